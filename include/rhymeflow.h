/*
 * rhymeflow.h -- C ABI of librhymeflow.so, the keyframe-query attention path
 * of RhymeFlow (asynchronous frame scheduling for video DiTs, arXiv 2606.06309)
 * on AMD Instinct MI355X (gfx950).
 *
 * At a denoising step where only keyframes are updated, the keyframes' query
 * tokens attend over the keys and values of every frame: the true states of
 * keyframes and the projected states of the skipped non-keyframes
 * (Sec. 3.2.3-3.2.4; App. B.2). This library provides the calls of that step:
 * keyframe-set normalisation, the latent trajectory projection of Eq. (3),
 * keyframe-query attention, and the frame gather/scatter around it; besides
 * them, the content-aware keyframe selection of Sec. 3.1 (frame similarity and
 * Alg. 1's scan), the per-layer rolling cache of App. B.2, whose projected
 * hidden states are the skipped frames' keys and values, and the progressive
 * asynchronous schedule (Eq. 2, Alg. 2) that says which step is which. Three
 * device probes, measurement support outside the method, report the rates the
 * matrix cores, LDS and HBM sustain on this device.
 *
 * Conventions shared by every call:
 *  - Return value: RF_OK (0) or a negative rf_status. No C++ exception crosses
 *    this ABI. rf_last_error() gives a thread-local description of the last
 *    failure on the calling thread.
 *  - Every argument is validated before any HIP call, so a rejected call has
 *    no effect on the device. The one HIP call that may come first is a query
 *    of the current device's compute-unit and XCD counts (bf16 attention and
 *    the plan queries with compute_units = 0), made once per device; a failed
 *    query returns RF_ERR_HIP.
 *  - Device buffers are owned by the caller, must stay alive until the stream
 *    has passed the launched work, and are never retained by the library.
 *    Host arrays are read during the call only; the caller may free them when
 *    the call returns. The library allocates no memory. The one piece of
 *    state that outlives a call, the rolling cache's bookkeeping, is a struct
 *    the caller owns and passes in.
 *  - `stream` is a hipStream_t (NULL = the default stream). Calls only enqueue
 *    work; they do not synchronise. Device faults surface at the caller's next
 *    synchronisation, not as a return code.
 *  - Calls may be made from several threads. The only state kept between
 *    calls is the per-device geometry above (read-only once queried).
 *  - Device pointers must be 16-byte aligned (128-bit accesses), otherwise
 *    RF_ERR_UNSUPPORTED, unless a call states a weaker requirement.
 */
#ifndef RHYMEFLOW_H
#define RHYMEFLOW_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RF_ABI_VERSION 2

/* Largest number of frames T a call accepts (keyframe ids travel inside the
   kernel arguments, which needs no device copy and no allocation). */
#define RF_MAX_FRAMES 256

/* Largest compute-unit count an attention plan query accepts. */
#define RF_MAX_COMPUTE_UNITS 65536

typedef enum {
    RF_OK = 0,
    RF_ERR_INVALID_ARG = -1,  /* NULL pointer, size <= 0, bad id list, NaN time */
    RF_ERR_UNSUPPORTED = -2,  /* valid request outside what the kernels cover */
    RF_ERR_RANGE = -3,        /* an id or size outside its range */
    RF_ERR_HIP = -4           /* the HIP runtime refused a launch */
} rf_status;

/* Element types; passed as int32_t. */
typedef enum { RF_BF16 = 0, RF_F32 = 1 } rf_dtype;

/* Flags of rf_select_keyframes. */
#define RF_SEL_NO_FORCE_FIRST 1u
/* Flags of rf_select_keyframes_adaptive. */
#define RF_SEL_INTENT_SIGN 1u

/* Name of a status code (static string). */
const char *rf_status_string(int status);
/* Description of the last failure on this thread ("" if none). */
const char *rf_last_error(void);
/* RF_ABI_VERSION of the loaded library. */
int rf_abi_version(void);

/*
 * Keyframe set from an explicit frame list (host only, integer, bit-exact).
 *
 * The keyframe set K is a set of frame indices; the first frame always belongs
 * to it, as the anchor of the video (Sec. 3.1; Alg. 1 starts K with the first
 * frame). Non-keyframes are the complement (Alg. 1).
 *
 * frame_ids [n_ids]: any order, duplicates allowed, each in [0, T).
 * T: frames, 1..RF_MAX_FRAMES.
 * flags: RF_SEL_NO_FORCE_FIRST leaves frame 0 out unless listed.
 * keyframe_ids_out [T capacity]: K sorted ascending, no duplicates.
 * num_keyframes_out: |K|.
 * keyframe_mask_out [T] (may be NULL): 1 for keyframes, 0 otherwise.
 * Errors: RF_ERR_INVALID_ARG (NULL outputs, n_ids < 0, frame_ids NULL with
 * n_ids > 0, empty result), RF_ERR_RANGE (an id outside [0, T) or T outside
 * 1..RF_MAX_FRAMES). Outputs are written only on success.
 */
int rf_select_keyframes(const int32_t *frame_ids, int32_t n_ids, int32_t T,
                        uint32_t flags, int32_t *keyframe_ids_out,
                        int32_t *num_keyframes_out, uint8_t *keyframe_mask_out);

/* Fixed-interval policy: frames 0, k, 2k, ... below T. ids_out has capacity T.
   Errors: RF_ERR_INVALID_ARG (NULL, k <= 0), RF_ERR_RANGE (T outside 1..RF_MAX_FRAMES). */
int rf_keyframes_stride(int32_t T, int32_t k, int32_t *ids_out, int32_t *n_out);

/* Evenly spaced policy ("Uniform" in the selection ablation, Sec. 4): M frames
   i*(T-1)/(M-1) rounded half up, i = 0..M-1, first and last included; M = 1
   gives frame 0. ids_out has capacity M.
   Errors: RF_ERR_INVALID_ARG (NULL), RF_ERR_RANGE (M outside 1..T, T outside
   1..RF_MAX_FRAMES). */
int rf_keyframes_uniform(int32_t T, int32_t M, int32_t *ids_out, int32_t *n_out);

/*
 * Latent trajectory projection, Eq. (3) (Sec. 3.2.4):
 *   z_hat(tau) = (1 - alpha) z(t_start) + alpha z(t_end),
 *   alpha = (t_start - tau) / (t_start - t_end),
 * for the non-keyframes; keyframes keep their current (true) state.
 *
 * latents: device [B][2][C][T][Hl][Wl], contiguous. Slot 0 holds z(t_start);
 *          slot 1 holds z(t_end) for non-keyframes and the current state for
 *          keyframes.
 * out:     device [B][C][T][Hl][Wl], contiguous. It may be exactly slot 1 of a
 *          single batch (B == 1, out == latents + C*T*Hl*Wl elements): keyframe
 *          planes are then left untouched. Any other overlap is an error.
 * timesteps: host {t_start, t_end, tau}, finite doubles (step indices or
 *          scheduler times; only their ratios matter). alpha is computed in
 *          double, kept inside [0, 1], and is 1 when t_start == t_end; it is
 *          then rounded once to float. Each element is evaluated as
 *          fmaf(alpha, z_end, (1 - alpha) * z_start) in fp32, so alpha = 0
 *          returns z_start and alpha = 1 returns z_end exactly.
 * keyframe_mask: host [T] bytes, nonzero = keyframe.
 * dtype:   RF_F32 or RF_BF16 storage for latents and out (fp32 arithmetic;
 *          bf16 results rounded to nearest even).
 * Errors: RF_ERR_INVALID_ARG (NULL, sizes <= 0, non-finite timesteps, partial
 *         overlap of out and latents), RF_ERR_RANGE (T > RF_MAX_FRAMES, sizes
 *         whose byte counts would pass 4e18), RF_ERR_UNSUPPORTED (unknown dtype,
 *         misaligned pointer), RF_ERR_HIP.
 */
int rf_project_latents(const void *latents, void *out, const double timesteps[3],
                       const uint8_t *keyframe_mask, int32_t B, int32_t C,
                       int32_t T, int32_t Hl, int32_t Wl, int32_t dtype,
                       void *stream);

/*
 * Keyframe-query attention (Sec. 3.2.3-3.2.4; App. B.2, attention at skipped
 * steps): the query rows are the N = H*W tokens of each keyframe; keys and
 * values are all S = T*N tokens of all frames. Per head,
 *   out = softmax(Q_kf K^T / sqrt(head_dim)) V,
 * with no mask. The query gather is fused: non-keyframe rows of q are never read.
 *
 * q, k, v: device [S][heads][head_dim], contiguous, token index
 *          f*N + y*W + x for frame f, row y, column x.
 * out:     device [M*N][heads][head_dim], contiguous; row r holds the query
 *          token keyframe_ids[r / N]*N + r % N (keyframe order). Must not
 *          overlap q, k or v.
 * keyframe_ids: host [M], strictly increasing, each in [0, T).
 * M = T with ids 0..T-1 is full 3D attention over all frames (warm-up steps
 * and Rhythmic Points, Sec. 3.2.1, 3.2.3).
 * head_dim: 64 or 128. dtype: RF_BF16 (bf16 inputs and output, bf16 matrix
 *          cores, fp32 softmax and accumulation, output rounded to nearest
 *          even) or RF_F32 (fp32 throughout, a correctness path).
 * Errors: RF_ERR_INVALID_ARG (NULL, sizes <= 0, ids not strictly increasing,
 *         out overlapping an input), RF_ERR_RANGE (an id outside [0, T), M > T,
 *         T > RF_MAX_FRAMES, sizes whose byte counts would pass 4e18),
 *         RF_ERR_UNSUPPORTED (head_dim, dtype, alignment), RF_ERR_HIP.
 */
int rf_keyframe_attention(const void *q, const void *k, const void *v, void *out,
                          const int32_t *keyframe_ids, int32_t M, int32_t T,
                          int32_t H, int32_t W, int32_t heads, int32_t head_dim,
                          int32_t dtype, void *stream);

/*
 * rf_keyframe_attention with a caller workspace for a split-key tail: one
 * bf16 workgroup of 256 query rows fills a compute unit, so ceil(M*N/256)*heads
 * workgroups run in whole rounds of the device's compute units (256 on
 * MI355X); the tiles beyond the last full round
 * are cut along the keys into parts that run side by side, and a second small
 * kernel combines each tile's parts (max of the parts' reference maxima,
 * rescaled sums, one bf16 rounding). Rows of split tiles differ from the
 * unsplit result only in fp32 summation order; which tiles are split depends
 * on the launch's size, so the row-for-row bitwise identity between launches
 * of different M that rf_keyframe_attention has does not hold here.
 *
 * workspace: device, 16-byte aligned, at least rf_attention_workspace bytes
 *   for the current device's compute units (compute_units = 0 there) (may be
 *   0: then nothing is split), not overlapping q, k, v or out; its
 *   contents are overwritten and meaningless afterwards. fp32 ignores it.
 * Other arguments and errors as rf_keyframe_attention; RF_ERR_INVALID_ARG also
 * for a NULL or too small workspace or an overlap.
 */
int rf_keyframe_attention_ws(const void *q, const void *k, const void *v, void *out,
                             const int32_t *keyframe_ids, int32_t M, int32_t T, int32_t H, int32_t W,
                             int32_t heads, int32_t head_dim, int32_t dtype, void *workspace,
                             int64_t workspace_bytes, void *stream);

/*
 * rf_keyframe_attention_ws without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc). The split-key tail's partial
 * results go to a static device array of RF_NOALLOC_SCRATCH_BYTES that the
 * library holds on every GPU it runs on until the process ends; the call
 * allocates nothing. Results equal rf_keyframe_attention_ws's bit for bit (the
 * same plan and kernels).
 *
 * Shapes whose split-key tail needs more than RF_NOALLOC_SCRATCH_BYTES on the
 * current device (rf_attention_workspace with compute_units = 0) are refused
 * with RF_ERR_RANGE; at 256 compute units that is only the case for
 * launches past about 200 tail tiles at head_dim 128, none of the paper's
 * shapes. All calls on one GPU share its array: two calls that overlap in time
 * on one GPU (different streams or threads) race on it, so serialise them.
 * The first call on each device looks up the array's device address (a HIP
 * query); a failure there returns RF_ERR_HIP.
 * Arguments and other errors as rf_keyframe_attention.
 */
#define RF_NOALLOC_SCRATCH_BYTES (160LL << 20)
int rf_keyframe_attention_noalloc(const void *q, const void *k, const void *v, void *out,
                                  const int32_t *keyframe_ids, int32_t M, int32_t T, int32_t H, int32_t W,
                                  int32_t heads, int32_t head_dim, int32_t dtype, void *stream);

/*
 * Bytes of workspace rf_keyframe_attention_ws (Mkv = T) or rf_frame_attention
 * (Mkv key/value frames) uses for these sizes on a device of compute_units
 * compute units (0 when nothing is split, always 0 for RF_F32). The split-key
 * tail fills the compute units a round of whole tiles leaves idle, so the plan
 * depends on their number: the launch uses the current device's count.
 * compute_units: 1..RF_MAX_COMPUTE_UNITS (host only, no HIP call), or 0 for the
 *   current device's count (queried once per device; 256 on MI355X).
 * Errors: RF_ERR_INVALID_ARG (NULL, sizes <= 0), RF_ERR_RANGE (T, M, Mkv,
 *         compute_units, sizes whose byte counts would pass 4e18),
 *         RF_ERR_UNSUPPORTED (head_dim, dtype), RF_ERR_HIP (compute_units = 0
 *         and no device to query).
 */
int rf_attention_workspace(int32_t M, int32_t Mkv, int32_t T, int32_t H, int32_t W, int32_t heads,
                           int32_t head_dim, int32_t dtype, int32_t compute_units, int64_t *bytes_out);

/* How a bf16 attention launch is cut (rf_attention_plan). A tile is 256 query
   rows of one head and runs as one workgroup filling one compute unit. */
typedef struct rf_attention_split {
    int64_t tiles;              /* ceil(M*N / 256) * heads */
    int64_t whole_tiles;        /* tiles computed over all keys in one workgroup */
    int64_t tail_tiles;         /* tiles past the last full round, cut along the keys */
    int32_t parts;              /* parts per tail tile (0: nothing is split) */
    int32_t key_tiles_per_part; /* key tiles per part (64 keys each; 128 at head_dim 64) */
    int64_t workspace_bytes;    /* tail_tiles * parts * 256 * (4 * head_dim + 8) */
    int32_t compute_units;      /* the count the plan is made for */
    int32_t reserved;
} rf_attention_split;

/*
 * The split plan rf_keyframe_attention_ws / rf_frame_attention use for these
 * sizes on compute_units compute units (arguments and errors as
 * rf_attention_workspace). For RF_F32 every count is 0 (no split).
 */
int rf_attention_plan(int32_t M, int32_t Mkv, int32_t T, int32_t H, int32_t W, int32_t heads, int32_t head_dim,
                      int32_t dtype, int32_t compute_units, rf_attention_split *plan_out);

/*
 * Attention under a frame-level key/value mask: the frame mask M_Rhyme (in
 * the Discussions, a per-step frame mask that can be multiplied with a token
 * mask) with one key set for all query frames. The query rows are the tokens
 * of frames q_frames, as in rf_keyframe_attention; the keys and values are the
 * tokens of frames kv_frames only, every other key being masked out:
 *   out = softmax(Q_q K_kv^T / sqrt(head_dim)) V_kv.
 * kv_frames = the keyframes gives the keyframe-only attention of Sec. 4's
 * ablations ("w/ keyframe-only attention"; "w/o projection", where keyframes
 * attend to the synchronised frames only). Masked frames' keys and values are
 * never read. The kernel walks the listed frames in key tiles that do not
 * cross a frame, so when N is not a multiple of 64 each frame's last tile is
 * partly idle.
 *
 * kv_frames [Mkv]: strictly increasing, each in [0, T), 1 <= Mkv <= T (Mkv = T
 * is rf_keyframe_attention). workspace / workspace_bytes: as
 * rf_keyframe_attention_ws, or NULL for no split. All other arguments,
 * layouts and errors as rf_keyframe_attention (q_frames / Mq are its
 * keyframe_ids / M).
 */
int rf_frame_attention(const void *q, const void *k, const void *v, void *out,
                       const int32_t *q_frames, int32_t Mq, const int32_t *kv_frames, int32_t Mkv,
                       int32_t T, int32_t H, int32_t W, int32_t heads, int32_t head_dim,
                       int32_t dtype, void *workspace, int64_t workspace_bytes, void *stream);

/*
 * Frame gather: dst_compact[m*N + n] = src_full[frame_ids[m]*N + n] for rows
 * of row_bytes bytes, N = rows_per_frame; every frame is one contiguous block
 * of N rows (the token layout of a frame-major sequence, App. B.1: S = F x N).
 * A bit-exact copy; standalone form of the query gather fused into
 * rf_keyframe_attention.
 *
 * src_full: device, T*N rows. dst_compact: device, M*N rows; no overlap.
 * frame_ids: host [M], strictly increasing, each in [0, T).
 * row_bytes: a multiple of 16.
 * Errors: RF_ERR_INVALID_ARG, RF_ERR_RANGE (ids, T, rows_per_frame * row_bytes *
 *         RF_MAX_FRAMES past 4e18), RF_ERR_UNSUPPORTED (alignment,
 *         row_bytes % 16), RF_ERR_HIP.
 */
int rf_gather_frames(const void *src_full, void *dst_compact,
                     const int32_t *frame_ids, int32_t M, int32_t T,
                     int64_t rows_per_frame, int64_t row_bytes, void *stream);

/*
 * Frame scatter, the inverse of rf_gather_frames: writes the keyframe rows of
 * a compact attention output back to their token positions,
 * dst_full[frame_ids[m]*N + n] = src_compact[m*N + n]. Rows of frames not
 * listed are left untouched (their outputs come from elsewhere, App. B.2).
 * Same arguments and errors as rf_gather_frames.
 */
int rf_scatter_frames(const void *src_compact, void *dst_full,
                      const int32_t *frame_ids, int32_t M, int32_t T,
                      int64_t rows_per_frame, int64_t row_bytes, void *stream);

/*
 * Cosine similarity between latent frames (content-aware keyframe selection,
 * Sec. 3.1: Eq. (1) compares a frame with the most recent keyframe by cosine
 * similarity; Alg. 1 computes it on the frames' clean-latent proxies).
 *
 * latents: device, [B][C][T][H][W] contiguous, RF_F32 or RF_BF16 (the proxies,
 *          e.g. a single-step clean-latent prediction; supplied by the caller).
 *          The vector of frame f of batch element b is its C*H*W elements.
 * sim_out: device, [B][T][T] doubles:
 *          sim[b][i][j] = <x_i, x_j> / (max(|x_i|, 1e-8) * max(|x_j|, 1e-8)),
 *          products and sums in double precision (a frame with zero norm has
 *          similarity 0 to every frame).
 * workspace: device scratch of at least workspace_bytes bytes, as returned by
 *          rf_frame_similarity_workspace for the same sizes; its contents are
 *          overwritten and are meaningless afterwards. It must not overlap
 *          latents or sim_out.
 * T: 1..RF_MAX_FRAMES. latents and workspace 16-byte aligned, sim_out 8-byte.
 * The result is deterministic (fixed-order reductions).
 * Errors: RF_ERR_INVALID_ARG (NULL, sizes <= 0, overlap, workspace too small),
 *         RF_ERR_RANGE (T), RF_ERR_UNSUPPORTED (dtype, alignment), RF_ERR_HIP.
 */
int rf_frame_similarity(const void *latents, double *sim_out, void *workspace,
                        int64_t workspace_bytes, int32_t B, int32_t C, int32_t T,
                        int32_t H, int32_t W, int32_t dtype, void *stream);

/*
 * Bytes of device workspace rf_frame_similarity needs for these sizes
 * (host only). Errors: RF_ERR_INVALID_ARG, RF_ERR_RANGE (T).
 */
int rf_frame_similarity_workspace(int32_t B, int32_t C, int32_t T, int32_t H, int32_t W,
                                  int64_t *bytes_out);

/*
 * Dynamic sequential keyframe selection (Alg. 1; Eq. 1) on a frame similarity
 * matrix (host only; the decisions are integer).
 *
 * The first frame seeds the set and is the first reference. Frames i = 1..T-1
 * are visited in order while fewer than M are selected; frame i joins when
 * sim[i][last] < tau, with `last` the most recent keyframe (strict <). On each
 * selection, the gap g = i - last is compared with L_avg = T / M (real
 * division): g >= L_avg + delta_up lowers tau by dtau, g <= L_avg - delta_down
 * raises it (Alg. 1 as printed). RF_SEL_INTENT_SIGN swaps the two adjustments
 * (the prose calls the large-gap adjustment encouraging, which under the
 * rule sim < tau is a raise).
 *
 * sim: host, [T][T] doubles, row-major (only sim[i][last] entries are read).
 * T: 1..RF_MAX_FRAMES. M: 1..T. tau, dtau, delta_up, delta_down: finite.
 * keyframe_ids_out: host, capacity T; *num_keyframes_out = selected count;
 * keyframe_mask_out: host [T] or NULL.
 * Errors: RF_ERR_INVALID_ARG (NULL, non-finite parameter, unknown flag),
 *         RF_ERR_RANGE (T, M).
 */
int rf_select_keyframes_adaptive(const double *sim, int32_t T, double tau, int32_t M,
                                 double dtau, double delta_up, double delta_down, uint32_t flags,
                                 int32_t *keyframe_ids_out, int32_t *num_keyframes_out,
                                 uint8_t *keyframe_mask_out);

/*
 * Per-layer rolling cache of post-attention hidden states (App. B.2).
 *
 * For each cached frame f (the non-keyframes, fixed when the keyframe set is
 * frozen at the end of warm-up) one layer's cache keeps two hidden states,
 * h_before and h_after, each the frame's N = rows_per_frame attention-output
 * rows of D = hidden elements (D = heads * head_dim), with their timesteps
 * t_before >= t_after. Diffusion timesteps decrease as denoising proceeds.
 *
 * The states live in a caller-owned device buffer `store` of 2 * n_cached
 * frame slots; slot s starts at store + s * frame_bytes (frame_bytes =
 * N * D * element size), and the i-th cached frame (in increasing frame order)
 * owns slots 2i and 2i+1. This host struct, also owned by the caller, records
 * which of the two slots holds which state: moving h_after into h_before at a
 * denoising step is a change of slot index, not a copy. The struct is plain
 * data: the calls below read and update it on the host when they are made, so
 * work enqueued on different streams must be ordered by the caller (the
 * projection reads the slots its call named; a later shift_store rewrites one
 * of them).
 */
typedef struct rf_rolling_cache {
    int32_t T;                  /* frames of the video, 1..RF_MAX_FRAMES */
    int32_t n_cached;           /* cached frames, 1..T */
    int64_t rows_per_frame;     /* N */
    int32_t hidden;             /* D */
    int32_t dtype;              /* RF_BF16 or RF_F32 */
    int64_t frame_bytes;        /* N * D * element size */
    uint32_t magic;             /* set by rf_cache_init */
    int32_t reserved;
    int16_t before_slot[RF_MAX_FRAMES];  /* slot of h_before of frame f, -1 if f is not cached */
    int16_t after_slot[RF_MAX_FRAMES];   /* slot of h_after of frame f, -1 if f is not cached */
    double t_before[RF_MAX_FRAMES];
    double t_after[RF_MAX_FRAMES];
} rf_rolling_cache;

/* Bytes of device store a cache of n_cached frames needs (host only):
   2 * n_cached * rows_per_frame * hidden * element size.
   Errors: RF_ERR_INVALID_ARG (NULL, sizes <= 0), RF_ERR_RANGE (n_cached >
   RF_MAX_FRAMES, size overflow), RF_ERR_UNSUPPORTED (dtype). */
int rf_cache_store_bytes(int32_t n_cached, int64_t rows_per_frame, int32_t hidden, int32_t dtype,
                         int64_t *bytes_out);

/*
 * Initialisation at the end of warm-up (step t_w): h_before = h_after = the
 * frame's attention output at t_w, t_before = t_after = t_w (App. B.2).
 *
 * cache: host struct, overwritten. frames [n]: the frames to cache, strictly
 * increasing, each in [0, T), 1 <= n <= T. Frame frames[i] gets slots 2i and
 * 2i+1; both of its indices point at slot 2i.
 * h_full: device [T*N][D] of dtype (the attention output of all frames at t_w,
 *   frame-major), or NULL to set up the bookkeeping only, the caller then
 *   writing slot 2i itself. When h_full is given, the rows of every listed
 *   frame are copied into its slot 2i of `store` (device, 16-byte aligned, at
 *   least rf_cache_store_bytes bytes, not overlapping h_full); store is not
 *   read when h_full is NULL.
 * hidden * element size must be a multiple of 16. t_w: finite.
 * Errors: RF_ERR_INVALID_ARG (NULL cache, bad frame list, sizes <= 0,
 *   non-finite t_w, overlap), RF_ERR_RANGE, RF_ERR_UNSUPPORTED (dtype,
 *   alignment, row size), RF_ERR_HIP. On error the struct is left unchanged.
 */
int rf_cache_init(rf_rolling_cache *cache, void *store, const void *h_full,
                  const int32_t *frames, int32_t n, int32_t T, int64_t rows_per_frame,
                  int32_t hidden, int32_t dtype, double t_w, void *stream);

/*
 * Shift-and-store at a denoising step (a Rhythmic Point) t_denoise (App. B.2):
 * for each listed frame, h_before <- h_after and t_before <- t_after (slot
 * indices only), then h_after <- the frame's new attention output, stored in
 * the frame's other slot, and t_after <- t_denoise.
 *
 * frames [n]: cached frames, strictly increasing; frames == NULL (n ignored)
 *   means every cached frame, the synchronised update of App. B.2.
 * h_full: device [T*N][D] (this step's attention output of all frames), or
 *   NULL to update the bookkeeping only (the caller then writes each frame's
 *   new after slot itself, before the next projection reads it).
 * t_denoise: finite and strictly below every listed frame's t_after.
 * Errors: RF_ERR_INVALID_ARG (NULL or uninitialised cache, a frame not cached,
 *   list not increasing, t_denoise not below t_after, overlap), RF_ERR_RANGE,
 *   RF_ERR_UNSUPPORTED (alignment), RF_ERR_HIP. On error the struct is left
 *   unchanged.
 */
int rf_cache_shift_store(rf_rolling_cache *cache, void *store, const void *h_full,
                         const int32_t *frames, int32_t n, double t_denoise, void *stream);

/*
 * The interpolation weight of frame f at t_skip (host only):
 *   alpha = (t_before - t_skip) / (t_before - t_after + 1e-8),
 * in double, kept inside [0, 1]. Right after initialisation (t_before =
 * t_after) any earlier step clamps to 1; both slots then hold one state.
 * Errors: RF_ERR_INVALID_ARG (NULL, uninitialised cache, f not cached,
 *   non-finite t_skip), RF_ERR_RANGE (f outside [0, T)).
 */
int rf_cache_alpha(const rf_rolling_cache *cache, int32_t frame, double t_skip, double *alpha_out);

/*
 * Keys and values of the cached frames at a skipped step t_skip (App. B.2):
 * for each listed frame f,
 *   h_hat = (1 - alpha_f) h_before + alpha_f h_after   (alpha_f from rf_cache_alpha),
 * evaluated per element as fmaf(alpha_f, h_after, (1 - alpha_f) * h_before) in
 * fp32 with alpha_f rounded once to float (bf16 results rounded to nearest
 * even), and written to the frame's rows of both k and v: the projected hidden
 * state serves as the frame's key and its value. Rows of other frames are not
 * touched; the keyframes' rows keep the keys and values the caller computed.
 *
 * store: the cache's device store. k, v: device [T*N][D] of the cache's dtype
 *   (D = heads * head_dim, the layout rf_keyframe_attention reads), 16-byte
 *   aligned, overlapping neither each other nor the store.
 * frames [n]: cached frames, strictly increasing; NULL means every cached frame.
 * Errors: RF_ERR_INVALID_ARG (NULL, uninitialised cache, a frame not cached,
 *   list not increasing, non-finite t_skip, overlap), RF_ERR_UNSUPPORTED
 *   (alignment), RF_ERR_HIP.
 */
int rf_cache_project_kv(const rf_rolling_cache *cache, const void *store, void *k, void *v,
                        const int32_t *frames, int32_t n, double t_skip, void *stream);

/*
 * Keyframe-query attention at a skipped step with the cached frames' projected
 * states as their keys and values, formed inside the attention kernel (App. B.2,
 * attention computation at skipped steps: every cached non-keyframe's key and
 * value are h = (1 - alpha) h_before + alpha h_after, alpha as in
 * rf_cache_alpha at t_skip). The result equals rf_cache_project_kv(cache, store,
 * k, v, NULL, 0, t_skip) followed by rf_keyframe_attention_ws on the modified k
 * and v, up to fp32 summation order, but k and v are neither written nor read
 * for cached frames: a key tile of a cached frame loads the frame's two cached
 * states and forms the projected tile in LDS (fp32 fmaf(alpha, h_after,
 * (1 - alpha) h_before), rounded once to bf16, as rf_cache_project_kv does). The
 * key loop walks frames in frame-aligned tiles (a frame's last tile partial when
 * N is not a multiple of the key tile).
 *
 * cache: initialised (rf_cache_init) for T frames of H*W rows of heads*head_dim
 *   elements in bf16; every cached frame is projected, the others take k and v.
 * store: the cache's device store (rf_cache_store_bytes bytes), 16-byte
 *   aligned, not overlapping out.
 * workspace / workspace_bytes: as rf_keyframe_attention_ws (the same plan and
 *   size, rf_attention_workspace with Mkv = T).
 * dtype: RF_BF16 only (RF_ERR_UNSUPPORTED otherwise).
 * Other arguments and errors as rf_keyframe_attention_ws; RF_ERR_INVALID_ARG
 * also for a cache that is not initialised, inconsistent, or of another shape
 * or dtype, a NULL store and a non-finite t_skip.
 */
int rf_keyframe_attention_cached(const void *q, const void *k, const void *v, void *out,
                                 const int32_t *keyframe_ids, int32_t M, int32_t T, int32_t H, int32_t W,
                                 int32_t heads, int32_t head_dim, int32_t dtype, const rf_rolling_cache *cache,
                                 const void *store, double t_skip, void *workspace, int64_t workspace_bytes,
                                 void *stream);

/*
 * Progressive asynchronous schedule (Eq. 2; Alg. 2), host only.
 *
 * For the denoising steps t = T down to 1: the first T_w steps (t > T - T_w)
 * are the synchronous warm-up, every frame taking one step with full
 * attention. Afterwards the keyframes take one step at every t, and the
 * non-keyframes, which all share one schedule, take a step of
 * n_skip(t) = n_small if T_mid < t <= T - T_w, n_large if t <= T_mid (Eq. 2),
 * stopping at 0, whenever their state time equals t. Such a step is a
 * Rhythmic Point: every frame is updated and attends over every frame. At the
 * other steps they are skipped: only the keyframes' queries are evaluated and
 * the non-keyframes' states at t are projected with Eq. (3) on the interval
 * they are crossing. Following the non-keyframes' state time gives Alg. 2's
 * test (T - T_w - t) mod n_skip == 0 whenever the stride does not change
 * between two of their updates, and stays consistent when it does.
 */
#define RF_STEP_WARMUP 0     /* every frame one step, full attention */
#define RF_STEP_RHYTHMIC 1   /* every frame updated, full attention; non-keyframes jump n_skip */
#define RF_STEP_SKIP 2       /* keyframes only, keyframe-query attention over projected non-keyframes */

typedef struct rf_step_plan {
    int32_t t;          /* the step: the time keyframes are at before it (T down to 1) */
    int32_t phase;      /* RF_STEP_WARMUP, RF_STEP_RHYTHMIC or RF_STEP_SKIP */
    int32_t n_skip;     /* Eq. (2) at t; 1 during warm-up */
    int32_t nonkey_to;  /* warm-up and Rhythmic Points: the time the non-keyframes reach
                           (t - 1, resp. max(t - n_skip, 0)); -1 at skipped steps */
    int32_t t_start;    /* skipped steps: the time the non-keyframes last left (Eq. 3's t_start); else -1 */
    int32_t t_end;      /* skipped steps: the time they reached (Eq. 3's t_end); else -1 */
    double alpha;       /* skipped steps: (t_start - t) / (t_start - t_end) in double, in (0, 1); else 0 */
} rf_step_plan;

/*
 * T: steps, 1..2^20. T_w, T_mid: 0..T. n_small, n_large: >= 1 (the paper uses
 * n_small < n_large, e.g. 2 and 3, with T_mid = T/2).
 * plan_out: host [T] records, step T first. n_rhythmic_out, n_skipped_out
 * (either may be NULL): counts of Rhythmic Points and of skipped steps.
 * Errors: RF_ERR_INVALID_ARG (NULL plan, a stride < 1), RF_ERR_RANGE (T, T_w, T_mid).
 */
int rf_async_schedule(int32_t T, int32_t T_w, int32_t T_mid, int32_t n_small, int32_t n_large,
                      rf_step_plan *plan_out, int32_t *n_rhythmic_out, int32_t *n_skipped_out);

/* ---- Device probes (measurement support, not part of the method) ----
 * Sustained whole-chip rates of this device under a pure load of one kind, to
 * set a kernel's achieved rate against what the device delivers besides the
 * published peaks (MI355X: dense bf16 matrix 2.5 PFLOP/s at 2.4 GHz, HBM3E
 * 8 TB/s); the chip runs below that clock when all matrix cores are busy.
 * Each enqueues one kernel on `stream` and returns at once; time them with
 * events on that stream.
 */

/*
 * Dense bf16 matrix cores: each of the workgroups' 4 waves runs 4 independent
 * accumulator chains of 32x32x16 bf16 matrix multiply-accumulates (fp32
 * accumulators), `rounds` rounds of 8 steps each. FLOP per launch:
 * workgroups * rounds * 2^22.
 * operands: device bf16 [12][64][8], 16-byte aligned: lane l holds A operands
 * i = 0..5 (operands[i][l][0..7]) and B operands (operands[6 + i][l][0..7]);
 * step u (0..7) of chain j adds A[(u + 2j) % 6] B[(3u + j) % 6], where an A
 * operand is the 32x16 matrix whose element (m, k) lane m + 32 (k / 8) holds
 * at k % 8, a B operand the 16x32 matrix whose element (k, n) lane
 * n + 32 (k / 8) holds at k % 8. Random operands make the matrix cores draw
 * the power of a real product; small integers make the result exact. The
 * kernel fits four waves on every SIMD.
 * sink: device float [workgroups * 256], 4-byte aligned; thread i of a wave
 * (lane l) writes the sum of its 64 accumulators, accumulator r of chain j
 * being element (8 (r / 4) + 4 (l / 32) + r % 4, l % 32) of chain j's product.
 * workgroups 1..2^20 (4 per compute unit give MI355X's 256 CUs 4 waves per
 * SIMD), rounds 1..2^22. Errors: RF_ERR_INVALID_ARG (NULL), RF_ERR_RANGE
 * (workgroups, rounds), RF_ERR_UNSUPPORTED (alignment).
 */
int rf_probe_mfma_bf16(const void *operands, int32_t workgroups, int32_t rounds, float *sink, void *stream);

/*
 * LDS reads: each of a workgroup's 4 waves reads the workgroup's 64 KB LDS
 * array (32-bit word i holds i * 2654435761 mod 2^32) in full `rounds` times,
 * with 16-byte reads (width 16) or with the transposing 8-byte reads of 16-bit
 * elements (width 8, the form that reads V^T operands for the matrix cores).
 * Width 16: round r reads the 64 rows of 1 KB in order, lane l at bytes
 * 16 ((l + r) % 64) .. +16 of each. Width 8: the array is 256 rows of 256
 * bytes; read t (0..127) of round r gives lane 16h + 4q + e (h, q, e = 0..3)
 * the 8 bytes at row 8 (t / 4) + 4 (h / 2) + q, byte
 * 32 ((2 ((t + r) % 4) + h % 2) XOR 2q) + 8e, which the hardware redistributes
 * within each group of 16 lanes (the layout the attention kernel reads V tiles
 * in). 64 KB of LDS per workgroup puts two workgroups on a compute unit.
 * Bytes per launch: workgroups * 4 * rounds * 65536.
 * sink: device uint32 [workgroups * 256], 4-byte aligned. Width 16: thread i
 * (lane l) writes the sum mod 2^32 of the 32-bit words it read. Width 8: a
 * thread writes the XOR of the 32-bit words it received; over a group of 16
 * lanes, that XOR folded to 16 bits (low half XOR high half) is the XOR of the
 * 16-bit elements the group addressed.
 * ticks: NULL, or device uint64 [workgroups], 8-byte aligned: the shader-clock
 * ticks (s_memtime) each workgroup spent between the barriers around its reads.
 * workgroups 1..2^20, rounds 1..2^22. Errors: RF_ERR_INVALID_ARG (NULL sink,
 * width), RF_ERR_RANGE (workgroups, rounds), RF_ERR_UNSUPPORTED (alignment).
 */
int rf_probe_lds_read(int32_t workgroups, int32_t rounds, int32_t width, uint32_t *sink, uint64_t *ticks,
                      void *stream);

/*
 * HBM reads: the workgroups read the device buffer src of `bytes` bytes once
 * (16-byte words, streaming loads): workgroup w of 1024 threads reads the
 * contiguous run of words [w P, (w + 1) P), P = ceil(words / workgroups), and
 * writes the XOR of the 32-bit words it read to sink[w], so the XOR of
 * sink[0 .. workgroups) is the XOR of every 32-bit word of src. Bytes per
 * launch: `bytes`. Runs of about 2 MB (workgroups = bytes / 2^21) read fastest
 * on MI355X.
 * src: 16-byte aligned, bytes a positive multiple of 16. sink: device
 * uint32 [workgroups], 4-byte aligned. workgroups 1..2^20.
 * Errors: RF_ERR_INVALID_ARG (NULL, bytes), RF_ERR_RANGE (workgroups),
 * RF_ERR_UNSUPPORTED (alignment).
 */
int rf_probe_hbm_read(const void *src, int64_t bytes, int32_t workgroups, uint32_t *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* RHYMEFLOW_H */
