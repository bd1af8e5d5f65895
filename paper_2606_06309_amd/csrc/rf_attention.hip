// Keyframe-query attention for gfx950 (CDNA4).
//
// Method (Sec. 3.2.3-3.2.4; App. B.2): at a step where only keyframes are
// denoised, the query tokens of the M keyframes attend over the keys and
// values of all T frames. Per head: out = softmax(Q_kf K^T / sqrt(d)) V.
//
// bf16 kernel design:
//  * A workgroup of 8 waves owns one (head, 256-row query tile); each wave
//    owns 32 query rows. Query rows are gathered straight from the keyframe
//    tokens (row r reads token kf[r / N] * N + r % N), so the gather is fused
//    and non-keyframe query rows are never read.
//  * Scores are computed transposed, S^T = K Q^T, with
//    v_mfma_f32_32x32x16_bf16: K rows are the A operand (from LDS), the
//    wave's query rows the B operand (held in registers for the whole loop).
//    In the 32x32 accumulator layout every lane then holds 16 scores of ONE
//    query column, so the softmax max and sum are in-lane reductions plus one
//    exchange with the lane 32 apart.
//  * The probabilities are already in the B-operand layout of the second
//    product, O^T = V^T P^T: the lane's 16 accumulators become two bf16x8
//    operands without any data movement. The V^T A operands are read from
//    the natural [key][dim] V tile with transposing LDS reads; the key order
//    inside an operand follows the accumulator layout (a reduction index may
//    be permuted freely as long as both operands agree).
//  * K and V tiles (64 keys; 128 at head dimension 64) go from HBM straight into LDS (buffer loads
//    with an LDS destination: no staging registers, no LDS write
//    instructions), double-buffered so the next tile streams in while the
//    current one is computed; the buffer range check zero-fills keys >= S and
//    the last tile masks their scores.
//  * Online softmax in the log2 domain with fp32 state, taken against a
//    reference that is a past row maximum: the row maximum of a tile is only
//    computed when the tile's row sum shows that a probability outgrew the
//    reference (first tile, or a jump by a factor of ~256), so the common tile
//    costs no max reduction. P is rounded to bf16 for the matrix cores and the
//    row sum adds those same rounded values.
//  * Workgroup ids are mapped XCD-aware: consecutive ids go round-robin to the
//    device's X XCDs (8 on MI355X), so tile = (id % X) * per_xcd + id / X gives
//    each XCD a contiguous, head-major range of tiles and the workgroups
//    resident on one XCD stream the same head's K/V through that XCD's L2.
//  * Split-key tail (when the caller provides a workspace): one workgroup
//    fills a CU, so a launch of n tiles runs in ceil(n / CUs) rounds (256 CUs
//    on MI355X; the count is queried from the device) and the
//    last round may leave most CUs idle. The tiles beyond the last full round
//    are then split along the keys into parts that run as extra workgroups;
//    each part writes its unnormalised (O, m, l) in fp32, and a small kernel
//    combines the parts of a tile (max of the references, rescaled sums).
//  * Frame-level key/value mask (the frame-list form): the key loop walks a list
//    of frames in key tiles that never cross a frame; masked frames are
//    never read.
//  * Projected keys and values at a skipped step (the cache form; App. B.2):
//    the key loop walks all frames in frame-aligned tiles; a tile of a cached
//    frame loads that frame's two cached hidden states h_before and h_after
//    instead of K and V, and the workgroup forms
//    h = fmaf(alpha, h_after, (1 - alpha) h_before), rounded once to bf16, in
//    LDS as both the key tile and the value tile, so the projected keys and
//    values are never written to HBM.
// The fp32 kernel at the end is a plain correctness path (fp32 throughout).
#include <atomic>

#include "rf_internal.h"

namespace rf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Data moves as 32-bit words; bf16 vectors are only ever formed by a
// whole-vector bitcast of a u32x4 (or of one scalar word) right before the
// instruction that consumes them.

// Tunables (compile-time): waves per workgroup (each owns 32 query rows), keys
// per LDS tile (at head dimension 128, and at 64), the largest row partial sum of a tile accepted before the
// softmax reference is rebased (so every probability stays below it), and how
// many LDS fragments the matrix core reads ahead.
#ifndef RF_ATTN_WAVES
#define RF_ATTN_WAVES 8
#endif
#ifndef RF_ATTN_BC
#define RF_ATTN_BC 64
#endif
#ifndef RF_ATTN_BC64
#define RF_ATTN_BC64 128
#endif
#ifndef RF_ATTN_REBASE_BOUND
#define RF_ATTN_REBASE_BOUND 256.0f
#endif
#ifndef RF_ATTN_K_LEAD
#define RF_ATTN_K_LEAD 4
#endif
#ifndef RF_ATTN_V_LEAD
#define RF_ATTN_V_LEAD 3
#endif

constexpr int kWaves = RF_ATTN_WAVES;
constexpr int kThreads = 64 * kWaves;
constexpr int kBr = 32 * kWaves;   // query rows per workgroup
// Keys per LDS tile. At head dimension 64 a tile of 64 keys carries half the
// matrix work of one at 128 for the same softmax, barrier and loop overhead, so
// it takes twice the keys (the registers and LDS that head dimension leaves free
// hold them).
__host__ __device__ constexpr int key_tile(int head_dim) { return head_dim == 64 ? RF_ATTN_BC64 : RF_ATTN_BC; }
// Split-key tail: the most parts a tail tile is cut into and the fewest key
// tiles a part may have. A round of whole tiles fills the device's compute
// units (one workgroup per CU), queried at launch.
constexpr int kMaxSplit = 8;
constexpr int kMinKvPerSplit = 8;
constexpr float kRebaseBound = RF_ATTN_REBASE_BOUND;   // largest tile row sum kept without a rebase
static_assert(key_tile(64) % 32 == 0 && key_tile(128) % 32 == 0, "key tile must be a multiple of 32");

struct AttnKArgs {
    const uint16_t *q;
    const uint16_t *k;
    const uint16_t *v;
    uint16_t *out;
    int64_t S;
    int64_t N;
    int64_t Mq;
    int32_t heads;
    int32_t n_qtiles;
    int32_t total_tiles;    // tiles computed whole (all tiles when there is no split)
    int32_t per_xcd;
    int32_t xcds;           // XCDs of the device: workgroup id i runs on XCD i % xcds
    int32_t grid_direct;    // workgroups of the whole tiles (per_xcd * xcds)
    int32_t split;          // parts per tail tile (0: no split)
    int32_t kv_per_split;   // key tiles per part
    float *ws_o;            // [tail tile * split + part][kBr][D] unnormalised O
    float *ws_ml;           // [tail tile * split + part][kBr][2] reference max (log2 domain), row sum
    float scale_log2;   // log2(e) / sqrt(d)
    int32_t kf[kMaxFrames];
    // key/value frame list (frame-masked form only): the keys are the tokens
    // of frames kvf[0..n_kv), walked frame by frame in tiles that never cross
    // a frame (tiles_per_frame = ceil(N / key tile); a frame's last tile is partial)
    int32_t n_kv;
    int32_t tiles_per_frame;
    // frame-list form: the listed frames; cache form (all T frames walked): per
    // frame the two cache slots (h_before | h_after << 16), or -1 when the frame
    // takes its keys and values from k and v
    int32_t kvf[kMaxFrames];
    const uint16_t *store;           // cache form: [slot][N][heads][head_dim] cached hidden states
    float calpha[kMaxFrames];        // cache form: each cached frame's weight alpha
};

// Kernel arguments travel in the kernarg segment: keep them within 4 KB.
static_assert(sizeof(AttnKArgs) <= 4096, "attention kernel arguments exceed 4 KB");

// Forms of the bf16 kernel's key loop.
constexpr int kFormDense = 0;    // all S tokens in order
constexpr int kFormFrames = 1;   // the tokens of the listed frames a.kvf
constexpr int kFormCache = 2;    // all frames; cached frames give projected keys = values

// Word 3 of a raw (untyped, stride 0) buffer resource on gfx9-class GPUs.
constexpr int kBufferWord3 = 0x00020000;

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// A pointer every lane holds the same value of, rebuilt from its first lane.
__device__ __forceinline__ void *uniform_ptr(const void *p) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
    return reinterpret_cast<void *>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Two floats -> two bf16 (round to nearest even) packed low-first in a word.
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
    const bf16x2_t v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ inline bf16x8_t as_bf16x8(u32x4_t w) { return __builtin_bit_cast(bf16x8_t, w); }

// lo + hi of a packed bf16 pair, accumulated in fp32 (v_dot2 against (1, 1)).
__device__ __forceinline__ float add_bf16x2(uint32_t word, float acc) {
    const bf16x2_t one = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, word), one, acc, false);
}

// Combine the values of lanes l and l ^ 32 with one VALU swap of the wave
// halves: r[0] holds lanes 0..31 in both halves, r[1] lanes 32..63.
__device__ __forceinline__ float halves_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS tile layout. A tile holds kBc keys of one head, K and V each in natural
// [key][dim] order with unpadded rows of 2*D bytes, so that the global->LDS
// loads can write whole 1 KB wave-chunks at consecutive addresses (lane l of a
// load lands at chunk + 16 l). Bank conflicts on the reads are removed by
// permuting the 16-byte slots of each row with an XOR of a key-dependent mask:
//   K: slot = chunk ^ kswz(key) makes the 16 lanes of one 128-bit read pass
//      (16 consecutive keys, same chunk) hit 16 different slot positions of
//      the 256-byte bank window;
//   V: slot = chunk ^ vswz(key) makes the 32 lanes of one transposing 64-bit
//      read pass (4 keys x 64 bytes) hit 8 different 32-byte positions.
template <int D>
struct TileLayout {
    static constexpr int kBc = key_tile(D);            // keys per tile
    static constexpr int kRow = 2 * D;                 // bytes per key row
    static constexpr int kSlots = kRow / 16;           // 16-byte slots per row
    static constexpr int kRowsPerWin = 256 / kRow;     // rows per 256-byte bank window
    static constexpr int kTileBytes = kBc * kRow;
    static constexpr int kRowsPerLoad = 1024 / kRow;   // rows one wave-wide 16-byte load fills
    static constexpr int kLoads = kTileBytes / 1024;   // wave-wide loads per tensor per tile
    __host__ __device__ static constexpr int kswz(int key) { return (key / kRowsPerWin) % kSlots; }
    __host__ __device__ static constexpr int vswz(int key) { return 4 * ((key / kRowsPerWin) % (kSlots / 4)); }
};

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

// 16 bytes per lane from a buffer resource straight into LDS: lane l's bytes
// land at dst + 16 l; offsets at or past the resource's range read as zero.
// (Kept out of the kernel template: the host pass drops the launch stub of a
// template that names this builtin.)
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t r, lds_void_t *dst, int voffset) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voffset, 0, 0, 0);
}

// S^T = K Q^T for one tile of kNB 32-key blocks. kofs[kk] is this lane's byte
// offset of its K fragment for reduction step kk inside block 0. The K
// fragments are read through a ring RF_ATTN_K_LEAD fragments ahead of the
// matrix core; the scheduling groups pin that order: LEAD reads, then
// (1 MFMA, 1 read) pairs, then the last LEAD MFMAs.
template <int D, int kNB>
__device__ __forceinline__ void scores_tile(const uint8_t *kb, const int (&kofs)[D / 16],
                                            const u32x4_t (&qf)[D / 16], f32x16_t (&sacc)[kNB]) {
    constexpr int kSteps = D / 16;
    constexpr int kNF = kNB * kSteps;
    constexpr int kLead = RF_ATTN_K_LEAD < kNF ? RF_ATTN_K_LEAD : kNF;
    u32x4_t ring[kLead];
    auto rd = [&](int i) {
        const int b = i / kSteps, kk = i % kSteps;
        return *reinterpret_cast<const u32x4_t *>(kb + kofs[kk] + b * 32 * TileLayout<D>::kRow);
    };
#pragma unroll
    for (int i = 0; i < kLead; ++i) ring[i] = rd(i);
#pragma unroll
    for (int i = 0; i < kNF; ++i) {
        const int b = i / kSteps, kk = i % kSteps;
        const f32x16_t c = kk == 0 ? f32x16_t{} : sacc[b];
        sacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(ring[i % kLead]), as_bf16x8(qf[kk]), c,
                                                          0, 0, 0);
        if (i + kLead < kNF) ring[i % kLead] = rd(i + kLead);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, kLead, 0);
#pragma unroll
    for (int i = 0; i < kNF - kLead; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kLead, 0);
}

// One A operand of O^T = V^T P^T: dims db*32 + (lane % 32) of the 16 keys
// c*16 .. c*16+15, in the key order of the probability operand (elements 0..3:
// keys c*16 + grp*4 + 0..3, elements 4..7: keys c*16 + 8 + grp*4 + 0..3).
// Each half is one transposing read: the 16 lanes of a group fetch 8 bytes of
// 4 key rows and the hardware redistributes them so lane i receives dim i of
// all four keys.
template <int D>
__device__ __forceinline__ u32x4_t vt_operand(const uint8_t *vb, int vofs, int c) {
    constexpr int kRow = TileLayout<D>::kRow;
    const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4_t *)(vb + vofs + c * 16 * kRow));
    const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4_t *)(vb + vofs + (c * 16 + 8) * kRow));
    const u32x2_t l2 = __builtin_bit_cast(u32x2_t, lo), h2 = __builtin_bit_cast(u32x2_t, hi);
    return __builtin_shufflevector(l2, h2, 0, 1, 2, 3);
}

// O^T += V^T P^T for one tile; operands are read RF_ATTN_V_LEAD ahead.
template <int D, int kNB>
__device__ __forceinline__ void pv_tile(const uint8_t *vb, const int (&vofs)[D / 32],
                                        const u32x4_t (&pw)[2 * kNB], f32x16_t (&oacc)[D / 32]) {
    constexpr int kNF = 2 * kNB * (D / 32);
    constexpr int kLead = RF_ATTN_V_LEAD < kNF ? RF_ATTN_V_LEAD : kNF;
    u32x4_t ring[kLead];
    auto rd = [&](int i) {
        const int c = i / (D / 32), db = i % (D / 32);
        return vt_operand<D>(vb, vofs[db], c);
    };
#pragma unroll
    for (int i = 0; i < kLead; ++i) ring[i] = rd(i);
#pragma unroll
    for (int i = 0; i < kNF; ++i) {
        const int c = i / (D / 32), db = i % (D / 32);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(ring[i % kLead]), as_bf16x8(pw[c]),
                                                           oacc[db], 0, 0, 0);
        if (i + kLead < kNF) ring[i % kLead] = rd(i + kLead);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * kLead, 0);
#pragma unroll
    for (int i = 0; i < kNF - kLead; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kLead, 0);
}

// Per-tile pipeline, double-buffered LDS, one barrier per tile:
//   issue the global->LDS loads of tile t+1 into the buffer tile t-1 used
//   math on tile t
//   wait for this wave's loads, barrier (tile t+1 visible, tile t released)
// The loads go through raw buffer resources rebased per tile in scalar
// registers whose range ends at the tile's last valid key, so the hardware
// range check zero-fills the keys past it (keys >= S, or past the end of a
// frame in the frame-masked form) and their scores are masked. The loop is
// unrolled by two so every LDS access names its buffer statically.
// kForm: kFormDense, kFormFrames (the keys are the tokens of the frames a.kvf,
// a frame-level mask) or kFormCache (every frame, cached frames projected).
template <int D, int kForm>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
void attn_bf16_kernel(const AttnKArgs a) {
    constexpr bool kKvList = kForm != kFormDense;   // frame-aligned tiles
    using L = TileLayout<D>;
    constexpr int kBc = L::kBc;
    constexpr int kNB = kBc / 32;                       // 32-key score blocks per tile
    constexpr int kLoadsPerWave = L::kLoads / kWaves;
    static_assert(L::kLoads % kWaves == 0, "tile loads must split evenly over the waves");

    __shared__ __attribute__((aligned(1024))) uint8_t k0[L::kTileBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t k1[L::kTileBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t v0[L::kTileBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t v1[L::kTileBytes];

    const int bid = blockIdx.x;
    int tile, part = -1;
    if (bid < a.grid_direct) {
        tile = (bid % a.xcds) * a.per_xcd + bid / a.xcds;
        if (tile >= a.total_tiles) return;
    } else {   // a part of a tail tile (tail tiles follow the whole ones in tile order)
        const int u = bid - a.grid_direct;
        const int tt = u / a.split;
        part = u - tt * a.split;
        tile = a.total_tiles + tt;
    }
    const int head = tile / a.n_qtiles;
    const int qt = tile - head * a.n_qtiles;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 31, grp = lane >> 5;
    const int64_t rs = static_cast<int64_t>(a.heads) * D;   // token stride in elements

    // ---- query fragments: B operand of S^T = K Q^T (fused keyframe gather) ----
    const int64_t row = static_cast<int64_t>(qt) * kBr + wave * 32 + col;
    u32x4_t qf[D / 16];
    if (row < a.Mq) {
        const int64_t f = row / a.N;
        const int64_t tok = static_cast<int64_t>(a.kf[f]) * a.N + (row - f * a.N);
        const uint16_t *qp = a.q + tok * rs + static_cast<int64_t>(head) * D + grp * 8;
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) qf[kk] = *reinterpret_cast<const u32x4_t *>(qp + kk * 16);
    } else {
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) qf[kk] = u32x4_t{0u, 0u, 0u, 0u};
    }

    // ---- per-lane offsets, fixed for the whole loop ----
    // global byte offsets (from the tile's first key) of this lane's 16 bytes in each load
    int kgo[kLoadsPerWave], vgo[kLoadsPerWave];
#pragma unroll
    for (int i = 0; i < kLoadsPerWave; ++i) {
        const int key = (wave * kLoadsPerWave + i) * L::kRowsPerLoad + lane / L::kSlots;
        const int slot = lane % L::kSlots;
        kgo[i] = static_cast<int>(key * rs * 2) + (slot ^ L::kswz(key)) * 16;
        vgo[i] = static_cast<int>(key * rs * 2) + (slot ^ L::vswz(key)) * 16;
    }
    // LDS byte offsets of the K fragment (block 0, step kk) and of the V^T operand halves
    int kofs[D / 16], vofs[D / 32];
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) kofs[kk] = col * L::kRow + (((2 * kk) ^ grp ^ L::kswz(col)) * 16);
    {
        const int g16 = (lane >> 4) & 1, j = lane & 15;
        const int rr = grp * 4 + j / 4;   // key row within each 8-key half of a 16-key group
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
            vofs[db] = rr * L::kRow + (((2 * db + g16) ^ (L::vswz(rr) / 2)) * 32) + 8 * (j % 4);
    }

    f32x16_t oacc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] = 0.0f;
    // m_run: reference max (log2 domain) the probabilities are taken against
    // (a past row maximum; see the softmax below).
    float m_run = -__builtin_huge_valf();
    float l_run = 0.0f;   // this lane's partial row sum

    const uint16_t *kbase = a.k + static_cast<int64_t>(head) * D;
    const uint16_t *vbase = a.v + static_cast<int64_t>(head) * D;
    // bytes from a head's first element to one past the last element it owns
    const int64_t head_bytes = ((a.S - 1) * rs + D) * 2;

    // Tile t: its first key's token, the bytes from there to the end of its last
    // valid key, and the number of valid keys (at most kBc).
    // Cache form: slots >= 0 for a tile of a cached frame (before | after << 16),
    // its rows' offset inside the frame and the frame's weight.
    struct Geom {
        int64_t tok0, left;
        int32_t valid;
        int32_t slots;
        int64_t frame_off;
        float alpha;
    };
    auto geom = [&](int64_t t) {
        Geom g;
        g.slots = -1;
        g.frame_off = 0;
        g.alpha = 0.0f;
        if constexpr (kKvList) {
            const int32_t m = static_cast<int32_t>(t) / a.tiles_per_frame;
            const int64_t o = (t - static_cast<int64_t>(m) * a.tiles_per_frame) * kBc;
            if constexpr (kForm == kFormCache) {
                g.tok0 = static_cast<int64_t>(m) * a.N + o;
                g.slots = a.kvf[m];
                g.frame_off = o;
                g.alpha = a.calpha[m];
            } else {
                g.tok0 = static_cast<int64_t>(a.kvf[m]) * a.N + o;
            }
            g.valid = static_cast<int32_t>(a.N - o < kBc ? a.N - o : kBc);
            g.left = ((g.valid - 1) * rs + D) * 2;
        } else {
            g.tok0 = t * kBc;
            g.left = head_bytes - g.tok0 * rs * 2;
            g.valid = static_cast<int32_t>(a.S - g.tok0 < kBc ? a.S - g.tok0 : kBc);
        }
        return g;
    };

    auto issue = [&](const Geom &g, uint8_t *kdst, uint8_t *vdst) {
        // The resources start at the tile's first key; their range ends at its last valid
        // key (clamped to 2^31 - 1: a tile never reaches that far past its first key).
        const int32_t rec = __builtin_amdgcn_readfirstlane(
            static_cast<int32_t>(g.left < 0x7fffffffLL ? g.left : 0x7fffffffLL));
        if constexpr (kForm == kFormCache) {
            if (g.slots >= 0) {
                // a cached frame: h_before into the key buffer, h_after into the value
                // buffer, both in the key layout (project_tile then writes both tiles)
                const uint16_t *hb = a.store + ((g.slots & 0xffff) * a.N + g.frame_off) * rs + head * D;
                const uint16_t *ha = a.store + ((g.slots >> 16) * a.N + g.frame_off) * rs + head * D;
                const __amdgpu_buffer_rsrc_t br =
                    __builtin_amdgcn_make_buffer_rsrc(uniform_ptr(hb), 0, rec, kBufferWord3);
                const __amdgpu_buffer_rsrc_t ar =
                    __builtin_amdgcn_make_buffer_rsrc(uniform_ptr(ha), 0, rec, kBufferWord3);
#pragma unroll
                for (int i = 0; i < kLoadsPerWave; ++i) {
                    const int chunk = (wave * kLoadsPerWave + i) * 1024;
                    load_lds16(br, (lds_void_t *)(kdst + chunk), kgo[i]);
                    load_lds16(ar, (lds_void_t *)(vdst + chunk), kgo[i]);
                }
                return;
            }
        }
        const __amdgpu_buffer_rsrc_t kr =
            __builtin_amdgcn_make_buffer_rsrc(uniform_ptr(kbase + g.tok0 * rs), 0, rec, kBufferWord3);
        const __amdgpu_buffer_rsrc_t vr =
            __builtin_amdgcn_make_buffer_rsrc(uniform_ptr(vbase + g.tok0 * rs), 0, rec, kBufferWord3);
#pragma unroll
        for (int i = 0; i < kLoadsPerWave; ++i) {
            const int chunk = (wave * kLoadsPerWave + i) * 1024;
            load_lds16(kr, (lds_void_t *)(kdst + chunk), kgo[i]);
            load_lds16(vr, (lds_void_t *)(vdst + chunk), vgo[i]);
        }
    };

    // Cache form: the projected state of a cached frame's tile, formed in LDS.
    // The key buffer holds h_before and the value buffer h_after, both in the key
    // layout; each wave owns whole key rows (kBc / 8 of them), reads its rows' 16-byte
    // slots of both, and writes h = fmaf(alpha, h_after, (1 - alpha) h_before),
    // rounded once to bf16, back into the key buffer at the same slot and into the
    // value buffer at the slot the value layout puts it. A wave's LDS instructions
    // run in order and no other wave touches its rows, so its reads see the loaded
    // states before its writes replace them. The caller's barrier then publishes
    // both tiles.
    auto project_tile = [&](uint8_t *kb, uint8_t *vb, float alpha) {
        constexpr int kRowsPerWave = kBc / kWaves;
        constexpr int kPerLane = kRowsPerWave * L::kSlots / 64;
        static_assert(kRowsPerWave * L::kSlots % 64 == 0, "a wave's rows must split evenly over its lanes");
        const float oma = 1.0f - alpha;
        u32x4_t hv[kPerLane];
        int pk[kPerLane], pv[kPerLane];
#pragma unroll
        for (int i = 0; i < kPerLane; ++i) {
            const int sidx = lane * kPerLane + i;
            const int key = wave * kRowsPerWave + sidx / L::kSlots;
            const int slot = sidx % L::kSlots;
            pk[i] = key * L::kRow + (slot ^ L::kswz(key)) * 16;
            pv[i] = key * L::kRow + (slot ^ L::vswz(key)) * 16;
            const u32x4_t b = *reinterpret_cast<const u32x4_t *>(kb + pk[i]);
            const u32x4_t af = *reinterpret_cast<const u32x4_t *>(vb + pk[i]);
            u32x4_t h;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float lo = fmaf(alpha, __uint_as_float(af[e] << 16), oma * __uint_as_float(b[e] << 16));
                const float hi = fmaf(alpha, __uint_as_float(af[e] & 0xffff0000u),
                                      oma * __uint_as_float(b[e] & 0xffff0000u));
                h[e] = pack_bf16x2(lo, hi);
            }
            hv[i] = h;
        }
#pragma unroll
        for (int i = 0; i < kPerLane; ++i) {
            *reinterpret_cast<u32x4_t *>(kb + pk[i]) = hv[i];
            *reinterpret_cast<u32x4_t *>(vb + pv[i]) = hv[i];
        }
    };
    // after a tile's loads are visible: form the projected tile if the frame is cached
    auto settle_tile = [&](const Geom &g, uint8_t *kb, uint8_t *vb) {
        if constexpr (kForm == kFormCache) {
            if (g.slots >= 0) {
                project_tile(kb, vb, g.alpha);
                __syncthreads();
            }
        }
    };

    const float sl2 = a.scale_log2;
    auto compute = [&](int32_t valid, const uint8_t *kb, const uint8_t *vb) {
        // ---- S^T = K Q^T : 32-key blocks ----
        f32x16_t sacc[kNB];
        scores_tile<D, kNB>(kb, kofs, qf, sacc);
        // accumulator r of block b holds key b*32 + (r/4)*8 + grp*4 + r%4 for query `col`
        if (valid < kBc) {
#pragma unroll
            for (int b = 0; b < kNB; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = b * 32 + (r / 4) * 8 + grp * 4 + (r % 4);
                    if (key >= valid) sacc[b][r] = -__builtin_huge_valf();
                }
        }

        // ---- online softmax (log2 domain), reference max moved only when needed ----
        // p = exp2(s * scale - m_run) against the current reference m_run. The
        // reference is a past row maximum, so p may exceed 1; that is harmless (O / l
        // does not depend on the reference and floating-point relative precision does
        // not depend on scale) until p grows large. The row sum bounds every p of the
        // tile, so a row whose tile sum exceeds kRebaseBound takes the exact
        // path: this tile's row maximum becomes the reference, O and l are
        // rescaled and P is recomputed. The first tile (m_run = -inf gives
        // p = inf) always takes it; afterwards it is rare.
        u32x4_t pw[2 * kNB];
        auto probs = [&]() {
            // probabilities, packed as the B operand of O^T = V^T P^T:
            // operand c takes accumulators 8*(c%2) .. 8*(c%2)+7 of block c/2.
            // The row sum adds the bf16-rounded values the matrix core consumes,
            // in four independent partial sums (a single chain of dependent adds
            // would hold up the end of the softmax).
            float lsp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int b = 0; b < kNB; ++b)
#pragma unroll
                for (int r = 0; r < 16; r += 2) {
                    const float p0 = fast_exp2(fmaf(sacc[b][r], sl2, -m_run));
                    const float p1 = fast_exp2(fmaf(sacc[b][r + 1], sl2, -m_run));
                    const uint32_t word = pack_bf16x2(p0, p1);
                    lsp[(r / 2) % 4] = add_bf16x2(word, lsp[(r / 2) % 4]);
                    pw[b * 2 + r / 8][(r % 8) / 2] = word;
                }
            return ((lsp[0] + lsp[1]) + lsp[2]) + lsp[3];
        };
        float ls = probs();
        // decided per query row (its two lanes agree), so a row's result depends on
        // its own scores only, whichever rows share the wave
        if (!(halves_sum(ls) <= kRebaseBound)) {   // rare; both lanes of a row take it
            float mx = -__builtin_huge_valf();
#pragma unroll
            for (int b = 0; b < kNB; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[b][r]);
            const float m_new = fmaxf(m_run, halves_max(mx) * sl2);
            const float corr = fast_exp2(m_run - m_new);   // 0 on the first tile
            m_run = m_new;
            l_run *= corr;
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int r = 0; r < 16; ++r) oacc[db][r] *= corr;
            ls = probs();
        }
        l_run += ls;

        // ---- O^T += V^T P^T ----
        pv_tile<D, kNB>(vb, vofs, pw, oacc);
    };
    auto tile_done = [&]() {
        __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0): this wave's loads have reached LDS
        __syncthreads();
    };

    const int64_t ntiles = kKvList ? static_cast<int64_t>(a.n_kv) * a.tiles_per_frame : (a.S + kBc - 1) / kBc;
    int64_t t_begin = 0, t_end = ntiles;
    if (part >= 0) {
        t_begin = static_cast<int64_t>(part) * a.kv_per_split;
        t_end = t_begin + a.kv_per_split < ntiles ? t_begin + a.kv_per_split : ntiles;
    }
    Geom cur = geom(t_begin);
    issue(cur, k0, v0);
    tile_done();
    settle_tile(cur, k0, v0);
    for (int64_t t = t_begin; t < t_end; t += 2) {
        Geom nxt = cur;
        if (t + 1 < t_end) {
            nxt = geom(t + 1);
            issue(nxt, k1, v1);
        }
        compute(cur.valid, k0, v0);
        tile_done();
        if (t + 1 >= t_end) break;
        // (a projected tile is formed while no load is in flight, so its barrier
        // waits for nothing but the projection itself)
        settle_tile(nxt, k1, v1);
        if (t + 2 < t_end) {
            cur = geom(t + 2);
            issue(cur, k0, v0);
        }
        compute(nxt.valid, k1, v1);
        tile_done();
        if (t + 2 < t_end) settle_tile(cur, k0, v0);
    }

    l_run = halves_sum(l_run);
    if (part >= 0) {
        // ---- a part of a tail tile: unnormalised O and (m, l) for the combine kernel ----
        if (row < a.Mq) {
            const int64_t slot = static_cast<int64_t>(tile - a.total_tiles) * a.split + part;
            const int64_t r = slot * kBr + wave * 32 + col;
            float *po = a.ws_o + r * D;
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4) {
                    const int rr = g4 * 4;
                    *reinterpret_cast<f32x4_t *>(po + db * 32 + g4 * 8 + grp * 4) =
                        f32x4_t{oacc[db][rr], oacc[db][rr + 1], oacc[db][rr + 2], oacc[db][rr + 3]};
                }
            if (grp == 0) *reinterpret_cast<f32x2_t *>(a.ws_ml + r * 2) = f32x2_t{m_run, l_run};
        }
        return;
    }

    // ---- epilogue: normalise, round to bf16, store the compact row ----
    if (row < a.Mq) {
        const float inv = 1.0f / l_run;
        uint16_t *op = a.out + row * rs + static_cast<int64_t>(head) * D;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
                // accumulator r holds dimension db*32 + (r/4)*8 + grp*4 + r%4
                const int r = g4 * 4;
                const u32x2_t w = {pack_bf16x2(oacc[db][r] * inv, oacc[db][r + 1] * inv),
                                   pack_bf16x2(oacc[db][r + 2] * inv, oacc[db][r + 3] * inv)};
                *reinterpret_cast<u32x2_t *>(op + db * 32 + g4 * 8 + grp * 4) = w;
            }
    }
}

// ---------------------------------------------------------------------------
// Combine of the split tail: for each row of a tail tile, the parts' reference
// maxima m_p (log2 domain), row sums l_p and unnormalised outputs O_p give
//   m = max_p m_p,  out = sum_p 2^(m_p - m) O_p / sum_p 2^(m_p - m) l_p,
// rounded to bf16. Each thread owns 8 output dimensions of one row.
// ---------------------------------------------------------------------------

struct CombineArgs {
    const float *ws_o;
    const float *ws_ml;
    uint16_t *out;
    int64_t Mq;
    int32_t heads;
    int32_t n_qtiles;
    int32_t first_tail;   // tile index of the first tail tile
    int32_t split;
};

constexpr int kCombineThreads = 256;

template <int D>
__global__ __launch_bounds__(kCombineThreads) void attn_combine_kernel(const CombineArgs a) {
    constexpr int kTpr = D / 8;                       // threads per row
    constexpr int kRows = kCombineThreads / kTpr;     // rows per workgroup
    constexpr int kGroups = kBr / kRows;              // workgroups per tail tile
    const int tt = blockIdx.x / kGroups;
    const int r = (blockIdx.x - tt * kGroups) * kRows + threadIdx.x / kTpr;
    const int c8 = threadIdx.x % kTpr;
    const int tile = a.first_tail + tt;
    const int head = tile / a.n_qtiles;
    const int qt = tile - head * a.n_qtiles;
    const int64_t row = static_cast<int64_t>(qt) * kBr + r;
    if (row >= a.Mq) return;
    const int64_t base = static_cast<int64_t>(tt) * a.split * kBr + r;   // slot of part 0 of this row
    float m = -__builtin_huge_valf();
    for (int p = 0; p < a.split; ++p) m = fmaxf(m, a.ws_ml[(base + static_cast<int64_t>(p) * kBr) * 2]);
    float l = 0.0f, o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = 0.0f;
    for (int p = 0; p < a.split; ++p) {
        const int64_t slot = base + static_cast<int64_t>(p) * kBr;
        const f32x2_t ml = *reinterpret_cast<const f32x2_t *>(a.ws_ml + slot * 2);
        const float wgt = fast_exp2(ml[0] - m);
        l = fmaf(wgt, ml[1], l);
        const f32x4_t *po = reinterpret_cast<const f32x4_t *>(a.ws_o + slot * D + c8 * 8);
        const f32x4_t x0 = po[0], x1 = po[1];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            o[e] = fmaf(wgt, x0[e], o[e]);
            o[e + 4] = fmaf(wgt, x1[e], o[e + 4]);
        }
    }
    const float inv = 1.0f / l;
    const int64_t rs = static_cast<int64_t>(a.heads) * D;
    const u32x4_t w = {pack_bf16x2(o[0] * inv, o[1] * inv), pack_bf16x2(o[2] * inv, o[3] * inv),
                       pack_bf16x2(o[4] * inv, o[5] * inv), pack_bf16x2(o[6] * inv, o[7] * inv)};
    *reinterpret_cast<u32x4_t *>(a.out + row * rs + static_cast<int64_t>(head) * D + c8 * 8) = w;
}

// ---------------------------------------------------------------------------
// fp32 path: a correctness path with fp32 arithmetic throughout. A workgroup
// of 128 lanes owns 64 query rows of one head; each row is shared by two
// adjacent lanes that each hold half of the head dimension.
// ---------------------------------------------------------------------------

constexpr int kF32Rows = 64;
constexpr int kF32Keys = 32;

struct AttnF32Args {
    const float *q;
    const float *k;
    const float *v;
    float *out;
    int64_t S;
    int64_t N;
    int64_t Mq;
    int32_t heads;
    float scale;       // 1 / sqrt(d)
    int32_t kf[kMaxFrames];
    int32_t n_kv;      // > 0: the keys are the tokens of frames kvf[0..n_kv), S = n_kv * N
    int32_t kvf[kMaxFrames];
};

template <int D>
__global__ __launch_bounds__(2 * kF32Rows) void attn_f32_kernel(const AttnF32Args a) {
    constexpr int HD = D / 2;
    __shared__ float ks[kF32Keys][D];
    __shared__ float vs[kF32Keys][D];
    const int head = blockIdx.y;
    const int tid = threadIdx.x;
    const int half = tid & 1;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * kF32Rows + (tid >> 1);
    const int64_t rs = static_cast<int64_t>(a.heads) * D;

    float qv[HD], o[HD];
    if (row < a.Mq) {
        const int64_t f = row / a.N;
        const int64_t tok = static_cast<int64_t>(a.kf[f]) * a.N + (row - f * a.N);
        const float *qp = a.q + tok * rs + static_cast<int64_t>(head) * D + half * HD;
#pragma unroll
        for (int c = 0; c < HD; ++c) qv[c] = qp[c];
    } else {
#pragma unroll
        for (int c = 0; c < HD; ++c) qv[c] = 0.0f;
    }
#pragma unroll
    for (int c = 0; c < HD; ++c) o[c] = 0.0f;
    float m = -__builtin_huge_valf(), l = 0.0f;

    for (int64_t j0 = 0; j0 < a.S; j0 += kF32Keys) {
        __syncthreads();
        for (int i = tid; i < kF32Keys * D; i += 2 * kF32Rows) {
            const int key = i / D, c = i % D;
            const int64_t j = j0 + key;
            int64_t tok = j;
            if (a.n_kv > 0 && j < a.S) {
                const int64_t m = j / a.N;
                tok = static_cast<int64_t>(a.kvf[m]) * a.N + (j - m * a.N);
            }
            const int64_t off = tok * rs + static_cast<int64_t>(head) * D + c;
            ks[key][c] = j < a.S ? a.k[off] : 0.0f;
            vs[key][c] = j < a.S ? a.v[off] : 0.0f;
        }
        __syncthreads();
        float s[kF32Keys];
        float mt = -__builtin_huge_valf();
#pragma unroll
        for (int jj = 0; jj < kF32Keys; ++jj) {
            float part = 0.0f;
#pragma unroll
            for (int c = 0; c < HD; ++c) part = fmaf(qv[c], ks[jj][half * HD + c], part);
            const float dot = part + __shfl_xor(part, 1);
            s[jj] = (j0 + jj < a.S) ? dot * a.scale : -__builtin_huge_valf();
            mt = fmaxf(mt, s[jj]);
        }
        const float m_new = fmaxf(m, mt);
        const float corr = expf(m - m_new);
        l *= corr;
#pragma unroll
        for (int c = 0; c < HD; ++c) o[c] *= corr;
#pragma unroll
        for (int jj = 0; jj < kF32Keys; ++jj) {
            const float p = expf(s[jj] - m_new);
            l += p;
#pragma unroll
            for (int c = 0; c < HD; ++c) o[c] = fmaf(p, vs[jj][half * HD + c], o[c]);
        }
        m = m_new;
    }
    if (row < a.Mq) {
        float *op = a.out + row * rs + static_cast<int64_t>(head) * D + half * HD;
        const float inv = 1.0f / l;
#pragma unroll
        for (int c = 0; c < HD; ++c) op[c] = o[c] * inv;
    }
}

}  // namespace

hipError_t device_geometry(DeviceGeometry *out) {
    constexpr int kMaxDevices = 64;
    static std::atomic<int64_t> cached[kMaxDevices];   // (cus << 32 | xcds), 0 until queried
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    int64_t v = cached[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        int cus = 0, xcds = 0;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        e = hipDeviceGetAttribute(&xcds, hipDeviceAttributeNumberOfXccs, dev);
        if (e != hipSuccess || xcds < 1) xcds = 1;   // no XCD count reported: one L2 domain
        if (cus < 1) return hipErrorInvalidDevice;
        if (xcds > cus) xcds = cus;
        v = (static_cast<int64_t>(cus) << 32) | static_cast<uint32_t>(xcds);
        cached[dev].store(v, std::memory_order_relaxed);
    }
    out->cus = static_cast<int32_t>(v >> 32);
    out->xcds = static_cast<int32_t>(v & 0xffffffff);
    return hipSuccess;
}

AttnSplit attention_split(int64_t Mq, int32_t heads, int32_t head_dim, int64_t N, int64_t S, int32_t n_kv,
                          int32_t cus, int32_t walk_frames) {
    AttnSplit sp{};
    const int64_t total = (Mq + kBr - 1) / kBr * heads;
    const int64_t kBc = key_tile(head_dim);
    const int64_t kv_tiles = n_kv > 0 ? static_cast<int64_t>(n_kv) * ((N + kBc - 1) / kBc) : (S + kBc - 1) / kBc;
    const int64_t tail = total % cus;
    sp.n_tiles = total;
    sp.n_direct = total;
    if (tail == 0) return sp;
    // tail time in rounds of whole tiles for s parts: ceil(tail * s / CUs) / s
    int best_s = 1;
    double best = 1.0;
    for (int s = 2; s <= kMaxSplit && kv_tiles / s >= kMinKvPerSplit; ++s) {
        const double cost = static_cast<double>((tail * s + cus - 1) / cus) / s;
        if (cost < best - 1e-9) {
            best = cost;
            best_s = s;
        }
    }
    if (best_s == 1) return sp;
    sp.n_direct = total - tail;
    sp.n_tail = tail;
    sp.split = best_s;
    // a frame-aligned walk has at least as many key tiles, so its parts keep >= kMinKvPerSplit
    const int64_t walk = walk_frames > 0 ? static_cast<int64_t>(walk_frames) * ((N + kBc - 1) / kBc) : kv_tiles;
    sp.kv_per_split = (walk + best_s - 1) / best_s;
    sp.ws_bytes = tail * best_s * kBr * (static_cast<int64_t>(head_dim) * 4 + 8);
    return sp;
}

hipError_t launch_attention(const AttnParams &p, hipStream_t stream) {
    const int64_t Mq = static_cast<int64_t>(p.M) * p.N;
    if (p.dtype == RF_BF16) {
        AttnKArgs a{};
        a.q = static_cast<const uint16_t *>(p.q);
        a.k = static_cast<const uint16_t *>(p.k);
        a.v = static_cast<const uint16_t *>(p.v);
        a.out = static_cast<uint16_t *>(p.out);
        a.S = p.S;
        a.N = p.N;
        a.Mq = Mq;
        a.heads = p.heads;
        const int64_t nq = (Mq + kBr - 1) / kBr;
        const int32_t xcds = p.geo.xcds;
        if (p.geo.cus < 1 || xcds < 1 || xcds > 64) return hipErrorInvalidValue;
        AttnSplit sp{};
        sp.n_direct = nq * p.heads;
        const int32_t walk = p.cache_form ? static_cast<int32_t>(p.S / p.N) : 0;
        if (p.ws) {
            sp = attention_split(Mq, p.heads, p.head_dim, p.N, p.S, p.n_kv, p.geo.cus, walk);
            if (sp.split > 0 && p.ws_bytes < sp.ws_bytes) return hipErrorInvalidValue;
        }
        const int64_t total = sp.n_direct;
        const int64_t per_xcd = (total + xcds - 1) / xcds;
        if (nq * p.heads > 0x7fffffffLL / 64) return hipErrorInvalidConfiguration;
        // per-lane load offsets inside a tile are 32-bit: a tile's token rows must span < 2 GiB
        const int64_t kBc = key_tile(p.head_dim);
        if (static_cast<int64_t>(p.heads) * p.head_dim * 2 * kBc >= 0x7fffffffLL) return hipErrorInvalidConfiguration;
        a.n_qtiles = static_cast<int32_t>(nq);
        a.total_tiles = static_cast<int32_t>(total);
        a.per_xcd = static_cast<int32_t>(per_xcd);
        a.xcds = xcds;
        a.grid_direct = static_cast<int32_t>(per_xcd * xcds);
        a.split = static_cast<int32_t>(sp.split);
        a.kv_per_split = static_cast<int32_t>(sp.kv_per_split);
        const int64_t n_parts = sp.n_tail * sp.split;
        if (sp.split > 0) {
            a.ws_o = static_cast<float *>(p.ws);
            a.ws_ml = a.ws_o + n_parts * kBr * p.head_dim;
        }
        a.scale_log2 = static_cast<float>(1.4426950408889634 / sqrt(static_cast<double>(p.head_dim)));
        for (int i = 0; i < p.M; ++i) a.kf[i] = p.kf[i];
        a.n_kv = p.n_kv;
        a.tiles_per_frame = static_cast<int32_t>((p.N + kBc - 1) / kBc);
        for (int i = 0; i < p.n_kv; ++i) a.kvf[i] = p.kvf[i];
        if (p.cache_form) {
            a.n_kv = walk;
            for (int i = 0; i < walk; ++i) {
                a.kvf[i] = p.cslot[i];
                a.calpha[i] = p.calpha[i];
            }
            a.store = static_cast<const uint16_t *>(p.store);
        }
        if (a.n_kv > 0 && static_cast<int64_t>(a.n_kv) * a.tiles_per_frame > 0x7fffffffLL)
            return hipErrorInvalidConfiguration;
        const dim3 grid(static_cast<uint32_t>(per_xcd * xcds + n_parts)), block(kThreads);
        if (p.cache_form) {
            if (p.head_dim == 128) hipLaunchKernelGGL((attn_bf16_kernel<128, kFormCache>), grid, block, 0, stream, a);
            else hipLaunchKernelGGL((attn_bf16_kernel<64, kFormCache>), grid, block, 0, stream, a);
        } else if (p.n_kv > 0) {
            if (p.head_dim == 128) hipLaunchKernelGGL((attn_bf16_kernel<128, kFormFrames>), grid, block, 0, stream, a);
            else hipLaunchKernelGGL((attn_bf16_kernel<64, kFormFrames>), grid, block, 0, stream, a);
        } else {
            if (p.head_dim == 128) hipLaunchKernelGGL((attn_bf16_kernel<128, kFormDense>), grid, block, 0, stream, a);
            else hipLaunchKernelGGL((attn_bf16_kernel<64, kFormDense>), grid, block, 0, stream, a);
        }
        if (sp.split == 0) return hipGetLastError();
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        CombineArgs c{};
        c.ws_o = a.ws_o;
        c.ws_ml = a.ws_ml;
        c.out = a.out;
        c.Mq = Mq;
        c.heads = p.heads;
        c.n_qtiles = a.n_qtiles;
        c.first_tail = a.total_tiles;
        c.split = a.split;
        const int rows_per_wg = kCombineThreads / (p.head_dim / 8);
        const dim3 cgrid(static_cast<uint32_t>(sp.n_tail * (kBr / rows_per_wg))), cblock(kCombineThreads);
        if (p.head_dim == 128) hipLaunchKernelGGL(attn_combine_kernel<128>, cgrid, cblock, 0, stream, c);
        else hipLaunchKernelGGL(attn_combine_kernel<64>, cgrid, cblock, 0, stream, c);
        return hipGetLastError();
    }
    AttnF32Args a{};
    a.q = static_cast<const float *>(p.q);
    a.k = static_cast<const float *>(p.k);
    a.v = static_cast<const float *>(p.v);
    a.out = static_cast<float *>(p.out);
    a.S = p.S;
    a.N = p.N;
    a.Mq = Mq;
    a.heads = p.heads;
    a.scale = static_cast<float>(1.0 / sqrt(static_cast<double>(p.head_dim)));
    for (int i = 0; i < p.M; ++i) a.kf[i] = p.kf[i];
    a.n_kv = p.n_kv;
    for (int i = 0; i < p.n_kv; ++i) a.kvf[i] = p.kvf[i];
    if (p.n_kv > 0) a.S = static_cast<int64_t>(p.n_kv) * p.N;
    const int64_t nq = (Mq + kF32Rows - 1) / kF32Rows;
    if (nq > 0x7fffffffLL || p.heads > 65535) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<uint32_t>(nq), static_cast<uint32_t>(p.heads)), block(2 * kF32Rows);
    if (p.head_dim == 128) hipLaunchKernelGGL(attn_f32_kernel<128>, grid, block, 0, stream, a);
    else hipLaunchKernelGGL(attn_f32_kernel<64>, grid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace rf
