// C ABI of librhymeflow.so: argument validation, kernel-argument packing and
// launch on the caller's stream. Every check runs before the first HIP call.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "rf_internal.h"

namespace {

thread_local char g_err[512] = "";

int fail(int status, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return status;
}

int ok() {
    g_err[0] = '\0';
    return RF_OK;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Byte counts are 64-bit: sizes whose product (computed in double) passes this
// are rejected before any of it is formed in integers.
constexpr double kMaxBytes = 4.0e18;

// Half-open byte ranges [a, a+na) and [b, b+nb) intersect.
bool overlaps(const void *a, int64_t na, const void *b, int64_t nb) {
    const uintptr_t pa = reinterpret_cast<uintptr_t>(a);
    const uintptr_t pb = reinterpret_cast<uintptr_t>(b);
    return pa < pb + static_cast<uintptr_t>(nb) && pb < pa + static_cast<uintptr_t>(na);
}

int launched(hipError_t e, const char *what) {
    if (e != hipSuccess)
        return fail(RF_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

// Strictly increasing ids in [0, T), copied into dst.
int check_id_list(const int32_t *ids, int32_t M, int32_t T, int32_t *dst, const char *what) {
    if (!ids) return fail(RF_ERR_INVALID_ARG, "%s: id list is NULL", what);
    if (M <= 0) return fail(RF_ERR_INVALID_ARG, "%s: M = %d must be positive", what, M);
    if (T <= 0) return fail(RF_ERR_INVALID_ARG, "%s: T = %d must be positive", what, T);
    if (T > RF_MAX_FRAMES)
        return fail(RF_ERR_RANGE, "%s: T = %d exceeds %d frames", what, T, RF_MAX_FRAMES);
    if (M > T) return fail(RF_ERR_RANGE, "%s: M = %d exceeds T = %d", what, M, T);
    for (int32_t i = 0; i < M; ++i) {
        if (ids[i] < 0 || ids[i] >= T)
            return fail(RF_ERR_RANGE, "%s: id %d at position %d outside [0, %d)", what, ids[i], i, T);
        if (i > 0 && ids[i] <= ids[i - 1])
            return fail(RF_ERR_INVALID_ARG, "%s: ids not strictly increasing at position %d", what, i);
        dst[i] = ids[i];
    }
    return RF_OK;
}

}  // namespace

extern "C" {

const char *rf_status_string(int status) {
    switch (status) {
        case RF_OK: return "RF_OK";
        case RF_ERR_INVALID_ARG: return "RF_ERR_INVALID_ARG";
        case RF_ERR_UNSUPPORTED: return "RF_ERR_UNSUPPORTED";
        case RF_ERR_RANGE: return "RF_ERR_RANGE";
        case RF_ERR_HIP: return "RF_ERR_HIP";
        default: return "RF_UNKNOWN_STATUS";
    }
}

const char *rf_last_error(void) { return g_err; }

int rf_abi_version(void) { return RF_ABI_VERSION; }

int rf_select_keyframes(const int32_t *frame_ids, int32_t n_ids, int32_t T, uint32_t flags,
                        int32_t *keyframe_ids_out, int32_t *num_keyframes_out,
                        uint8_t *keyframe_mask_out) {
    if (!keyframe_ids_out || !num_keyframes_out)
        return fail(RF_ERR_INVALID_ARG, "rf_select_keyframes: NULL output");
    if (n_ids < 0) return fail(RF_ERR_INVALID_ARG, "rf_select_keyframes: n_ids < 0");
    if (n_ids > 0 && !frame_ids)
        return fail(RF_ERR_INVALID_ARG, "rf_select_keyframes: frame_ids is NULL");
    if (T <= 0 || T > RF_MAX_FRAMES)
        return fail(RF_ERR_RANGE, "rf_select_keyframes: T = %d outside 1..%d", T, RF_MAX_FRAMES);
    if (flags & ~RF_SEL_NO_FORCE_FIRST)
        return fail(RF_ERR_INVALID_ARG, "rf_select_keyframes: unknown flags 0x%x", flags);
    uint8_t member[RF_MAX_FRAMES] = {0};
    for (int32_t i = 0; i < n_ids; ++i) {
        if (frame_ids[i] < 0 || frame_ids[i] >= T)
            return fail(RF_ERR_RANGE, "rf_select_keyframes: id %d outside [0, %d)", frame_ids[i], T);
        member[frame_ids[i]] = 1;
    }
    if (!(flags & RF_SEL_NO_FORCE_FIRST)) member[0] = 1;  // the first frame anchors the video
    int32_t n = 0;
    for (int32_t f = 0; f < T; ++f) n += member[f];
    if (n == 0) return fail(RF_ERR_INVALID_ARG, "rf_select_keyframes: empty keyframe set");
    n = 0;
    for (int32_t f = 0; f < T; ++f)
        if (member[f]) keyframe_ids_out[n++] = f;
    *num_keyframes_out = n;
    if (keyframe_mask_out)
        for (int32_t f = 0; f < T; ++f) keyframe_mask_out[f] = member[f];
    return ok();
}

int rf_keyframes_stride(int32_t T, int32_t k, int32_t *ids_out, int32_t *n_out) {
    if (!ids_out || !n_out) return fail(RF_ERR_INVALID_ARG, "rf_keyframes_stride: NULL output");
    if (k <= 0) return fail(RF_ERR_INVALID_ARG, "rf_keyframes_stride: k = %d must be positive", k);
    if (T <= 0 || T > RF_MAX_FRAMES)
        return fail(RF_ERR_RANGE, "rf_keyframes_stride: T = %d outside 1..%d", T, RF_MAX_FRAMES);
    int32_t n = 0;
    for (int32_t f = 0; f < T; f += k) ids_out[n++] = f;
    *n_out = n;
    return ok();
}

int rf_keyframes_uniform(int32_t T, int32_t M, int32_t *ids_out, int32_t *n_out) {
    if (!ids_out || !n_out) return fail(RF_ERR_INVALID_ARG, "rf_keyframes_uniform: NULL output");
    if (T <= 0 || T > RF_MAX_FRAMES)
        return fail(RF_ERR_RANGE, "rf_keyframes_uniform: T = %d outside 1..%d", T, RF_MAX_FRAMES);
    if (M <= 0 || M > T)
        return fail(RF_ERR_RANGE, "rf_keyframes_uniform: M = %d outside 1..%d", M, T);
    if (M == 1) {
        ids_out[0] = 0;
        *n_out = 1;
        return ok();
    }
    // nearest integer to i*(T-1)/(M-1), halves rounded up: floor((2i(T-1) + (M-1)) / (2(M-1)))
    for (int32_t i = 0; i < M; ++i) {
        const int64_t num = 2LL * i * (T - 1) + (M - 1);
        ids_out[i] = static_cast<int32_t>(num / (2LL * (M - 1)));
    }
    *n_out = M;
    return ok();
}

int rf_project_latents(const void *latents, void *out, const double timesteps[3],
                       const uint8_t *keyframe_mask, int32_t B, int32_t C, int32_t T,
                       int32_t Hl, int32_t Wl, int32_t dtype, void *stream) {
    const char *fn = "rf_project_latents";
    if (!latents || !out || !timesteps || !keyframe_mask)
        return fail(RF_ERR_INVALID_ARG, "%s: NULL argument", fn);
    if (B <= 0 || C <= 0 || T <= 0 || Hl <= 0 || Wl <= 0)
        return fail(RF_ERR_INVALID_ARG, "%s: sizes must be positive (B=%d C=%d T=%d Hl=%d Wl=%d)",
                    fn, B, C, T, Hl, Wl);
    if (T > RF_MAX_FRAMES) return fail(RF_ERR_RANGE, "%s: T = %d exceeds %d", fn, T, RF_MAX_FRAMES);
    if (dtype != RF_F32 && dtype != RF_BF16)
        return fail(RF_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
    if (static_cast<double>(B) * 2.0 * C * T * Hl * Wl * 4.0 > kMaxBytes)
        return fail(RF_ERR_RANGE, "%s: sizes overflow 64-bit byte counts", fn);
    const double t_start = timesteps[0], t_end = timesteps[1], tau = timesteps[2];
    if (!isfinite(t_start) || !isfinite(t_end) || !isfinite(tau))
        return fail(RF_ERR_INVALID_ARG, "%s: timesteps must be finite", fn);
    if (!aligned16(latents) || !aligned16(out))
        return fail(RF_ERR_UNSUPPORTED, "%s: pointers must be 16-byte aligned", fn);

    const int64_t elem = dtype == RF_F32 ? 4 : 2;
    const int64_t plane = static_cast<int64_t>(Hl) * Wl;
    const int64_t slot_bytes = static_cast<int64_t>(C) * T * plane * elem;
    const int64_t lat_bytes = static_cast<int64_t>(B) * 2 * slot_bytes;
    const int64_t out_bytes = static_cast<int64_t>(B) * slot_bytes;
    const char *slot1 = static_cast<const char *>(latents) + slot_bytes;
    int skip_keyframes = 0;
    if (B == 1 && out == slot1) {
        skip_keyframes = 1;  // out is slot 1 itself: keyframe planes already hold their state
    } else if (overlaps(latents, lat_bytes, out, out_bytes)) {
        return fail(RF_ERR_INVALID_ARG, "%s: out overlaps latents (only out == slot 1 with B == 1 is allowed)", fn);
    }

    rf::ProjParams p{};
    p.latents = latents;
    p.out = out;
    p.plane = plane;
    p.B = B;
    p.C = C;
    p.T = T;
    p.dtype = dtype;
    p.skip_keyframes = skip_keyframes;
    // Eq. (3): alpha = (t_start - tau) / (t_start - t_end), in double, kept in
    // [0, 1]; equal endpoints (both snapshots the same state) give 1.
    double alpha = 1.0;
    if (t_start != t_end) {
        alpha = (t_start - tau) / (t_start - t_end);
        alpha = alpha < 0.0 ? 0.0 : (alpha > 1.0 ? 1.0 : alpha);
    }
    p.alpha = static_cast<float>(alpha);
    for (int32_t f = 0; f < T; ++f) p.is_key[f] = keyframe_mask[f] ? 1 : 0;
    return launched(rf::launch_projection(p, static_cast<hipStream_t>(stream)), fn);
}

// Shared validation and launch of the two attention entry points.
// Bytes of split-tail workspace a bf16 attention of these sizes uses on a device
// of `cus` compute units (0 for fp32 or when nothing is split); the sizes must
// already be valid.
static int64_t attention_ws_need(int32_t M, int32_t n_kv, int32_t T, int64_t N, int32_t heads, int32_t head_dim,
                                 int32_t dtype, int32_t cus) {
    if (dtype != RF_BF16) return 0;
    return rf::attention_split(static_cast<int64_t>(M) * N, heads, head_dim, N, N * T, n_kv, cus).ws_bytes;
}

// The current device's geometry, as an rf_status.
static int query_geometry(rf::DeviceGeometry *geo, const char *fn) {
    const hipError_t e = rf::device_geometry(geo);
    if (e != hipSuccess)
        return fail(RF_ERR_HIP, "%s: cannot query the current device: %s", fn, hipGetErrorString(e));
    return RF_OK;
}

// The cache form of an attention call: the cached frames' projected states at
// t_skip replace their keys and values (already validated).
struct CacheForm {
    const rf_rolling_cache *cache;
    const void *store;
    double t_skip;
};

static double cache_alpha(const rf_rolling_cache &c, int32_t f, double t_skip);

// use_scratch: the split tail takes the library's static scratch (the
// allocation-free entry point) instead of a caller workspace.
static int attention_call(const void *q, const void *k, const void *v, void *out, const int32_t *q_ids,
                          int32_t M, const int32_t *kv_ids, int32_t Mkv, int32_t T, int32_t H, int32_t W,
                          int32_t heads, int32_t head_dim, int32_t dtype, void *ws, int64_t ws_bytes,
                          void *stream, const char *fn, bool use_scratch = false,
                          const CacheForm *cf = nullptr) {
    if (!q || !k || !v || !out) return fail(RF_ERR_INVALID_ARG, "%s: NULL tensor", fn);
    if (H <= 0 || W <= 0 || heads <= 0 || head_dim <= 0)
        return fail(RF_ERR_INVALID_ARG, "%s: sizes must be positive (H=%d W=%d heads=%d head_dim=%d)",
                    fn, H, W, heads, head_dim);
    if (static_cast<double>(H) * W * (T > 0 ? T : 1) * heads * head_dim * 4.0 > kMaxBytes)
        return fail(RF_ERR_RANGE, "%s: sizes overflow 64-bit byte counts (T=%d H=%d W=%d heads=%d head_dim=%d)",
                    fn, T, H, W, heads, head_dim);
    rf::AttnParams p{};
    int rc = check_id_list(q_ids, M, T, p.kf, fn);
    if (rc != RF_OK) return rc;
    int32_t kvf[RF_MAX_FRAMES];
    if (kv_ids) {
        rc = check_id_list(kv_ids, Mkv, T, kvf, fn);
        if (rc != RF_OK) return rc;
    }
    if (head_dim != 64 && head_dim != 128)
        return fail(RF_ERR_UNSUPPORTED, "%s: head_dim %d not in {64, 128}", fn, head_dim);
    if (dtype != RF_BF16 && dtype != RF_F32)
        return fail(RF_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
        return fail(RF_ERR_UNSUPPORTED, "%s: pointers must be 16-byte aligned", fn);

    const int64_t N = static_cast<int64_t>(H) * W;
    const int64_t S = N * T;
    const int64_t row = static_cast<int64_t>(heads) * head_dim * (dtype == RF_F32 ? 4 : 2);
    const int64_t in_bytes = S * row;
    const int64_t out_bytes = N * M * row;
    if (overlaps(out, out_bytes, q, in_bytes) || overlaps(out, out_bytes, k, in_bytes) ||
        overlaps(out, out_bytes, v, in_bytes))
        return fail(RF_ERR_INVALID_ARG, "%s: out overlaps q, k or v", fn);
    const int32_t n_kv = (kv_ids && Mkv < T) ? Mkv : 0;
    if (cf) {
        const rf_rolling_cache &c = *cf->cache;
        const int64_t store_bytes = 2 * static_cast<int64_t>(c.n_cached) * c.frame_bytes;
        if (overlaps(out, out_bytes, cf->store, store_bytes))
            return fail(RF_ERR_INVALID_ARG, "%s: out overlaps the cache store", fn);
        p.cache_form = 1;
        p.store = cf->store;
        for (int32_t f = 0; f < T; ++f) {
            p.cslot[f] = -1;
            p.calpha[f] = 0.0f;
            if (c.after_slot[f] >= 0) {
                p.cslot[f] = static_cast<int32_t>(c.before_slot[f]) | (static_cast<int32_t>(c.after_slot[f]) << 16);
                p.calpha[f] = static_cast<float>(cache_alpha(c, f, cf->t_skip));
            }
        }
    }
    if (ws) {
        if (ws_bytes < 0) return fail(RF_ERR_INVALID_ARG, "%s: workspace_bytes < 0", fn);
        if (!aligned16(ws)) return fail(RF_ERR_UNSUPPORTED, "%s: workspace must be 16-byte aligned", fn);
        if (ws_bytes > 0 && (overlaps(ws, ws_bytes, q, in_bytes) || overlaps(ws, ws_bytes, k, in_bytes) ||
                             overlaps(ws, ws_bytes, v, in_bytes) || overlaps(ws, ws_bytes, out, out_bytes)))
            return fail(RF_ERR_INVALID_ARG, "%s: workspace overlaps q, k, v or out", fn);
    }
    // every argument is valid: the bf16 split plan and tile order follow the device
    p.geo.cus = p.geo.xcds = 1;
    if (dtype == RF_BF16) {
        rc = query_geometry(&p.geo, fn);
        if (rc != RF_OK) return rc;
    }
    if (use_scratch) {
        const int64_t need = attention_ws_need(M, n_kv, T, N, heads, head_dim, dtype, p.geo.cus);
        if (need > rf::kAttentionScratchBytes)
            return fail(RF_ERR_RANGE,
                        "%s: the split-key tail needs %lld bytes of scratch on %d compute units, the static "
                        "scratch holds %lld (rf_keyframe_attention_ws takes a workspace of any size)",
                        fn, static_cast<long long>(need), p.geo.cus,
                        static_cast<long long>(rf::kAttentionScratchBytes));
        if (need > 0) {
            const hipError_t e = rf::attention_scratch(&p.ws);
            if (e != hipSuccess)
                return fail(RF_ERR_HIP, "%s: cannot look up the static scratch: %s", fn, hipGetErrorString(e));
            p.ws_bytes = rf::kAttentionScratchBytes;
        }
    } else if (ws) {
        const int64_t need = attention_ws_need(M, n_kv, T, N, heads, head_dim, dtype, p.geo.cus);
        if (ws_bytes < need)
            return fail(RF_ERR_INVALID_ARG, "%s: workspace of %lld bytes, %lld needed on %d compute units", fn,
                        static_cast<long long>(ws_bytes), static_cast<long long>(need), p.geo.cus);
        p.ws = need > 0 ? ws : nullptr;
        p.ws_bytes = ws_bytes;
    }

    p.q = q;
    p.k = k;
    p.v = v;
    p.out = out;
    p.S = S;
    p.N = N;
    p.M = M;
    p.heads = heads;
    p.head_dim = head_dim;
    p.dtype = dtype;
    // every frame listed: the unmasked kernel
    p.n_kv = n_kv;
    for (int32_t i = 0; i < p.n_kv; ++i) p.kvf[i] = kvf[i];
    return launched(rf::launch_attention(p, static_cast<hipStream_t>(stream)), fn);
}

int rf_keyframe_attention(const void *q, const void *k, const void *v, void *out,
                          const int32_t *keyframe_ids, int32_t M, int32_t T, int32_t H,
                          int32_t W, int32_t heads, int32_t head_dim, int32_t dtype,
                          void *stream) {
    return attention_call(q, k, v, out, keyframe_ids, M, nullptr, 0, T, H, W, heads, head_dim, dtype,
                          nullptr, 0, stream, "rf_keyframe_attention");
}

int rf_keyframe_attention_ws(const void *q, const void *k, const void *v, void *out,
                             const int32_t *keyframe_ids, int32_t M, int32_t T, int32_t H, int32_t W,
                             int32_t heads, int32_t head_dim, int32_t dtype, void *workspace,
                             int64_t workspace_bytes, void *stream) {
    const char *fn = "rf_keyframe_attention_ws";
    if (!workspace) return fail(RF_ERR_INVALID_ARG, "%s: NULL workspace", fn);
    return attention_call(q, k, v, out, keyframe_ids, M, nullptr, 0, T, H, W, heads, head_dim, dtype,
                          workspace, workspace_bytes, stream, fn);
}

int rf_keyframe_attention_noalloc(const void *q, const void *k, const void *v, void *out,
                                  const int32_t *keyframe_ids, int32_t M, int32_t T, int32_t H, int32_t W,
                                  int32_t heads, int32_t head_dim, int32_t dtype, void *stream) {
    return attention_call(q, k, v, out, keyframe_ids, M, nullptr, 0, T, H, W, heads, head_dim, dtype, nullptr, 0,
                          stream, "rf_keyframe_attention_noalloc", true);
}

int rf_frame_attention(const void *q, const void *k, const void *v, void *out,
                       const int32_t *q_frames, int32_t Mq, const int32_t *kv_frames, int32_t Mkv,
                       int32_t T, int32_t H, int32_t W, int32_t heads, int32_t head_dim,
                       int32_t dtype, void *workspace, int64_t workspace_bytes, void *stream) {
    const char *fn = "rf_frame_attention";
    if (!kv_frames) return fail(RF_ERR_INVALID_ARG, "%s: kv_frames is NULL", fn);
    return attention_call(q, k, v, out, q_frames, Mq, kv_frames, Mkv, T, H, W, heads, head_dim, dtype,
                          workspace, workspace_bytes, stream, fn);
}

// Sizes of an attention plan query, and the compute units it is planned for
// (0: the current device's, which needs a device query).
static int plan_args(int32_t M, int32_t Mkv, int32_t T, int32_t H, int32_t W, int32_t heads, int32_t head_dim,
                     int32_t dtype, int32_t compute_units, int32_t *cus, const char *fn) {
    if (H <= 0 || W <= 0 || heads <= 0 || T <= 0 || M <= 0 || Mkv <= 0)
        return fail(RF_ERR_INVALID_ARG, "%s: sizes must be positive", fn);
    if (T > RF_MAX_FRAMES) return fail(RF_ERR_RANGE, "%s: T = %d exceeds %d", fn, T, RF_MAX_FRAMES);
    if (M > T || Mkv > T) return fail(RF_ERR_RANGE, "%s: M = %d or Mkv = %d exceeds T = %d", fn, M, Mkv, T);
    if (head_dim != 64 && head_dim != 128)
        return fail(RF_ERR_UNSUPPORTED, "%s: head_dim %d not in {64, 128}", fn, head_dim);
    if (dtype != RF_BF16 && dtype != RF_F32) return fail(RF_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
    if (static_cast<double>(H) * W * T * heads * head_dim * 4.0 > kMaxBytes)
        return fail(RF_ERR_RANGE, "%s: sizes overflow 64-bit byte counts", fn);
    if (compute_units < 0 || compute_units > RF_MAX_COMPUTE_UNITS)
        return fail(RF_ERR_RANGE, "%s: compute_units = %d outside 0..%d", fn, compute_units, RF_MAX_COMPUTE_UNITS);
    if (compute_units > 0) {
        *cus = compute_units;
        return RF_OK;
    }
    rf::DeviceGeometry geo;
    const int rc = query_geometry(&geo, fn);
    if (rc != RF_OK) return rc;
    *cus = geo.cus;
    return RF_OK;
}

int rf_attention_workspace(int32_t M, int32_t Mkv, int32_t T, int32_t H, int32_t W, int32_t heads,
                           int32_t head_dim, int32_t dtype, int32_t compute_units, int64_t *bytes_out) {
    const char *fn = "rf_attention_workspace";
    if (!bytes_out) return fail(RF_ERR_INVALID_ARG, "%s: NULL output", fn);
    int32_t cus = 0;
    const int rc = plan_args(M, Mkv, T, H, W, heads, head_dim, dtype, compute_units, &cus, fn);
    if (rc != RF_OK) return rc;
    *bytes_out = attention_ws_need(M, Mkv < T ? Mkv : 0, T, static_cast<int64_t>(H) * W, heads, head_dim, dtype,
                                   cus);
    return ok();
}

int rf_attention_plan(int32_t M, int32_t Mkv, int32_t T, int32_t H, int32_t W, int32_t heads, int32_t head_dim,
                      int32_t dtype, int32_t compute_units, rf_attention_split *plan_out) {
    const char *fn = "rf_attention_plan";
    if (!plan_out) return fail(RF_ERR_INVALID_ARG, "%s: NULL output", fn);
    int32_t cus = 0;
    const int rc = plan_args(M, Mkv, T, H, W, heads, head_dim, dtype, compute_units, &cus, fn);
    if (rc != RF_OK) return rc;
    const int64_t N = static_cast<int64_t>(H) * W;
    rf_attention_split out;
    memset(&out, 0, sizeof out);
    out.compute_units = cus;
    if (dtype == RF_BF16) {
        const rf::AttnSplit sp = rf::attention_split(static_cast<int64_t>(M) * N, heads, head_dim, N, N * T,
                                                     Mkv < T ? Mkv : 0, cus);
        out.tiles = sp.n_tiles;
        out.whole_tiles = sp.n_direct;
        out.tail_tiles = sp.n_tail;
        out.parts = static_cast<int32_t>(sp.split);
        out.key_tiles_per_part = static_cast<int32_t>(sp.kv_per_split);
        out.workspace_bytes = sp.ws_bytes;
    }
    *plan_out = out;
    return ok();
}

static int frame_copy(const void *src, void *dst, const int32_t *frame_ids, int32_t M, int32_t T,
                      int64_t rows_per_frame, int64_t row_bytes, void *stream, int scatter,
                      const char *fn) {
    if (!src || !dst) return fail(RF_ERR_INVALID_ARG, "%s: NULL buffer", fn);
    if (rows_per_frame <= 0 || row_bytes <= 0)
        return fail(RF_ERR_INVALID_ARG, "%s: rows_per_frame and row_bytes must be positive", fn);
    if (static_cast<double>(rows_per_frame) * static_cast<double>(row_bytes) * RF_MAX_FRAMES > kMaxBytes)
        return fail(RF_ERR_RANGE, "%s: rows_per_frame x row_bytes overflows 64-bit byte counts", fn);
    rf::FrameCopyParams p{};
    int32_t ids[RF_MAX_FRAMES];
    const int rc = check_id_list(frame_ids, M, T, ids, fn);
    if (rc != RF_OK) return rc;
    if (row_bytes % 16 != 0)
        return fail(RF_ERR_UNSUPPORTED, "%s: row_bytes %lld not a multiple of 16", fn,
                    static_cast<long long>(row_bytes));
    if (!aligned16(src) || !aligned16(dst))
        return fail(RF_ERR_UNSUPPORTED, "%s: pointers must be 16-byte aligned", fn);
    const int64_t frame_bytes = rows_per_frame * row_bytes;
    const int64_t full = frame_bytes * T, compact = frame_bytes * M;
    if (overlaps(src, scatter ? compact : full, dst, scatter ? full : compact))
        return fail(RF_ERR_INVALID_ARG, "%s: source and destination overlap", fn);
    p.src = src;
    p.dst = dst;
    p.frame_bytes = frame_bytes;
    p.M = M;
    for (int32_t m = 0; m < M; ++m) {
        p.src_idx[m] = scatter ? m : ids[m];
        p.dst_idx[m] = scatter ? ids[m] : m;
    }
    return launched(rf::launch_frame_copy(p, static_cast<hipStream_t>(stream)), fn);
}

int rf_gather_frames(const void *src_full, void *dst_compact, const int32_t *frame_ids, int32_t M,
                     int32_t T, int64_t rows_per_frame, int64_t row_bytes, void *stream) {
    return frame_copy(src_full, dst_compact, frame_ids, M, T, rows_per_frame, row_bytes, stream, 0,
                      "rf_gather_frames");
}

int rf_scatter_frames(const void *src_compact, void *dst_full, const int32_t *frame_ids, int32_t M,
                      int32_t T, int64_t rows_per_frame, int64_t row_bytes, void *stream) {
    return frame_copy(src_compact, dst_full, frame_ids, M, T, rows_per_frame, row_bytes, stream, 1,
                      "rf_scatter_frames");
}

int rf_frame_similarity_workspace(int32_t B, int32_t C, int32_t T, int32_t H, int32_t W,
                                  int64_t *bytes_out) {
    const char *fn = "rf_frame_similarity_workspace";
    if (!bytes_out) return fail(RF_ERR_INVALID_ARG, "%s: NULL output", fn);
    if (B <= 0 || C <= 0 || T <= 0 || H <= 0 || W <= 0)
        return fail(RF_ERR_INVALID_ARG, "%s: sizes must be positive (B=%d C=%d T=%d H=%d W=%d)",
                    fn, B, C, T, H, W);
    if (T > RF_MAX_FRAMES) return fail(RF_ERR_RANGE, "%s: T = %d exceeds %d", fn, T, RF_MAX_FRAMES);
    const rf::SimGeometry g = rf::similarity_geometry(B, C, T, static_cast<int64_t>(H) * W);
    if (static_cast<double>(B) * static_cast<double>(g.n_runs) * g.NBP * 128.0 > kMaxBytes ||
        static_cast<double>(C) * H * W * T * B > kMaxBytes)
        return fail(RF_ERR_RANGE, "%s: workspace size overflows", fn);
    *bytes_out = g.workspace_bytes;
    return ok();
}

int rf_frame_similarity(const void *latents, double *sim_out, void *workspace,
                        int64_t workspace_bytes, int32_t B, int32_t C, int32_t T, int32_t H,
                        int32_t W, int32_t dtype, void *stream) {
    const char *fn = "rf_frame_similarity";
    if (!latents || !sim_out || !workspace) return fail(RF_ERR_INVALID_ARG, "%s: NULL argument", fn);
    int64_t need = 0;
    const int rc = rf_frame_similarity_workspace(B, C, T, H, W, &need);
    if (rc != RF_OK) return rc;
    if (dtype != RF_F32 && dtype != RF_BF16)
        return fail(RF_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
    if (!aligned16(latents) || !aligned16(workspace) || (reinterpret_cast<uintptr_t>(sim_out) & 7u))
        return fail(RF_ERR_UNSUPPORTED, "%s: latents/workspace must be 16-byte and sim_out 8-byte aligned", fn);
    if (workspace_bytes < need)
        return fail(RF_ERR_INVALID_ARG, "%s: workspace of %lld bytes, %lld needed", fn,
                    static_cast<long long>(workspace_bytes), static_cast<long long>(need));
    const int64_t plane = static_cast<int64_t>(H) * W;
    const int64_t lat_bytes = static_cast<int64_t>(B) * C * T * plane * (dtype == RF_F32 ? 4 : 2);
    const int64_t sim_bytes = static_cast<int64_t>(B) * T * T * 8;
    if (overlaps(sim_out, sim_bytes, latents, lat_bytes) || overlaps(sim_out, sim_bytes, workspace, need) ||
        overlaps(workspace, need, latents, lat_bytes))
        return fail(RF_ERR_INVALID_ARG, "%s: latents, sim_out and workspace must not overlap", fn);
    rf::SimParams p{};
    p.latents = latents;
    p.sim = sim_out;
    p.workspace = static_cast<double *>(workspace);
    p.plane = plane;
    p.B = B;
    p.C = C;
    p.T = T;
    p.dtype = dtype;
    return launched(rf::launch_similarity(p, static_cast<hipStream_t>(stream)), fn);
}

int rf_select_keyframes_adaptive(const double *sim, int32_t T, double tau, int32_t M, double dtau,
                                 double delta_up, double delta_down, uint32_t flags,
                                 int32_t *keyframe_ids_out, int32_t *num_keyframes_out,
                                 uint8_t *keyframe_mask_out) {
    const char *fn = "rf_select_keyframes_adaptive";
    if (!sim || !keyframe_ids_out || !num_keyframes_out)
        return fail(RF_ERR_INVALID_ARG, "%s: NULL argument", fn);
    if (T <= 0 || T > RF_MAX_FRAMES) return fail(RF_ERR_RANGE, "%s: T = %d outside 1..%d", fn, T, RF_MAX_FRAMES);
    if (M <= 0 || M > T) return fail(RF_ERR_RANGE, "%s: M = %d outside 1..%d", fn, M, T);
    if (!isfinite(tau) || !isfinite(dtau) || !isfinite(delta_up) || !isfinite(delta_down))
        return fail(RF_ERR_INVALID_ARG, "%s: tau, dtau, delta_up and delta_down must be finite", fn);
    if (flags & ~RF_SEL_INTENT_SIGN) return fail(RF_ERR_INVALID_ARG, "%s: unknown flags 0x%x", fn, flags);
    const bool intent = (flags & RF_SEL_INTENT_SIGN) != 0;
    // Alg. 1: the first frame seeds the set; expected interval L_avg = T / M.
    const double l_avg = static_cast<double>(T) / static_cast<double>(M);
    int32_t n = 0, last = 0;
    keyframe_ids_out[n++] = 0;
    for (int32_t i = 1; i < T && n < M; ++i) {
        // Eq. (1): compare with the most recent keyframe, strictly below the threshold
        if (sim[static_cast<int64_t>(i) * T + last] < tau) {
            const double gap = static_cast<double>(i - last);
            if (gap >= l_avg + delta_up)
                tau = intent ? tau + dtau : tau - dtau;
            else if (gap <= l_avg - delta_down)
                tau = intent ? tau - dtau : tau + dtau;
            keyframe_ids_out[n++] = i;
            last = i;
        }
    }
    *num_keyframes_out = n;
    if (keyframe_mask_out) {
        for (int32_t f = 0; f < T; ++f) keyframe_mask_out[f] = 0;
        for (int32_t m = 0; m < n; ++m) keyframe_mask_out[keyframe_ids_out[m]] = 1;
    }
    return ok();
}

// ---------------------------------------------------------------------------
// Rolling cache (App. B.2)
// ---------------------------------------------------------------------------

static const uint32_t kCacheMagic = 0x52464331u;
static const double kHiddenEps = 1e-8;

static int64_t elem_bytes(int32_t dtype) { return dtype == RF_F32 ? 4 : 2; }

static int cache_store_bytes(int32_t n_cached, int64_t rows_per_frame, int32_t hidden, int32_t dtype,
                             int64_t *bytes_out, const char *fn) {
    if (n_cached <= 0 || rows_per_frame <= 0 || hidden <= 0)
        return fail(RF_ERR_INVALID_ARG, "%s: sizes must be positive", fn);
    if (n_cached > RF_MAX_FRAMES)
        return fail(RF_ERR_RANGE, "%s: n_cached = %d exceeds %d", fn, n_cached, RF_MAX_FRAMES);
    if (dtype != RF_F32 && dtype != RF_BF16) return fail(RF_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
    if (static_cast<double>(rows_per_frame) * hidden * elem_bytes(dtype) * 2.0 * n_cached * RF_MAX_FRAMES > kMaxBytes)
        return fail(RF_ERR_RANGE, "%s: size overflows", fn);
    *bytes_out = 2 * static_cast<int64_t>(n_cached) * rows_per_frame * hidden * elem_bytes(dtype);
    return RF_OK;
}

int rf_cache_store_bytes(int32_t n_cached, int64_t rows_per_frame, int32_t hidden, int32_t dtype,
                         int64_t *bytes_out) {
    const char *fn = "rf_cache_store_bytes";
    if (!bytes_out) return fail(RF_ERR_INVALID_ARG, "%s: NULL output", fn);
    const int rc = cache_store_bytes(n_cached, rows_per_frame, hidden, dtype, bytes_out, fn);
    return rc == RF_OK ? ok() : rc;
}

// An initialised cache struct whose sizes and slot indices are consistent.
static int check_cache(const rf_rolling_cache *c, const char *fn) {
    if (!c) return fail(RF_ERR_INVALID_ARG, "%s: NULL cache", fn);
    if (c->magic != kCacheMagic) return fail(RF_ERR_INVALID_ARG, "%s: cache not initialised by rf_cache_init", fn);
    if (c->T <= 0 || c->T > RF_MAX_FRAMES || c->n_cached <= 0 || c->n_cached > c->T ||
        c->rows_per_frame <= 0 || c->hidden <= 0 || (c->dtype != RF_F32 && c->dtype != RF_BF16) ||
        static_cast<double>(c->rows_per_frame) * c->hidden * 4.0 * 2.0 * RF_MAX_FRAMES > kMaxBytes ||
        c->frame_bytes != c->rows_per_frame * c->hidden * elem_bytes(c->dtype))
        return fail(RF_ERR_INVALID_ARG, "%s: cache struct is inconsistent", fn);
    for (int32_t f = 0; f < c->T; ++f) {
        const int b = c->before_slot[f], a = c->after_slot[f];
        if (b < 0 && a < 0) continue;
        if (b < 0 || a < 0 || b >= 2 * c->n_cached || a >= 2 * c->n_cached || (b >> 1) != (a >> 1))
            return fail(RF_ERR_INVALID_ARG, "%s: cache struct has bad slots for frame %d", fn, f);
        if (!isfinite(c->t_before[f]) || !isfinite(c->t_after[f]) || !(c->t_after[f] <= c->t_before[f]))
            return fail(RF_ERR_INVALID_ARG, "%s: cache struct has bad timesteps for frame %d", fn, f);
    }
    return RF_OK;
}

// The listed frames (NULL: every cached frame), strictly increasing and cached.
static int cache_frames(const rf_rolling_cache *c, const int32_t *frames, int32_t n, int32_t *out,
                        int32_t *n_out, const char *fn) {
    if (!frames) {
        int32_t k = 0;
        for (int32_t f = 0; f < c->T; ++f)
            if (c->after_slot[f] >= 0) out[k++] = f;
        *n_out = k;
        return RF_OK;
    }
    if (n <= 0 || n > c->T) return fail(RF_ERR_INVALID_ARG, "%s: n = %d outside 1..%d", fn, n, c->T);
    for (int32_t i = 0; i < n; ++i) {
        if (frames[i] < 0 || frames[i] >= c->T)
            return fail(RF_ERR_RANGE, "%s: frame %d outside [0, %d)", fn, frames[i], c->T);
        if (i > 0 && frames[i] <= frames[i - 1])
            return fail(RF_ERR_INVALID_ARG, "%s: frames not strictly increasing at position %d", fn, i);
        if (c->after_slot[frames[i]] < 0) return fail(RF_ERR_INVALID_ARG, "%s: frame %d is not cached", fn, frames[i]);
        out[i] = frames[i];
    }
    *n_out = n;
    return RF_OK;
}

// Copies the rows of each listed frame of h_full into its after slot.
static int store_after(const rf_rolling_cache &c, void *store, const void *h_full, const int32_t *fr,
                       int32_t n, void *stream, const char *fn) {
    if (!store) return fail(RF_ERR_INVALID_ARG, "%s: NULL store", fn);
    if (!aligned16(store) || !aligned16(h_full))
        return fail(RF_ERR_UNSUPPORTED, "%s: store and h_full must be 16-byte aligned", fn);
    const int64_t store_bytes = 2 * static_cast<int64_t>(c.n_cached) * c.frame_bytes;
    if (overlaps(store, store_bytes, h_full, c.frame_bytes * c.T))
        return fail(RF_ERR_INVALID_ARG, "%s: store overlaps h_full", fn);
    rf::FrameCopyParams p{};
    p.src = h_full;
    p.dst = store;
    p.frame_bytes = c.frame_bytes;
    p.M = n;
    for (int32_t i = 0; i < n; ++i) {
        p.src_idx[i] = fr[i];
        p.dst_idx[i] = c.after_slot[fr[i]];
    }
    return launched(rf::launch_frame_copy(p, static_cast<hipStream_t>(stream)), fn);
}

int rf_cache_init(rf_rolling_cache *cache, void *store, const void *h_full, const int32_t *frames,
                  int32_t n, int32_t T, int64_t rows_per_frame, int32_t hidden, int32_t dtype,
                  double t_w, void *stream) {
    const char *fn = "rf_cache_init";
    if (!cache) return fail(RF_ERR_INVALID_ARG, "%s: NULL cache", fn);
    int32_t ids[RF_MAX_FRAMES];
    int rc = check_id_list(frames, n, T, ids, fn);
    if (rc != RF_OK) return rc;
    int64_t need = 0;
    rc = cache_store_bytes(n, rows_per_frame, hidden, dtype, &need, fn);
    if (rc != RF_OK) return rc;
    if ((static_cast<int64_t>(hidden) * elem_bytes(dtype)) % 16 != 0)
        return fail(RF_ERR_UNSUPPORTED, "%s: a row of %d elements is not a multiple of 16 bytes", fn, hidden);
    if (!isfinite(t_w)) return fail(RF_ERR_INVALID_ARG, "%s: t_w must be finite", fn);
    if (h_full && !store) return fail(RF_ERR_INVALID_ARG, "%s: NULL store", fn);

    rf_rolling_cache c;
    memset(&c, 0, sizeof c);
    c.T = T;
    c.n_cached = n;
    c.rows_per_frame = rows_per_frame;
    c.hidden = hidden;
    c.dtype = dtype;
    c.frame_bytes = rows_per_frame * hidden * elem_bytes(dtype);
    c.magic = kCacheMagic;
    for (int32_t f = 0; f < RF_MAX_FRAMES; ++f) {
        c.before_slot[f] = c.after_slot[f] = -1;
        c.t_before[f] = c.t_after[f] = 0.0;
    }
    // h_before = h_after = the state at t_w: both indices name slot 2i
    for (int32_t i = 0; i < n; ++i) {
        c.before_slot[ids[i]] = c.after_slot[ids[i]] = static_cast<int16_t>(2 * i);
        c.t_before[ids[i]] = c.t_after[ids[i]] = t_w;
    }
    if (h_full) {
        rc = store_after(c, store, h_full, ids, n, stream, fn);
        if (rc != RF_OK) return rc;
    }
    *cache = c;
    return ok();
}

int rf_cache_shift_store(rf_rolling_cache *cache, void *store, const void *h_full, const int32_t *frames,
                         int32_t n, double t_denoise, void *stream) {
    const char *fn = "rf_cache_shift_store";
    int rc = check_cache(cache, fn);
    if (rc != RF_OK) return rc;
    int32_t fr[RF_MAX_FRAMES], k = 0;
    rc = cache_frames(cache, frames, n, fr, &k, fn);
    if (rc != RF_OK) return rc;
    if (!isfinite(t_denoise)) return fail(RF_ERR_INVALID_ARG, "%s: t_denoise must be finite", fn);
    for (int32_t i = 0; i < k; ++i)
        if (!(t_denoise < cache->t_after[fr[i]]))
            return fail(RF_ERR_INVALID_ARG, "%s: t_denoise %g is not below t_after %g of frame %d", fn,
                        t_denoise, cache->t_after[fr[i]], fr[i]);
    rf_rolling_cache c = *cache;
    for (int32_t i = 0; i < k; ++i) {
        const int32_t f = fr[i];
        // h_before <- h_after, t_before <- t_after; h_after goes to the other slot of the pair
        c.before_slot[f] = c.after_slot[f];
        c.t_before[f] = c.t_after[f];
        c.after_slot[f] = static_cast<int16_t>(c.before_slot[f] ^ 1);
        c.t_after[f] = t_denoise;
    }
    if (h_full) {
        rc = store_after(c, store, h_full, fr, k, stream, fn);
        if (rc != RF_OK) return rc;
    }
    *cache = c;
    return ok();
}

// App. B.2's weight with its epsilon, clamped to [0, 1].
static double cache_alpha(const rf_rolling_cache &c, int32_t f, double t_skip) {
    const double a = (c.t_before[f] - t_skip) / (c.t_before[f] - c.t_after[f] + kHiddenEps);
    return a < 0.0 ? 0.0 : (a > 1.0 ? 1.0 : a);
}

int rf_cache_alpha(const rf_rolling_cache *cache, int32_t frame, double t_skip, double *alpha_out) {
    const char *fn = "rf_cache_alpha";
    int rc = check_cache(cache, fn);
    if (rc != RF_OK) return rc;
    if (!alpha_out) return fail(RF_ERR_INVALID_ARG, "%s: NULL output", fn);
    if (frame < 0 || frame >= cache->T) return fail(RF_ERR_RANGE, "%s: frame %d outside [0, %d)", fn, frame, cache->T);
    if (cache->after_slot[frame] < 0) return fail(RF_ERR_INVALID_ARG, "%s: frame %d is not cached", fn, frame);
    if (!isfinite(t_skip)) return fail(RF_ERR_INVALID_ARG, "%s: t_skip must be finite", fn);
    *alpha_out = cache_alpha(*cache, frame, t_skip);
    return ok();
}

int rf_cache_project_kv(const rf_rolling_cache *cache, const void *store, void *k, void *v,
                        const int32_t *frames, int32_t n, double t_skip, void *stream) {
    const char *fn = "rf_cache_project_kv";
    int rc = check_cache(cache, fn);
    if (rc != RF_OK) return rc;
    if (!store || !k || !v) return fail(RF_ERR_INVALID_ARG, "%s: NULL buffer", fn);
    int32_t fr[RF_MAX_FRAMES], cnt = 0;
    rc = cache_frames(cache, frames, n, fr, &cnt, fn);
    if (rc != RF_OK) return rc;
    if (!isfinite(t_skip)) return fail(RF_ERR_INVALID_ARG, "%s: t_skip must be finite", fn);
    if (!aligned16(store) || !aligned16(k) || !aligned16(v))
        return fail(RF_ERR_UNSUPPORTED, "%s: pointers must be 16-byte aligned", fn);
    const int64_t store_bytes = 2 * static_cast<int64_t>(cache->n_cached) * cache->frame_bytes;
    const int64_t kv_bytes = cache->frame_bytes * cache->T;
    if (overlaps(k, kv_bytes, v, kv_bytes) || overlaps(k, kv_bytes, store, store_bytes) ||
        overlaps(v, kv_bytes, store, store_bytes))
        return fail(RF_ERR_INVALID_ARG, "%s: k, v and store must not overlap", fn);
    rf::CacheProjParams p{};
    p.store = store;
    p.k = k;
    p.v = v;
    p.frame_bytes = cache->frame_bytes;
    p.n = cnt;
    p.dtype = cache->dtype;
    for (int32_t i = 0; i < cnt; ++i) {
        const int32_t f = fr[i];
        p.before[i] = cache->before_slot[f];
        p.after[i] = cache->after_slot[f];
        p.dst[i] = static_cast<uint8_t>(f);
        p.alpha[i] = static_cast<float>(cache_alpha(*cache, f, t_skip));
    }
    return launched(rf::launch_cache_projection(p, static_cast<hipStream_t>(stream)), fn);
}

int rf_keyframe_attention_cached(const void *q, const void *k, const void *v, void *out,
                                 const int32_t *keyframe_ids, int32_t M, int32_t T, int32_t H, int32_t W,
                                 int32_t heads, int32_t head_dim, int32_t dtype, const rf_rolling_cache *cache,
                                 const void *store, double t_skip, void *workspace, int64_t workspace_bytes,
                                 void *stream) {
    const char *fn = "rf_keyframe_attention_cached";
    int rc = check_cache(cache, fn);
    if (rc != RF_OK) return rc;
    if (!store) return fail(RF_ERR_INVALID_ARG, "%s: NULL store", fn);
    if (!aligned16(store)) return fail(RF_ERR_UNSUPPORTED, "%s: store must be 16-byte aligned", fn);
    if (!isfinite(t_skip)) return fail(RF_ERR_INVALID_ARG, "%s: t_skip must be finite", fn);
    if (dtype != RF_BF16)
        return fail(RF_ERR_UNSUPPORTED, "%s: the projected keys and values are formed in bf16 attention only", fn);
    if (cache->T != T || H <= 0 || W <= 0 || cache->rows_per_frame != static_cast<int64_t>(H) * W ||
        heads <= 0 || head_dim <= 0 || cache->hidden != static_cast<int64_t>(heads) * head_dim ||
        cache->dtype != dtype)
        return fail(RF_ERR_INVALID_ARG,
                    "%s: the cache (T=%d, %lld rows of %d, dtype %d) does not match the attention "
                    "(T=%d, %d x %d rows of %d x %d, dtype %d)", fn, cache->T,
                    static_cast<long long>(cache->rows_per_frame), cache->hidden, cache->dtype, T, H, W, heads,
                    head_dim, dtype);
    if (!workspace) return fail(RF_ERR_INVALID_ARG, "%s: NULL workspace", fn);
    const CacheForm cf{cache, store, t_skip};
    return attention_call(q, k, v, out, keyframe_ids, M, nullptr, 0, T, H, W, heads, head_dim, dtype, workspace,
                          workspace_bytes, stream, fn, false, &cf);
}

// ---------------------------------------------------------------------------
// Progressive asynchronous schedule (Eq. 2, Alg. 2)
// ---------------------------------------------------------------------------

int rf_async_schedule(int32_t T, int32_t T_w, int32_t T_mid, int32_t n_small, int32_t n_large,
                      rf_step_plan *plan_out, int32_t *n_rhythmic_out, int32_t *n_skipped_out) {
    const char *fn = "rf_async_schedule";
    if (!plan_out) return fail(RF_ERR_INVALID_ARG, "%s: NULL plan", fn);
    if (T < 1 || T > (1 << 20)) return fail(RF_ERR_RANGE, "%s: T = %d outside 1..%d", fn, T, 1 << 20);
    if (T_w < 0 || T_w > T) return fail(RF_ERR_RANGE, "%s: T_w = %d outside 0..T", fn, T_w);
    if (T_mid < 0 || T_mid > T) return fail(RF_ERR_RANGE, "%s: T_mid = %d outside 0..T", fn, T_mid);
    if (n_small < 1 || n_large < 1)
        return fail(RF_ERR_INVALID_ARG, "%s: strides must be >= 1 (n_small=%d n_large=%d)", fn, n_small, n_large);
    int32_t state = T;   // the non-keyframes' state time
    int32_t left = -1;   // the time of their last update
    int32_t n_rp = 0, n_sk = 0;
    for (int32_t t = T, i = 0; t >= 1; --t, ++i) {
        rf_step_plan p;
        p.t = t;
        p.nonkey_to = p.t_start = p.t_end = -1;
        p.alpha = 0.0;
        if (t > T - T_w) {  // synchronous warm-up
            p.phase = RF_STEP_WARMUP;
            p.n_skip = 1;
            p.nonkey_to = state = t - 1;
        } else {
            p.n_skip = t > T_mid ? n_small : n_large;   // Eq. (2)
            if (state == t) {  // the non-keyframes are at t: a Rhythmic Point
                p.phase = RF_STEP_RHYTHMIC;
                p.nonkey_to = t - p.n_skip > 0 ? t - p.n_skip : 0;
                left = t;
                state = p.nonkey_to;
                ++n_rp;
            } else {           // skipped: project on the interval [state, left]
                p.phase = RF_STEP_SKIP;
                p.t_start = left;
                p.t_end = state;
                p.alpha = static_cast<double>(left - t) / static_cast<double>(left - state);
                ++n_sk;
            }
        }
        plan_out[i] = p;
    }
    if (n_rhythmic_out) *n_rhythmic_out = n_rp;
    if (n_skipped_out) *n_skipped_out = n_sk;
    return ok();
}

int rf_probe_mfma_bf16(const void *operands, int32_t workgroups, int32_t rounds, float *sink, void *stream) {
    const char *fn = "rf_probe_mfma_bf16";
    if (!operands || !sink) return fail(RF_ERR_INVALID_ARG, "%s: NULL argument", fn);
    if (workgroups < 1 || workgroups > (1 << 20) || rounds < 1 || rounds > (1 << 22))
        return fail(RF_ERR_RANGE, "%s: workgroups %d (1..2^20) or rounds %d (1..2^22) out of range", fn,
                    workgroups, rounds);
    if (!aligned16(operands) || (reinterpret_cast<uintptr_t>(sink) & 3u))
        return fail(RF_ERR_UNSUPPORTED, "%s: operands must be 16-byte and sink 4-byte aligned", fn);
    return launched(rf::launch_mfma_probe(operands, workgroups, rounds, sink, static_cast<hipStream_t>(stream)),
                    fn);
}

int rf_probe_lds_read(int32_t workgroups, int32_t rounds, int32_t width, uint32_t *sink, uint64_t *ticks,
                      void *stream) {
    const char *fn = "rf_probe_lds_read";
    if (!sink) return fail(RF_ERR_INVALID_ARG, "%s: NULL sink", fn);
    if (width != 16 && width != 8) return fail(RF_ERR_INVALID_ARG, "%s: width %d is not 16 or 8", fn, width);
    if (workgroups < 1 || workgroups > (1 << 20) || rounds < 1 || rounds > (1 << 22))
        return fail(RF_ERR_RANGE, "%s: workgroups %d (1..2^20) or rounds %d (1..2^22) out of range", fn,
                    workgroups, rounds);
    if ((reinterpret_cast<uintptr_t>(sink) & 3u) || (reinterpret_cast<uintptr_t>(ticks) & 7u))
        return fail(RF_ERR_UNSUPPORTED, "%s: sink must be 4-byte and ticks 8-byte aligned", fn);
    return launched(
        rf::launch_lds_read_probe(workgroups, rounds, width, sink, ticks, static_cast<hipStream_t>(stream)), fn);
}

int rf_probe_hbm_read(const void *src, int64_t bytes, int32_t workgroups, uint32_t *sink, void *stream) {
    const char *fn = "rf_probe_hbm_read";
    if (!src || !sink) return fail(RF_ERR_INVALID_ARG, "%s: NULL argument", fn);
    if (bytes < 16 || bytes % 16 != 0)
        return fail(RF_ERR_INVALID_ARG, "%s: bytes = %lld must be a positive multiple of 16", fn,
                    static_cast<long long>(bytes));
    if (workgroups < 1 || workgroups > (1 << 20))
        return fail(RF_ERR_RANGE, "%s: workgroups %d out of range (1..2^20)", fn, workgroups);
    if (!aligned16(src) || (reinterpret_cast<uintptr_t>(sink) & 3u))
        return fail(RF_ERR_UNSUPPORTED, "%s: src must be 16-byte and sink 4-byte aligned", fn);
    return launched(rf::launch_hbm_read_probe(src, bytes, workgroups, sink, static_cast<hipStream_t>(stream)), fn);
}

}  // extern "C"
