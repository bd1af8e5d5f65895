// Rolling-cache projection (App. B.2) for gfx950.
//
// At a skipped step every cached non-keyframe provides its projected hidden
// state h_hat = (1 - alpha) h_before + alpha h_after as both its key and its
// value. This kernel forms h_hat element by element from the two cache slots
// and writes it into the frame's block of K and of V, so the attention kernel
// then reads one ordinary [S][heads][head_dim] key and value sequence.
//
// Bandwidth-bound elementwise work (two 16-byte loads and two 16-byte stores
// per vector, no LDS, no matrix cores). A workgroup covers one contiguous
// chunk of one frame, so the slot offsets and alpha are workgroup-uniform and
// live in scalar registers; every access is a coalesced streaming access.
#include "rf_internal.h"

namespace rf {
namespace {

// Launch shape: one wave per workgroup, one 16-byte vector per thread and
// stream (the fastest of 64..512 threads x 1..4 vectors measured on MI355X).
#ifndef RF_CACHE_THREADS
#define RF_CACHE_THREADS 64
#endif
#ifndef RF_CACHE_UNROLL
#define RF_CACHE_UNROLL 1
#endif
constexpr int kThreads = RF_CACHE_THREADS;
constexpr int kUnroll = RF_CACHE_UNROLL;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4_t ld16(const u32x4_t *p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st16(u32x4_t *p, u32x4_t v) { __builtin_nontemporal_store(v, p); }

struct CacheKArgs {
    const u32x4_t *store;
    u32x4_t *k;
    u32x4_t *v;
    int64_t frame_vecs;       // 16-byte vectors per frame block
    int32_t blocks_per_frame;
    int16_t before[kMaxFrames];
    int16_t after[kMaxFrames];
    uint8_t dst[kMaxFrames];
    float alpha[kMaxFrames];
};

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round to nearest even; NaN stays NaN.
__device__ inline uint32_t to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

template <bool kBf16>
__device__ inline u32x4_t lerp_vec(u32x4_t b, u32x4_t a, float al, float oma) {
    const uint32_t wb[4] = {b.x, b.y, b.z, b.w};
    const uint32_t wa[4] = {a.x, a.y, a.z, a.w};
    uint32_t r[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (kBf16) {
            const float lo = fmaf(al, bf16_lo(wa[e]), oma * bf16_lo(wb[e]));
            const float hi = fmaf(al, bf16_hi(wa[e]), oma * bf16_hi(wb[e]));
            r[e] = to_bf16(lo) | (to_bf16(hi) << 16);
        } else {
            r[e] = __float_as_uint(fmaf(al, __uint_as_float(wa[e]), oma * __uint_as_float(wb[e])));
        }
    }
    return u32x4_t{r[0], r[1], r[2], r[3]};
}

template <bool kBf16>
__global__ __launch_bounds__(kThreads) void cache_project_kernel(const CacheKArgs a) {
    const int m = blockIdx.x / a.blocks_per_frame;
    const int chunk = blockIdx.x - m * a.blocks_per_frame;
    const u32x4_t *hb = a.store + static_cast<int64_t>(a.before[m]) * a.frame_vecs;
    const u32x4_t *ha = a.store + static_cast<int64_t>(a.after[m]) * a.frame_vecs;
    const int64_t out = static_cast<int64_t>(a.dst[m]) * a.frame_vecs;
    u32x4_t *k = a.k + out;
    u32x4_t *v = a.v + out;
    const float al = a.alpha[m];
    // (1 - alpha) in float: exactly 1 at alpha = 0 and 0 at alpha = 1, so the
    // endpoints return the cached states bit for bit.
    const float oma = 1.0f - al;
    const int64_t base = static_cast<int64_t>(chunk) * kThreads * kUnroll + threadIdx.x;
    u32x4_t xb[kUnroll], xa[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const int64_t i = base + u * kThreads;
        if (i < a.frame_vecs) {
            xb[u] = ld16(hb + i);
            xa[u] = ld16(ha + i);
        }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const int64_t i = base + u * kThreads;
        if (i < a.frame_vecs) {
            const u32x4_t r = lerp_vec<kBf16>(xb[u], xa[u], al, oma);
            st16(k + i, r);
            st16(v + i, r);
        }
    }
}

}  // namespace

hipError_t launch_cache_projection(const CacheProjParams &p, hipStream_t stream) {
    CacheKArgs a{};
    a.store = static_cast<const u32x4_t *>(p.store);
    a.k = static_cast<u32x4_t *>(p.k);
    a.v = static_cast<u32x4_t *>(p.v);
    a.frame_vecs = p.frame_bytes / 16;
    for (int m = 0; m < p.n; ++m) {
        a.before[m] = p.before[m];
        a.after[m] = p.after[m];
        a.dst[m] = p.dst[m];
        a.alpha[m] = p.alpha[m];
    }
    const int64_t per_block = static_cast<int64_t>(kThreads) * kUnroll;
    const int64_t bpf = (a.frame_vecs + per_block - 1) / per_block;
    const int64_t blocks = bpf * p.n;
    if (bpf > 0x7fffffffLL || blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    a.blocks_per_frame = static_cast<int32_t>(bpf);
    const dim3 grid(static_cast<uint32_t>(blocks)), block(kThreads);
    if (p.dtype == RF_BF16) hipLaunchKernelGGL(cache_project_kernel<true>, grid, block, 0, stream, a);
    else hipLaunchKernelGGL(cache_project_kernel<false>, grid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace rf
