// Latent trajectory projection, Eq. (3) (Sec. 3.2.4), for gfx950.
//
// out = fmaf(alpha, z_end, (1 - alpha) * z_start) for non-keyframe planes,
// out = z_end (the current state) for keyframe planes.
//
// Bandwidth-bound elementwise work: no matrix cores, no LDS. A workgroup
// covers one contiguous chunk of one (b, c, f) plane, so alpha and the
// keyframe flag are workgroup-uniform (scalar registers) and every access is
// a coalesced 128-bit streaming load or store.
#include "rf_internal.h"

namespace rf {
namespace {

// Launch shape (measured on MI355X against 64..1024 threads and 1..4 vectors per
// thread): 128 threads x 2 vectors per workgroup, streaming (nontemporal)
// 16-byte accesses, since each byte is touched once.
#ifndef RF_PROJ_THREADS
#define RF_PROJ_THREADS 128
#endif
#ifndef RF_PROJ_UNROLL
#define RF_PROJ_UNROLL 2
#endif
constexpr int kThreads = RF_PROJ_THREADS;
constexpr int kUnroll = RF_PROJ_UNROLL;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4_t ld16(const u32x4_t *p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st16(u32x4_t *p, u32x4_t v) { __builtin_nontemporal_store(v, p); }

struct ProjKArgs {
    const void *lat;
    void *out;
    int64_t plane;          // elements per (b, c, f) plane
    int64_t ctp;            // C * T * plane
    int32_t C, T;
    int32_t blocks_per_plane;
    int32_t skip_keyframes;
    float alpha;
    float one_minus_alpha;
    uint8_t is_key[kMaxFrames];
};

__device__ inline float bf16_bits_to_float(uint32_t b16) { return __uint_as_float(b16 << 16); }

// Round to nearest even; NaN stays NaN.
__device__ inline uint32_t float_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ inline float lerp3(float a, float b, float alpha, float oma) {
    return fmaf(alpha, b, oma * a);
}

// One workgroup: kThreads * kUnroll 16-byte vectors of one plane.
// Requires plane % (elements per 16 bytes) == 0 and 16-byte aligned bases.
template <bool kBf16>
__global__ __launch_bounds__(kThreads) void project_vec_kernel(const ProjKArgs a) {
    constexpr int kPer = kBf16 ? 8 : 4;  // elements per 16-byte vector
    const int64_t pl = blockIdx.x / a.blocks_per_plane;
    const int chunk = blockIdx.x - static_cast<int>(pl * a.blocks_per_plane);
    const int f = static_cast<int>(pl % a.T);
    const int64_t bc = pl / a.T;
    const int64_t c = bc % a.C, b = bc / a.C;
    const bool key = a.is_key[f] != 0;
    if (key && a.skip_keyframes) return;

    const int64_t in_plane = (c * a.T + f) * a.plane;
    const u32x4_t *s0 = reinterpret_cast<const u32x4_t *>(
        static_cast<const char *>(a.lat) + (b * 2 * a.ctp + in_plane) * (kBf16 ? 2 : 4));
    const u32x4_t *s1 = reinterpret_cast<const u32x4_t *>(
        static_cast<const char *>(a.lat) + ((b * 2 + 1) * a.ctp + in_plane) * (kBf16 ? 2 : 4));
    u32x4_t *o = reinterpret_cast<u32x4_t *>(
        static_cast<char *>(a.out) + (b * a.ctp + in_plane) * (kBf16 ? 2 : 4));
    const int64_t nvec = a.plane / kPer;
    const int64_t base = static_cast<int64_t>(chunk) * kThreads * kUnroll + threadIdx.x;

    if (key) {  // keyframe: current state passes through
        u32x4_t r[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t i = base + u * kThreads;
            if (i < nvec) r[u] = ld16(s1 + i);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t i = base + u * kThreads;
            if (i < nvec) st16(o + i, r[u]);
        }
        return;
    }

    u32x4_t x0[kUnroll], x1[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const int64_t i = base + u * kThreads;
        if (i < nvec) {
            x0[u] = ld16(s0 + i);
            x1[u] = ld16(s1 + i);
        }
    }
    const float al = a.alpha, oma = a.one_minus_alpha;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const int64_t i = base + u * kThreads;
        if (i >= nvec) continue;
        const uint32_t w0[4] = {x0[u].x, x0[u].y, x0[u].z, x0[u].w};
        const uint32_t w1[4] = {x1[u].x, x1[u].y, x1[u].z, x1[u].w};
        uint32_t r[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (kBf16) {
                const float lo = lerp3(bf16_bits_to_float(w0[e] & 0xffffu),
                                       bf16_bits_to_float(w1[e] & 0xffffu), al, oma);
                const float hi = lerp3(bf16_bits_to_float(w0[e] >> 16),
                                       bf16_bits_to_float(w1[e] >> 16), al, oma);
                r[e] = float_to_bf16_bits(lo) | (float_to_bf16_bits(hi) << 16);
            } else {
                r[e] = __float_as_uint(lerp3(__uint_as_float(w0[e]), __uint_as_float(w1[e]), al, oma));
            }
        }
        st16(o + i, u32x4_t{r[0], r[1], r[2], r[3]});
    }
}

// Element-at-a-time form for planes whose size is not a multiple of the vector.
template <bool kBf16>
__global__ __launch_bounds__(kThreads) void project_scalar_kernel(const ProjKArgs a) {
    const int64_t pl = blockIdx.x / a.blocks_per_plane;
    const int chunk = blockIdx.x - static_cast<int>(pl * a.blocks_per_plane);
    const int f = static_cast<int>(pl % a.T);
    const int64_t bc = pl / a.T;
    const int64_t c = bc % a.C, b = bc / a.C;
    const bool key = a.is_key[f] != 0;
    if (key && a.skip_keyframes) return;
    const int64_t in_plane = (c * a.T + f) * a.plane;
    const int64_t i0 = b * 2 * a.ctp + in_plane, i1 = (b * 2 + 1) * a.ctp + in_plane;
    const int64_t io = b * a.ctp + in_plane;
    const int64_t base = static_cast<int64_t>(chunk) * kThreads * kUnroll + threadIdx.x;
    for (int u = 0; u < kUnroll; ++u) {
        const int64_t e = base + u * kThreads;
        if (e >= a.plane) break;
        if (kBf16) {
            const uint16_t *l = static_cast<const uint16_t *>(a.lat);
            uint16_t *o = static_cast<uint16_t *>(a.out);
            const uint32_t z1 = l[i1 + e];
            if (key) {
                o[io + e] = static_cast<uint16_t>(z1);
            } else {
                const float r = lerp3(bf16_bits_to_float(l[i0 + e]), bf16_bits_to_float(z1),
                                      a.alpha, a.one_minus_alpha);
                o[io + e] = static_cast<uint16_t>(float_to_bf16_bits(r));
            }
        } else {
            const float *l = static_cast<const float *>(a.lat);
            float *o = static_cast<float *>(a.out);
            o[io + e] = key ? l[i1 + e] : lerp3(l[i0 + e], l[i1 + e], a.alpha, a.one_minus_alpha);
        }
    }
}

}  // namespace

hipError_t launch_projection(const ProjParams &p, hipStream_t stream) {
    ProjKArgs a{};
    a.lat = p.latents;
    a.out = p.out;
    a.plane = p.plane;
    a.ctp = static_cast<int64_t>(p.C) * p.T * p.plane;
    a.C = p.C;
    a.T = p.T;
    a.skip_keyframes = p.skip_keyframes;
    a.alpha = p.alpha;
    // (1 - alpha) in float: exactly 1 at alpha = 0 and exactly 0 at alpha = 1,
    // so the endpoints return z_start and z_end bit for bit.
    a.one_minus_alpha = 1.0f - p.alpha;
    for (int f = 0; f < p.T; ++f) a.is_key[f] = p.is_key[f];
    const bool bf16 = p.dtype == RF_BF16;
    const int per = bf16 ? 8 : 4;
    const bool vec = p.plane % per == 0;
    const int64_t units = vec ? p.plane / per : p.plane;
    const int64_t per_block = static_cast<int64_t>(kThreads) * kUnroll;
    a.blocks_per_plane = static_cast<int32_t>((units + per_block - 1) / per_block);
    const int64_t planes = static_cast<int64_t>(p.B) * p.C * p.T;
    const int64_t blocks = planes * a.blocks_per_plane;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<uint32_t>(blocks)), block(kThreads);
    if (vec) {
        if (bf16) hipLaunchKernelGGL(project_vec_kernel<true>, grid, block, 0, stream, a);
        else hipLaunchKernelGGL(project_vec_kernel<false>, grid, block, 0, stream, a);
    } else {
        if (bf16) hipLaunchKernelGGL(project_scalar_kernel<true>, grid, block, 0, stream, a);
        else hipLaunchKernelGGL(project_scalar_kernel<false>, grid, block, 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace rf
