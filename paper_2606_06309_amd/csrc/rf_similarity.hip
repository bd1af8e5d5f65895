// Cosine similarity between latent frames for gfx950 (content-aware keyframe
// selection: Eq. (1) compares frames by cosine similarity, Sec. 3.1; Alg. 1).
//
// The frames of a batch element form a matrix X = [T][F] (F = C*H*W elements,
// channel after channel); the similarity is the Gram matrix G = X X^T scaled
// by the frame norms. F is large (10^5 .. 10^6) and T small (<= 256), so the
// work is a bandwidth-bound reduction over F, split into chunks:
//  1. gram_partial_kernel: a workgroup walks a run of consecutive feature
//     chunks; for each it stages the chunk of all T frames in LDS (as
//     [element][frame], frames padded to a multiple of 4) and accumulates 4x4
//     frame blocks of the Gram matrix in double precision (fp32 x fp32
//     products are exact in double). The run's partial blocks go to the
//     workspace. fp32 latents of at most 64 frames whose planes are a
//     multiple of 4 take gram_partial_dma_kernel instead: the chunk's frame
//     rows stream from HBM into LDS through the load units, double-buffered.
//     At most 512 workgroups in all (one round at two per compute unit),
//     at least one per batch element, cover the batch.
//  2. gram_reduce_kernel: a workgroup per 4x4 block pair sums the partials of
//     all runs in a fixed order (deterministic) into the output matrix.
//  3. cosine_normalize_kernel: one workgroup per batch element turns G into
//     G_ij / (max(|x_i|, eps) * max(|x_j|, eps)) in place.
#include "rf_internal.h"

namespace rf {
namespace {

constexpr int kThreads = 256;
constexpr int kTileFloats = 16384;     // LDS floats for one staged chunk (64 KB)
constexpr int kMaxChunk = 256;         // feature elements per chunk
constexpr double kNormFloor = 1e-8;
#ifndef RF_SIM_TARGET_WORKGROUPS
#define RF_SIM_TARGET_WORKGROUPS 512
#endif
constexpr int64_t kTargetWorkgroups = RF_SIM_TARGET_WORKGROUPS;   // partial-Gram workgroups per launch
constexpr int kNarrowFrames = 64;            // padded frame count of the register-sum path
static_assert(kNarrowFrames * kThreads <= kTileFloats, "narrow chunk must fit the LDS tile");

typedef float f32x4_t __attribute__((ext_vector_type(4)));

struct PartialArgs {
    const void *x;
    double *ws;
    int64_t plane;
    int64_t chunks_per_plane;
    int64_t n_chunks;
    int64_t run;              // chunks per workgroup
    int64_t n_runs;           // workgroups per batch element
    int32_t C, T, Tp, NB, NBP, L, KS;   // KS element slices per block pair (NBP < kThreads)
};

__device__ inline float load_elem(const void *x, int64_t i, bool bf16) {
    if (bf16) return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t *>(x)[i]) << 16);
    return static_cast<const float *>(x)[i];
}

// Block pair index -> (bi, bj), bi <= bj, enumerated row after row.
__device__ inline void block_pair(int bp, int NB, int &bi, int &bj) {
    int row = 0, rem = bp;
    while (rem >= NB - row) {
        rem -= NB - row;
        ++row;
    }
    bi = row;
    bj = row + rem;
}

// kWide = false (T <= 64): chunks of kThreads elements, at most kThreads block
// pairs; each thread owns one block pair (or an element slice of one, KS > 1)
// for the whole run of chunks and keeps its 16 sums in registers. kWide = true
// (T > 64): shorter chunks, runs of one chunk; a thread walks several block
// pairs and writes each one's sums when done.
template <bool kBf16, bool kWide>
__global__ __launch_bounds__(kThreads) void gram_partial_kernel(const PartialArgs a) {
    extern __shared__ __attribute__((aligned(16))) float tile[];   // Tp * L floats (<= kTileFloats)
    const int64_t b = blockIdx.x / a.n_runs;
    const int64_t rn = blockIdx.x - b * a.n_runs;
    const int tid = threadIdx.x;
    const int n_items = a.KS > 1 ? a.NBP * a.KS : a.NBP;
    double *dst = a.ws + (b * a.n_runs + rn) * a.NBP * 16;

    auto stage = [&](int64_t chunk) {   // wide path: [element k][frame f], padding as 0
        const int64_t c = chunk / a.chunks_per_plane;
        const int64_t p0 = (chunk - c * a.chunks_per_plane) * a.L;
        const int64_t frame0 = (b * a.C + c) * a.T;
        for (int idx = tid; idx < a.Tp * a.L; idx += kThreads) {
            const int f = idx / a.L, k = idx - f * a.L;
            float v = 0.0f;
            if (f < a.T && p0 + k < a.plane) v = load_elem(a.x, (frame0 + f) * a.plane + p0 + k, kBf16);
            tile[k * a.Tp + f] = v;
        }
    };
    // 16 sums of one 4x4 frame block pair over this chunk's elements k = ks, ks + KS, ...
    auto accumulate = [&](int item, double (&acc)[16]) {
        const int bp = a.KS > 1 ? item / a.KS : item;
        const int ks = a.KS > 1 ? item - bp * a.KS : 0;
        int bi, bj;
        block_pair(bp, a.NB, bi, bj);
        const f32x4_t *t4 = reinterpret_cast<const f32x4_t *>(tile);
        const int row4 = a.Tp / 4;
        auto step = [&](int k) {
            const f32x4_t u = t4[k * row4 + bi];
            const f32x4_t w = t4[k * row4 + bj];
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    acc[r * 4 + q] = fma(static_cast<double>(u[r]), static_cast<double>(w[q]), acc[r * 4 + q]);
        };
        int k = ks;
        for (; k + 3 * a.KS < a.L; k += 4 * a.KS) {   // four elements' reads in flight
            step(k);
            step(k + a.KS);
            step(k + 2 * a.KS);
            step(k + 3 * a.KS);
        }
        for (; k < a.L; k += a.KS) step(k);
    };

    if constexpr (kWide) {
        stage(rn);   // a run is one chunk
        __syncthreads();
        for (int item = tid; item < n_items; item += kThreads) {
            double acc[16];
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[e] = 0.0;
            accumulate(item, acc);
#pragma unroll
            for (int e = 0; e < 16; ++e) dst[item * 16 + e] = acc[e];
        }
    } else {
        double acc[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[e] = 0.0;
        const int64_t c0 = rn * a.run;
        const int64_t c1 = (c0 + a.run < a.n_chunks) ? c0 + a.run : a.n_chunks;
        for (int64_t chunk = c0; chunk < c1; ++chunk) {
            const int64_t c = chunk / a.chunks_per_plane;
            const int64_t p0 = (chunk - c * a.chunks_per_plane) * a.L;
            const bool in = p0 + tid < a.plane;
            const int64_t src = (b * a.C + c) * a.T * a.plane + (in ? p0 + tid : 0);
            __syncthreads();   // the previous chunk is no longer read
            // thread = element: its frames' values go out kBatch loads at a time
            // (addresses clamped to a valid element, the values then masked) so
            // the loads overlap instead of waiting one by one
            constexpr int kBatch = 16;
            for (int f0 = 0; f0 < a.Tp; f0 += kBatch) {
                float v[kBatch];
#pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const int f = f0 + u;
                    const int fc = f < a.T ? f : a.T - 1;
                    const float x = load_elem(a.x, src + static_cast<int64_t>(fc) * a.plane, kBf16);
                    v[u] = (f < a.T && in) ? x : 0.0f;
                }
#pragma unroll
                for (int u = 0; u < kBatch; ++u)
                    if (f0 + u < a.Tp) tile[tid * a.Tp + f0 + u] = v[u];
            }
            __syncthreads();
            if (tid < n_items) accumulate(tid, acc);
        }
        if (a.KS == 1) {
            if (tid < n_items) {
#pragma unroll
                for (int e = 0; e < 16; ++e) dst[tid * 16 + e] = acc[e];
            }
        } else {
            double *red = reinterpret_cast<double *>(tile);   // NBP * KS * 16 <= kThreads * 16 doubles
            __syncthreads();
            if (tid < n_items) {
#pragma unroll
                for (int e = 0; e < 16; ++e) red[tid * 16 + e] = acc[e];
            }
            __syncthreads();
            for (int t = tid; t < a.NBP * 16; t += kThreads) {
                const int bq = t / 16, e = t - bq * 16;
                double sum = 0.0;
                for (int j = 0; j < a.KS; ++j) sum += red[(bq * a.KS + j) * 16 + e];
                dst[t] = sum;
            }
        }
    }
}

// 16 bytes per lane from a buffer resource straight into LDS (lane l lands at
// dst + 16 l); offsets at or past the resource's range read as zero.
__device__ __forceinline__ void sim_load_lds16(__amdgpu_buffer_rsrc_t r, __attribute__((address_space(3))) void *dst,
                                               int voffset) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voffset, 0, 0, 0);
}

constexpr int kBufferWord3 = 0x00020000;   // raw buffer resource, gfx9-class GPUs

// A pointer every lane holds the same value of, rebuilt from its first lane.
__device__ __forceinline__ void *sim_uniform_ptr(const void *p) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
    return reinterpret_cast<void *>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Narrow path for fp32 latents whose planes are a multiple of 4 elements: a
// chunk's frame rows (256 elements = 1 KB each, [frame][element] order) go
// from HBM straight into LDS, one wave-wide 16-byte-per-lane load per row,
// double-buffered so the next chunk streams in while this one is summed;
// elements past the plane read as zero through the load's range check, the
// padding frames' rows are zeroed once. A thread accumulates its 4x4 block pair
// over groups of 4 consecutive elements (8 LDS reads of 16 bytes per 64 fused
// multiply-adds).
__global__ __launch_bounds__(kThreads) void gram_partial_dma_kernel(const PartialArgs a) {
    constexpr int kL = kThreads;
    constexpr int kGroups = kL / 4;
    extern __shared__ __attribute__((aligned(1024))) float tile[];   // 2 x [Tp][kL] floats
    const int64_t b = blockIdx.x / a.n_runs;
    const int64_t rn = blockIdx.x - b * a.n_runs;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n_items = a.KS > 1 ? a.NBP * a.KS : a.NBP;
    double *dst = a.ws + (b * a.n_runs + rn) * a.NBP * 16;
    const int buf_floats = a.Tp * kL;

    // padding frames: zero rows in both buffers (never loaded)
    for (int i = tid; i < 2 * (a.Tp - a.T) * kL; i += kThreads) {
        const int bufi = i / ((a.Tp - a.T) * kL);
        const int rem = i - bufi * (a.Tp - a.T) * kL;
        tile[bufi * buf_floats + a.T * kL + rem] = 0.0f;
    }

    const int64_t c0 = rn * a.run;
    const int64_t c1 = (c0 + a.run < a.n_chunks) ? c0 + a.run : a.n_chunks;
    // loads of chunk `chunk` into buffer `bufi`: wave w takes frames w, w + 4, ...
    auto issue = [&](int64_t chunk, int bufi) {
        const int64_t c = chunk / a.chunks_per_plane;
        const int64_t p0 = (chunk - c * a.chunks_per_plane) * kL;
        const float *base = static_cast<const float *>(a.x) + ((b * a.C + c) * a.T) * a.plane + p0;
        const int64_t left = (static_cast<int64_t>(a.T) * a.plane - p0) * 4;
        const int32_t rec = __builtin_amdgcn_readfirstlane(
            static_cast<int32_t>(left < 0x7fffffffLL ? left : 0x7fffffffLL));
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(sim_uniform_ptr(base), 0, rec,
                                                                            kBufferWord3);
        const bool in = p0 + 4 * lane < a.plane;
        for (int f = wave; f < a.T; f += kThreads / 64) {
            const int off = in ? static_cast<int>(f * a.plane * 4 + lane * 16) : static_cast<int>(0xfffffff0u);
            sim_load_lds16(r, (__attribute__((address_space(3))) void *)(
                                  reinterpret_cast<char *>(tile) + (bufi * buf_floats + f * kL) * 4),
                           off);
        }
    };
    auto done = [&]() {
        __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0): this wave's loads have reached LDS
        __syncthreads();
    };

    double acc[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.0;
    int bi = 0, bj = 0, ks = 0;
    if (tid < n_items) {
        const int bp = a.KS > 1 ? tid / a.KS : tid;
        ks = a.KS > 1 ? tid - bp * a.KS : 0;
        block_pair(bp, a.NB, bi, bj);
    }
    auto sum_chunk = [&](int bufi) {
        if (tid >= n_items) return;
        const f32x4_t *t4 = reinterpret_cast<const f32x4_t *>(tile + bufi * buf_floats);
        for (int g = ks; g < kGroups; g += a.KS) {
            f32x4_t u[4], w[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                u[r] = t4[(4 * bi + r) * kGroups + g];
                w[r] = t4[(4 * bj + r) * kGroups + g];
            }
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        acc[r * 4 + q] = fma(static_cast<double>(u[r][e]), static_cast<double>(w[q][e]),
                                             acc[r * 4 + q]);
        }
    };
    if (c0 < c1) issue(c0, 0);
    done();
    for (int64_t chunk = c0; chunk < c1; chunk += 2) {
        if (chunk + 1 < c1) issue(chunk + 1, 1);
        sum_chunk(0);
        done();
        if (chunk + 1 >= c1) break;
        if (chunk + 2 < c1) issue(chunk + 2, 0);
        sum_chunk(1);
        done();
    }
    if (a.KS == 1) {
        if (tid < n_items) {
#pragma unroll
            for (int e = 0; e < 16; ++e) dst[tid * 16 + e] = acc[e];
        }
    } else {
        double *red = reinterpret_cast<double *>(tile);
        __syncthreads();
        if (tid < n_items) {
#pragma unroll
            for (int e = 0; e < 16; ++e) red[tid * 16 + e] = acc[e];
        }
        __syncthreads();
        for (int t = tid; t < a.NBP * 16; t += kThreads) {
            const int bq = t / 16, e = t - bq * 16;
            double sum = 0.0;
            for (int j = 0; j < a.KS; ++j) sum += red[(bq * a.KS + j) * 16 + e];
            dst[t] = sum;
        }
    }
}

struct ReduceArgs {
    const double *ws;
    double *sim;
    int64_t n_runs;
    int32_t T, NB, NBP;
};

// One workgroup per (batch element, block pair): kReduceLanes lanes per Gram
// entry sum the runs' partials with stride kReduceLanes, then the lane sums
// are added in lane order.
constexpr int kReduceThreads = 1024;
constexpr int kReduceLanes = kReduceThreads / 16;

__global__ __launch_bounds__(kReduceThreads) void gram_reduce_kernel(const ReduceArgs a) {
    __shared__ double lane_sum[kReduceThreads];
    const int64_t b = blockIdx.x / a.NBP;
    const int bp = static_cast<int>(blockIdx.x - b * a.NBP);
    const int e = threadIdx.x % 16, lane = threadIdx.x / 16;
    const double *src = a.ws + (b * a.n_runs * a.NBP + bp) * 16 + e;
    double s = 0.0;
#pragma unroll 4
    for (int64_t r = lane; r < a.n_runs; r += kReduceLanes) s += src[r * a.NBP * 16];
    lane_sum[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x < 16) {
        double g = 0.0;
        for (int l = 0; l < kReduceLanes; ++l) g += lane_sum[l * 16 + e];
        int bi, bj;
        block_pair(bp, a.NB, bi, bj);
        const int i = 4 * bi + e / 4, j = 4 * bj + e % 4;
        if (i < a.T && j < a.T) {
            double *out = a.sim + b * a.T * a.T;
            out[static_cast<int64_t>(i) * a.T + j] = g;
            out[static_cast<int64_t>(j) * a.T + i] = g;   // same value twice on diagonal blocks
        }
    }
}

__global__ __launch_bounds__(kThreads) void cosine_normalize_kernel(double *sim, int32_t T) {
    __shared__ double norm[kMaxFrames];
    double *g = sim + static_cast<int64_t>(blockIdx.x) * T * T;
    for (int i = threadIdx.x; i < T; i += kThreads) {
        const double n = sqrt(g[static_cast<int64_t>(i) * T + i]);
        norm[i] = n > kNormFloor ? n : kNormFloor;
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < T * T; idx += kThreads) {
        const int i = idx / T, j = idx - i * T;
        g[idx] = g[idx] / (norm[i] * norm[j]);
    }
}

}  // namespace

SimGeometry similarity_geometry(int32_t B, int32_t C, int32_t T, int64_t plane) {
    SimGeometry g{};
    g.Tp = (T + 3) / 4 * 4;
    g.NB = g.Tp / 4;
    g.NBP = g.NB * (g.NB + 1) / 2;
    // T <= 64: chunks of exactly kThreads elements; larger T: as many as fit the tile
    const int L = (kTileFloats / g.Tp) / 16 * 16;
    g.L = g.Tp <= kNarrowFrames ? kThreads : (L < kMaxChunk ? L : kMaxChunk);
    g.chunks_per_plane = (plane + g.L - 1) / g.L;
    g.n_chunks = static_cast<int64_t>(C) * g.chunks_per_plane;
    // at most kTargetWorkgroups workgroups over the whole batch (one round at two
    // per compute unit: a partly filled second round would double the time of
    // the workgroups in it), at least one per batch element; each is a run of
    // chunks (one chunk per run when a thread has to walk several block pairs)
    const int64_t per_b = kTargetWorkgroups / B > 0 ? kTargetWorkgroups / B : 1;
    g.run = g.Tp > kNarrowFrames ? 1 : (g.n_chunks + per_b - 1) / per_b;
    g.n_runs = (g.n_chunks + g.run - 1) / g.run;
    g.workspace_bytes = static_cast<int64_t>(B) * g.n_runs * g.NBP * 16 * static_cast<int64_t>(sizeof(double));
    return g;
}

hipError_t launch_similarity(const SimParams &p, hipStream_t stream) {
    const SimGeometry g = similarity_geometry(p.B, p.C, p.T, p.plane);
    PartialArgs a{};
    a.x = p.latents;
    a.ws = p.workspace;
    a.plane = p.plane;
    a.chunks_per_plane = g.chunks_per_plane;
    a.n_chunks = g.n_chunks;
    a.run = g.run;
    a.n_runs = g.n_runs;
    a.C = p.C;
    a.T = p.T;
    a.Tp = g.Tp;
    a.NB = g.NB;
    a.NBP = g.NBP;
    a.L = g.L;
    a.KS = g.NBP >= kThreads ? 1 : kThreads / g.NBP;
    const int64_t blocks = static_cast<int64_t>(p.B) * g.n_runs;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<uint32_t>(blocks)), block(kThreads);
    const bool wide = g.Tp > kNarrowFrames;
    // the staged chunk, or the element-slice sums of the narrow path if larger
    size_t lds = static_cast<size_t>(g.Tp) * g.L * sizeof(float);
    const size_t red = static_cast<size_t>(kThreads) * 16 * sizeof(double);
    if (!wide && a.KS > 1 && lds < red) lds = red;
    // fp32, at most 64 frames, planes of a multiple of 4 elements and frame blocks
    // addressable with 32-bit offsets: chunks streamed into LDS by the load units
    const bool dma = p.dtype == RF_F32 && !wide && p.plane % 4 == 0 &&
                     static_cast<int64_t>(p.T) * p.plane * 4 < 0x7ffff000LL;
    if (dma) {
        const size_t two = 2 * static_cast<size_t>(g.Tp) * g.L * sizeof(float);
        const size_t bytes = two > lds ? two : lds;
        if (bytes > 65536) {   // more than 64 KB of dynamic LDS must be allowed explicitly
            const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&gram_partial_dma_kernel),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     static_cast<int>(bytes));
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(gram_partial_dma_kernel, grid, block, bytes, stream, a);
    } else if (p.dtype == RF_BF16) {
        if (wide) hipLaunchKernelGGL((gram_partial_kernel<true, true>), grid, block, lds, stream, a);
        else hipLaunchKernelGGL((gram_partial_kernel<true, false>), grid, block, lds, stream, a);
    } else {
        if (wide) hipLaunchKernelGGL((gram_partial_kernel<false, true>), grid, block, lds, stream, a);
        else hipLaunchKernelGGL((gram_partial_kernel<false, false>), grid, block, lds, stream, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    ReduceArgs r{};
    r.ws = p.workspace;
    r.sim = p.sim;
    r.n_runs = g.n_runs;
    r.T = p.T;
    r.NB = g.NB;
    r.NBP = g.NBP;
    const int64_t rblocks = static_cast<int64_t>(p.B) * g.NBP;
    if (rblocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(gram_reduce_kernel, dim3(static_cast<uint32_t>(rblocks)), dim3(kReduceThreads), 0, stream, r);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(cosine_normalize_kernel, dim3(static_cast<uint32_t>(p.B)), dim3(kThreads), 0, stream,
                       p.sim, p.T);
    return hipGetLastError();
}

}  // namespace rf
