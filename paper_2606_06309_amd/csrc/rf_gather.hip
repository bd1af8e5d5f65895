// Frame gather / scatter for gfx950: bit-exact copies of whole frames.
//
// A frame-major token sequence stores each frame as one contiguous block of
// rows_per_frame rows, so gathering the keyframes' rows is a copy of M
// contiguous blocks, and scattering is the reverse; storing frames into the
// rolling cache's slots is the same copy with another index pair per block. Bandwidth-bound: every
// access is a coalesced 16-byte load or store, no LDS, no matrix cores.
#include "rf_internal.h"

namespace rf {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Launch shape: one wave per workgroup copying 1 KB, one 16-byte vector per
// thread (the fastest of 64..1024 threads x 1..4 vectors measured on MI355X:
// many small workgroups keep more copies in flight than few large ones).
#ifndef RF_COPY_THREADS
#define RF_COPY_THREADS 64
#endif
#ifndef RF_COPY_UNROLL
#define RF_COPY_UNROLL 1
#endif
constexpr int kThreads = RF_COPY_THREADS;
constexpr int kUnroll = RF_COPY_UNROLL;

struct CopyKArgs {
    const u32x4 *src;
    u32x4 *dst;
    int64_t frame_vecs;       // 16-byte vectors per frame
    int32_t blocks_per_frame;
    int32_t src_idx[kMaxFrames];
    int32_t dst_idx[kMaxFrames];
};

__global__ __launch_bounds__(kThreads) void frame_copy_kernel(const CopyKArgs a) {
    const int m = blockIdx.x / a.blocks_per_frame;
    const int chunk = blockIdx.x - m * a.blocks_per_frame;
    const int64_t src_frame = a.src_idx[m];
    const int64_t dst_frame = a.dst_idx[m];
    const u32x4 *s = a.src + src_frame * a.frame_vecs;
    u32x4 *d = a.dst + dst_frame * a.frame_vecs;
    const int64_t base = static_cast<int64_t>(chunk) * kThreads * kUnroll + threadIdx.x;
    u32x4 r[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const int64_t i = base + u * kThreads;
        if (i < a.frame_vecs) r[u] = __builtin_nontemporal_load(s + i);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const int64_t i = base + u * kThreads;
        if (i < a.frame_vecs) __builtin_nontemporal_store(r[u], d + i);
    }
}

}  // namespace

hipError_t launch_frame_copy(const FrameCopyParams &p, hipStream_t stream) {
    CopyKArgs a{};
    a.src = static_cast<const u32x4 *>(p.src);
    a.dst = static_cast<u32x4 *>(p.dst);
    a.frame_vecs = p.frame_bytes / 16;
    for (int m = 0; m < p.M; ++m) {
        a.src_idx[m] = p.src_idx[m];
        a.dst_idx[m] = p.dst_idx[m];
    }
    const int64_t per_block = static_cast<int64_t>(kThreads) * kUnroll;
    const int64_t bpf = (a.frame_vecs + per_block - 1) / per_block;
    const int64_t blocks = bpf * p.M;
    if (bpf > 0x7fffffffLL || blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    a.blocks_per_frame = static_cast<int32_t>(bpf);
    hipLaunchKernelGGL(frame_copy_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0,
                       stream, a);
    return hipGetLastError();
}

}  // namespace rf
