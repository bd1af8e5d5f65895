// Device probes for gfx950: the sustained whole-chip rate of the dense bf16
// matrix cores and of HBM reads. They are measurement support, not part of the
// method: a kernel's achieved rate is set against the published peaks and
// against what this device sustains under a pure load of the same kind (the
// chip lowers its clock below the 2.4 GHz of the published matrix peak when
// every matrix core is busy).
//
//  * mfma_probe_kernel: every wave runs kChains independent accumulator chains
//    of v_mfma_f32_32x32x16_bf16 (independent chains keep the matrix core fed
//    without waiting for a result). A lane holds 6 A and 6 B operands, and step
//    u of a round multiplies A[(u + 2j) % 6] by B[(3u + j) % 6] in chain j, so
//    consecutive instructions see different data, as in a real product (the
//    power a matrix core draws, and with it the clock the chip holds, depends
//    on how much its inputs change). A round is 8 steps of every chain: 2^22
//    FLOP per (workgroup, round). The operands go from the caller's buffer into
//    LDS and from there into registers, the path real kernels feed the matrix
//    cores by: loaded straight from global memory into the operand registers,
//    the same loop sustained well under the rate the hardware reaches. The
//    kernel is held to four waves per SIMD (114 registers) so that a grid of 4
//    workgroups per CU runs in one round.
//  * hbm_read_kernel: a grid-stride read of 16-byte words (four loads in
//    flight per thread), folded with XOR into one 32-bit word per thread, so
//    the XOR of all sink words equals the XOR of all words of the buffer.
#include "rf_internal.h"

namespace rf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kChains = 4;
constexpr int kOps = 6;   // A and B operands per lane
constexpr int kSteps = 8; // steps of every chain per round

__global__ __launch_bounds__(kProbeThreads) __attribute__((amdgpu_waves_per_eu(4, 4)))
void mfma_probe_kernel(const u32x4_t *ops, int32_t rounds, float *sink) {
    __shared__ __attribute__((aligned(16))) u32x4_t staged[2 * kOps * 64];
    for (int t = threadIdx.x; t < 2 * kOps * 64; t += kProbeThreads) staged[t] = ops[t];
    __syncthreads();
    const int lane = threadIdx.x & 63;
    u32x4_t A[kOps], B[kOps];
#pragma unroll
    for (int i = 0; i < kOps; ++i) {
        A[i] = staged[i * 64 + lane];
        B[i] = staged[(kOps + i) * 64 + lane];
    }
    f32x16_t c[kChains];
#pragma unroll
    for (int j = 0; j < kChains; ++j) c[j] = f32x16_t{};
    for (int32_t it = 0; it < rounds; ++it) {
#pragma unroll
        for (int u = 0; u < kSteps; ++u)
#pragma unroll
            for (int j = 0; j < kChains; ++j) {
                const bf16x8_t a = __builtin_bit_cast(bf16x8_t, A[(u + 2 * j) % kOps]);
                const bf16x8_t b = __builtin_bit_cast(bf16x8_t, B[(3 * u + j) % kOps]);
                c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[j], 0, 0, 0);
            }
    }
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < kChains; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += c[j][r];
    sink[static_cast<int64_t>(blockIdx.x) * kProbeThreads + threadIdx.x] = s;
}

__global__ __launch_bounds__(kProbeThreads) void hbm_read_kernel(const u32x4_t *src, int64_t n_words,
                                                                 uint32_t *sink) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kProbeThreads;
    int64_t i = static_cast<int64_t>(blockIdx.x) * kProbeThreads + threadIdx.x;
    u32x4_t acc = {0u, 0u, 0u, 0u};
    for (; i + 3 * stride < n_words; i += 4 * stride) {
        const u32x4_t w0 = __builtin_nontemporal_load(src + i);
        const u32x4_t w1 = __builtin_nontemporal_load(src + i + stride);
        const u32x4_t w2 = __builtin_nontemporal_load(src + i + 2 * stride);
        const u32x4_t w3 = __builtin_nontemporal_load(src + i + 3 * stride);
        acc ^= (w0 ^ w1) ^ (w2 ^ w3);
    }
    for (; i < n_words; i += stride) acc ^= src[i];
    sink[static_cast<int64_t>(blockIdx.x) * kProbeThreads + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

}  // namespace

hipError_t launch_mfma_probe(const void *ops, int32_t workgroups, int32_t rounds, float *sink,
                             hipStream_t stream) {
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(static_cast<uint32_t>(workgroups)), dim3(kProbeThreads), 0,
                       stream, static_cast<const u32x4_t *>(ops), rounds, sink);
    return hipGetLastError();
}

hipError_t launch_hbm_read_probe(const void *src, int64_t bytes, int32_t workgroups, uint32_t *sink,
                                 hipStream_t stream) {
    hipLaunchKernelGGL(hbm_read_kernel, dim3(static_cast<uint32_t>(workgroups)), dim3(kProbeThreads), 0,
                       stream, static_cast<const u32x4_t *>(src), bytes / 16, sink);
    return hipGetLastError();
}

}  // namespace rf
