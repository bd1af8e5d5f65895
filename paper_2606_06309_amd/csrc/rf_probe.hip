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
//  * hbm_read_kernel: workgroups of 1024 threads, each reading one contiguous
//    run of the buffer in 16-byte words (four loads in flight per thread),
//    folded with XOR into one 32-bit word per workgroup, so the XOR of all
//    sink words equals the XOR of all words of the buffer. Runs of about 2 MB
//    read fastest here (about 7 TB/s on MI355X); a grid stride over the whole
//    buffer reads slower, and runs of 16 KB pay the workgroup's closing
//    reduction for every 16 KB.
//  * lds_read_kernel: every wave of a workgroup reads a 64 KB LDS array in
//    full per round, with 16-byte reads or with the transposing 8-byte reads
//    the attention kernel takes its V^T operands with, as many in flight as
//    the compiler keeps, and adds what it reads into two 32-bit sums. The workgroup's elapsed
//    shader-clock ticks over its read loop give the bytes per clock; 64 KB of
//    LDS per workgroup puts two workgroups (8 waves) on a compute unit, the
//    attention kernel's occupancy.
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

__global__ __launch_bounds__(kHbmThreads) void hbm_read_kernel(const u32x4_t *src, int64_t n_words, int64_t per,
                                                              uint32_t *sink) {
    const int64_t b0 = static_cast<int64_t>(blockIdx.x) * per;
    const int64_t b1 = b0 + per < n_words ? b0 + per : n_words;
    u32x4_t acc = {0u, 0u, 0u, 0u};
    int64_t i = b0 + threadIdx.x;
    for (; i + 3 * kHbmThreads < b1; i += 4 * kHbmThreads) {
        const u32x4_t w0 = __builtin_nontemporal_load(src + i);
        const u32x4_t w1 = __builtin_nontemporal_load(src + i + kHbmThreads);
        const u32x4_t w2 = __builtin_nontemporal_load(src + i + 2 * kHbmThreads);
        const u32x4_t w3 = __builtin_nontemporal_load(src + i + 3 * kHbmThreads);
        acc ^= (w0 ^ w1) ^ (w2 ^ w3);
    }
    for (; i < b1; i += kHbmThreads) acc ^= src[i];
    uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
    for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o);
    __shared__ uint32_t red[kHbmThreads / 64];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0u;
        for (int w = 0; w < kHbmThreads / 64; ++w) t ^= red[w];
        sink[blockIdx.x] = t;
    }
}

constexpr int kLdsWords = 16384;   // 64 KB of LDS per workgroup

// The 16-byte form reads the array row by row (64 rows of 64 lanes x 16
// bytes), lane l in round r at column (l + r) % 64, and sums 32-bit words.
// The transposing form addresses LDS as the attention kernel addresses a V
// tile of 256-byte key rows: in read t of round r, lanes 16h + 4q + e (h = 0..3,
// q, e = 0..3) take the 8 bytes at row 8 (t / 4) + 4 (h / 2) + q, 32-byte chunk
// (2 ((t + r) % 4) + h % 2) ^ 2q, byte 8e, so the 16 lanes of a group cover
// 4 rows x 32 bytes and a wave 8 rows x 64 bytes; the hardware hands lane
// 16h + i the i-th 16-bit element of each of the group's 4 rows. That form
// XORs the 32-bit words it receives: a group's XOR, folded to 16 bits (low half
// XOR high half), is the XOR of the 16-bit elements the group addressed however
// they are distributed. Either way each round of each wave reads every byte once
// and a lane's bytes change from round to round.
template <int kWidth>
__global__ __launch_bounds__(kProbeThreads) void lds_read_kernel(int32_t rounds, uint32_t *sink,
                                                                 uint64_t *ticks) {
    __shared__ __attribute__((aligned(16))) uint32_t buf[kLdsWords];
    for (int i = threadIdx.x; i < kLdsWords; i += kProbeThreads) buf[i] = static_cast<uint32_t>(i) * 2654435761u;
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const uint8_t *base = reinterpret_cast<const uint8_t *>(buf);
    uint32_t s0 = 0u, s1 = 0u;
    const uint64_t t0 = __builtin_amdgcn_s_memtime();
    if constexpr (kWidth == 16) {
        for (int32_t r = 0; r < rounds; ++r) {
            const uint8_t *col = base + ((lane + r) & 63) * 16;
#pragma unroll
            for (int j = 0; j < 64; ++j) {
                const u32x4_t w = *reinterpret_cast<const u32x4_t *>(col + j * 1024);
                s0 += w[0] + w[1];
                s1 += w[2] + w[3];
            }
        }
    } else {
        typedef short i16x4_t __attribute__((ext_vector_type(4)));
        typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;
        typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
        const int h = lane >> 4, q = (lane >> 2) & 3, e = lane & 3;
        const int row_ofs = (4 * (h >> 1) + q) * 256 + 8 * e;
        for (int32_t r = 0; r < rounds; ++r) {
            int po[4];
#pragma unroll
            for (int p = 0; p < 4; ++p) po[p] = row_ofs + (((2 * ((p + r) & 3) + (h & 1)) ^ (2 * q)) * 32);
#pragma unroll
            for (int t = 0; t < 128; ++t) {
                const i16x4_t v =
                    __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)(base + (t / 4) * 2048 + po[t % 4]));
                const u32x2_t w = __builtin_bit_cast(u32x2_t, v);
                s0 ^= w[0];
                s1 ^= w[1];
            }
        }
    }
    __syncthreads();
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
    sink[static_cast<int64_t>(blockIdx.x) * kProbeThreads + threadIdx.x] = kWidth == 16 ? s0 + s1 : s0 ^ s1;
    if (ticks && threadIdx.x == 0) ticks[blockIdx.x] = t1 - t0;
}

}  // namespace

hipError_t launch_lds_read_probe(int32_t workgroups, int32_t rounds, int32_t width, uint32_t *sink,
                                 uint64_t *ticks, hipStream_t stream) {
    if (width == 16)
        hipLaunchKernelGGL(lds_read_kernel<16>, dim3(static_cast<uint32_t>(workgroups)), dim3(kProbeThreads), 0,
                           stream, rounds, sink, ticks);
    else
        hipLaunchKernelGGL(lds_read_kernel<8>, dim3(static_cast<uint32_t>(workgroups)), dim3(kProbeThreads), 0,
                           stream, rounds, sink, ticks);
    return hipGetLastError();
}

hipError_t launch_mfma_probe(const void *ops, int32_t workgroups, int32_t rounds, float *sink,
                             hipStream_t stream) {
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(static_cast<uint32_t>(workgroups)), dim3(kProbeThreads), 0,
                       stream, static_cast<const u32x4_t *>(ops), rounds, sink);
    return hipGetLastError();
}

hipError_t launch_hbm_read_probe(const void *src, int64_t bytes, int32_t workgroups, uint32_t *sink,
                                 hipStream_t stream) {
    const int64_t n_words = bytes / 16;
    const int64_t per = (n_words + workgroups - 1) / workgroups;
    hipLaunchKernelGGL(hbm_read_kernel, dim3(static_cast<uint32_t>(workgroups)), dim3(kHbmThreads), 0,
                       stream, static_cast<const u32x4_t *>(src), n_words, per, sink);
    return hipGetLastError();
}

}  // namespace rf
