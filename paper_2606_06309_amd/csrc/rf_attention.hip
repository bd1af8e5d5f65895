// Keyframe-query attention for gfx950 (CDNA4).
//
// Method (Sec. 3.2.3-3.2.4; App. B.2): at a step where only keyframes are
// denoised, the query tokens of the M keyframes attend over the keys and
// values of all T frames. Per head: out = softmax(Q_kf K^T / sqrt(d)) V.
//
// bf16 kernel design:
//  * A workgroup of 4 waves owns one (head, 128-row query tile); each wave
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
//    operands without any data movement. V is staged transposed in LDS
//    ([d][key]) so each A operand is two 64-bit LDS reads; the key order
//    inside an operand follows the accumulator layout (a reduction index may
//    be permuted freely as long as both operands agree).
//  * Online softmax in the log2 domain with fp32 state; P is rounded to bf16
//    for the matrix cores, the row sum uses the unrounded fp32 values.
//  * K/V tiles of 64 keys are prefetched into registers while the current
//    tile is computed; the last tile masks keys >= S.
//  * Workgroup ids are mapped XCD-aware: consecutive ids go round-robin to the
//    8 XCDs, so tile = (id % 8) * per_xcd + id / 8 gives each XCD a contiguous,
//    head-major range of tiles and the workgroups resident on one XCD stream
//    the same head's K/V through that XCD's L2.
#include "rf_internal.h"

namespace rf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Data moves as 32-bit words; bf16 vectors are only ever formed by a
// whole-vector bitcast of a u32x4 (or of one scalar word) right before the
// instruction that consumes them.

// Tunables (compile-time): waves per workgroup (each owns 32 query rows), keys
// per LDS tile, the log2-domain slack before the running max is rebased (0:
// the reference is always the exact running max, so the largest probability
// is exactly 1), and how many LDS fragments the matrix core reads ahead.
#ifndef RF_ATTN_WAVES
#define RF_ATTN_WAVES 8
#endif
#ifndef RF_ATTN_BC
#define RF_ATTN_BC 64
#endif
#ifndef RF_ATTN_RESCALE_SLACK
#define RF_ATTN_RESCALE_SLACK 0.0f
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
constexpr int kBc = RF_ATTN_BC;    // keys per LDS tile
constexpr int kKPad = 8;           // bf16 padding per K row in LDS (row = 272 B at d=128)
constexpr int kVPad = 8;           // bf16 padding per V^T row in LDS (row = 144 B at 64 keys)
constexpr int kXcds = 8;
static_assert(kBc % 32 == 0, "key tile must be a multiple of 32");

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
    int32_t total_tiles;
    int32_t per_xcd;
    float scale_log2;   // log2(e) / sqrt(d)
    int32_t kf[kMaxFrames];
};

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

// S^T = K Q^T for one tile of kNB 32-key blocks, with the K fragments read
// from LDS through a ring RF_ATTN_K_LEAD fragments ahead of the matrix core.
// The scheduling groups pin that order: LEAD reads, then (1 MFMA, 1 read)
// pairs, then the last LEAD MFMAs.
template <int D, int kNB, int kKRow>
__device__ __forceinline__ void scores_tile(const uint16_t *kb, const u32x4_t (&qf)[D / 16],
                                            f32x16_t (&sacc)[kNB], int col, int grp) {
    constexpr int kSteps = D / 16;
    constexpr int kNF = kNB * kSteps;
    constexpr int kLead = RF_ATTN_K_LEAD < kNF ? RF_ATTN_K_LEAD : kNF;
    u32x4_t ring[kLead];
    auto rd = [&](int i) {
        const int b = i / kSteps, kk = i % kSteps;
        return *reinterpret_cast<const u32x4_t *>(&kb[(b * 32 + col) * kKRow + kk * 16 + grp * 8]);
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

// Column of key k in a transposed V row: within every 16-key group the middle
// two 4-key quarters are swapped, so the 8 keys one lane contributes to an A
// operand (keys grp*4 + 0..3 and 8 + grp*4 + 0..3 of the group, following the
// score accumulator layout) sit in 8 consecutive columns: one 128-bit read.
__host__ __device__ constexpr int vt_column(int k) {
    return (k & ~15) | ((((k >> 2) & 3) == 1 ? 2 : (((k >> 2) & 3) == 2 ? 1 : ((k >> 2) & 3))) << 2) | (k & 3);
}

// O^T += V^T P^T for one tile; each A operand is one 128-bit read of the
// transposed V tile, issued RF_ATTN_V_LEAD operands ahead.
template <int D, int kNB, int kVRow>
__device__ __forceinline__ void pv_tile(const uint16_t *vb, const u32x4_t (&pw)[2 * kNB],
                                        f32x16_t (&oacc)[D / 32], int col, int grp) {
    constexpr int kNF = 2 * kNB * (D / 32);
    constexpr int kLead = RF_ATTN_V_LEAD < kNF ? RF_ATTN_V_LEAD : kNF;
    u32x4_t ring[kLead];
    auto rd = [&](int i) {
        const int c = i / (D / 32), db = i % (D / 32);
        return *reinterpret_cast<const u32x4_t *>(&vb[(db * 32 + col) * kVRow + c * 16 + grp * 8]);
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
    __builtin_amdgcn_sched_group_barrier(0x100, kLead, 0);
#pragma unroll
    for (int i = 0; i < kNF - kLead; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kLead, 0);
}

// Per-tile pipeline with double-buffered LDS and one barrier per tile:
//   global loads of tile t+1 -> registers   (in flight during the math)
//   math on LDS buffer t%2
//   registers -> LDS buffer (t+1)%2          (last read during tile t-1)
//   barrier
// kBuf: K/V staging through raw buffer loads whose resource is rebased per
// tile in scalar registers, so the hardware range check zero-fills keys >= S
// and no per-tile vector address arithmetic is needed (tensors below 2 GiB).
template <int D, bool kBuf>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
void attn_bf16_kernel(const AttnKArgs a) {
    constexpr int kKRow = D + kKPad;                    // bf16 elements per K row
    constexpr int kVRow = kBc + kVPad;                  // bf16 elements per V^T row
    constexpr int kKTotal = kBc * D / 8;                // 16-byte K chunks per tile
    constexpr int kVTotal = (kBc / 2) * (D / 8);        // (2 keys x 8 dims) V chunks per tile
    constexpr int kKChunks = (kKTotal + kThreads - 1) / kThreads;
    constexpr int kVChunks = (kVTotal + kThreads - 1) / kThreads;
    constexpr int kNB = kBc / 32;                       // 32-key score blocks per tile
    constexpr int kKBufs = 2;                           // K tile buffers (see the loop below)
    constexpr int kVBufs = 2;                           // V tile buffers

    __shared__ __attribute__((aligned(16))) uint16_t ks[kKBufs][kBc * kKRow];
    __shared__ __attribute__((aligned(16))) uint16_t vt[kVBufs][D * kVRow];

    const int tile = static_cast<int>(blockIdx.x % kXcds) * a.per_xcd + static_cast<int>(blockIdx.x / kXcds);
    if (tile >= a.total_tiles) return;
    const int head = tile / a.n_qtiles;
    const int qt = tile - head * a.n_qtiles;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
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

    f32x16_t oacc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] = 0.0f;
    // m_run: reference max (log2 domain) the probabilities are taken against.
    // It is rebased when the running max exceeds it by more than the slack, so
    // p <= 2^slack; the final O / l does not depend on the reference. The
    // accumulators are rescaled only on tiles where some lane rebased.
    float m_run = -__builtin_huge_valf();
    float l_run = 0.0f;   // this lane's partial row sum

    const uint16_t *kbase = a.k + static_cast<int64_t>(head) * D;
    const uint16_t *vbase = a.v + static_cast<int64_t>(head) * D;
    const u32x4_t zero4 = {0u, 0u, 0u, 0u};
    // bytes from a head's first element to one past the last element it owns
    const int64_t head_bytes = ((a.S - 1) * rs + D) * 2;

    u32x4_t kreg[kKChunks], vreg0[kVChunks], vreg1[kVChunks];

    auto load_tile = [&](int64_t j0) {
        if constexpr (kBuf) {
            // scalar rebase: the resource starts at key j0, its range ends at the head's last key.
            // The inputs are workgroup-uniform; readfirstlane states that to the compiler so the
            // resource lives in scalar registers (no per-load uniformity loop).
            const int64_t off = j0 * rs * 2;
            const int32_t rec = __builtin_amdgcn_readfirstlane(static_cast<int32_t>(head_bytes - off));
            const __amdgpu_buffer_rsrc_t kr =
                __builtin_amdgcn_make_buffer_rsrc(uniform_ptr(kbase + j0 * rs), 0, rec, kBufferWord3);
            const __amdgpu_buffer_rsrc_t vr =
                __builtin_amdgcn_make_buffer_rsrc(uniform_ptr(vbase + j0 * rs), 0, rec, kBufferWord3);
#pragma unroll
            for (int i = 0; i < kKChunks; ++i) {
                const int c = tid + i * kThreads;
                if (kKTotal % kThreads != 0 && c >= kKTotal) break;
                const int key = c / (D / 8), c8 = c % (D / 8);
                kreg[i] = __builtin_amdgcn_raw_buffer_load_b128(
                    kr, static_cast<int32_t>((key * rs + c8 * 8) * 2), 0, 0);
            }
#pragma unroll
            for (int i = 0; i < kVChunks; ++i) {
                const int p = tid + i * kThreads;
                if (kVTotal % kThreads != 0 && p >= kVTotal) break;
                const int kp = p % (kBc / 2), c8 = p / (kBc / 2);
                const int32_t o = static_cast<int32_t>((2 * kp * rs + c8 * 8) * 2);
                vreg0[i] = __builtin_amdgcn_raw_buffer_load_b128(vr, o, 0, 0);
                vreg1[i] = __builtin_amdgcn_raw_buffer_load_b128(vr, o + static_cast<int32_t>(rs * 2), 0, 0);
            }
        } else {
#pragma unroll
            for (int i = 0; i < kKChunks; ++i) {
                const int c = tid + i * kThreads;
                if (kKTotal % kThreads != 0 && c >= kKTotal) break;
                const int key = c / (D / 8), c8 = c % (D / 8);
                const int64_t j = j0 + key;
                kreg[i] = j < a.S ? *reinterpret_cast<const u32x4_t *>(kbase + j * rs + c8 * 8) : zero4;
            }
#pragma unroll
            for (int i = 0; i < kVChunks; ++i) {
                const int p = tid + i * kThreads;
                if (kVTotal % kThreads != 0 && p >= kVTotal) break;
                const int kp = p % (kBc / 2), c8 = p / (kBc / 2);
                const int64_t j = j0 + 2 * kp;
                vreg0[i] = j < a.S ? *reinterpret_cast<const u32x4_t *>(vbase + j * rs + c8 * 8) : zero4;
                vreg1[i] =
                    j + 1 < a.S ? *reinterpret_cast<const u32x4_t *>(vbase + (j + 1) * rs + c8 * 8) : zero4;
            }
        }
    };
    auto store_tile = [&](int kbuf, int vbuf) {
#pragma unroll
        for (int i = 0; i < kKChunks; ++i) {
            const int c = tid + i * kThreads;
            if (kKTotal % kThreads != 0 && c >= kKTotal) break;
            const int key = c / (D / 8), c8 = c % (D / 8);
            *reinterpret_cast<u32x4_t *>(&ks[kbuf][key * kKRow + c8 * 8]) = kreg[i];
        }
#pragma unroll
        for (int i = 0; i < kVChunks; ++i) {
            const int p = tid + i * kThreads;
            if (kVTotal % kThreads != 0 && p >= kVTotal) break;
            const int kp = p % (kBc / 2), c8 = p / (kBc / 2);
            uint32_t *dst = reinterpret_cast<uint32_t *>(&vt[vbuf][(c8 * 8) * kVRow + vt_column(2 * kp)]);
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                // word w holds dims 2w (low half) and 2w+1 (high half) of one key;
                // the transposed row of a dim holds keys 2kp (low) and 2kp+1
                // (high) side by side (vt_column keeps even/odd key pairs adjacent)
                const uint32_t x0 = vreg0[i][w], x1 = vreg1[i][w];
                dst[(2 * w) * (kVRow / 2)] = __builtin_amdgcn_perm(x1, x0, 0x05040100u);
                dst[(2 * w + 1) * (kVRow / 2)] = __builtin_amdgcn_perm(x1, x0, 0x07060302u);
            }
        }
    };

    // Per-tile pipeline with double-buffered LDS and one barrier per tile:
    //   global loads of tile t+1 -> registers   (in flight during the math)
    //   math on LDS buffer t%2
    //   registers -> LDS buffer (t+1)%2          (last read during tile t-1)
    //   barrier
    const int64_t ntiles = (a.S + kBc - 1) / kBc;
    const float sl2 = a.scale_log2;
    load_tile(0);
    store_tile(0, 0);
    __syncthreads();
    for (int64_t t = 0; t < ntiles; ++t) {
        const int buf = static_cast<int>(t & 1);
        if (t + 1 < ntiles) load_tile((t + 1) * kBc);   // in flight during this tile's math

        // ---- S^T = K Q^T : 32-key blocks ----
        f32x16_t sacc[kNB];
        scores_tile<D, kNB, kKRow>(ks[buf], qf, sacc, col, grp);
        // accumulator r of block b holds key b*32 + (r/4)*8 + grp*4 + r%4 for query `col`

        const int64_t j0 = t * kBc;
        if (j0 + kBc > a.S) {
#pragma unroll
            for (int b = 0; b < kNB; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t key = j0 + b * 32 + (r / 4) * 8 + grp * 4 + (r % 4);
                    if (key >= a.S) sacc[b][r] = -__builtin_huge_valf();
                }
        }

        // ---- online softmax (log2 domain) ----
        float mx = -__builtin_huge_valf();
#pragma unroll
        for (int b = 0; b < kNB; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[b][r]);
        mx = halves_max(mx) * sl2;
        const bool rebase = mx > m_run + RF_ATTN_RESCALE_SLACK;
        if (__builtin_amdgcn_ballot_w64(rebase)) {   // wave-uniform branch, rarer as the max settles
            const float m_new = rebase ? mx : m_run;
            const float corr = fast_exp2(m_run - m_new);
            m_run = m_new;
            l_run *= corr;
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int r = 0; r < 16; ++r) oacc[db][r] *= corr;
        }

        // probabilities, packed as the B operand of O^T = V^T P^T:
        // operand c takes accumulators 8*(c%2) .. 8*(c%2)+7 of block c/2.
        // The row sum adds the bf16-rounded values the matrix core consumes.
        u32x4_t pw[2 * kNB];
        float ls = 0.0f;
#pragma unroll
        for (int b = 0; b < kNB; ++b)
#pragma unroll
            for (int r = 0; r < 16; r += 2) {
                const float p0 = fast_exp2(fmaf(sacc[b][r], sl2, -m_run));
                const float p1 = fast_exp2(fmaf(sacc[b][r + 1], sl2, -m_run));
                const uint32_t word = pack_bf16x2(p0, p1);
                ls = add_bf16x2(word, ls);
                pw[b * 2 + r / 8][(r % 8) / 2] = word;
            }
        l_run += ls;

        // ---- O^T += V^T P^T ----
        pv_tile<D, kNB, kVRow>(vt[buf], pw, oacc, col, grp);

        if (t + 1 < ntiles) store_tile(buf ^ 1, buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue: normalise, round to bf16, store the compact row ----
    l_run = halves_sum(l_run);
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
            const int64_t off = j * rs + static_cast<int64_t>(head) * D + c;
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
        const int64_t total = nq * p.heads;
        const int64_t per_xcd = (total + kXcds - 1) / kXcds;
        if (total > 0x7fffffffLL / kXcds) return hipErrorInvalidConfiguration;
        a.n_qtiles = static_cast<int32_t>(nq);
        a.total_tiles = static_cast<int32_t>(total);
        a.per_xcd = static_cast<int32_t>(per_xcd);
        a.scale_log2 = static_cast<float>(1.4426950408889634 / sqrt(static_cast<double>(p.head_dim)));
        for (int i = 0; i < p.M; ++i) a.kf[i] = p.kf[i];
        const dim3 grid(static_cast<uint32_t>(per_xcd * kXcds)), block(kThreads);
        // buffer addressing covers a head's keys with 32-bit byte offsets
        const bool buf = p.S * p.heads * p.head_dim * 2 < 0x7fffffffLL;
        if (p.head_dim == 128) {
            if (buf) hipLaunchKernelGGL((attn_bf16_kernel<128, true>), grid, block, 0, stream, a);
            else hipLaunchKernelGGL((attn_bf16_kernel<128, false>), grid, block, 0, stream, a);
        } else {
            if (buf) hipLaunchKernelGGL((attn_bf16_kernel<64, true>), grid, block, 0, stream, a);
            else hipLaunchKernelGGL((attn_bf16_kernel<64, false>), grid, block, 0, stream, a);
        }
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
    const int64_t nq = (Mq + kF32Rows - 1) / kF32Rows;
    if (nq > 0x7fffffffLL || p.heads > 65535) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<uint32_t>(nq), static_cast<uint32_t>(p.heads)), block(2 * kF32Rows);
    if (p.head_dim == 128) hipLaunchKernelGGL(attn_f32_kernel<128>, grid, block, 0, stream, a);
    else hipLaunchKernelGGL(attn_f32_kernel<64>, grid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace rf
