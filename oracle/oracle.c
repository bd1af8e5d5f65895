/*
 * Plain, slow fp64 CPU oracle for the keyframe-query attention path of
 * RhymeFlow (arXiv 2606.06309).
 *
 * TEST INFRASTRUCTURE ONLY. This library exists to check the HIP library.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load it. It shares no source, header, table or constant with the HIP
 * library, and nothing in the product path may call it.
 *
 * Conventions:
 *  - Every tensor is read as the exact bits the GPU receives: fp32 values or
 *    bf16 bit patterns are widened exactly to double before any arithmetic.
 *  - All arithmetic is double precision, without fast-math.
 *  - Every reduction is a plain sequential loop in ascending index order.
 *  - exp is libm's double exp.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F64 = 0, ORC_F32 = 1, ORC_BF16 = 2 };

/* Exact widening of element idx of a tensor stored as fp64, fp32 or bf16. */
static double widen(const void *base, int dtype, int64_t idx)
{
    if (dtype == ORC_F64)
        return ((const double *)base)[idx];
    if (dtype == ORC_F32)
        return (double)((const float *)base)[idx];
    /* bf16 is the upper half of an IEEE binary32 word. */
    uint32_t bits = ((uint32_t)((const uint16_t *)base)[idx]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of later parallel loops started from the calling thread (timing only). */
void orc_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/*
 * Scaled dot-product attention for a list of (query token, head) pairs.
 *
 * Method: at a step where only keyframes are denoised, each keyframe query
 * token attends over the keys and values of every frame -- true keyframe
 * states and projected non-keyframe states alike (Sec. 3.2.3-3.2.4;
 * App. B.2, attention at skipped steps). Each head computes the standard
 * attention of App. B.1 (scores Q K^T / sqrt(d), softmax, weighted sum of V),
 * with no mask (bidirectional video attention).
 *
 * q, k, v: [S][heads][d] row-major tensors of the given dtype (q may hold
 *          more tokens than k/v; only the listed tokens are read).
 * S:       number of key/value tokens.
 * q_tokens, q_heads: the n_pairs (token, head) pairs to compute.
 * out:     [n_pairs][d] doubles.
 * probs:   optional [n_pairs][S] doubles, the softmax row of each pair.
 *
 * For one pair (i, h):
 *   s_j = (sum_c q[i,h,c] * k[j,h,c]) / sqrt(d)      j = 0..S-1
 *   m   = max_j s_j
 *   p_j = exp(s_j - m)
 *   l   = sum_j p_j
 *   out[c] = (sum_j p_j * v[j,h,c]) / l
 * Subtracting m changes nothing mathematically (it cancels in p_j / l) and
 * keeps exp in range.
 *
 * Returns 0, or -1 on an invalid argument.
 */
int orc_attention_pairs(const void *q, const void *k, const void *v, int dtype,
                        int64_t S, int64_t heads, int64_t d,
                        const int64_t *q_tokens, const int64_t *q_heads,
                        int64_t n_pairs, double *out, double *probs)
{
    if (!q || !k || !v || !q_tokens || !q_heads || !out)
        return -1;
    if (S <= 0 || heads <= 0 || d <= 0 || n_pairs < 0)
        return -1;
    if (dtype != ORC_F64 && dtype != ORC_F32 && dtype != ORC_BF16)
        return -1;
    for (int64_t p = 0; p < n_pairs; ++p)
        if (q_tokens[p] < 0 || q_heads[p] < 0 || q_heads[p] >= heads)
            return -1;

    const double scale = 1.0 / sqrt((double)d);
    int failed = 0;

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < n_pairs; ++p) {
        double *s = (double *)malloc((size_t)S * sizeof(double));
        if (!s) {
#pragma omp atomic write
            failed = 1;
            continue;
        }
        const int64_t i = q_tokens[p];
        const int64_t h = q_heads[p];

        /* scores */
        for (int64_t j = 0; j < S; ++j) {
            double dot = 0.0;
            for (int64_t c = 0; c < d; ++c)
                dot += widen(q, dtype, (i * heads + h) * d + c) *
                       widen(k, dtype, (j * heads + h) * d + c);
            s[j] = dot * scale;
        }

        /* softmax */
        double m = s[0];
        for (int64_t j = 1; j < S; ++j)
            if (s[j] > m)
                m = s[j];
        double l = 0.0;
        for (int64_t j = 0; j < S; ++j) {
            s[j] = exp(s[j] - m);
            l += s[j];
        }

        /* weighted sum of values */
        for (int64_t c = 0; c < d; ++c) {
            double acc = 0.0;
            for (int64_t j = 0; j < S; ++j)
                acc += s[j] * widen(v, dtype, (j * heads + h) * d + c);
            out[p * d + c] = acc / l;
        }
        if (probs)
            for (int64_t j = 0; j < S; ++j)
                probs[p * S + j] = s[j] / l;
        free(s);
    }
    return failed ? -1 : 0;
}

/*
 * Interpolation weight of the latent trajectory projection, Eq. (3):
 *   alpha = (t_start - tau) / (t_start - t_end).
 * Readings where the paper leaves the value open:
 *  - alpha is kept inside [0, 1], the range App. B.2 states for it;
 *  - t_start == t_end (the state right after warm-up, where both stored
 *    snapshots are the same state) gives alpha = 1.
 */
double orc_projection_alpha(double t_start, double t_end, double tau)
{
    if (t_start == t_end)
        return 1.0;
    double a = (t_start - tau) / (t_start - t_end);
    if (a < 0.0)
        a = 0.0;
    if (a > 1.0)
        a = 1.0;
    return a;
}

/*
 * Latent trajectory projection, Eq. (3), applied to a latent batch.
 *
 * latents: [B][2][C][T][P] of the given dtype, where P = Hl*Wl. Slot 0 holds
 *          z at t_start; slot 1 holds z at t_end for non-keyframes and the
 *          current true state for keyframes.
 * keyframe_mask: [T] bytes, nonzero for keyframes.
 * out:     [B][C][T][P] doubles.
 *
 * Non-keyframe f: out = (1 - alpha) * z_start + alpha * z_end   (Eq. 3)
 * Keyframe f:     out = current state (slot 1); keyframes are denoised every
 *                 step and need no projection (Sec. 3.2.3; the context set
 *                 of Alg. 2 takes keyframes' true states).
 */
int orc_project_latents(const void *latents, int dtype, int64_t B, int64_t C,
                        int64_t T, int64_t P, const uint8_t *keyframe_mask,
                        double t_start, double t_end, double tau, double *out)
{
    if (!latents || !keyframe_mask || !out)
        return -1;
    if (B <= 0 || C <= 0 || T <= 0 || P <= 0)
        return -1;
    if (dtype != ORC_F64 && dtype != ORC_F32 && dtype != ORC_BF16)
        return -1;
    const double alpha = orc_projection_alpha(t_start, t_end, tau);
    for (int64_t b = 0; b < B; ++b)
        for (int64_t c = 0; c < C; ++c)
            for (int64_t f = 0; f < T; ++f)
                for (int64_t e = 0; e < P; ++e) {
                    const int64_t i0 = (((b * 2 + 0) * C + c) * T + f) * P + e;
                    const int64_t i1 = (((b * 2 + 1) * C + c) * T + f) * P + e;
                    const int64_t o = ((b * C + c) * T + f) * P + e;
                    const double z_start = widen(latents, dtype, i0);
                    const double z_end = widen(latents, dtype, i1);
                    if (keyframe_mask[f])
                        out[o] = z_end;
                    else
                        out[o] = (1.0 - alpha) * z_start + alpha * z_end;
                }
    return 0;
}

/*
 * Cosine similarity between the latent frames of a batch element (Sec. 3.1:
 * Eq. (1) compares frames with psi_sim, the cosine similarity; Alg. 1 applies
 * it to the clean-latent proxies of the frames).
 *
 * latents: [B][C][T][P] of the given dtype (P = h*w). The vector of frame f of
 *          batch element b is its C*P elements, channel after channel.
 * sim:     [B][T][T] doubles,
 *          sim[b][i][j] = <x_i, x_j> / (max(|x_i|, 1e-8) * max(|x_j|, 1e-8)),
 *          so a frame with zero norm has similarity 0 to every frame.
 */
int orc_frame_cosine(const void *latents, int dtype, int64_t B, int64_t C,
                     int64_t T, int64_t P, double *sim)
{
    if (!latents || !sim)
        return -1;
    if (B <= 0 || C <= 0 || T <= 0 || P <= 0)
        return -1;
    if (dtype != ORC_F64 && dtype != ORC_F32 && dtype != ORC_BF16)
        return -1;
    const double eps = 1e-8;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t i = 0; i < T; ++i)
            for (int64_t j = 0; j < T; ++j) {
                double dot = 0.0, ni = 0.0, nj = 0.0;
                for (int64_t c = 0; c < C; ++c)
                    for (int64_t e = 0; e < P; ++e) {
                        const double xi = widen(latents, dtype, ((b * C + c) * T + i) * P + e);
                        const double xj = widen(latents, dtype, ((b * C + c) * T + j) * P + e);
                        dot += xi * xj;
                        ni += xi * xi;
                        nj += xj * xj;
                    }
                const double di = sqrt(ni) > eps ? sqrt(ni) : eps;
                const double dj = sqrt(nj) > eps ? sqrt(nj) : eps;
                sim[(b * T + i) * T + j] = dot / (di * dj);
            }
    return 0;
}
