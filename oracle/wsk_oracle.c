/*
 * Oracle for the partitioned-KV decode path -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, fp64 definitions of what the GPU path computes.  Nothing in the
 * product links this file: only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load it.  It shares no code, header or table
 * with the HIP library.
 *
 * Inputs are the same bf16 bytes the GPU reads (widened exactly to fp64);
 * every sum is an fp64 sum in plain index order; scores are materialised and
 * the softmax is taken in two passes (max, then normalised weights).
 *
 * Passages followed (Yu, Dong, Liao: "Physically Partitioned KVCache Format
 * for CPU-GPU Load Balancing in MoE Inference"):
 *   - Sec. 5.1 (Sequence-Dimension Splitting): both engines attend every head
 *     over disjoint sequence ranges; the two partial outputs merge exactly by
 *     log-sum-exp rescaling.
 *   - Sec. 4.2 (Batched Write-Time Routing in Decode), last paragraph: each
 *     side returns its partial output and normaliser; one LSE join per step.
 *   - Sec. 6.1 (CPU kernel), "Compressed-MLA variant": MLA attention is a
 *     query-side projection into the latent space, attention over the shared
 *     latent, and an output-side expansion.
 *   - Sec. 4.3 (Interface and Semantics), semantic (iv) exactness: the result
 *     is the exact attention over the whole context, nothing dropped.
 *
 * Readings where the paper is silent (the normaliser is one natural-log LSE of
 * the scaled scores per query head; an empty range yields O = 0, LSE = -inf;
 * query head h reads KV head floor(h / G)) are the ones the build documents.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* bf16 bits -> fp64, exactly: bf16 is the upper half of an IEEE binary32. */
static double bf16_to_double(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * Exact softmax attention of every query head over keys [a, e).
 *
 *   query head h reads KV head g = floor(h / G);
 *   s_j  = scale * sum_d q[h][d] * K[g][j][d]            for j in [a, e)
 *   m    = max_j s_j
 *   l    = sum_j exp(s_j - m)
 *   O[h] = sum_j exp(s_j - m) * V[g][j][:] / l
 *   LSE  = m + ln l
 *   empty range: O = 0, LSE = -inf
 *
 * q   : fp64 [H][dk]
 * key of head g, token j   : k + g*k_head + j*k_row   (dk bf16 elements)
 * value of head g, token j : v + g*v_head + j*v_row   (dv bf16 elements)
 * o   : fp64 [H][dv], lse: fp64 [H]
 * Returns 0, or -1 on bad arguments / allocation failure.
 */
int oracle_attend(int H, int G, int dk, int dv,
                  const double *q,
                  const uint16_t *k, int64_t k_row, int64_t k_head,
                  const uint16_t *v, int64_t v_row, int64_t v_head,
                  int64_t a, int64_t e, double scale,
                  double *o, double *lse)
{
    if (H <= 0 || G <= 0 || H % G != 0 || dk <= 0 || dv <= 0 || a < 0 || e < a)
        return -1;
    int64_t T = e - a;
    int failed = 0;

#pragma omp parallel for schedule(dynamic, 1)
    for (int h = 0; h < H; ++h) {
        double *oh = o + (int64_t)h * dv;
        if (T == 0) {
            for (int d = 0; d < dv; ++d) oh[d] = 0.0;
            lse[h] = -INFINITY;
            continue;
        }
        int g = h / G;
        const double *qh = q + (int64_t)h * dk;
        double *s = (double *)malloc((size_t)T * sizeof(double));
        if (!s) {
#pragma omp atomic write
            failed = 1;
            continue;
        }
        /* pass 1: scores and their maximum */
        double m = -INFINITY;
        for (int64_t j = 0; j < T; ++j) {
            const uint16_t *kj = k + g * k_head + (a + j) * k_row;
            double dot = 0.0;
            for (int d = 0; d < dk; ++d)
                dot += qh[d] * bf16_to_double(kj[d]);
            s[j] = scale * dot;
            if (s[j] > m) m = s[j];
        }
        /* pass 2: normaliser and weighted sum of values */
        for (int d = 0; d < dv; ++d) oh[d] = 0.0;
        double l = 0.0;
        for (int64_t j = 0; j < T; ++j) {
            double w = exp(s[j] - m);
            l += w;
            const uint16_t *vj = v + g * v_head + (a + j) * v_row;
            for (int d = 0; d < dv; ++d)
                oh[d] += w * bf16_to_double(vj[d]);
        }
        for (int d = 0; d < dv; ++d) oh[d] /= l;
        lse[h] = m + log(l);
        free(s);
    }
    return failed ? -1 : 0;
}

/*
 * LSE merge of two normalised partials over disjoint key sets (Sec. 5.1):
 *   m = max(lse_a, lse_b); if m = -inf: O = 0, LSE = -inf
 *   else w_x = exp(lse_x - m), O = (w_a O_a + w_b O_b) / (w_a + w_b),
 *        LSE = m + ln(w_a + w_b)
 * Arrays are [rows][width] (O) and [rows] (LSE), fp64.  Outputs may alias inputs.
 */
int oracle_merge(int64_t rows, int width,
                 const double *o_a, const double *lse_a,
                 const double *o_b, const double *lse_b,
                 double *o_out, double *lse_out)
{
    if (rows < 0 || width <= 0) return -1;
    for (int64_t r = 0; r < rows; ++r) {
        double la = lse_a[r], lb = lse_b[r];
        double m = la > lb ? la : lb;
        const double *xa = o_a + r * width, *xb = o_b + r * width;
        double *y = o_out + r * width;
        if (m == -INFINITY) {
            for (int d = 0; d < width; ++d) y[d] = 0.0;
            lse_out[r] = -INFINITY;
            continue;
        }
        double wa = exp(la - m), wb = exp(lb - m);
        for (int d = 0; d < width; ++d)
            y[d] = (wa * xa[d] + wb * xb[d]) / (wa + wb);
        lse_out[r] = m + log(wa + wb);
    }
    return 0;
}

/*
 * MLA query-side projection (Sec. 6.1, compressed-MLA variant): a head's
 * non-RoPE query is carried into the latent space,
 *   q_lat[h][l] = sum_i q_nope[h][i] * W_UK[h][i][l].
 * q_nope: bf16 [H][dn], w_uk: bf16 [H][dn][dl], out: fp64 [H][dl].
 */
int oracle_mla_absorb(int H, int dn, int dl, const uint16_t *q_nope,
                      const uint16_t *w_uk, double *q_lat)
{
    if (H <= 0 || dn <= 0 || dl <= 0) return -1;
    for (int h = 0; h < H; ++h)
        for (int l = 0; l < dl; ++l) {
            double acc = 0.0;
            for (int i = 0; i < dn; ++i)
                acc += bf16_to_double(q_nope[(int64_t)h * dn + i]) *
                       bf16_to_double(w_uk[((int64_t)h * dn + i) * dl + l]);
            q_lat[(int64_t)h * dl + l] = acc;
        }
    return 0;
}

/*
 * MLA output-side expansion (Sec. 6.1): a head's latent output is carried to
 * its value width,  O[h][j] = sum_l O_lat[h][l] * W_UV[h][l][j].
 * o_lat: fp64 [H][dl], w_uv: bf16 [H][dl][dv], out: fp64 [H][dv].
 */
int oracle_mla_expand(int H, int dl, int dv, const double *o_lat,
                      const uint16_t *w_uv, double *o)
{
    if (H <= 0 || dl <= 0 || dv <= 0) return -1;
    for (int h = 0; h < H; ++h)
        for (int j = 0; j < dv; ++j) {
            double acc = 0.0;
            for (int l = 0; l < dl; ++l)
                acc += o_lat[(int64_t)h * dl + l] *
                       bf16_to_double(w_uv[((int64_t)h * dl + l) * dv + j]);
            o[(int64_t)h * dv + j] = acc;
        }
    return 0;
}

/*
 * Round fp64 values to bf16 (round to nearest, ties to even), returning bits.
 * bf16 keeps 8 significant bits and binary32's exponent range; results past
 * the largest finite bf16 become +-inf, tiny ones become bf16 subnormals.
 */
static uint16_t double_to_bf16(double x)
{
    if (isnan(x)) return 0x7fc0;
    uint16_t sign = signbit(x) ? 0x8000 : 0;
    double ax = fabs(x);
    if (ax == 0.0) return sign;
    int ex;
    frexp(ax, &ex);                       /* ax = f * 2^ex, f in [0.5, 1) */
    int e2 = ex - 1;                      /* ax in [2^e2, 2^(e2+1)) */
    if (e2 < -126) e2 = -126;             /* subnormal spacing below 2^-126 */
    double ulp = ldexp(1.0, e2 - 7);      /* 8 significant bits */
    double n = ax / ulp;                  /* exact: power-of-two scaling */
    double r = floor(n);
    double frac = n - r;
    if (frac > 0.5 || (frac == 0.5 && fmod(r, 2.0) != 0.0)) r += 1.0;
    double y = r * ulp;                   /* may carry to the next binade: still exact */
    if (y > 3.3895313892515355e38)        /* largest finite bf16 */
        return sign | 0x7f80;
    float f = (float)y;                   /* exact: y has <= 8 significant bits */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return sign | (uint16_t)(u >> 16);
}

int oracle_round_bf16(int64_t n, const double *x, uint16_t *out)
{
    if (n < 0) return -1;
    for (int64_t i = 0; i < n; ++i) out[i] = double_to_bf16(x[i]);
    return 0;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the following calls (timing only; results do not depend on it). */
int oracle_set_threads(int n)
{
    if (n < 1) return -1;
#ifdef _OPENMP
    omp_set_num_threads(n);
#endif
    return 0;
}
