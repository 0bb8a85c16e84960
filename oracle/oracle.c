/*
 * oracle.c -- plain, slow, fp64 CPU reference for the attention of
 * "Speed Is All You Need: On-Device Acceleration of Large Diffusion Models via
 * GPU-Aware Optimizations" (Chen et al., CVPR 2023 workshop).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark do.  It shares no code, header, table or helper with the
 * HIP library.
 *
 * What it computes (Sec. 3.2.1 "Partially Fused Softmax"):
 *   Eq. 3  Attention(Q, K, V) = softmax(Q K^T / sqrt(d)) V,
 *          Q in R^{N x d}, K, V in R^{M x d}.
 *   Eq. 4  L_i = max_j a_ij,  S_i = sum_j exp(a_ij - max_k a_ik)  for the
 *          matrix A = Q K^T / sqrt(d), followed by the element-wise
 *          normalisation exp(a_ij - L_i) / S_i (the text after Eq. 4).
 *
 * Each output row is computed in three passes, exactly as the definition
 * reads: (1) the logits a_ij and their maximum L_i, (2) the shifted
 * exponential sum S_i, (3) the normalised weights times V.  All arithmetic is
 * IEEE double with libm exp; inputs are widened exactly from binary16,
 * bfloat16 or binary32; the scale is the binary32 value the GPU receives,
 * widened exactly.  The caller picks the scale (1/sqrt(d) with the true head
 * dimension d in the UNet).  No blocking, fusion or reordering beyond the
 * definition.  Rows are independent, so OpenMP splits the work by row; the
 * result does not depend on the thread count.
 *
 * Also the steps around the attention (the projections and the multi-head
 * block), the specialised kernels of Sec. 3.1 (group normalisation, Eq. 1;
 * GELU, Eq. 2, with its split and multiply) and the 3x3 convolution that
 * Sec. 3.3 computes with Winograd's algorithm, each written out from its
 * definition below.
 *
 * Build: gcc -O2 -fopenmp -fPIC -shared (no -ffast-math).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* element type codes of the oracle's inputs */
enum { OR_F16 = 0, OR_BF16 = 1, OR_F32 = 2, OR_F64 = 3 };

/* IEEE 754 binary16 -> double, from the format's definition:
 * 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
static double or_from_binary16(uint16_t bits)
{
    const int sign = bits >> 15;
    const int expo = (bits >> 10) & 0x1f;
    const int frac = bits & 0x3ff;
    double mag;
    if (expo == 0)            /* zero or subnormal: frac * 2^-24 */
        mag = ldexp((double)frac, -24);
    else if (expo == 31)      /* infinity or NaN */
        mag = frac ? NAN : INFINITY;
    else                      /* normal: (1024 + frac) * 2^(expo - 25) */
        mag = ldexp((double)(frac | 0x400), expo - 25);
    return sign ? -mag : mag;
}

/* bfloat16 is the upper half of a binary32 word */
static double or_from_bfloat16(uint16_t bits)
{
    uint32_t word = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &word, sizeof f);
    return (double)f;
}

static double or_elem(const void *base, int dtype, int64_t idx)
{
    switch (dtype) {
    case OR_F16:  return or_from_binary16(((const uint16_t *)base)[idx]);
    case OR_BF16: return or_from_bfloat16(((const uint16_t *)base)[idx]);
    case OR_F32:  return (double)((const float *)base)[idx];
    default:      return ((const double *)base)[idx];
    }
}

int oracle_num_threads(int requested)
{
#ifdef _OPENMP
    return requested > 0 ? requested : omp_get_max_threads();
#else
    (void)requested;
    return 1;
#endif
}

/* Widen n elements of `src` (type `dtype`) into `dst` as double. */
int oracle_widen(const void *src, int dtype, int64_t n, double *dst)
{
    if (!src || !dst || n < 0 || dtype < OR_F16 || dtype > OR_F64)
        return 1;
    for (int64_t i = 0; i < n; ++i)
        dst[i] = or_elem(src, dtype, i);
    return 0;
}

/*
 * Attention, Eq. 3, for Q [B,H,Lq,D], K and V [B,H,Lk,D] (contiguous,
 * D innermost), all of element type `dtype`.
 *
 * rows: NULL for every query row, else `nrows` flat row indices
 *       r = (b*H + h)*Lq + i selecting the rows to compute.
 * out:  [nrows or B*H*Lq][D] doubles, row by row in the order asked for.
 * L, S: optional [same rows] doubles receiving Eq. 4's L_i and S_i.
 * dev:  optional [same rows][D] doubles receiving, after the three passes,
 *       dev_id = sum_j p_ij |v_jd - o_id| with p_ij = exp(a_ij - L_i) / S_i:
 *       the mean absolute deviation of the value column under the weights.
 *       It is not part of Eq. 3; the GPU parity tests derive from it how far
 *       a relative rounding of every weight can move o_id (first order: by at
 *       most that relative size times dev_id).
 * Returns 0, or 1 on a bad argument.
 */
int oracle_attention_f64(const void *q, const void *k, const void *v, int dtype,
                         int B, int H, int Lq, int Lk, int D, float scale,
                         const int64_t *rows, int64_t nrows, int nthreads,
                         double *out, double *L, double *S, double *dev)
{
    if (!q || !k || !v || !out || B < 1 || H < 1 || Lq < 1 || Lk < 1 || D < 1 ||
        dtype < OR_F16 || dtype > OR_F64)
        return 1;
    const int64_t total = (int64_t)B * H * Lq;
    const int64_t n = rows ? nrows : total;
    if (n < 0)
        return 1;
    if (rows)
        for (int64_t t = 0; t < n; ++t)
            if (rows[t] < 0 || rows[t] >= total)
                return 1;
    const double sc = (double)scale;
    int bad = 0;

#pragma omp parallel num_threads(oracle_num_threads(nthreads)) reduction(| : bad)
    {
        double *a = (double *)malloc(sizeof(double) * (size_t)Lk);
        if (!a) {
            bad = 1;
        } else {
#pragma omp for schedule(static)
            for (int64_t t = 0; t < n; ++t) {
                const int64_t r = rows ? rows[t] : t;
                const int64_t bh = r / Lq;             /* (b, h) pair */
                const int64_t qrow = r * D;            /* start of q_i */
                const int64_t kv0 = bh * Lk * D;       /* start of K, V of this head */

                /* pass 1: a_ij = scale * <q_i, k_j>, and L_i = max_j a_ij */
                double Li = -INFINITY;
                for (int j = 0; j < Lk; ++j) {
                    double dot = 0.0;
                    for (int d = 0; d < D; ++d)
                        dot += or_elem(q, dtype, qrow + d) *
                               or_elem(k, dtype, kv0 + (int64_t)j * D + d);
                    a[j] = sc * dot;
                    if (a[j] > Li)
                        Li = a[j];
                }
                /* pass 2: S_i = sum_j exp(a_ij - L_i) */
                double Si = 0.0;
                for (int j = 0; j < Lk; ++j)
                    Si += exp(a[j] - Li);
                /* pass 3: o_i = sum_j exp(a_ij - L_i) / S_i * v_j */
                double *o = out + t * D;
                for (int d = 0; d < D; ++d)
                    o[d] = 0.0;
                for (int j = 0; j < Lk; ++j) {
                    const double pij = exp(a[j] - Li) / Si;
                    for (int d = 0; d < D; ++d)
                        o[d] += pij * or_elem(v, dtype, kv0 + (int64_t)j * D + d);
                }
                if (dev) {
                    double *e = dev + t * D;
                    for (int d = 0; d < D; ++d)
                        e[d] = 0.0;
                    for (int j = 0; j < Lk; ++j) {
                        const double pij = exp(a[j] - Li) / Si;
                        for (int d = 0; d < D; ++d)
                            e[d] += pij * fabs(or_elem(v, dtype, kv0 + (int64_t)j * D + d) - o[d]);
                    }
                }
                if (L)
                    L[t] = Li;
                if (S)
                    S[t] = Si;
            }
            free(a);
        }
    }
    return bad;
}

/*
 * The reduction step of Eq. 4 on a given matrix A [rows][cols] of type
 * `dtype`, with the scale applied first (a_ij = scale * A_ij):
 *   ls[2r]   = L_r = max_j a_rj
 *   ls[2r+1] = S_r = sum_j exp(a_rj - L_r)
 * and, when p is not NULL, the element-wise step p_rj = exp(a_rj - L_r) / S_r.
 */
int oracle_softmax_rows_f64(const void *a, int dtype, int64_t rows, int64_t cols,
                            float scale, int nthreads, double *ls, double *p)
{
    if (!a || !ls || rows < 1 || cols < 1 || dtype < OR_F16 || dtype > OR_F64)
        return 1;
    const double sc = (double)scale;

#pragma omp parallel for schedule(static) num_threads(oracle_num_threads(nthreads))
    for (int64_t r = 0; r < rows; ++r) {
        const int64_t base = r * cols;
        double Lr = -INFINITY;
        for (int64_t j = 0; j < cols; ++j) {
            const double x = sc * or_elem(a, dtype, base + j);
            if (x > Lr)
                Lr = x;
        }
        double Sr = 0.0;
        for (int64_t j = 0; j < cols; ++j)
            Sr += exp(sc * or_elem(a, dtype, base + j) - Lr);
        ls[2 * r] = Lr;
        ls[2 * r + 1] = Sr;
        if (p)
            for (int64_t j = 0; j < cols; ++j)
                p[base + j] = exp(sc * or_elem(a, dtype, base + j) - Lr) / Sr;
    }
    return 0;
}

/*
 * The partially fused softmax of Sec. 3.2.1 splits Eq. 3 into three steps:
 * the logit matrix, Eq. 4's reduction (oracle_softmax_rows_f64 above), and
 * the element-wise normalisation fused with the product by V.  The first and
 * last steps follow.
 *
 * Logits: out[t][j] = scale * <q_i, k_j> for the query row r = (b*H + h)*Lq + i
 * (all B*H*Lq rows when `rows` is NULL, else the `nrows` rows listed), Q
 * [B,H,Lq,D] and K [B,H,Lk,D] of element type `dtype`.  out: [n][Lk] doubles.
 */
int oracle_logits_f64(const void *q, const void *k, int dtype, int B, int H, int Lq, int Lk,
                      int D, float scale, const int64_t *rows, int64_t nrows, int nthreads,
                      double *out)
{
    if (!q || !k || !out || B < 1 || H < 1 || Lq < 1 || Lk < 1 || D < 1 ||
        dtype < OR_F16 || dtype > OR_F64)
        return 1;
    const int64_t total = (int64_t)B * H * Lq;
    const int64_t n = rows ? nrows : total;
    if (n < 0)
        return 1;
    if (rows)
        for (int64_t t = 0; t < n; ++t)
            if (rows[t] < 0 || rows[t] >= total)
                return 1;
    const double sc = (double)scale;

#pragma omp parallel for schedule(static) num_threads(oracle_num_threads(nthreads))
    for (int64_t t = 0; t < n; ++t) {
        const int64_t r = rows ? rows[t] : t;
        const int64_t qrow = r * D;
        const int64_t k0 = (r / Lq) * Lk * D;
        for (int j = 0; j < Lk; ++j) {
            double dot = 0.0;
            for (int d = 0; d < D; ++d)
                dot += or_elem(q, dtype, qrow + d) * or_elem(k, dtype, k0 + (int64_t)j * D + d);
            out[t * Lk + j] = sc * dot;
        }
    }
    return 0;
}

/*
 * Normalise and multiply by V: for each selected row r of the logit matrix A
 * [B,H,Lq,Lk] (element type a_dtype, the scale already applied) and V
 * [B,H,Lk,D] (element type v_dtype),
 *   o[t][d] = sum_j exp(a_rj - L_r) / S_r * v_jd,
 * with (L_r, S_r) = ls[2r], ls[2r+1] when `ls` is given ([B*H*Lq][2]
 * doubles), else Eq. 4 computed from A's row: L_r = max_j a_rj,
 * S_r = sum_j exp(a_rj - L_r).  out: [n][D] doubles.
 */
int oracle_softmax_pv_f64(const void *a, int a_dtype, const double *ls, const void *v,
                          int v_dtype, int B, int H, int Lq, int Lk, int D, const int64_t *rows,
                          int64_t nrows, int nthreads, double *out)
{
    if (!a || !v || !out || B < 1 || H < 1 || Lq < 1 || Lk < 1 || D < 1 ||
        a_dtype < OR_F16 || a_dtype > OR_F64 || v_dtype < OR_F16 || v_dtype > OR_F64)
        return 1;
    const int64_t total = (int64_t)B * H * Lq;
    const int64_t n = rows ? nrows : total;
    if (n < 0)
        return 1;
    if (rows)
        for (int64_t t = 0; t < n; ++t)
            if (rows[t] < 0 || rows[t] >= total)
                return 1;

#pragma omp parallel for schedule(static) num_threads(oracle_num_threads(nthreads))
    for (int64_t t = 0; t < n; ++t) {
        const int64_t r = rows ? rows[t] : t;
        const int64_t arow = r * Lk;
        const int64_t v0 = (r / Lq) * Lk * D;
        double Lr, Sr;
        if (ls) {
            Lr = ls[2 * r];
            Sr = ls[2 * r + 1];
        } else {
            Lr = -INFINITY;
            for (int j = 0; j < Lk; ++j) {
                const double x = or_elem(a, a_dtype, arow + j);
                if (x > Lr)
                    Lr = x;
            }
            Sr = 0.0;
            for (int j = 0; j < Lk; ++j)
                Sr += exp(or_elem(a, a_dtype, arow + j) - Lr);
        }
        double *o = out + t * D;
        for (int d = 0; d < D; ++d)
            o[d] = 0.0;
        for (int j = 0; j < Lk; ++j) {
            const double pij = exp(or_elem(a, a_dtype, arow + j) - Lr) / Sr;
            for (int d = 0; d < D; ++d)
                o[d] += pij * or_elem(v, v_dtype, v0 + (int64_t)j * D + d);
        }
    }
    return 0;
}

/*
 * The steps either side of the attention in SD's UNet transformer blocks:
 * a linear layer, and the attention block built from them.
 *
 * Linear layer with weights stored [out, in]:
 *   y[m][n] = sum_k x[m][k] * w[n][k] + bias[n]   (bias may be NULL)
 * x [M][K] of x_dtype, w [N][K] of w_dtype, bias [N] of w_dtype; y [M][N] doubles.
 */
int oracle_linear_f64(const void *x, int x_dtype, const void *w, int w_dtype, const void *bias,
                      int64_t M, int K, int N, int nthreads, double *y)
{
    if (!x || !w || !y || M < 1 || K < 1 || N < 1 || x_dtype < OR_F16 || x_dtype > OR_F64 ||
        w_dtype < OR_F16 || w_dtype > OR_F64)
        return 1;

#pragma omp parallel for schedule(static) num_threads(oracle_num_threads(nthreads))
    for (int64_t m = 0; m < M; ++m) {
        for (int n = 0; n < N; ++n) {
            double acc = 0.0;
            for (int k = 0; k < K; ++k)
                acc += or_elem(x, x_dtype, m * K + k) * or_elem(w, w_dtype, (int64_t)n * K + k);
            y[m * N + n] = acc + (bias ? or_elem(bias, w_dtype, n) : 0.0);
        }
    }
    return 0;
}

/*
 * The attention block (multi-head attention over Eq. 3), all tensors of one
 * element type `dtype`:
 *   x   [B][Lq][C]   latent tokens          ctx [B][Lk][Cc]  context tokens
 *   wq  [C][C], wk [C][Cc], wv [C][Cc], wo [C][C]  (weights [out, in]); bo [C]
 *   Q = x wq^T, K = ctx wk^T, V = ctx wv^T, each split into H heads of D = C/H
 *   channels (head h holds channels h*D .. h*D + D - 1);
 *   O_h = softmax(scale Q_h K_h^T) V_h per head (Eq. 3);
 *   out = [O_0 | O_1 | ... | O_{H-1}] wo^T + bo.
 * Q, K, V and O stay in fp64 between the steps.  rows: NULL for all B*Lq
 * rows, else `nrows` flat rows b*Lq + i.  out: [n][C] doubles.
 */
int oracle_attention_block_f64(const void *x, const void *ctx, const void *wq, const void *wk,
                               const void *wv, const void *wo, const void *bo, int dtype, int B,
                               int Lq, int Lk, int C, int Cc, int H, float scale,
                               const int64_t *rows, int64_t nrows, int nthreads, double *out)
{
    if (!x || !ctx || !wq || !wk || !wv || !wo || !out || B < 1 || Lq < 1 || Lk < 1 || C < 1 ||
        Cc < 1 || H < 1 || C % H != 0 || dtype < OR_F16 || dtype > OR_F64)
        return 1;
    const int D = C / H;
    const int64_t total = (int64_t)B * Lq;
    const int64_t n = rows ? nrows : total;
    if (n < 0)
        return 1;
    if (rows)
        for (int64_t t = 0; t < n; ++t)
            if (rows[t] < 0 || rows[t] >= total)
                return 1;
    /* K and V of every context token: [B][Lk][C] each */
    double *Kf = (double *)malloc(sizeof(double) * (size_t)B * Lk * C);
    double *Vf = (double *)malloc(sizeof(double) * (size_t)B * Lk * C);
    if (!Kf || !Vf) {
        free(Kf);
        free(Vf);
        return 1;
    }
    if (oracle_linear_f64(ctx, dtype, wk, dtype, NULL, (int64_t)B * Lk, Cc, C, nthreads, Kf) ||
        oracle_linear_f64(ctx, dtype, wv, dtype, NULL, (int64_t)B * Lk, Cc, C, nthreads, Vf)) {
        free(Kf);
        free(Vf);
        return 1;
    }
    const double sc = (double)scale;
    int bad = 0;

#pragma omp parallel num_threads(oracle_num_threads(nthreads)) reduction(| : bad)
    {
        double *q = (double *)malloc(sizeof(double) * (size_t)C);
        double *o = (double *)malloc(sizeof(double) * (size_t)C);
        double *a = (double *)malloc(sizeof(double) * (size_t)Lk);
        if (!q || !o || !a) {
            bad = 1;
        } else {
#pragma omp for schedule(static)
            for (int64_t t = 0; t < n; ++t) {
                const int64_t r = rows ? rows[t] : t;
                const int64_t b = r / Lq;
                /* q = x_r wq^T */
                for (int c = 0; c < C; ++c) {
                    double acc = 0.0;
                    for (int k = 0; k < C; ++k)
                        acc += or_elem(x, dtype, r * C + k) * or_elem(wq, dtype, (int64_t)c * C + k);
                    q[c] = acc;
                }
                /* each head: Eq. 3 in three passes (max, exp-sum, normalise times V) */
                for (int h = 0; h < H; ++h) {
                    double Lh = -INFINITY;
                    for (int j = 0; j < Lk; ++j) {
                        const double *kj = Kf + ((size_t)b * Lk + j) * C + (size_t)h * D;
                        double dot = 0.0;
                        for (int d = 0; d < D; ++d)
                            dot += q[h * D + d] * kj[d];
                        a[j] = sc * dot;
                        if (a[j] > Lh)
                            Lh = a[j];
                    }
                    double Sh = 0.0;
                    for (int j = 0; j < Lk; ++j)
                        Sh += exp(a[j] - Lh);
                    for (int d = 0; d < D; ++d)
                        o[h * D + d] = 0.0;
                    for (int j = 0; j < Lk; ++j) {
                        const double pij = exp(a[j] - Lh) / Sh;
                        const double *vj = Vf + ((size_t)b * Lk + j) * C + (size_t)h * D;
                        for (int d = 0; d < D; ++d)
                            o[h * D + d] += pij * vj[d];
                    }
                }
                /* out = o wo^T + bo */
                for (int c = 0; c < C; ++c) {
                    double acc = 0.0;
                    for (int k = 0; k < C; ++k)
                        acc += o[k] * or_elem(wo, dtype, (int64_t)c * C + k);
                    out[t * C + c] = acc + (bo ? or_elem(bo, dtype, c) : 0.0);
                }
            }
        }
        free(q);
        free(o);
        free(a);
    }
    free(Kf);
    free(Vf);
    return bad;
}

/*
 * Group normalisation (Sec. 3.1, Eq. 1) of feature maps x [B][C][HW] (the
 * channel-major layout of the UNet's convolution outputs) of type `dtype`.
 * The C channels form G groups of C/G consecutive channels; group (b, g)
 * holds the (C/G)*HW values of channels g*C/G .. (g+1)*C/G - 1 of batch b.
 *   mu  = the group's mean,  var = the mean of (x - mu)^2  (a second pass),
 *   y_i = (x_i - mu) / sqrt(var + eps) * gamma_c + beta_c   (c: x_i's channel).
 * Eq. 1 is the case eps = 0 without the per-channel affine terms; gamma and
 * beta (type `dtype`, [C]) may be NULL for 1 and 0.  mean and rstd, when not
 * NULL, receive mu and 1/sqrt(var + eps) per group, [B][G].
 */
int oracle_group_norm_f64(const void *x, int dtype, const void *gamma, const void *beta, int B,
                          int C, int64_t HW, int G, double eps, int nthreads, double *y,
                          double *mean, double *rstd)
{
    if (!x || !y || B < 1 || C < 1 || HW < 1 || G < 1 || C % G != 0 || eps < 0.0 ||
        dtype < OR_F16 || dtype > OR_F64)
        return 1;
    const int cpg = C / G;
    const int64_t n = (int64_t)cpg * HW;

#pragma omp parallel for schedule(static) num_threads(oracle_num_threads(nthreads))
    for (int64_t bg = 0; bg < (int64_t)B * G; ++bg) {
        const int64_t base = bg * n;   /* the group's values are contiguous */
        double s = 0.0;
        for (int64_t i = 0; i < n; ++i)
            s += or_elem(x, dtype, base + i);
        const double mu = s / (double)n;
        double s2 = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            const double d = or_elem(x, dtype, base + i) - mu;
            s2 += d * d;
        }
        const double var = s2 / (double)n;
        const double inv = 1.0 / sqrt(var + eps);
        const int g = (int)(bg % G);
        for (int64_t i = 0; i < n; ++i) {
            const int c = g * cpg + (int)(i / HW);
            const double ga = gamma ? or_elem(gamma, dtype, c) : 1.0;
            const double be = beta ? or_elem(beta, dtype, c) : 0.0;
            y[base + i] = (or_elem(x, dtype, base + i) - mu) * inv * ga + be;
        }
        if (mean)
            mean[bg] = mu;
        if (rstd)
            rstd[bg] = inv;
    }
    return 0;
}

/* GELU of Eq. 2, element-wise: out_i = x_i / 2 * (1 + erf(x_i / sqrt(2))). */
int oracle_gelu_f64(const void *x, int dtype, int64_t n, double *out)
{
    if (!x || !out || n < 0 || dtype < OR_F16 || dtype > OR_F64)
        return 1;
    for (int64_t i = 0; i < n; ++i) {
        const double v = or_elem(x, dtype, i);
        out[i] = 0.5 * v * (1.0 + erf(v / sqrt(2.0)));
    }
    return 0;
}

/*
 * The GELU of Eq. 2 with the split and multiply around it (the gated
 * feed-forward of the transformer block): h [M][2F] of type `dtype` is split
 * along its last axis into a value half and a gate half,
 *   out[m][f] = h[m][f] * GELU(h[m][F + f]),   out [M][F] doubles.
 */
int oracle_geglu_f64(const void *h, int dtype, int64_t M, int F, int nthreads, double *out)
{
    if (!h || !out || M < 1 || F < 1 || dtype < OR_F16 || dtype > OR_F64)
        return 1;

#pragma omp parallel for schedule(static) num_threads(oracle_num_threads(nthreads))
    for (int64_t m = 0; m < M; ++m) {
        for (int f = 0; f < F; ++f) {
            const double a = or_elem(h, dtype, m * 2 * F + f);
            const double g = or_elem(h, dtype, m * 2 * F + F + f);
            out[m * F + f] = a * (0.5 * g * (1.0 + erf(g / sqrt(2.0))));
        }
    }
    return 0;
}

/*
 * 3x3 convolution, stride 1, zero padding 1 (the layers Sec. 3.3 accelerates
 * with Winograd's algorithm; the oracle is the convolution's definition):
 *   y[b][o][i][j] = bias[o] + sum_{c, u, v} w[o][c][u][v] * x[b][c][i + u - 1][j + v - 1]
 * with x taken as 0 outside the H x W map.  x [B][Ci][H][W], w [Co][Ci][3][3],
 * bias [Co] or NULL, all of type `dtype`; y [B][Co][H][W] doubles.
 */
int oracle_conv3x3_f64(const void *x, const void *w, const void *bias, int dtype, int B, int Ci,
                       int Co, int H, int W, int nthreads, double *y)
{
    if (!x || !w || !y || B < 1 || Ci < 1 || Co < 1 || H < 1 || W < 1 || dtype < OR_F16 ||
        dtype > OR_F64)
        return 1;

#pragma omp parallel for schedule(static) num_threads(oracle_num_threads(nthreads))
    for (int64_t bo = 0; bo < (int64_t)B * Co; ++bo) {
        const int64_t b = bo / Co;
        const int o = (int)(bo % Co);
        const double bo_v = bias ? or_elem(bias, dtype, o) : 0.0;
        for (int i = 0; i < H; ++i) {
            for (int j = 0; j < W; ++j) {
                double acc = 0.0;
                for (int c = 0; c < Ci; ++c) {
                    for (int u = 0; u < 3; ++u) {
                        const int ii = i + u - 1;
                        if (ii < 0 || ii >= H)
                            continue;
                        for (int v = 0; v < 3; ++v) {
                            const int jj = j + v - 1;
                            if (jj < 0 || jj >= W)
                                continue;
                            acc += or_elem(w, dtype, (((int64_t)o * Ci + c) * 3 + u) * 3 + v) *
                                   or_elem(x, dtype, ((b * Ci + c) * H + ii) * (int64_t)W + jj);
                        }
                    }
                }
                y[(bo * H + i) * (int64_t)W + j] = acc + bo_v;
            }
        }
    }
    return 0;
}
