/*
 * fp64 CPU oracle of the MonarchAttention forward pass.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain reference that the
 * HIP library is checked against.  Only the test suite, the smoke check and
 * the benchmark's CPU-baseline leg may build, load or call it; the product
 * path never does, and it shares no code, header or table with the HIP path.
 *
 * What it computes (paper, Sec. 3 "MonarchAttention" and its "Implementation"
 * paragraph; the algorithm of Fig. "Python-like code for MonarchAttention"):
 * for every (batch, head) slice with Q, K, V in R^{N x d}, N = m*b (see below
 * for N < m*b),
 *
 *   Qbar[j][l] = Q[l*b + j],  Kbar[k][i] = K[k*b + i],  Vbar[k][i] = V[k*b + i]
 *                        (row (l,j) of the "transpose" permutation P, Sec. 2)
 *   L^(0)[j][k][l] = delta_kl                            (init, Sec. 3)
 *   for t = 1..T:
 *     alpha_R[k][j] = sum_l L[j][k][l] Qbar[j][l]        (eq. beta_r)
 *     c_R[k][j]     = sum_l L[j][k][l]                   (eq. beta_r)
 *     beta_R[k][j][i] = <alpha_R[k][j], Kbar[k][i]>      (eq. beta_r)
 *     R[k][j][:]    = softmax_i(beta_R[k][j][:] / c_R[k][j])       (eq. R_update)
 *     alpha_L[j][k] = sum_i R[k][j][i] Kbar[k][i]        (eq. beta_l)
 *     c_L[j][k]     = sum_i R[k][j][i] log R[k][j][i]    (eq. beta_l)
 *     beta_L[j][k][l] = <alpha_L[j][k], Qbar[j][l]>      (eq. beta_l)
 *     L[j][:][l]    = softmax_k(beta_L[j][:][l] - c_L[j][:])       (eq. L_update)
 *   Y[j][k]     = sum_i R[k][j][i] Vbar[k][i]            (eq. monarch_multiply)
 *   O[l*b + j]  = sum_k L[j][k][l] Y[j][k]               (eq. monarch_multiply)
 *
 * The scores use Q K^T / sqrt(d): the factor s = 1/sqrt(d) is absorbed into Q
 * (Sec. 2, footnote on attention), i.e. Qbar above holds s * Q.
 *
 * Organisation: the state form of the Implementation paragraph, in which L and
 * R are never stored; only alpha_R, c_R, alpha_L, c_L (and Y) are kept.  At
 * t = 1 the identity L^(0) gives alpha_R[k][j] = Qbar[j][k] = s*Q[k*b + j] and
 * c_R = 1.  The R half-step runs over all (k, j) and the L half-step over all
 * (j, l); in the last iteration the L half-step is fused with the second
 * Monarch product, exactly as the paper's last two kernels do.  OpenMP
 * distributes the independent (head, k) and (head, j) units; it does not
 * change any element's arithmetic.
 *
 * c_L follows its definition: sum_i R log R, with the limit 0 * log 0 = 0 for
 * entries that underflow to zero.
 *
 * Sequence lengths that are not a multiple of b (Appendix "Padding and
 * Masking"): with m = ceil(N / b), Q, K and V are post-padded with zero rows
 * to N' = m*b (the paper leaves the pad value open; zero is the reading taken
 * here, and the padded query rows take part in the iteration like any other
 * row), the mask omega adds -inf to Z_R for every key position k*b + i >= N
 * before the softmax of eq. R_update, so that the last N' - N columns of M
 * are zero, and only the first N rows of O are returned.
 *
 * Batched sequences padded to a common length (the same appendix): with
 * ma_oracle_fwd_varlen_f64, head h of batch element beta has lens[beta] <= N
 * real rows and keeps the batch's m and b, so whole key blocks can be
 * padding.  Such a block has no defined R softmax (every entry of its omega
 * row is -inf); the reading taken here gives it R = 0 (so alpha_L, c_L and Y
 * of that block are zero) and leaves it out of the L softmax (Z_L = -inf),
 * so that M keeps unit row sums; with no real key at all L = 0.  Rows >=
 * lens[beta] of O are zero.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Index of the calling thread within the current parallel region (0 without OpenMP). */
static int thread_index(void)
{
#ifdef _OPENMP
    return omp_get_thread_num();
#else
    return 0;
#endif
}

#define MO_OK 0
#define MO_EINVAL 1
#define MO_ENOMEM 4

/* One R half-step for unit (head, k), eq. R_update, beta_r, beta_l.
 * aR[k][j][:] and cR[k][j] are the inputs; writes aL[j][k][:], cL[j][k] and,
 * when y != NULL, Y[j][k][:].  kreal[k*b + i] is 0 where key position
 * k*b + i is padding: the mask omega = -inf is added to its Z_R (Appendix
 * "Padding and Masking"). */
static void r_half_step(const double *Kh, const double *Vh, const double *aR, const double *cR,
                        double *aL, double *cL, double *Y, int64_t m, int64_t b, int64_t d,
                        int64_t k, const unsigned char *kreal, double *z)
{
    const double *Kk = Kh + k * b * d; /* Kbar[k][i] = K[k*b + i] */
    const double *Vk = Vh ? Vh + k * b * d : NULL;
    int64_t nkeys = 0; /* real keys of block k */
    for (int64_t i = 0; i < b; ++i) nkeys += kreal[k * b + i] != 0;
    if (nkeys == 0) { /* a block of padding only: R[k] = 0 */
        for (int64_t j = 0; j < b; ++j) {
            cL[j * m + k] = 0.0;
            memset(aL + (j * m + k) * d, 0, (size_t)d * sizeof(double));
            if (Y) memset(Y + (j * m + k) * d, 0, (size_t)d * sizeof(double));
        }
        return;
    }
    for (int64_t j = 0; j < b; ++j) {
        const double *a = aR + (k * b + j) * d;
        const double c = cR[k * b + j];
        double zmax = -INFINITY;
        for (int64_t i = 0; i < b; ++i) {
            double beta = 0.0;
            for (int64_t v = 0; v < d; ++v) beta += a[v] * Kk[i * d + v];
            z[i] = kreal[k * b + i] ? beta / c : -INFINITY; /* + omega[k][j][i] */
            if (z[i] > zmax) zmax = z[i];
        }
        double sum = 0.0;
        for (int64_t i = 0; i < b; ++i) {
            z[i] = exp(z[i] - zmax);
            sum += z[i];
        }
        double neg_entropy = 0.0;
        for (int64_t i = 0; i < b; ++i) {
            z[i] /= sum; /* z now holds R[k][j][:] */
            if (z[i] > 0.0) neg_entropy += z[i] * log(z[i]);
        }
        cL[j * m + k] = neg_entropy;
        double *al = aL + (j * m + k) * d;
        for (int64_t v = 0; v < d; ++v) {
            double acc = 0.0;
            for (int64_t i = 0; i < b; ++i) acc += z[i] * Kk[i * d + v];
            al[v] = acc;
        }
        if (Y) {
            double *y = Y + (j * m + k) * d;
            for (int64_t v = 0; v < d; ++v) {
                double acc = 0.0;
                for (int64_t i = 0; i < b; ++i) acc += z[i] * Vk[i * d + v];
                y[v] = acc;
            }
        }
    }
}

/* One L half-step for unit (head, j), eq. L_update and beta_l.  Qs is s*Q of
 * this head.  When O == NULL it accumulates aR[k][j][:] and cR[k][j] for the
 * next R half-step (eq. beta_r); otherwise it forms O[l*b + j] from Y (eq.
 * monarch_multiply).  When fj != NULL it also accumulates aR, cR and writes
 * to *fj the share of class j of the objective f(M) of the current factors,
 * in the separable form of Sec. 3 ("Softmax Objective"):
 *   sum_k <alpha_R[k][j], alpha_L[j][k]> + (1^T R_kj) H(L_jk) + (1^T L_jk) H(R_kj),
 * with 1^T R_kj = 1, 1^T L_jk = c_R[k][j], H(R_kj) = -c_L[j][k] and
 * H(L_jk) = -sum_l L log L (hl: m doubles of scratch).  Key blocks k with
 * blive[k] == 0 hold no real key (batch padding): Z_L = -inf for them, and
 * L = 0 when no block holds one. */
static void l_half_step(const double *Qs, const double *aL, const double *cL, const double *Y,
                        double *aR, double *cR, double *O, int64_t m, int64_t b, int64_t d,
                        int64_t j, const unsigned char *blive, double *z, double *fj, double *hl)
{
    int64_t live = 0; /* key blocks holding a real key */
    for (int64_t k = 0; k < m; ++k) live += blive[k] != 0;
    if (fj) {
        for (int64_t k = 0; k < m; ++k) hl[k] = 0.0;
    }
    if (!O || fj) {
        for (int64_t k = 0; k < m; ++k) {
            cR[k * b + j] = 0.0;
            memset(aR + (k * b + j) * d, 0, (size_t)d * sizeof(double));
        }
    }
    for (int64_t l = 0; l < m; ++l) {
        const double *qb = Qs + (l * b + j) * d; /* Qbar[j][l] = Q[l*b + j] */
        double zmax = -INFINITY;
        for (int64_t k = 0; k < m; ++k) {
            const double *al = aL + (j * m + k) * d;
            double beta = 0.0;
            for (int64_t v = 0; v < d; ++v) beta += al[v] * qb[v];
            z[k] = blive[k] ? beta - cL[j * m + k] : -INFINITY;
            if (z[k] > zmax) zmax = z[k];
        }
        if (live > 0) {
            double sum = 0.0;
            for (int64_t k = 0; k < m; ++k) {
                z[k] = exp(z[k] - zmax);
                sum += z[k];
            }
            for (int64_t k = 0; k < m; ++k) z[k] /= sum; /* z now holds L[j][:][l] */
        } else {
            for (int64_t k = 0; k < m; ++k) z[k] = 0.0;
        }
        if (fj) {
            for (int64_t k = 0; k < m; ++k)
                if (z[k] > 0.0) hl[k] -= z[k] * log(z[k]);
        }
        if (!O || fj) {
            for (int64_t k = 0; k < m; ++k) {
                cR[k * b + j] += z[k];
                double *ar = aR + (k * b + j) * d;
                for (int64_t v = 0; v < d; ++v) ar[v] += z[k] * qb[v];
            }
        }
        if (O) {
            double *o = O + (l * b + j) * d;
            for (int64_t v = 0; v < d; ++v) {
                double acc = 0.0;
                for (int64_t k = 0; k < m; ++k) acc += z[k] * Y[(j * m + k) * d + v];
                o[v] = acc;
            }
        }
    }
    if (fj) {
        double f = 0.0;
        for (int64_t k = 0; k < m; ++k) {
            const double *ar = aR + (k * b + j) * d, *al = aL + (j * m + k) * d;
            double dot = 0.0;
            for (int64_t v = 0; v < d; ++v) dot += ar[v] * al[v];
            f += dot + hl[k] - cR[k * b + j] * cL[j * m + k];
        }
        *fj = f;
    }
}

/* The forward pass; obj (NULL, or B*H*T doubles) receives f(M^(t); Q, K)
 * after every step t (the objective of Sec. 3 with the factors of step t, on
 * all m*b rows of the padded problem): obj[(h * T) + t - 1].  lens (NULL, or
 * B lengths <= N) gives the real rows of each batch element.
 *
 * Placement of the n real rows of a head (n = lens[e] or N) in the padded
 * sequence of Np = m*b positions (Appendix "Padding and Masking"):
 *   post-padding (pre = 0): the first n rows of the tensor at positions
 *                           0 .. n-1; positions n .. Np-1 are padding;
 *   pre-padding  (pre = 1): the last n rows of the tensor (rows N-n .. N-1)
 *                           at positions Np-n .. Np-1; positions below
 *                           Np-n are padding.
 * Padded positions hold zero rows and their keys are masked (omega = -inf
 * on Z_R); O is written at the real rows and is zero on the others. */
static int forward(const double *q, const double *k, const double *v, double *out, double *obj,
                   const int64_t *lens, int pre, int64_t B, int64_t H, int64_t N, int64_t d, int64_t m,
                   int64_t b, int32_t T, int32_t threads)
{
    if (!q || !k || !v || !out) return MO_EINVAL;
    if (B < 1 || H < 1 || d < 1 || m < 1 || b < 1 || T < 1 || N < 1) return MO_EINVAL;
    if (N > m * b || N <= (m - 1) * b) return MO_EINVAL; /* m = ceil(N / b) */
    if (lens) {
        if (obj) return MO_EINVAL;
        for (int64_t e = 0; e < B; ++e)
            if (lens[e] < 0 || lens[e] > N) return MO_EINVAL;
    }
    const int64_t BH = B * H, Np = m * b, nd = Np * d;
    const double s = 1.0 / sqrt((double)d);
    /* Q (scaled), K, V post-padded with zero rows to Np = m*b; O on Np rows */
    double *Qs = calloc((size_t)(BH * nd), sizeof(double));
    double *Kp = calloc((size_t)(BH * nd), sizeof(double));
    double *Vp = calloc((size_t)(BH * nd), sizeof(double));
    double *Op = malloc(sizeof(double) * (size_t)(BH * nd));
    double *aR = malloc(sizeof(double) * (size_t)(BH * nd));
    double *aL = malloc(sizeof(double) * (size_t)(BH * nd));
    double *Y = malloc(sizeof(double) * (size_t)(BH * nd));
    double *cR = malloc(sizeof(double) * (size_t)(BH * Np));
    double *cL = malloc(sizeof(double) * (size_t)(BH * Np));
    double *fpart = malloc(sizeof(double) * (size_t)(BH * b)); /* objective share of (head, j) */
    unsigned char *kreal = calloc((size_t)(BH * Np), 1);         /* real key positions of each head */
    unsigned char *blive = calloc((size_t)(BH * m), 1);          /* key blocks holding a real key */
    if (!Qs || !Kp || !Vp || !Op || !aR || !aL || !Y || !cR || !cL || !fpart || !kreal || !blive) {
        free(Qs); free(Kp); free(Vp); free(Op); free(aR); free(aL); free(Y); free(cR); free(cL); free(fpart);
        free(kreal); free(blive);
        return MO_ENOMEM;
    }
#ifdef _OPENMP
    const int nt = threads > 0 ? threads : omp_get_max_threads(); /* this call only */
#else
    const int nt = 1;
    (void)threads;
#endif
    const int64_t zlen = (m > b ? m : b);
    /* per-thread scratch rows, allocated (and checked) before the parallel regions */
    double *zbuf = malloc(sizeof(double) * (size_t)(nt * zlen));
    double *hbuf = malloc(sizeof(double) * (size_t)(nt * m));
    if (!zbuf || !hbuf) {
        free(zbuf); free(hbuf);
        free(Qs); free(Kp); free(Vp); free(Op); free(aR); free(aL); free(Y); free(cR); free(cL); free(fpart);
        free(kreal); free(blive);
        return MO_ENOMEM;
    }

#pragma omp parallel for schedule(static) num_threads(nt)
    for (int64_t h = 0; h < BH; ++h) {
        const int64_t n = lens ? lens[h / H] : N;
        const int64_t row0 = pre ? N - n : 0, pos0 = pre ? Np - n : 0; /* first real row, its position */
        for (int64_t r = 0; r < n; ++r) {
            for (int64_t e = 0; e < d; ++e) {
                Qs[h * nd + (pos0 + r) * d + e] = s * q[(h * N + row0 + r) * d + e]; /* scale absorbed into Q */
                Kp[h * nd + (pos0 + r) * d + e] = k[(h * N + row0 + r) * d + e];
                Vp[h * nd + (pos0 + r) * d + e] = v[(h * N + row0 + r) * d + e];
            }
            kreal[h * Np + pos0 + r] = 1;
            blive[h * m + (pos0 + r) / b] = 1;
        }
    }
    /* t = 1 state from L^(0) = I: alpha_R[k][j] = s*Q[k*b+j], c_R = 1. */
#pragma omp parallel for schedule(static) num_threads(nt)
    for (int64_t e = 0; e < BH * nd; ++e) aR[e] = Qs[e];
#pragma omp parallel for schedule(static) num_threads(nt)
    for (int64_t e = 0; e < BH * Np; ++e) cR[e] = 1.0;

    for (int32_t t = 1; t <= T; ++t) {
        const int last = (t == T);
#pragma omp parallel num_threads(nt)
        {
            double *z = zbuf + (size_t)thread_index() * (size_t)zlen;
            double *hl = hbuf + (size_t)thread_index() * (size_t)m;
#pragma omp for collapse(2) schedule(static)
            for (int64_t h = 0; h < BH; ++h)
                for (int64_t kk = 0; kk < m; ++kk)
                    r_half_step(Kp + h * nd, last ? Vp + h * nd : NULL, aR + h * nd, cR + h * Np,
                                aL + h * nd, cL + h * Np, last ? Y + h * nd : NULL, m, b, d, kk, kreal + h * Np, z);
#pragma omp for collapse(2) schedule(static)
            for (int64_t h = 0; h < BH; ++h)
                for (int64_t j = 0; j < b; ++j)
                    l_half_step(Qs + h * nd, aL + h * nd, cL + h * Np, Y + h * nd, aR + h * nd,
                                cR + h * Np, last ? Op + h * nd : NULL, m, b, d, j, blive + h * m, z,
                                obj ? fpart + h * b + j : NULL, hl);
        }
        if (obj) {
            for (int64_t h = 0; h < BH; ++h) {
                double f = 0.0;
                for (int64_t j = 0; j < b; ++j) f += fpart[h * b + j];
                obj[h * T + (t - 1)] = f;
            }
        }
    }
    /* O at the real rows of every head, zero on the others */
#pragma omp parallel for schedule(static) num_threads(nt)
    for (int64_t h = 0; h < BH; ++h) {
        const int64_t n = lens ? lens[h / H] : N;
        const int64_t row0 = pre ? N - n : 0, pos0 = pre ? Np - n : 0;
        memset(out + h * N * d, 0, sizeof(double) * (size_t)(N * d));
        memcpy(out + (h * N + row0) * d, Op + h * nd + pos0 * d, sizeof(double) * (size_t)(n * d));
    }
    free(Qs); free(Kp); free(Vp); free(Op); free(aR); free(aL); free(Y); free(cR); free(cL); free(fpart);
    free(kreal); free(blive);
    free(zbuf); free(hbuf);
    return MO_OK;
}

int ma_oracle_fwd_obj_f64(const double *q, const double *k, const double *v, double *out, double *obj,
                          int64_t B, int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T,
                          int32_t threads)
{
    return forward(q, k, v, out, obj, NULL, 0, B, H, N, d, m, b, T, threads);
}

/* Batch padding: lens[B] real rows per batch element (0 <= lens <= N). */
int ma_oracle_fwd_varlen_f64(const double *q, const double *k, const double *v, double *out,
                             const int64_t *lens, int64_t B, int64_t H, int64_t N, int64_t d, int64_t m,
                             int64_t b, int32_t T, int32_t threads)
{
    if (!lens) return MO_EINVAL;
    return forward(q, k, v, out, NULL, lens, 0, B, H, N, d, m, b, T, threads);
}

/* Pre-padded sequences (the last sentence of Appendix "Padding and
 * Masking"): the padding rows come before the real ones.  lens == NULL: all
 * N rows are real and the sequence is pre-padded to m*b; otherwise batch
 * element e holds lens[e] real rows as the LAST lens[e] rows of its N
 * (a left-padded batch), pre-padded to m*b, and its other rows of out are
 * zero. */
int ma_oracle_fwd_prepad_f64(const double *q, const double *k, const double *v, double *out, const int64_t *lens,
                             int64_t B, int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T,
                             int32_t threads)
{
    return forward(q, k, v, out, NULL, lens, 1, B, H, N, d, m, b, T, threads);
}

int ma_oracle_fwd_f64(const double *q, const double *k, const double *v, double *out, int64_t B,
                      int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T,
                      int32_t threads)
{
    return ma_oracle_fwd_obj_f64(q, k, v, out, NULL, B, H, N, d, m, b, T, threads);
}

/* Exact softmax attention O = softmax(Q K^T / sqrt(d)) V (eq. softmax_attention),
 * used only for the approximation-quality number.  rows: number of query rows
 * of each head to evaluate (row indices given in `row_idx`, or the first
 * `rows` rows when row_idx == NULL); out is [B*H, rows, d]. */
int ma_oracle_dense_attn_f64(const double *q, const double *k, const double *v, double *out,
                             int64_t BH, int64_t N, int64_t d, const int64_t *row_idx,
                             int64_t rows, int32_t threads)
{
    if (!q || !k || !v || !out || BH < 1 || N < 1 || d < 1 || rows < 1) return MO_EINVAL;
#ifdef _OPENMP
    const int nt = threads > 0 ? threads : omp_get_max_threads(); /* this call only */
#else
    const int nt = 1;
    (void)threads;
#endif
    const double s = 1.0 / sqrt((double)d);
    double *zbuf = malloc(sizeof(double) * (size_t)nt * (size_t)N); /* one score row per thread */
    if (!zbuf) return MO_ENOMEM;
#pragma omp parallel num_threads(nt)
    {
        double *z = zbuf + (size_t)thread_index() * (size_t)N;
#pragma omp for collapse(2) schedule(static)
        for (int64_t h = 0; h < BH; ++h)
            for (int64_t r = 0; r < rows; ++r) {
                const int64_t row = row_idx ? row_idx[r] : r;
                const double *qr = q + (h * N + row) * d;
                const double *kh = k + h * N * d, *vh = v + h * N * d;
                double zmax = -INFINITY, sum = 0.0;
                for (int64_t c = 0; c < N; ++c) {
                    double acc = 0.0;
                    for (int64_t e = 0; e < d; ++e) acc += qr[e] * kh[c * d + e];
                    z[c] = s * acc;
                    if (z[c] > zmax) zmax = z[c];
                }
                for (int64_t c = 0; c < N; ++c) {
                    z[c] = exp(z[c] - zmax);
                    sum += z[c];
                }
                double *o = out + (h * rows + r) * d;
                for (int64_t e = 0; e < d; ++e) o[e] = 0.0;
                for (int64_t c = 0; c < N; ++c) {
                    const double w = z[c] / sum;
                    for (int64_t e = 0; e < d; ++e) o[e] += w * vh[c * d + e];
                }
            }
    }
    free(zbuf);
    return MO_OK;
}

int ma_oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
