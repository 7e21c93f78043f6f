/*
 * Driver of the C oracle for the AddressSanitizer / UndefinedBehaviorSanitizer
 * build (tests/test_sanitizers.py): every exported entry point on small
 * shapes (square, rectangular, post-padded, batch-padded lengths including
 * 0 and whole blocks of padding, the objective, exact attention on sampled
 * rows) and the argument checks.  Inputs come from a 64-bit LCG; the driver
 * checks only that the outputs are finite and that rows past a length are
 * zero, the sanitizers check the memory accesses and the arithmetic.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int ma_oracle_fwd_f64(const double *q, const double *k, const double *v, double *out, int64_t B, int64_t H,
                      int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t threads);
int ma_oracle_fwd_obj_f64(const double *q, const double *k, const double *v, double *out, double *obj, int64_t B,
                          int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t threads);
int ma_oracle_fwd_varlen_f64(const double *q, const double *k, const double *v, double *out, const int64_t *lens,
                             int64_t B, int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T,
                             int32_t threads);
int ma_oracle_dense_attn_f64(const double *q, const double *k, const double *v, double *out, int64_t BH, int64_t N,
                             int64_t d, const int64_t *row_idx, int64_t rows, int32_t threads);

static uint64_t state = 0x9e3779b97f4a7c15ull;

static double draw(void)
{
    state = state * 6364136223846793005ull + 1442695040888963407ull;
    return ((double)(state >> 11) / 9007199254740992.0 - 0.5) * 3.0;
}

static double *filled(size_t n)
{
    double *x = malloc(n * sizeof(double));
    if (!x) exit(3);
    for (size_t i = 0; i < n; ++i) x[i] = draw();
    return x;
}

static int finite_all(const double *x, size_t n)
{
    for (size_t i = 0; i < n; ++i)
        if (!isfinite(x[i])) return 0;
    return 1;
}

static int fails = 0;

static void expect(int cond, const char *what)
{
    if (!cond) {
        fprintf(stderr, "FAILED: %s\n", what);
        ++fails;
    }
}

static void run_shape(int64_t B, int64_t H, int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t threads)
{
    const size_t n = (size_t)(B * H * N * d);
    double *q = filled(n), *k = filled(n), *v = filled(n), *o = filled(n);
    double *obj = malloc(sizeof(double) * (size_t)(B * H * T));
    if (!obj) exit(3);
    expect(ma_oracle_fwd_f64(q, k, v, o, B, H, N, d, m, b, T, threads) == 0, "fwd status");
    expect(finite_all(o, n), "fwd finite");
    expect(ma_oracle_fwd_obj_f64(q, k, v, o, obj, B, H, N, d, m, b, T, threads) == 0, "objective status");
    expect(finite_all(obj, (size_t)(B * H * T)), "objective finite");
    int64_t *lens = malloc(sizeof(int64_t) * (size_t)B);
    if (!lens) exit(3);
    for (int64_t e = 0; e < B; ++e) lens[e] = (e % 4 == 0) ? N : (e % 4 == 1) ? 0 : (e % 4 == 2) ? 1 : N / 3;
    expect(ma_oracle_fwd_varlen_f64(q, k, v, o, lens, B, H, N, d, m, b, T, threads) == 0, "varlen status");
    expect(finite_all(o, n), "varlen finite");
    for (int64_t e = 0; e < B; ++e)
        for (int64_t h = 0; h < H; ++h)
            for (int64_t r = lens[e]; r < N; ++r)
                for (int64_t c = 0; c < d; ++c) expect(o[((e * H + h) * N + r) * d + c] == 0.0, "varlen zero rows");
    int64_t rows[3] = {0, N / 2, N - 1};
    double *dense = malloc(sizeof(double) * (size_t)(B * H * 3 * d));
    if (!dense) exit(3);
    expect(ma_oracle_dense_attn_f64(q, k, v, dense, B * H, N, d, rows, 3, threads) == 0, "dense status");
    expect(finite_all(dense, (size_t)(B * H * 3 * d)), "dense finite");
    free(q); free(k); free(v); free(o); free(obj); free(lens); free(dense);
}

int main(void)
{
    run_shape(1, 1, 16, 8, 4, 4, 1, 1);
    run_shape(2, 3, 30, 12, 5, 6, 3, 4);      /* rectangular, several heads */
    run_shape(4, 1, 37, 8, 5, 8, 2, 3);       /* post-padded: 37 rows in 5 blocks of 8 */
    run_shape(1, 2, 7, 4, 1, 7, 2, 2);        /* one block */
    run_shape(1, 1, 9, 4, 9, 1, 2, 2);        /* b = 1 */
    run_shape(3, 2, 64, 16, 8, 8, 4, 8);
    /* argument checks */
    double x[64] = {0};
    expect(ma_oracle_fwd_f64(NULL, x, x, x, 1, 1, 4, 4, 2, 2, 1, 1) != 0, "null q rejected");
    expect(ma_oracle_fwd_f64(x, x, x, x, 1, 1, 4, 4, 1, 2, 1, 1) != 0, "m != ceil(N/b) rejected");
    expect(ma_oracle_fwd_f64(x, x, x, x, 1, 1, 4, 4, 2, 2, 0, 1) != 0, "T = 0 rejected");
    int64_t bad = 5;
    expect(ma_oracle_fwd_varlen_f64(x, x, x, x, &bad, 1, 1, 4, 4, 2, 2, 1, 1) != 0, "length > N rejected");
    if (fails) return 1;
    printf("oracle sanitizer run: ok\n");
    return 0;
}
