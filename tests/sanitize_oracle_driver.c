/*
 * Drives every entry point of the CPU oracle (oracle/pam_oracle.c) on small
 * seeded inputs, for a build with AddressSanitizer and UndefinedBehaviour-
 * Sanitizer (tests/test_sanitizers.py).  Checks a few invariants on the way;
 * exits non-zero on a failed check (the sanitizers abort on their own).
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

double orc_alpha(int d);
void orc_embedding_matrix(int d, double *E);
double orc_raw_scale(int d);
int orc_simplex(const float *p, int64_t n, int d, int32_t *keys, double *bary, int32_t *rank, double *xelev);
int64_t orc_lattice(int64_t n, int d, const int32_t *keys, int32_t *vert, int32_t *ukeys);
void orc_neighbours(int64_t M, int d, const int32_t *ukeys, int32_t *nbr);
void orc_splat(int64_t n, int d, int C, const int32_t *vert, const double *bary, const double *val, int64_t M,
               double *L);
int orc_blur(int64_t M, int d, int C, const int32_t *nbr, int reverse, double *L);
void orc_slice(int64_t n, int d, int C, const int32_t *vert, const double *bary, const double *L, double *out);
void orc_vertex_dots(int64_t n, int d, int C, const int32_t *vert, const double *a, const double *L, double *h);
void orc_embed_grad(int64_t n, int d, const int32_t *rank, const double *h, double *df);
void orc_gauss_bruteforce(int64_t n, int d, int C, const double *p, const double *v, double *out);

static uint64_t state = 1907;
static double uniform(void)
{
    state = state * 6364136223846793005ull + 1442695040888963407ull;
    return (double)(state >> 11) / 9007199254740992.0;
}

static int run(int d, int64_t n, int C)
{
    const int d1 = d + 1;
    float *p = malloc(sizeof(float) * n * d);
    double *pd = malloc(sizeof(double) * n * d), *val = malloc(sizeof(double) * n * C);
    for (int64_t i = 0; i < n * d; ++i) {
        p[i] = (float)(4.0 * uniform());
        pd[i] = p[i];
    }
    for (int64_t i = 0; i < n * C; ++i)
        val[i] = uniform() - 0.5;
    int32_t *keys = malloc(sizeof(int32_t) * n * d1 * d), *rank = malloc(sizeof(int32_t) * n * d1);
    double *bary = malloc(sizeof(double) * n * d1), *xel = malloc(sizeof(double) * n * d1);
    double *E = malloc(sizeof(double) * d1 * d);
    orc_embedding_matrix(d, E);
    if (orc_simplex(p, n, d, keys, bary, rank, xel) != 0)
        return 1;
    int32_t *vert = malloc(sizeof(int32_t) * n * d1), *ukeys = malloc(sizeof(int32_t) * n * d1 * d);
    const int64_t M = orc_lattice(n, d, keys, vert, ukeys);
    if (M <= 0 || M > n * d1)
        return 2;
    int32_t *nbr = malloc(sizeof(int32_t) * M * d1 * 2);
    orc_neighbours(M, d, ukeys, nbr);
    double *L = malloc(sizeof(double) * M * C), *out = malloc(sizeof(double) * n * C);
    double *h = malloc(sizeof(double) * n * d1), *df = malloc(sizeof(double) * n * d);
    double *ex = malloc(sizeof(double) * n * C);
    orc_splat(n, d, C, vert, bary, val, M, L);
    for (int rev = 0; rev < 2; ++rev)
        if (orc_blur(M, d, C, nbr, rev, L) != 0)
            return 3;
    orc_slice(n, d, C, vert, bary, L, out);
    orc_vertex_dots(n, d, C, vert, val, L, h);
    orc_embed_grad(n, d, rank, h, df);
    orc_gauss_bruteforce(n, d, C, pd, val, ex);
    for (int64_t i = 0; i < n; ++i) {
        double sb = 0.0;
        for (int k = 0; k < d1; ++k)
            sb += bary[i * d1 + k];
        if (fabs(sb - 1.0) > 1e-12)
            return 4;
    }
    for (int64_t e = 0; e < n * d1; ++e)
        if (vert[e] < 0 || vert[e] >= M)
            return 5;
    if (!(orc_alpha(d) > 0.0) || !(orc_raw_scale(d) > 0.0))
        return 6;
    free(p); free(pd); free(val); free(keys); free(rank); free(bary); free(xel); free(E); free(vert); free(ukeys);
    free(nbr); free(L); free(out); free(h); free(df); free(ex);
    return 0;
}

int main(void)
{
    const int dims[] = {1, 2, 3, 5, 8, 16};
    for (unsigned j = 0; j < sizeof(dims) / sizeof(dims[0]); ++j) {
        const int rc = run(dims[j], 300, 3);
        if (rc) {
            fprintf(stderr, "check %d failed for d=%d\n", rc, dims[j]);
            return rc;
        }
    }
    if (run(3, 1, 2) || run(2, 2, 1))  /* a lone point, two points */
        return 7;
    printf("oracle under sanitizers: ok\n");
    return 0;
}
