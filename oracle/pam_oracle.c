/*
 * pam_oracle.c -- plain, slow CPU oracle of the permutohedral-lattice filter
 * used by the Permutohedral Attention Module (PAM; Joutard et al., 2019).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or constant generator
 * with the GPU library.
 *
 * What it computes (paper, Section 2 "Permutohedral Attention Module"):
 *   v'_i = sum_j K(f_i, f_j) v_j  (eq. 4-5), approximated in four steps,
 *   Embedding E, Splat S, Blur B, Slice Sl (eq. 6 and the Fig. 1 caption);
 *   the value gradient is the same filter with the blur directions taken in
 *   reverse order (eq. 7 and the notation paragraph after eq. 8); the
 *   embedding gradient combines the blurred lattices of v and of dL/dv'
 *   through the embedding matrix and the permutation found by E (eq. 8).
 *
 * The paper leaves the lattice algorithm itself to its reference [PL]; the
 * steps below follow the permutohedral lattice as the paper uses it, written
 * from its mathematics:
 *   * elevation x = E p onto the hyperplane sum(x) = 0 of R^{d+1}, with
 *     E = alpha * Q, Q an orthonormal basis of that hyperplane, and
 *     alpha = (d+1) sqrt(2/3), which makes the whole filter a unit-variance
 *     Gaussian in input units;
 *   * the enclosing simplex: nearest remainder-0 point (all coordinates
 *     multiples of d+1, sum 0), ranks of the residuals, barycentric weights;
 *   * splat with those weights, d+1 blur passes of taps [1 2 1] along the
 *     lattice directions u_j = (d+1) e_j - 1 over the touched vertices only
 *     (absent neighbours read as 0), slice with the same weights.
 *
 * Precision.  Every integer decision (the remainder-0 point, the ranks and
 * therefore the vertex keys) is taken in fp32 with a fixed operation order:
 * the elevation is an fmaf chain over the nonzero entries of E in ascending
 * input index, rounding is rintf(x * fp32(1/(d+1))) (ties to even), and the
 * residuals are single fp32 subtractions.  All values (barycentric weights,
 * lattice contents, outputs, gradients) are computed in fp64 from a
 * double-precision elevation of the same fp32 inputs, using the integer
 * decisions above.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared (no fast-math).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_MAX_D 16

/* ---------------------------------------------------------------------- */
/* Constants                                                              */
/* ---------------------------------------------------------------------- */

/* Scale of the elevation: alpha = (d+1) sqrt(2/3).  With it the d+1 blur
 * passes plus splat/slice give unit variance per input dimension. */
double orc_alpha(int d) { return (double)(d + 1) * sqrt(2.0 / 3.0); }

/* The position embedding matrix E of eq. (8) (the notation paragraph calls
 * it the position embedding matrix), (d+1) x d row-major:
 *   E[i][j] = alpha / sqrt((j+1)(j+2))          if i <= j
 *           = -alpha (j+1) / sqrt((j+1)(j+2))   if i == j+1
 *           = 0                                 otherwise.
 * Its columns are orthogonal, each of norm alpha, and each sums to zero. */
void orc_embedding_matrix(int d, double *E)
{
    double a = orc_alpha(d);
    for (int i = 0; i <= d; ++i) {
        for (int j = 0; j < d; ++j) {
            double nrm = sqrt((double)(j + 1) * (double)(j + 2));
            double q = 0.0;
            if (i <= j)
                q = 1.0 / nrm;
            else if (i == j + 1)
                q = -(double)(j + 1) / nrm;
            E[i * d + j] = a * q;
        }
    }
}

/* Scale of the raw (unnormalised) filter: s_d = 1 / G_d where
 * G_d = 4^{d+1} * covol / (2 pi)^{d/2} is the mass of the lattice kernel
 * (each of the d+1 [1 2 1] passes multiplies mass by 4; slicing integrates
 * to the lattice covolume (3/2)^{d/2}/sqrt(d+1) in input units) divided by
 * the mass of exp(-|x|^2/2).  With it the raw output approximates
 * sum_j exp(-|f_i - f_j|^2 / 2) v_j in scale as well as in shape. */
double orc_raw_scale(int d)
{
    double G = pow(4.0, d + 1) * pow(3.0 / (4.0 * M_PI), 0.5 * d) / sqrt((double)(d + 1));
    return 1.0 / G;
}

/* ---------------------------------------------------------------------- */
/* Embedding: enclosing simplex of every point (operator E of eq. 6)       */
/* ---------------------------------------------------------------------- */

/* For each of the n points p_i (n x d fp32):
 *   keys  [n][d+1][d] int32: the d stored coordinates of the d+1 simplex
 *         vertices (coordinate d is minus the sum of the others); vertex k
 *         has every coordinate congruent to k modulo d+1;
 *   bary  [n][d+1] fp64: barycentric weight of vertex k;
 *   rank  [n][d+1] int32: rank of each elevated coordinate after the
 *         remainder-0 fix-up (the permutation sigma_i of eq. 8);
 *   xelev [n][d+1] fp64 (may be NULL): the fp64 elevation.
 * Returns 0, or -1 if a point is not finite or lies so far out
 * (|x| > 2^24) that its key would not be representable. */
int orc_simplex(const float *p, int64_t n, int d, int32_t *keys, double *bary,
                int32_t *rank, double *xelev)
{
    if (d < 1 || d > ORC_MAX_D)
        return -1;
    const int d1 = d + 1;
    double E[(ORC_MAX_D + 1) * ORC_MAX_D];
    float E32[(ORC_MAX_D + 1) * ORC_MAX_D];
    orc_embedding_matrix(d, E);
    for (int t = 0; t < d1 * d; ++t)
        E32[t] = (float)E[t];
    const float inv32 = (float)(1.0 / (double)d1);

    for (int64_t i = 0; i < n; ++i) {
        const float *pi = p + i * d;
        float x32[ORC_MAX_D + 1], delta[ORC_MAX_D + 1];
        double x64[ORC_MAX_D + 1], y[ORC_MAX_D + 2], b[ORC_MAX_D + 2];
        int r[ORC_MAX_D + 1], rk[ORC_MAX_D + 1];

        /* 1. elevate: fp32 fma chain (decisions) and fp64 sum (values) */
        for (int c = 0; c < d1; ++c) {
            float acc = 0.0f;
            double acc64 = 0.0;
            for (int j = (c > 0 ? c - 1 : 0); j < d; ++j) {
                acc = fmaf(E32[c * d + j], pi[j], acc);
                acc64 += E[c * d + j] * (double)pi[j];
            }
            if (!isfinite(acc) || fabsf(acc) > 16777216.0f)
                return -1;
            x32[c] = acc;
            x64[c] = acc64;
        }

        /* 2. nearest remainder-0 point, coordinate by coordinate */
        int s = 0;
        for (int c = 0; c < d1; ++c) {
            int q = (int)rintf(x32[c] * inv32);
            r[c] = q * d1;
            s += q;
            delta[c] = x32[c] - (float)r[c];
        }

        /* 3. rank the residuals: rank 0 is the largest; equal residuals
         *    give the lower coordinate index the lower rank */
        for (int c = 0; c < d1; ++c) {
            int k = 0;
            for (int c2 = 0; c2 < d1; ++c2) {
                if (delta[c2] > delta[c])
                    ++k;
                else if (delta[c2] == delta[c] && c2 < c)
                    ++k;
            }
            rk[c] = k;
        }

        /* 4. restore sum(r) = 0: move the s coordinates with the smallest
         *    residual down by d+1 (s > 0), or the -s coordinates with the
         *    largest residual up by d+1 (s < 0); the moved coordinates
         *    become the extreme ones and the ranks rotate by s. */
        if (s > 0) {
            for (int c = 0; c < d1; ++c) {
                if (rk[c] >= d1 - s) {
                    r[c] -= d1;
                    rk[c] += s - d1;
                } else {
                    rk[c] += s;
                }
            }
        } else if (s < 0) {
            for (int c = 0; c < d1; ++c) {
                if (rk[c] < -s) {
                    r[c] += d1;
                    rk[c] += s + d1;
                } else {
                    rk[c] += s;
                }
            }
        }

        /* 5. barycentric weights (fp64): with y = (x - r)/(d+1), vertex k
         *    gets y of the coordinate ranked d-k minus y of the coordinate
         *    ranked d+1-k, and vertex 0 additionally 1 - y(rank 0). */
        for (int k = 0; k < d1 + 1; ++k)
            b[k] = 0.0;
        for (int c = 0; c < d1; ++c) {
            y[c] = (x64[c] - (double)r[c]) / (double)d1;
            b[d - rk[c]] += y[c];
            b[d1 - rk[c]] -= y[c];
        }
        b[0] += 1.0 + b[d1];

        /* 6. vertices: vertex k is r + k on every coordinate, minus d+1 on
         *    the coordinates whose rank exceeds d-k */
        for (int k = 0; k < d1; ++k) {
            for (int c = 0; c < d; ++c)
                keys[(i * d1 + k) * d + c] = r[c] + k - (rk[c] > d - k ? d1 : 0);
            bary[i * d1 + k] = b[k];
        }
        for (int c = 0; c < d1; ++c) {
            rank[i * d1 + c] = rk[c];
            if (xelev)
                xelev[i * d1 + c] = x64[c];
        }
    }
    return 0;
}

/* ---------------------------------------------------------------------- */
/* The sparse lattice: unique vertex set, ids, neighbours                  */
/* ---------------------------------------------------------------------- */

static int g_cmp_d;            /* key length for the qsort comparator */
static const int32_t *g_cmp_keys;

static int cmp_key_index(const void *a, const void *b)
{
    int64_t ia = *(const int64_t *)a, ib = *(const int64_t *)b;
    const int32_t *ka = g_cmp_keys + ia * g_cmp_d;
    const int32_t *kb = g_cmp_keys + ib * g_cmp_d;
    for (int c = 0; c < g_cmp_d; ++c) {
        if (ka[c] != kb[c])
            return ka[c] < kb[c] ? -1 : 1;
    }
    return (ia > ib) - (ia < ib);
}

/* Vertex set V = all distinct keys among the n(d+1) simplex vertices.
 * Vertex ids are positions in lexicographic key order.
 *   keys  [n(d+1)][d]  input;
 *   vert  [n(d+1)]     output: id of every (point, vertex) pair;
 *   ukeys [n(d+1)][d]  output: the M distinct keys, sorted (capacity n(d+1)).
 * Returns M (or -1 on allocation failure). */
int64_t orc_lattice(int64_t n, int d, const int32_t *keys, int32_t *vert, int32_t *ukeys)
{
    const int64_t total = n * (int64_t)(d + 1);
    if (total == 0)
        return 0;
    int64_t *idx = (int64_t *)malloc((size_t)total * sizeof(int64_t));
    if (!idx)
        return -1;
    for (int64_t t = 0; t < total; ++t)
        idx[t] = t;
    g_cmp_d = d;
    g_cmp_keys = keys;
    qsort(idx, (size_t)total, sizeof(int64_t), cmp_key_index);
    int64_t M = 0;
    for (int64_t t = 0; t < total; ++t) {
        const int32_t *k = keys + idx[t] * d;
        if (M == 0 || memcmp(k, ukeys + (M - 1) * d, (size_t)d * sizeof(int32_t)) != 0) {
            memcpy(ukeys + M * d, k, (size_t)d * sizeof(int32_t));
            ++M;
        }
        vert[idx[t]] = (int32_t)(M - 1);
    }
    free(idx);
    return M;
}

static int64_t find_key(int64_t M, int d, const int32_t *ukeys, const int32_t *key)
{
    int64_t lo = 0, hi = M;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        const int32_t *k = ukeys + mid * d;
        int c = 0;
        while (c < d && k[c] == key[c])
            ++c;
        if (c == d)
            return mid;
        if (k[c] < key[c])
            lo = mid + 1;
        else
            hi = mid;
    }
    return -1;
}

/* Neighbours along the d+1 lattice directions.  On the d stored
 * coordinates, u_j is +d at coordinate j and -1 elsewhere (j < d); u_d is -1
 * everywhere.  nbr[m][j][0] = id(key_m - u_j), nbr[m][j][1] = id(key_m + u_j),
 * -1 where that vertex is not in V. */
void orc_neighbours(int64_t M, int d, const int32_t *ukeys, int32_t *nbr)
{
    int32_t key[ORC_MAX_D];
    for (int64_t m = 0; m < M; ++m) {
        for (int j = 0; j <= d; ++j) {
            for (int sgn = 0; sgn < 2; ++sgn) {
                int step = sgn ? 1 : -1;
                for (int c = 0; c < d; ++c) {
                    int u = (c == j) ? d : -1;
                    key[c] = ukeys[m * d + c] + step * u;
                }
                nbr[(m * (d + 1) + j) * 2 + sgn] = (int32_t)find_key(M, d, ukeys, key);
            }
        }
    }
}

/* ---------------------------------------------------------------------- */
/* Splat, Blur, Slice (operators S, B and Sl of eq. 6-7)                   */
/* ---------------------------------------------------------------------- */

/* L[m] = sum over (i,k) with vert[i][k] = m of bary[i][k] * val[i]. */
void orc_splat(int64_t n, int d, int C, const int32_t *vert, const double *bary,
               const double *val, int64_t M, double *L)
{
    memset(L, 0, (size_t)(M * C) * sizeof(double));
    for (int64_t i = 0; i < n; ++i)
        for (int k = 0; k <= d; ++k) {
            double w = bary[i * (d + 1) + k];
            double *row = L + (int64_t)vert[i * (d + 1) + k] * C;
            for (int c = 0; c < C; ++c)
                row[c] += w * val[i * C + c];
        }
}

/* d+1 passes L <- L[n-] + 2 L + L[n+] along directions 0..d (reverse = 0)
 * or d..0 (reverse = 1); each pass reads only the previous pass's values;
 * absent neighbours contribute 0.  Returns -1 on allocation failure. */
int orc_blur(int64_t M, int d, int C, const int32_t *nbr, int reverse, double *L)
{
    double *tmp = (double *)malloc((size_t)(M * C > 0 ? M * C : 1) * sizeof(double));
    if (!tmp)
        return -1;
    for (int t = 0; t <= d; ++t) {
        int j = reverse ? d - t : t;
        for (int64_t m = 0; m < M; ++m) {
            int32_t lo = nbr[(m * (d + 1) + j) * 2 + 0];
            int32_t hi = nbr[(m * (d + 1) + j) * 2 + 1];
            for (int c = 0; c < C; ++c) {
                double acc = 2.0 * L[m * C + c];
                if (lo >= 0)
                    acc += L[(int64_t)lo * C + c];
                if (hi >= 0)
                    acc += L[(int64_t)hi * C + c];
                tmp[m * C + c] = acc;
            }
        }
        memcpy(L, tmp, (size_t)(M * C) * sizeof(double));
    }
    free(tmp);
    return 0;
}

/* out[i] = sum_k bary[i][k] * L[vert[i][k]]. */
void orc_slice(int64_t n, int d, int C, const int32_t *vert, const double *bary,
               const double *L, double *out)
{
    for (int64_t i = 0; i < n; ++i) {
        double *o = out + i * C;
        for (int c = 0; c < C; ++c)
            o[c] = 0.0;
        for (int k = 0; k <= d; ++k) {
            double w = bary[i * (d + 1) + k];
            const double *row = L + (int64_t)vert[i * (d + 1) + k] * C;
            for (int c = 0; c < C; ++c)
                o[c] += w * row[c];
        }
    }
}

/* h[i][k] = <a_i, L[vert[i][k]]> (C-dim dot products). */
void orc_vertex_dots(int64_t n, int d, int C, const int32_t *vert, const double *a,
                     const double *L, double *h)
{
    for (int64_t i = 0; i < n; ++i)
        for (int k = 0; k <= d; ++k) {
            const double *row = L + (int64_t)vert[i * (d + 1) + k] * C;
            double acc = 0.0;
            for (int c = 0; c < C; ++c)
                acc += a[i * C + c] * row[c];
            h[i * (d + 1) + k] = acc;
        }
}

/* Embedding gradient (eq. 8).  h[i][k] = dL/d(bary[i][k]).  Inside the
 * simplex of point i, d bary_k / d x_c = ([k = d - rank_c]
 * - [k = (d + 1 - rank_c) mod (d+1)]) / (d+1), so
 *   gx_c = (h[d - rank_c] - h[(d + 1 - rank_c) mod (d+1)]) / (d+1),
 * and with x = E p the gradient is df_i = E^T gx. */
void orc_embed_grad(int64_t n, int d, const int32_t *rank, const double *h, double *df)
{
    double E[(ORC_MAX_D + 1) * ORC_MAX_D];
    orc_embedding_matrix(d, E);
    const int d1 = d + 1;
    for (int64_t i = 0; i < n; ++i) {
        double gx[ORC_MAX_D + 1];
        for (int c = 0; c < d1; ++c) {
            int rc = rank[i * d1 + c];
            int k_plus = d - rc;
            int k_minus = (d1 - rc) % d1;
            gx[c] = (h[i * d1 + k_plus] - h[i * d1 + k_minus]) / (double)d1;
        }
        for (int j = 0; j < d; ++j) {
            double acc = 0.0;
            for (int c = 0; c < d1; ++c)
                acc += E[c * d + j] * gx[c];
            df[i * d + j] = acc;
        }
    }
}

/* ---------------------------------------------------------------------- */
/* Exact Gaussian filter (eq. 4 with the kernel read as exp(-|.|^2/2))     */
/* ---------------------------------------------------------------------- */

/* out_i = sum_j exp(-|p_i - p_j|^2 / 2) v_j, O(n^2); small n only. */
void orc_gauss_bruteforce(int64_t n, int d, int C, const double *p, const double *v,
                          double *out)
{
    for (int64_t i = 0; i < n; ++i) {
        double *o = out + i * C;
        for (int c = 0; c < C; ++c)
            o[c] = 0.0;
        for (int64_t j = 0; j < n; ++j) {
            double r2 = 0.0;
            for (int t = 0; t < d; ++t) {
                double diff = p[i * d + t] - p[j * d + t];
                r2 += diff * diff;
            }
            double w = exp(-0.5 * r2);
            for (int c = 0; c < C; ++c)
                o[c] += w * v[j * C + c];
        }
    }
}
