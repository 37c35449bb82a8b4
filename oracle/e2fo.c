/*
 * e2fo.c -- fp64 CPU oracle of the Wigner-6j convolution (E2Former,
 * arXiv 2501.19216).  TEST INFRASTRUCTURE ONLY: nothing in the product
 * library links, loads or calls this file; it is used by the tests, the
 * smoke check and the CPU-baseline leg of the benchmark.
 *
 * It is plain, slow and written to be checked against the paper by eye:
 *   - Wigner 3j symbol by Racah's closed form (App. C.1);
 *   - complex Clebsch-Gordan coefficients from the 3j symbol (Condon-Shortley);
 *   - real-basis CG (Def. 2.2) by the unitary complex->real change of basis
 *     of the real spherical harmonics of Def. 2.1 (sin for m<0, cos for m>0,
 *     no Condon-Shortley sign in the real functions);
 *   - real regular solid harmonics R^(l) as the stretched power
 *     R^(l) = [R^(l-1) (x) R^(1)]^(l), R^(1)(v) = (y, z, x) (Def. 2.1 and the
 *     projection identity of Thm. 3.2);
 *   - Wigner 6j symbol by Racah's single-sum formula (App. C.2; the four-3j
 *     sum printed there has inconsistent m indices and is not used);
 *   - the recoupling weights X of Def. 2.3 as an overlap of coupling trees;
 *   - the radius graph: every ordered pair i != j of one graph with
 *     |r_i - r_j| < cutoff, evaluated exactly on the 2^-16 A grid;
 *   - the attention weights of the edges (Alg. 1 input alpha; E2Attention
 *     of App. E): scalar q.k logits plus a radial basis, softmax over each
 *     receiver's neighbours, cosine envelope;
 *   - the k-nearest-neighbour graph of the paper's sparse scaling workloads
 *     (Sec. 4.1, Fig. 2): per atom the k others of its graph that come first
 *     in (squared grid distance, index) order;
 *   - the layer by its definition (Def. 3.1 with attention weights, App. D.2
 *     setup): y_i = sum_j alpha_ij sum_{a,f} w_afo [h_j^(a) (x) R^(f)(r_i - r_j)]^(o);
 *   - the layer by the node factorisation of Thm. 3.3 / Alg. 1 (for the
 *     equality check of the two forms only);
 *   - the per-irrep linear channel mix of App. F;
 *   - the attention-weighted aggregation of stored node tensors, Alg. 1's
 *     einsum "ijh,jhds->ihds" summed over the graph's edges;
 *   - the vector-Jacobian products of the layer with respect to the features
 *     and the attention weights, by the definition (the layer is linear in
 *     both).
 *
 * Accumulation is in double; the row loops are parallel (OpenMP) over
 * receivers, each row summed in ascending sender order.
 */
#include <complex.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define MAXL 12 /* largest degree any table here is asked for */

static int iabs_(int x) { return x < 0 ? -x : x; }
static int imin_(int a, int b) { return a < b ? a : b; }
static int imax_(int a, int b) { return a > b ? a : b; }
static double sgn_pow(int k) { return (k % 2 == 0) ? 1.0 : -1.0; } /* (-1)^k, k may be < 0 */

static long double fact(int n) {
    long double r = 1.0L;
    for (int k = 2; k <= n; ++k) r *= (long double)k;
    return r;
}

static int triangle(int a, int b, int c) { return c >= iabs_(a - b) && c <= a + b; }

/* ---------- Wigner 3j: Racah's closed form (App. C.1) ---------- */
double e2fo_wigner3j(int j1, int j2, int j3, int m1, int m2, int m3) {
    if (m1 + m2 + m3 != 0) return 0.0;
    if (!triangle(j1, j2, j3)) return 0.0;
    if (iabs_(m1) > j1 || iabs_(m2) > j2 || iabs_(m3) > j3) return 0.0;
    long double tri = fact(j1 + j2 - j3) * fact(j1 - j2 + j3) * fact(-j1 + j2 + j3) / fact(j1 + j2 + j3 + 1);
    long double mm = fact(j1 + m1) * fact(j1 - m1) * fact(j2 + m2) * fact(j2 - m2) * fact(j3 + m3) * fact(j3 - m3);
    int zmin = imax_(0, imax_(j2 - j3 - m1, j1 - j3 + m2));
    int zmax = imin_(j1 + j2 - j3, imin_(j1 - m1, j2 + m2));
    long double s = 0.0L;
    for (int z = zmin; z <= zmax; ++z) {
        long double den = fact(z) * fact(j1 + j2 - j3 - z) * fact(j1 - m1 - z) * fact(j2 + m2 - z) *
                          fact(j3 - j2 + m1 + z) * fact(j3 - j1 - m2 + z);
        s += ((z % 2) ? -1.0L : 1.0L) / den;
    }
    return (double)(sgn_pow(j1 - j2 - m3) * sqrtl(tri) * sqrtl(mm) * s);
}

/* Complex (Condon-Shortley) CG <l1 m1; l2 m2 | l3 m3> from the 3j symbol. */
double e2fo_cg_complex(int l1, int m1, int l2, int m2, int l3, int m3) {
    return sgn_pow(l1 - l2 + m3) * sqrt(2.0 * l3 + 1.0) * e2fo_wigner3j(l1, l2, l3, m1, m2, -m3);
}

/* Row m' (real function index) of the complex->real map S = U Y for degree l:
 * m'>0: S = ((-1)^m' Y^m' + Y^-m')/sqrt2 ; m'<0: S = i (Y^-|m'| - (-1)^|m'| Y^|m'|)/sqrt2. */
static double complex umat(int l, int mp, int m) {
    (void)l;
    const double r = 1.0 / sqrt(2.0);
    if (mp == 0) return (m == 0) ? 1.0 : 0.0;
    if (mp > 0) {
        if (m == mp) return sgn_pow(mp) * r;
        if (m == -mp) return r;
        return 0.0;
    }
    int mu = -mp;
    if (m == -mu) return I * r;
    if (m == mu) return -I * sgn_pow(mu) * r;
    return 0.0;
}

/* Real-basis CG for (l1,l2,l3): out[(m1+l1)][(m2+l2)][(m3+l3)] such that
 * [A (x) B]^(l3)_m3 = sum C[m1][m2][m3] A_m1 B_m2 for real-basis irreps A, B.
 * The transformed coefficients are purely real when l1+l2+l3 is even and
 * purely imaginary when odd; the real part (even) or the imaginary part
 * (odd) is returned.  Returns 0 on success, 1 if the discarded part was not
 * negligible (a convention error), 2 if the triangle rule fails. */
int e2fo_cg_real(int l1, int l2, int l3, double *out) {
    int n1 = 2 * l1 + 1, n2 = 2 * l2 + 1, n3 = 2 * l3 + 1;
    memset(out, 0, sizeof(double) * n1 * n2 * n3);
    if (!triangle(l1, l2, l3)) return 2;
    int odd = (l1 + l2 + l3) % 2;
    double worst = 0.0;
    for (int p1 = -l1; p1 <= l1; ++p1)
        for (int p2 = -l2; p2 <= l2; ++p2)
            for (int p3 = -l3; p3 <= l3; ++p3) {
                double complex acc = 0.0;
                for (int m1 = -l1; m1 <= l1; ++m1) {
                    double complex u1 = conj(umat(l1, p1, m1));
                    if (u1 == 0.0) continue;
                    for (int m2 = -l2; m2 <= l2; ++m2) {
                        double complex u2 = conj(umat(l2, p2, m2));
                        if (u2 == 0.0) continue;
                        int m3 = m1 + m2;
                        if (iabs_(m3) > l3) continue;
                        double complex u3 = umat(l3, p3, m3);
                        if (u3 == 0.0) continue;
                        acc += u3 * e2fo_cg_complex(l1, m1, l2, m2, l3, m3) * u1 * u2;
                    }
                }
                double keep = odd ? cimag(acc) : creal(acc);
                double drop = odd ? creal(acc) : cimag(acc);
                if (fabs(drop) > worst) worst = fabs(drop);
                out[((p1 + l1) * n2 + (p2 + l2)) * n3 + (p3 + l3)] = keep;
            }
    return worst > 1e-12 ? 1 : 0;
}

/* ---------- cached real CG tables for degrees <= MAXL ---------- */
static double *g_cg[MAXL + 1][MAXL + 1][2 * MAXL + 1];

static const double *cg(int l1, int l2, int l3) {
    if (!g_cg[l1][l2][l3]) {
        int n = (2 * l1 + 1) * (2 * l2 + 1) * (2 * l3 + 1);
        double *t = (double *)malloc(sizeof(double) * n);
        e2fo_cg_real(l1, l2, l3, t);
        g_cg[l1][l2][l3] = t;
    }
    return g_cg[l1][l2][l3];
}

/* Fill every table up to the given degrees before threads read them. */
static void warm_cg(int lmax_in, int lmax_out) {
    for (int a = 0; a <= lmax_in; ++a)
        for (int b = 0; b <= lmax_in; ++b)
            for (int c = iabs_(a - b); c <= imin_(a + b, lmax_out); ++c) cg(a, b, c);
}

/* CG coupling of two real irreps: out[m3] = sum C[m1][m2][m3] x[m1] y[m2]. */
static void couple(int l1, const double *x, int l2, const double *y, int l3, double *out) {
    const double *c = cg(l1, l2, l3);
    int n2 = 2 * l2 + 1, n3 = 2 * l3 + 1;
    for (int k = 0; k < n3; ++k) out[k] = 0.0;
    for (int i = 0; i < 2 * l1 + 1; ++i)
        for (int j = 0; j < n2; ++j) {
            double xy = x[i] * y[j];
            if (xy == 0.0) continue;
            for (int k = 0; k < n3; ++k) out[k] += c[(i * n2 + j) * n3 + k] * xy;
        }
}

/* ---------- real regular solid harmonics (Def. 2.1), stretched power ---------- */
void e2fo_solid_harmonics(int lmax, const double *v, double *out) {
    out[0] = 1.0;
    if (lmax < 1) return;
    double r1[3] = {v[1], v[2], v[0]}; /* m = -1, 0, +1  <->  y, z, x */
    out[1] = r1[0]; out[2] = r1[1]; out[3] = r1[2];
    for (int l = 2; l <= lmax; ++l) couple(l - 1, out + (l - 1) * (l - 1), 1, r1, l, out + l * l);
}

/* Gradient of the solid harmonics: out[x*nk + k] = dR_k / dv_x (x, y, z),
 * by the product rule on the recursion R^(l) = [R^(l-1) (x) R^(1)]^(l), whose
 * coupling is bilinear: dR^(l) = [dR^(l-1) (x) R^(1)] + [R^(l-1) (x) dR^(1)]. */
void e2fo_solid_harmonics_grad(int lmax, const double *v, double *out) {
    int nk = (lmax + 1) * (lmax + 1);
    double R[49], t1[13], t2[13];
    e2fo_solid_harmonics(lmax, v, R);
    for (int x = 0; x < 3; ++x) {
        double *d = out + (size_t)x * nk;
        d[0] = 0.0;
        if (lmax < 1) continue;
        /* R^(1) = (v_y, v_z, v_x) */
        double d1[3] = {x == 1 ? 1.0 : 0.0, x == 2 ? 1.0 : 0.0, x == 0 ? 1.0 : 0.0};
        double r1[3] = {v[1], v[2], v[0]};
        d[1] = d1[0]; d[2] = d1[1]; d[3] = d1[2];
        for (int l = 2; l <= lmax; ++l) {
            couple(l - 1, d + (l - 1) * (l - 1), 1, r1, l, t1);
            couple(l - 1, R + (l - 1) * (l - 1), 1, d1, l, t2);
            for (int k = 0; k < 2 * l + 1; ++k) d[l * l + k] = t1[k] + t2[k];
        }
    }
}

/* ---------- Wigner 6j: Racah's single-sum formula ---------- */
static long double delta_tri(int a, int b, int c) {
    return sqrtl(fact(a + b - c) * fact(a - b + c) * fact(-a + b + c) / fact(a + b + c + 1));
}

double e2fo_wigner6j(int j1, int j2, int j3, int j4, int j5, int j6) {
    if (!triangle(j1, j2, j3) || !triangle(j1, j5, j6) || !triangle(j4, j2, j6) || !triangle(j4, j5, j3)) return 0.0;
    int a1 = j1 + j2 + j3, a2 = j1 + j5 + j6, a3 = j4 + j2 + j6, a4 = j4 + j5 + j3;
    int b1 = j1 + j2 + j4 + j5, b2 = j2 + j3 + j5 + j6, b3 = j3 + j1 + j6 + j4;
    int tmin = imax_(imax_(a1, a2), imax_(a3, a4));
    int tmax = imin_(b1, imin_(b2, b3));
    long double s = 0.0L;
    for (int t = tmin; t <= tmax; ++t) {
        long double den = fact(t - a1) * fact(t - a2) * fact(t - a3) * fact(t - a4) * fact(b1 - t) * fact(b2 - t) * fact(b3 - t);
        s += ((t % 2) ? -1.0L : 1.0L) * fact(t + 1) / den;
    }
    return (double)(delta_tri(j1, j2, j3) * delta_tri(j1, j5, j6) * delta_tri(j4, j2, j6) * delta_tri(j4, j5, j3) * s);
}

/* ---------- recoupling weights (Def. 2.3) as an overlap of coupling trees ----------
 * With A of degree a, B of degree b, C of degree u and f = b + u:
 *   [A (x) [C (x) B]^(f)]^(o) = sum_d X_d [C (x) [A (x) B]^(d)]^(o).
 * T2[al,be,ga,M]   = sum_ka C^{f ka}_{u ga, b be} C^{o M}_{a al, f ka}   (left tree)
 * T1_d[al,be,ga,M] = sum_de C^{d de}_{a al, b be} C^{o M}_{u ga, d de}   (right tree)
 * The right trees are orthogonal with squared norm 2o+1 (CG orthogonality,
 * App. C.1), so X_d = <T2, T1_d> / (2o+1). */
double e2fo_recoupling_x(int a, int b, int u, int o, int d) {
    int f = b + u;
    if (!triangle(a, f, o) || !triangle(a, b, d) || !triangle(u, d, o)) return 0.0;
    const double *cub_f = cg(u, b, f), *caf_o = cg(a, f, o), *cab_d = cg(a, b, d), *cud_o = cg(u, d, o);
    int na = 2 * a + 1, nb = 2 * b + 1, nu = 2 * u + 1, no = 2 * o + 1, nf = 2 * f + 1, nd = 2 * d + 1;
    double acc = 0.0;
    for (int al = 0; al < na; ++al)
        for (int be = 0; be < nb; ++be)
            for (int ga = 0; ga < nu; ++ga)
                for (int M = 0; M < no; ++M) {
                    double t2 = 0.0, t1 = 0.0;
                    for (int ka = 0; ka < nf; ++ka)
                        t2 += cub_f[(ga * nb + be) * nf + ka] * caf_o[(al * nf + ka) * no + M];
                    for (int de = 0; de < nd; ++de)
                        t1 += cab_d[(al * nb + be) * nd + de] * cud_o[(ga * nd + de) * no + M];
                    acc += t2 * t1;
                }
    return acc / (double)no;
}

/* ---------- radius graph (Alg. 1 step 2), exact on the 2^-16 grid ---------- */
static int in_range(const float *pos, int i, int j, double r2) {
    double d2 = 0.0;
    for (int k = 0; k < 3; ++k) {
        int64_t xi = llrint((double)pos[3 * i + k] * 65536.0), xj = llrint((double)pos[3 * j + k] * 65536.0);
        int64_t dx = xi - xj;
        d2 += (double)(dx * dx); /* integers below 2^53: exact */
    }
    return d2 < r2;
}

/* Every ordered pair (i, j), i != j, of one graph with |r_i - r_j| < cutoff.
 * Rows ascending in j.  Returns E; col_idx is written only if E <= cap. */
int64_t e2fo_neighbor_list(const float *pos, const int32_t *graph_id, int n, float cutoff, int64_t *row_ptr,
                           int32_t *col_idx, int64_t cap) {
    double rc = (double)cutoff * 65536.0;
    double r2 = rc * rc;
    int64_t *cnt = (int64_t *)calloc((size_t)n, sizeof(int64_t));
#pragma omp parallel for schedule(dynamic, 64)
    for (int i = 0; i < n; ++i) {
        int64_t c = 0;
        for (int j = 0; j < n; ++j)
            if (j != i && (!graph_id || graph_id[i] == graph_id[j]) && in_range(pos, i, j, r2)) ++c;
        cnt[i] = c;
    }
    row_ptr[0] = 0;
    for (int i = 0; i < n; ++i) row_ptr[i + 1] = row_ptr[i] + cnt[i];
    int64_t E = row_ptr[n];
    free(cnt);
    if (!col_idx || E > cap) return E;
#pragma omp parallel for schedule(dynamic, 64)
    for (int i = 0; i < n; ++i) {
        int64_t e = row_ptr[i];
        for (int j = 0; j < n; ++j)
            if (j != i && (!graph_id || graph_id[i] == graph_id[j]) && in_range(pos, i, j, r2)) col_idx[e++] = j;
    }
    return E;
}

/* ---------- k-nearest-neighbour graph (Sec. 4.1, Fig. 2 sparse graphs) ----------
 * Row i holds the min(k, n_g - 1) atoms j != i of i's graph (n_g atoms) that
 * come first in the order of (squared distance on the 2^-16 A grid, then
 * index j); the row lists them by ascending j.  Distances are exact unsigned
 * 64-bit integers (|x| < 16384 A keeps each of the three squares below 2^62).
 * Returns E; col_idx is written only if E <= cap. */
typedef struct {
    uint64_t d2;
    int32_t j;
} knn_cand;

static int cmp_i32_knn(const void *x, const void *y) {
    int32_t a = *(const int32_t *)x, b = *(const int32_t *)y;
    return (a > b) - (a < b);
}

static int cmp_cand(const void *x, const void *y) {
    const knn_cand *a = (const knn_cand *)x, *b = (const knn_cand *)y;
    if (a->d2 != b->d2) return (a->d2 > b->d2) - (a->d2 < b->d2);
    return (a->j > b->j) - (a->j < b->j);
}

static uint64_t grid_d2(const float *pos, int i, int j) {
    uint64_t d2 = 0;
    for (int k = 0; k < 3; ++k) {
        int64_t dx = llrint((double)pos[3 * i + k] * 65536.0) - llrint((double)pos[3 * j + k] * 65536.0);
        d2 += (uint64_t)(dx * dx);
    }
    return d2;
}

int64_t e2fo_knn_graph(const float *pos, const int32_t *graph_id, int n, int k, int64_t *row_ptr, int32_t *col_idx,
                       int64_t cap) {
    int64_t *cnt = (int64_t *)calloc((size_t)n, sizeof(int64_t));
#pragma omp parallel for schedule(dynamic, 64)
    for (int i = 0; i < n; ++i) {
        int64_t c = 0;
        for (int j = 0; j < n; ++j)
            if (j != i && (!graph_id || graph_id[i] == graph_id[j])) ++c;
        cnt[i] = c < k ? c : k;
    }
    row_ptr[0] = 0;
    for (int i = 0; i < n; ++i) row_ptr[i + 1] = row_ptr[i] + cnt[i];
    const int64_t E = row_ptr[n];
    free(cnt);
    if (!col_idx || E > cap) return E;
#pragma omp parallel
    {
        knn_cand *cand = (knn_cand *)malloc(sizeof(knn_cand) * (size_t)(n > 0 ? n : 1));
        int32_t *row = (int32_t *)malloc(sizeof(int32_t) * (size_t)(k > 0 ? k : 1));
#pragma omp for schedule(dynamic, 16)
        for (int i = 0; i < n; ++i) {
            int m = 0;
            for (int j = 0; j < n; ++j)
                if (j != i && (!graph_id || graph_id[i] == graph_id[j])) {
                    cand[m].d2 = grid_d2(pos, i, j);
                    cand[m].j = j;
                    ++m;
                }
            qsort(cand, (size_t)m, sizeof(knn_cand), cmp_cand);
            const int take = m < k ? m : k;
            for (int q = 0; q < take; ++q) row[q] = cand[q].j;
            qsort(row, (size_t)take, sizeof(int32_t), cmp_i32_knn);
            for (int q = 0; q < take; ++q) col_idx[row_ptr[i] + q] = row[q];
        }
        free(cand);
        free(row);
    }
    return E;
}

/* ---------- attention weights (Alg. 1 input alpha; App. E E2Attention) ----------
 * For the edge e = (i, j) of row i and head h:
 *   logit = sum_t q[i][h][t] k[j][h][t] + sum_r w[h][r] exp(-((d - mu_r)/sigma)^2),
 *   mu_r = r cutoff / (R - 1), sigma = cutoff / (R - 1), d = |r_i - r_j|,
 *   alpha[e][h] = env(d) exp(logit) / sum over the row of exp(logit),
 *   env(d) = (cos(pi d / cutoff) + 1) / 2 for d < cutoff, else 0. */
void e2fo_attention_weights(const float *pos, const float *q, const float *k, int n, int heads, int dk,
                            const float *rbf_w, int n_rbf, float cutoff, const int64_t *row_ptr,
                            const int32_t *col_idx, float *alpha) {
    const double rc = cutoff, sigma = rc / (double)(n_rbf - 1);
#pragma omp parallel for schedule(dynamic, 16)
    for (int i = 0; i < n; ++i) {
        const int64_t e0 = row_ptr[i], e1 = row_ptr[i + 1];
        if (e1 == e0) continue;
        double *lg = (double *)malloc(sizeof(double) * (size_t)(e1 - e0));
        double *env = (double *)malloc(sizeof(double) * (size_t)(e1 - e0));
        for (int h = 0; h < heads; ++h) {
            double mx = -INFINITY;
            for (int64_t e = e0; e < e1; ++e) {
                const int j = col_idx[e];
                double d2 = 0.0;
                for (int c = 0; c < 3; ++c) {
                    const double dx = (double)pos[3 * i + c] - (double)pos[3 * j + c];
                    d2 += dx * dx;
                }
                const double d = sqrt(d2);
                double l = 0.0;
                for (int t = 0; t < dk; ++t)
                    l += (double)q[((size_t)i * heads + h) * dk + t] * (double)k[((size_t)j * heads + h) * dk + t];
                for (int r = 0; r < n_rbf; ++r) {
                    const double z = (d - r * sigma) / sigma;
                    l += (double)rbf_w[h * n_rbf + r] * exp(-z * z);
                }
                lg[e - e0] = l;
                env[e - e0] = d < rc ? 0.5 * (cos(acos(-1.0) * d / rc) + 1.0) : 0.0;
                if (l > mx) mx = l;
            }
            double den = 0.0;
            for (int64_t e = e0; e < e1; ++e) den += exp(lg[e - e0] - mx);
            for (int64_t e = e0; e < e1; ++e)
                alpha[e * heads + h] = (float)(env[e - e0] * exp(lg[e - e0] - mx) / den);
        }
        free(lg);
        free(env);
    }
}

/* The same graph through a uniform cell grid (cell side >= cutoff), for
 * systems where the all-pairs loop is too slow.  Same predicate, same
 * ascending rows (each row is sorted after collection). */
static int cmp_i32(const void *x, const void *y) {
    int32_t a = *(const int32_t *)x, b = *(const int32_t *)y;
    return (a > b) - (a < b);
}

int64_t e2fo_neighbor_list_cells(const float *pos, const int32_t *graph_id, int n, float cutoff, int64_t *row_ptr,
                                 int32_t *col_idx, int64_t cap) {
    double rc = (double)cutoff * 65536.0, r2 = rc * rc;
    double lo[3] = {1e300, 1e300, 1e300}, hi[3] = {-1e300, -1e300, -1e300};
    for (int i = 0; i < n; ++i)
        for (int k = 0; k < 3; ++k) {
            double x = pos[3 * i + k];
            if (x < lo[k]) lo[k] = x;
            if (x > hi[k]) hi[k] = x;
        }
    int dim[3];
    for (int k = 0; k < 3; ++k) {
        dim[k] = (int)floor((hi[k] - lo[k]) / (double)cutoff) + 1;
        if (dim[k] < 1) dim[k] = 1;
    }
    int64_t ncell = (int64_t)dim[0] * dim[1] * dim[2];
    int *cell = (int *)malloc(sizeof(int) * (size_t)n);
    int64_t *start = (int64_t *)calloc((size_t)ncell + 1, sizeof(int64_t));
    int *members = (int *)malloc(sizeof(int) * (size_t)n);
    for (int i = 0; i < n; ++i) {
        int c[3];
        for (int k = 0; k < 3; ++k) {
            c[k] = (int)floor(((double)pos[3 * i + k] - lo[k]) / (double)cutoff);
            if (c[k] >= dim[k]) c[k] = dim[k] - 1;
        }
        cell[i] = (c[2] * dim[1] + c[1]) * dim[0] + c[0];
        start[cell[i] + 1]++;
    }
    for (int64_t c = 0; c < ncell; ++c) start[c + 1] += start[c];
    int64_t *fillp = (int64_t *)malloc(sizeof(int64_t) * (size_t)ncell);
    memcpy(fillp, start, sizeof(int64_t) * (size_t)ncell);
    for (int i = 0; i < n; ++i) members[fillp[cell[i]]++] = i;
    free(fillp);
    int64_t *cnt = (int64_t *)calloc((size_t)n, sizeof(int64_t));
    for (int pass = 0; pass < 2; ++pass) {
        if (pass == 1) {
            row_ptr[0] = 0;
            for (int i = 0; i < n; ++i) row_ptr[i + 1] = row_ptr[i] + cnt[i];
            if (!col_idx || row_ptr[n] > cap) break;
        }
#pragma omp parallel for schedule(dynamic, 64)
        for (int i = 0; i < n; ++i) {
            int ci = cell[i];
            int cx = ci % dim[0], cy = (ci / dim[0]) % dim[1], cz = ci / (dim[0] * dim[1]);
            int64_t c = 0, e = pass ? row_ptr[i] : 0;
            for (int dz = -1; dz <= 1; ++dz)
                for (int dy = -1; dy <= 1; ++dy)
                    for (int dx = -1; dx <= 1; ++dx) {
                        int x = cx + dx, y = cy + dy, z = cz + dz;
                        if (x < 0 || y < 0 || z < 0 || x >= dim[0] || y >= dim[1] || z >= dim[2]) continue;
                        int64_t cc = ((int64_t)z * dim[1] + y) * dim[0] + x;
                        for (int64_t q = start[cc]; q < start[cc + 1]; ++q) {
                            int j = members[q];
                            if (j != i && (!graph_id || graph_id[i] == graph_id[j]) && in_range(pos, i, j, r2)) {
                                if (pass) col_idx[e++] = j;
                                else ++c;
                            }
                        }
                    }
            if (pass) qsort(col_idx + row_ptr[i], (size_t)(row_ptr[i + 1] - row_ptr[i]), sizeof(int32_t), cmp_i32);
            else cnt[i] = c;
        }
    }
    int64_t E = row_ptr[n];
    free(cnt); free(cell); free(start); free(members);
    return E;
}

/* ---------- the layer by its definition (Def. 3.1 with attention weights) ----------
 * y_i^(o)[m,c] = sum_{j in N(i)} alpha[e(i,j), c/dh] sum_{a,f} w[a][f][o]
 *                  sum_{ma,mf} C^{o m}_{a ma, f mf} h_j^(a)[ma,c] R^(f)_mf(r_i - r_j)
 * Only the listed rows are evaluated (the definition is separable per row).
 * out: [n_rows][(L+1)^2][C]. */
int e2fo_conv_edge(int L, int C, int H, const float *pos, const float *feat, int n, const int64_t *row_ptr,
                   const int32_t *col_idx, const float *alpha, const double *path_w, const int32_t *rows, int n_rows,
                   int y_norm, double *out) {
    if (L < 0 || L > 6 || C < 1 || H < 1 || C % H) return 1;
    (void)n;
    int nk = (L + 1) * (L + 1), dh = C / H;
    warm_cg(L, L);
#pragma omp parallel for schedule(dynamic, 4)
    for (int r = 0; r < n_rows; ++r) {
        int i = rows[r];
        double *y = out + (size_t)r * nk * C;
        memset(y, 0, sizeof(double) * (size_t)nk * C);
        double R[49];
        for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            int j = col_idx[e];
            double v[3] = {(double)pos[3 * i] - pos[3 * j], (double)pos[3 * i + 1] - pos[3 * j + 1],
                           (double)pos[3 * i + 2] - pos[3 * j + 2]};
            e2fo_solid_harmonics(L, v, R);
            /* y_norm: Alg. 1's per-degree weights alpha / D^f, D = |r_i - r_j|
             * (filters Y^(f) of the unit vector); 0 for f > 0 at D = 0 */
            double dpow[7] = {1, 1, 1, 1, 1, 1, 1};
            if (y_norm) {
                double D = sqrt(v[0] * v[0] + v[1] * v[1] + v[2] * v[2]);
                for (int f = 1; f <= L; ++f) dpow[f] = D > 0.0 ? dpow[f - 1] / D : 0.0;
            }
            const float *hj = feat + (size_t)j * nk * C;
            for (int a = 0; a <= L; ++a)
                for (int f = 0; f <= L; ++f)
                    for (int o = iabs_(a - f); o <= imin_(a + f, L); ++o) {
                        double w = path_w[(a * (L + 1) + f) * (L + 1) + o] * dpow[f];
                        if (w == 0.0) continue;
                        const double *c3 = cg(a, f, o);
                        for (int ma = 0; ma < 2 * a + 1; ++ma)
                            for (int mf = 0; mf < 2 * f + 1; ++mf)
                                for (int m = 0; m < 2 * o + 1; ++m) {
                                    double cgv = c3[(ma * (2 * f + 1) + mf) * (2 * o + 1) + m];
                                    if (cgv == 0.0) continue;
                                    double k = w * cgv * R[f * f + mf];
                                    const float *hrow = hj + (size_t)(a * a + ma) * C;
                                    double *yrow = y + (size_t)(o * o + m) * C;
                                    for (int c = 0; c < C; ++c)
                                        yrow[c] += (double)alpha[e * H + c / dh] * k * (double)hrow[c];
                                }
                    }
        }
    }
    return 0;
}

/* ---------- vector-Jacobian products of the layer by its definition ----------
 * The layer is linear in h and in alpha.  For the output gradient gy
 * [n][(L+1)^2][C] (double):
 *   gfeat[j][a al][c] = sum over edges e = (i, j) of alpha[e][c/dh]
 *       sum_{f,o} w_afo sum_{mf,m} C^{o m}_{a al, f mf} R^(f)_mf(r_i - r_j) gy[i][o m][c],
 *   galpha[e][h] = sum_{c of head h} sum_{a,f,o} w_afo
 *       sum_{al,mf,m} C^{o m}_{a al, f mf} R^(f)_mf(r_i - r_j) h_j[a al][c] gy[i][o m][c].
 * Either output may be NULL.  galpha is computed for the edges of the
 * receivers arows (all if NULL), gfeat for the senders frows (all if NULL);
 * the rest stays zero.  gfeat is gathered per sender j over a transposed edge
 * list, so every sum runs in a fixed order. */
int e2fo_conv_edge_vjp(int L, int C, int H, const float *pos, const float *feat, const double *gy, int n,
                       const int64_t *row_ptr, const int32_t *col_idx, const float *alpha, const double *path_w,
                       const int32_t *arows, int n_arows, const int32_t *frows, int n_frows, double *gfeat,
                       double *galpha) {
    if (L < 0 || L > 6 || C < 1 || H < 1 || C % H) return 1;
    const int nk = (L + 1) * (L + 1), dh = C / H;
    const int64_t E = row_ptr[n];
    warm_cg(L, L);
    if (galpha) {
        memset(galpha, 0, sizeof(double) * (size_t)E * H);
        const int na = arows ? n_arows : n;
#pragma omp parallel for schedule(dynamic, 4)
        for (int r = 0; r < na; ++r) {
            const int i = arows ? arows[r] : r;
            double R[49];
            const double *gyi = gy + (size_t)i * nk * C;
            for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                const int j = col_idx[e];
                double v[3] = {(double)pos[3 * i] - pos[3 * j], (double)pos[3 * i + 1] - pos[3 * j + 1],
                               (double)pos[3 * i + 2] - pos[3 * j + 2]};
                e2fo_solid_harmonics(L, v, R);
                const float *hj = feat + (size_t)j * nk * C;
                for (int h = 0; h < H; ++h) galpha[e * H + h] = 0.0;
                for (int a = 0; a <= L; ++a)
                    for (int f = 0; f <= L; ++f)
                        for (int o = iabs_(a - f); o <= imin_(a + f, L); ++o) {
                            const double w = path_w[(a * (L + 1) + f) * (L + 1) + o];
                            if (w == 0.0) continue;
                            const double *c3 = cg(a, f, o);
                            for (int ma = 0; ma < 2 * a + 1; ++ma)
                                for (int mf = 0; mf < 2 * f + 1; ++mf)
                                    for (int m = 0; m < 2 * o + 1; ++m) {
                                        const double cgv = c3[(ma * (2 * f + 1) + mf) * (2 * o + 1) + m];
                                        if (cgv == 0.0) continue;
                                        const double k = w * cgv * R[f * f + mf];
                                        const float *hrow = hj + (size_t)(a * a + ma) * C;
                                        const double *grow = gyi + (size_t)(o * o + m) * C;
                                        for (int c = 0; c < C; ++c) galpha[e * H + c / dh] += k * hrow[c] * grow[c];
                                    }
                        }
            }
        }
    }
    if (gfeat) {
        /* transposed edge list: for every sender j the edges (i, j), by ascending e */
        int64_t *tptr = (int64_t *)calloc((size_t)n + 1, sizeof(int64_t));
        int64_t *tedge = (int64_t *)malloc(sizeof(int64_t) * (size_t)(E > 0 ? E : 1));
        int32_t *trecv = (int32_t *)malloc(sizeof(int32_t) * (size_t)(E > 0 ? E : 1));
        for (int64_t e = 0; e < E; ++e) tptr[col_idx[e] + 1]++;
        for (int j = 0; j < n; ++j) tptr[j + 1] += tptr[j];
        int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
        for (int j = 0; j < n; ++j) fill[j] = tptr[j];
        for (int i = 0; i < n; ++i)
            for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                const int64_t t = fill[col_idx[e]]++;
                tedge[t] = e;
                trecv[t] = i;
            }
        free(fill);
        memset(gfeat, 0, sizeof(double) * (size_t)n * nk * C);
        const int nf = frows ? n_frows : n;
#pragma omp parallel for schedule(dynamic, 4)
        for (int r = 0; r < nf; ++r) {
            const int j = frows ? frows[r] : r;
            double R[49];
            double *g = gfeat + (size_t)j * nk * C;
            for (int64_t t = tptr[j]; t < tptr[j + 1]; ++t) {
                const int64_t e = tedge[t];
                const int i = trecv[t];
                double v[3] = {(double)pos[3 * i] - pos[3 * j], (double)pos[3 * i + 1] - pos[3 * j + 1],
                               (double)pos[3 * i + 2] - pos[3 * j + 2]};
                e2fo_solid_harmonics(L, v, R);
                const double *gyi = gy + (size_t)i * nk * C;
                for (int a = 0; a <= L; ++a)
                    for (int f = 0; f <= L; ++f)
                        for (int o = iabs_(a - f); o <= imin_(a + f, L); ++o) {
                            const double w = path_w[(a * (L + 1) + f) * (L + 1) + o];
                            if (w == 0.0) continue;
                            const double *c3 = cg(a, f, o);
                            for (int ma = 0; ma < 2 * a + 1; ++ma)
                                for (int mf = 0; mf < 2 * f + 1; ++mf)
                                    for (int m = 0; m < 2 * o + 1; ++m) {
                                        const double cgv = c3[(ma * (2 * f + 1) + mf) * (2 * o + 1) + m];
                                        if (cgv == 0.0) continue;
                                        const double k = w * cgv * R[f * f + mf];
                                        double *grow = g + (size_t)(a * a + ma) * C;
                                        const double *yrow = gyi + (size_t)(o * o + m) * C;
                                        for (int c = 0; c < C; ++c)
                                            grow[c] += (double)alpha[e * H + c / dh] * k * yrow[c];
                                    }
                        }
            }
        }
        free(tptr);
        free(tedge);
        free(trecv);
    }
    return 0;
}

/* ---------- gradient with respect to the positions (forces) ----------
 * For the output gradient gy, the edge e = (i, j) with r = r_i - r_j carries
 *   g_e[x] = sum_{o,m,c} gy_i[o,m,c] alpha_{e,h(c)} sum_{a,f} w_afo
 *            sum_{ma,mf} C^{o m}_{a ma, f mf} h_j^(a)[ma,c] dR^(f)_mf(r)/dr_x,
 * which adds to atom i and subtracts from atom j (r depends on r_i - r_j
 * only).  out[r][x] for the atoms atoms[r] (all n in order if atoms is NULL):
 * the sum over the edges of which the atom is receiver, minus the sum over
 * those of which it is sender, each in ascending edge order. */
static void edge_force(int L, int C, int H, const float *pos, const float *feat, const double *gy, int i, int j,
                       int64_t e, const float *alpha, const double *path_w, double g[3]) {
    const int nk = (L + 1) * (L + 1), dh = C / H;
    double v[3] = {(double)pos[3 * i] - pos[3 * j], (double)pos[3 * i + 1] - pos[3 * j + 1],
                   (double)pos[3 * i + 2] - pos[3 * j + 2]};
    double dR[3 * 49];
    e2fo_solid_harmonics_grad(L, v, dR);
    const float *hj = feat + (size_t)j * nk * C;
    const double *gyi = gy + (size_t)i * nk * C;
    g[0] = g[1] = g[2] = 0.0;
    for (int a = 0; a <= L; ++a)
        for (int f = 0; f <= L; ++f)
            for (int o = iabs_(a - f); o <= imin_(a + f, L); ++o) {
                const double w = path_w[(a * (L + 1) + f) * (L + 1) + o];
                if (w == 0.0) continue;
                const double *c3 = cg(a, f, o);
                for (int ma = 0; ma < 2 * a + 1; ++ma)
                    for (int mf = 0; mf < 2 * f + 1; ++mf)
                        for (int m = 0; m < 2 * o + 1; ++m) {
                            const double cgv = c3[(ma * (2 * f + 1) + mf) * (2 * o + 1) + m];
                            if (cgv == 0.0) continue;
                            const float *hrow = hj + (size_t)(a * a + ma) * C;
                            const double *grow = gyi + (size_t)(o * o + m) * C;
                            double s = 0.0;
                            for (int c = 0; c < C; ++c) s += (double)alpha[e * H + c / dh] * hrow[c] * grow[c];
                            for (int x = 0; x < 3; ++x) g[x] += w * cgv * dR[x * nk + f * f + mf] * s;
                        }
            }
}

int e2fo_conv_edge_grad_pos(int L, int C, int H, const float *pos, const float *feat, const double *gy, int n,
                            const int64_t *row_ptr, const int32_t *col_idx, const float *alpha, const double *path_w,
                            const int32_t *atoms, int n_atoms, double *out) {
    if (L < 0 || L > 6 || C < 1 || H < 1 || C % H) return 1;
    const int64_t E = row_ptr[n];
    warm_cg(L, L);
    /* the edges of every sender, by ascending e */
    int64_t *tptr = (int64_t *)calloc((size_t)n + 1, sizeof(int64_t));
    int64_t *tedge = (int64_t *)malloc(sizeof(int64_t) * (size_t)(E > 0 ? E : 1));
    int32_t *trecv = (int32_t *)malloc(sizeof(int32_t) * (size_t)(E > 0 ? E : 1));
    int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!tptr || !tedge || !trecv || !fill) { free(tptr); free(tedge); free(trecv); free(fill); return 2; }
    for (int64_t e = 0; e < E; ++e) tptr[col_idx[e] + 1]++;
    for (int j = 0; j < n; ++j) tptr[j + 1] += tptr[j];
    for (int j = 0; j < n; ++j) fill[j] = tptr[j];
    for (int i = 0; i < n; ++i)
        for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            const int64_t t = fill[col_idx[e]]++;
            tedge[t] = e;
            trecv[t] = i;
        }
    free(fill);
    const int na = atoms ? n_atoms : n;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 2)
    for (int r = 0; r < na; ++r) {
        const int a = atoms ? atoms[r] : r;
        double *o3 = out + (size_t)r * 3;
        o3[0] = o3[1] = o3[2] = 0.0;
        if (a < 0 || a >= n) { bad = 1; continue; }
        double g[3];
        for (int64_t e = row_ptr[a]; e < row_ptr[a + 1]; ++e) {
            edge_force(L, C, H, pos, feat, gy, a, col_idx[e], e, alpha, path_w, g);
            for (int x = 0; x < 3; ++x) o3[x] += g[x];
        }
        for (int64_t t = tptr[a]; t < tptr[a + 1]; ++t) {
            edge_force(L, C, H, pos, feat, gy, trecv[t], a, tedge[t], alpha, path_w, g);
            for (int x = 0; x < 3; ++x) o3[x] -= g[x];
        }
    }
    free(tptr); free(tedge); free(trecv);
    return bad;
}

/* ---------- the layer by node factorisation (Thm. 3.3, Alg. 1) ----------
 * p = r - origin.  T_j^(a,b,d) = [h_j^(a) (x) R^(b)(p_j)]^(d) for every
 * triangle-valid (a,b,d);  S_i = sum_j alpha_ij T_j;
 * y_i^(o) = sum_{a,f} w_afo sum_{u=0}^{f} (-1)^(f-u) binom(f,u)
 *           sum_d X(a, f-u, u, o; d) [R^(u)(p_i) (x) S_i^(a,f-u,d)]^(o).
 * Dense scratch of size n * (L+1)^2 * (2L+1) * (4L+1) * C doubles: tiny
 * graphs only.  out: [n][(L+1)^2][C]. */
static double binom_(int n, int k) {
    double r = 1.0;
    for (int t = 1; t <= k; ++t) r = r * (n - k + t) / t;
    return r;
}

/* i-side recoupling of one node (blue box of Thm. 3.3; Wigner6jTP of Alg. 1):
 * y^(o) = sum_{a,f} w_afo sum_{u<=f} (-1)^(f-u) binom(f,u) sum_d X(a,f-u,u,o;d)
 *         [R^(u)(p_i) (x) S^(a,f-u,d)]^(o),
 * with S indexed [a][b][d][delta][c] (d < 2L+1, delta < 4L+1) and Ru = R(p_i). */
static void iside(int L, int C, const double *Ru0, const double *S, const double *path_w, double *y) {
    int nk = (L + 1) * (L + 1), L1 = L + 1, DM = 4 * L + 1;
    memset(y, 0, sizeof(double) * (size_t)nk * C);
    for (int a = 0; a <= L; ++a)
        for (int f = 0; f <= L; ++f)
            for (int o = iabs_(a - f); o <= imin_(a + f, L); ++o) {
                double w = path_w[(a * L1 + f) * L1 + o];
                if (w == 0.0) continue;
                for (int u = 0; u <= f; ++u) {
                    int b = f - u;
                    double coef = w * sgn_pow(f - u) * binom_(f, u);
                    for (int d = iabs_(a - b); d <= a + b; ++d) {
                        double x = e2fo_recoupling_x(a, b, u, o, d);
                        if (x == 0.0) continue;
                        const double *c3 = cg(u, d, o);
                        const double *Ru = Ru0 + u * u;
                        for (int ga = 0; ga < 2 * u + 1; ++ga)
                            for (int de = 0; de < 2 * d + 1; ++de)
                                for (int m = 0; m < 2 * o + 1; ++m) {
                                    double k = coef * x * c3[(ga * (2 * d + 1) + de) * (2 * o + 1) + m] * Ru[ga];
                                    if (k == 0.0) continue;
                                    double *yrow = y + (size_t)(o * o + m) * C;
                                    const double *srow = S + ((((size_t)a * L1 + b) * (2 * L + 1) + d) * DM + de) * C;
                                    for (int c = 0; c < C; ++c) yrow[c] += k * srow[c];
                                }
                    }
                }
            }
}

/* j-side product of one node (red box of Thm. 3.3): T^(a,b,d) = [h^(a) (x) R^(b)(p)]^(d)
 * added with weight s into T indexed like S above. */
static void jside_add(int L, int C, const double *Rb0, const float *h, double s, double *T) {
    int L1 = L + 1, DM = 4 * L + 1;
    for (int a = 0; a <= L; ++a)
        for (int b = 0; b <= L; ++b)
            for (int d = iabs_(a - b); d <= a + b; ++d) {
                const double *c3 = cg(a, b, d);
                const double *Rb = Rb0 + b * b;
                double *Tb = T + (((size_t)a * L1 + b) * (2 * L + 1) + d) * DM * C;
                for (int al = 0; al < 2 * a + 1; ++al)
                    for (int be = 0; be < 2 * b + 1; ++be)
                        for (int de = 0; de < 2 * d + 1; ++de) {
                            double k = s * c3[(al * (2 * b + 1) + be) * (2 * d + 1) + de] * Rb[be];
                            if (k == 0.0) continue;
                            for (int c = 0; c < C; ++c) Tb[(size_t)de * C + c] += k * (double)h[(size_t)(a * a + al) * C + c];
                        }
            }
}

int e2fo_conv_factorised(int L, int C, int H, const float *pos, const float *feat, int n, const int64_t *row_ptr,
                         const int32_t *col_idx, const float *alpha, const double *path_w, const double *origin,
                         double *out) {
    if (L < 0 || L > 6 || C < 1 || H < 1 || C % H) return 1;
    int nk = (L + 1) * (L + 1), dh = C / H, L1 = L + 1, DM = 4 * L + 1;
    warm_cg(2 * L, 2 * L);
    /* T index: [node][a][b][d][delta][c] with d in 0..2L, delta < 4L+1 */
    size_t per_node = (size_t)L1 * L1 * (2 * L + 1) * DM * C;
    double *T = (double *)calloc((size_t)n * per_node, sizeof(double));
    double *S = (double *)calloc((size_t)n * per_node, sizeof(double));
    double *Rp = (double *)malloc(sizeof(double) * (size_t)n * nk);
    if (!T || !S || !Rp) { free(T); free(S); free(Rp); return 2; }
    for (int i = 0; i < n; ++i) {
        double p[3] = {(double)pos[3 * i] - origin[0], (double)pos[3 * i + 1] - origin[1], (double)pos[3 * i + 2] - origin[2]};
        e2fo_solid_harmonics(L, p, Rp + (size_t)i * nk);
    }
    /* j-side tensor products (red box of Thm. 3.3; T_k of Alg. 1) */
    for (int j = 0; j < n; ++j) jside_add(L, C, Rp + (size_t)j * nk, feat + (size_t)j * nk * C, 1.0, T + (size_t)j * per_node);
    /* attention-weighted aggregation (einsum "ijh,jhds->ihds" of Alg. 1) */
    for (int i = 0; i < n; ++i)
        for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            int j = col_idx[e];
            for (size_t q = 0; q < per_node; ++q) {
                int c = (int)(q % (size_t)C);
                S[(size_t)i * per_node + q] += (double)alpha[e * H + c / dh] * T[(size_t)j * per_node + q];
            }
        }
    /* i-side recoupling (blue box of Thm. 3.3; Wigner6jTP of Alg. 1) */
    for (int i = 0; i < n; ++i)
        iside(L, C, Rp + (size_t)i * nk, S + (size_t)i * per_node, path_w, out + (size_t)i * nk * C);
    free(T); free(S); free(Rp);
    return 0;
}

/* ---------- uniform attention over the whole graph (App. G) ----------
 * alpha_ij = 1 for every pair i, j of the n atoms, j = i included.  With
 * p = r - origin, the moments M^(a,b,d) = sum_j [h_j^(a) (x) R^(b)(p_j)]^(d)
 * are summed once (O(n)) and every node contracts them with its own R^(u)(p_i)
 * exactly as in the factorised layer: y_i = iside(R(p_i), M).
 * out: [n_rows][(L+1)^2][C] for the nodes rows[] (all n if rows is NULL). */
int e2fo_conv_global(int L, int C, const float *pos, const float *feat, int n, const double *path_w,
                     const double *origin, const int32_t *rows, int n_rows, double *out) {
    if (L < 0 || L > 6 || C < 1) return 1;
    int nk = (L + 1) * (L + 1), L1 = L + 1, DM = 4 * L + 1;
    warm_cg(2 * L, 2 * L);
    size_t per_node = (size_t)L1 * L1 * (2 * L + 1) * DM * C;
    double *M = (double *)calloc(per_node, sizeof(double));
    double *Rp = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * nk);
    if (!M || !Rp) { free(M); free(Rp); return 2; }
    for (int i = 0; i < n; ++i) {
        double p[3] = {(double)pos[3 * i] - origin[0], (double)pos[3 * i + 1] - origin[1], (double)pos[3 * i + 2] - origin[2]};
        e2fo_solid_harmonics(L, p, Rp + (size_t)i * nk);
    }
    for (int j = 0; j < n; ++j) jside_add(L, C, Rp + (size_t)j * nk, feat + (size_t)j * nk * C, 1.0, M);
    /* out row r belongs to node rows[r] (every node in order if rows is NULL) */
    int nr = rows ? n_rows : n;
    for (int r = 0; r < nr; ++r) {
        int i = rows ? rows[r] : r;
        if (i < 0 || i >= n) { free(M); free(Rp); return 1; }
        iside(L, C, Rp + (size_t)i * nk, M, path_w, out + (size_t)r * nk * C);
    }
    free(M); free(Rp);
    return 0;
}

/* ---------- per-irrep linear self-mix (App. F) ----------
 * out[i][(o,m)][c'] = sum_c W[o][c'][c] y[i][(o,m)][c]. */
void e2fo_mix(int L, int C, int n_rows, const double *y, const float *W, double *out) {
    int nk = (L + 1) * (L + 1);
#pragma omp parallel for schedule(static)
    for (int r = 0; r < n_rows; ++r)
        for (int o = 0; o <= L; ++o)
            for (int m = 0; m < 2 * o + 1; ++m) {
                const double *yrow = y + ((size_t)r * nk + o * o + m) * C;
                double *orow = out + ((size_t)r * nk + o * o + m) * C;
                for (int cp = 0; cp < C; ++cp) {
                    double s = 0.0;
                    for (int c = 0; c < C; ++c) s += (double)W[((size_t)o * C + cp) * C + c] * yrow[c];
                    orow[cp] = s;
                }
            }
}

/* ---------- aggregation of stored node tensors (Alg. 1's einsum "ijh,jhds->ihds") ----------
 * For the receivers rows[r] (all n if rows is NULL):
 *     out[r][h][k] = sum over the edges e = (i, j) of row i of alpha[e][h] T[j][h][k],
 * T [n][H][W] (W = the values per head), alpha [E][H] or NULL (ones).
 * Returns 1 for a receiver or sender index outside [0, n), else 0. */
int e2fo_aggregate(int n, int H, int64_t W, const float *T, const int64_t *row_ptr, const int32_t *col_idx,
                   const float *alpha, const int32_t *rows, int n_rows, double *out) {
    int nr = rows ? n_rows : n;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 4) reduction(|:err)
    for (int r = 0; r < nr; ++r) {
        int i = rows ? rows[r] : r;
        if (i < 0 || i >= n) { err = 1; continue; }
        double *o = out + (size_t)r * H * W;
        for (int64_t q = 0; q < (int64_t)H * W; ++q) o[q] = 0.0;
        for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            int j = col_idx[e];
            if (j < 0 || j >= n) { err = 1; break; }
            for (int h = 0; h < H; ++h) {
                double a = alpha ? (double)alpha[e * H + h] : 1.0;
                const float *t = T + ((size_t)j * H + h) * W;
                double *oh = o + (size_t)h * W;
                for (int64_t q = 0; q < W; ++q) oh[q] += a * (double)t[q];
            }
        }
    }
    return err;
}
