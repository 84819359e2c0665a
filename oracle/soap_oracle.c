/*
 * SOAP oracle: a plain, slow CPU implementation of the descriptor and its
 * analytic Jacobian, written from the paper's equations.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, the smoke check and the bench's
 * CPU-baseline leg load this library.  It shares no code with the HIP path.
 *
 * Precision: float64 throughout, long double (x87, 64-bit mantissa) for the
 * Loewdin-weighted radial sums and the monomial evaluation of the harmonics,
 * where cancellation would otherwise cost digits, and __float128 for the
 * Laplace form's monomial sums, which cancel the most.  Compiled with
 * -ffp-contract=off so the cutoff test below is evaluated exactly as written.
 *
 * Paper passages followed (Sec. = section of the paper):
 *  - density, projection, power spectrum, product rule: Sec. 2.1,
 *    Eqs. (density), (projection), (powerspectrum), (powerspectrum-derivative);
 *    translational invariance for the center's own block, end of Sec. 2.1.
 *  - GTO coefficients and gradient: Sec. 2.2, Eqs. (gto-coefficients),
 *    (gto-derivative) (the ladder terms are the gradient of the solid
 *    harmonic r^l Y_lm; here that gradient is taken directly from the
 *    polynomial form of r^l Y_lm).
 *  - polynomial coefficients: Sec. 2.3, Eqs. (poly-coefficients-exact),
 *    (poly-radial-integral), with the radial integral done by the fixed
 *    Gauss-Legendre rule of Sec. 3.1; gradient by the chain rule
 *    Eq. (poly-cartesian-derivative) with df/dr from differentiating the same
 *    quadrature under the integral sign (i_l' = i_{l+1} + (l/x) i_l).
 *  - polynomial coefficients, Laplace form: Sec. 2.3, Eqs. (poly-laplace),
 *    (poly-coefficients), (poly-radial-derivative), the same chain rule.
 *  - neighbour set and the on-site term: Sec. 3.1 (zero-length edges are
 *    dropped and the position-independent l = 0 self term is added).
 *  - feature order: Sec. 3.1, species pair (mu <= nu), then n, then n'
 *    (n' >= n on the diagonal), then l innermost.
 */
#include <math.h>
#include <omp.h>
#include <quadmath.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef long double ld;
typedef __float128 qd;

typedef struct {
    int32_t S, n, lmax, rbf; /* rbf: 0 = GTO, 1 = polynomial (quadrature), 2 = polynomial (Laplace) */
    double rc, sigma;
    /* GTO: alpha[l][k], beta[l][n][k] */
    const double *alpha_hi, *alpha_lo, *beta_hi, *beta_lo;
    /* polynomial: G[n][q] = w_q r_q^2 g_n(r_q), nodes r_q */
    int32_t Q;
    const double *G_hi, *G_lo, *rq_hi, *rq_lo;
    /* real solid harmonics up to sh_lmax as monomials */
    int32_t sh_lmax;
    const int32_t *sh_ptr, *sh_exp;
    const double *sh_c_hi, *sh_c_lo;
    /* polynomial, Laplace variant: W_nk / N_k (rbf 2; G and rq still give the on-site term) */
    const double *wn_hi, *wn_lo;
} oracle_params;

#define LD(h, l) ((ld)(h) + (ld)(l))

/* ---------------------------------------------------------------- neighbours
 * j is a neighbour of center i iff j != i and |r_j - r_i|^2 < r_cut^2, with
 * the squared distance summed as ((dx*dx + dy*dy) + dz*dz) in float64. */
static int is_neighbour(const double *pi, const double *pj, double rc2) {
    double dx = pj[0] - pi[0], dy = pj[1] - pi[1], dz = pj[2] - pi[2];
    double d2 = dx * dx + dy * dy;
    d2 = d2 + dz * dz;
    return d2 < rc2;
}

/* brute force over all atoms; cols sorted ascending by construction */
int64_t oracle_neighbors(int64_t n_atoms, const double *pos, double rc, const int64_t *centers, int64_t nc,
                         int64_t *row_ptr, int32_t *cols, int64_t cap) {
    double rc2 = rc * rc;
    int64_t e = 0;
    row_ptr[0] = 0;
    for (int64_t c = 0; c < nc; ++c) {
        int64_t i = centers ? centers[c] : c;
        for (int64_t j = 0; j < n_atoms; ++j) {
            if (j == i) continue;
            if (is_neighbour(pos + 3 * i, pos + 3 * j, rc2)) {
                if (cols && e < cap) cols[e] = (int32_t)j;
                ++e;
            }
        }
        row_ptr[c + 1] = e;
    }
    return e;
}

/* Periodic images, brute force.  cell[9] holds the lattice vectors a, b, c as
 * rows; pbc[3] marks the periodic directions; nimg[3] bounds the image index
 * per direction (0 where not periodic).  An edge (i -> j, n) exists for every
 * atom j and integer image n with |n_k| <= nimg[k], (j, n) != (i, 0), whose
 * image r_j + s(n), s(n) = ((n_a a + n_b b) + n_c c) evaluated in float64 in
 * that order (and rounded to float32 when f32 != 0, the float32-mode reading),
 * passes the cutoff test against r_i.  Rows: ascending j, then n in
 * lexicographic (n_a, n_b, n_c) order.  Writes cols[e] = j and img[e][3] = n
 * when cols is not NULL; returns the edge count. */
static double image_coord(const double *pos, const double *cell, int64_t j, const int *n, int d, int f32) {
    double s = (double)n[0] * cell[d];
    s = s + (double)n[1] * cell[3 + d];
    s = s + (double)n[2] * cell[6 + d];
    double v = pos[3 * j + d] + s;
    return f32 ? (double)(float)v : v;
}

int64_t oracle_neighbors_periodic(int64_t n_atoms, const double *pos, double rc, const double *cell,
                                  const int32_t *nimg, int f32, const int64_t *centers, int64_t nc,
                                  int64_t *row_ptr, int32_t *cols, int32_t *img, int64_t cap) {
    double rc2 = rc * rc;
    int64_t e = 0;
    row_ptr[0] = 0;
    for (int64_t c = 0; c < nc; ++c) {
        int64_t i = centers ? centers[c] : c;
        for (int64_t j = 0; j < n_atoms; ++j)
            for (int na = -nimg[0]; na <= nimg[0]; ++na)
                for (int nb = -nimg[1]; nb <= nimg[1]; ++nb)
                    for (int ncc = -nimg[2]; ncc <= nimg[2]; ++ncc) {
                        if (j == i && na == 0 && nb == 0 && ncc == 0) continue;
                        int n[3] = {na, nb, ncc};
                        double q[3];
                        for (int d = 0; d < 3; ++d) q[d] = image_coord(pos, cell, j, n, d, f32);
                        if (is_neighbour(pos + 3 * i, q, rc2)) {
                            if (cols && e < cap) {
                                cols[e] = (int32_t)j;
                                img[3 * e] = na;
                                img[3 * e + 1] = nb;
                                img[3 * e + 2] = ncc;
                            }
                            ++e;
                        }
                    }
        row_ptr[c + 1] = e;
    }
    return e;
}

/* A second, separately written neighbour builder on a uniform grid (cells of
 * edge >= r_cut), for structures too large for the all-pairs loop.  Returns
 * the directed edge count; cols ascending per row. */
static int cmp_i32(const void *a, const void *b) {
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

int64_t oracle_neighbors_grid(int64_t n_atoms, const double *pos, double rc, int64_t *row_ptr, int32_t *cols,
                              int64_t cap) {
    double lo[3] = {INFINITY, INFINITY, INFINITY}, hi[3] = {-INFINITY, -INFINITY, -INFINITY};
    for (int64_t i = 0; i < n_atoms; ++i)
        for (int d = 0; d < 3; ++d) {
            if (pos[3 * i + d] < lo[d]) lo[d] = pos[3 * i + d];
            if (pos[3 * i + d] > hi[d]) hi[d] = pos[3 * i + d];
        }
    int64_t dim[3];
    for (int d = 0; d < 3; ++d) {
        dim[d] = (int64_t)floor((hi[d] - lo[d]) / rc) + 1;
        if (dim[d] < 1) dim[d] = 1;
    }
    int64_t ncell = dim[0] * dim[1] * dim[2];
    int64_t *start = (int64_t *)calloc((size_t)ncell + 1, sizeof(int64_t));
    int64_t *cell = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_atoms ? n_atoms : 1));
    int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_atoms ? n_atoms : 1));
    int64_t (*cc)[3] = malloc(sizeof(int64_t[3]) * (size_t)(n_atoms ? n_atoms : 1));
    if (!start || !cell || !order || !cc) return -1;
    for (int64_t i = 0; i < n_atoms; ++i) {
        for (int d = 0; d < 3; ++d) {
            int64_t v = (int64_t)floor((pos[3 * i + d] - lo[d]) / rc);
            if (v >= dim[d]) v = dim[d] - 1;
            if (v < 0) v = 0;
            cc[i][d] = v;
        }
        cell[i] = (cc[i][0] * dim[1] + cc[i][1]) * dim[2] + cc[i][2];
        start[cell[i] + 1]++;
    }
    for (int64_t c = 0; c < ncell; ++c) start[c + 1] += start[c];
    int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)ncell);
    memcpy(fill, start, sizeof(int64_t) * (size_t)ncell);
    for (int64_t i = 0; i < n_atoms; ++i) order[fill[cell[i]]++] = i;
    free(fill);
    double rc2 = rc * rc;
    int64_t e = 0;
    row_ptr[0] = 0;
    for (int64_t i = 0; i < n_atoms; ++i) {
        int64_t e0 = e;
        for (int64_t a = cc[i][0] - 1; a <= cc[i][0] + 1; ++a)
            for (int64_t b = cc[i][1] - 1; b <= cc[i][1] + 1; ++b)
                for (int64_t c = cc[i][2] - 1; c <= cc[i][2] + 1; ++c) {
                    if (a < 0 || b < 0 || c < 0 || a >= dim[0] || b >= dim[1] || c >= dim[2]) continue;
                    int64_t k = (a * dim[1] + b) * dim[2] + c;
                    for (int64_t t = start[k]; t < start[k + 1]; ++t) {
                        int64_t j = order[t];
                        if (j == i) continue;
                        if (is_neighbour(pos + 3 * i, pos + 3 * j, rc2)) {
                            if (cols && e < cap) cols[e] = (int32_t)j;
                            ++e;
                        }
                    }
                }
        if (cols && e <= cap) qsort(cols + e0, (size_t)(e - e0), sizeof(int32_t), cmp_i32);
        row_ptr[i + 1] = e;
    }
    free(start); free(cell); free(order); free(cc);
    return e;
}

/* ------------------------------------------------------- solid harmonics
 * Y[lm] = Y_lm(u) and G[3][lm] = grad of the polynomial r^l Y_lm at u, for a
 * unit vector u, by summing the monomial expansion in long double. */
static void solid_harmonics_unit(const oracle_params *P, int lmax, const ld u[3], ld *Y, ld *G) {
    int L = (lmax + 1) * (lmax + 1);
    ld pw[3][32];
    for (int d = 0; d < 3; ++d) {
        pw[d][0] = 1.0L;
        for (int k = 1; k <= lmax + 1; ++k) pw[d][k] = pw[d][k - 1] * u[d];
    }
    for (int lm = 0; lm < L; ++lm) {
        ld y = 0, gx = 0, gy = 0, gz = 0;
        for (int t = P->sh_ptr[lm]; t < P->sh_ptr[lm + 1]; ++t) {
            int a = P->sh_exp[3 * t], b = P->sh_exp[3 * t + 1], c = P->sh_exp[3 * t + 2];
            ld k = LD(P->sh_c_hi[t], P->sh_c_lo[t]);
            y += k * pw[0][a] * pw[1][b] * pw[2][c];
            if (a > 0) gx += k * a * pw[0][a - 1] * pw[1][b] * pw[2][c];
            if (b > 0) gy += k * b * pw[0][a] * pw[1][b - 1] * pw[2][c];
            if (c > 0) gz += k * c * pw[0][a] * pw[1][b] * pw[2][c - 1];
        }
        Y[lm] = y;
        if (G) { G[lm] = gx; G[L + lm] = gy; G[2 * L + lm] = gz; }
    }
}

/* exported for tests: Y (L) and grad of r^l Y_lm at the unit vector of v (3L) */
void oracle_solid_harmonics(const oracle_params *P, int lmax, const double *v, double *Y, double *G) {
    int L = (lmax + 1) * (lmax + 1);
    ld r = sqrtl((ld)v[0] * v[0] + (ld)v[1] * v[1] + (ld)v[2] * v[2]);
    ld u[3] = {v[0] / r, v[1] / r, v[2] / r};
    ld *y = malloc(sizeof(ld) * 4 * L);
    solid_harmonics_unit(P, lmax, u, y, y + L);
    for (int k = 0; k < L; ++k) Y[k] = (double)y[k];
    if (G) for (int k = 0; k < 3 * L; ++k) G[k] = (double)y[L + k];
    free(y);
}

/* ----------------------------------------------- modified spherical Bessel
 * i_l(x) for l = 0..lmax (unscaled, long double).  The two highest orders come
 * from the power series
 *   i_l(x) = x^l sum_k (x^2/2)^k / (k! (2l+2k+1)!!)
 * (all terms positive), the rest by the downward recurrence
 *   i_{l-1}(x) = i_{l+1}(x) + (2l+1)/x i_l(x), which is stable downward. */
static ld bessel_series(int l, ld x) {
    ld dfact = 1.0L; /* (2l+1)!! */
    for (int k = 1; k <= 2 * l + 1; k += 2) dfact *= k;
    ld term = powl(x, l) / dfact, sum = term, h = 0.5L * x * x;
    for (int k = 1; k < 100000; ++k) {
        term *= h / ((ld)k * (ld)(2 * l + 2 * k + 1));
        sum += term;
        /* stop once past the largest term and negligible */
        if (term < sum * 1e-22L && (ld)k * (ld)(2 * l + 2 * k + 1) > h) break;
    }
    return sum;
}

void oracle_bessel_il(int lmax, double xd, double *out) {
    ld x = xd;
    ld *v = malloc(sizeof(ld) * (lmax + 2));
    if (x == 0) {
        for (int l = 0; l <= lmax; ++l) out[l] = (l == 0) ? 1.0 : 0.0;
        free(v);
        return;
    }
    v[lmax + 1] = bessel_series(lmax + 1, x);
    v[lmax] = bessel_series(lmax, x);
    for (int l = lmax; l >= 1; --l) v[l - 1] = v[l + 1] + (ld)(2 * l + 1) / x * v[l];
    for (int l = 0; l <= lmax; ++l) out[l] = (double)v[l];
    free(v);
}

static void bessel_all(int lmax, ld x, ld *v) { /* v[0..lmax+1] */
    v[lmax + 1] = bessel_series(lmax + 1, x);
    v[lmax] = bessel_series(lmax, x);
    for (int l = lmax; l >= 1; --l) v[l - 1] = v[l + 1] + (ld)(2 * l + 1) / x * v[l];
}

/* ----------------------------------------------------------- radial parts
 * For one neighbour at distance r (r > 0), fill for every (n, l):
 *   GTO (Eq. gto-coefficients):  R[n][l] = sum_k beta^l_nk (2 pi)^{3/2} sigma^3
 *        exp(-alpha r^2/(1+2 sigma^2 alpha)) / (1+2 sigma^2 alpha)^{l+3/2}
 *     so that c_nlm = R[n][l] r^l Y_lm; and dR[n][l] = dR/dr.
 *   polynomial (Eq. poly-coefficients-exact with Gauss-Legendre):
 *     R[n][l] = f_nl(r) = 4 pi exp(-r^2/2s^2) sum_q G[n][q] exp(-r_q^2/2s^2) i_l(r_q r/s^2)
 *     so that c_nlm = f_nl Y_lm; and dR[n][l] = f'_nl(r). */
static void radial(const oracle_params *P, ld r, ld *R, ld *dR) {
    int n = P->n, lmax = P->lmax;
    ld s2 = (ld)P->sigma * P->sigma;
    if (P->rbf == 0) {
        ld pref = powl(2.0L * 3.14159265358979323846264338327950288L, 1.5L) * s2 * (ld)P->sigma;
        for (int l = 0; l <= lmax; ++l)
            for (int a = 0; a < n; ++a) {
                ld acc = 0, dacc = 0;
                for (int k = 0; k < n; ++k) {
                    ld al = LD(P->alpha_hi[l * n + k], P->alpha_lo[l * n + k]);
                    ld be = LD(P->beta_hi[(l * n + a) * n + k], P->beta_lo[(l * n + a) * n + k]);
                    ld den = 1.0L + 2.0L * s2 * al;
                    ld e = expl(-al * r * r / den) / powl(den, (ld)l + 1.5L);
                    acc += be * e;
                    dacc += be * e * (-2.0L * al * r / den);
                }
                R[a * (lmax + 1) + l] = pref * acc;
                dR[a * (lmax + 1) + l] = pref * dacc;
            }
    } else if (P->rbf == 2) {
        /* Eqs. (poly-coefficients) and (poly-radial-derivative), the Laplace
           (steepest-descent) form to first order in sigma^2, k = 1..n_max:
           f_nl = (2 pi)^{3/2} s^3 sum_k W_nk/N_k (rc-r)^{k+2}
                  [1 - l(l+1)s^2/(2r^2) - (k+2)s^2/(r(rc-r)) + (k+2)(k+1)s^2/(2(rc-r)^2)]
           f'_nl = (2 pi)^{3/2} s^3 sum_k W_nk/N_k (rc-r)^{k+1}
                  [-(k+2) + l(l+1)s^2(rc-r)/r^3 + (k+2)(l(l+1)+2)s^2/(2r^2)
                   + (k+1)(k+2)s^2/(r(rc-r)) - k(k+1)(k+2)s^2/(2(rc-r)^2)] */
        /* The sums over k cancel heavily: W_nk/N_k grow large with alternating
           signs, and at n_max = 16 long double keeps only ~9 digits of f.  They
           run in __float128, W_nk/N_k taken from its (hi, lo) pair. */
        const qd pi = 3.14159265358979323846264338327950288Q, sg = (qd)P->sigma, qs2 = sg * sg;
        const qd pref = 2 * pi * sqrtq(2 * pi) * qs2 * sg;
        const qd rq = (qd)r, u = (qd)P->rc - rq;
        for (int a = 0; a < n; ++a)
            for (int l = 0; l <= lmax; ++l) {
                qd ll = (qd)(l * (l + 1)), acc = 0, dacc = 0;
                for (int b = 0; b < n; ++b) {
                    qd k = (qd)(b + 1), wn = (qd)P->wn_hi[a * n + b] + (qd)P->wn_lo[a * n + b];
                    qd uk1 = 1; /* u^(k+1) */
                    for (int e = 0; e < b + 2; ++e) uk1 *= u;
                    qd br = 1 - ll * qs2 / (2 * rq * rq) - (k + 2) * qs2 / (rq * u) + (k + 2) * (k + 1) * qs2 / (2 * u * u);
                    qd dbr = -(k + 2) + ll * qs2 * u / (rq * rq * rq) + (k + 2) * (ll + 2) * qs2 / (2 * rq * rq) +
                             (k + 1) * (k + 2) * qs2 / (rq * u) - k * (k + 1) * (k + 2) * qs2 / (2 * u * u);
                    acc += wn * uk1 * u * br;
                    dacc += wn * uk1 * dbr;
                }
                R[a * (lmax + 1) + l] = (ld)(pref * acc);
                dR[a * (lmax + 1) + l] = (ld)(pref * dacc);
            }
    } else {
        int Q = P->Q;
        ld *iv = malloc(sizeof(ld) * (size_t)Q * (lmax + 3));
        ld *gq = malloc(sizeof(ld) * (size_t)Q);
        for (int q = 0; q < Q; ++q) {
            ld rq = LD(P->rq_hi[q], P->rq_lo[q]);
            bessel_all(lmax + 1, rq * r / s2, iv + (size_t)q * (lmax + 3));
            gq[q] = expl(-(rq * rq + r * r) / (2.0L * s2));
        }
        ld fourpi = 4.0L * 3.14159265358979323846264338327950288L;
        for (int a = 0; a < n; ++a)
            for (int l = 0; l <= lmax; ++l) {
                ld acc = 0, dacc = 0;
                for (int q = 0; q < Q; ++q) {
                    ld rq = LD(P->rq_hi[q], P->rq_lo[q]);
                    ld G = LD(P->G_hi[a * Q + q], P->G_lo[a * Q + q]);
                    ld x = rq * r / s2;
                    ld il = iv[(size_t)q * (lmax + 3) + l], il1 = iv[(size_t)q * (lmax + 3) + l + 1];
                    ld dil = il1 + (ld)l / x * il; /* d i_l / dx */
                    acc += G * gq[q] * il;
                    dacc += G * gq[q] * (-(r / s2) * il + (rq / s2) * dil);
                }
                R[a * (lmax + 1) + l] = fourpi * acc;
                dR[a * (lmax + 1) + l] = fourpi * dacc;
            }
        free(iv);
        free(gq);
    }
}

/* position-independent on-site l = 0 term of the center's own species */
static void onsite(const oracle_params *P, double *c0) {
    int n = P->n;
    ld s2 = (ld)P->sigma * P->sigma, pi = 3.14159265358979323846264338327950288L;
    for (int a = 0; a < n; ++a) {
        ld acc = 0;
        if (P->rbf == 0) { /* sqrt(2) pi sigma^3 sum_k beta^0_nk / (1 + 2 s^2 alpha_k0)^{3/2} */
            for (int k = 0; k < n; ++k) {
                ld al = LD(P->alpha_hi[k], P->alpha_lo[k]);
                acc += LD(P->beta_hi[a * n + k], P->beta_lo[a * n + k]) / powl(1.0L + 2.0L * s2 * al, 1.5L);
            }
            acc *= sqrtl(2.0L) * pi * s2 * (ld)P->sigma;
        } else { /* 4 pi Y_00 sum_q G[n][q] exp(-r_q^2 / 2 s^2), i_0(0) = 1 */
            for (int q = 0; q < P->Q; ++q) {
                ld rq = LD(P->rq_hi[q], P->rq_lo[q]);
                acc += LD(P->G_hi[a * P->Q + q], P->G_lo[a * P->Q + q]) * expl(-rq * rq / (2.0L * s2));
            }
            acc *= 4.0L * pi / sqrtl(4.0L * pi);
        }
        c0[a] = (double)acc;
    }
}

/* ----------------------------------------------------------- features */
/* Worker threads of the per-center loop: n > 0 sets them; returns the count
 * the next oracle_soap call uses. */
int oracle_threads(int n) {
    if (n > 0) omp_set_num_threads(n);
    return omp_get_max_threads();
}

int64_t oracle_num_features(int S, int n, int lmax) {
    int64_t F = 0;
    for (int mu = 0; mu < S; ++mu)
        for (int nu = mu; nu < S; ++nu)
            for (int a = 0; a < n; ++a)
                for (int b = (mu == nu ? a : 0); b < n; ++b) F += lmax + 1;
    return F;
}

/* -------------------------------------------------------------- main entry
 * For each requested center (centers[c], or c when centers is NULL), using the
 * neighbour rows nb_ptr/nb_col (ascending j):
 *   desc[c][F]                     power spectrum
 *   cout[c][S][n][L] (optional)    expansion coefficients c^mu_nlm
 *   if jac: blocks for j in N(i) and i itself, in ascending atom index,
 *   blk_ptr[c] .. blk_ptr[c+1] (= row length + 1), atom index in blk_j,
 *   jac[b][3][F] = d p_i / d r_j;
 *   dcout (optional) [e][3][n][L] for the e-th neighbour edge of the rows
 *   (row order): d c^{s_j}_{nlm}(i) / d r_j, the gradient of Eqs.
 *   (gto-derivative) / (poly-cartesian-derivative); only the neighbour's own
 *   species block of c depends on r_j.
 * Returns 0, or -1 on allocation failure. */
int oracle_soap(const oracle_params *P, int64_t n_atoms, const double *pos, const int32_t *spec,
                const int64_t *centers, int64_t nc, const int64_t *nb_ptr, const int32_t *nb_col,
                double *desc, double *cout, int want_jac, const int64_t *blk_ptr, int32_t *blk_j, double *jac,
                double *dcout) {
    (void)n_atoms;
    const int S = P->S, n = P->n, lmax = P->lmax, L = (lmax + 1) * (lmax + 1);
    const int64_t F = oracle_num_features(S, n, lmax);
    const size_t CSZ = (size_t)S * n * L;
    double c0[64];
    if (n > 64) return -1;
    onsite(P, c0);
    int fail = 0;

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t ci = 0; ci < nc; ++ci) {
        int64_t i = centers ? centers[ci] : ci;
        int64_t e0 = nb_ptr[ci], deg = nb_ptr[ci + 1] - e0;
        const int want_dc = want_jac || dcout != NULL;
        double *c = calloc(CSZ, sizeof(double));
        double *dc = want_dc ? calloc((size_t)(deg > 0 ? deg : 1) * 3 * n * L, sizeof(double)) : NULL;
        ld *Y = malloc(sizeof(ld) * 4 * L), *R = malloc(sizeof(ld) * 2 * n * (lmax + 1));
        if (!c || (want_dc && !dc) || !Y || !R) {
            fail = 1;
            free(c); free(dc); free(Y); free(R);
            continue;
        }
        ld *G = Y + L, *dR = R + n * (lmax + 1);
        /* on-site term of the center itself (its own species, l = 0) */
        for (int a = 0; a < n; ++a) c[((size_t)spec[i] * n + a) * L + 0] += c0[a];
        for (int64_t e = 0; e < deg; ++e) {
            int64_t j = nb_col[e0 + e];
            int s = spec[j];
            ld v[3] = {(ld)pos[3 * j] - (ld)pos[3 * i], (ld)pos[3 * j + 1] - (ld)pos[3 * i + 1],
                       (ld)pos[3 * j + 2] - (ld)pos[3 * i + 2]};
            ld r = sqrtl(v[0] * v[0] + v[1] * v[1] + v[2] * v[2]);
            if (r == 0) { /* coincident atom: its on-site term only, no gradient */
                for (int a = 0; a < n; ++a) c[((size_t)s * n + a) * L] += c0[a];
                continue;
            }
            ld u[3] = {v[0] / r, v[1] / r, v[2] / r};
            solid_harmonics_unit(P, lmax, u, Y, G);
            radial(P, r, R, dR);
            for (int a = 0; a < n; ++a)
                for (int l = 0; l <= lmax; ++l) {
                    ld Rv = R[a * (lmax + 1) + l], dRv = dR[a * (lmax + 1) + l];
                    for (int m = -l; m <= l; ++m) {
                        int lm = l * l + l + m;
                        ld y = Y[lm];
                        if (P->rbf == 0) {
                            /* c += R r^l Y ; grad = R' r^l Y u + R grad(r^l Y) ,
                               grad(r^l Y)(v) = r^(l-1) grad-poly(u) */
                            ld rl = powl(r, l);
                            c[((size_t)s * n + a) * L + lm] += (double)(Rv * rl * y);
                            if (want_dc)
                                for (int d = 0; d < 3; ++d) {
                                    ld g = (l > 0) ? powl(r, l - 1) * G[d * L + lm] : 0.0L;
                                    dc[((size_t)(e * 3 + d) * n + a) * L + lm] =
                                        (double)(dRv * rl * y * u[d] + Rv * g);
                                }
                        } else {
                            /* Eq. (poly-cartesian-derivative):
                               dc/dx = (x/r) Y f' + f dY/dx,  dY/dx = (grad-poly(u) - l Y u)/r */
                            c[((size_t)s * n + a) * L + lm] += (double)(Rv * y);
                            if (want_dc)
                                for (int d = 0; d < 3; ++d) {
                                    ld dY = (G[d * L + lm] - (ld)l * y * u[d]) / r;
                                    dc[((size_t)(e * 3 + d) * n + a) * L + lm] = (double)(u[d] * y * dRv + Rv * dY);
                                }
                        }
                    }
                }
        }
        if (cout) memcpy(cout + ci * CSZ, c, CSZ * sizeof(double));
        if (dcout && deg > 0) memcpy(dcout + (size_t)e0 * 3 * n * L, dc, (size_t)deg * 3 * n * L * sizeof(double));
        /* Eq. (powerspectrum) */
        double *drow = desc + ci * F;
        int64_t f = 0;
        for (int mu = 0; mu < S; ++mu)
            for (int nu = mu; nu < S; ++nu)
                for (int a = 0; a < n; ++a)
                    for (int b = (mu == nu ? a : 0); b < n; ++b)
                        for (int l = 0; l <= lmax; ++l) {
                            double acc = 0;
                            for (int m = -l; m <= l; ++m) {
                                int lm = l * l + l + m;
                                acc += c[((size_t)mu * n + a) * L + lm] * c[((size_t)nu * n + b) * L + lm];
                            }
                            drow[f++] = M_PI * sqrt(8.0 / (2 * l + 1)) * acc;
                        }
        if (want_jac) {
            /* blocks in ascending atom index, the center inserted at its place */
            int64_t b0 = blk_ptr[ci];
            int64_t self_slot = -1, k = 0;
            for (int64_t e = 0; e <= deg; ++e) {
                int64_t j = (e < deg) ? nb_col[e0 + e] : INT64_MAX;
                if (self_slot < 0 && i < j) { self_slot = b0 + k; blk_j[b0 + k] = (int32_t)i; ++k; }
                if (e < deg) { blk_j[b0 + k] = (int32_t)j; ++k; }
            }
            double *Js = jac + (size_t)self_slot * 3 * F;
            memset(Js, 0, sizeof(double) * 3 * F);
            k = 0;
            for (int64_t e = 0; e < deg; ++e) {
                int64_t slot = b0 + k;
                if (slot == self_slot) { ++k; slot = b0 + k; }
                ++k;
                int s = spec[nb_col[e0 + e]];
                double *Je = jac + (size_t)slot * 3 * F;
                /* Eq. (powerspectrum-derivative): only this edge's own dc is
                   non-zero, and only in the block of its species s */
                for (int d = 0; d < 3; ++d) {
                    const double *g = dc + (size_t)(e * 3 + d) * n * L;
                    int64_t ff = 0;
                    for (int mu = 0; mu < S; ++mu)
                        for (int nu = mu; nu < S; ++nu)
                            for (int a = 0; a < n; ++a)
                                for (int b = (mu == nu ? a : 0); b < n; ++b)
                                    for (int l = 0; l <= lmax; ++l) {
                                        double acc = 0;
                                        for (int m = -l; m <= l; ++m) {
                                            int lm = l * l + l + m;
                                            if (s == mu) acc += g[(size_t)a * L + lm] * c[((size_t)nu * n + b) * L + lm];
                                            if (s == nu) acc += c[((size_t)mu * n + a) * L + lm] * g[(size_t)b * L + lm];
                                        }
                                        double val = M_PI * sqrt(8.0 / (2 * l + 1)) * acc;
                                        Je[(size_t)d * F + ff] = val;
                                        Js[(size_t)d * F + ff] -= val; /* translational invariance */
                                        ++ff;
                                    }
                }
            }
        }
        free(c); free(dc); free(Y); free(R);
    }
    return fail ? -1 : 0;
}

/* exported for tests: radial parts R[n][l], dR[n][l] at distance r > 0 and the
 * on-site terms c0[n] */
void oracle_radial(const oracle_params *P, double r, double *R, double *dR, double *c0) {
    int m = P->n * (P->lmax + 1);
    ld *t = malloc(sizeof(ld) * 2 * m);
    radial(P, (ld)r, t, t + m);
    for (int k = 0; k < m; ++k) { R[k] = (double)t[k]; dR[k] = (double)t[m + k]; }
    free(t);
    if (c0) onsite(P, c0);
}
