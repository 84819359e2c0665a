// Host-side basis constants (see basis.cpp).  Internal to the library.
#pragma once

#ifdef __cplusplus
extern "C" {
#endif

// GTO basis (Sec. 2.2).  Outputs, all row-major:
//   betaC [l][n][k] = beta^l_nk * (2 pi)^{3/2} sigma^3 / (1 + 2 sigma^2 alpha_kl)^{l+3/2}
//   betaCa[l][n][k] = -2 * betaC[l][n][k] * aprime[l][k]
//   aprime[l][k]    = alpha_kl / (1 + 2 sigma^2 alpha_kl)
//   c0[n]           = on-site l = 0 term of Eq. (gto-coefficients)
// so that B_nl(r) = sum_k betaC e^{-aprime r^2} and c_nlm = B_nl r^l Y_lm.
// betaC_lo, betaCa_lo, aprime_lo (each may be NULL): the rounding remainders
// x - (double)x of the three tables, for the compensated float64 evaluation.
// Returns 0, or -1 with a message in err.
int soap_basis_gto(double r_cut, int n_max, int l_max, double sigma, double *betaC, double *betaCa,
                   double *aprime, double *c0, char *err, int errlen, double *betaC_lo, double *betaCa_lo,
                   double *aprime_lo);

// Polynomial basis (Sec. 2.3) with a quad_n-point Gauss-Legendre rule on
// [0, r_cut]:  G[n][q] = 4 pi w_q r_q^2 g_n(r_q),  rq[q] = r_q,
// c0[n] = on-site l = 0 term.  Returns 0 or -1.
int soap_basis_poly(double r_cut, int n_max, double sigma, int quad_n, double *G, double *rq, double *c0,
                    char *err, int errlen);

// Laplace form of the polynomial basis (Eqs. poly-coefficients,
// poly-radial-derivative).  With u = r_cut - r and WN_nk = (2 pi)^{3/2}
// sigma^3 W_nk / N_k (k = 1..n_max), the radial factors need
//   P_n0(u) = sum_k WN_nk u^{k+2}  and its u-derivatives P_n1, P_n2, P_n3.
// Their monomial coefficients grow large with alternating signs as n_max
// grows, so they are handed over as Chebyshev series on [0, r_cut]:
//   P_nj(u) = sum_{i < n_max + 3} CH[n][i][j] T_i(2u / r_cut - 1),
// from interpolation at n_max + 3 Chebyshev points in 113-bit arithmetic
// (exact for degree n_max + 2).  Returns 0 or -1.
int soap_basis_poly_laplace(double r_cut, int n_max, double sigma, double *CH, char *err, int errlen);

// Real solid-harmonic normalisation N[l][m], 0 <= m <= l, row stride l_max+1.
void soap_basis_sh_norms(int l_max, double *Nlm);

// 2^(j/64), j = 0..63, as pairs t[2j] = (double)v, t[2j+1] = v - t[2j]
// (v in 113-bit arithmetic): the table of the exponential of the GTO
// radial factors.
void soap_exp2_table64(double *t);

#ifdef __cplusplus
}
#endif
