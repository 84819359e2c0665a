// SOAP descriptor and Jacobian kernels for gfx950 (wave64).
//
// Both kernels evaluate, per directed edge e = (i -> j) with r = r_j - r_i
// formed in float64 (exact for float32 inputs):
//   * real solid harmonics S_lm(r) = r^l Y_lm(r_hat) and their Cartesian
//     gradients, by the recurrences below (one thread per (edge, |m|));
//   * radial factors B_nl(r) and Bh_nl(r) = (1/r) dB_nl/dr such that the
//     edge's contribution to the coefficients is c_nlm += B_nl S_lm and its
//     gradient is dc_nlm/dr_j = Bh_nl r S_lm + B_nl grad S_lm:
//       GTO (Eq. gto-coefficients, gto-derivative):
//         B_nl = sum_k betaC^l_nk exp(-a'_kl r^2),  Bh_nl = -2 sum_k betaC a' exp(..)
//       polynomial (Eq. poly-coefficients-exact with Gauss-Legendre, and the
//         chain rule Eq. poly-cartesian-derivative written for S_lm):
//         B_nl  = r^-l sum_q G_nq e^{-(r_q-r)^2/2s^2} ii_l(r_q r/s^2)
//         Bh_nl = r^-(l+1) / s^2 sum_q G_nq e^{-(r_q-r)^2/2s^2} (r_q ii_{l+1} - r ii_l)
//       with ii_l(x) = e^-x i_l(x) and d/dx (x^-l i_l) = x^-l i_{l+1}.
//
// k_density: one workgroup per (center, l-group).  Accumulates c (and, for
//   the Jacobian, D = sum over edges of dc, i.e. minus the derivative of c
//   with respect to the center) in LDS, then writes the power spectrum
//   Eq. (powerspectrum) and the center's own Jacobian block
//   -K_l sum_m (D^mu c^nu + c^mu D^nu) (Eq. powerspectrum-derivative with
//   translational invariance).  c goes to a float64 scratch for k_jacobian.
// k_jacobian: one workgroup per center, edges in chunks.  Per edge it forms
//   U^nu_{n'l} = sum_m S_lm c^nu_{n'lm} and V = sum_m grad S_lm c^nu_{n'lm}
//   (the per-edge precontraction the paper describes in Sec. 3.2), then each
//   output is K_l (Bh_nl r_x U + B_nl V_x) [+ the mirrored term on a
//   diagonal species pair]: no (2l+1)-long sums in the store loop.
//   Output rows are the F_e features whose pair contains species(j).
// All arithmetic is float64; outputs are converted once at the store.
#include "soap_internal.h"

namespace soap {
namespace {

constexpr int BS = 256; // workgroup size of both kernels

__device__ __forceinline__ int isqrt_lm(int lm) { // l such that l*l <= lm < (l+1)^2
    int l = (int)sqrtf((float)lm);
    while (l * l > lm) --l;
    while ((l + 1) * (l + 1) <= lm) ++l;
    return l;
}

template <typename T> __device__ __forceinline__ void store_nt(T *p, double v) {
    __builtin_nontemporal_store((T)v, p);
}

// ---------------------------------------------------------------------------
// Real solid harmonics for one |m| column.
//   (C_m + i S_m) = (x + i y)^m
//   Q_m^m = (2m-1)!!,  Q_{m+1}^m = (2m+1) z Q_m^m,
//   Q_l^m = ((2l-1) z Q_{l-1}^m - (l+m-1) r^2 Q_{l-2}^m) / (l-m)
//   S_l0 = N_l0 Q_l^0,  S_{l,m} = N_lm Q_l^m C_m,  S_{l,-m} = N_lm Q_l^m S_m
//   dQ_l^m/dx = -x Q_{l-1}^{m+1}, dQ_l^m/dy = -y Q_{l-1}^{m+1},
//   dQ_l^m/dz = (l+m) Q_{l-1}^m;  dC_m/dx = m C_{m-1}, dC_m/dy = -m S_{m-1},
//   dS_m/dx = m S_{m-1}, dS_m/dy = m C_{m-1}.
// Writes Y[lm - lm0] and dY[d*ldd + lm - lm0] for l in [l_lo, l_hi).
// grad = false skips the gradient.  zero_grad forces the gradient to 0.
// ---------------------------------------------------------------------------
template <bool GRAD>
__device__ void sh_column(int m, int l_lo, int l_hi, double x, double y, double z, const double *__restrict__ Nlm,
                          int ldN, double *__restrict__ Y, double *__restrict__ dY, int ldd, int lm0,
                          bool zero_grad) {
    const double r2 = x * x + y * y + z * z;
    double c = 1.0, s = 0.0, cm1 = 0.0, sm1 = 0.0;
    for (int k = 1; k <= m; ++k) {
        cm1 = c;
        sm1 = s;
        double cn = x * c - y * s;
        s = x * s + y * c;
        c = cn;
    }
    double dfm = 1.0; // (2m-1)!!
    for (int k = 1; k <= m; ++k) dfm *= (double)(2 * k - 1);
    // column m: q1 = Q_{l-1}^m, q2 = Q_{l-2}^m ; column m+1: p1 = Q_{l-2}^{m+1} ... tracked as "prev"
    double q1 = 0.0, q2 = 0.0; // Q_{l-1}^m, Q_{l-2}^m
    double p1 = 0.0, p2 = 0.0; // Q_{l-2}^{m+1}, Q_{l-3}^{m+1}
    for (int l = m; l < l_hi; ++l) {
        double q; // Q_l^m
        if (l == m) q = dfm;
        else if (l == m + 1) q = (double)(2 * m + 1) * z * dfm;
        else q = ((double)(2 * l - 1) * z * q1 - (double)(l + m - 1) * r2 * q2) / (double)(l - m);
        double p; // Q_{l-1}^{m+1}
        const int lp = l - 1;
        if (lp < m + 1) p = 0.0;
        else if (lp == m + 1) p = dfm * (double)(2 * m + 1);
        else if (lp == m + 2) p = (double)(2 * m + 3) * z * dfm * (double)(2 * m + 1);
        else p = ((double)(2 * lp - 1) * z * p1 - (double)(lp + m) * r2 * p2) / (double)(lp - m - 1);
        if (l >= l_lo) {
            const double N = Nlm[l * ldN + m];
            const int base = l * l + l - lm0;
            if (m == 0) {
                Y[base] = N * q;
                if (GRAD) {
                    double gx = -N * x * p, gy = -N * y * p, gz = N * (double)l * q1;
                    if (zero_grad) gx = gy = gz = 0.0;
                    dY[base] = gx;
                    dY[ldd + base] = gy;
                    dY[2 * ldd + base] = gz;
                }
            } else {
                Y[base + m] = N * q * c;
                Y[base - m] = N * q * s;
                if (GRAD) {
                    const double qm = (double)m * q, dz = N * (double)(l + m) * q1;
                    double gxc = N * (-x * p * c + qm * cm1), gyc = N * (-y * p * c - qm * sm1), gzc = dz * c;
                    double gxs = N * (-x * p * s + qm * sm1), gys = N * (-y * p * s + qm * cm1), gzs = dz * s;
                    if (zero_grad) gxc = gyc = gzc = gxs = gys = gzs = 0.0;
                    dY[base + m] = gxc;
                    dY[ldd + base + m] = gyc;
                    dY[2 * ldd + base + m] = gzc;
                    dY[base - m] = gxs;
                    dY[ldd + base - m] = gys;
                    dY[2 * ldd + base - m] = gzs;
                }
            }
        }
        q2 = q1;
        q1 = q;
        p2 = p1;
        p1 = p;
    }
}

// ---------------------------------------------------------------------------
// Scaled modified spherical Bessel functions ii_l(x) = e^-x i_l(x), l = 0..Lt.
// x >= Lt(Lt+1)/6.9: upward recurrence from the closed forms of ii_0, ii_1
//   (error growth bounded by about e^{Lt(Lt+1)/x} <= 1e3);
// otherwise: power series for the two highest orders (positive terms),
//   i_l(x) = x^l sum_k (x^2/2)^k / (k! (2l+2k+1)!!), then the downward
//   recurrence i_{l-1} = i_{l+1} + (2l+1)/x i_l (stable downward).
// ---------------------------------------------------------------------------
__device__ double bessel_series_scaled(int l, double x) {
    double t = 1.0;
    for (int k = 0; k < l; ++k) t *= x / (double)(2 * k + 3);
    t /= 1.0; // x^l / (2l+1)!! built as prod x/(2k+3) times 1/1
    double s = t;
    const double h = 0.5 * x * x;
    for (int k = 1; k < 400; ++k) {
        t *= h / ((double)k * (double)(2 * l + 2 * k + 1));
        s += t;
        if (t < 1e-17 * s && (double)k * (double)(2 * l + 2 * k + 1) > h) break;
    }
    return s * exp(-x);
}

__device__ void bessel_scaled_all(int Lt, double x, double *v /* [LT_MAX+1] */) {
    if (x == 0.0) {
#pragma unroll
        for (int k = 0; k <= LT_MAX; ++k) v[k] = (k == 0) ? 1.0 : 0.0;
        return;
    }
    const double ix = 1.0 / x;
    if (x * 6.9 >= (double)(Lt * (Lt + 1))) {
        const double em = exp(-2.0 * x);
        v[0] = 0.5 * (1.0 - em) * ix;
        v[1] = 0.5 * (1.0 + em) * ix - 0.5 * (1.0 - em) * ix * ix;
#pragma unroll
        for (int k = 1; k < LT_MAX; ++k)
            if (k < Lt) v[k + 1] = v[k - 1] - (double)(2 * k + 1) * ix * v[k];
    } else {
        // seeds at Lt and Lt-1, then downward
        double top = bessel_series_scaled(Lt, x);
        double nxt = (Lt >= 1) ? bessel_series_scaled(Lt - 1, x) : 0.0;
#pragma unroll
        for (int k = 0; k <= LT_MAX; ++k) {
            if (k == Lt) v[k] = top;
            if (k == Lt - 1) v[k] = nxt;
        }
#pragma unroll
        for (int k = LT_MAX - 1; k >= 1; --k)
            if (k < Lt) v[k - 1] = v[k + 1] + (double)(2 * k + 1) * ix * v[k];
    }
}

// ---------------------------------------------------------------------------
// Per-chunk edge staging, shared by both kernels.  LDS arrays:
//   geo[EC][4] (x, y, z, r), sp[EC] species,
//   Y[EC][Lg], dY[EC][3][Lg] (harmonics for lm in [lm0, lm0+Lg)),
//   B[EC][n][lgc], Bh[EC][n][lgc] (radial factors for l in [lg0, lg0+lgc)),
//   T[EC][Q][lgc+1] polynomial quadrature scratch.
// scaleK multiplies B and Bh by K_l = pi sqrt(8/(2l+1)).
// ---------------------------------------------------------------------------
struct Stage {
    double *geo, *Y, *dY, *B, *Bh, *T;
    int *sp;
};

template <bool GRAD>
__device__ void stage_angular_radial(const Params &P, const Stage &st, int nb, int lg0, int lg1, bool scaleK) {
    const int tid = threadIdx.x;
    const int lm0 = lg0 * lg0, Lg = lg1 * lg1 - lm0, lgc = lg1 - lg0, n = P.n;
    // harmonics: items (edge, m), m < lg1
    for (int it = tid; it < nb * lg1; it += BS) {
        const int e = it / lg1, m = it - e * lg1;
        const double *g = st.geo + 4 * e;
        sh_column<GRAD>(m, lg0 > m ? lg0 : m, lg1, g[0], g[1], g[2], P.Nlm, P.lmax + 1, st.Y + e * Lg,
                        GRAD ? st.dY + e * 3 * Lg : nullptr, Lg, lm0, g[3] == 0.0);
    }
    if (P.rbf == 0) {
        // GTO: items (edge, l)
        for (int it = tid; it < nb * lgc; it += BS) {
            const int e = it / lgc, lc = it - e * lgc, l = lg0 + lc;
            const double r = st.geo[4 * e + 3], r2 = r * r;
            double E[NMAX];
#pragma unroll
            for (int k = 0; k < NMAX; ++k) E[k] = (k < n) ? exp(-P.aprime[l * n + k] * r2) : 0.0;
            const double K = scaleK ? M_PI * sqrt(8.0 / (double)(2 * l + 1)) : 1.0;
            for (int a = 0; a < n; ++a) {
                const double *bc = P.betaC + ((size_t)l * n + a) * n;
                double b = 0.0;
#pragma unroll
                for (int k = 0; k < NMAX; ++k)
                    if (k < n) b += bc[k] * E[k];
                st.B[(e * n + a) * lgc + lc] = K * b;
                if (GRAD) {
                    const double *ba = P.betaCa + ((size_t)l * n + a) * n;
                    double bh = 0.0;
#pragma unroll
                    for (int k = 0; k < NMAX; ++k)
                        if (k < n) bh += ba[k] * E[k];
                    st.Bh[(e * n + a) * lgc + lc] = K * bh;
                }
            }
        }
    } else {
        // polynomial: items (edge, q) fill T = e^{-(r_q - r)^2/2s^2} ii_l(r_q r/s^2), l in [lg0, lg1]
        const int Q = P.Q, tw = lgc + 1;
        for (int it = tid; it < nb * Q; it += BS) {
            const int e = it / Q, q = it - e * Q;
            const double r = st.geo[4 * e + 3], rq = P.rq[q];
            const double gq = exp(-0.5 * (rq - r) * (rq - r) * P.inv_s2);
            double v[LT_MAX + 1];
            bessel_scaled_all(lg1, rq * r * P.inv_s2, v);
            double *t = st.T + ((size_t)e * Q + q) * tw;
#pragma unroll
            for (int k = 0; k <= LT_MAX; ++k)
                if (k >= lg0 && k <= lg1) t[k - lg0] = gq * v[k];
        }
        __syncthreads();
        for (int it = tid; it < nb * n * lgc; it += BS) {
            const int e = it / (n * lgc), rem = it - e * (n * lgc), a = rem / lgc, lc = rem - a * lgc;
            const int l = lg0 + lc;
            const double r = st.geo[4 * e + 3];
            const double *G = P.G + (size_t)a * Q;
            const double *t = st.T + (size_t)e * Q * tw;
            double b = 0.0, bh = 0.0;
            for (int q = 0; q < Q; ++q) {
                const double tl = t[q * tw + lc];
                b += G[q] * tl;
                if (GRAD) bh += G[q] * (P.rq[q] * t[q * tw + lc + 1] - r * tl);
            }
            const double K = scaleK ? M_PI * sqrt(8.0 / (double)(2 * l + 1)) : 1.0;
            if (r == 0.0) {
                b = (l == 0) ? b : 0.0;
                bh = 0.0;
            } else {
                double ir = 1.0 / r, rl = 1.0;
                for (int k = 0; k < l; ++k) rl *= ir;
                b *= rl;
                bh *= rl * ir * P.inv_s2;
            }
            st.B[(e * n + a) * lgc + lc] = K * b;
            if (GRAD) st.Bh[(e * n + a) * lgc + lc] = K * bh;
        }
    }
}

template <typename PosT>
__device__ __forceinline__ void stage_geometry(const Stage &st, const PosT *__restrict__ pos,
                                               const uint8_t *__restrict__ spec, const int32_t *__restrict__ cols,
                                               int64_t base, int nb, double3 pi) {
    const int tid = threadIdx.x;
    if (tid < nb) {
        const int64_t j = cols[base + tid];
        const double x = (double)pos[3 * j] - pi.x, y = (double)pos[3 * j + 1] - pi.y,
                     z = (double)pos[3 * j + 2] - pi.z;
        st.geo[4 * tid] = x;
        st.geo[4 * tid + 1] = y;
        st.geo[4 * tid + 2] = z;
        st.geo[4 * tid + 3] = sqrt(x * x + y * y + z * z);
        st.sp[tid] = spec[j];
    }
}

__device__ __forceinline__ size_t align8(size_t b) { return (b + 7) & ~(size_t)7; }

// ---------------------------------------------------------------------------
// k_density
// ---------------------------------------------------------------------------
template <typename PosT, typename OutT, bool JAC>
__global__ __launch_bounds__(BS) void k_density(Params P, Rows R, const PosT *__restrict__ pos, int EC,
                                                OutT *__restrict__ desc, OutT *__restrict__ c_out,
                                                OutT *__restrict__ jself, double *__restrict__ c_scratch) {
    extern __shared__ double smem[];
    const int G = P.n_groups;
    const int64_t ci = blockIdx.x / G;
    const int g = blockIdx.x - (int)(ci * G);
    const int lg0 = P.lgrp[g], lg1 = P.lgrp[g + 1], lgc = lg1 - lg0;
    const int lm0 = lg0 * lg0, Lg = lg1 * lg1 - lm0;
    const int S = P.S, n = P.n, tid = threadIdx.x;
    const int nL = n * Lg, SnL = S * nL;

    double *cacc = smem;
    double *Dacc = cacc + SnL; // [3][S][n][Lg]
    Stage st;
    st.geo = Dacc + (JAC ? 3 * SnL : 0);
    st.Y = st.geo + 4 * EC;
    st.dY = st.Y + EC * Lg;
    st.B = st.dY + (JAC ? 3 * EC * Lg : 0);
    st.Bh = st.B + EC * n * lgc;
    st.T = st.Bh + (JAC ? EC * n * lgc : 0);
    st.sp = (int *)(st.T + (P.rbf ? (size_t)EC * P.Q * (lgc + 1) : 0));

    for (int k = tid; k < SnL * (JAC ? 4 : 1); k += BS) cacc[k] = 0.0;

    const int64_t i = R.centers ? (int64_t)R.centers[ci] : ci;
    const double3 pi = make_double3((double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]);
    const int64_t e0 = R.row_ptr[ci], e1 = R.row_ptr[ci + 1];

    for (int64_t base = e0; base < e1; base += EC) {
        const int nb = (int)((e1 - base) < EC ? (e1 - base) : EC);
        __syncthreads();
        stage_geometry(st, pos, R.spec, R.cols, base, nb, pi);
        __syncthreads();
        stage_angular_radial<JAC>(P, st, nb, lg0, lg1, false);
        __syncthreads();
        // accumulate: each thread owns entries (a, lm) for every species
        for (int ent = tid; ent < nL; ent += BS) {
            const int a = ent / Lg, lmg = ent - a * Lg;
            const int lc = isqrt_lm(lmg + lm0) - lg0;
            double acc = 0.0, ax = 0.0, ay = 0.0, az = 0.0;
            int cur = st.sp[0];
            for (int e = 0; e < nb; ++e) {
                const int s = st.sp[e];
                if (s != cur) {
                    cacc[cur * nL + ent] += acc;
                    if (JAC) {
                        Dacc[cur * nL + ent] += ax;
                        Dacc[SnL + cur * nL + ent] += ay;
                        Dacc[2 * SnL + cur * nL + ent] += az;
                    }
                    acc = ax = ay = az = 0.0;
                    cur = s;
                }
                const double b = st.B[(e * n + a) * lgc + lc], y = st.Y[e * Lg + lmg];
                acc += b * y;
                if (JAC) {
                    const double bh = st.Bh[(e * n + a) * lgc + lc] * y;
                    const double *gg = st.geo + 4 * e;
                    const double *dy = st.dY + e * 3 * Lg + lmg;
                    ax += bh * gg[0] + b * dy[0];
                    ay += bh * gg[1] + b * dy[Lg];
                    az += bh * gg[2] + b * dy[2 * Lg];
                }
            }
            if (nb > 0) {
                cacc[cur * nL + ent] += acc;
                if (JAC) {
                    Dacc[cur * nL + ent] += ax;
                    Dacc[SnL + cur * nL + ent] += ay;
                    Dacc[2 * SnL + cur * nL + ent] += az;
                }
            }
        }
    }
    __syncthreads();
    // on-site term of the center (its species, l = 0)
    if (lg0 == 0)
        for (int a = tid; a < n; a += BS) cacc[(int)R.spec[i] * nL + a * Lg] += P.c0[a];
    __syncthreads();

    const int lw = P.lmax + 1;
    // power spectrum for the group's l
    if (desc) {
        for (int it = tid; it < P.nq_full * lgc; it += BS) {
            const int q = it / lgc, lc = it - q * lgc, l = lg0 + lc;
            const uint32_t f = P.fq[q];
            const int mu = f & 0xff, nu = (f >> 8) & 0xff, a = (f >> 16) & 0xff, b = f >> 24;
            const double *x = cacc + mu * nL + a * Lg + l * l - lm0;
            const double *y = cacc + nu * nL + b * Lg + l * l - lm0;
            double acc = 0.0;
            for (int m = 0; m < 2 * l + 1; ++m) acc += x[m] * y[m];
            desc[ci * P.F + q * lw + l] = (OutT)(M_PI * sqrt(8.0 / (double)(2 * l + 1)) * acc);
        }
    }
    const int Lfull = P.L;
    if (c_out)
        for (int it = tid; it < SnL; it += BS) {
            const int sa = it / Lg, lmg = it - sa * Lg;
            c_out[(ci * S * n + sa) * Lfull + lm0 + lmg] = (OutT)cacc[it];
        }
    if (JAC) {
        for (int it = tid; it < SnL; it += BS) {
            const int sa = it / Lg, lmg = it - sa * Lg;
            c_scratch[(ci * S * n + sa) * Lfull + lm0 + lmg] = cacc[it];
        }
        // center block: -K_l sum_m (D^mu_{n l m} c^nu_{n' l m} + c^mu D^nu)
        for (int it = tid; it < 3 * P.nq_full * lgc; it += BS) {
            const int d = it / (P.nq_full * lgc), rem = it - d * (P.nq_full * lgc);
            const int q = rem / lgc, lc = rem - q * lgc, l = lg0 + lc;
            const uint32_t f = P.fq[q];
            const int mu = f & 0xff, nu = (f >> 8) & 0xff, a = (f >> 16) & 0xff, b = f >> 24;
            const int oa = mu * nL + a * Lg + l * l - lm0, ob = nu * nL + b * Lg + l * l - lm0;
            const double *Dd = Dacc + d * SnL;
            double acc = 0.0;
            for (int m = 0; m < 2 * l + 1; ++m) acc += Dd[oa + m] * cacc[ob + m] + cacc[oa + m] * Dd[ob + m];
            jself[(ci * 3 + d) * P.F + q * lw + l] = (OutT)(-M_PI * sqrt(8.0 / (double)(2 * l + 1)) * acc);
        }
    }
}

// ---------------------------------------------------------------------------
// k_jacobian
// ---------------------------------------------------------------------------
template <typename PosT, typename OutT>
__global__ __launch_bounds__(BS) void k_jacobian(Params P, Rows R, const PosT *__restrict__ pos, int EB,
                                                 const double *__restrict__ c_scratch, OutT *__restrict__ jedge) {
    extern __shared__ double smem[];
    const int64_t ci = blockIdx.x;
    const int S = P.S, n = P.n, lw = P.lmax + 1, L = P.L, Sn = S * n, tid = threadIdx.x;
    const int Fe = P.Fe;
    const int64_t e0 = R.row_ptr[ci], e1 = R.row_ptr[ci + 1];
    if (e1 == e0) return;

    double *cc = smem;                // [S][n][L]
    double *U4 = cc + (size_t)Sn * L; // [EB][Sn][lw][4]
    Stage st;
    st.geo = U4 + (size_t)EB * Sn * lw * 4;
    st.Y = st.geo + 4 * EB;
    st.dY = st.Y + EB * L;
    st.B = st.dY + 3 * EB * L;
    st.Bh = st.B + EB * n * lw;
    st.T = st.Bh + EB * n * lw;
    st.sp = (int *)(st.T + (P.rbf ? (size_t)EB * P.Q * (lw + 1) : 0));

    const double *cg = c_scratch + ci * (size_t)Sn * L;
    for (int k = tid; k < Sn * L; k += BS) cc[k] = cg[k];
    const int64_t i = R.centers ? (int64_t)R.centers[ci] : ci;
    const double3 pi = make_double3((double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]);

    for (int64_t base = e0; base < e1; base += EB) {
        const int nb = (int)((e1 - base) < EB ? (e1 - base) : EB);
        __syncthreads();
        stage_geometry(st, pos, R.spec, R.cols, base, nb, pi);
        __syncthreads();
        stage_angular_radial<true>(P, st, nb, 0, lw, true);
        __syncthreads();
        // U/V precontraction: items (edge, u = (nu, n'), l)
        for (int it = tid; it < nb * Sn * lw; it += BS) {
            const int e = it / (Sn * lw), rem = it - e * (Sn * lw), u = rem / lw, l = rem - u * lw;
            const double *c = cc + (size_t)u * L + l * l;
            const double *y = st.Y + e * L + l * l;
            const double *dy = st.dY + e * 3 * L + l * l;
            double U = 0.0, Vx = 0.0, Vy = 0.0, Vz = 0.0;
            for (int m = 0; m < 2 * l + 1; ++m) {
                const double cv = c[m];
                U += y[m] * cv;
                Vx += dy[m] * cv;
                Vy += dy[L + m] * cv;
                Vz += dy[2 * L + m] * cv;
            }
            double *o = U4 + (size_t)it * 4;
            o[0] = U;
            o[1] = Vx;
            o[2] = Vy;
            o[3] = Vz;
        }
        __syncthreads();
        // assembly: items (edge, compressed feature)
        for (int it = tid; it < nb * Fe; it += BS) {
            const int e = it / Fe, fe = it - e * Fe;
            const int s = st.sp[e];
            const uint2 t = P.fe[(size_t)s * Fe + fe];
            const int l = t.x & 0xff, nb1 = (t.x >> 8) & 0xff, u1 = (t.x >> 16) & 0xff, two = t.x >> 24;
            const double *g = st.geo + 4 * e;
            const double bh1 = st.Bh[(e * n + nb1) * lw + l] , b1 = st.B[(e * n + nb1) * lw + l];
            const double *w1 = U4 + ((size_t)(e * Sn + u1) * lw + l) * 4;
            double hu = bh1 * w1[0];
            double jx = b1 * w1[1], jy = b1 * w1[2], jz = b1 * w1[3];
            if (two) {
                const int nb2 = t.y & 0xff, u2 = (t.y >> 8) & 0xff;
                const double bh2 = st.Bh[(e * n + nb2) * lw + l], b2 = st.B[(e * n + nb2) * lw + l];
                const double *w2 = U4 + ((size_t)(e * Sn + u2) * lw + l) * 4;
                hu += bh2 * w2[0];
                jx += b2 * w2[1];
                jy += b2 * w2[2];
                jz += b2 * w2[3];
            }
            OutT *o = jedge + ((base + e) * 3) * Fe + fe;
            store_nt(o, hu * g[0] + jx);
            store_nt(o + Fe, hu * g[1] + jy);
            store_nt(o + 2 * Fe, hu * g[2] + jz);
        }
    }
}

// dense[ci][j][3][F]: zero-filled by the caller; each stored block is copied
template <typename OutT>
__global__ void k_scatter_dense(Params P, Rows R, const OutT *__restrict__ jedge, const OutT *__restrict__ jself,
                                const int32_t *__restrict__ fmap, OutT *__restrict__ dense) {
    const int64_t ci = blockIdx.x;
    const int F = P.F, Fe = P.Fe;
    const int64_t i = R.centers ? (int64_t)R.centers[ci] : ci;
    OutT *row = dense + ci * R.n_atoms * 3 * F;
    for (int k = threadIdx.x; k < 3 * F; k += blockDim.x) row[i * 3 * F + k] = jself[ci * 3 * F + k];
    for (int64_t e = R.row_ptr[ci]; e < R.row_ptr[ci + 1]; ++e) {
        const int64_t j = R.cols[e];
        const int s = R.spec[j];
        for (int k = threadIdx.x; k < 3 * Fe; k += blockDim.x) {
            const int d = k / Fe, fe = k - d * Fe;
            row[(j * 3 + d) * F + fmap[s * Fe + fe]] = jedge[(e * 3 + d) * Fe + fe];
        }
    }
}

} // namespace

size_t density_lds_bytes(const Params &P, int jac, int lg0, int lg1, int EC) {
    const size_t Lg = (size_t)(lg1 * lg1 - lg0 * lg0), lgc = (size_t)(lg1 - lg0);
    const size_t SnL = (size_t)P.S * P.n * Lg;
    size_t d = SnL * (jac ? 4 : 1);
    d += (size_t)EC * (4 + Lg * (jac ? 4 : 1) + P.n * lgc * (jac ? 2 : 1) + (P.rbf ? P.Q * (lgc + 1) : 0));
    return d * 8 + (size_t)EC * 4;
}

size_t jacobian_lds_bytes(const Params &P, int EB) {
    const size_t L = (size_t)P.L, lw = (size_t)P.lmax + 1, Sn = (size_t)P.S * P.n;
    size_t d = Sn * L + (size_t)EB * (Sn * lw * 4 + 4 + 4 * L + 2 * P.n * lw + (P.rbf ? P.Q * (lw + 1) : 0));
    return d * 8 + (size_t)EB * 4;
}

hipError_t set_lds_limits() {
    const int lim = 160 * 1024;
    hipError_t e = hipSuccess;
#define SOAP_SET(K)                                                                                          \
    if (e == hipSuccess) e = hipFuncSetAttribute((const void *)(K), hipFuncAttributeMaxDynamicSharedMemorySize, lim);
    SOAP_SET((k_density<float, float, false>));
    SOAP_SET((k_density<float, float, true>));
    SOAP_SET((k_density<double, double, false>));
    SOAP_SET((k_density<double, double, true>));
    SOAP_SET((k_jacobian<float, float>));
    SOAP_SET((k_jacobian<double, double>));
#undef SOAP_SET
    return e;
}

hipError_t launch_density(const Params &P, const Rows &R, const void *pos, bool f64, bool jac,
                          const DensityLaunch &cfg, void *desc, void *c_out, void *jself, double *c_scratch,
                          hipStream_t st) {
    const int64_t blocks = R.nc * P.n_groups;
    if (blocks <= 0) return hipSuccess;
    dim3 grid((unsigned)blocks), block(BS);
    if (f64) {
        if (jac)
            hipLaunchKernelGGL((k_density<double, double, true>), grid, block, cfg.lds, st, P, R, (const double *)pos,
                               cfg.EC, (double *)desc, (double *)c_out, (double *)jself, c_scratch);
        else
            hipLaunchKernelGGL((k_density<double, double, false>), grid, block, cfg.lds, st, P, R,
                               (const double *)pos, cfg.EC, (double *)desc, (double *)c_out, (double *)jself,
                               c_scratch);
    } else {
        if (jac)
            hipLaunchKernelGGL((k_density<float, float, true>), grid, block, cfg.lds, st, P, R, (const float *)pos,
                               cfg.EC, (float *)desc, (float *)c_out, (float *)jself, c_scratch);
        else
            hipLaunchKernelGGL((k_density<float, float, false>), grid, block, cfg.lds, st, P, R, (const float *)pos,
                               cfg.EC, (float *)desc, (float *)c_out, (float *)jself, c_scratch);
    }
    return hipGetLastError();
}

hipError_t launch_jacobian(const Params &P, const Rows &R, const void *pos, bool f64, const JacLaunch &cfg,
                           const double *c_scratch, void *jedge, hipStream_t st) {
    if (R.nc <= 0) return hipSuccess;
    dim3 grid((unsigned)R.nc), block(BS);
    if (f64)
        hipLaunchKernelGGL((k_jacobian<double, double>), grid, block, cfg.lds, st, P, R, (const double *)pos, cfg.EB,
                           c_scratch, (double *)jedge);
    else
        hipLaunchKernelGGL((k_jacobian<float, float>), grid, block, cfg.lds, st, P, R, (const float *)pos, cfg.EB,
                           c_scratch, (float *)jedge);
    return hipGetLastError();
}

hipError_t launch_scatter_dense(const Params &P, const Rows &R, bool f64, const void *jedge, const void *jself,
                                const int32_t *fmap, void *dense, hipStream_t st) {
    if (R.nc <= 0) return hipSuccess;
    if (f64)
        hipLaunchKernelGGL(k_scatter_dense<double>, dim3((unsigned)R.nc), dim3(256), 0, st, P, R,
                           (const double *)jedge, (const double *)jself, fmap, (double *)dense);
    else
        hipLaunchKernelGGL(k_scatter_dense<float>, dim3((unsigned)R.nc), dim3(256), 0, st, P, R,
                           (const float *)jedge, (const float *)jself, fmap, (float *)dense);
    return hipGetLastError();
}

} // namespace soap
