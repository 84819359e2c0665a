// Device code of the SOAP descriptor and Jacobian kernels for gfx950 (wave64),
// shared by the translation units that instantiate the kernels.
//
// Both kernels evaluate, per directed edge e = (i -> j) with r = r_j - r_i
// formed in float64 (exact for float32 inputs):
//   * real solid harmonics S_lm(r) = r^l Y_lm(r_hat) by a division-free
//     column recurrence, and their Cartesian gradients from the degree l-1
//     harmonics (stage_edges);
//   * radial factors B_nl(r) and Bh_nl(r) = (1/r) dB_nl/dr such that the
//     edge's contribution to the coefficients is c_nlm += B_nl S_lm and its
//     gradient is dc_nlm/dr_j = Bh_nl r S_lm + B_nl grad S_lm:
//       GTO (Eq. gto-coefficients, gto-derivative):
//         B_nl = sum_k betaC^l_nk exp(-a'_kl r^2),  Bh_nl = -2 sum_k betaC a' exp(..)
//       polynomial (Eq. poly-coefficients-exact with Gauss-Legendre, and the
//         chain rule Eq. poly-cartesian-derivative written for S_lm):
//         B_nl  = r^-l sum_q G_nq e^{-(r_q-r)^2/2s^2} ii_l(r_q r/s^2)
//         Bh_nl = r^-(l+1) / s^2 sum_q G_nq e^{-(r_q-r)^2/2s^2} (r_q ii_{l+1} - r ii_l)
//       with ii_l(x) = e^-x i_l(x) and d/dx (x^-l i_l) = x^-l i_{l+1};
//       polynomial, Laplace form (Eqs. poly-coefficients, poly-radial-derivative):
//         B_nl = r^-l f_nl,  Bh_nl = r^-(l+1) (f'_nl - l f_nl / r)  (see stage_edges);
//       GTO, compensated (float64 mode, larger n_max): the GTO sums with every
//         exponential in double-double arithmetic and compensated dot products.
//
// k_density: persistent workgroups, each bound to one l-group and taking
//   centers from a counter.  Accumulates c (and, for the Jacobian, D = sum
//   over edges of dc, i.e. minus the derivative of c with respect to the
//   center), then writes the power spectrum Eq. (powerspectrum) and the
//   center's own Jacobian block -K_l sum_m (D^mu c^nu + c^mu D^nu)
//   (Eq. powerspectrum-derivative with translational invariance).  c goes to
//   a scratch for k_jacobian, at the staging precision (float32 in the mixed
//   mode, where every reader rounds it to float32 anyway).
// k_jacobian: one workgroup per center; per edge the precontraction
//   U = sum_m S_lm c, V = sum_m grad S_lm c on the matrix cores, then the
//   neighbour block from U, V, B, Bh (see the kernel).
// Arithmetic is float64, except the Jacobian's final two-term assembly, which
// runs at the output precision (see k_jacobian).
#pragma once

#include "soap_internal.h"

#include <algorithm>

namespace soap {
namespace dev {

// Output stores are plain (write-back) stores: on this chip non-temporal
// stores of the neighbour blocks' partial-line runs write back at about half
// the bandwidth.
template <typename T> __device__ __forceinline__ void store_out(T *p, double v) { *p = (T)v; }
__device__ __forceinline__ void store_out(float *p, float v) { *p = v; }

// (value, companion) pairs in LDS at the precision T
template <typename T> struct Pair;
template <> struct Pair<double> {
    using type = double2;
    static __device__ __forceinline__ double2 make(double a, double b) { return make_double2(a, b); }
};
template <> struct Pair<float> {
    using type = float2;
    static __device__ __forceinline__ float2 make(double a, double b) { return make_float2((float)a, (float)b); }
};

// four consecutive LDS values (16-byte aligned) as float64
__device__ __forceinline__ void load4(const double *p, double &a, double &b, double &c, double &d) {
    const double2 u = *(const double2 *)p, v = *(const double2 *)(p + 2);
    a = u.x;
    b = u.y;
    c = v.x;
    d = v.y;
}
__device__ __forceinline__ void load4(const float *p, double &a, double &b, double &c, double &d) {
    const float4 u = *(const float4 *)p;
    a = u.x;
    b = u.y;
    c = u.z;
    d = u.w;
}

// floor(x / d) for 0 <= x < 2^22 with inv = 1/d correctly rounded: the
// relative error of (x + 1/2) * inv stays below 1/(2d) of the gap to the
// next integer
__device__ __forceinline__ int qdiv(int x, float inv) { return (int)(((float)x + 0.5f) * inv); }

// Read-only basis tables seen through the constant address space: a
// wave-uniform read then compiles to a scalar load from the scalar cache.
// Through a generic pointer, which may alias the kernel's own LDS and
// global stores, it stays a per-lane vector load on the latency path.
typedef const __attribute__((address_space(4))) double *cdptr;
__device__ __forceinline__ cdptr as_const(const double *p) { return (cdptr)p; }

// ---------------------------------------------------------------------------
// Double-double arithmetic (unevaluated sums hi + lo) for the compensated GTO
// radial sums: Knuth's two-sum, the fused multiply-add two-product.  Device
// code is compiled with multiply-add contraction on; fused into the sums, a
// product's rounding no longer matches the remainder taken from it, and the
// compensated sums lose more than they gain.  Every function here, and every
// block that uses them, turns contraction off.
// ---------------------------------------------------------------------------
struct dd {
    double hi, lo;
};
__device__ __forceinline__ dd dd_fast_sum(double a, double b) { // |a| >= |b|
#pragma clang fp contract(off)
    const double s = a + b;
    return dd{s, b - (s - a)};
}
__device__ __forceinline__ dd dd_two_sum(double a, double b) {
#pragma clang fp contract(off)
    const double s = a + b, bb = s - a;
    return dd{s, (a - (s - bb)) + (b - bb)};
}
__device__ __forceinline__ dd dd_add(dd a, dd b) {
#pragma clang fp contract(off)
    dd s = dd_two_sum(a.hi, b.hi);
    const dd t = dd_two_sum(a.lo, b.lo);
    s.lo += t.hi;
    s = dd_fast_sum(s.hi, s.lo);
    s.lo += t.lo;
    return dd_fast_sum(s.hi, s.lo);
}
__device__ __forceinline__ dd dd_mul(dd a, dd b) {
#pragma clang fp contract(off)
    const double p = a.hi * b.hi;
    double e = fma(a.hi, b.hi, -p);
    e = fma(a.hi, b.lo, e);
    e = fma(a.lo, b.hi, e);
    return dd_fast_sum(p, e);
}
// exp(-x) for x >= 0 to ~1e-30 relative: x = k ln 2 + t with ln 2 split in
// three parts (the first with 32 significant bits, so k times it is exact),
// then exp(-t) = (exp(-t / 256))^256, the inner factor by its Taylor series
// to degree 9 (|t| / 256 < 1.4e-3: remainder below 1e-35) and eight squarings.
__device__ __forceinline__ dd dd_exp_neg(dd x) {
#pragma clang fp contract(off)
    if (x.hi > 700.0) return dd{0.0, 0.0};
    constexpr double L1 = 0.6931471803691238, L2 = 1.9082149292705877e-10, L3 = 1.1612227229362532e-26;
    // 1/j!, j = 0..9, as (hi, lo)
    constexpr double FH[10] = {1.0, 1.0, 0.5, 0.16666666666666666, 0.041666666666666664, 0.008333333333333333,
                               0.001388888888888889, 0.0001984126984126984, 2.48015873015873e-05,
                               2.7557319223985893e-06};
    constexpr double FL[10] = {0.0, 0.0, 0.0, 9.25185853854297e-18, 2.3129646346357427e-18, 1.1564823173178714e-19,
                               -5.300543954373577e-20, 1.7209558293420705e-22, 2.1511947866775882e-23,
                               -1.858393274046472e-22};
    const double k = rint(x.hi * 1.4426950408889634);
    const double t1 = fma(-k, L1, x.hi); // exact
    const double p2 = k * L2, e2 = fma(k, L2, -p2);
    dd t = dd_add(dd{t1, x.lo}, dd{-p2, -e2});
    t.lo -= k * L3;
    const dd y{-t.hi * (1.0 / 256.0), -t.lo * (1.0 / 256.0)};
    dd p{FH[9], FL[9]};
#pragma unroll
    for (int j = 8; j >= 0; --j) p = dd_add(dd_mul(p, y), dd{FH[j], FL[j]});
#pragma unroll
    for (int j = 0; j < 8; ++j) p = dd_mul(p, p);
    const int ki = (int)k;
    return dd{ldexp(p.hi, -ki), ldexp(p.lo, -ki)};
}

// e^{-x} for x >= 0 to about half an ulp, by the table-driven reduction of
// Tang (ACM TOMS 15(2), 1989): -x = (64 k + j) ln2/64 + r with |r| <=
// ln2/128, e^{-x} = 2^k 2^{j/64} e^r, 2^{j/64} as (value, remainder) pairs
// t2[2j], t2[2j+1] (in LDS) and e^r - 1 = r + r^2 (1/2 + r/6) + r^4/24 (1 +
// r/5 + r^2/30), whose first omitted term is below 3e-20.  The polynomial
// takes its constants only as multiplicands or inline constants, so no
// constant is an accumulator that has to be copied first.  Branch-free;
// below e^-745 the result flushes to zero in the final ldexp (arguments past
// 746 are clamped there first, which keeps the integer part in range).
__device__ __forceinline__ double exp_neg_tab(double x, const double *__restrict__ t2) {
#pragma clang fp contract(off)
    const double y = -__builtin_fmin(x, 746.0);
    const double nn = __builtin_rint(y * 92.33248261689366); // 64 / ln 2
    const int k = (int)nn;
    double r = __builtin_fma(nn, -0.010830424696249145, y); // ln 2 / 64: leading part
    r = __builtin_fma(nn, -3.623510646634843e-19, r);       // and the rest
    const double2 tj = *(const double2 *)(t2 + 2 * (k & 63));
    const double r2 = r * r;
    const double A = __builtin_fma(r, 0.16666666666666666, 0.5);
    double t = __builtin_fma(r, 0.2, 1.0);
    t = __builtin_fma(r2, 0.03333333333333333, t);
    const double r4c = r2 * (r2 * 0.041666666666666664);
    double p = __builtin_fma(r2, A, r);
    p = __builtin_fma(r4c, t, p);
    return __builtin_ldexp(tj.x + __builtin_fma(tj.x, p, tj.y), k >> 6);
}

// ---------------------------------------------------------------------------
// Real solid harmonics of one column m without gradients and without
// divisions.  With (C_m + i S_m) = (x + i y)^m, R_m = 1, R_{m+1} = (2m+1) z,
//   R_l = (2l-1) z R_{l-1} - (l+m-1)(l-m-1) r^2 R_{l-2},
// the associated Legendre part is Q_l^m = (2m-1)!! R_l / (l-m)!, so
//   S_l,m = Nt_lm R_l C_m, S_l,-m = Nt_lm R_l S_m, Nt_lm = N_lm (2m-1)!! / (l-m)!.
// Stores l in [l_lo, l_hi) at Y[(l^2 + l +- m - lm_base) * ls].
// ---------------------------------------------------------------------------
template <typename YT, typename NtPtr = const double *__restrict__>
__device__ __forceinline__ void sh_col_y(int m, int l_lo, int l_hi, double x, double y, double z, NtPtr Nt, int ldN,
                                         YT *__restrict__ Y, int ls, int lm_base) {
    const double r2 = x * x + y * y + z * z;
    double c = 1.0, s = 0.0;
    for (int k = 0; k < m; ++k) {
        const double cn = x * c - y * s;
        s = x * s + y * c;
        c = cn;
    }
    double R1 = 0.0, R = 1.0; // R_{l-1}, R_l
    for (int l = m; l < l_hi; ++l) {
        if (l > m) {
            const double a = (double)(2 * l - 1), b = (double)((l + m - 1) * (l - m - 1));
            const double Rn = a * z * R - b * r2 * R1;
            R1 = R;
            R = Rn;
        }
        if (l >= l_lo) {
            const double v = Nt[l * ldN + m] * R;
            const int o = l * l + l - lm_base;
            if (m == 0) {
                Y[o * ls] = (YT)v;
            } else {
                Y[(o + m) * ls] = (YT)(v * c);
                Y[(o - m) * ls] = (YT)(v * s);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Scaled modified spherical Bessel functions ii_l(x) = e^-x i_l(x), l = 0..Lt
// (the radial integral of the polynomial basis, Eq. bessel-integral).
// x >= Lt(Lt+1)/6.9: upward recurrence from the closed forms of ii_0, ii_1
//   (error growth bounded by about e^{Lt(Lt+1)/x} <= 1e3);
// otherwise Miller's method: the downward recurrence
//   i_{l-1} = i_{l+1} + (2l+1)/x i_l
// started at N = Lt + 12 + floor(x) from (f_{N+1}, f_N) = (0, 1), where i_l
// is the dominant solution, then normalised by the closed form
// ii_0 = -expm1(-2x) / (2x) (relative error <= 1.3e-15 against 40-digit
// values for Lt <= 15 over that x range).  The running pair is rescaled by
// 1e-150 above 1e150 before the stored orders, and the stored orders by
// 1e-200 should they pass 1e200 (only for x far below 1e-6).
// ---------------------------------------------------------------------------
// Writes ii_l(x) * g for l = 0..Lt to t[0..Lt] (LDS).
__device__ __forceinline__ void bessel_scaled_lds(int Lt, double x, double g, double *t) {
    if (x == 0.0) {
        t[0] = g;
        for (int k = 1; k <= Lt; ++k) t[k] = 0.0;
        return;
    }
    const double ix = 1.0 / x;
    if (x * 6.9 >= (double)(Lt * (Lt + 1))) {
        const double em = exp(-2.0 * x);
        double a = 0.5 * (1.0 - em) * ix;              // ii_0
        double b = 0.5 * (1.0 + em) * ix - a * ix;     // ii_1
        t[0] = g * a;
        if (Lt >= 1) t[1] = g * b;
        for (int k = 1; k < Lt; ++k) {
            const double c = a - (double)(2 * k + 1) * ix * b;
            t[k + 1] = g * c;
            a = b;
            b = c;
        }
    } else {
        const int N = Lt + 12 + (int)x;
        double a = 0.0, b = 1.0; // f_{k+1}, f_k
        for (int k = N; k > Lt; --k) {
            const double c = a + (double)(2 * k + 1) * ix * b;
            a = b;
            b = c;
            if (fabs(b) > 1e150) {
                a *= 1e-150;
                b *= 1e-150;
            }
        }
        t[Lt] = b;
        for (int k = Lt; k > 0; --k) {
            const double c = a + (double)(2 * k + 1) * ix * b; // f_{k-1}
            t[k - 1] = c;
            a = b;
            b = c;
            if (fabs(b) > 1e200) {
                for (int j = k - 1; j <= Lt; ++j) t[j] *= 1e-200;
                a *= 1e-200;
                b *= 1e-200;
            }
        }
        const double sc = g * (-expm1(-2.0 * x) * 0.5 * ix) / b; // b = f_0
        for (int k = 0; k <= Lt; ++k) t[k] *= sc;
    }
}

// ---------------------------------------------------------------------------
// LDS layout helpers.  Every region starts on a 16-byte boundary.
// ---------------------------------------------------------------------------
__host__ __device__ __forceinline__ size_t even(size_t nd) { return (nd + 1) & ~(size_t)1; }

struct Carver {
    double *base;
    size_t off = 0;
    __device__ __forceinline__ double *take(size_t nd) {
        double *p = base + off;
        off += even(nd);
        return p;
    }
};

// Neighbour rows are prefetched into LDS in blocks of row_block(EC) edges.
__host__ __device__ __forceinline__ int row_block(int EC) { return EC >= 128 ? EC : EC * (128 / EC); }

// Basis tables copied to LDS once per workgroup (for l in [lg0, lg1)), so
// that no global load sits on the per-edge path: with the chip's store
// traffic in flight, global load latency runs to microseconds.
struct Tables {
    const double *Kl;      // K_l = pi sqrt(8/(2l+1)), l < 16
    const double2 *bcp;    // GTO: [k][n][lc] = (betaC, -2 betaC a') of B_nl = sum_k betaC_nk e^{-a'_kl r^2}
    const double *aprime;  // GTO: [k][lc]
    const double *WN, *B0; // polynomial, Laplace form: [n][n+3][4] Chebyshev coefficients (stage_edges); B_n0(0) [n]
    const double2 *bcdd;   // GTO, compensated: [k][n][lc] = (betaC, its remainder)
    const double2 *apdd;   // GTO, compensated: [k][lc] = (a', its remainder)
    const double *Nt;      // [ldN][ldN] N_lm (2m-1)!! / (l-m)!, for sh_col_y
    const double2 *gcoef;  // [(l, m >= 0)][2]: (cA, cB), (cC, l | m << 8), see stage_edges
};

__host__ __device__ __forceinline__ int grad_pairs(int lmax) { return (lmax + 1) * (lmax + 2) / 2; }

__host__ __device__ __forceinline__ size_t table_doubles(const Params &P, int lgc) {
    const size_t ldN = (size_t)P.lmax + 2, n = (size_t)P.n;
    size_t d = 16 + even(ldN * ldN) + 4 * (size_t)grad_pairs(P.lmax);
    if (P.rbf == 0) d += 2 * (size_t)lgc * n * n + even((size_t)lgc * n);
    else if (P.rbf == 2) d += 4 * n * (n + 3) + even(n);
    else if (P.rbf == 3) d += 2 * (size_t)lgc * n * n + 2 * (size_t)lgc * n;
    return d; // the polynomial quadrature reads its radial factors from k_radial: no tables
}

// RBF: the radial basis fixed at compile time (0 GTO), or -1 to read it from P
template <int NT = 0, int LWT = 0, int RBF = -1>
__device__ __forceinline__ void load_tables(const Params &P, Carver &cv, Tables &T, int lg0, int lg1) {
    const int n = NT ? NT : P.n, lmax = LWT ? LWT - 1 : P.lmax;
    const int ldN = lmax + 2, lgc = lg1 - lg0, tid = threadIdx.x, bs = blockDim.x;
    // every pointer is assigned on every path, so the struct stays in
    // registers and the compiler keeps LDS (ds_*) addressing for it
    double *Kl = cv.take(16);
    double *Ntl = cv.take((size_t)ldN * ldN);
    double *gc = cv.take(4 * (size_t)grad_pairs(lmax));
    const int rbf = RBF >= 0 ? RBF : P.rbf;
    if (tid < 16) Kl[tid] = M_PI * sqrt(8.0 / (double)(2 * tid + 1));
    // (betaC, betaCa) pairs | G | WN | (betaC, remainder) pairs, then aprime | rq | B0 | (a', remainder) pairs
    const size_t szA = rbf == 0 ? 2 * (size_t)lgc * n * n
                                : (rbf == 1 ? 0 : (rbf == 2 ? 4 * (size_t)n * (n + 3) : 2 * (size_t)lgc * n * n));
    const size_t szB = rbf == 0 ? (size_t)lgc * n : (rbf == 1 ? 0 : (rbf == 2 ? (size_t)n : 2 * (size_t)lgc * n));
    double *A = cv.take(szA), *B = cv.take(szB);
    for (int k = tid; k < ldN * ldN; k += bs) Ntl[k] = P.Nt[k];
    for (int k = tid; k < 4 * grad_pairs(lmax); k += bs) gc[k] = P.gcoef[k];
    if (rbf == 0) {
        // global [l][n][k] -> LDS [k][n][lc]; global [l][k] -> LDS [k][lc]
        const size_t o = (size_t)lg0 * n * n;
        for (int s = tid; s < (int)(szA / 2); s += bs) {
            const int lc = s / (n * n), r = s - lc * n * n, a = r / n, k = r - a * n;
            const int d = (k * n + a) * lgc + lc;
            A[2 * d] = P.betaC[o + s];
            A[2 * d + 1] = P.betaCa[o + s];
        }
        for (int s = tid; s < (int)szB; s += bs) {
            const int lc = s / n, k = s - lc * n;
            B[k * lgc + lc] = P.aprime[(size_t)lg0 * n + s];
        }
    } else if (rbf == 3) {
        // global [l][n][k] -> LDS [k][n][lc] pairs; global [l][k] -> LDS [k][lc] pairs
        const size_t o = (size_t)lg0 * n * n;
        for (int s = tid; s < (int)(szA / 2); s += bs) {
            const int lc = s / (n * n), r = s - lc * n * n, a = r / n, k = r - a * n;
            const int d = (k * n + a) * lgc + lc;
            A[2 * d] = P.betaC[o + s];
            A[2 * d + 1] = P.betaC_lo[o + s];
        }
        for (int s = tid; s < (int)(szB / 2); s += bs) {
            const int lc = s / n, k = s - lc * n;
            B[2 * (k * lgc + lc)] = P.aprime[(size_t)lg0 * n + s];
            B[2 * (k * lgc + lc) + 1] = P.aprime_lo[(size_t)lg0 * n + s];
        }
    } else if (rbf == 2) {
        // a neighbour at distance 0 adds the on-site term: B_n0 S_00 = c0_n
        for (int k = tid; k < (int)szA; k += bs) A[k] = P.WN[k];
        for (int k = tid; k < (int)szB; k += bs) B[k] = P.c0[k] * sqrt(4.0 * M_PI);
    }
    T.Kl = Kl;
    T.Nt = Ntl;
    T.gcoef = (const double2 *)gc;
    T.bcp = (const double2 *)A;
    T.WN = A;
    T.aprime = B;
    T.B0 = B;
    T.bcdd = (const double2 *)A;
    T.apdd = (const double2 *)B;
}

// X scratch per edge: GTO exponentials n * lgc; none for the polynomial
// quadrature (its radial factors come from k_radial); Laplace form: the four
// l-independent values P_j per n, 4 n; compensated GTO: the exponentials in
// double-double, 2 n * lgc
__host__ __device__ __forceinline__ size_t stage_x_doubles(const Params &P, int lgc, int lg1) {
    (void)lg1;
    return P.rbf == 0 ? (size_t)P.n * lgc : (P.rbf == 1 ? 0 : (P.rbf == 2 ? 4 * (size_t)P.n : 2 * (size_t)P.n * lgc));
}

// Synchronisation inside one wave: LDS writes become visible to the other
// lanes and the compiler keeps LDS accesses on their side of the point.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

// Workgroup barrier ordering LDS only.  __syncthreads() also fences global
// memory, which makes every wave wait for all of its outstanding output
// stores; nothing here reads another wave's global writes, so the output
// stream keeps flowing across the barrier.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// ---------------------------------------------------------------------------
// Per-tile edge staging (one wave, nb edges), shared by both kernels, for
// l in [lg0, lg1).
//   YY: harmonics, element (edge e, component c, lm) at
//       e es + c cs + (lm - lmY0) ls; component 0 = S, 1..3 = dS/dx_d (GRAD).
//       Degrees from lgY0 = lg0 - 1 (GRAD and lg0 > 0) or lg0 are stored.
//   BB[e][n][lc] = K (B_nl, Bh_nl), K = K_l if scaleK else 1, stored at precision BT
//   X: GTO exponentials [e][k][lc], the polynomial table [e][q][0..lg1], or
//      the Laplace form's P_j [e][n][j]
// Phase 1 runs the harmonic columns (edge, m), then the radial scratch;
// phase 2 the gradients, then the radial factors.  Each gradient component
// is at most two degree l-1 harmonics: with H_l^m = (x + iy)^m Q_l^m (so
// S_l,m = N_lm Re H, S_l,-m = N_lm Im H),
//   d/dz H_l^m = (l+m) H_{l-1}^m,  (d/dx + i d/dy) H_l^m = -H_{l-1}^{m+1},
//   (d/dx - i d/dy) H_l^m = (l+m)(l+m-1) H_{l-1}^{m-1}.
// Per (l, m >= 0), with S' = S_{l-1,.} and gcoef = (cA, cB, cC):
//   m = 0:  grad S_l0 = (-cA S'_1, -cA S'_-1, cC S'_0)
//   m > 0:  grad S_lm  = (-cA S'_{m+1} + cB S'_{m-1}, -cA S'_{-(m+1)} - cB S'_{-(m-1)}, cC S'_m)
//           grad S_l-m = (-cA S'_{-(m+1)} + cB S'_{-(m-1)}, cA S'_{m+1} + cB S'_{m-1}, cC S'_-m)
// (S'_k = 0 for |k| > l-1, S'_-0 = 0).  A zero-length edge gets a zero gradient.
// ---------------------------------------------------------------------------
struct YLayout {
    int es, cs, ls, lmY0;
};

template <bool GRAD, typename BT = double, int NT = 0, int LWT = 0, typename YT = double, int RBF = -1>
__device__ __forceinline__ void stage_edges(const Params &P, const Tables &T, YT *__restrict__ YY, YLayout yl,
                                            typename Pair<BT>::type *__restrict__ BB, double *__restrict__ X,
                                            const double *__restrict__ geo, int nb, int lane, int lg0, int lg1,
                                            bool scaleK, int64_t r0) {
    const int n = NT ? NT : P.n, ldN = (LWT ? LWT - 1 : P.lmax) + 2, lgc = lg1 - lg0, nlc = n * lgc;
    const int lgY0 = (GRAD && lg0 > 0) ? lg0 - 1 : lg0;
    const float inv_lg1 = 1.0f / (float)lg1, inv_nlc = 1.0f / (float)nlc, inv_lgc = 1.0f / (float)lgc;
    const int rbf = RBF >= 0 ? RBF : P.rbf;
    // phase 1: harmonic columns (edge, m), then the radial scratch (two
    // independent exponentials per lane trip)
    for (int it = lane; it < nb * lg1; it += 64) {
        const int e = qdiv(it, inv_lg1), m = it - e * lg1;
        const double *g = geo + 4 * e;
        sh_col_y(m, m > lgY0 ? m : lgY0, lg1, g[0], g[1], g[2], T.Nt, ldN, YY + e * yl.es, yl.ls, yl.lmY0);
    }
    if constexpr (RBF == 3) {
#pragma clang fp contract(off)
        // compensated GTO: x = a' r^2 in double-double (a' as hi + remainder), then exp(-x)
        for (int it = lane; it < nb * nlc; it += 64) {
            const int e = qdiv(it, inv_nlc), t = it - e * nlc; // t = k lgc + lc
            const double r = geo[4 * e + 3], s2r = r * r;
            const double2 ap = T.apdd[t];
            const double xh = ap.x * s2r;
            const dd v = dd_exp_neg(dd_fast_sum(xh, fma(ap.x, s2r, -xh) + ap.y * s2r));
            X[2 * it] = v.hi;
            X[2 * it + 1] = v.lo;
        }
    } else if (rbf == 0) {
        const int nx = nb * nlc;
        for (int it = lane; it < nx; it += 128) {
            const int i2 = it + 64 < nx ? it + 64 : it;
            const int e1 = qdiv(it, inv_nlc), e2 = qdiv(i2, inv_nlc);
            const double r1 = geo[4 * e1 + 3], r2 = geo[4 * e2 + 3];
            const double v1 = exp(-T.aprime[it - e1 * nlc] * r1 * r1), v2 = exp(-T.aprime[i2 - e2 * nlc] * r2 * r2);
            X[it] = v1;
            X[i2] = v2;
        }
    } else if (rbf == 2) {
        // the Laplace form's P_j(u) = d^j/du^j sum_k WN_nk u^(k+2), u = r_cut - r, at [e][n][j]
        // from their Chebyshev series in t = 2u/r_cut - 1 (Clenshaw's recurrence)
        const int per = 4 * n;
        const float inv_per = 1.0f / (float)per;
        for (int it = lane; it < nb * per; it += 64) {
            const int e = qdiv(it, inv_per), q = it - e * per;
            const double r = geo[4 * e + 3];
            const double tt = (P.rc - r) * P.inv_rc2 - 1.0, t2 = tt + tt;
            const double *ch = T.WN + (size_t)(q >> 2) * (n + 3) * 4 + (q & 3);
            double b1 = 0.0, b2 = 0.0;
            for (int i = n + 2; i >= 1; --i) {
                const double nb1 = t2 * b1 - b2 + ch[4 * i];
                b2 = b1;
                b1 = nb1;
            }
            X[it] = tt * b1 - b2 + ch[0];
        }
    }
    wave_sync();
    // phase 2: gradients (edge, (l, m >= 0)), then the radial factors (edge, n, lc)
    if (GRAD) {
        const int t0 = lg0 * (lg0 + 1) / 2, Tg = lg1 * (lg1 + 1) / 2 - t0;
        const float inv_T = 1.0f / (float)Tg;
        for (int it = lane; it < nb * Tg; it += 64) {
            const int e = qdiv(it, inv_T), t = it - e * Tg + t0;
            const double2 c01 = T.gcoef[2 * t], c2p = T.gcoef[2 * t + 1];
            const int lm = (int)c2p.y, l = lm & 0xff, m = lm >> 8;
            YT *Y = YY + e * yl.es;
            const int lp = l > 0 ? l - 1 : 0, c0 = lp * lp + lp - yl.lmY0;
            const bool live = geo[4 * e + 3] != 0.0 && l > 0;
            // S'_k for k in {m+1, -(m+1), m-1, -(m-1), m, -m}, clamped into degree l-1
            auto sp = [&](int k) -> double {
                const int kc = k < -lp ? -lp : (k > lp ? lp : k);
                const double v = (double)Y[(c0 + kc) * yl.ls];
                return (live && k >= -lp && k <= lp) ? v : 0.0;
            };
            const double cA = c01.x, cB = c01.y, cC = c2p.x;
            YT *Dx = Y + yl.cs, *Dy = Y + 2 * yl.cs, *Dz = Y + 3 * yl.cs;
            const int o = l * l + l - yl.lmY0;
            if (m == 0) {
                Dx[o * yl.ls] = (YT)(-cA * sp(1));
                Dy[o * yl.ls] = (YT)(-cA * sp(-1));
                Dz[o * yl.ls] = (YT)(cC * sp(0));
            } else {
                const double pp = sp(m + 1), pn = sp(-(m + 1)), qp = sp(m - 1), qn = m > 1 ? sp(-(m - 1)) : 0.0;
                const double zp = sp(m), zn = sp(-m);
                Dx[(o + m) * yl.ls] = (YT)(-cA * pp + cB * qp);
                Dy[(o + m) * yl.ls] = (YT)(-cA * pn - cB * qn);
                Dz[(o + m) * yl.ls] = (YT)(cC * zp);
                Dx[(o - m) * yl.ls] = (YT)(-cA * pn + cB * qn);
                Dy[(o - m) * yl.ls] = (YT)(cA * pp + cB * qp);
                Dz[(o - m) * yl.ls] = (YT)(cC * zn);
            }
        }
    }
    const int nd = nb * nlc;
    if constexpr (RBF == 3) {
#pragma clang fp contract(off)
        // compensated dot products (two-product and two-sum per term, the
        // errors summed apart): B = sum_k betaC e_k, Bh = -2 sum_k (betaC a') e_k
        // with betaC a' formed in double-double (no second table: the LDS
        // then holds what the plain GTO path holds)
        for (int it = lane; it < nd; it += 64) {
            const int e = qdiv(it, inv_nlc), t = it - e * nlc, lc = t - qdiv(t, inv_lgc) * lgc;
            const double2 *bc = T.bcdd + t; // [k][n][lc]
            const double2 *apk = T.apdd + lc; // [k][lc]
            const double *E = X + 2 * ((size_t)e * nlc + lc);
            double sb = 0.0, cb = 0.0, sh = 0.0, ch = 0.0;
            for (int k = 0; k < n; ++k) {
                const double2 c = bc[(size_t)k * nlc], ap = apk[k * lgc];
                const dd m = dd_mul(dd{c.x, c.y}, dd{ap.x, ap.y});
                const double eh = E[2 * k * lgc], el = E[2 * k * lgc + 1];
                const double pb = c.x * eh, ph = m.hi * eh;
                const dd tb = dd_two_sum(sb, pb), th = dd_two_sum(sh, ph);
                sb = tb.hi;
                sh = th.hi;
                cb += (fma(c.x, eh, -pb) + tb.lo) + (c.x * el + c.y * eh);
                ch += (fma(m.hi, eh, -ph) + th.lo) + (m.hi * el + m.lo * eh);
            }
            const double K = scaleK ? T.Kl[lg0 + lc] : 1.0;
            BB[it] = Pair<BT>::make(K * (sb + cb), -2.0 * K * (sh + ch));
        }
    } else if (rbf == 0) {
        for (int it = lane; it < nd; it += 128) {
            const int i2 = it + 64 < nd ? it + 64 : it;
            const int e1 = qdiv(it, inv_nlc), t1 = it - e1 * nlc, l1 = t1 - qdiv(t1, inv_lgc) * lgc;
            const int e2 = qdiv(i2, inv_nlc), t2 = i2 - e2 * nlc, l2 = t2 - qdiv(t2, inv_lgc) * lgc;
            const double2 *bc1 = T.bcp + t1, *bc2 = T.bcp + t2; // [k][n][lc]: t = a lgc + lc
            const double *E1 = X + (size_t)e1 * nlc + l1, *E2 = X + (size_t)e2 * nlc + l2;
            double b1 = 0.0, h1 = 0.0, b2 = 0.0, h2 = 0.0;
#pragma unroll 2
            for (int k = 0; k < n; ++k) {
                const double2 c1 = bc1[k * nlc], c2 = bc2[k * nlc];
                const double v1 = E1[k * lgc], v2 = E2[k * lgc];
                b1 += c1.x * v1;
                h1 += c1.y * v1;
                b2 += c2.x * v2;
                h2 += c2.y * v2;
            }
            const double K1 = scaleK ? T.Kl[lg0 + l1] : 1.0, K2 = scaleK ? T.Kl[lg0 + l2] : 1.0;
            BB[it] = Pair<BT>::make(K1 * b1, K1 * h1);
            BB[i2] = Pair<BT>::make(K2 * b2, K2 * h2);
        }
    } else if (rbf == 2) {
        // Laplace form, u = r_cut - r, k = 1..n: the bracket of Eq. (poly-coefficients) summed over k
        // is f = P_0 (1 - l(l+1) h/2) - s^2/r P_1 + s^2/2 P_2 with h = s^2/r^2 and P_j = d^j/du^j
        // sum_k WN_nk u^(k+2) (phase 1); Eq. (poly-radial-derivative) likewise is
        // f' = l(l+1) h/r P_0 + ((l(l+1)+2) h/2 - 1) P_1 + s^2/r P_2 - s^2/2 P_3.
        // s2, hs2 and inv_rc2 come in as kernel arguments: computed here, the
        // compiler hoists them into vector registers held through the kernel
        const double s2 = P.s2, hs2 = P.hs2;
        for (int it = lane; it < nd; it += 64) {
            const int e = qdiv(it, inv_nlc), t = it - e * nlc, a = qdiv(t, inv_lgc), l = lg0 + t - a * lgc;
            const double r = geo[4 * e + 3];
            double b, bh;
            if (r == 0.0) {
                b = (l == 0) ? T.B0[a] : 0.0;
                bh = 0.0;
            } else {
                const double *ps = X + 4 * ((size_t)e * n + a);
                const double p0 = ps[0], p1 = ps[1], p2 = ps[2], p3 = ps[3];
                const double ir = 1.0 / r, ll = (double)(l * (l + 1)), h = s2 * ir * ir;
                const double f = p0 * (1.0 - 0.5 * ll * h) - s2 * ir * p1 + hs2 * p2;
                const double fp = ll * h * ir * p0 + (0.5 * (ll + 2.0) * h - 1.0) * p1 + s2 * ir * p2 - hs2 * p3;
                double rl = 1.0;
                for (int k = 0; k < l; ++k) rl *= ir;
                b = rl * f;
                bh = rl * ir * (fp - (double)l * f * ir);
            }
            const double K = scaleK ? T.Kl[l] : 1.0;
            BB[it] = Pair<BT>::make(K * b, K * bh);
        }
    } else {
        // polynomial quadrature: the factors k_radial left for this call's edges, [edge][n][l]
        const int lwa = P.lmax + 1;
        const double2 *rad = P.rad + (r0 - P.rad_e0) * (size_t)n * lwa + lg0;
        for (int it = lane; it < nd; it += 64) {
            const int e = qdiv(it, inv_nlc), t = it - e * nlc, a = qdiv(t, inv_lgc), lc = t - a * lgc;
            const double2 v = rad[((size_t)e * n + a) * lwa + lc];
            const double K = scaleK ? T.Kl[lg0 + lc] : 1.0;
            BB[it] = Pair<BT>::make(K * v.x, K * v.y);
        }
    }
    wave_sync();
}

// Prefetch the rows [r0, r0+cnt) of the center: edge vectors r_j - r_i in
// float64 (exact for float32 inputs), |r|, species.
template <typename PosT>
__device__ __forceinline__ void load_rows(double *geo, int *sp, const PosT *__restrict__ pos,
                                          const uint8_t *__restrict__ spec, const int32_t *__restrict__ cols,
                                          int64_t r0, int cnt, double3 pi) {
    for (int t = threadIdx.x; t < cnt; t += blockDim.x) {
        const int64_t j = cols[r0 + t];
        const double x = (double)pos[3 * j] - pi.x, y = (double)pos[3 * j + 1] - pi.y,
                     z = (double)pos[3 * j + 2] - pi.z;
        geo[4 * t] = x;
        geo[4 * t + 1] = y;
        geo[4 * t + 2] = z;
        geo[4 * t + 3] = sqrt(x * x + y * y + z * z);
        sp[t] = spec[j];
    }
}

// ---------------------------------------------------------------------------
// k_radial: the polynomial basis's radial factors of every edge of a range of
// centers, evaluated once per call and read by every density and Jacobian
// kernel (quadrature form of the radial integral, Sec. 2.3: the sums over the
// basis and over the nodes swapped, G[n][q] = w_q r_q^2 g_n(r_q) 4 pi):
//   B_nl  = r^-l sum_q G_nq ii_l(x_q) g_q,
//   Bh_nl = (1/r) dB_nl/dr
//         = r^-l (1/r) sigma^-2 sum_q G_nq (r_q ii_{l+1}(x_q) - r ii_l(x_q)) g_q,
// x_q = r r_q / sigma^2, g_q = exp(-(r_q - r)^2 / (2 sigma^2)) (ii_l the
// exponentially scaled modified spherical Bessel function, the derivative
// from i_l' = i_{l+1} + (l/x) i_l), and for an edge of length 0 only the
// l = 0 factor, B_n0(0).  Output [edge - e_base][n][l] = (B_nl, Bh_nl) for
// l <= l_max, unscaled by K_l.
// A workgroup takes a block of cb consecutive centers, whose edges are
// contiguous; its waves take four edges at a time, round-robin, each lane
// finding its edge's center in the block's row offsets.  Per four edges the
// Bessel values of (edge, node) for 16 nodes at once go to the wave's LDS
// slab, then lane = (edge, l) accumulates all NA radial indices over those
// nodes (G broadcast from LDS).  The node sums run in node order, as in the
// in-kernel evaluation.
// ---------------------------------------------------------------------------
constexpr int NWR = 4, BSR = 64 * NWR;
constexpr int RAD_EC = 4, RAD_QC = 16; // edges per wave pass; nodes per Bessel slab
constexpr int RAD_CB_MAX = 256;        // centers per workgroup block

__host__ __device__ __forceinline__ int radial_qpad(int Q) { return (Q + RAD_QC - 1) / RAD_QC * RAD_QC; }
// LDS doubles of k_radial: the block's row offsets [RAD_CB_MAX + 1], G [NA][Qp], r_q [Qp], and
// per wave the Bessel slab [64][l_max + 2]
__host__ __device__ __forceinline__ size_t radial_lds_doubles(const Params &P, int na) {
    const size_t qp = (size_t)radial_qpad(P.Q);
    return even(RAD_CB_MAX + 1) + even((size_t)na * qp) + even(qp) + NWR * even(64 * ((size_t)P.lmax + 2));
}

template <typename PosT, int NA>
__global__ __launch_bounds__(BSR) void k_radial(Params P, Rows R, const PosT *__restrict__ pos, int64_t e_base,
                                                int cb, double2 *__restrict__ out) {
    extern __shared__ __align__(16) double smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = P.n, Q = P.Q, Qp = radial_qpad(Q), lw = P.lmax + 1, tw = lw + 1;
    Carver cv{smem};
    int64_t *rp = (int64_t *)cv.take(RAD_CB_MAX + 1);
    double *G = cv.take((size_t)NA * Qp);
    double *rq = cv.take((size_t)Qp);
    double *slab = cv.take(0) + (size_t)wave * even(64 * (size_t)tw);
    for (int k = tid; k < NA * Qp; k += BSR) {
        const int a = k / Qp, q = k - a * Qp;
        G[k] = (a < n && q < Q) ? P.G[(size_t)a * Q + q] : 0.0;
    }
    for (int k = tid; k < Qp; k += BSR) rq[k] = k < Q ? P.rq[k] : 0.0;
    const int es = lane >> 4, sub = lane & 15; // edge slot; node (Bessel phase) or l (sum phase)
    double *mine = slab + (size_t)lane * tw;          // this lane's (edge, node) Bessel row
    const double *col = slab + (size_t)es * RAD_QC * tw; // this lane's edge, all 16 nodes
    const int l = sub < lw ? sub : lw - 1;
    for (int64_t c0 = (int64_t)blockIdx.x * cb; c0 < R.nc; c0 += (int64_t)gridDim.x * cb) {
        const int ncb = (int)((R.nc - c0) < cb ? (R.nc - c0) : cb);
        __syncthreads(); // the tables; the previous block's readers of rp
        for (int t = tid; t <= ncb; t += BSR) rp[t] = R.row_ptr[c0 + t];
        __syncthreads();
        const int64_t E1 = rp[ncb];
        for (int64_t eb = rp[0] + (int64_t)RAD_EC * wave; eb < E1; eb += (int64_t)RAD_EC * NWR) {
            const int64_t e = eb + es;
            const bool live = e < E1;
            double r = 0.0;
            if (live) {
                int lo = 0, hi = ncb - 1; // the center of e: the last k with rp[k] <= e
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (rp[mid] <= e) lo = mid;
                    else hi = mid - 1;
                }
                const int64_t ci = c0 + lo;
                const int64_t i = R.centers ? (int64_t)R.centers[ci] : R.c_base + ci;
                const int64_t j = R.cols[e];
                const double x = (double)pos[3 * j] - (double)pos[3 * i], y = (double)pos[3 * j + 1] - (double)pos[3 * i + 1],
                             z = (double)pos[3 * j + 2] - (double)pos[3 * i + 2];
                r = sqrt(x * x + y * y + z * z);
            }
            double b[NA], h[NA];
#pragma unroll
            for (int a = 0; a < NA; ++a) b[a] = h[a] = 0.0;
            for (int q0 = 0; q0 < Qp; q0 += RAD_QC) {
                const int q = q0 + sub;
                if (live && q < Q) {
                    const double xq = rq[q];
                    const double gq = exp(-0.5 * (xq - r) * (xq - r) * P.inv_s2);
                    bessel_scaled_lds(lw, xq * r * P.inv_s2, gq, mine);
                } else {
                    for (int k = 0; k < tw; ++k) mine[k] = 0.0;
                }
                wave_sync();
#pragma unroll 2
                for (int qq = 0; qq < RAD_QC; ++qq) {
                    const double tl = col[qq * tw + l], d = rq[q0 + qq] * col[qq * tw + l + 1] - r * tl;
                    const double *g = G + q0 + qq;
#pragma unroll
                    for (int a = 0; a < NA; ++a) {
                        const double ga = g[(size_t)a * Qp];
                        b[a] += ga * tl;
                        h[a] += ga * d;
                    }
                }
                wave_sync(); // the slab is read before the next nodes overwrite it
            }
            if (live && sub < lw) {
                double sb = 1.0, sh = 0.0;
                if (r == 0.0) {
                    sb = l == 0 ? 1.0 : 0.0;
                } else {
                    const double ir = 1.0 / r;
                    double rl = 1.0;
                    for (int k = 0; k < l; ++k) rl *= ir;
                    sb = rl;
                    sh = rl * ir * P.inv_s2;
                }
                double2 *o = out + (e - e_base) * (size_t)n * lw + l;
#pragma unroll
                for (int a = 0; a < NA; ++a)
                    if (a < n) o[(size_t)a * lw] = make_double2(b[a] * sb, h[a] * sh);
            }
        }
    }
}

typedef double dbl4 __attribute__((ext_vector_type(4)));

// Workgroup copy of cnt doubles from global memory to LDS (as DT) with U
// loads in flight per thread (a plain strided loop waits for each load in turn).
template <int BS, int U, typename DT = double, typename SRT = double>
__device__ __forceinline__ void copy_to_lds(DT *__restrict__ dst, const SRT *__restrict__ src, int cnt,
                                            int tid) {
    for (int base = 0; base < cnt; base += U * BS) {
        double v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = base + u * BS + tid;
            v[u] = src[k < cnt ? k : cnt - 1];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = base + u * BS + tid;
            if (k < cnt) dst[k] = (DT)v[u];
        }
    }
}

__host__ __device__ __forceinline__ int chunks_below(int l) { // sum over l' < l of ceil((2l'+1)/4)
    const int a = l >> 1;
    return (l & 1) ? (a + 1) * (a + 1) : a * (a + 1);
}

// Coefficients of one l-range as a matrix view: entry (u, lm) at
// C[u * ldu + (lm - lm0) * ldm], u = species * n + radial index; D holds
// one Cartesian component of the center derivative in the same layout.
// coefficients c (and one component of D) in LDS, entry (u, lm) at
// u * ldu + lm * ldm, stored at precision T (read as float64)
template <typename T = double> struct CoefView {
    const T *C, *D;
    int ldu, ldm;
};

// Power spectrum (comp < 0) or one Cartesian component d = comp of the
// center block, for l in [lg0, lg0 + lgc): 16 x 16 fp64 matrix-core tiles
// (ti <= tj) of u = (species, n) rows by v = (species, n') columns,
//   p(u, v, l)       =  K_l sum_m c_ulm c_vlm,
//   dp/dr_i(u, v, l) = -K_l sum_m (D_ulm c_vlm + c_ulm D_vlm),
// feature (u <= v, l) written to row[q * ldq + l - lbase] (Eqs.
// powerspectrum and powerspectrum-derivative, the center term from
// translational invariance).  Items (l, tile pair) go round-robin over the
// nw waves; only u <= v, the stored pairs (mu <= nu, n' >= n on mu = nu),
// are written.
//
// Pair index q of rows u <= v (u = species * n + n'), -1 for u > v: the
// position of the block (mu, nu, n, n') in the feature order (species pairs
// mu <= nu, then n, then n' with n' >= n on mu = nu).  Computed rather than
// read from a table: a global load among the output stores would wait for
// all of them (one vmcnt counter covers loads and stores).
struct PairIndex {
    int S, n;
    float inv_n;
    __device__ __forceinline__ int operator()(int u, int v) const {
        if (u > v) return -1;
        const int mu = qdiv(u, inv_n), a = u - mu * n, nu = qdiv(v, inv_n), b = v - nu * n;
        const int D = n * (n + 1) / 2, O = n * n;
        const int q = mu * D + O * (mu * (S - 1) - mu * (mu - 1) / 2); // pairs before (mu, mu)
        if (mu == nu) return q + a * n - a * (a + 1) / 2 + b;
        return q + D + (nu - mu - 1) * O + a * n + b;
    }
};
// the four pair indices of a lane's results: rows u = 16 ti + kk + 4 r of column v = 16 tj + ro
__device__ __forceinline__ void lane_pair_index(const PairIndex &pq, int Sn, int ti, int tj, int kk, int ro, int q[4]) {
    const int v = 16 * tj + ro;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int u = 16 * ti + kk + 4 * r;
        q[r] = (u < Sn && v < Sn) ? pq(u, v) : -1;
    }
}

// qtab (may be NULL): the lanes' pair indices per tile pair, [tile pair][lane][4]
// (pair_index_table), read instead of computed per item
// The pair indices of every lane for every tile pair (ti <= tj, in the order
// power_tiles deals them), [tile pair][lane][4] as shorts (pair indices are
// below Sn (Sn + 1) / 2, which fits for the Sn <= 80 the table is kept for),
// built by all threads.
__device__ __forceinline__ void pair_index_table(const PairIndex &pq, int Sn, short *__restrict__ qtab, int tid,
                                                 int nthreads) {
    const int ntile = (Sn + 15) >> 4, ntp = ntile * (ntile + 1) / 2;
    for (int k = tid; k < 64 * ntp; k += nthreads) {
        const int tpi = k >> 6, ln = k & 63;
        int tp = tpi, ti = 0;
        while (tp >= ntile - ti) {
            tp -= ntile - ti;
            ++ti;
        }
        int q[4];
        lane_pair_index(pq, Sn, ti, ti + tp, ln >> 4, ln & 15, q);
        short4 v;
        v.x = (short)q[0];
        v.y = (short)q[1];
        v.z = (short)q[2];
        v.w = (short)q[3];
        *(short4 *)(qtab + 4 * k) = v;
    }
}

template <typename OutT, typename CT = double>
__device__ __forceinline__ void power_tiles(const CoefView<CT> cv, int comp, int Sn, int lm0, int lg0, int lgc,
                                            OutT *__restrict__ row, int ldq, int lbase, const PairIndex pq,
                                            int wave, int nw, int lane, const double *__restrict__ Kl,
                                            const short *__restrict__ qtab = nullptr) {
    const int ntile = (Sn + 15) >> 4, ntp = ntile * (ntile + 1) / 2;
    const int nitem = lgc * ntp;
    const int ro = lane & 15, kk = lane >> 4;
    int q[4];
    if (ntp == 1) lane_pair_index(pq, Sn, 0, 0, kk, ro, q);
    // items dealt in snake order over the waves, longest chains first (an
    // item's chain has (l >> 1) + 1 chunks): every wave gets about the same
    // number of products, and the slowest wave sets the end of the phase
    for (int rd = 0;; ++rd) { // uniform per wave
        const int pos = rd * nw + ((rd & 1) ? nw - 1 - wave : wave);
        if (pos >= nitem) break;
        const int item = nitem - 1 - pos;
        const int lc = item / ntp, l = lg0 + lc;
        const int tpi = item - lc * ntp;
        int tp = tpi, ti = 0;
        while (tp >= ntile - ti) {
            tp -= ntile - ti;
            ++ti;
        }
        const int tj = ti + tp;
        if (ntp > 1) {
            if (qtab) {
                const short4 qs = *(const short4 *)(qtab + 4 * (64 * tpi + lane));
                q[0] = qs.x;
                q[1] = qs.y;
                q[2] = qs.z;
                q[3] = qs.w;
            } else {
                lane_pair_index(pq, Sn, ti, tj, kk, ro, q);
            }
        }
        const int ua = 16 * ti + ro, vb = 16 * tj + ro; // A row, B column of this lane
        const bool uok = ua < Sn, vok = vb < Sn;
        const int oa = (uok ? ua : 0) * cv.ldu + (l * l - lm0) * cv.ldm;
        const int ob = (vok ? vb : 0) * cv.ldu + (l * l - lm0) * cv.ldm;
        dbl4 acc = {0.0, 0.0, 0.0, 0.0};
        // one loop per kind (comp is uniform): a branch inside the chain made
        // the two kinds' accumulators meet in copies at every chunk
        if (comp < 0) {
            for (int ch = 0; ch < (l >> 1) + 1; ++ch) {
                const int m = 4 * ch + kk;
                const bool mok = m <= 2 * l;
                const int mo = (mok ? m : 0) * cv.ldm;
                const double ca = (double)cv.C[oa + mo], cb = (double)cv.C[ob + mo];
                const double xa = (mok && uok) ? ca : 0.0, xb = (mok && vok) ? cb : 0.0;
                acc = __builtin_amdgcn_mfma_f64_16x16x4f64(xa, xb, acc, 0, 0, 0);
            }
        } else {
            for (int ch = 0; ch < (l >> 1) + 1; ++ch) {
                const int m = 4 * ch + kk;
                const bool mok = m <= 2 * l;
                const int mo = (mok ? m : 0) * cv.ldm;
                const double ca = (double)cv.C[oa + mo], cb = (double)cv.C[ob + mo];
                const double xa = (mok && uok) ? ca : 0.0, xb = (mok && vok) ? cb : 0.0;
                const double da = (double)cv.D[oa + mo], db = (double)cv.D[ob + mo];
                acc = __builtin_amdgcn_mfma_f64_16x16x4f64((mok && uok) ? da : 0.0, xb, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f64_16x16x4f64(xa, (mok && vok) ? db : 0.0, acc, 0, 0, 0);
            }
        }
        // lane holds rows u = 16 ti + kk + 4 r of column v = 16 tj + ro
        const double K = comp < 0 ? Kl[l] : -Kl[l];
        OutT *rl = row + (l - lbase);
#pragma unroll
        for (int r = 0; r < 4; ++r)
            if (q[r] >= 0) store_out(rl + q[r] * ldq, K * acc[r]);
    }
}

// The four output rows of one center at once, for l in [lg0, lg0 + lgc):
// the power spectrum and the three center block components, from c (X) and
// D_x, D_y, D_z (X + d * xs, same layout as c: entry (u, lm) at
// u * ldu + (lm - lm0) * ldm).  Per item (l, tile pair) the c chunk is read
// once and the four accumulators are independent matrix-core chains.
// Feature (q, l) of the power spectrum goes to r0[q * ldq + l - lbase], of
// component d to r1[d * rs + q * ldq + l - lbase].
template <typename OutT>
__device__ __forceinline__ void power_tiles4(const double *__restrict__ X, int xs, int ldu, int ldm, int Sn, int lm0,
                                             int lg0, int lgc, OutT *__restrict__ r0, OutT *__restrict__ r1, int rs,
                                             int ldq, int lbase, const PairIndex pq, int wave, int nw,
                                             int lane, const double *__restrict__ Kl) {
    const int ntile = (Sn + 15) >> 4, ntp = ntile * (ntile + 1) / 2;
    const int nitem = lgc * ntp;
    const int ro = lane & 15, kk = lane >> 4;
    int q[4];
    if (ntp == 1) lane_pair_index(pq, Sn, 0, 0, kk, ro, q);
    // items dealt in snake order over the waves, longest chains first (an
    // item's chain has (l >> 1) + 1 chunks): every wave gets about the same
    // number of products, and the slowest wave sets the end of the phase
    for (int rd = 0;; ++rd) { // uniform per wave
        const int pos = rd * nw + ((rd & 1) ? nw - 1 - wave : wave);
        if (pos >= nitem) break;
        const int item = nitem - 1 - pos;
        const int lc = item / ntp, l = lg0 + lc;
        int tp = item - lc * ntp, ti = 0;
        while (tp >= ntile - ti) {
            tp -= ntile - ti;
            ++ti;
        }
        const int tj = ti + tp;
        if (ntp > 1) lane_pair_index(pq, Sn, ti, tj, kk, ro, q);
        const int ua = 16 * ti + ro, vb = 16 * tj + ro; // A row, B column of this lane
        const bool uok = ua < Sn, vok = vb < Sn;
        const int oa = (uok ? ua : 0) * ldu + (l * l - lm0) * ldm;
        const int ob = (vok ? vb : 0) * ldu + (l * l - lm0) * ldm;
        dbl4 p = {0.0, 0.0, 0.0, 0.0}, jx = p, jy = p, jz = p;
        for (int ch = 0; ch < (l >> 1) + 1; ++ch) {
            const int m = 4 * ch + kk;
            const bool mok = m <= 2 * l;
            const int mo = (mok ? m : 0) * ldm;
            const bool ma = mok && uok, mb = mok && vok;
            const double ca = ma ? X[oa + mo] : 0.0, cb = mb ? X[ob + mo] : 0.0;
            const double xa = ma ? X[xs + oa + mo] : 0.0, xb = mb ? X[xs + ob + mo] : 0.0;
            const double ya = ma ? X[2 * xs + oa + mo] : 0.0, yb = mb ? X[2 * xs + ob + mo] : 0.0;
            const double za = ma ? X[3 * xs + oa + mo] : 0.0, zb = mb ? X[3 * xs + ob + mo] : 0.0;
            p = __builtin_amdgcn_mfma_f64_16x16x4f64(ca, cb, p, 0, 0, 0);
            jx = __builtin_amdgcn_mfma_f64_16x16x4f64(xa, cb, jx, 0, 0, 0);
            jy = __builtin_amdgcn_mfma_f64_16x16x4f64(ya, cb, jy, 0, 0, 0);
            jz = __builtin_amdgcn_mfma_f64_16x16x4f64(za, cb, jz, 0, 0, 0);
            jx = __builtin_amdgcn_mfma_f64_16x16x4f64(ca, xb, jx, 0, 0, 0);
            jy = __builtin_amdgcn_mfma_f64_16x16x4f64(ca, yb, jy, 0, 0, 0);
            jz = __builtin_amdgcn_mfma_f64_16x16x4f64(ca, zb, jz, 0, 0, 0);
        }
        // lane holds rows u = 16 ti + kk + 4 r of column v = 16 tj + ro
        const double K = Kl[l];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            if (q[r] >= 0) {
                const int f = q[r] * ldq + l - lbase;
                store_out(r0 + f, K * p[r]);
                store_out(r1 + f, -K * jx[r]);
                store_out(r1 + (rs + f), -K * jy[r]);
                store_out(r1 + (2 * rs + f), -K * jz[r]);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// k_density
//
// Persistent: a workgroup is bound to one l-group g (blockIdx % G), keeps
// that group's basis tables in LDS, and takes centers from an atomic work
// counter after a first, static one (64-bit, zeroed with the neighbour list
// and never reset between launches: a launch subtracts the count taken
// before it, base).  Per center, each wave runs its own tiles of W edges: staging
// (harmonics, gradients, radial factors) in the wave's LDS, then every lane
// adds each edge's contribution to the coefficient entries (a, lm) it owns,
// in registers that persist over the wave's tiles:
//   c^s_{a lm} += B_al S_lm,
//   D^s_{a lm} += Bh_al r S_lm + B_al grad S_lm
// (D = sum over neighbours of dc/dr_j = -dc/dr_i).  Rows are sorted by
// species, so the registers are flushed into the shared LDS accumulators
// only when the species changes and at the end.  The flushes of one species
// go in wave order (each wave waits for its turn on that species, adds, and
// hands the turn on), so every sum is formed in the same order on every run:
// the results are bitwise repeatable and do not depend on which workgroup,
// launch or center batch computes a center.  Then
// the descriptor path writes the power spectrum of the group's l
// (power_tiles); the Jacobian path leaves c and D in scratch for k_outputs
// and k_jacobian.
// ---------------------------------------------------------------------------
constexpr int NWD = 4, BSD = 64 * NWD;

constexpr int KE = DENSITY_KE; // coefficient entries owned per lane: n * Lg <= 64 * KE

// Wave-ordered flushes: a wave waits for its turn on a species at most this
// many sleeps (~27 ns each; a turn comes within the time the lower waves take
// to reach the same species boundary).  The order argument (wave 0 never
// waits; wave w waits only for wave w-1 to pass a species that wave w-1
// passes before its next workgroup barrier) makes every wait end; the bound
// only guarantees it: past it the wave adds without its turn, which stays
// correct (the adds are LDS atomics) but gives up the fixed summation order.
constexpr int TURN_SPIN_LIMIT = 1 << 18;
constexpr int MAX_SPECIES = 64;

__host__ __device__ __forceinline__ int dens_lgY0(int jac, int lg0) { return (jac && lg0 > 0) ? lg0 - 1 : lg0; }

// Per-wave staging of k_density, in doubles: harmonics YY and radial pairs BB
// at the output precision (sb = 4 or 8 bytes), the radial scratch X in
// float64 (it enters dot products with cancelling basis coefficients).
__host__ __device__ __forceinline__ size_t dens_wave_doubles(const Params &P, int jac, int lg0, int lg1, int W,
                                                            int sb) {
    const int lgY0 = dens_lgY0(jac, lg0);
    const size_t LY = (size_t)(lg1 * lg1 - lgY0 * lgY0), lgc = (size_t)(lg1 - lg0);
    return even((W * LY * (jac ? 4 : 1) * sb + 7) / 8) + even((2 * W * P.n * lgc * sb + 7) / 8) +
           even(W * stage_x_doubles(P, (int)lgc, lg1));
}

// MODE: 0 descriptor (c, power spectrum); 1 descriptor + Jacobian (c and D);
// 2 coefficient Jacobian ("cc": c, every edge's dc/dr_j, and -D).
// RBF: the radial basis, fixed at compile time (0 GTO, 1 polynomial by
// quadrature, 2 polynomial in the Laplace form, 3 GTO compensated).  The other bases' branches of
// the staging then drop out, and with them up to 40 VGPRs: the GTO descriptor
// kernel runs four waves per SIMD instead of three.
// Resident waves per SIMD: a second variant (HI) of the coefficient Jacobian
// asks for 2 (it otherwise takes all 256 VGPRs and runs one wave), and of the
// Jacobian path of GTO and the Laplace form for 3 (a small spill).  More
// workgroups per CU split the LDS further, so the host takes HI only where
// the LDS plan stays as good (density_has_high and plan_launches).
constexpr bool dens_has_high(int mode, int rbf) { return mode == 2 || (mode == 1 && (rbf == 0 || rbf == 2)); }
constexpr int dens_min_waves(int mode, int rbf, bool hi) {
    return (hi && dens_has_high(mode, rbf)) ? (mode == 2 ? 2 : 3) : 1;
}

// ST: precision of the staged harmonics and radial factors (OutT, or double
// for float64 arithmetic with float32 outputs), and of the coefficient scratch.
template <typename PosT, typename OutT, int MODE, int RBF, bool HI, typename ST = OutT>
__global__ __launch_bounds__(BSD, dens_min_waves(MODE, RBF, HI)) void k_density(Params P, Rows R, const PosT *__restrict__ pos, int W,
                                                 unsigned long long *__restrict__ work, WorkBase base,
                                                 OutT *__restrict__ desc,
                                                 OutT *__restrict__ c_out, OutT *__restrict__ jself,
                                                 ST *__restrict__ c_scratch, OutT *__restrict__ jc_edge) {
    constexpr bool JAC = MODE != 0, CCJ = MODE == 2;
    // 16-byte aligned: the carved regions are read with 16-byte LDS accesses
    extern __shared__ __align__(16) double smem[];
    __shared__ int64_t s_next;
    __shared__ int s_turn[MAX_SPECIES]; // per species: the wave whose partial sums go in next
    const int G = P.n_groups;
    const int g = blockIdx.x % G;
    const int lg0 = P.lgrp[g], lg1 = P.lgrp[g + 1], lgc = lg1 - lg0;
    const int lm0 = lg0 * lg0, Lg = lg1 * lg1 - lm0;
    const int lgY0 = dens_lgY0(JAC, lg0), lmY0 = lgY0 * lgY0, LY = lg1 * lg1 - lmY0;
    const int S = P.S, n = P.n, tid = threadIdx.x, lane = tid & 63;
    // wave-uniform (the compiler cannot prove tid >> 6 uniform by itself): per-wave
    // loops then compile to scalar control flow
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nL = n * Lg, SnL = S * nL, lw = P.lmax + 1, Lfull = P.L, Sn = S * n, nlc = n * lgc;
    const int RBk = row_block(NWD * W);

    Carver cv{smem};
    Tables T;
    load_tables<0, 0, RBF>(P, cv, T, lg0, lg1);
    double *cacc = cv.take((size_t)SnL * (JAC ? 4 : 1)); // [s][a][lmg], then D [3][s][a][lmg]
    double *Dacc = cacc + SnL;
    double *rgeo = cv.take(4 * (size_t)RBk);
    int *rsp = (int *)cv.take((RBk + 1) / 2);
    double *c0 = cv.take((size_t)n);
    // staging at precision ST (by default the output precision): the
    // harmonics and radial factors enter the float64 accumulators as
    // products with relative rounding error of ST's order, which float32
    // outputs carry anyway
    using ST2 = typename Pair<ST>::type;
    constexpr int SB = sizeof(ST);
    Carver wv{cv.take(0) + (size_t)wave * dens_wave_doubles(P, JAC, lg0, lg1, W, SB)};
    // harmonics interleaved per lm as (S, dS/dx, dS/dy, dS/dz) for the Jacobian
    const YLayout yl = JAC ? YLayout{4 * LY, 1, 4, lmY0} : YLayout{LY, 0, 1, lmY0};
    ST *YY = (ST *)wv.take(((size_t)W * yl.es * SB + 7) / 8);
    ST2 *BB = (ST2 *)wv.take((2 * (size_t)W * nlc * SB + 7) / 8);
    double *X = wv.take((size_t)W * stage_x_doubles(P, lgc, lg1));

    // the coefficient entries this lane owns: (a, lm) = ent / Lg, ent % Lg;
    // oC: its offset a L + lm in a coefficient block of one species (unsigned,
    // so the gradient stores take the scalar-base + 32-bit-offset form instead
    // of per-lane 64-bit addresses, which the compiler hoists and spills)
    int oY[KE], oB[KE];
    uint32_t oC[KE];
    bool own[KE];
#pragma unroll
    for (int k = 0; k < KE; ++k) {
        const int e = lane + 64 * k;
        own[k] = e < nL;
        const int a = e / Lg, lmg = e - a * Lg;
        const int lm = lm0 + (own[k] ? lmg : 0);
        oC[k] = (uint32_t)(a * Lfull + lm);
        int l = (int)sqrtf((float)lm);
        while (l * l > lm) --l;
        while ((l + 1) * (l + 1) <= lm) ++l;
        oY[k] = (lm - lmY0) * (JAC ? 4 : 1);
        oB[k] = own[k] ? a * lgc + (l - lg0) : 0;
    }

    // on-site terms in LDS: no global load may sit between output stores
    // (vmcnt counts loads and stores together)
    for (int k = tid; k < n; k += BSD) c0[k] = P.c0[k];
    // structure index of the batch's first edge: edge outputs are batch-local
    const int64_t ebase = CCJ ? *R.e_origin : 0;

    // the next center: its rows are loaded before the current center's
    // outputs are stored, so those loads never wait behind the stores
    int64_t ci = 0, i = 0, e0 = 0, e1 = 0;
    int spec_i = 0;
    double3 pi = make_double3(0.0, 0.0, 0.0);
    // the first center of each workgroup is static (blockIdx / G); the later
    // ones come from the group's counter, past the per_group static ones
    // (a burst of one atomic per workgroup on one address at the start would
    // serialise)
    const int64_t per_group = gridDim.x / G;
    bool first = true;
    auto fetch = [&]() {
        if (first) {
            ci = blockIdx.x / G;
            first = false;
        } else {
            if (tid == 0) s_next = per_group + (int64_t)(atomicAdd(&work[g], 1ull) - base.b[g]);
            lds_barrier();
            ci = __builtin_amdgcn_readfirstlane((int)s_next); // uniform: scalar addressing
            lds_barrier();                                    // s_next is rewritten by the next fetch
        }
        if (ci >= R.nc) return;
        i = R.centers ? (int64_t)R.centers[ci] : R.c_base + ci;
        pi = make_double3((double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]);
        spec_i = R.spec[i];
        e0 = R.row_ptr[ci];
        e1 = R.row_ptr[ci + 1];
        const int64_t cnt = (e1 - e0) < RBk ? (e1 - e0) : RBk;
        load_rows(rgeo, rsp, pos, R.spec, R.cols, e0, (int)cnt, pi);
    };
    fetch();
    const float inv_Lg = 1.0f / (float)Lg, inv_Sn = 1.0f / (float)Sn;
    const PairIndex pq{S, n, 1.0f / (float)n};

    while (ci < R.nc) {
        for (int k = tid; k < SnL * (JAC ? 4 : 1); k += BSD) cacc[k] = 0.0;
        for (int k = tid; k < S; k += BSD) s_turn[k] = 0;
        lds_barrier(); // rows of this center, the cleared accumulators and turns

        double acc[KE][4];
#pragma unroll
        for (int k = 0; k < KE; ++k) acc[k][0] = acc[k][1] = acc[k][2] = acc[k][3] = 0.0;
        int cur = -1;  // species of the registers' partial sums (-1: none held)
        int nextp = 0; // the lowest species this wave has not passed yet
        // Pass every species t in [nextp, upto): wait for this wave's turn on
        // t, add the registers into the shared accumulators if they hold t,
        // and hand the turn to the next wave.  Species go in increasing order
        // (the rows are sorted), so each wave passes each species once per
        // center and the sums of a species are taken in wave order.
        auto pass = [&](int upto) {
            for (int t = nextp; t < upto; ++t) {
                bool turn = false;
                for (int spin = 0; spin < TURN_SPIN_LIMIT; ++spin) {
                    const int w = __hip_atomic_load(&s_turn[t], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
                    if (__builtin_amdgcn_readfirstlane(w) == wave) {
                        turn = true;
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                }
                if (t == cur) {
                    // LDS atomic adds (one instruction each): while the wave
                    // holds the turn no other wave adds to species t, so the
                    // order is the wave order
#pragma unroll
                    for (int k = 0; k < KE; ++k) {
                        if (!own[k]) continue;
                        const int idx = cur * nL + lane + 64 * k;
                        atomicAdd(&cacc[idx], acc[k][0]);
                        if (JAC) {
                            atomicAdd(&Dacc[idx], acc[k][1]);
                            atomicAdd(&Dacc[SnL + idx], acc[k][2]);
                            atomicAdd(&Dacc[2 * SnL + idx], acc[k][3]);
                        }
                        acc[k][0] = acc[k][1] = acc[k][2] = acc[k][3] = 0.0;
                    }
                    cur = -1;
                }
                if (turn) __hip_atomic_store(&s_turn[t], wave + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
            }
            nextp = upto > nextp ? upto : nextp;
        };

        for (int64_t rb0 = e0; rb0 < e1; rb0 += RBk) {
            const int rbn = (int)((e1 - rb0) < RBk ? (e1 - rb0) : RBk);
            if (rb0 != e0) { // further row blocks of a long row (no output stores are pending here)
                // before the barrier, pass the species below the last one of
                // the block just done: a wave waiting for its turn on one of
                // them is then never left waiting on a wave held at the barrier
                pass(__builtin_amdgcn_readfirstlane(rsp[RBk - 1])); // the previous block is full
                lds_barrier();
                load_rows(rgeo, rsp, pos, R.spec, R.cols, rb0, rbn, pi);
                lds_barrier();
            }
            for (int off = wave * W; off < rbn; off += NWD * W) {
                const int nb = (rbn - off) < W ? (rbn - off) : W;
                const double *geo = rgeo + 4 * off;
                stage_edges<JAC, ST, 0, 0, ST, RBF>(P, T, YY, yl, BB, X, geo, nb, lane, lg0, lg1, false, rb0 + off);
                for (int e = 0; e < nb; ++e) {
                    const int s = __builtin_amdgcn_readfirstlane(rsp[off + e]);
                    if (s != cur) {
                        pass(s); // adds the registers if they hold a lower species
                        cur = s;
                    }
                    const double rx = geo[4 * e], ry = geo[4 * e + 1], rz = geo[4 * e + 2];
                    const ST *Ye = YY + e * yl.es;
                    const ST2 *Be = BB + e * nlc;
                    // this edge's block of the coefficient Jacobian: [3][n][L],
                    // one wave-uniform base per row.  The base is made opaque:
                    // strength-reduced over the edges, it became one 64-bit
                    // pointer per lane and entry, which spilled.
                    OutT *je = nullptr;
                    if (CCJ) {
                        je = jc_edge + (size_t)(rb0 + off + e - ebase) * 3 * n * Lfull;
                        __asm__ volatile("" : "+s"(je));
                    }
                    OutT *const je1 = je + (size_t)n * Lfull, *const je2 = je + 2 * (size_t)n * Lfull;
#pragma unroll
                    for (int k = 0; k < KE; ++k) {
                        if (!own[k]) continue;
                        const ST2 b2 = Be[oB[k]];
                        const double bx = (double)b2.x, by = (double)b2.y;
                        if (JAC) {
                            double y0, y1, y2, y3;
                            load4(Ye + oY[k], y0, y1, y2, y3);
                            const double bh = by * y0;
                            // dc/dr_j = Bh r S + B grad S (Eqs. gto-derivative, poly-cartesian-derivative)
                            const double gx = bh * rx + bx * y1, gy = bh * ry + bx * y2, gz = bh * rz + bx * y3;
                            acc[k][0] += bx * y0;
                            acc[k][1] += gx;
                            acc[k][2] += gy;
                            acc[k][3] += gz;
                            if (CCJ) {
                                store_out(je + oC[k], gx);
                                store_out(je1 + oC[k], gy);
                                store_out(je2 + oC[k], gz);
                            }
                        } else {
                            acc[k][0] += bx * (double)Ye[oY[k]];
                        }
                    }
                }
                wave_sync(); // the next tile's staging overwrites YY and BB
            }
        }
        pass(S);
        lds_barrier();
        // on-site term of the center (its species, l = 0)
        if (lg0 == 0)
            for (int a = tid; a < n; a += BSD) cacc[spec_i * nL + a * Lg] += c0[a];
        // the next center's rows go in while this center's outputs are written
        const int64_t cw = ci;
        fetch(); // its barriers also publish the on-site term
        // power spectrum (descriptor path): per l, 16 x 16 matrix-core tiles
        // (ti <= tj) of u = (species, n) rows and v = (species, n') columns
        if (!JAC && desc)
            power_tiles<OutT>(CoefView<double>{cacc, nullptr, Lg, 1}, -1, Sn, lm0, lg0, lgc, desc + cw * P.F, lw, 0, pq,
                              wave, NWD, lane, T.Kl);
        if (c_out)
            for (int it = tid; it < SnL; it += BSD) {
                const int sa = qdiv(it, inv_Lg), lmg = it - sa * Lg;
                store_out(c_out + (cw * Sn + sa) * Lfull + lm0 + lmg, cacc[it]);
            }
        if (CCJ) {
            // center block of the coefficient Jacobian: dc/dr_i = -D, [3][S][n][L]
            for (int it = tid; it < 3 * SnL; it += BSD) {
                const int d = it / SnL, rem = it - d * SnL;
                const int sa = qdiv(rem, inv_Lg), lmg = rem - sa * Lg;
                store_out(jself + ((cw * 3 + d) * Sn + sa) * Lfull + lm0 + lmg, -Dacc[it]);
            }
        } else if (JAC) {
            // with one l-group the workgroup holds all of c and D: it writes
            // the power spectrum and the center block itself (whole rows of
            // one center from one workgroup, so their lines fill in one L2);
            // the scratch then only needs c.  Otherwise c and D go to
            // scratch for k_outputs.  Both transposed to [comp][lm][s n]: c
            // is the Jacobian kernel's matrix-core operand.
            const bool whole = G == 1;
            if (whole)
                power_tiles4<OutT>(cacc, SnL, Lg, 1, Sn, 0, 0, lw, desc + cw * P.F, jself + cw * 3 * P.F, P.F, lw, 0,
                                   pq, wave, NWD, lane, T.Kl);
            // in destination order (consecutive lanes, consecutive addresses);
            // the transposition falls on the LDS reads
            ST *sc = c_scratch + cw * 4 * (size_t)Lfull * Sn;
            for (int it = tid; it < (whole ? 1 : 4) * SnL; it += BSD) {
                const int comp = it / SnL, rem = it - comp * SnL;
                const int lmg = qdiv(rem, inv_Sn), sa = rem - lmg * Sn;
                sc[((size_t)comp * Lfull + lm0 + lmg) * Sn + sa] = (ST)cacc[comp * SnL + sa * Lg + lmg];
            }
        }
        lds_barrier(); // the outputs are read from cacc before the next center clears it
    }
}

// All real solid harmonics of one edge per lane (l < lw), by the column
// recurrence of sh_col_y, into Y[lm * ls]; Nt in LDS (wave-uniform reads).
template <typename YT>
__device__ __forceinline__ void sh_all_lane(double x, double y, double z, const double *__restrict__ Nt, int ldN,
                                            int lw, YT *__restrict__ Y, int ls) {
#pragma clang fp contract(off) // the roundings of sh_all_fixed, bit for bit
    const double r2 = x * x + y * y + z * z;
    double c = 1.0, s = 0.0; // (x + i y)^m
    for (int m = 0; m < lw; ++m) {
        double R1 = 0.0, R = 1.0; // R_{l-1}, R_l
        for (int l = m; l < lw; ++l) {
            if (l > m) {
                const double a = (double)(2 * l - 1), b = (double)((l + m - 1) * (l - m - 1));
                const double Rn = __builtin_fma(a * z, R, -(b * r2 * R1));
                R1 = R;
                R = Rn;
            }
            const double v = Nt[l * ldN + m] * R;
            const int o = l * l + l;
            if (m == 0) {
                Y[o * ls] = (YT)v;
            } else {
                Y[(o + m) * ls] = (YT)(v * c);
                Y[(o - m) * ls] = (YT)(v * s);
            }
        }
        const double cn = __builtin_fma(x, c, -(y * s));
        s = __builtin_fma(x, s, y * c);
        c = cn;
    }
}

// sh_all_lane for a degree count LW and a row stride LS fixed at compile
// time (Nt rows of LW + 1 entries): the same recurrence fully unrolled, so
// that the constants a, b, the table and store offsets and the loop control
// are resolved at compile time; what stays is the per-lane arithmetic and
// the LDS traffic.
template <int LW, int LS, typename YT>
__device__ __forceinline__ void sh_all_fixed(double x, double y, double z, const double *__restrict__ Nt,
                                             YT *__restrict__ Y) {
#pragma clang fp contract(off) // the roundings of sh_all_lane, bit for bit
    constexpr int ls = LS;
    constexpr int ldN = LW + 1;
    // the edge vector passes through an empty asm: the unrolled products
    // depend only on it, and hoisted out of the caller's task loop they
    // would all be live across the other tasks
    __asm__ volatile("" : "+v"(x), "+v"(y), "+v"(z));
    const double r2 = x * x + y * y + z * z;
    double c = 1.0, s = 0.0; // (x + i y)^m
#pragma unroll
    for (int m = 0; m < LW; ++m) {
        // an opaque zero offset per column keeps the table reads here (the
        // table is invariant too)
        int t0 = 0;
        __asm__ volatile("" : "+s"(t0));
        const double *Ntc = Nt + t0;
        double R1 = 0.0, R = 1.0; // R_{l-1}, R_l
#pragma unroll
        for (int l = m; l < LW; ++l) {
            if (l > m) {
                const double a = (double)(2 * l - 1), b = (double)((l + m - 1) * (l - m - 1));
                const double Rn = __builtin_fma(a * z, R, -(b * r2 * R1));
                R1 = R;
                R = Rn;
            }
            const double v = Ntc[l * ldN + m] * R;
            const int o = l * l + l;
            if (m == 0) {
                Y[o * ls] = (YT)v;
            } else {
                Y[(o + m) * ls] = (YT)(v * c);
                Y[(o - m) * ls] = (YT)(v * s);
            }
        }
        const double cn = __builtin_fma(x, c, -(y * s));
        s = __builtin_fma(x, s, y * c);
        c = cn;
    }
}

// the solid harmonics of one edge per lane: unrolled for lw <= 8 at the row
// stride of 64-edge chunks (both uniform, so one case runs per wave), else
// the loop
template <typename YT>
__device__ __forceinline__ void sh_all_any(double x, double y, double z, const double *__restrict__ Nt, int ldN,
                                           int lw, YT *__restrict__ Y, int ls) {
    constexpr int LS = 65;
    if (ls != LS) {
        sh_all_lane(x, y, z, Nt, ldN, lw, Y, ls);
        return;
    }
    switch (lw) {
    case 2: sh_all_fixed<2, LS>(x, y, z, Nt, Y); break;
    case 3: sh_all_fixed<3, LS>(x, y, z, Nt, Y); break;
    case 4: sh_all_fixed<4, LS>(x, y, z, Nt, Y); break;
    case 5: sh_all_fixed<5, LS>(x, y, z, Nt, Y); break;
    case 6: sh_all_fixed<6, LS>(x, y, z, Nt, Y); break;
    case 7: sh_all_fixed<7, LS>(x, y, z, Nt, Y); break;
    case 8: sh_all_fixed<8, LS>(x, y, z, Nt, Y); break;
    default: sh_all_lane(x, y, z, Nt, ldN, lw, Y, ls); break;
    }
}

// ---------------------------------------------------------------------------
// k_desc: the descriptor (and coefficients) of the GTO basis.  Persistent
// workgroups of NWC waves, one center at a time per workgroup (centers
// blockIdx + k gridDim), in two phases per chunk of up to W edges of the
// center's row:
//   1. staging, lane = edge, split over the waves by task: task l < l_max + 1
//      is the radial factors of degree l, B_nl = sum_k betaC^l_nk e^{-a'_kl r^2}
//      (Eq. gto-coefficients); task l_max + 1 is the real solid harmonics
//      S_lm (sh_all_any).  Wave w runs tasks w, w + NWC, ...  Every
//      coefficient read is wave-uniform (the tables sit in LDS, copied once
//      per workgroup), and every lane works on its own edge;
//   2. projection, thread = (lm, group of AG radial indices a): each thread
//      owns those coefficients c_{a lm} in float64 registers, one set per
//      species (SR >= S slots), and adds B_al S_lm over the chunk's edges in
//      row order (Eq. projection); one harmonic read serves AG products.
//      Rows are sorted by species, so each species is a contiguous run of the
//      chunk.  After the row the owner of (l = 0, a) of the center's species
//      adds the on-site term, and the registers go to the center's
//      coefficient block (its own LDS region).
// Every coefficient has one owner thread and every sum runs in row order:
// the results are bitwise repeatable with no ordering protocol.  Then the
// power spectrum on the matrix cores (power_tiles, Eq. powerspectrum).
// Two barriers per center of one chunk: staging -> projection, and block ->
// power spectrum.  The block's next writers pass the next center's first
// barrier, which every wave reaches only after its power spectrum tiles; the
// staging's next writers come after the block barrier, which every wave
// reaches only after its projection reads.  The next center's first chunk of edge vectors is
// gathered into registers before this center's output stores: a load issued
// after a run of stores waits for all of them.
// ST: staging precision (the output precision, or double for float64
// arithmetic with float32 outputs).  QT (lm, group) tasks per thread, AG
// radial indices per group and NA >= n_max, fixed at compile time so that
// the accumulators stay in registers.
// ---------------------------------------------------------------------------
constexpr int NWC = 4, BSC = 64 * NWC;

// LDS of k_desc.  Float64: K_l, the harmonic normalisations Nt, a'_kl [l][k],
// betaC [l][n][k], the on-site terms, the exponential's table, the
// coefficient block [S][n][L].  Then the staging buffers.
// Staging, at the staging precision: harmonics [lm][W + 1] and radial
// factors [l][n][W + 1] (edge fastest: the staging lanes, one per edge,
// write consecutive words), the rows of one l padded to an odd length
// desc_ldl; the odd strides put the projection threads, which read one edge
// at different lm (or l), on different banks.  Then the chunk's species run
// bounds.
__host__ __device__ __forceinline__ int desc_ldl(int n, int W) { return (n * (W + 1)) | 1; }
__host__ __device__ __forceinline__ size_t desc_lds_doubles(const Params &P, int W, int sb) {
    const size_t ldN = (size_t)P.lmax + 2, lw = (size_t)P.lmax + 1, n = (size_t)P.n, L = (size_t)P.L;
    const size_t stage = even((L * (W + 1) * sb + 7) / 8) + even((lw * desc_ldl((int)n, W) * sb + 7) / 8) + 16;
    const size_t block = (size_t)P.S * n * L;
    return 16 + even(ldN * ldN) + even(lw * n) + even(lw * n * n) + even(n) + 128 + even(block) + even(stage);
}
// (lm, group of ag radial indices) tasks per thread
__host__ __device__ __forceinline__ int desc_tasks(const Params &P, int ag) {
    return (P.L * ((P.n + ag - 1) / ag) + BSC - 1) / BSC;
}

template <typename PosT, typename OutT, typename ST, int QT, int AG, int NA, int SR>
__global__ __launch_bounds__(BSC) void k_desc(Params P, Rows R, const PosT *__restrict__ pos, int W,
                                              OutT *__restrict__ desc, OutT *__restrict__ c_out) {
    extern __shared__ __align__(16) double smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int S = P.S, n = P.n, lmax = P.lmax, lw = lmax + 1, L = P.L, ldN = lmax + 2, Sn = S * n;
    const int nL = n * L, SnL = S * nL, np = (n + AG - 1) / AG;
    constexpr int SB = sizeof(ST);
    Carver cv{smem};
    double *Kl = cv.take(16);
    double *Nt = cv.take((size_t)ldN * ldN);
    double *apr = cv.take((size_t)lw * n);
    double *bcf = cv.take((size_t)lw * n * n);
    double *c0 = cv.take((size_t)n);
    double *e2 = cv.take(128);               // 2^(j/64) pairs of exp_neg_tab
    double *cb = cv.take((size_t)S * n * L); // [S][n][L], written after the row
    double *stage = cv.take(0);
    const int WP = W + 1, ldl = desc_ldl(n, W);
    Carver sv{stage};
    ST *Yl = (ST *)sv.take(((size_t)L * WP * SB + 7) / 8);  // [lm][W + 1]
    ST *Bl = (ST *)sv.take(((size_t)lw * ldl * SB + 7) / 8); // [l][n][W + 1], rows of l padded to ldl
    int *run = (int *)sv.take(16);                           // species run bounds of the chunk
    if (tid < 16) Kl[tid] = M_PI * sqrt(8.0 / (double)(2 * tid + 1));
    for (int k = tid; k < ldN * ldN; k += BSC) Nt[k] = P.Nt[k];
    for (int k = tid; k < lw * n; k += BSC) apr[k] = P.aprime[k];
    for (int k = tid; k < lw * n * n; k += BSC) bcf[k] = P.betaC[k];
    for (int k = tid; k < n; k += BSC) c0[k] = P.c0[k];
    for (int k = tid; k < 128; k += BSC) e2[k] = P.e2t[k];

    // this thread's projection tasks: (lm, radial group) = (t % L, t / L), t = tid + BSC q
    int lm_q[QT], l_q[QT], a_q[QT], goff[QT][AG];
    bool ok_q[QT];
#pragma unroll
    for (int q = 0; q < QT; ++q) {
        const int t = tid + BSC * q, ap = t / L, lm = t - ap * L;
        int l = (int)sqrtf((float)lm);
        while (l * l > lm) --l;
        while ((l + 1) * (l + 1) <= lm) ++l;
        ok_q[q] = ap < np;
        lm_q[q] = ok_q[q] ? lm : 0;
        l_q[q] = ok_q[q] ? l : 0;
        a_q[q] = ok_q[q] ? AG * ap : 0;
#pragma unroll
        for (int g = 0; g < AG; ++g) goff[q][g] = (a_q[q] + g < n ? g : 0) * WP;
    }
    int64_t ci = blockIdx.x;
    const int64_t stride = gridDim.x;
    // the first chunk of a center's row, gathered by every wave, lane = edge:
    // edge vector (float64, exact for float32 inputs) and species
    double gx = 0.0, gy = 0.0, gz = 0.0;
    int gs = 0;
    int64_t e0 = 0, e1 = 0;
    double3 pi = make_double3(0.0, 0.0, 0.0);
    int spec_i = 0;
    auto gather = [&](int64_t cs, int nb) {
        if (lane < nb) {
            const int64_t j = R.cols[cs + lane];
            gx = (double)pos[3 * j] - pi.x;
            gy = (double)pos[3 * j + 1] - pi.y;
            gz = (double)pos[3 * j + 2] - pi.z;
            gs = R.spec[j];
        }
    };
    auto fetch = [&]() { // the center ci: its atom, row and first chunk
        if (ci >= R.nc) return;
        const int64_t i = R.centers ? (int64_t)R.centers[ci] : R.c_base + ci;
        pi = make_double3((double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]);
        spec_i = R.spec[i];
        e0 = R.row_ptr[ci];
        e1 = R.row_ptr[ci + 1];
        gather(e0, (int)((e1 - e0) < W ? (e1 - e0) : W));
    };
    fetch();
    lds_barrier(); // the tables
    while (ci < R.nc) {
        double acc[SR][QT][AG];
#pragma unroll
        for (int sr = 0; sr < SR; ++sr)
#pragma unroll
            for (int q = 0; q < QT; ++q)
#pragma unroll
                for (int g = 0; g < AG; ++g) acc[sr][q][g] = 0.0;
        for (int64_t cs = e0; cs < e1; cs += W) {
            const int nb = (int)((e1 - cs) < W ? (e1 - cs) : W);
            if (cs != e0) { // later chunks of a long row (no stores pending)
                gather(cs, nb);
                lds_barrier(); // the previous chunk is read
            }
            // ---- phase 1: staging, lane = edge, tasks over the waves ----
            if (wave == 0) {
                // run bounds: the chunk's edges of species below sr (rows are sorted by species)
#pragma unroll
                for (int sr = 0; sr <= SR; ++sr) {
                    const int cnt = __popcll(__ballot(lane < nb && gs < sr));
                    if (lane == 0) run[sr] = cnt;
                }
            }
            if (lane < nb) {
                const double r2 = gx * gx + gy * gy + gz * gz;
                for (int task = wave; task <= lw; task += NWC) {
                    if (task == lw) {
                        sh_all_any(gx, gy, gz, Nt, ldN, lw, Yl + lane, WP);
                        continue;
                    }
                    const int l = task;
                    // exponentials past n_max are zero, so the clamped
                    // coefficient reads past the row multiply zero
                    double ex[NA];
#pragma unroll
                    for (int k = 0; k < NA; ++k) {
                        const double v = exp_neg_tab(apr[l * n + (k < n ? k : n - 1)] * r2, e2);
                        ex[k] = k < n ? v : 0.0;
                    }
                    ST *bo = Bl + (size_t)l * ldl + lane;
                    const double *bc = bcf + (size_t)l * n * n;
                    if (n == NA) {
                        // unrolled: compile-time coefficient offsets and NA
                        // independent sums (the same sums, in the same order)
#pragma unroll
                        for (int a = 0; a < NA; ++a) {
                            double b = 0.0;
#pragma unroll
                            for (int k = 0; k < NA; ++k) b += bc[a * NA + k] * ex[k];
                            bo[a * WP] = (ST)b;
                        }
                    } else {
                        for (int a = 0; a < n; ++a) {
                            double b = 0.0;
#pragma unroll
                            for (int k = 0; k < NA; ++k) b += bc[a * n + (k < n ? k : n - 1)] * ex[k];
                            bo[a * WP] = (ST)b;
                        }
                    }
                }
            }
            lds_barrier();
            // ---- phase 2: projection, thread = (lm, radial group), species run by run ----
#pragma unroll
            for (int sr = 0; sr < SR; ++sr) {
                const int lo = run[sr], hi = run[sr + 1];
#pragma unroll 4
                for (int e = lo; e < hi; ++e) {
#pragma unroll
                    for (int q = 0; q < QT; ++q) {
                        // every load unconditional (a guarded load becomes a branch that waits for it
                        // alone): a thread with no task reads lm 0, a radial index past n_max reads
                        // index a_q; neither sum is ever written
                        const double yv = (double)Yl[lm_q[q] * WP + e];
                        const ST *bp = Bl + (size_t)l_q[q] * ldl + a_q[q] * WP + e;
#pragma unroll
                        for (int g = 0; g < AG; ++g) acc[sr][q][g] += (double)bp[goff[q][g]] * yv;
                    }
                }
            }
        }
        // on-site term of the center (its species, l = 0), added by the owner
        // after the row's sum
#pragma unroll
        for (int sr = 0; sr < SR; ++sr)
#pragma unroll
            for (int q = 0; q < QT; ++q)
#pragma unroll
                for (int g = 0; g < AG; ++g)
                    if (sr == spec_i && lm_q[q] == 0 && ok_q[q] && a_q[q] + g < n) acc[sr][q][g] += c0[a_q[q] + g];
#pragma unroll
        for (int sr = 0; sr < SR; ++sr)
#pragma unroll
            for (int q = 0; q < QT; ++q)
#pragma unroll
                for (int g = 0; g < AG; ++g)
                    if (sr < S && ok_q[q] && a_q[q] + g < n) cb[(sr * n + a_q[q] + g) * L + lm_q[q]] = acc[sr][q][g];
        lds_barrier(); // the block is complete (and every wave is done with the staging)
        // the next center's first chunk goes in before this center's stores
        const int64_t cw = ci;
        ci += stride;
        fetch();
        if (desc)
            power_tiles<OutT>(CoefView<double>{cb, nullptr, L, 1}, -1, Sn, 0, 0, lw, desc + cw * P.F, lw, 0,
                              PairIndex{S, n, 1.0f / (float)n}, wave, NWC, lane, Kl);
        if (c_out)
            for (int k = tid; k < SnL; k += BSC) store_out(c_out + cw * SnL + k, cb[k]);
    }
}

// ---------------------------------------------------------------------------
// k_djac: the density step of the Jacobian path for the GTO basis, in the
// layout of k_desc (one center per workgroup of NWC waves, 64-edge chunks,
// staging lane = edge split over the waves by task, every accumulated entry
// owned by one thread):
//   staging: task l: B_nl and Bh_nl = (1/r) dB_nl/dr = sum_k betaCa e_kl
//     (Eqs. gto-coefficients, gto-derivative); the last task: the solid
//     harmonics; wave 0 also keeps the chunk's edge vectors and species;
//   projection, thread = (lm, pair of radial indices): per edge
//       c_{a lm}  += B_al S_lm,
//       D_{a lm}  += Bh_al r S_lm + B_al grad S_lm,
//     (D = sum over neighbours of dc/dr_j = -dc/dr_i), the gradient of S_lm
//     from at most five degree l-1 harmonics by the ladder identities of
//     stage_edges (zero for an edge of length 0).  The sums of each species
//     stay in registers (species slots SR >= S): the rows are sorted by
//     species, so each species is a contiguous run of the chunk.
// At the end of the row the registers go to the coefficient block [c, Dx, Dy,
// Dz][S][n][L] (aliasing the staging buffers), the on-site term is added, and
// the workgroup writes the power spectrum and the center block
// -K_l sum_m (D^mu c^nu + c^mu D^nu) (power_tiles4, Eqs. powerspectrum,
// powerspectrum-derivative with translational invariance) and the
// coefficients, transposed to [lm][species n], for k_jacobian.  Each sum runs
// in row order: deterministic with no ordering protocol.
// ---------------------------------------------------------------------------
// LDS doubles of k_djac: tables (K_l, Nt, a', betaC, c0), then the
// larger of the staging buffers (harmonics [lm][W+1], B and Bh [l][n][W+1]
// with odd row lengths, edge vectors [W][4], species [W], species run bounds)
// and the coefficient block 4 S n L
__host__ __device__ __forceinline__ size_t djac_table_doubles(const Params &P) {
    const size_t ldN = (size_t)P.lmax + 2, lw = (size_t)P.lmax + 1, n = (size_t)P.n;
    return 16 + even(ldN * ldN) + even(lw * n) + even(lw * n * n) + even(n) + 128;
}
__host__ __device__ __forceinline__ size_t djac_stage_doubles(const Params &P, int W, int sb) {
    const size_t L = (size_t)P.L, lw = (size_t)P.lmax + 1, n = (size_t)P.n;
    const size_t stage = even((L * (W + 1) * sb + 7) / 8) + 2 * even((lw * desc_ldl((int)n, W) * sb + 7) / 8) +
                         4 * (size_t)W + even(((size_t)W + 1) / 2) + 16;
    const size_t block = 4 * (size_t)P.S * n * L;
    return stage > block ? stage : block;
}
__host__ __device__ __forceinline__ size_t djac_lds_doubles(const Params &P, int W, int sb) {
    return djac_table_doubles(P) + djac_stage_doubles(P, W, sb);
}

template <typename PosT, typename OutT, typename ST, int QT, int NA, int SR>
__global__ __launch_bounds__(BSC) void k_djac(Params P, Rows R, const PosT *__restrict__ pos, int W,
                                              OutT *__restrict__ desc, OutT *__restrict__ jself,
                                              ST *__restrict__ c_scratch) {
    extern __shared__ __align__(16) double smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int S = P.S, n = P.n, lmax = P.lmax, lw = lmax + 1, L = P.L, ldN = lmax + 2, Sn = S * n;
    const int nL = n * L, SnL = S * nL, np = (n + 1) / 2;
    constexpr int SB = sizeof(ST);
    Carver cv{smem};
    double *Kl = cv.take(16);
    double *Nt = cv.take((size_t)ldN * ldN);
    double *apr = cv.take((size_t)lw * n);
    double *bcf = cv.take((size_t)lw * n * n);
    double *c0 = cv.take((size_t)n);
    double *e2 = cv.take(128); // 2^(j/64) pairs of exp_neg_tab
    double *stage = cv.take(0);
    const int WP = W + 1, ldl = desc_ldl(n, W);
    Carver sv{stage};
    ST *Yl = (ST *)sv.take(((size_t)L * WP * SB + 7) / 8);  // [lm][W + 1]
    ST *Bl = (ST *)sv.take(((size_t)lw * ldl * SB + 7) / 8); // [l][n][W + 1]
    ST *Hl = (ST *)sv.take(((size_t)lw * ldl * SB + 7) / 8); // [l][n][W + 1]
    double *geo = sv.take(4 * (size_t)W);                    // [W][x, y, z, r]
    int *esp = (int *)sv.take(((size_t)W + 1) / 2);          // species of the chunk's edges
    int *run = (int *)sv.take(16);                           // species run bounds of the chunk
    double *cb = stage;                                      // [c, Dx, Dy, Dz][S][n][L], after the row
    if (tid < 16) Kl[tid] = M_PI * sqrt(8.0 / (double)(2 * tid + 1));
    for (int k = tid; k < ldN * ldN; k += BSC) Nt[k] = P.Nt[k];
    for (int k = tid; k < lw * n; k += BSC) apr[k] = P.aprime[k];
    for (int k = tid; k < lw * n * n; k += BSC) bcf[k] = P.betaC[k];
    for (int k = tid; k < n; k += BSC) c0[k] = P.c0[k];
    for (int k = tid; k < 128; k += BSC) e2[k] = P.e2t[k];

    // this thread's tasks: (lm, radial pair) = (t % L, t / L), t = tid + BSC q,
    // and the gradient of its S_lm: gx = g0 Y'_0 + g1 Y'_1, gy = g2 Y'_2 + g3 Y'_3,
    // gz = g4 Y'_4, Y'_k = the degree l-1 harmonic gi[k] (coefficient 0 where
    // the identity has no term or the order is out of range)
    int lm_q[QT], l_q[QT], a_q[QT], o1_q[QT], gi[QT][5];
    double gc[QT][5];
    bool ok_q[QT];
#pragma unroll
    for (int q = 0; q < QT; ++q) {
        const int t = tid + BSC * q, ap = t / L, lm = t - ap * L;
        int l = (int)sqrtf((float)lm);
        while (l * l > lm) --l;
        while ((l + 1) * (l + 1) <= lm) ++l;
        ok_q[q] = ap < np;
        lm_q[q] = ok_q[q] ? lm : 0;
        l_q[q] = ok_q[q] ? l : 0;
        a_q[q] = ok_q[q] ? 2 * ap : 0;
        o1_q[q] = a_q[q] + 1 < n ? WP : 0;
        const int m = lm_q[q] - l_q[q] * l_q[q] - l_q[q], mm = m < 0 ? -m : m, lp = l_q[q] - 1;
        const int tg = l_q[q] * (l_q[q] + 1) / 2 + mm;
        const double cA = P.gcoef[4 * tg], cB = P.gcoef[4 * tg + 1], cC = P.gcoef[4 * tg + 2];
        int k[5];
        double c[5];
        if (m == 0) {
            k[0] = 1; c[0] = -cA; k[1] = 0; c[1] = 0.0;
            k[2] = -1; c[2] = -cA; k[3] = 0; c[3] = 0.0;
            k[4] = 0; c[4] = cC;
        } else if (m > 0) {
            k[0] = m + 1; c[0] = -cA; k[1] = m - 1; c[1] = cB;
            k[2] = -(m + 1); c[2] = -cA; k[3] = -(m - 1); c[3] = m > 1 ? -cB : 0.0;
            k[4] = m; c[4] = cC;
        } else {
            k[0] = -(mm + 1); c[0] = -cA; k[1] = -(mm - 1); c[1] = mm > 1 ? cB : 0.0;
            k[2] = mm + 1; c[2] = cA; k[3] = mm - 1; c[3] = cB;
            k[4] = -mm; c[4] = cC;
        }
#pragma unroll
        for (int j = 0; j < 5; ++j) {
            const bool in = ok_q[q] && lp >= 0 && k[j] >= -lp && k[j] <= lp;
            gi[q][j] = in ? lp * lp + lp + k[j] : 0;
            gc[q][j] = in ? c[j] : 0.0;
        }
    }
    int64_t ci = blockIdx.x;
    const int64_t stride = gridDim.x;
    double gx = 0.0, gy = 0.0, gz = 0.0;
    int gs = 0;
    int64_t e0 = 0, e1 = 0;
    double3 pi = make_double3(0.0, 0.0, 0.0);
    int spec_i = 0;
    auto gather = [&](int64_t cs, int nb) {
        if (lane < nb) {
            const int64_t j = R.cols[cs + lane];
            gx = (double)pos[3 * j] - pi.x;
            gy = (double)pos[3 * j + 1] - pi.y;
            gz = (double)pos[3 * j + 2] - pi.z;
            gs = R.spec[j];
        }
    };
    auto fetch = [&]() {
        if (ci >= R.nc) return;
        const int64_t i = R.centers ? (int64_t)R.centers[ci] : R.c_base + ci;
        pi = make_double3((double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]);
        spec_i = R.spec[i];
        e0 = R.row_ptr[ci];
        e1 = R.row_ptr[ci + 1];
        gather(e0, (int)((e1 - e0) < W ? (e1 - e0) : W));
    };
    fetch();
    while (ci < R.nc) {
        double acc[SR][QT][2][4];
#pragma unroll
        for (int sr = 0; sr < SR; ++sr)
#pragma unroll
            for (int q = 0; q < QT; ++q)
#pragma unroll
                for (int a = 0; a < 2; ++a)
#pragma unroll
                    for (int d = 0; d < 4; ++d) acc[sr][q][a][d] = 0.0;
        for (int64_t cs = e0; cs < e1; cs += W) {
            const int nb = (int)((e1 - cs) < W ? (e1 - cs) : W);
            if (cs != e0) gather(cs, nb);
            lds_barrier(); // the tables; the previous chunk's (or center's) readers of the staging region
            // ---- staging, lane = edge, tasks over the waves ----
            if (wave == 0) {
                if (lane < nb) {
                    esp[lane] = gs;
                    geo[4 * lane] = gx;
                    geo[4 * lane + 1] = gy;
                    geo[4 * lane + 2] = gz;
                    geo[4 * lane + 3] = sqrt(gx * gx + gy * gy + gz * gz);
                }
                // run bounds: the chunk's edges of species below sr (rows are sorted by species)
#pragma unroll
                for (int sr = 0; sr <= SR; ++sr) {
                    const int cnt = __popcll(__ballot(lane < nb && gs < sr));
                    if (lane == 0) run[sr] = cnt;
                }
            }
            if (lane < nb) {
                const double r2 = gx * gx + gy * gy + gz * gz;
                for (int task = wave; task <= lw; task += NWC) {
                    if (task == lw) {
                        sh_all_any(gx, gy, gz, Nt, ldN, lw, Yl + lane, WP);
                        continue;
                    }
                    const int l = task;
                    // e_k and -2 a'_k e_k: Bh = sum_k betaC (-2 a'_k) e_k
                    double ex[NA], ea[NA];
#pragma unroll
                    for (int k = 0; k < NA; ++k) {
                        const double ap = apr[l * n + (k < n ? k : n - 1)];
                        const double v = exp_neg_tab(ap * r2, e2);
                        ex[k] = k < n ? v : 0.0;
                        ea[k] = -2.0 * ap * ex[k];
                    }
                    ST *bo = Bl + (size_t)l * ldl + lane, *ho = Hl + (size_t)l * ldl + lane;
                    const double *bc = bcf + (size_t)l * n * n;
                    for (int a = 0; a < n; ++a) {
                        double b = 0.0, h = 0.0;
#pragma unroll
                        for (int k = 0; k < NA; ++k) {
                            const double cf = bc[a * n + (k < n ? k : n - 1)];
                            b += cf * ex[k];
                            h += cf * ea[k];
                        }
                        bo[a * WP] = (ST)b;
                        ho[a * WP] = (ST)h;
                    }
                }
            }
            lds_barrier();
            // ---- projection, thread = (lm, radial pair), species run by run ----
#pragma unroll
            for (int sr = 0; sr < SR; ++sr) {
                const int lo = run[sr], hi = run[sr + 1];
                // two edges per iteration at one task per thread; at two
                // tasks the second edge's operands would cost the kernel its
                // second wave per SIMD
                constexpr int EU = QT == 1 ? 2 : 1;
#pragma unroll EU
                for (int e = lo; e < hi; ++e) {
                    const double rx = geo[4 * e], ry = geo[4 * e + 1], rz = geo[4 * e + 2];
                    const double live = geo[4 * e + 3] != 0.0 ? 1.0 : 0.0;
#pragma unroll
                    for (int q = 0; q < QT; ++q) {
                        const double y = (double)Yl[lm_q[q] * WP + e];
                        const double t0 = (double)Yl[gi[q][0] * WP + e], t1 = (double)Yl[gi[q][1] * WP + e];
                        const double t2 = (double)Yl[gi[q][2] * WP + e], t3 = (double)Yl[gi[q][3] * WP + e];
                        const double t4 = (double)Yl[gi[q][4] * WP + e];
                        const double dx = live * (gc[q][0] * t0 + gc[q][1] * t1);
                        const double dy = live * (gc[q][2] * t2 + gc[q][3] * t3);
                        const double dz = live * (gc[q][4] * t4);
                        // unconditional loads (a guarded load becomes a branch that waits for
                        // it alone): radial index a_q + 1 past n_max reads index a_q, a sum
                        // that is never written
                        const ST *bp = Bl + (size_t)l_q[q] * ldl + a_q[q] * WP + e;
                        const ST *hp = Hl + (size_t)l_q[q] * ldl + a_q[q] * WP + e;
#pragma unroll
                        for (int a = 0; a < 2; ++a) {
                            const int o = a == 0 ? 0 : o1_q[q];
                            const double b = (double)bp[o];
                            const double hs = (double)hp[o] * y;
                            // two fused steps per component, no separate sum
                            acc[sr][q][a][0] = __builtin_fma(b, y, acc[sr][q][a][0]);
                            acc[sr][q][a][1] = __builtin_fma(b, dx, __builtin_fma(hs, rx, acc[sr][q][a][1]));
                            acc[sr][q][a][2] = __builtin_fma(b, dy, __builtin_fma(hs, ry, acc[sr][q][a][2]));
                            acc[sr][q][a][3] = __builtin_fma(b, dz, __builtin_fma(hs, rz, acc[sr][q][a][3]));
                        }
                    }
                }
            }
        }
        lds_barrier(); // the staging region is read: the coefficient block goes over it
#pragma unroll
        for (int sr = 0; sr < SR; ++sr)
#pragma unroll
            for (int q = 0; q < QT; ++q)
#pragma unroll
                for (int a = 0; a < 2; ++a)
                    if (sr < S && ok_q[q] && a_q[q] + a < n)
#pragma unroll
                        for (int d = 0; d < 4; ++d)
                            cb[(size_t)d * SnL + (sr * n + a_q[q] + a) * L + lm_q[q]] = acc[sr][q][a][d];
        lds_barrier();
        // on-site term of the center (its species, l = 0)
        if (tid < n) cb[(spec_i * n + tid) * L] += c0[tid];
        lds_barrier();
        const int64_t cw = ci;
        ci += stride;
        fetch(); // the next center's first chunk before this center's stores
        power_tiles4<OutT>(cb, SnL, L, 1, Sn, 0, 0, lw, desc + cw * P.F, jself + cw * 3 * P.F, P.F, lw, 0,
                           PairIndex{S, n, 1.0f / (float)n}, wave, NWC, lane, Kl);
        // the coefficients for k_jacobian, [lm][species n], in destination order
        ST *sc = c_scratch + cw * 4 * (size_t)L * Sn;
        for (int it = tid; it < SnL; it += BSC) {
            const int lm = it / Sn, sa = it - lm * Sn;
            sc[it] = (ST)cb[sa * L + lm];
        }
    }
}

// ---------------------------------------------------------------------------
// k_djs: the density step of the Jacobian path with the coefficients
// streamed to scratch.  The layout of k_djac (one center per workgroup of NWC
// waves, chunks of W edges of the row, staging lane = edge, every
// accumulated entry owned by one thread), for the bases whose coefficient
// block c, D does not fit on chip beside the staging (the polynomial basis of
// the multi-species workloads) or whose projection exceeds k_djac's two tasks
// per thread.  A thread's sums hold one species at a time: rows are sorted by
// species, so when the row reaches a new species the sums of the previous one
// go straight to the scratch [c, Dx, Dy, Dz][lm][species n] (each entry
// written once, by its owner; a species without neighbours gets zeros, and c
// of the center's own species its on-site term).  The output kernel then
// writes the power spectrum and the center block from the scratch, and
// k_jacobian reads c from it.
//   staging: the chunk's edge vectors and species (wave 0); the radial
//     factors B_nl, Bh_nl: GTO (RBF 0) from the exponentials as in k_djac,
//     one l per task over the waves; polynomial quadrature (RBF 1) copied
//     from the factors k_radial left for the call's edges, all threads, in
//     the buffer's order; the solid harmonics, their columns m spread over
//     the waves (sh_cols_lane);
//   projection: thread = (radial pair, lm), per edge
//       c_{a lm} += B_al S_lm,  D_{a lm} += Bh_al r S_lm + B_al grad S_lm,
//     each sum in row order (deterministic with no ordering protocol).
// Task t is radial pair t % np of harmonic lm = t / np, so that neighbouring
// threads own neighbouring entries of a scratch row.
// ---------------------------------------------------------------------------
// the real solid harmonics of columns m = m0, m0 + ms, ... (lane = edge; the
// column recurrence of sh_all_lane, (x + i y)^m advanced by (x + i y)^ms)
template <typename YT>
__device__ __forceinline__ void sh_cols_lane(double x, double y, double z, const double *__restrict__ Nt, int ldN,
                                             int lw, YT *__restrict__ Y, int ls, int m0, int ms) {
    const double r2 = x * x + y * y + z * z;
    double c = 1.0, s = 0.0, cs = 1.0, ss = 0.0;
    for (int k = 0; k < m0; ++k) {
        const double cn = x * c - y * s;
        s = x * s + y * c;
        c = cn;
    }
    for (int k = 0; k < ms; ++k) {
        const double cn = x * cs - y * ss;
        ss = x * ss + y * cs;
        cs = cn;
    }
    for (int m = m0; m < lw; m += ms) {
        double R1 = 0.0, R = 1.0; // R_{l-1}, R_l
        for (int l = m; l < lw; ++l) {
            if (l > m) {
                const double a = (double)(2 * l - 1), b = (double)((l + m - 1) * (l - m - 1));
                const double Rn = a * z * R - b * r2 * R1;
                R1 = R;
                R = Rn;
            }
            const double v = Nt[l * ldN + m] * R;
            const int o = l * l + l;
            if (m == 0) {
                Y[o * ls] = (YT)v;
            } else {
                Y[(o + m) * ls] = (YT)(v * c);
                Y[(o - m) * ls] = (YT)(v * s);
            }
        }
        const double cn = c * cs - s * ss;
        s = c * ss + s * cs;
        c = cn;
    }
}

// LDS doubles of k_djs: tables (Nt, on-site terms; GTO: a', betaC), then the
// staging (harmonics [lm][W+1], B and Bh [l][n][W+1] with odd row lengths,
// edge vectors [W][4], species [W], species run bounds)
__host__ __device__ __forceinline__ size_t djs_lds_doubles(const Params &P, int W, int sb) {
    const size_t ldN = (size_t)P.lmax + 2, lw = (size_t)P.lmax + 1, n = (size_t)P.n, L = (size_t)P.L;
    const size_t tables = even(ldN * ldN) + even(n) + (P.rbf == 0 ? even(lw * n) + even(lw * n * n) : 0);
    return tables + even((L * (W + 1) * sb + 7) / 8) + 2 * even((lw * desc_ldl((int)n, W) * sb + 7) / 8) +
           4 * (size_t)W + even(((size_t)W + 1) / 2) + 16;
}
// (radial pair, lm) tasks per thread
__host__ __device__ __forceinline__ int djs_tasks(const Params &P) {
    return (P.L * ((P.n + 1) / 2) + BSC - 1) / BSC;
}

template <typename PosT, typename ST, int QT, int NA, int RBF>
__global__ __launch_bounds__(BSC) void k_djs(Params P, Rows R, const PosT *__restrict__ pos, int W,
                                             ST *__restrict__ c_scratch) {
    extern __shared__ __align__(16) double smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int S = P.S, n = P.n, lmax = P.lmax, lw = lmax + 1, L = P.L, ldN = lmax + 2, Sn = S * n;
    const int np = (n + 1) / 2;
    constexpr int SB = sizeof(ST);
    Carver cv{smem};
    double *Nt = cv.take((size_t)ldN * ldN);
    double *c0 = cv.take((size_t)n);
    double *apr = RBF == 0 ? cv.take((size_t)lw * n) : nullptr;
    double *bcf = RBF == 0 ? cv.take((size_t)lw * n * n) : nullptr;
    const int WP = W + 1, ldl = desc_ldl(n, W);
    ST *Yl = (ST *)cv.take(((size_t)L * WP * SB + 7) / 8);  // [lm][W + 1]
    ST *Bl = (ST *)cv.take(((size_t)lw * ldl * SB + 7) / 8); // [l][n][W + 1]
    ST *Hl = (ST *)cv.take(((size_t)lw * ldl * SB + 7) / 8); // [l][n][W + 1]
    double *geo = cv.take(4 * (size_t)W);                    // [W][x, y, z, r]
    int *run = (int *)cv.take(16);                           // species run bounds of the chunk
    for (int k = tid; k < ldN * ldN; k += BSC) Nt[k] = P.Nt[k];
    for (int k = tid; k < n; k += BSC) c0[k] = P.c0[k];
    if constexpr (RBF == 0) {
        for (int k = tid; k < lw * n; k += BSC) apr[k] = P.aprime[k];
        for (int k = tid; k < lw * n * n; k += BSC) bcf[k] = P.betaC[k];
    }
    lds_barrier(); // the tables (a center without neighbours reads the on-site terms before any chunk)

    // this thread's tasks: (radial pair, lm) = (t % np, t / np), t = tid + BSC q,
    // and the gradient of its S_lm (as in k_djac)
    int lm_q[QT], l_q[QT], a_q[QT], o1_q[QT], gi[QT][5];
    double gc[QT][5];
    bool ok_q[QT];
#pragma unroll
    for (int q = 0; q < QT; ++q) {
        const int t = tid + BSC * q, lm = t / np, ap = t - lm * np;
        int l = (int)sqrtf((float)lm);
        while (l * l > lm) --l;
        while ((l + 1) * (l + 1) <= lm) ++l;
        ok_q[q] = lm < L;
        lm_q[q] = ok_q[q] ? lm : 0;
        l_q[q] = ok_q[q] ? l : 0;
        a_q[q] = ok_q[q] ? 2 * ap : 0;
        o1_q[q] = a_q[q] + 1 < n ? WP : 0;
        const int m = lm_q[q] - l_q[q] * l_q[q] - l_q[q], mm = m < 0 ? -m : m, lp = l_q[q] - 1;
        const int tg = l_q[q] * (l_q[q] + 1) / 2 + mm;
        const double cA = P.gcoef[4 * tg], cB = P.gcoef[4 * tg + 1], cC = P.gcoef[4 * tg + 2];
        int k[5];
        double c[5];
        if (m == 0) {
            k[0] = 1; c[0] = -cA; k[1] = 0; c[1] = 0.0;
            k[2] = -1; c[2] = -cA; k[3] = 0; c[3] = 0.0;
            k[4] = 0; c[4] = cC;
        } else if (m > 0) {
            k[0] = m + 1; c[0] = -cA; k[1] = m - 1; c[1] = cB;
            k[2] = -(m + 1); c[2] = -cA; k[3] = -(m - 1); c[3] = m > 1 ? -cB : 0.0;
            k[4] = m; c[4] = cC;
        } else {
            k[0] = -(mm + 1); c[0] = -cA; k[1] = -(mm - 1); c[1] = mm > 1 ? cB : 0.0;
            k[2] = mm + 1; c[2] = cA; k[3] = mm - 1; c[3] = cB;
            k[4] = -mm; c[4] = cC;
        }
#pragma unroll
        for (int j = 0; j < 5; ++j) {
            const bool in = ok_q[q] && lp >= 0 && k[j] >= -lp && k[j] <= lp;
            gi[q][j] = in ? lp * lp + lp + k[j] : 0;
            gc[q][j] = in ? c[j] : 0.0;
        }
    }
    const int per = n * lw;
    const float inv_per = 1.0f / (float)per, inv_lw = 1.0f / (float)lw;
    int64_t ci = blockIdx.x;
    const int64_t stride = gridDim.x;
    double gx = 0.0, gy = 0.0, gz = 0.0;
    int gs = 0;
    int64_t e0 = 0, e1 = 0;
    double3 pi = make_double3(0.0, 0.0, 0.0);
    int spec_i = 0;
    auto gather = [&](int64_t cs, int nb) {
        if (lane < nb) {
            const int64_t j = R.cols[cs + lane];
            gx = (double)pos[3 * j] - pi.x;
            gy = (double)pos[3 * j + 1] - pi.y;
            gz = (double)pos[3 * j + 2] - pi.z;
            gs = R.spec[j];
        }
    };
    auto fetch = [&]() {
        if (ci >= R.nc) return;
        const int64_t i = R.centers ? (int64_t)R.centers[ci] : R.c_base + ci;
        pi = make_double3((double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]);
        spec_i = R.spec[i];
        e0 = R.row_ptr[ci];
        e1 = R.row_ptr[ci + 1];
        gather(e0, (int)((e1 - e0) < W ? (e1 - e0) : W));
    };
    fetch();
    while (ci < R.nc) {
        double acc[QT][2][4];
        const int64_t cw = ci;
        const int spec_c = spec_i;
        ST *sc = c_scratch + cw * 4 * (size_t)L * Sn; // [c, Dx, Dy, Dz][lm][species n]
        // the sums of species s (or zeros) to the scratch; c of the center's
        // own species gets the on-site term
        auto flush = [&](int s, bool sums) {
#pragma unroll
            for (int q = 0; q < QT; ++q)
#pragma unroll
                for (int a = 0; a < 2; ++a)
                    if (ok_q[q] && a_q[q] + a < n) {
                        ST *o = sc + (size_t)lm_q[q] * Sn + s * n + a_q[q] + a;
#pragma unroll
                        for (int d = 0; d < 4; ++d) {
                            double v = sums ? acc[q][a][d] : 0.0;
                            if (d == 0 && s == spec_c && lm_q[q] == 0) v += c0[a_q[q] + a];
                            o[(size_t)d * L * Sn] = (ST)v;
                        }
                    }
        };
#pragma unroll
        for (int q = 0; q < QT; ++q)
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int d = 0; d < 4; ++d) acc[q][a][d] = 0.0;
        int cur = 0; // the species the sums hold
        for (int64_t cs = e0; cs < e1; cs += W) {
            const int nb = (int)((e1 - cs) < W ? (e1 - cs) : W);
            if (cs != e0) gather(cs, nb);
            lds_barrier(); // the tables; the previous chunk's (or center's) readers of the staging region
            // ---- staging, lane = edge ----
            if (wave == 0) {
                if (lane < nb) {
                    geo[4 * lane] = gx;
                    geo[4 * lane + 1] = gy;
                    geo[4 * lane + 2] = gz;
                    geo[4 * lane + 3] = sqrt(gx * gx + gy * gy + gz * gz);
                }
                // run bounds: the chunk's edges of species below s (rows are sorted by species)
                for (int s = 0; s <= S; ++s) {
                    const int cnt = __popcll(__ballot(lane < nb && gs < s));
                    if (lane == 0) run[s] = cnt;
                }
            }
            if constexpr (RBF == 1) {
                // the chunk's radial factors, [edge][n][l] in the buffer, contiguous over the chunk
                const double2 *rad = P.rad + (cs - P.rad_e0) * (size_t)per;
                for (int k = tid; k < nb * per; k += BSC) {
                    const int e = qdiv(k, inv_per), t = k - e * per, a = qdiv(t, inv_lw), l = t - a * lw;
                    const double2 v = rad[k];
                    Bl[l * ldl + a * WP + e] = (ST)v.x;
                    Hl[l * ldl + a * WP + e] = (ST)v.y;
                }
            }
            if (lane < nb) {
                if constexpr (RBF == 0) {
                    const double r2 = gx * gx + gy * gy + gz * gz;
                    for (int l = wave; l < lw; l += NWC) {
                        // e_k and -2 a'_k e_k: Bh = sum_k betaC (-2 a'_k) e_k
                        double ex[NA], ea[NA];
#pragma unroll
                        for (int k = 0; k < NA; ++k) {
                            const double ap = apr[l * n + (k < n ? k : n - 1)];
                            ex[k] = k < n ? exp(-ap * r2) : 0.0;
                            ea[k] = -2.0 * ap * ex[k];
                        }
                        ST *bo = Bl + (size_t)l * ldl + lane, *ho = Hl + (size_t)l * ldl + lane;
                        const double *bc = bcf + (size_t)l * n * n;
                        for (int a = 0; a < n; ++a) {
                            double b = 0.0, h = 0.0;
#pragma unroll
                            for (int k = 0; k < NA; ++k) {
                                const double cf = bc[a * n + (k < n ? k : n - 1)];
                                b += cf * ex[k];
                                h += cf * ea[k];
                            }
                            bo[a * WP] = (ST)b;
                            ho[a * WP] = (ST)h;
                        }
                    }
                }
                sh_cols_lane(gx, gy, gz, Nt, ldN, lw, Yl + lane, WP, wave, NWC);
            }
            lds_barrier();
            // ---- projection, thread = (radial pair, lm), species run by run ----
            for (int s = 0; s < S; ++s) {
                const int lo = run[s], hi = run[s + 1];
                if (lo == hi) continue; // uniform
                if (s != cur) {
                    flush(cur, true);
                    for (int z = cur + 1; z < s; ++z) flush(z, false);
                    cur = s;
#pragma unroll
                    for (int q = 0; q < QT; ++q)
#pragma unroll
                        for (int a = 0; a < 2; ++a)
#pragma unroll
                            for (int d = 0; d < 4; ++d) acc[q][a][d] = 0.0;
                }
                for (int e = lo; e < hi; ++e) {
                    const double rx = geo[4 * e], ry = geo[4 * e + 1], rz = geo[4 * e + 2];
                    const double live = geo[4 * e + 3] != 0.0 ? 1.0 : 0.0;
#pragma unroll
                    for (int q = 0; q < QT; ++q) {
                        const double y = (double)Yl[lm_q[q] * WP + e];
                        const double t0 = (double)Yl[gi[q][0] * WP + e], t1 = (double)Yl[gi[q][1] * WP + e];
                        const double t2 = (double)Yl[gi[q][2] * WP + e], t3 = (double)Yl[gi[q][3] * WP + e];
                        const double t4 = (double)Yl[gi[q][4] * WP + e];
                        const double dx = live * (gc[q][0] * t0 + gc[q][1] * t1);
                        const double dy = live * (gc[q][2] * t2 + gc[q][3] * t3);
                        const double dz = live * (gc[q][4] * t4);
                        // unconditional loads: radial index a_q + 1 past n_max reads
                        // index a_q, a sum that is never written
                        const ST *bp = Bl + (size_t)l_q[q] * ldl + a_q[q] * WP + e;
                        const ST *hp = Hl + (size_t)l_q[q] * ldl + a_q[q] * WP + e;
#pragma unroll
                        for (int a = 0; a < 2; ++a) {
                            const int o = a == 0 ? 0 : o1_q[q];
                            const double b = (double)bp[o];
                            const double hs = (double)hp[o] * y;
                            acc[q][a][0] += b * y;
                            acc[q][a][1] += hs * rx + b * dx;
                            acc[q][a][2] += hs * ry + b * dy;
                            acc[q][a][3] += hs * rz + b * dz;
                        }
                    }
                }
            }
        }
        ci += stride;
        fetch(); // the next center's first chunk before this center's last stores
        flush(cur, true);
        for (int z = cur + 1; z < S; ++z) flush(z, false);
    }
}

// ---------------------------------------------------------------------------
// k_outputs: power spectrum and center block for the Jacobian path, from the
// coefficients c and D that k_density left in scratch
// ([center][c, Dx, Dy, Dz][lm][species n]).  One workgroup per center.  Per
// l-group of O (usually one group covering every l), the four slabs (c, Dx,
// Dy, Dz) of the group go to LDS in one pass (all loads in flight together),
// the matrix-core tiles of the four output rows (descriptor, d/dx, d/dy,
// d/dz) fill LDS copies of the rows, spread evenly over the waves, and the
// rows leave in whole, contiguous lines.  One load phase and one store
// phase per group: the kernel is latency-bound, not bandwidth-bound.
// ---------------------------------------------------------------------------
constexpr int BSO = 256;

__host__ __device__ __forceinline__ size_t outputs_group_doubles(const Params &P, int lg0, int lg1, int out_bytes) {
    const size_t Sn = (size_t)P.S * P.n, slab = (size_t)(lg1 * lg1 - lg0 * lg0) * Sn;
    return 4 * even(slab) + 4 * even(((size_t)P.nq_full * (lg1 - lg0) * out_bytes + 7) / 8);
}

template <typename OutT, typename ST = OutT>
__global__ __launch_bounds__(BSO) void k_outputs(Params P, OutPlan O, const ST *__restrict__ scratch,
                                                 OutT *__restrict__ desc, OutT *__restrict__ jself) {
    extern __shared__ __align__(16) double smem[];
    __shared__ double Kl[16];
    const int64_t ci = blockIdx.x;
    const int S = P.S, n = P.n, Sn = S * n, L = P.L, lw = P.lmax + 1, nq = P.nq_full, F = P.F, tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    constexpr int NW = BSO / 64;
    if (tid < 16) Kl[tid] = M_PI * sqrt(8.0 / (double)(2 * tid + 1));
    double *base = smem;
    const PairIndex pq{P.S, P.n, 1.0f / (float)P.n};
    const ST *src = scratch + ci * 4 * (size_t)L * Sn;
    OutT *drow = desc + ci * F, *jrow = jself + ci * 3 * F; // jself rows d = 0..2 are consecutive
    for (int g = 0; g < O.n_groups; ++g) {
        const int lg0 = O.lgrp[g], lg1 = O.lgrp[g + 1], lgc = lg1 - lg0, lm0 = lg0 * lg0;
        const int slab = (lg1 * lg1 - lm0) * Sn, sstr = (int)even((size_t)slab);
        const int rlen = nq * lgc, rstr = (int)even(((size_t)rlen * sizeof(OutT) + 7) / 8) * (8 / (int)sizeof(OutT));
        double *X = base;                        // [comp][slab], comp = c, Dx, Dy, Dz
        OutT *rows = (OutT *)(base + 4 * sstr);  // [row][rlen], row = descriptor, d/dx, d/dy, d/dz
        // the four slabs, eight loads in flight per thread (the barrier after
        // them also orders the previous group's row reads before the tiles)
        for (int k0 = 0; k0 < 4 * slab; k0 += 8 * BSO) {
            double v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int k = k0 + u * BSO + tid, kk = k < 4 * slab ? k : 4 * slab - 1;
                const int comp = kk / slab, r = kk - comp * slab;
                v[u] = src[((size_t)comp * L + lm0) * Sn + r];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int k = k0 + u * BSO + tid;
                if (k < 4 * slab) {
                    const int comp = k / slab, r = k - comp * slab;
                    X[comp * sstr + r] = v[u];
                }
            }
        }
        lds_barrier();
        power_tiles4<OutT>(X, sstr, 1, Sn, Sn, lm0, lg0, lgc, rows, rows + rstr, rstr, lgc, lg0, pq, wave, NW, lane,
                           Kl);
        lds_barrier();
        if (lgc == lw) {
            for (int f = tid; f < F; f += BSO) drow[f] = rows[f];
            for (int f = tid; f < 3 * F; f += BSO) {
                const int d = f >= F ? (f >= 2 * F ? 2 : 1) : 0;
                jrow[f] = rows[(d + 1) * rstr + (f - d * F)];
            }
        } else {
            for (int t = tid; t < 4 * rlen; t += BSO) {
                const int c = t / rlen, r = t - c * rlen, q = r / lgc, lc = r - q * lgc;
                OutT *dst = c == 0 ? drow : jrow + (size_t)(c - 1) * F;
                dst[q * lw + lg0 + lc] = rows[c * rstr + r];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// k_outputs_rows: the output kernel for bases whose c and one component of D
// (every l) fit in LDS beside one output row.  One workgroup of NWO waves per
// center, four passes: the power spectrum from c, then the three components
// of the center block from c and D_x, D_y, D_z (power_tiles).  c stays in LDS
// for all four; the next component of D is loaded into registers while the
// current pass runs its tiles.  Each pass leaves one whole output row in LDS,
// which goes out in contiguous lines (an l-group split writes part of every
// line of a row per group).
// ---------------------------------------------------------------------------
constexpr int NWO = 8, BSO2 = 64 * NWO;
constexpr int OUT_PF = 24; // prefetched doubles per thread: one slab of at most OUT_PF * BSO2

// sb: bytes per staged coefficient (ST)
// the pair-index table of k_outputs_rows, in doubles: kept for up to five 16-row
// tiles (S n <= 80: at most 15 tile pairs, 7.5 KB), else the indices are
// computed per item
__host__ __device__ __forceinline__ size_t outputs_qtab_doubles(const Params &P) {
    const size_t ntile = ((size_t)P.S * P.n + 15) / 16, ntp = ntile * (ntile + 1) / 2;
    return (ntile > 1 && ntile <= 5) ? ntp * 64 : 0;
}
__host__ __device__ __forceinline__ size_t outputs_rows_doubles(const Params &P, int out_bytes, int sb) {
    const size_t slab = (size_t)P.L * P.S * P.n;
    // c, one component of D, a row, the pair-index table
    return 2 * even((slab * sb + 7) / 8) + even(((size_t)P.F * out_bytes + 7) / 8) + outputs_qtab_doubles(P);
}

// ST: precision of the staged c and D (float64, or float32 in the mixed mode;
// the products and sums stay float64 on the matrix cores)
template <typename OutT, typename ST>
__global__ __launch_bounds__(BSO2) void k_outputs_rows(Params P, const ST *__restrict__ scratch,
                                                       OutT *__restrict__ desc, OutT *__restrict__ jself) {
    extern __shared__ __align__(16) double smem[];
    __shared__ double Kl[16];
    const int64_t ci = blockIdx.x;
    const int S = P.S, n = P.n, Sn = S * n, lw = P.lmax + 1, F = P.F, tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int slab = P.L * Sn, sstr = (int)even(((size_t)slab * sizeof(ST) + 7) / 8);
    if (tid < 16) Kl[tid] = M_PI * sqrt(8.0 / (double)(2 * tid + 1));
    ST *Xc = (ST *)smem, *Xd = (ST *)(smem + sstr);
    OutT *row = (OutT *)(smem + 2 * sstr);
    const int rstr = (int)even(((size_t)F * sizeof(OutT) + 7) / 8);
    // [tile pair][lane][4], built below, read after the barrier (NULL: computed per item)
    short *qtab = outputs_qtab_doubles(P) ? (short *)(smem + 2 * sstr + rstr) : nullptr;
    const ST *src = scratch + ci * 4 * (size_t)slab; // [c, Dx, Dy, Dz][lm][species n]
    // c and D_x, eight loads in flight per thread
    for (int k0 = 0; k0 < 2 * slab; k0 += 8 * BSO2) {
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int k = k0 + u * BSO2 + tid;
            v[u] = src[k < 2 * slab ? k : 0];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int k = k0 + u * BSO2 + tid;
            if (k < 2 * slab) (k < slab ? Xc[k] : Xd[k - slab]) = (ST)v[u];
        }
    }
    const PairIndex pq{S, n, 1.0f / (float)n};
    if (qtab) pair_index_table(pq, Sn, qtab, tid, BSO2);
    lds_barrier();
    for (int p = 0; p < 4; ++p) {
        ST pf[OUT_PF];
        if (p == 1 || p == 2) {
            const ST *nx = src + (size_t)(p + 1) * slab;
#pragma unroll
            for (int u = 0; u < OUT_PF; ++u) {
                const int k = u * BSO2 + tid;
                pf[u] = nx[k < slab ? k : 0];
            }
        }
        power_tiles<OutT, ST>(CoefView<ST>{Xc, Xd, 1, Sn}, p - 1, Sn, 0, 0, lw, row, lw, 0, pq, wave, NWO, lane, Kl,
                              qtab);
        lds_barrier(); // the row is complete; D of this pass is read
        OutT *dst = p == 0 ? desc + ci * F : jself + (ci * 3 + (p - 1)) * F;
        for (int f = tid; f < F; f += BSO2) dst[f] = row[f];
        if (p == 1 || p == 2) {
#pragma unroll
            for (int u = 0; u < OUT_PF; ++u) {
                const int k = u * BSO2 + tid;
                if (k < slab) Xd[k] = (ST)pf[u];
            }
        }
        lds_barrier(); // the row is read and the next D is in place before the next pass
    }
}

// ---------------------------------------------------------------------------
// Averaged modes: column means over the centers (float64 sums in row chunks,
// then the chunk sums) and the power spectrum of one coefficient set.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_colsum_partial(const T *__restrict__ in, int64_t rows, int64_t cols,
                                                        int64_t chunk_rows, double *__restrict__ part) {
    const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x, ch = blockIdx.y;
    if (col >= cols) return;
    const int64_t r0 = ch * chunk_rows, r1 = r0 + chunk_rows < rows ? r0 + chunk_rows : rows;
    double s = 0.0;
    for (int64_t r = r0; r < r1; ++r) s += (double)in[r * cols + col];
    part[ch * cols + col] = s;
}

template <typename T>
__global__ __launch_bounds__(256) void k_colmean_finish(const double *__restrict__ part, int nchunk, int64_t cols,
                                                        int64_t rows, T *__restrict__ out, double *__restrict__ mean) {
    const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (col >= cols) return;
    double s = 0.0;
    for (int k = 0; k < nchunk; ++k) s += part[(int64_t)k * cols + col];
    const double m = s / (double)rows;
    mean[col] = m;
    if (out) out[col] = (T)m;
}

// one workgroup: Eq. (powerspectrum) of c[S][n][L] (float64) into out[F]
template <typename OutT>
__global__ __launch_bounds__(256) void k_power_single(Params P, const double *__restrict__ c, OutT *__restrict__ out) {
    extern __shared__ __align__(16) double smem[];
    __shared__ double Kl[16];
    const int Sn = P.S * P.n, L = P.L, tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    if (tid < 16) Kl[tid] = M_PI * sqrt(8.0 / (double)(2 * tid + 1));
    copy_to_lds<256, 4>(smem, c, Sn * L, tid);
    lds_barrier();
    power_tiles<OutT>(CoefView<double>{smem, nullptr, L, 1}, -1, Sn, 0, 0, P.lmax + 1, out, P.lmax + 1, 0,
                      PairIndex{P.S, P.n, 1.0f / (float)P.n}, wave, 4,
                      lane, Kl);
}

// ---------------------------------------------------------------------------
// k_jacobian
//
// One workgroup of NWJ waves per center.  The workgroup shares the basis
// tables, the center's coefficients (transposed, cT[lm][u], u = species * n
// + n') and the prefetched neighbour rows; each wave then runs its own
// pipeline over tiles of W <= 4 edges, synchronising only within the wave:
//
//   1. harmonics S_lm and grad S_lm, radial factors K_l B_nl and K_l Bh_nl;
//   2. the precontraction U^u_l = sum_m S_lm c^u_lm, V^u_l = sum_m grad S_lm
//      c^u_lm on the matrix cores: per l, a 16 x 16 x 4 float64 MFMA chain
//      with A rows (component, edge) = (S, dS/dx, dS/dy, dS/dz) of up to four
//      edges, K = m (2l + 1 padded to a multiple of 4), B columns = u;
//   3. assembly of the neighbour block of each edge j (species s), whose
//      slots are the features with s in their species pair, in feature
//      order: pairs (mu, s), mu < s; the diagonal pair (s, s), n' >= n;
//      pairs (s, nu), nu > s.  With r = r_j - r_i,
//        (mu, s):  K_l [U^mu_nl Bh_n'l r + V^mu_nl B_n'l]
//        (s, nu):  K_l [Bh_nl r U^nu_n'l + B_nl V^nu_n'l]
//        (s, s):   both of the above with mu = nu = s
//      (Eq. powerspectrum-derivative).  On the off-diagonal pairs a lane owns
//      one (n', l) and walks n, so consecutive lanes store consecutive
//      floats; the diagonal triangle is walked flat with a decode table.
// ---------------------------------------------------------------------------
constexpr int NWJ = 4, BSJ = 64 * NWJ;
constexpr int JAC_MAX_W = 4;  // edges per MFMA tile: A rows are (component, edge)
constexpr int JAC_MAX_NP = 4; // lanes passes over (n', l): n * (l_max + 1) <= 256
constexpr int JB = 8;         // MFMA operand pairs loaded ahead of their chain


// The assembly works at the output precision (ab = 4 or 8 bytes): U/V and
// B/Bh are rounded once to it, which keeps the float32 kernel's LDS small
// enough for three workgroups per CU.
__host__ __device__ __forceinline__ size_t jac_xu_doubles(const Params &P, int ab) {
    const size_t lw = (size_t)P.lmax + 1, Sn = (size_t)P.S * P.n;
    const size_t xd = stage_x_doubles(P, (int)lw, (int)lw), ud = 4 * Sn * lw * ab / 8;
    return xd > ud ? xd : ud;
}

__host__ __device__ __forceinline__ size_t jac_wave_doubles(const Params &P, int W, int ab) {
    const size_t L = (size_t)P.L, lw = (size_t)P.lmax + 1;
    return even(W * 4 * L) + even(2 * W * P.n * lw * ab / 8) + even(W * jac_xu_doubles(P, ab));
}

// o: wave-uniform row base; idx: per-lane offset (unsigned, so the stores
// can take the scalar-base + 32-bit-offset form)
template <typename T, typename V>
__device__ __forceinline__ void store3(T *o, uint32_t Fe, uint32_t idx, V x, V y, V z) {
    store_out(o + idx, x);
    store_out(o + (Fe + idx), y);
    store_out(o + (2 * Fe + idx), z);
}

// float64 edge blocks are stored 16 bytes (two values) per lane and row.
// For float32 output, 8- and 16-byte stores measured slower than one value
// per lane (the per-slot decode and the strided LDS reads cost more than the
// wider stores save), so only the float64 kernels carry this path.
typedef double jv_f64x2 __attribute__((ext_vector_type(2)));
template <typename T> struct Vec16;
template <> struct Vec16<double> {
    using type = jv_f64x2;
    static constexpr int N = 2;
};
template <typename T> constexpr bool jac_vector_stores() { return sizeof(T) == 8; }
template <typename T, typename V = typename Vec16<T>::type>
__device__ __forceinline__ void store3v(T *o, uint32_t Fe, uint32_t idx, const V &x, const V &y, const V &z) {
    *(V *)(o + idx) = x;
    *(V *)(o + (Fe + idx)) = y;
    *(V *)(o + (2 * Fe + idx)) = z;
}
// next slot (n, n' lw + l) of an off-diagonal pair block, nl = n_max lw
__device__ __forceinline__ void jac_next_slot(int &a, int &tt, int &l, int nl, int lw) {
    ++tt;
    ++l;
    if (l == lw) l = 0;
    if (tt == nl) {
        tt = 0;
        ++a;
    }
}

// NT, LWT: n_max and l_max + 1 fixed at compile time (0 = from P).  Three
// resident waves per SIMD for the float32 kernel of small bases (its LDS
// allows three workgroups per CU); larger bases keep the registers to avoid
// spills (at l_max 6 from n_max 10 on, the three-wave budget of 168
// registers spilled and ran ~1.4x slower than two waves).
constexpr int jac_min_waves(int ab, int NT, int LWT) {
    return (ab == 4 && (LWT == 0 || LWT <= 5 || (LWT == 7 && NT <= 8))) ? 3 : 2;
}

// RBF: -1 reads the radial basis from P (0..2); 3 is the compensated GTO
// AT: precision of the final assembly (OutT, or double for float64
// arithmetic with float32 outputs).
template <typename PosT, typename OutT, int NT, int LWT, int RBF = -1, typename AT = OutT>
__global__ __launch_bounds__(BSJ, jac_min_waves(sizeof(AT), NT, LWT)) void k_jacobian(Params P, Rows R, const PosT *__restrict__ pos,
                                                                            int W, int vec, const AT *__restrict__ c_scratch,
                                                                            OutT *__restrict__ jedge) {
    using AT2 = typename Pair<AT>::type;
    constexpr int ab = sizeof(AT);
    // 16-byte aligned: the carved regions are read with 16-byte LDS accesses
    extern __shared__ __align__(16) double smem[];
    const int S = P.S, n = NT ? NT : P.n, lw = LWT ? LWT : P.lmax + 1, L = lw * lw, Sn = S * n, tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6); // wave-uniform: scalar control flow
    const int Fe = P.Fe, nl = n * lw, nnl = n * nl, tri_lw = P.tri_lw;
    const int RBk = row_block(NWJ * W);

    Carver cv{smem};
    Tables T;
    load_tables<NT, LWT, RBF>(P, cv, T, 0, lw);
    // [L][Sn] at the assembly precision: in the mixed mode the coefficients
    // enter the (float64) precontraction rounded to float32, which halves the
    // largest LDS table (the bases of four species and l_max 10 then keep
    // two workgroups per CU instead of one)
    AT *cT = (AT *)cv.take(((size_t)Sn * L * ab + 7) / 8);
    double *rgeo = cv.take(4 * (size_t)RBk);
    int *rsp = (int *)cv.take((RBk + 1) / 2);
    uint32_t *dtab = (uint32_t *)cv.take(((size_t)tri_lw + 1) / 2);
    // this wave's private staging
    Carver wv{cv.take(0) + (size_t)wave * jac_wave_doubles(P, W, ab)};
    double *YY = wv.take((size_t)W * 4 * L); // [e][S, dS/dx, dS/dy, dS/dz][L]
    AT2 *BB = (AT2 *)wv.take(2 * (size_t)W * nl * ab / 8); // [e][n][l] = K_l (B, Bh)
    double *XU = wv.take((size_t)W * jac_xu_doubles(P, ab));
    // precontraction results, aliasing the radial scratch: U2a[e][u][l] =
    // (U, Vx), U2b[e][u][l] = (Vy, Vz)
    AT2 *U2a = (AT2 *)XU, *U2b = U2a + (size_t)W * Sn * lw;

    for (int k = tid; k < tri_lw; k += BSJ) dtab[k] = P.dtab[k];

    // lane roles.  MFMA operands: A row (lane & 15) = (component, edge) =
    // (row >> 2, row & 3), B column (lane & 15) = u within the tile, K index
    // lane >> 4; result register r of lane holds row (lane >> 4) + 4 r, i.e.
    // component r of edge lane >> 4.
    const int a_comp = (lane & 15) >> 2, a_e = lane & 3, kk = lane >> 4, bj = lane & 15, o_e = lane >> 4;
    const int ntile = (Sn + 15) >> 4, nj = chunks_below(lw);
    // assembly: lane pass p owns tt = lane + 64 p = n' lw + l
    const float inv_lw = 1.0f / (float)lw, inv_nl = 1.0f / (float)nl;
    const int NP = (nl + 63) >> 6;
    int tp[JAC_MAX_NP], lp[JAC_MAX_NP];
#pragma unroll
    for (int p = 0; p < JAC_MAX_NP; ++p) {
        tp[p] = lane + 64 * p;
        lp[p] = tp[p] - qdiv(tp[p], inv_lw) * lw;
    }

    // One center per workgroup.  (A persistent loop over centers is slower:
    // vmcnt counts loads and stores together, so the next center's row and
    // coefficient loads would wait for all of the previous center's output
    // stores to drain.)
    {
    const int64_t ci = blockIdx.x;
    const int64_t e0 = R.row_ptr[ci], e1 = R.row_ptr[ci + 1], ebase = *R.e_origin;
    if (e1 == e0) return;
    const AT *cg = c_scratch + ci * 4 * (size_t)Sn * L; // component c of [c, Dx, Dy, Dz]
    copy_to_lds<BSJ, 4>(cT, cg, Sn * L, tid);
    const int64_t i = R.centers ? (int64_t)R.centers[ci] : R.c_base + ci;
    const double3 pi = make_double3((double)pos[3 * i], (double)pos[3 * i + 1], (double)pos[3 * i + 2]);

    for (int64_t rb0 = e0; rb0 < e1; rb0 += RBk) {
        const int rbn = (int)((e1 - rb0) < RBk ? (e1 - rb0) : RBk);
        lds_barrier();
        load_rows(rgeo, rsp, pos, R.spec, R.cols, rb0, rbn, pi);
        lds_barrier();
        // full rounds of NWJ tiles of W edges, then the remaining edges split
        // as evenly as possible over the waves (at most W each): the slowest
        // wave, which sets the workgroup's end, carries at most one edge more
        // than the others in the last round instead of a whole tile
        const int FW = NWJ * W, nfull = rbn / FW, rem = rbn - nfull * FW;
        const int rq = rem / NWJ, rr = rem - rq * NWJ, mine = rq + (wave < rr ? 1 : 0);
        const int ntiles = nfull + (mine > 0 ? 1 : 0);
        for (int t = 0; t < ntiles; ++t) { // uniform per wave
            const int off = t < nfull ? t * FW + wave * W : nfull * FW + wave * rq + (wave < rr ? wave : rr);
            const int nb = t < nfull ? W : mine;
            const int64_t base = rb0 + off - ebase; // batch-local edge index
            const double *geo = rgeo + 4 * off;
            const int *spc = rsp + off;
            stage_edges<true, AT, NT, LWT, double, RBF>(P, T, YY, YLayout{4 * L, L, 1, 0}, BB, XU, geo, nb, lane, 0, lw,
                                                        true, rb0 + off);

            // ---- precontraction on the matrix cores ----
            // chunks j = (l, ch) in l-major order, operands loaded JB at a time
            {
                const bool aok = a_e < nb;
                const double *Arow = YY + ((aok ? a_e : 0) * 4 + a_comp) * L;
                for (int t = 0; t < ntile; ++t) {
                    const int u = 16 * t + bj;
                    const bool uok = u < Sn;
                    const int uc = uok ? u : Sn - 1;
                    dbl4 acc = {0.0, 0.0, 0.0, 0.0};
                    int l = 0, ch = 0;
                    for (int j0 = 0; j0 < nj; j0 += JB) {
                        double av[JB], bv[JB];
                        int lq = l, cq = ch;
#pragma unroll
                        for (int q = 0; q < JB; ++q) {
                            const int m = 4 * cq + kk;
                            const bool ok = j0 + q < nj && m <= 2 * lq;
                            const int row = lq * lq + (ok ? m : 0);
                            const double a = Arow[row], b = (double)cT[row * Sn + uc];
                            av[q] = (ok && aok) ? a : 0.0;
                            bv[q] = (ok && uok) ? b : 0.0;
                            if (++cq == (lq >> 1) + 1) {
                                cq = 0;
                                lq = lq + 1 < lw ? lq + 1 : lq;
                            }
                        }
#pragma unroll
                        for (int q = 0; q < JB; ++q) {
                            if (j0 + q < nj) {
                                acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av[q], bv[q], acc, 0, 0, 0);
                                if (++ch == (l >> 1) + 1) {
                                    if (o_e < nb && uok) {
                                        const size_t qq = (size_t)(o_e * Sn + u) * lw + l;
                                        U2a[qq] = Pair<AT>::make(acc[0], acc[1]);
                                        U2b[qq] = Pair<AT>::make(acc[2], acc[3]);
                                    }
                                    acc = dbl4{0.0, 0.0, 0.0, 0.0};
                                    ch = 0;
                                    ++l;
                                }
                            }
                        }
                    }
                }
            }
            wave_sync();

            // ---- assembly and stores ----
            for (int e = 0; e < nb; ++e) {
                const int s = __builtin_amdgcn_readfirstlane(spc[e]);
                const AT rx = (AT)geo[4 * e], ry = (AT)geo[4 * e + 1], rz = (AT)geo[4 * e + 2];
                const AT2 *Be = BB + (size_t)e * nl;
                const AT2 *Ua = U2a + (size_t)e * Sn * lw, *Ub = U2b + (size_t)e * Sn * lw;
                OutT *o = jedge + (base + e) * 3 * Fe;
                if constexpr (jac_vector_stores<OutT>()) if (vec) {
                    // the same slots, a lane owning VN consecutive ones (one
                    // 16-byte store per row); the host enables this when
                    // n nl and tri_lw are multiples of VN and jedge is
                    // 16-byte aligned, so every vector is aligned and whole
                    using OV = typename Vec16<OutT>::type;
                    constexpr int VN = Vec16<OutT>::N;
                    // the lane index made opaque here: the slot decode below
                    // is the same for every edge, and hoisted out of the tile
                    // loops it would hold ~20 registers through the whole kernel
                    int vl = lane;
                    __asm__ volatile("" : "+v"(vl));
                    // pairs (mu, s), mu < s
                    for (int mu = 0; mu < s; ++mu) {
                        const AT2 *Uma = Ua + mu * nl, *Umb = Ub + mu * nl;
                        OutT *ob = o + mu * nnl;
                        for (int g0 = VN * vl; g0 < nnl; g0 += 64 * VN) {
                            int a = qdiv(g0, inv_nl), tt = g0 - a * nl, l = tt - qdiv(tt, inv_lw) * lw;
                            OV vx, vy, vz;
#pragma unroll
                            for (int v = 0; v < VN; ++v) {
                                const AT2 bb = Be[tt], q0 = Uma[a * lw + l], q1 = Umb[a * lw + l];
                                const AT bhx = bb.y * rx, bhy = bb.y * ry, bhz = bb.y * rz;
                                vx[v] = q0.x * bhx + q0.y * bb.x;
                                vy[v] = q0.x * bhy + q1.x * bb.x;
                                vz[v] = q0.x * bhz + q1.y * bb.x;
                                jac_next_slot(a, tt, l, nl, lw);
                            }
                            store3v(ob, Fe, g0, vx, vy, vz);
                        }
                    }
                    // diagonal pair (s, s), n' >= n, flat over (n, n', l)
                    {
                        OutT *ob = o + s * nnl;
                        const AT2 *Usa = Ua + s * nl, *Usb = Ub + s * nl;
                        for (int f0 = VN * vl; f0 < tri_lw; f0 += 64 * VN) {
                            OV vx, vy, vz;
#pragma unroll
                            for (int v = 0; v < VN; ++v) {
                                const uint32_t d = dtab[f0 + v];
                                const int ta = d & 0xffff, tb = d >> 16;
                                const AT2 A = Be[ta], B = Be[tb];
                                const AT2 a0 = Usa[ta], a1 = Usb[ta], b0 = Usa[tb], b1 = Usb[tb];
                                const AT hu = B.y * a0.x + A.y * b0.x;
                                vx[v] = hu * rx + (B.x * a0.y + A.x * b0.y);
                                vy[v] = hu * ry + (B.x * a1.x + A.x * b1.x);
                                vz[v] = hu * rz + (B.x * a1.y + A.x * b1.y);
                            }
                            store3v(ob, Fe, f0, vx, vy, vz);
                        }
                    }
                    // pairs (s, nu), nu > s
                    for (int nu = s + 1; nu < S; ++nu) {
                        const AT2 *Una = Ua + nu * nl, *Unb = Ub + nu * nl;
                        OutT *ob = o + s * nnl + tri_lw + (nu - s - 1) * nnl;
                        for (int g0 = VN * vl; g0 < nnl; g0 += 64 * VN) {
                            int a = qdiv(g0, inv_nl), tt = g0 - a * nl, l = tt - qdiv(tt, inv_lw) * lw;
                            OV vx, vy, vz;
#pragma unroll
                            for (int v = 0; v < VN; ++v) {
                                const AT2 q0 = Una[tt], q1 = Unb[tt], bb = Be[a * lw + l];
                                const AT ux = q0.x * rx, uy = q0.x * ry, uz = q0.x * rz;
                                vx[v] = bb.y * ux + bb.x * q0.y;
                                vy[v] = bb.y * uy + bb.x * q1.x;
                                vz[v] = bb.y * uz + bb.x * q1.y;
                                jac_next_slot(a, tt, l, nl, lw);
                            }
                            store3v(ob, Fe, g0, vx, vy, vz);
                        }
                    }
                    continue;
                }
                // pairs (mu, s), mu < s
                if (s > 0) {
#pragma unroll
                    for (int p = 0; p < JAC_MAX_NP; ++p) {
                        if (p >= NP || tp[p] >= nl) continue;
                        const int tt = tp[p], l = lp[p];
                        const AT2 bb = Be[tt];
                        const AT bhx = bb.y * rx, bhy = bb.y * ry, bhz = bb.y * rz;
                        for (int mu = 0; mu < s; ++mu) {
                            const AT2 *Uma = Ua + mu * nl + l, *Umb = Ub + mu * nl + l;
                            OutT *ob = o + mu * nnl;
                            for (int a = 0; a < n; ++a) {
                                const AT2 q0 = Uma[a * lw], q1 = Umb[a * lw];
                                store3(ob + a * nl, Fe, tt, q0.x * bhx + q0.y * bb.x, q0.x * bhy + q1.x * bb.x,
                                       q0.x * bhz + q1.y * bb.x);
                            }
                        }
                    }
                }
                // diagonal pair (s, s), n' >= n, flat over (n, n', l)
                {
                    OutT *ob = o + s * nnl;
                    const AT2 *Usa = Ua + s * nl, *Usb = Ub + s * nl;
                    for (int f = lane; f < tri_lw; f += 64) {
                        const uint32_t d = dtab[f];
                        const int ta = d & 0xffff, tb = d >> 16; // n lw + l, n' lw + l
                        const AT2 A = Be[ta], B = Be[tb];
                        const AT2 a0 = Usa[ta], a1 = Usb[ta], b0 = Usa[tb], b1 = Usb[tb];
                        const AT hu = B.y * a0.x + A.y * b0.x;
                        store3(ob, Fe, f, hu * rx + (B.x * a0.y + A.x * b0.y), hu * ry + (B.x * a1.x + A.x * b1.x),
                               hu * rz + (B.x * a1.y + A.x * b1.y));
                    }
                }
                // pairs (s, nu), nu > s
                if (s + 1 < S) {
#pragma unroll
                    for (int p = 0; p < JAC_MAX_NP; ++p) {
                        if (p >= NP || tp[p] >= nl) continue;
                        const int tt = tp[p], l = lp[p];
                        for (int nu = s + 1; nu < S; ++nu) {
                            const AT2 q0 = Ua[nu * nl + tt], q1 = Ub[nu * nl + tt];
                            const AT ux = q0.x * rx, uy = q0.x * ry, uz = q0.x * rz;
                            OutT *ob = o + s * nnl + tri_lw + (nu - s - 1) * nnl;
                            const AT2 *Bl = Be + l;
                            for (int a = 0; a < n; ++a) {
                                const AT2 bb = Bl[a * lw];
                                store3(ob + a * nl, Fe, tt, bb.y * ux + bb.x * q0.y, bb.y * uy + bb.x * q1.x,
                                       bb.y * uz + bb.x * q1.y);
                            }
                        }
                    }
                }
            }
            wave_sync();
        }
    }
    } // center
}

// dense[ci][j][3][F]: zero-filled by the caller; each stored block is copied
template <typename OutT>
__global__ void k_scatter_dense(Params P, Rows R, const OutT *__restrict__ jedge, const OutT *__restrict__ jself,
                                const int32_t *__restrict__ fmap, const int32_t *__restrict__ atom_of,
                                OutT *__restrict__ dense) {
    const int64_t ci = blockIdx.x;
    const int F = P.F, Fe = P.Fe;
    const int64_t i = R.centers ? (int64_t)R.centers[ci] : R.c_base + ci;
    const int64_t ebase = *R.e_origin;
    OutT *row = dense + ci * R.n_atoms * 3 * F;
    for (int k = threadIdx.x; k < 3 * F; k += blockDim.x) row[i * 3 * F + k] = jself[ci * 3 * F + k];
    __syncthreads(); // a periodic image of the center adds to the center block
    // thread k always owns component k / Fe, slot k % Fe, so the blocks of
    // several images of one atom are summed by one thread, in edge order
    for (int64_t e = R.row_ptr[ci]; e < R.row_ptr[ci + 1]; ++e) {
        const int64_t x = R.cols[e], j = atom_of ? (int64_t)atom_of[x] : x;
        const int s = R.spec[x];
        for (int k = threadIdx.x; k < 3 * Fe; k += blockDim.x) {
            const int d = k / Fe, fe = k - d * Fe;
            OutT *o = row + (j * 3 + d) * F + fmap[s * Fe + fe];
            if (atom_of) *o += jedge[((e - ebase) * 3 + d) * Fe + fe];
            else *o = jedge[((e - ebase) * 3 + d) * Fe + fe];
        }
    }
}

} // namespace dev
} // namespace soap
