// Host-side basis constants in 113-bit binary floating point (__float128).
//
// The Loewdin orthonormalisation of both radial bases is severely
// ill-conditioned (Sec. 3.1 notes coefficients of order 1e6 and heavy
// cancellation; the overlap matrices reach condition numbers of 1e15 (GTO,
// r_cut 6, n_max 12) and 1e17 (polynomial, n_max 12)), so the inverse square
// roots and everything that sums Loewdin-weighted terms into a table are
// formed here in quad precision and rounded once to float64.
//
// Compiled by the host C++ compiler only (no device code).
#include "basis.h"

#include <quadmath.h>

#include <cmath>
#include <cstring>
#include <vector>

namespace {

typedef __float128 q128;

const q128 PI_Q = M_PIq;

// Unevaluated sum hi + lo of two __float128 values (about 226 bits), for the
// polynomial overlap matrix, whose condition number reaches 5.6e25 at
// n_max = 16: its inverse square root in 113 bits would keep ~9 digits.
// Error-free transformations: Knuth's two-sum and the fused multiply-add
// product; division and square root by one Newton correction.
struct qq {
    q128 hi = 0, lo = 0;
    qq() = default;
    qq(q128 h) : hi(h), lo(0) {}
    qq(int v) : hi((q128)v), lo(0) {}
    qq(q128 h, q128 l) : hi(h), lo(l) {}
    explicit operator q128() const { return hi + lo; }
};
inline qq fast_sum(q128 a, q128 b) { // |a| >= |b|
    q128 s = a + b;
    return qq(s, b - (s - a));
}
inline qq two_sum(q128 a, q128 b) {
    q128 s = a + b, bb = s - a;
    return qq(s, (a - (s - bb)) + (b - bb));
}
inline qq operator+(const qq &a, const qq &b) {
    qq s = two_sum(a.hi, b.hi), t = two_sum(a.lo, b.lo);
    s.lo += t.hi;
    s = fast_sum(s.hi, s.lo);
    s.lo += t.lo;
    return fast_sum(s.hi, s.lo);
}
inline qq operator-(const qq &a) { return qq(-a.hi, -a.lo); }
inline qq operator-(const qq &a, const qq &b) { return a + (-b); }
inline qq operator*(const qq &a, const qq &b) {
    q128 p = a.hi * b.hi, e = fmaq(a.hi, b.hi, -p);
    e += a.hi * b.lo + a.lo * b.hi;
    return fast_sum(p, e);
}
inline qq operator/(const qq &a, const qq &b) {
    q128 q1 = a.hi / b.hi;
    qq r = a - b * qq(q1);
    q128 q2 = r.hi / b.hi;
    r = r - b * qq(q2);
    q128 q3 = r.hi / b.hi;
    qq q = fast_sum(q1, q2);
    return q + qq(q3);
}
inline qq &operator+=(qq &a, const qq &b) { return a = a + b; }
inline bool operator>=(const qq &a, const qq &b) { return a.hi > b.hi || (a.hi == b.hi && a.lo >= b.lo); }
inline bool operator<=(const qq &a, const qq &b) { return b >= a; }
inline bool operator>(const qq &a, const qq &b) { return !(b >= a); }
inline bool operator==(const qq &a, int b) { return a.hi == (q128)b && a.lo == 0; }
inline qq qsqrt(const qq &a) {
    if (!(a.hi > 0)) return qq(0);
    q128 x = sqrtq(a.hi);
    qq r = a - qq(x) * qq(x);
    return qq(x) + qq(r.hi / (2 * x));
}
inline qq qabs(const qq &a) { return a.hi < 0 ? -a : a; }
inline q128 qsqrt(q128 a) { return sqrtq(a); }
inline q128 qabs(q128 a) { return fabsq(a); }

// off-diagonal / diagonal squared-norm ratio at which the Jacobi sweeps stop
template <typename T> constexpr double jacobi_tol();
template <> constexpr double jacobi_tol<q128>() { return 1e-66; }
template <> constexpr double jacobi_tol<qq>() { return 1e-130; }

// Cyclic Jacobi eigen-decomposition of a symmetric n x n matrix A (row major,
// destroyed).  V receives the eigenvectors as columns, w the eigenvalues.
template <typename T>
bool jacobi_eigen(int n, std::vector<T> &A, std::vector<T> &V, std::vector<T> &w) {
    V.assign((size_t)n * n, T(0));
    for (int i = 0; i < n; ++i) V[(size_t)i * n + i] = T(1);
    const T tol = T((q128)jacobi_tol<T>());
    for (int sweep = 0; sweep < 200; ++sweep) {
        T off = T(0), diag = T(0);
        for (int p = 0; p < n; ++p) {
            diag += A[(size_t)p * n + p] * A[(size_t)p * n + p];
            for (int q = p + 1; q < n; ++q) off += A[(size_t)p * n + q] * A[(size_t)p * n + q];
        }
        if (off <= diag * tol) break;
        for (int p = 0; p < n; ++p)
            for (int q = p + 1; q < n; ++q) {
                T apq = A[(size_t)p * n + q];
                if (apq == 0) continue;
                T app = A[(size_t)p * n + p], aqq = A[(size_t)q * n + q];
                T theta = (aqq - app) / (T(2) * apq);
                T t = T(theta >= T(0) ? 1 : -1) / (qabs(theta) + qsqrt(theta * theta + T(1)));
                T c = T(1) / qsqrt(t * t + T(1)), s = t * c;
                for (int k = 0; k < n; ++k) { // columns p, q
                    T akp = A[(size_t)k * n + p], akq = A[(size_t)k * n + q];
                    A[(size_t)k * n + p] = c * akp - s * akq;
                    A[(size_t)k * n + q] = s * akp + c * akq;
                }
                for (int k = 0; k < n; ++k) { // rows p, q
                    T apk = A[(size_t)p * n + k], aqk = A[(size_t)q * n + k];
                    A[(size_t)p * n + k] = c * apk - s * aqk;
                    A[(size_t)q * n + k] = s * apk + c * aqk;
                }
                for (int k = 0; k < n; ++k) {
                    T vkp = V[(size_t)k * n + p], vkq = V[(size_t)k * n + q];
                    V[(size_t)k * n + p] = c * vkp - s * vkq;
                    V[(size_t)k * n + q] = s * vkp + c * vkq;
                }
            }
    }
    w.resize(n);
    for (int i = 0; i < n; ++i) w[i] = A[(size_t)i * n + i];
    return true;
}

// Principal inverse square root of a symmetric positive-definite matrix.
template <typename T>
bool inv_sqrt_spd(int n, const std::vector<T> &S, std::vector<T> &X) {
    std::vector<T> A = S, V, w;
    jacobi_eigen(n, A, V, w);
    for (int i = 0; i < n; ++i)
        if (!(w[i] > T(0))) return false;
    X.assign((size_t)n * n, T(0));
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j) {
            T acc = T(0);
            for (int k = 0; k < n; ++k) acc += V[(size_t)i * n + k] * V[(size_t)j * n + k] / qsqrt(w[k]);
            X[(size_t)i * n + j] = acc;
        }
    return true;
}

q128 half_int_pow(q128 x, int l) { // x^(l + 3/2)
    return powq(x, (q128)l) * x * sqrtq(x);
}

void set_err(char *err, int errlen, const char *msg) {
    if (err && errlen > 0) {
        std::strncpy(err, msg, (size_t)errlen - 1);
        err[errlen - 1] = 0;
    }
}

} // namespace

extern "C" void soap_exp2_table64(double *t) {
    for (int j = 0; j < 64; ++j) {
        const q128 v = exp2q((q128)j / 64);
        t[2 * j] = (double)v;
        t[2 * j + 1] = (double)(v - (q128)t[2 * j]);
    }
}

extern "C" int soap_basis_gto(double r_cut, int n_max, int l_max, double sigma, double *betaC, double *betaCa,
                              double *aprime, double *c0, char *err, int errlen, double *betaC_lo, double *betaCa_lo,
                              double *aprime_lo) {
    const int n = n_max;
    const q128 rc = r_cut, sg = sigma, s2 = sg * sg;
    std::vector<q128> z(n);
    for (int k = 0; k < n; ++k) z[k] = (n == 1) ? (q128)1 : 1 + (q128)k * (rc - 1) / (q128)(n - 1);
    const q128 ln1000 = logq((q128)1000);
    const q128 pref = powq(2 * PI_Q, (q128)1.5Q) * s2 * sg; // (2 pi)^{3/2} sigma^3
    std::vector<q128> beta0;
    for (int l = 0; l <= l_max; ++l) {
        // Eq. (gto-alphas): alpha_kl = -ln(1e-3 / z_k^l) / z_k^2
        std::vector<q128> al(n);
        for (int k = 0; k < n; ++k) al[k] = (ln1000 + (q128)l * logq(z[k])) / (z[k] * z[k]);
        // Eq. (gto-overlap-approx): Gamma(l+3/2) / (2 (a_k + a_k')^{l+3/2})
        q128 gam = sqrtq(PI_Q);
        for (int j = 0; j <= l; ++j) gam *= ((q128)j + (q128)0.5Q);
        std::vector<q128> S((size_t)n * n), B;
        for (int a = 0; a < n; ++a)
            for (int b = 0; b < n; ++b) S[(size_t)a * n + b] = gam / (2 * half_int_pow(al[a] + al[b], l));
        if (!inv_sqrt_spd(n, S, B)) { // Eq. (gto-lowdin)
            set_err(err, errlen, "GTO overlap matrix is not positive definite");
            return -1;
        }
        if (l == 0) beta0 = B;
        for (int k = 0; k < n; ++k) {
            q128 den = 1 + 2 * s2 * al[k];
            q128 ap = al[k] / den;              // envelope exponent of Eq. (gto-coefficients)
            q128 C = pref / half_int_pow(den, l); // prefactor of Eq. (gto-coefficients)
            aprime[l * n + k] = (double)ap;
            if (aprime_lo) aprime_lo[l * n + k] = (double)(ap - (q128)aprime[l * n + k]);
            for (int a = 0; a < n; ++a) {
                const size_t o = ((size_t)l * n + a) * n + k;
                const q128 bc = B[(size_t)a * n + k] * C, bca = -2 * bc * ap;
                betaC[o] = (double)bc;
                betaCa[o] = (double)bca;
                if (betaC_lo) betaC_lo[o] = (double)(bc - (q128)betaC[o]);
                if (betaCa_lo) betaCa_lo[o] = (double)(bca - (q128)betaCa[o]);
            }
        }
    }
    // on-site term: sqrt(2) pi sigma^3 sum_k beta^0_nk / (1 + 2 sigma^2 alpha_k0)^{3/2}
    for (int a = 0; a < n; ++a) {
        q128 acc = 0;
        for (int k = 0; k < n; ++k) {
            q128 al = ln1000 / (z[k] * z[k]);
            acc += beta0[(size_t)a * n + k] / half_int_pow(1 + 2 * s2 * al, 0);
        }
        c0[a] = (double)(sqrtq((q128)2) * PI_Q * s2 * sg * acc);
    }
    return 0;
}

// Norms N_k of (r_cut - r)^{k+2} (Eq. poly-norm) and the Loewdin weights
// W = S^{-1/2} of their overlap matrix (Eq. poly-overlap), k = 1..n.
// The overlap matrix and its inverse square root are formed in double
// __float128 (qq), then W is rounded to __float128.
static bool poly_weights(q128 rc, int n, std::vector<q128> &N, std::vector<q128> &W, char *err, int errlen) {
    std::vector<qq> S((size_t)n * n), Wq;
    N.assign(n, 0);
    for (int a = 0; a < n; ++a) {
        int k = a + 1;
        N[a] = sqrtq(powq(rc, (q128)(2 * k + 5)) / (q128)(2 * k + 5));
    }
    for (int a = 0; a < n; ++a)
        for (int b = 0; b < n; ++b) {
            int k = a + 1, kp = b + 1;
            S[(size_t)a * n + b] = qsqrt(qq((5 + 2 * k) * (5 + 2 * kp))) / qq(5 + k + kp);
        }
    if (!inv_sqrt_spd(n, S, Wq)) {
        set_err(err, errlen, "polynomial overlap matrix is not positive definite");
        return false;
    }
    W.resize(Wq.size());
    for (size_t i = 0; i < Wq.size(); ++i) W[i] = (q128)Wq[i];
    return true;
}

extern "C" int soap_basis_poly(double r_cut, int n_max, double sigma, int quad_n, double *G, double *rq_out,
                               double *c0, char *err, int errlen) {
    const int n = n_max, Q = quad_n;
    const q128 rc = r_cut, s2 = (q128)sigma * (q128)sigma;
    std::vector<q128> N, W;
    if (!poly_weights(rc, n, N, W, err, errlen)) return -1;
    // Gauss-Legendre nodes on [-1, 1] by Newton iteration on P_Q
    std::vector<q128> t(Q), wt(Q);
    for (int i = 0; i < Q; ++i) {
        q128 x = std::cos(M_PI * (i + 0.75) / (Q + 0.5));
        q128 dp = 1;
        for (int it = 0; it < 100; ++it) {
            q128 p0 = 1, p1 = x;
            for (int k = 2; k <= Q; ++k) {
                q128 p2 = ((2 * k - 1) * x * p1 - (k - 1) * p0) / k;
                p0 = p1;
                p1 = p2;
            }
            dp = (q128)Q * (x * p1 - p0) / (x * x - 1);
            q128 dx = p1 / dp;
            x -= dx;
            if (fabsq(dx) < (q128)1e-33Q) break;
        }
        q128 p0 = 1, p1 = x;
        for (int k = 2; k <= Q; ++k) {
            q128 p2 = ((2 * k - 1) * x * p1 - (k - 1) * p0) / k;
            p0 = p1;
            p1 = p2;
        }
        dp = (q128)Q * (x * p1 - p0) / (x * x - 1);
        t[i] = x;
        wt[i] = 2 / ((1 - x * x) * dp * dp);
    }
    // g_n(r_q) of Eq. (poly-basis), summed in quad; then G[n][q] = 4 pi w_q r_q^2 g_n(r_q)
    const q128 fourpi = 4 * PI_Q;
    std::vector<q128> g((size_t)n * Q), phi(n);
    for (int q = 0; q < Q; ++q) {
        const q128 r = rc * (t[q] + 1) / 2, w = rc * wt[q] / 2, u = rc - r;
        q128 up = u * u * u; // (r_cut - r)^{k+2}, k = 1..n
        for (int b = 0; b < n; ++b, up *= u) phi[b] = up / N[b];
        rq_out[q] = (double)r;
        for (int a = 0; a < n; ++a) {
            q128 acc = 0;
            for (int b = 0; b < n; ++b) acc += W[(size_t)a * n + b] * phi[b];
            g[(size_t)a * Q + q] = acc;
            G[(size_t)a * Q + q] = (double)(fourpi * w * r * r * acc);
        }
    }
    // on-site term: sqrt(4 pi) sum_q w_q r_q^2 g_n(r_q) exp(-r_q^2 / 2 sigma^2)
    for (int a = 0; a < n; ++a) {
        q128 acc = 0;
        for (int q = 0; q < Q; ++q) {
            const q128 r = rc * (t[q] + 1) / 2, w = rc * wt[q] / 2;
            acc += w * r * r * g[(size_t)a * Q + q] * expq(-r * r / (2 * s2));
        }
        c0[a] = (double)(sqrtq(fourpi) * acc);
    }
    return 0;
}

extern "C" int soap_basis_poly_laplace(double r_cut, int n_max, double sigma, double *CH, char *err, int errlen) {
    const int n = n_max, M = n + 3; // P_0 has degree n + 2
    std::vector<q128> N, W;
    if (!poly_weights((q128)r_cut, n, N, W, err, errlen)) return -1;
    const q128 rc = r_cut, s = sigma, pref = powq(2 * PI_Q, (q128)1.5) * s * s * s;
    // P_j(u) = d^j/du^j sum_k WN_k u^{k+2} at the Chebyshev points t_p = cos(pi (p + 1/2) / M)
    std::vector<q128> val((size_t)M * 4);
    for (int a = 0; a < n; ++a) {
        for (int p = 0; p < M; ++p) {
            const q128 t = cosq(PI_Q * ((q128)p + 0.5Q) / (q128)M), u = (t + 1) * rc / 2;
            q128 P[4] = {0, 0, 0, 0}, up = 1; // up = u^{k-1}
            for (int k = 1; k <= n; ++k) {
                const q128 v = pref * W[(size_t)a * n + k - 1] / N[k - 1] * up;
                P[0] += v * u * u * u;
                P[1] += (q128)(k + 2) * v * u * u;
                P[2] += (q128)((k + 1) * (k + 2)) * v * u;
                P[3] += (q128)(k * (k + 1) * (k + 2)) * v;
                up *= u;
            }
            for (int j = 0; j < 4; ++j) val[(size_t)p * 4 + j] = P[j];
        }
        // c_i = (2 - [i = 0]) / M sum_p P(t_p) T_i(t_p)
        for (int i = 0; i < M; ++i)
            for (int j = 0; j < 4; ++j) {
                q128 acc = 0;
                for (int p = 0; p < M; ++p) acc += val[(size_t)p * 4 + j] * cosq(PI_Q * (q128)i * ((q128)p + 0.5Q) / (q128)M);
                CH[((size_t)a * M + i) * 4 + j] = (double)(acc * (i == 0 ? 1 : 2) / (q128)M);
            }
    }
    return 0;
}

// Normalisation of the real solid harmonics: N[l][m] for 0 <= m <= l,
// sqrt((2l+1)/(4 pi) (l-m)!/(l+m)!) times sqrt(2) when m > 0.
extern "C" void soap_basis_sh_norms(int l_max, double *Nlm) {
    for (int l = 0; l <= l_max; ++l)
        for (int m = 0; m <= l; ++m) {
            q128 ratio = 1;
            for (int k = l - m + 1; k <= l + m; ++k) ratio /= (q128)k;
            q128 v = sqrtq((q128)(2 * l + 1) / (4 * PI_Q) * ratio);
            if (m > 0) v *= sqrtq((q128)2);
            Nlm[l * (l_max + 1) + m] = (double)v;
        }
}
