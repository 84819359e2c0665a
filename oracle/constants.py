"""Basis constants for the SOAP oracle, in 50-digit arithmetic (mpmath).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
package; only tests/, the smoke check and the bench's CPU-baseline leg do.

Every quantity is computed from its definition in the paper (Sec. 2):

* GTO radial basis (Sec. 2.2): primitive widths from Eq. (gto-alphas),
  primitive overlap Eq. (gto-overlap-approx) (complete gamma function, i.e. the
  radial range extended to infinity, the same extension the closed-form
  coefficients of Eq. (gto-coefficients) rely on), Loewdin coefficients
  Eq. (gto-lowdin) as the principal inverse square root of the overlap.
* Polynomial radial basis (Sec. 2.3): Eqs. (poly-basis), (poly-norm),
  (poly-overlap), W = S^(-1/2); Gauss-Legendre nodes on [0, r_cut] for the
  radial integral Eq. (poly-radial-integral) (Sec. 3.1 states that these
  integrals use a fixed Gauss-Legendre rule).  The basis function values at
  the nodes, g_n(r_q), are summed in 50 digits: the Loewdin sum is
  ill-conditioned (condition numbers of S reach 1e16-1e17 at n_max 10-12).
* Real solid harmonics r^l Y_lm (the real, DScribe-style harmonics of
  Sec. 2.1) as explicit homogeneous polynomials in x, y, z: m > 0 follows
  cos(m phi), m < 0 follows sin(|m| phi), sqrt(2) normalisation for m != 0,
  no Condon-Shortley phase.

Values are returned as (hi, lo) float64 pairs so the C oracle can rebuild
them in long double.
"""
from __future__ import annotations

import functools
from fractions import Fraction
from math import comb, factorial

import mpmath as mp
import numpy as np

DPS = 50


def _split(x) -> tuple[float, float]:
    hi = float(x)
    lo = float(x - mp.mpf(hi))
    return hi, lo


def _split_array(vals) -> tuple[np.ndarray, np.ndarray]:
    hi = np.array([float(v) for v in vals], dtype=np.float64)
    lo = np.array([float(v - mp.mpf(h)) for v, h in zip(vals, hi)], dtype=np.float64)
    return hi, lo


def inv_sqrt_spd(A: "mp.matrix") -> "mp.matrix":
    """Principal inverse square root of a symmetric positive-definite matrix."""
    E, Q = mp.eigsy(A)
    n = A.rows
    for i in range(n):
        if E[i] <= 0:
            raise ValueError("overlap matrix is not positive definite at %d digits" % mp.mp.dps)
    out = mp.matrix(n, n)
    for i in range(n):
        for j in range(n):
            out[i, j] = mp.fsum(Q[i, k] * Q[j, k] / mp.sqrt(E[k]) for k in range(n))
    return out


# --------------------------------------------------------------------------
# GTO basis: Eqs. (gto-basis), (gto-overlap-approx), (gto-lowdin), (gto-alphas)
# --------------------------------------------------------------------------

@functools.lru_cache(maxsize=64)
def gto_mp(r_cut: float, n_max: int, l_max: int):
    """Return (z[k], alpha[l][k], beta[l] (n x n mp.matrix)), all 50-digit."""
    with mp.workdps(DPS):
        rc = mp.mpf(r_cut)
        if n_max == 1:
            z = [mp.mpf(1)]
        else:
            z = [1 + k * (rc - 1) / (n_max - 1) for k in range(n_max)]
        alpha = [[-mp.log(mp.mpf("1e-3") / zk ** l) / zk ** 2 for zk in z] for l in range(l_max + 1)]
        beta = []
        for l in range(l_max + 1):
            S = mp.matrix(n_max, n_max)
            g = mp.gamma(l + mp.mpf(3) / 2)
            for a in range(n_max):
                for b in range(n_max):
                    S[a, b] = g / (2 * (alpha[l][a] + alpha[l][b]) ** (l + mp.mpf(3) / 2))
            beta.append(inv_sqrt_spd(S))
        return z, alpha, beta


def gto_arrays(r_cut: float, n_max: int, l_max: int) -> dict:
    z, alpha, beta = gto_mp(r_cut, n_max, l_max)
    with mp.workdps(DPS):
        a_flat = [alpha[l][k] for l in range(l_max + 1) for k in range(n_max)]
        b_flat = [beta[l][n, k] for l in range(l_max + 1) for n in range(n_max) for k in range(n_max)]
        ah, al = _split_array(a_flat)
        bh, bl = _split_array(b_flat)
    return dict(alpha_hi=ah, alpha_lo=al, beta_hi=bh, beta_lo=bl)


# --------------------------------------------------------------------------
# Polynomial basis: Eqs. (poly-basis), (poly-norm), (poly-overlap)
# --------------------------------------------------------------------------

@functools.lru_cache(maxsize=64)
def gauss_legendre_mp(q: int):
    """Nodes and weights of the q-point Gauss-Legendre rule on [-1, 1], 50 digits
    (Newton iteration on the three-term Legendre recurrence)."""
    with mp.workdps(DPS + 10):
        xs, ws = [], []
        for i in range(1, q + 1):
            x = mp.cos(mp.pi * (i - mp.mpf(1) / 4) / (q + mp.mpf(1) / 2))
            for _ in range(100):
                p0, p1 = mp.mpf(1), x
                for k in range(2, q + 1):
                    p0, p1 = p1, ((2 * k - 1) * x * p1 - (k - 1) * p0) / k
                dp = q * (x * p1 - p0) / (x * x - 1)
                dx = p1 / dp
                x -= dx
                if abs(dx) < mp.mpf(10) ** (-(DPS + 5)):
                    break
            p0, p1 = mp.mpf(1), x
            for k in range(2, q + 1):
                p0, p1 = p1, ((2 * k - 1) * x * p1 - (k - 1) * p0) / k
            dp = q * (x * p1 - p0) / (x * x - 1)
            xs.append(x)
            ws.append(2 / ((1 - x * x) * dp * dp))
        return xs, ws


@functools.lru_cache(maxsize=64)
def poly_mp(r_cut: float, n_max: int, quad_n: int):
    """Return (N[k], W (mp.matrix), r_q, w_q, g[n][q]) for the polynomial basis."""
    with mp.workdps(DPS):
        rc = mp.mpf(r_cut)
        ks = range(1, n_max + 1)
        N = [mp.sqrt(rc ** (2 * k + 5) / (2 * k + 5)) for k in ks]
        S = mp.matrix(n_max, n_max)
        for a, k in enumerate(ks):
            for b, kp in enumerate(ks):
                S[a, b] = mp.sqrt(mp.mpf((5 + 2 * k) * (5 + 2 * kp))) / (5 + k + kp)
        W = inv_sqrt_spd(S)
        t, w = gauss_legendre_mp(quad_n)
        rq = [rc * (ti + 1) / 2 for ti in t]
        wq = [rc * wi / 2 for wi in w]
        g = [[mp.fsum(W[n, a] * (rc - r) ** (k + 2) / N[a] for a, k in enumerate(ks)) for r in rq]
             for n in range(n_max)]
        return N, W, rq, wq, g


def poly_laplace_arrays(r_cut: float, n_max: int) -> dict:
    """W_nk / N_k of the polynomial basis (Eqs. poly-norm, poly-overlap), the
    coefficients of the Laplace-form radial factors (Eq. poly-coefficients)."""
    N, W, _, _, _ = poly_mp(r_cut, n_max, 2)
    with mp.workdps(DPS):
        wn = [W[a, b] / N[b] for a in range(n_max) for b in range(n_max)]
        h, l = _split_array(wn)
    return dict(wn_hi=h, wn_lo=l)


def poly_arrays(r_cut: float, n_max: int, quad_n: int) -> dict:
    N, W, rq, wq, g = poly_mp(r_cut, n_max, quad_n)
    with mp.workdps(DPS):
        G = [wq[q] * rq[q] ** 2 * g[n][q] for n in range(n_max) for q in range(quad_n)]
        Gh, Gl = _split_array(G)
        rh, rl = _split_array(rq)
    return dict(G_hi=Gh, G_lo=Gl, rq_hi=rh, rq_lo=rl)


# --------------------------------------------------------------------------
# Real solid harmonics as monomial expansions
# --------------------------------------------------------------------------

def _pi_lm(l: int, m: int):
    """Coefficients of r^(l-m) P_l^m(z/r) / (1 - z^2/r^2)^(m/2) (no Condon-Shortley
    phase) as {(power of r^2, power of z): Fraction}."""
    out = {}
    for k in range((l - m) // 2 + 1):
        c = Fraction((-1) ** k * comb(l, k) * comb(2 * l - 2 * k, l) * factorial(l - 2 * k),
                     2 ** l * factorial(l - 2 * k - m))
        out[(k, l - 2 * k - m)] = c
    return out


def _ab_m(m: int, which: str):
    """Re (x + i y)^m ('c') or Im (x + i y)^m ('s') as {(px, py): int}."""
    out = {}
    for p in range(m + 1):
        e = m - p  # power of i*y
        # i^e: real for even e, imaginary for odd e
        if which == "c" and e % 2 == 0:
            out[(p, e)] = comb(m, p) * (-1) ** (e // 2)
        if which == "s" and e % 2 == 1:
            out[(p, e)] = comb(m, p) * (-1) ** ((e - 1) // 2)
    return out


@functools.lru_cache(maxsize=32)
def solid_harmonic_monomials(l_max: int):
    """For l <= l_max, m = -l..l: list of (a, b, c, coefficient) with
    r^l Y_lm = sum coefficient * x^a y^b z^c.  Index lm = l*l + l + m."""
    table = []
    with mp.workdps(DPS):
        for l in range(l_max + 1):
            for m in range(-l, l + 1):
                am = abs(m)
                norm = mp.sqrt(mp.mpf(2 * l + 1) / (4 * mp.pi) * mp.factorial(l - am) / mp.factorial(l + am))
                if m != 0:
                    norm *= mp.sqrt(2)
                pi = _pi_lm(l, am)
                xy = _ab_m(am, "c" if m >= 0 else "s") if am > 0 else {(0, 0): 1}
                poly = {}
                for (k, pz), cz in pi.items():
                    # r^(2k) = sum over i+j+h = k of k!/(i! j! h!) x^2i y^2j z^2h
                    for i in range(k + 1):
                        for j in range(k - i + 1):
                            h = k - i - j
                            mult = factorial(k) // (factorial(i) * factorial(j) * factorial(h))
                            for (px, py), cxy in xy.items():
                                key = (2 * i + px, 2 * j + py, 2 * h + pz)
                                poly[key] = poly.get(key, Fraction(0)) + cz * mult * cxy
                terms = [(a, b, c, mp.mpf(v.numerator) / v.denominator * norm)
                         for (a, b, c), v in sorted(poly.items()) if v != 0]
                table.append(terms)
    return table


def solid_harmonic_arrays(l_max: int) -> dict:
    table = solid_harmonic_monomials(l_max)
    ptr = [0]
    exps = []
    coefs = []
    for terms in table:
        for a, b, c, v in terms:
            exps.extend((a, b, c))
            coefs.append(v)
        ptr.append(len(coefs))
    with mp.workdps(DPS):
        ch, cl = _split_array(coefs)
    return dict(sh_ptr=np.array(ptr, dtype=np.int32), sh_exp=np.array(exps, dtype=np.int32),
                sh_c_hi=ch, sh_c_lo=cl)
