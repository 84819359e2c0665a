"""CPU checks of the C-ABI library: it loads, exports every entry point the
header declares, and its host-side basis setup matches the oracle's 50-digit
constants.  No GPU is used."""
import ctypes
import os
import re

import mpmath as mp
import numpy as np
import pytest

from oracle import constants

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_05709_amd", "libsoap.so")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2609_05709_amd import build
        build.build()
    return ctypes.CDLL(LIB)


def test_header_symbols_exported(lib):
    hdr = open(os.path.join(ROOT, "include", "soap.h")).read()
    names = set(re.findall(r"^\s*(?:int|int64_t|void|const char \*)\s*\*?(soap_\w+)\s*\(", hdr, re.M))
    from paper_2609_05709_amd.soap import ABI_SYMBOLS
    assert names == set(ABI_SYMBOLS)
    for n in names:
        assert hasattr(lib, n), n


def test_python_binding_declares_abi(lib):
    from paper_2609_05709_amd import soap
    L = soap.load_library()
    for n in soap.ABI_SYMBOLS:
        assert getattr(L, n).restype is not None or n == "soap_destroy"


def test_host_exp2_table(lib):
    """The table of the GTO kernels' exponential: 2^(j/64) as a double and
    its remainder, against 50-digit values (the double correctly rounded,
    the pair exact to ~2^-106 relative)."""
    t = np.empty(128)
    f = lib.soap_exp2_table64
    f.argtypes = [ctypes.c_void_p]
    f.restype = None
    f(t.ctypes.data)
    with mp.workdps(50):
        for j in range(64):
            v = mp.power(2, mp.mpf(j) / 64)
            assert t[2 * j] == float(v), j
            assert abs((mp.mpf(t[2 * j]) + mp.mpf(t[2 * j + 1]) - v) / v) < mp.mpf(2) ** -104, j


@pytest.mark.parametrize("r_cut,n_max,l_max,sigma", [(5.0, 4, 4, 0.5), (6.0, 8, 6, 0.5), (6.0, 12, 12, 0.5),
                                                     (6.0, 1, 2, 0.4)])
def test_host_gto_constants_match_oracle(lib, r_cut, n_max, l_max, sigma):
    n, lw = n_max, l_max + 1
    bc = np.empty(lw * n * n)
    ba = np.empty(lw * n * n)
    ap = np.empty(lw * n)
    c0 = np.empty(n)
    bcl, bal, apl = np.empty_like(bc), np.empty_like(ba), np.empty_like(ap)
    err = ctypes.create_string_buffer(256)
    f = lib.soap_basis_gto
    f.argtypes = ([ctypes.c_double, ctypes.c_int, ctypes.c_int, ctypes.c_double] + [ctypes.c_void_p] * 5 + [ctypes.c_int]
                  + [ctypes.c_void_p] * 3)
    assert f(r_cut, n, l_max, sigma, bc.ctypes.data, ba.ctypes.data, ap.ctypes.data, c0.ctypes.data, err, 256,
             bcl.ctypes.data, bal.ctypes.data, apl.ctypes.data) == 0
    z, alpha, beta = constants.gto_mp(r_cut, n, l_max)
    with mp.workdps(50):
        s2 = mp.mpf(sigma) ** 2
        for l in range(lw):
            for k in range(n):
                den = 1 + 2 * s2 * alpha[l][k]
                C = (2 * mp.pi) ** 1.5 * mp.mpf(sigma) ** 3 / den ** (l + mp.mpf(3) / 2)
                assert abs(ap[l * n + k] - float(alpha[l][k] / den)) <= 2e-16 * abs(float(alpha[l][k] / den))
                # the remainders make hi + lo the value to the 113-bit setup's accuracy (~1e-22);
                # the compensated float64 path uses both parts
                apr = alpha[l][k] / den
                assert abs(mp.mpf(ap[l * n + k]) + mp.mpf(apl[l * n + k]) - apr) <= 1e-28 * abs(apr)
                for a in range(n):
                    ref = beta[l][a, k] * C
                    got = bc[(l * n + a) * n + k]
                    assert abs(got - float(ref)) <= 1e-15 * abs(float(ref)) + 1e-300, (l, a, k, got, ref)
                    i = (l * n + a) * n + k
                    assert abs(mp.mpf(bc[i]) + mp.mpf(bcl[i]) - ref) <= 1e-20 * abs(ref) + 1e-300, (l, a, k)
                    refa = -2 * ref * apr
                    assert abs(mp.mpf(ba[i]) + mp.mpf(bal[i]) - refa) <= 1e-20 * abs(refa) + 1e-300, (l, a, k)
        for a in range(n):
            ref = mp.sqrt(2) * mp.pi * mp.mpf(sigma) ** 3 * mp.fsum(
                beta[0][a, k] / (1 + 2 * s2 * alpha[0][k]) ** 1.5 for k in range(n))
            assert abs(c0[a] - float(ref)) <= 1e-14 * max(1.0, abs(float(ref)))


@pytest.mark.parametrize("n_max,Q", [(4, 64), (10, 64), (12, 48), (15, 64), (16, 64)])
def test_host_poly_constants_match_oracle(lib, n_max, Q):
    """Up to n_max = 16, where the overlap matrix's condition number is 5.6e25."""
    r_cut, sigma = 5.0, 0.4
    G = np.empty(n_max * Q)
    rq = np.empty(Q)
    c0 = np.empty(n_max)
    err = ctypes.create_string_buffer(256)
    f = lib.soap_basis_poly
    f.argtypes = [ctypes.c_double, ctypes.c_int, ctypes.c_double, ctypes.c_int] + [ctypes.c_void_p] * 4 + [ctypes.c_int]
    assert f(r_cut, n_max, sigma, Q, G.ctypes.data, rq.ctypes.data, c0.ctypes.data, err, 256) == 0
    ref = constants.poly_arrays(r_cut, n_max, Q)
    Gr = (ref["G_hi"] + ref["G_lo"]) * 4 * np.pi
    assert np.allclose(np.sort(rq), np.sort(ref["rq_hi"]), rtol=0, atol=1e-15)
    order = np.argsort(rq)
    oref = np.argsort(ref["rq_hi"])
    Gg = G.reshape(n_max, Q)[:, order]
    Gr = Gr.reshape(n_max, Q)[:, oref]
    assert np.abs(Gg - Gr).max() <= 1e-14 * np.abs(Gr).max()


@pytest.mark.parametrize("r_cut,n_max,sigma", [(5.0, 1, 0.4), (6.0, 8, 0.5), (5.0, 12, 0.5), (4.0, 16, 0.3)])
def test_host_poly_laplace_chebyshev_series(lib, r_cut, n_max, sigma):
    """The Laplace form's P_j(u) = d^j/du^j sum_k (2 pi)^{3/2} sigma^3 W_nk/N_k
    u^(k+2), j = 0..3, handed over as Chebyshev series on [0, r_cut], equal
    the monomial sums with the oracle's 50-digit W and N, to 4e-15 of their
    largest value on the interval (the series evaluated in float64)."""
    n, M = n_max, n_max + 3
    CH = np.empty((n, M, 4))
    err = ctypes.create_string_buffer(256)
    f = lib.soap_basis_poly_laplace
    f.argtypes = [ctypes.c_double, ctypes.c_int, ctypes.c_double, ctypes.c_void_p, ctypes.c_char_p, ctypes.c_int]
    assert f(r_cut, n, sigma, CH.ctypes.data, err, 256) == 0, err.value
    N, W, _, _, _ = constants.poly_mp(r_cut, n, 2)
    us = np.linspace(0.0, r_cut, 41)
    t = 2 * us / r_cut - 1
    with mp.workdps(50):
        pref = (2 * mp.pi) ** mp.mpf(1.5) * mp.mpf(sigma) ** 3
        for a in range(n):
            got = np.polynomial.chebyshev.chebval(t, CH[a]).T  # [u][j]
            for j in range(4):
                ref = np.array([float(mp.fsum(pref * W[a, k - 1] / N[k - 1] * mp.ff(k + 2, j) * mp.mpf(u) ** (k + 2 - j)
                                              for k in range(1, n + 1))) for u in us])
                assert np.abs(got[:, j] - ref).max() <= 4e-15 * np.abs(ref).max(), (a, j)
