"""GPU parity over the hyperparameter map of the 3000-atom water cluster (the
n_max x l_max map of the paper's Sec. 4.2): every (n_max, l_max) in
{2, 4, ..., 12}^2 for the GTO basis and both forms of the polynomial basis, in
the float32 mode (which runs a kernel compiled for that fixed basis size at
every grid point), and in the float64 mode at the four corners and at
(8, 6).  Per point: the neighbour rows of every center, the descriptor rows
of a seeded sample of centers, and every Jacobian block of a smaller sample,
against the oracle."""
import numpy as np
import pytest

import oracle
from paper_2609_05709_amd import workloads
from tests.parity import TOL, check_rows, gpu_run, jacobian_errors, row_errors

pytestmark = pytest.mark.gpu

_st = {}


def _water1000():
    if "s" not in _st:
        _st["s"] = workloads.WATER1000.structure()
    return _st["s"]


def sampled_check(wl, dtype, n_desc=32, n_jac=8, seed=0):
    st = _water1000()
    n = st.n_atoms
    rng = np.random.default_rng(seed)
    jac_idx = np.sort(rng.choice(n, size=n_jac, replace=False))
    desc_idx = np.sort(np.union1d(rng.choice(n, size=n_desc, replace=False), jac_idx))
    print(f"[grid] {wl.name} {dtype}", flush=True)
    g = gpu_run(wl, st, dtype, sample=jac_idx.tolist())
    check_rows(g, st, wl.r_cut, np.arange(n), wl.species)
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    ref = o.compute(st.pos64, st.Z, centers=desc_idx)
    ed = row_errors(g["desc"][desc_idx], ref["desc"]).max()
    refj = o.compute(st.pos64, st.Z, centers=jac_idx, jacobian=True)
    ej = jacobian_errors(g, refj, st, wl.species, jac_idx.tolist(), jac_idx)
    print(f"[grid] {wl.name} {dtype}: desc {ed:.2e}  jac {ej:.2e}", flush=True)
    assert ed < TOL[dtype]
    assert ej < TOL[dtype]


GRID = [(n, l) for n in workloads.GRID_NL for l in workloads.GRID_NL]
CORNERS = [(2, 2), (2, 12), (12, 2), (12, 12), (8, 6)]


@pytest.mark.parametrize("rbf", ["gto", "polynomial", "polynomial-laplace"])
@pytest.mark.parametrize("nl", GRID, ids=[f"n{n}l{l}" for n, l in GRID])
def test_grid_float32(rbf, nl):
    wl = workloads.WATER1000.with_basis(nl[0], nl[1], rbf)
    sampled_check(wl, "float32", seed=nl[0] * 13 + nl[1])


@pytest.mark.parametrize("rbf", ["gto", "polynomial", "polynomial-laplace"])
@pytest.mark.parametrize("nl", CORNERS, ids=[f"n{n}l{l}" for n, l in CORNERS])
def test_grid_float64(rbf, nl):
    wl = workloads.WATER1000.with_basis(nl[0], nl[1], rbf)
    sampled_check(wl, "float64", seed=nl[0] * 17 + nl[1])


@pytest.mark.parametrize("nl", [(8, 6), (12, 12), (2, 12)], ids=["n8l6", "n12l12", "n2l12"])
def test_grid_float64_arithmetic(nl):
    """float32 outputs from float64 internal arithmetic (option "arith"):
    the generic kernels with float64 staging and assembly."""
    wl = workloads.WATER1000.with_basis(nl[0], nl[1], "gto")
    st = _water1000()
    rng = np.random.default_rng(nl[0] + nl[1])
    jac_idx = np.sort(rng.choice(st.n_atoms, size=8, replace=False))
    g = gpu_run(wl, st, "float32", sample=jac_idx.tolist(), arith="fp64")
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    ref = o.compute(st.pos64, st.Z, centers=jac_idx, jacobian=True)
    ed = row_errors(g["desc"][jac_idx], ref["desc"]).max()
    ej = jacobian_errors(g, ref, st, wl.species, jac_idx.tolist(), jac_idx)
    print(f"[grid] {wl.name} float32 out, float64 arithmetic: desc {ed:.2e}  jac {ej:.2e}", flush=True)
    # float64 arithmetic leaves only the final rounding to float32: at most
    # 2^-24 of each value, so normwise below 6e-8 (plus float64 error)
    assert ed < 1e-7
    assert ej < 1e-7
