"""GPU parity of the coefficient ("cc") Jacobian and of the averaged descriptors
against the oracle, on the same seeded inputs.  Tolerances as for the
descriptor: 1e-5 (float32 mode) and 1e-10 (float64 mode), normwise per block
(coefficient set of one center, gradient block of one (center, atom) pair) or
per averaged row."""
import numpy as np
import pytest

import oracle
from paper_2609_05709_amd import workloads
from tests.parity import TOL, block_error

pytestmark = pytest.mark.gpu


def _wl(species=(1, 8), rbf="gto", r_cut=5.0, sigma=0.5, n_max=4, l_max=4):
    return workloads.Workload("modes", tuple(species), rbf, r_cut, sigma, n_max, l_max, True, ("none",))


def _soap(wl, dtype):
    from paper_2609_05709_amd.soap import Soap
    return Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, dtype=dtype)


def _inputs(st, dtype):
    import torch
    tdt = torch.float64 if dtype == "float64" else torch.float32
    pos = torch.from_numpy(st.pos.astype(np.float64) if dtype == "float64" else st.pos).to("cuda", tdt)
    return pos, torch.from_numpy(st.Z).to("cuda")


def check_cc(wl, st, dtype, sample=None):
    import torch
    sp = _soap(wl, dtype)
    pos, Z = _inputs(st, dtype)
    E = sp.build_neighbors(pos, Z)
    row, cols = [t.cpu().numpy() for t in sp.neighbors()]
    c, je, js = sp.coefficient_derivatives()
    torch.cuda.synchronize()
    c, js = c.cpu().double().numpy(), js.cpu().double().numpy()
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    ref = o.compute(st.pos64, st.Z, coefficients=True, coefficient_jacobian=True)
    orow, ocols = ref["row_ptr"], ref["cols"]
    idx = range(st.n_atoms) if sample is None else sample
    worst = 0.0
    for ci in idx:
        worst = max(worst, block_error(c[ci], ref["c"][ci]), block_error(js[ci], ref["dc_self"][ci]))
        g = {int(j): e for e, j in zip(range(int(row[ci]), int(row[ci + 1])), cols[row[ci]:row[ci + 1]])}
        r = {int(j): e for e, j in zip(range(int(orow[ci]), int(orow[ci + 1])), ocols[orow[ci]:orow[ci + 1]])}
        assert g.keys() == r.keys(), ci
        if g:
            eg = np.array([g[j] for j in r])
            blocks = je[torch.from_numpy(eg).cuda()].cpu().double().numpy()
            for k, j in enumerate(r):
                worst = max(worst, block_error(blocks[k], ref["dc"][r[j]]))
    print(f"[parity] cc {wl.name} {wl.rbf} {dtype}: {worst:.2e} E={E}", flush=True)
    assert worst < TOL[dtype]
    sp.close()


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_cc_water64(dtype):
    check_cc(workloads.WATER64, workloads.WATER64.structure(), dtype)


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_cc_water1000_sampled(dtype):
    wl = workloads.WATER1000
    rng = np.random.default_rng(11)
    check_cc(wl, wl.structure(), dtype, sample=sorted(rng.choice(3000, size=60, replace=False).tolist()))


@pytest.mark.parametrize("rbf", ["gto", "polynomial", "polynomial-laplace"])
@pytest.mark.parametrize("nl", [(1, 0), (6, 9), (12, 3)])
def test_cc_small_bases(rbf, nl):
    wl = _wl(species=(1, 6, 8), rbf=rbf, n_max=nl[0], l_max=nl[1])
    st = workloads.random_small(30, 17, 3.5, species=(1, 6, 8))
    for dtype in ("float32", "float64"):
        check_cc(wl, st, dtype)


def test_cc_isolated_and_coincident_atoms():
    wl = _wl()
    st = workloads.Structure(np.array([[0, 0, 0], [20, 0, 0], [20, 0, 0], [0.9, 0.2, -0.3]], dtype=np.float32),
                             np.array([8, 1, 1, 1], dtype=np.int32), 0.0, 0)
    check_cc(wl, st, "float64")
    lone = workloads.Structure(np.array([[1.0, 2.0, 3.0]], dtype=np.float32), np.array([8], dtype=np.int32), 0.0, 0)
    check_cc(wl, lone, "float32")


def check_averaged(wl, st, dtype):
    import torch
    sp = _soap(wl, dtype)
    pos, Z = _inputs(st, dtype)
    sp.build_neighbors(pos, Z)
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    for mode in ("inner", "outer"):
        got = sp.compute_averaged(mode)
        torch.cuda.synchronize()
        ref = o.averaged(st.pos64, st.Z, mode)
        err = np.abs(got.cpu().double().numpy() - ref).max() / np.abs(ref).max()
        print(f"[parity] average {mode} {wl.name} {dtype}: {err:.2e}", flush=True)
        assert err < TOL[dtype]
    sp.close()


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_averaged_water1000(dtype):
    check_averaged(workloads.WATER1000, workloads.WATER1000.structure(), dtype)


def test_averaged_chno4096():
    check_averaged(workloads.CHNO4096, workloads.CHNO4096.structure(), "float32")


def test_averaged_single_atom_and_dimer():
    wl = _wl(species=(8,), n_max=4, l_max=5)
    for pos in ([[0.3, -0.2, 0.1]], [[0.3, -0.2, 0.1], [1.1, 0.9, -0.6]]):
        st = workloads.Structure(np.array(pos, dtype=np.float32), np.full(len(pos), 8, dtype=np.int32), 0.0, 0)
        check_averaged(wl, st, "float64")


def test_modes_reject_bad_arguments():
    import torch
    from paper_2609_05709_amd.soap import SoapError
    wl = _wl()
    sp = _soap(wl, "float32")
    with pytest.raises(SoapError):
        sp.compute_averaged("outer")  # no neighbour list yet
    st = workloads.random_small(10, 3, 3.0)
    pos, Z = _inputs(st, "float32")
    sp.build_neighbors(pos, Z)
    with pytest.raises(ValueError):
        sp.compute_averaged("middle")
    rc = sp._L.soap_compute_averaged(sp._h, 7, torch.empty(sp.n_features, device="cuda").data_ptr(), None)
    assert rc != 0
    sp.close()
