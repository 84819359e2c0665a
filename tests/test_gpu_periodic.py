"""GPU parity for periodic cells: neighbour rows as sets of (atom, image), the
descriptor, the Jacobian blocks per (atom, image), the dense expansion that
sums the images of an atom, and the coefficient Jacobian, against the
oracle's brute-force periodic images.  float32 mode uses the float32 image
positions on both sides (the reading documented in soap.h)."""
import numpy as np
import pytest

import oracle
from paper_2609_05709_amd import workloads
from tests.parity import TOL, block_error, row_errors

pytestmark = pytest.mark.gpu


def _wl(species=(1, 8), rbf="gto", r_cut=4.5, sigma=0.5, n_max=4, l_max=4):
    return workloads.Workload("pbc", tuple(species), rbf, r_cut, sigma, n_max, l_max, True, ("none",))


def _case(seed, n=9, cell=None):
    rng = np.random.default_rng(seed)
    if cell is None:
        cell = np.array([[4.3, 0.0, 0.0], [0.9, 4.1, 0.0], [-0.4, 0.6, 4.6]])
    pos = (rng.uniform(0, 1, size=(n, 3)) @ cell).astype(np.float32)
    Z = np.array([1, 8] * n, dtype=np.int32)[:n]
    return pos, Z, np.asarray(cell, dtype=np.float64)


def run_gpu(wl, pos, Z, cell, pbc, dtype, what="derivatives"):
    import torch
    from paper_2609_05709_amd.soap import Soap
    tdt = torch.float64 if dtype == "float64" else torch.float32
    sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, dtype=dtype)
    sp.set_cell(cell, pbc)
    p = torch.from_numpy(pos.astype(np.float64) if dtype == "float64" else pos).to("cuda", tdt)
    E = sp.build_neighbors(p, torch.from_numpy(Z).cuda())
    row, cols = [t.cpu().numpy() for t in sp.neighbors()]
    img = sp.neighbor_images().cpu().numpy()
    out = dict(E=E, row=row, cols=cols, img=img, fmaps=[sp.feature_map(k) for k in range(len(wl.species))])
    if what == "derivatives":
        d, je, js = sp.derivatives()
        dense = sp.scatter_dense(je, js)
        torch.cuda.synchronize()
        out.update(desc=d.cpu().double().numpy(), je=je.cpu().double().numpy(), js=js.cpu().double().numpy(),
                   dense=dense.cpu().double().numpy())
    else:
        c, je, js = sp.coefficient_derivatives()
        torch.cuda.synchronize()
        out.update(c=c.cpu().double().numpy(), je=je.cpu().double().numpy(), js=js.cpu().double().numpy())
    sp.close()
    return out


def _keys(cols, img, r0, r1):
    return {(int(cols[e]),) + tuple(int(v) for v in img[e]): e for e in range(int(r0), int(r1))}


def check(wl, pos, Z, cell, pbc, dtype):
    f32 = dtype == "float32"
    g = run_gpu(wl, pos, Z, cell, pbc, dtype)
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    ref = o.compute_periodic(pos.astype(np.float64), Z, cell, pbc, f32=f32, jacobian=True)
    n = len(pos)
    spec = {z: k for k, z in enumerate(sorted(wl.species))}
    assert row_errors(g["desc"], ref["desc"]).max() < TOL[dtype]
    worst = 0.0
    for c in range(n):
        gk = _keys(g["cols"], g["img"], g["row"][c], g["row"][c + 1])
        b0, b1 = ref["blk_ptr"][c], ref["blk_ptr"][c + 1]
        rk, total = {}, {}
        for b in range(b0, b1):
            x = int(ref["blk_j"][b])
            key = (int(ref["img_atom"][x]),) + tuple(int(v) for v in ref["img_shift"][x])
            if x == c:
                worst = max(worst, block_error(g["js"][c], ref["jac"][b]))
            else:
                rk[key] = b
            a = key[0]
            total[a] = total.get(a, 0) + ref["jac"][b]
        assert gk.keys() == rk.keys(), c
        for key, e in gk.items():
            fm = g["fmaps"][spec[int(Z[key[0]])]]
            worst = max(worst, block_error(g["je"][e], ref["jac"][rk[key]][:, fm]))
        for a, J in total.items():
            worst = max(worst, block_error(g["dense"][c, a], J))
    print(f"[parity] periodic {wl.rbf} {dtype} pbc={pbc}: desc/jac {worst:.2e} E={g['E']}", flush=True)
    assert worst < TOL[dtype]


@pytest.mark.parametrize("dtype", ["float32", "float64"])
@pytest.mark.parametrize("rbf", ["gto", "polynomial", "polynomial-laplace"])
def test_periodic_small_triclinic_cell(rbf, dtype):
    """A cell smaller than 2 r_cut: several images of each atom and of the
    center itself are neighbours."""
    pos, Z, cell = _case(3)
    check(_wl(rbf=rbf), pos, Z, cell, (1, 1, 1), dtype)


def test_periodic_slab_and_atoms_outside_the_cell():
    pos, Z, cell = _case(8, n=12)
    pos = pos + np.array([5.0, -9.0, 2.0], dtype=np.float32)  # images are built around the atoms as given
    check(_wl(species=(1, 8), n_max=3, l_max=5), pos, Z, cell, (1, 1, 0), "float32")


def test_periodic_water_box():
    st = workloads.WATER64.structure()
    lo = st.pos.min(axis=0) - 0.8
    cell = np.diag(st.pos.max(axis=0) - lo + 1.6)
    check(_wl(r_cut=5.0), (st.pos - lo).astype(np.float32), st.Z, cell, (1, 1, 1), "float32")


def test_periodic_rows_match_oracle_and_large_cell_is_the_cluster():
    import torch
    s = workloads.random_small(20, 9, 3.0, species=(1, 8))
    wl = _wl()
    big = np.diag([70.0, 70.0, 70.0])
    moved = s.pos + np.float32(30.0)
    g = run_gpu(wl, moved, s.Z, big, (1, 1, 1), "float64")
    assert not g["img"].any()
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    ref = o.compute(moved.astype(np.float64), s.Z)["desc"]
    assert row_errors(g["desc"], ref).max() < TOL["float64"]
    pos, Z, cell = _case(5)
    g = run_gpu(wl, pos, Z, cell, (1, 1, 1), "float32", what="cc")
    row, cols, img = oracle.neighbors_periodic(pos.astype(np.float64), wl.r_cut, cell, (1, 1, 1), f32=True)
    for c in range(len(pos)):
        assert _keys(g["cols"], g["img"], g["row"][c], g["row"][c + 1]).keys() == _keys(cols, img, row[c], row[c + 1]).keys()


def test_periodic_coefficient_jacobian():
    pos, Z, cell = _case(6)
    wl = _wl(n_max=3, l_max=3)
    g = run_gpu(wl, pos, Z, cell, (1, 1, 1), "float64", what="cc")
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    ref = o.compute_periodic(pos.astype(np.float64), Z, cell, (1, 1, 1), f32=False, coefficients=True,
                             coefficient_jacobian=True)
    worst = 0.0
    for c in range(len(pos)):
        worst = max(worst, block_error(g["c"][c], ref["c"][c]), block_error(g["js"][c], ref["dc_self"][c]))
        oc = {}
        for e in range(int(ref["row_ptr"][c]), int(ref["row_ptr"][c + 1])):
            x = int(ref["cols"][e])
            oc[(int(ref["img_atom"][x]),) + tuple(int(v) for v in ref["img_shift"][x])] = e
        gk = _keys(g["cols"], g["img"], g["row"][c], g["row"][c + 1])
        assert gk.keys() == oc.keys(), c
        for key, e in gk.items():
            worst = max(worst, block_error(g["je"][e], ref["dc"][oc[key]]))
    assert worst < TOL["float64"]


def test_set_cell_errors_and_reset():
    import torch
    from paper_2609_05709_amd.soap import Soap, SoapError
    wl = _wl()
    sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    with pytest.raises(SoapError):
        sp.set_cell(np.array([[1.0, 0, 0], [2.0, 0, 0], [0, 0, 1.0]]))
    pos, Z, cell = _case(2)
    p, z = torch.from_numpy(pos).cuda(), torch.from_numpy(Z).cuda()
    sp.set_cell(cell)
    e1 = sp.build_neighbors(p, z)
    sp.set_cell(None)
    e0 = sp.build_neighbors(p, z)
    assert e1 > e0 and not sp.neighbor_images().cpu().numpy().any()
    sp.close()
