"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI
and compare with the oracle.

Error metric (normwise per unit): descriptor row of a center -> max |delta| /
max |oracle row|; Jacobian block (center i, atom j) -> max |delta| / max
|oracle block|; a unit whose oracle values are all zero must be exactly zero.
"""
from __future__ import annotations

import numpy as np

import oracle

TOL = {"float32": 1e-5, "float64": 1e-10}


def gpu_run(wl, st, dtype="float32", centers=None, jacobian=True, sample=None, coefficients=False, quad_n=None,
            arith="mixed"):
    """Run the HIP path; copy back the descriptor, neighbour rows and, for the
    centers in `sample` (indices into the center list; None = all), their
    Jacobian blocks."""
    import torch
    from paper_2609_05709_amd.soap import Soap
    tdt = torch.float64 if dtype == "float64" else torch.float32
    sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, dtype=dtype, quad_n=quad_n, arith=arith)
    pos = torch.from_numpy(st.pos.astype(np.float64) if dtype == "float64" else st.pos).to("cuda", tdt)
    Z = torch.from_numpy(st.Z).to("cuda")
    cen = None if centers is None else torch.from_numpy(np.asarray(centers, dtype=np.int32)).to("cuda")
    E = sp.build_neighbors(pos, Z, cen)
    out = dict(E=E, F=sp.n_features, Fe=sp.n_edge_features, fmaps=[sp.feature_map(k) for k in range(len(wl.species))],
               labels=sp.feature_labels())
    row, cols = sp.neighbors()
    out["row"], out["cols"] = row.cpu().numpy(), cols.cpu().numpy()
    if coefficients:
        out["c"] = sp.coefficients().cpu().double().numpy()
    if jacobian:
        desc, jedge, jself = sp.derivatives()
        torch.cuda.synchronize()
        out["desc"] = desc.cpu().double().numpy()
        nc = out["row"].shape[0] - 1
        idx = range(nc) if sample is None else sample
        out["jedge"], out["jself"] = {}, {}
        for c in idx:
            r0, r1 = int(out["row"][c]), int(out["row"][c + 1])
            out["jedge"][c] = jedge[r0:r1].cpu().double().numpy()
            out["jself"][c] = jself[c].cpu().double().numpy()
        del jedge, jself
    else:
        out["desc"] = sp.compute().cpu().double().numpy()
    torch.cuda.synchronize()
    sp.close()
    return out


def row_errors(got, ref):
    scale = np.abs(ref).max(axis=1)
    err = np.abs(got - ref).max(axis=1)
    zero = scale == 0
    assert np.all(err[zero] == 0), "non-zero output where the oracle row is zero"
    return np.where(zero, 0.0, err / np.where(zero, 1.0, scale))


def block_error(got, ref):
    s = np.abs(ref).max()
    if s == 0:
        assert np.all(got == 0), "non-zero block where the oracle block is zero"
        return 0.0
    return float(np.abs(got - ref).max() / s)


def jacobian_errors(gpu, ref, st, species, centers_idx, center_atoms):
    """Worst normwise error over all (center, atom) blocks of the given centers.
    ref = oracle output computed for center_atoms (same order as centers_idx)."""
    spec = {z: k for k, z in enumerate(sorted(species))}
    worst = 0.0
    for k, c in enumerate(centers_idx):
        i = int(center_atoms[k])
        b0, b1 = int(ref["blk_ptr"][k]), int(ref["blk_ptr"][k + 1])
        blocks = dict(zip(ref["blk_j"][b0:b1].tolist(), range(b0, b1)))
        worst = max(worst, block_error(gpu["jself"][c], ref["jac"][blocks[i]]))
        r0 = int(gpu["row"][c])
        cols = gpu["cols"][r0:int(gpu["row"][c + 1])]
        assert len(cols) == b1 - b0 - 1
        for e, j in enumerate(cols.tolist()):
            Jr = ref["jac"][blocks[j]]
            fm = gpu["fmaps"][spec[int(st.Z[j])]]
            mask = np.ones(Jr.shape[1], bool)
            mask[fm] = False
            assert np.all(Jr[:, mask] == 0), "oracle has non-zeros outside the neighbour's species pairs"
            worst = max(worst, block_error(gpu["jedge"][c][e], Jr[:, fm]))
    return worst


def check_rows(gpu, st, r_cut, center_atoms, species):
    """Neighbour rows: same index sets as the oracle's all-pairs search, ordered
    by (species index, atom index)."""
    row_o, col_o = oracle.neighbors(st.pos64, r_cut, np.asarray(center_atoms, dtype=np.int64))
    assert np.array_equal(np.diff(gpu["row"]), np.diff(row_o))
    spec = {z: k for k, z in enumerate(sorted(species))}
    s_of = np.array([spec[int(z)] for z in st.Z])
    for c in range(len(center_atoms)):
        g = gpu["cols"][gpu["row"][c]:gpu["row"][c + 1]]
        o = col_o[row_o[c]:row_o[c + 1]]
        assert set(g.tolist()) == set(o.tolist()), c
        key = s_of[g].astype(np.int64) * (1 << 32) + g
        assert np.all(np.diff(key) > 0), "row not ordered by (species, atom)"
