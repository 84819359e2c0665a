"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs, element by element.  Tolerances: 1e-5 (float32 mode) and
1e-10 (float64 mode), normwise per descriptor row / Jacobian block."""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2609_05709_amd import workloads
from tests.parity import TOL, check_rows, gpu_run, jacobian_errors, row_errors

pytestmark = pytest.mark.gpu

_structs = {}


def structure(wl):
    key = wl.make
    if key not in _structs:
        _structs[key] = wl.structure()
    return _structs[key]


def oracle_for(wl, **kw):
    return oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, **kw)


def full_check(wl, dtype, sample=None, seed=0):
    st = structure(wl)
    print(f"[parity] {wl.name} {dtype} atoms={st.n_atoms}", flush=True)
    n = st.n_atoms
    if sample is not None:
        rng = np.random.default_rng(seed)
        sample = np.sort(rng.choice(n, size=min(sample, n), replace=False))
    g = gpu_run(wl, st, dtype, sample=None if sample is None else sample.tolist())
    o = oracle_for(wl)
    check_rows(g, st, wl.r_cut, np.arange(n), wl.species)
    # descriptor: every center
    ref_d = o.compute(st.pos64, st.Z)["desc"]
    ed = row_errors(g["desc"], ref_d)
    # Jacobian: all or sampled centers
    idx = np.arange(n) if sample is None else sample
    ref = o.compute(st.pos64, st.Z, centers=idx, jacobian=True)
    ej = jacobian_errors(g, ref, st, wl.species, idx.tolist(), idx)
    print(f"[parity] {wl.name} {dtype}: desc {ed.max():.2e}  jac {ej:.2e}  E={g['E']}", flush=True)
    assert ed.max() < TOL[dtype]
    assert ej < TOL[dtype]
    return ed.max(), ej


def all_centers_check(wl, dtype, batch=512):
    """Every center and every block; the oracle's Jacobian is computed and
    compared in batches of centers to bound its memory."""
    st = structure(wl)
    print(f"[parity] {wl.name} {dtype} all centers, atoms={st.n_atoms}", flush=True)
    n = st.n_atoms
    g = gpu_run(wl, st, dtype)
    o = oracle_for(wl)
    check_rows(g, st, wl.r_cut, np.arange(n), wl.species)
    ed = row_errors(g["desc"], o.compute(st.pos64, st.Z)["desc"]).max()
    ej = 0.0
    for b0 in range(0, n, batch):
        idx = np.arange(b0, min(n, b0 + batch))
        ref = o.compute(st.pos64, st.Z, centers=idx, jacobian=True)
        ej = max(ej, jacobian_errors(g, ref, st, wl.species, idx.tolist(), idx))
        del ref
    print(f"[parity] {wl.name} {dtype} all centers: desc {ed:.2e}  jac {ej:.2e}  E={g['E']}", flush=True)
    assert ed < TOL[dtype]
    assert ej < TOL[dtype]


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_water1000_gto_n8l6_all_centers(dtype):
    all_centers_check(workloads.WATER1000, dtype)


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_chno4096_poly_n10l10_all_centers(dtype):
    all_centers_check(workloads.CHNO4096, dtype)


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_water64_gto_full(dtype):
    full_check(workloads.WATER64, dtype)


def test_water64_coefficients_match_oracle():
    wl = workloads.WATER64
    st = structure(wl)
    g = gpu_run(wl, st, "float64", jacobian=False, coefficients=True)
    ref = oracle_for(wl).compute(st.pos64, st.Z, coefficients=True)["c"]
    err = row_errors(g["c"].reshape(st.n_atoms, -1), ref.reshape(st.n_atoms, -1))
    assert err.max() < 1e-10, err.max()


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_water1000_gto_n8l6(dtype):
    full_check(workloads.WATER1000, dtype, sample=24, seed=1)


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_chno4096_poly_n10l10(dtype):
    full_check(workloads.CHNO4096, dtype, sample=32, seed=3)


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_water64_polynomial_laplace_full(dtype):
    full_check(workloads.WATER64.with_basis(4, 4, "polynomial-laplace"), dtype)


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_water1000_polynomial_laplace_n8l6(dtype):
    full_check(workloads.WATER1000.with_basis(8, 6, "polynomial-laplace"), dtype, sample=24, seed=5)


@pytest.mark.parametrize("dtype", ["float32", "float64"])
@pytest.mark.parametrize("rbf", ["gto", "polynomial", "polynomial-laplace"])
def test_largest_radial_basis(rbf, dtype):
    """n_max = 16, the library's largest: the polynomial overlap matrix has
    condition number 5.6e25 there, and the GTO Loewdin coefficients amplify
    float64 rounding of the radial sums by ~5e8 (the compensated path)."""
    wl = workloads.WATER64.with_basis(16, 4, rbf)
    full_check(wl, dtype, sample=12, seed=16)


@pytest.mark.parametrize("n_max,l_max,sigma", [(10, 6, 0.5), (12, 12, 0.5), (14, 4, 0.3), (16, 8, 0.5)])
def test_gto_float64_compensated(n_max, l_max, sigma):
    """GTO in float64 from n_max 10 on: every exponential in double-double and
    compensated sums over the Loewdin coefficients keep the 1e-10 bar."""
    wl = dataclasses.replace(workloads.WATER64.with_basis(n_max, l_max, "gto"), sigma=sigma)
    full_check(wl, "float64", sample=12, seed=n_max + l_max)


def test_water1m_descriptor_sampled():
    import torch
    from paper_2609_05709_amd.soap import Soap
    wl = workloads.WATER1M
    st = structure(wl)
    print(f"[parity] {wl.name} atoms={st.n_atoms}", flush=True)
    sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    pos = torch.from_numpy(st.pos).cuda()
    Z = torch.from_numpy(st.Z).cuda()
    E = sp.build_neighbors(pos, Z)
    desc = sp.compute()
    row, cols = sp.neighbors()
    rng = np.random.default_rng(4)
    sample = np.sort(rng.choice(st.n_atoms, 200, replace=False))
    got = desc[torch.from_numpy(sample).cuda()].cpu().double().numpy()
    row, cols = row.cpu().numpy(), cols.cpu().numpy()
    sp.close()
    # full neighbour sets against the oracle's uniform-grid search
    row_g, col_g = oracle.neighbors_grid(st.pos64, wl.r_cut)
    assert E == len(col_g)
    assert np.array_equal(row, row_g)
    for i in sample:
        assert set(cols[row[i]:row[i + 1]].tolist()) == set(col_g[row_g[i]:row_g[i + 1]].tolist())
    ref = oracle_for(wl).compute(st.pos64, st.Z, centers=sample)["desc"]
    err = row_errors(got, ref)
    print(f"[parity] {wl.name}: desc {err.max():.2e} E={E}", flush=True)
    assert err.max() < TOL["float32"]


@pytest.mark.parametrize("seed", range(12))
def test_fuzz_small_structures(seed):
    rng = np.random.default_rng(100 + seed)
    S = int(rng.integers(1, 5))
    species = tuple(sorted(rng.choice([1, 6, 7, 8, 16], size=S, replace=False).tolist()))
    n_max = int(rng.integers(1, 13))
    l_max = int(rng.integers(0, 13))
    rbf = "gto" if seed % 2 == 0 else "polynomial"
    n_atoms = int(rng.integers(2, 40))
    st = workloads.random_small(n_atoms, 200 + seed, 4.0, species=species, dmin=0.8)
    wl = workloads.Workload(f"fuzz{seed}", species, rbf, 4.5, float(rng.uniform(0.3, 0.6)), n_max, l_max, True,
                            ("none",))
    _structs[wl.make] = st
    ref_d = oracle_for(wl).compute(st.pos64, st.Z)["desc"]
    for dtype in ("float32", "float64"):
        full_check(wl, dtype)
        # the descriptor-only path (its own kernels) on the same structure
        d = gpu_run(wl, st, dtype, jacobian=False)
        ed = row_errors(d["desc"], ref_d).max()
        print(f"[parity] {wl.name} {dtype}: descriptor path {ed:.2e}", flush=True)
        assert ed < TOL[dtype]
    _structs.pop(wl.make)


@pytest.mark.parametrize("dtype", ["float32", "float64"])
@pytest.mark.parametrize("nl", [(4, 4), (8, 6), (2, 2), (12, 7), (8, 10), (1, 0)])
def test_descriptor_kernel_chunk_widths(dtype, nl):
    """The GTO descriptor path (one wave per center) at every chunk width and
    the shared density kernel (desc_tile -1): sampled rows against the
    oracle; the chunk widths give the same bits (each wave sums its center's
    edges in row order whatever the chunking); the coefficients too."""
    import torch
    from paper_2609_05709_amd.soap import Soap
    wl = workloads.WATER1000.with_basis(nl[0], nl[1], "gto")
    st = structure(wl)
    tdt = torch.float64 if dtype == "float64" else torch.float32
    pos = torch.from_numpy(st.pos.astype(np.float64) if dtype == "float64" else st.pos).to("cuda", tdt)
    Z = torch.from_numpy(st.Z).cuda()
    rng = np.random.default_rng(nl[0] * 31 + nl[1])
    idx = np.sort(rng.choice(st.n_atoms, size=24, replace=False))
    ref = oracle_for(wl).compute(st.pos64, st.Z, centers=idx, coefficients=True)
    first = None
    for tile in (64, 32, 16, -1):
        sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, dtype=dtype)
        sp._check(sp._L.soap_set_option(sp._h, b"desc_tile", tile))
        sp.build_neighbors(pos, Z)
        d = sp.compute()
        c = sp.coefficients()
        torch.cuda.synchronize()
        err = row_errors(d.cpu().double().numpy()[idx], ref["desc"]).max()
        cerr = row_errors(c.cpu().double().numpy()[idx].reshape(len(idx), -1), ref["c"].reshape(len(idx), -1)).max()
        print(f"[desc] {wl.name} {dtype} tile {tile}: desc {err:.2e} c {cerr:.2e}", flush=True)
        assert err < TOL[dtype] and cerr < TOL[dtype]
        if tile > 0:
            if first is None:
                first = (d.clone(), c.clone())
            else:
                assert torch.equal(d, first[0]) and torch.equal(c, first[1])
        sp.close()


@pytest.mark.parametrize("dtype", ["float32", "float64"])
@pytest.mark.parametrize("case", ["water64", "water1000", "water1000_n4l8", "three_species", "four_species_n6l4"])
def test_jacobian_density_kernel_chunk_widths(dtype, case):
    """The one-workgroup-per-center density step of the Jacobian path (GTO)
    at both chunk widths: descriptor and every block of sampled centers
    against the oracle, and the same bits at both widths."""
    import torch
    from paper_2609_05709_amd.soap import Soap
    if case == "water64":
        wl, st, sample = workloads.WATER64, structure(workloads.WATER64), None
    elif case.startswith("water1000"):
        wl = workloads.WATER1000 if case == "water1000" else workloads.WATER1000.with_basis(4, 8, "gto")
        st, sample = structure(wl), 16
    else:
        species = (1, 6, 8) if case == "three_species" else (1, 6, 7, 8)
        nl = (5, 5) if case == "three_species" else (6, 4)
        wl = workloads.Workload(case, species, "gto", 5.0, 0.45, nl[0], nl[1], True, ("none",))
        st = workloads.random_small(90, 31 + len(species), 5.0, species=species, dmin=0.85)
        sample = None
    n = st.n_atoms
    idx = np.arange(n) if sample is None else np.sort(np.random.default_rng(7).choice(n, sample, replace=False))
    ref = oracle_for(wl).compute(st.pos64, st.Z, centers=idx, jacobian=True)
    tdt = torch.float64 if dtype == "float64" else torch.float32
    pos = torch.from_numpy(st.pos.astype(np.float64) if dtype == "float64" else st.pos).to("cuda", tdt)
    Z = torch.from_numpy(st.Z).cuda()
    first = None
    for tile in (64, 32):
        sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, dtype=dtype)
        sp._check(sp._L.soap_set_option(sp._h, b"djac_tile", tile))
        sp.build_neighbors(pos, Z)
        d, je, js = sp.derivatives()
        row, cols = sp.neighbors()
        torch.cuda.synchronize()
        g = dict(row=row.cpu().numpy(), cols=cols.cpu().numpy(), fmaps=[sp.feature_map(k) for k in range(len(wl.species))],
                 jedge={}, jself={})
        for c in idx:
            r0, r1 = int(g["row"][c]), int(g["row"][c + 1])
            g["jedge"][int(c)] = je[r0:r1].cpu().double().numpy()
            g["jself"][int(c)] = js[int(c)].cpu().double().numpy()
        ed = row_errors(d.cpu().double().numpy()[idx], ref["desc"]).max()
        ej = jacobian_errors(g, ref, st, wl.species, idx.tolist(), idx)
        print(f"[djac] {case} {dtype} tile {tile}: desc {ed:.2e} jac {ej:.2e}", flush=True)
        assert ed < TOL[dtype] and ej < TOL[dtype]
        if first is None:
            first = (d.clone(), je.clone(), js.clone())
        else:
            for x, y in zip((d, je, js), first):
                assert torch.equal(x, y)
        sp.close()


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_jacobian_kernel_tile_widths(dtype):
    """The edge Jacobian kernel at every matrix-core tile width that fits
    (option "jac_tile"): every block of the 64-water cluster against the
    oracle, and the same bits at every width (a tile's rows are the
    (component, edge) pairs of its edges, each summed on its own)."""
    import torch
    from paper_2609_05709_amd.soap import Soap
    wl, st = workloads.WATER64, structure(workloads.WATER64)
    idx = np.arange(st.n_atoms)
    ref = oracle_for(wl).compute(st.pos64, st.Z, centers=idx, jacobian=True)
    tdt = torch.float64 if dtype == "float64" else torch.float32
    pos = torch.from_numpy(st.pos.astype(np.float64) if dtype == "float64" else st.pos).to("cuda", tdt)
    Z = torch.from_numpy(st.Z).cuda()
    first, ran = None, 0
    for tile in (1, 2, 3, 4):
        sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, dtype=dtype)
        sp._check(sp._L.soap_set_option(sp._h, b"jac_tile", tile))
        if sp.get_option("jacobian_tile") != tile:
            sp.close()  # this width does not fit on chip
            continue
        sp.build_neighbors(pos, Z)
        d, je, js = sp.derivatives()
        row, cols = sp.neighbors()
        torch.cuda.synchronize()
        g = dict(row=row.cpu().numpy(), cols=cols.cpu().numpy(), fmaps=[sp.feature_map(k) for k in range(len(wl.species))],
                 jedge={}, jself={})
        for c in idx:
            r0, r1 = int(g["row"][c]), int(g["row"][c + 1])
            g["jedge"][int(c)] = je[r0:r1].cpu().double().numpy()
            g["jself"][int(c)] = js[int(c)].cpu().double().numpy()
        ej = jacobian_errors(g, ref, st, wl.species, idx.tolist(), idx)
        print(f"[jac] {wl.name} {dtype} tile {tile}: jac {ej:.2e}", flush=True)
        assert ej < TOL[dtype]
        ran += 1
        if first is None:
            first = je.clone()
        else:
            assert torch.equal(je, first)
        sp.close()
    assert ran >= 2


@pytest.mark.parametrize("dtype", ["float32", "float64"])
@pytest.mark.parametrize("case", ["chno_poly_n10l10", "chno_poly_n6l8", "water_poly_n12l12"])
def test_output_kernel_rows_and_groups(dtype, case):
    """The output kernel of the Jacobian path (power spectrum and center block
    from the coefficient scratch) writing whole rows and in l-groups:
    descriptor and every block of every center against the oracle, and in
    float64 the same bits both ways (the mixed mode stages the whole-row
    kernel's coefficients in float32, the l-group kernel's in float64)."""
    import torch
    from paper_2609_05709_amd.soap import Soap
    if case.startswith("chno"):
        nl = (10, 10) if case.endswith("n10l10") else (6, 8)
        wl = workloads.Workload(case, (1, 6, 7, 8), "polynomial", 5.0, 0.4, nl[0], nl[1], True, ("none",))
        st = workloads.random_small(60, 41, 5.0, species=(1, 6, 7, 8), dmin=0.85)
    else:
        wl = workloads.Workload(case, (1, 8), "polynomial", 5.0, 0.5, 12, 12, True, ("none",))
        st = workloads.random_small(48, 43, 4.5, species=(1, 8), dmin=0.85)
    idx = np.arange(st.n_atoms)
    ref = oracle_for(wl).compute(st.pos64, st.Z, centers=idx, jacobian=True)
    tdt = torch.float64 if dtype == "float64" else torch.float32
    pos = torch.from_numpy(st.pos.astype(np.float64) if dtype == "float64" else st.pos).to("cuda", tdt)
    Z = torch.from_numpy(st.Z).cuda()
    first = None
    for rows in (1, 0):
        sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, dtype=dtype)
        sp._check(sp._L.soap_set_option(sp._h, b"out_rows", rows))
        groups, used_rows = sp.get_option("jacobian_l_groups"), sp.get_option("output_kernel_rows")
        sp.build_neighbors(pos, Z)
        d, je, js = sp.derivatives()
        row, cols = sp.neighbors()
        torch.cuda.synchronize()
        g = dict(row=row.cpu().numpy(), cols=cols.cpu().numpy(), fmaps=[sp.feature_map(k) for k in range(len(wl.species))],
                 jedge={}, jself={})
        for c in idx:
            r0, r1 = int(g["row"][c]), int(g["row"][c + 1])
            g["jedge"][int(c)] = je[r0:r1].cpu().double().numpy()
            g["jself"][int(c)] = js[int(c)].cpu().double().numpy()
        ed = row_errors(d.cpu().double().numpy()[idx], ref["desc"]).max()
        ej = jacobian_errors(g, ref, st, wl.species, idx.tolist(), idx)
        print(f"[outputs] {case} {dtype} out_rows {rows} (groups {groups}, rows kernel {used_rows}): "
              f"desc {ed:.2e} jac {ej:.2e}", flush=True)
        assert ed < TOL[dtype] and ej < TOL[dtype]
        if rows == 0:
            assert used_rows == 0
        if first is None:
            first = (d.clone(), je.clone(), js.clone())
        elif dtype == "float64":
            for x, y in zip((d, je, js), first):
                assert torch.equal(x, y)
        sp.close()


@pytest.mark.parametrize("dtype", ["float32", "float64"])
@pytest.mark.parametrize("case", ["chno_poly_n10l10", "water_poly_n8l6", "water_gto_n8l12", "five_species_gto_n4l4"])
def test_streamed_density_kernel(dtype, case):
    """The density step of the Jacobian path that streams the coefficients to
    the scratch (one workgroup per center, one species' sums in registers at
    a time; the output kernel then writes the descriptor and center blocks):
    descriptor and every block of every center against the oracle at each
    chunk width that fits, the same bits at every width, and the shared
    density kernel (l-groups) within the tolerance of the oracle too."""
    import torch
    from paper_2609_05709_amd.soap import Soap
    if case == "chno_poly_n10l10":
        wl = workloads.Workload(case, (1, 6, 7, 8), "polynomial", 5.0, 0.4, 10, 10, True, ("none",))
        st = workloads.random_small(60, 41, 5.0, species=(1, 6, 7, 8), dmin=0.85)
    elif case == "water_poly_n8l6":
        wl = dataclasses.replace(workloads.WATER64, name=case, rbf="polynomial", n_max=8, l_max=6)
        st = structure(workloads.WATER64)
    elif case == "water_gto_n8l12":
        wl = dataclasses.replace(workloads.WATER64, name=case, n_max=8, l_max=12)
        st = structure(workloads.WATER64)
    else:
        wl = workloads.Workload(case, (1, 6, 7, 8, 16), "gto", 5.0, 0.45, 4, 4, True, ("none",))
        st = workloads.random_small(70, 53, 5.0, species=(1, 6, 7, 8, 16), dmin=0.85)
    idx = np.arange(st.n_atoms)
    ref = oracle_for(wl).compute(st.pos64, st.Z, centers=idx, jacobian=True)
    tdt = torch.float64 if dtype == "float64" else torch.float32
    pos = torch.from_numpy(st.pos.astype(np.float64) if dtype == "float64" else st.pos).to("cuda", tdt)
    Z = torch.from_numpy(st.Z).cuda()
    first, ran = None, 0
    for tile in (64, 32, 16, -1):
        sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, dtype=dtype)
        sp._check(sp._L.soap_set_option(sp._h, b"djs_tile", tile))
        kern, got = sp.get_option("jacobian_density_kernel"), sp.get_option("jacobian_density_tile")
        if tile > 0 and (kern != 2 or got != tile):
            sp.close()  # this width does not fit the on-chip plan
            continue
        if tile == -1:
            assert kern == 0
        sp.build_neighbors(pos, Z)
        d, je, js = sp.derivatives()
        row, cols = sp.neighbors()
        torch.cuda.synchronize()
        g = dict(row=row.cpu().numpy(), cols=cols.cpu().numpy(), fmaps=[sp.feature_map(k) for k in range(len(wl.species))],
                 jedge={}, jself={})
        for c in idx:
            r0, r1 = int(g["row"][c]), int(g["row"][c + 1])
            g["jedge"][int(c)] = je[r0:r1].cpu().double().numpy()
            g["jself"][int(c)] = js[int(c)].cpu().double().numpy()
        ed = row_errors(d.cpu().double().numpy()[idx], ref["desc"]).max()
        ej = jacobian_errors(g, ref, st, wl.species, idx.tolist(), idx)
        print(f"[djs] {case} {dtype} tile {tile} (kernel {kern}): desc {ed:.2e} jac {ej:.2e}", flush=True)
        assert ed < TOL[dtype] and ej < TOL[dtype]
        if tile > 0:
            ran += 1
            if first is None:
                first = (d.clone(), je.clone(), js.clone())
            else:
                for x, y in zip((d, je, js), first):
                    assert torch.equal(x, y)
        sp.close()
    assert ran >= 1
