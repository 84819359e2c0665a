"""Center batches (Sec. 3.3: centers streamed through the device in batches
that bound the memory of one call), bitwise repeatability, the degree limit,
and the density kernel's work counters across modes."""
import numpy as np
import pytest

import oracle
from paper_2609_05709_amd import workloads
from tests.parity import TOL, gpu_run, jacobian_errors, row_errors

pytestmark = pytest.mark.gpu


def _ctx(wl, st, dtype="float32", **kw):
    import torch
    from paper_2609_05709_amd.soap import Soap
    tdt = torch.float64 if dtype == "float64" else torch.float32
    sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, dtype=dtype, **kw)
    pos = torch.from_numpy(st.pos.astype(np.float64) if dtype == "float64" else st.pos).to("cuda", tdt)
    Z = torch.from_numpy(st.Z).cuda()
    sp.build_neighbors(pos, Z)
    return sp


def test_batches_descriptor_million_atoms_bitwise():
    """The 1,000,002-atom water descriptor streamed in batches sized by a
    memory budget equals the single call bit for bit."""
    import torch
    wl = workloads.WATER1M
    st = wl.structure()
    print(f"[batch] {wl.name} atoms={st.n_atoms}", flush=True)
    sp = _ctx(wl, st)
    whole = sp.compute()
    budget = st.n_atoms * sp.n_features * 4 // 5 + 1
    cf, _ = sp.plan_batches(budget, jacobian=False)
    assert len(cf) - 1 >= 4
    out = torch.empty_like(whole[: int(np.diff(cf).max())])
    for k in range(len(cf) - 1):
        a, b = int(cf[k]), int(cf[k + 1])
        part = sp.compute_batch(a, b - a, out=out[: b - a])
        assert torch.equal(part, whole[a:b]), k
    torch.cuda.synchronize()
    print(f"[batch] {len(cf) - 1} batches bitwise equal", flush=True)
    sp.close()


@pytest.mark.parametrize("dtype", ["float32", "float64"])
def test_batches_derivatives_30k_water(dtype):
    """Descriptor + Jacobian of a 30,000-atom water cluster (GTO n8 l6,
    r_cut 6): batches sized by a budget equal the single call bit for bit,
    and sampled centers match the oracle."""
    import torch
    wl = workloads.Workload("water10000_gto_n8l6", (1, 8), "gto", 6.0, 0.5, 8, 6, True, ("water", 10000, 7))
    st = wl.structure()
    print(f"[batch] {wl.name} {dtype} atoms={st.n_atoms}", flush=True)
    sp = _ctx(wl, st, dtype)
    desc, jedge, jself = sp.derivatives()
    row, cols = sp.neighbors()
    total = desc.numel() * desc.element_size() * 4 + jedge.numel() * jedge.element_size()
    cf, ef = sp.plan_batches(total // 6, jacobian=True)
    nb = len(cf) - 1
    assert nb >= 6
    assert np.array_equal(ef, row.cpu().numpy()[cf])
    for k in range(nb):
        a, b = int(cf[k]), int(cf[k + 1])
        d, je, js = sp.derivatives_batch(a, b - a, int(ef[k + 1] - ef[k]))
        assert torch.equal(d, desc[a:b]) and torch.equal(js, jself[a:b]), k
        assert torch.equal(je, jedge[int(ef[k]):int(ef[k + 1])]), k
        del d, je, js
    torch.cuda.synchronize()
    print(f"[batch] {nb} batches bitwise equal", flush=True)
    # sampled centers against the oracle
    rng = np.random.default_rng(11)
    idx = np.sort(rng.choice(st.n_atoms, size=12, replace=False))
    g = dict(row=row.cpu().numpy(), cols=cols.cpu().numpy(), fmaps=[sp.feature_map(s) for s in range(2)],
             jedge={}, jself={})
    for c in idx:
        r0, r1 = int(g["row"][c]), int(g["row"][c + 1])
        g["jedge"][int(c)] = jedge[r0:r1].cpu().double().numpy()
        g["jself"][int(c)] = jself[int(c)].cpu().double().numpy()
    got_d = desc[torch.from_numpy(idx).cuda()].cpu().double().numpy()
    sp.close()
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    ref = o.compute(st.pos64, st.Z, centers=idx, jacobian=True)
    ed = row_errors(got_d, ref["desc"]).max()
    ej = jacobian_errors(g, ref, st, wl.species, idx.tolist(), idx)
    print(f"[batch] {wl.name} {dtype}: desc {ed:.2e} jac {ej:.2e}", flush=True)
    assert ed < TOL[dtype] and ej < TOL[dtype]


def test_plan_batches_budget_and_errors():
    """Every planned batch fits the budget; a budget below one center's
    outputs is a capacity error; a batch outside the centers is rejected."""
    from paper_2609_05709_amd.soap import SOAP_ECAPACITY, SOAP_EINVAL, SoapError
    wl = workloads.WATER64
    st = wl.structure()
    sp = _ctx(wl, st)
    row, _ = sp.neighbors()
    row = row.cpu().numpy()
    F, Fe, S, L = sp.n_features, sp.n_edge_features, 2, (wl.l_max + 1) ** 2
    # float32 outputs and, in the mixed mode, a float32 coefficient scratch
    per_c = 4 * F * 4 + 16 * S * wl.n_max * L
    budget = 20 * per_c
    cf, ef = sp.plan_batches(budget, jacobian=True)
    assert cf[0] == 0 and cf[-1] == st.n_atoms and np.all(np.diff(cf) > 0)
    for k in range(len(cf) - 1):
        a, b = cf[k], cf[k + 1]
        used = (b - a) * per_c + (row[b] - row[a]) * 3 * Fe * 4
        assert used <= budget
        if b < st.n_atoms:  # greedy: the next center would not have fit
            assert used + per_c + (row[b + 1] - row[b]) * 3 * Fe * 4 > budget
    with pytest.raises(SoapError) as ei:
        sp.plan_batches(per_c // 2, jacobian=True)
    assert ei.value.code == SOAP_ECAPACITY
    with pytest.raises(SoapError) as ei:
        sp.compute_batch(st.n_atoms - 2, 3)
    assert ei.value.code == SOAP_EINVAL
    sp.close()


@pytest.mark.parametrize("which", ["water1000", "chno4096"])
def test_repeatable_bitwise_float64(which):
    """Two runs of descriptor + Jacobian in float64 give the same bits: the
    per-center sums run in a fixed order (no arrival-order atomics)."""
    import torch
    wl = {"water1000": workloads.WATER1000, "chno4096": workloads.CHNO4096}[which]
    st = wl.structure()
    print(f"[repeat] {wl.name} float64", flush=True)
    sp = _ctx(wl, st, "float64")
    a = [t.clone() for t in sp.derivatives()]
    b = sp.derivatives()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    c = sp.coefficients()
    assert torch.equal(c, sp.coefficients())
    sp.close()


def test_degree_above_limit_is_a_capacity_error():
    """A center with more than 2048 neighbours: soap_build_neighbors returns
    SOAP_ECAPACITY and leaves no neighbour list (nothing is computed); 2048
    neighbours exactly are accepted and match the oracle."""
    import torch
    from paper_2609_05709_amd.soap import SOAP_ECAPACITY, SOAP_ESTATE, Soap, SoapError
    wl = workloads.Workload("dense", (1, 8), "gto", 5.0, 0.5, 2, 2, True, ("none",))
    rng = np.random.default_rng(5)
    for n_atoms, ok in ((2050, False), (2049, True)):
        v = rng.normal(size=(n_atoms, 3))
        pos = (v / np.linalg.norm(v, axis=1, keepdims=True) * 2.0 * rng.uniform(0, 1, (n_atoms, 1)) ** (1 / 3))
        st = workloads.Structure(pos.astype(np.float32), np.array([1, 8] * (n_atoms // 2) + [1] * (n_atoms % 2),
                                                                 dtype=np.int32), 2.0, 0)
        print(f"[capacity] {n_atoms} atoms in a 2 A ball, r_cut 5", flush=True)
        if not ok:
            sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
            with pytest.raises(SoapError) as ei:
                sp.build_neighbors(torch.from_numpy(st.pos).cuda(), torch.from_numpy(st.Z).cuda())
            assert ei.value.code == SOAP_ECAPACITY
            with pytest.raises(SoapError) as ei:
                sp.compute()
            assert ei.value.code == SOAP_ESTATE
            sp.close()
            continue
        sample = [0, 1, 777, 2048]
        g = gpu_run(wl, st, "float32", sample=sample)
        assert np.all(np.diff(g["row"]) == 2048)
        o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
        ref = o.compute(st.pos64, st.Z, centers=np.asarray(sample), jacobian=True)
        assert row_errors(g["desc"][sample], ref["desc"]).max() < TOL["float32"]
        assert jacobian_errors(g, ref, st, wl.species, sample, np.asarray(sample)) < TOL["float32"]


def _shared_density_kernel(sp):
    """Route the Jacobian path through the shared (work-counter) density
    kernel, as the streaming one would otherwise take these bases."""
    sp._check(sp._L.soap_set_option(sp._h, b"djs_tile", -1))
    assert sp.get_option("jacobian_density_kernel") == 0
    return sp


@pytest.mark.parametrize("case", ["8species_n8l6", "chno_quad128"])
@pytest.mark.parametrize("density", ["shared", "auto"])
def test_modes_with_different_group_counts(case, density):
    """Descriptor, Jacobian and coefficient calls in any order on one
    neighbour list, for bases whose density modes split l into different
    numbers of groups (each group's work counter keeps its own count): every
    result equals a fresh context's, and the first ones match the oracle.
    "shared": the Jacobian path on the shared density kernel as well (three
    modes, three group counts); "auto": the planner's choice."""
    import torch
    if case == "8species_n8l6":
        species = tuple(range(1, 9))
        wl = workloads.Workload("s8", species, "gto", 5.0, 0.5, 8, 6, True, ("none",))
        st = workloads.random_small(80, 21, 4.5, species=species, dmin=0.8)
        kw = {}
    else:
        wl = workloads.Workload("chno", (1, 6, 7, 8), "polynomial", 5.0, 0.4, 10, 10, True, ("none",))
        st = workloads.random_small(80, 22, 5.0, species=(1, 6, 7, 8), dmin=0.9)
        kw = dict(quad_n=128)
    print(f"[modes] {case}", flush=True)
    sp = _ctx(wl, st, **kw)
    fresh = _ctx(wl, st, **kw)
    if density == "shared":
        sp, fresh = _shared_density_kernel(sp), _shared_density_kernel(fresh)
    d0 = fresh.compute().clone()
    j0 = [t.clone() for t in fresh.derivatives()]
    c0 = fresh.coefficients().clone()
    fresh.close()
    for _ in range(2):
        assert torch.equal(sp.compute(), d0)
        for x, y in zip(sp.derivatives(), j0):
            assert torch.equal(x, y)
        assert torch.equal(sp.coefficients(), c0)
        assert torch.equal(sp.compute(), d0)
    sp.close()
    idx = np.arange(0, st.n_atoms, 9)
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, **kw)
    ref = o.compute(st.pos64, st.Z, centers=idx)
    assert row_errors(d0.cpu().double().numpy()[idx], ref["desc"]).max() < TOL["float32"]


def test_basis_too_large_for_the_jacobian_path():
    """16 species at n_max 8, l_max 6 (S n = 128): the descriptor path fits
    and matches the oracle; the Jacobian paths are refused with SOAP_EINVAL."""
    from paper_2609_05709_amd.soap import SOAP_EINVAL, SoapError
    species = tuple(range(1, 17))
    wl = workloads.Workload("s16", species, "gto", 5.0, 0.5, 8, 6, True, ("none",))
    st = workloads.random_small(64, 23, 4.5, species=species, dmin=0.8)
    sp = _ctx(wl, st)
    desc = sp.compute().cpu().double().numpy()
    with pytest.raises(SoapError) as ei:
        sp.derivatives()
    assert ei.value.code == SOAP_EINVAL
    sp.close()
    idx = np.arange(0, st.n_atoms, 7)
    ref = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf).compute(
        st.pos64, st.Z, centers=idx)
    assert row_errors(desc[idx], ref["desc"]).max() < TOL["float32"]


@pytest.mark.parametrize("chunks,wg", [(2, 0), (3, 1), (4, 2)])
def test_pipelined_derivatives_bitwise(chunks, wg):
    """The pipelined derivatives (center chunks, the Jacobian kernel of a
    chunk on a second stream beside the density kernel of the next) give the
    same bits as the single-stream call, for the whole list and for a batch."""
    import torch
    wl = workloads.WATER1000
    st = wl.structure()
    sp = _ctx(wl, st)
    ref = [t.clone() for t in sp.derivatives()]
    cf, ef = sp.plan_batches(10**9, jacobian=True)
    a, b = 700, 1500
    row, _ = sp.neighbors()
    row = row.cpu().numpy()
    ref_b = [t.clone() for t in sp.derivatives_batch(a, b - a, int(row[b] - row[a]))]
    sp._check(sp._L.soap_set_option(sp._h, b"pipeline", chunks))
    sp._check(sp._L.soap_set_option(sp._h, b"pipeline_density_wg", wg))
    for _ in range(2):
        for x, y in zip(sp.derivatives(), ref):
            assert torch.equal(x, y)
        for x, y in zip(sp.derivatives_batch(a, b - a, int(row[b] - row[a])), ref_b):
            assert torch.equal(x, y)
    sp.close()


@pytest.mark.parametrize("case", ["water1000", "chno4096"])
def test_batch_centers_option(case):
    """soap_derivatives with the "batch_centers" option (the call's centers in
    consecutive batches, the scratch sized for one batch): every output bit
    for bit equal to one batch; the context reports its device."""
    import torch
    wl = workloads.WATER1000 if case == "water1000" else workloads.CHNO4096
    st = wl.structure()
    print(f"[batch_centers] {case}", flush=True)
    sp = _ctx(wl, st)
    assert sp.get_option("device") == torch.cuda.current_device()
    ref = [t.clone() for t in sp.derivatives()]
    for B in (997, 64):
        sp.set_option("batch_centers", B)
        assert sp.get_option("batch_centers") == B
        out = sp.derivatives()
        torch.cuda.synchronize()
        for x, y in zip(out, ref):
            assert torch.equal(x, y), (case, B)
    sp.set_option("batch_centers", 0)
    sp.close()
