"""The bench's algorithmic byte model (the numerator of its roofline
fraction) against an independent count: the oracle's enumerated feature list
and its brute-force neighbour rows."""
import numpy as np

import bench
import oracle
from paper_2609_05709_amd import workloads


def test_feature_counts_match_the_enumerated_features():
    for species, n, l in [((1, 8), 8, 6), ((1, 6, 7, 8), 10, 10), ((8,), 3, 2)]:
        o = oracle.OracleSOAP(species, 5.0, n, l, 0.5, "gto")
        feats = o.features()
        S = len(species)
        assert len(feats) == (l + 1) * (S * n) * (S * n + 1) // 2
        for s in range(S):
            fe = sum(1 for (mu, nu, a, b, ll) in feats if s in (mu, nu))
            assert fe == (l + 1) * (n * (n + 1) // 2 + (S - 1) * n * n)


def test_algorithmic_bytes_of_the_headline_workload():
    wl = workloads.WATER1000
    st = wl.structure()
    row, cols = oracle.neighbors(st.pos64, wl.r_cut)
    E = len(cols)
    assert E == 204662
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    feats = o.features()
    F = len(feats)
    spec = {z: k for k, z in enumerate(sorted(wl.species))}
    fe_of = [sum(1 for (mu, nu, a, b, l) in feats if s in (mu, nu)) for s in range(len(wl.species))]
    # float32 outputs that can be non-zero: every descriptor entry, every
    # center-block entry, and per edge the features of pairs containing the
    # neighbour's species
    edge_vals = 3 * sum(fe_of[spec[int(z)]] for z in st.Z[cols])
    expect_jac = 4 * edge_vals
    expect_step = 4 * (st.n_atoms * F + 3 * st.n_atoms * F) + expect_jac
    alg = bench.algorithmic(wl, st.n_atoms, E, F, fe_of[0], 4, True)
    assert alg["jacobian"] == expect_jac == 1_719_160_800
    assert alg["step"] == expect_step == 1_764_856_800
    assert alg["density"] + alg["jacobian"] == alg["step"]
    assert np.all(np.diff(row) >= 0)
