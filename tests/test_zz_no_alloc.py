"""soap_derivatives_batch_noalloc (the allocation-free variant, for callers
that cannot allocate) against soap_derivatives_batch, called through the C
ABI: two calls in a row, the second with a smaller input, bitwise equal; a
batch above the static scratch is refused."""
import ctypes

import numpy as np
import pytest

from paper_2609_05709_amd import workloads

pytestmark = pytest.mark.gpu


def _run_pair(L, wl, st, first, count):
    """One context: outputs of centers [first, first + count) from the
    existing batch entry point and from the allocation-free one."""
    import torch
    from paper_2609_05709_amd.soap import RBF_CODES, SOAP_OK
    z = np.ascontiguousarray(sorted(wl.species), dtype=np.int32)
    h = ctypes.c_void_p()
    assert L.soap_create(z.ctypes.data, len(z), wl.r_cut, wl.n_max, wl.l_max, wl.sigma, RBF_CODES[wl.rbf],
                         ctypes.byref(h)) == SOAP_OK
    pos = torch.from_numpy(st.pos).cuda()
    Z = torch.from_numpy(st.Z).cuda()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    E = ctypes.c_int64()
    assert L.soap_build_neighbors(h, st.n_atoms, pos.data_ptr(), Z.data_ptr(), st.n_atoms, None, ctypes.byref(E),
                                  stream) == SOAP_OK
    F, Fe = L.soap_num_features(h), L.soap_num_edge_features(h)
    row = torch.empty(st.n_atoms + 1, dtype=torch.int64, device="cuda")
    assert L.soap_get_neighbors(h, row.data_ptr(), None, stream) == SOAP_OK
    torch.cuda.synchronize()
    eb = int(row[first + count] - row[first])
    outs = []
    for fn in (L.soap_derivatives_batch, L.soap_derivatives_batch_noalloc):
        desc = torch.full((count, F), float("nan"), device="cuda")
        je = torch.full((max(eb, 1), 3, Fe), float("nan"), device="cuda")
        js = torch.full((count, 3, F), float("nan"), device="cuda")
        assert fn(h, first, count, desc.data_ptr(), je.data_ptr(), js.data_ptr(), stream) == SOAP_OK, \
            L.soap_last_error(h)
        torch.cuda.synchronize()
        outs.append((desc, je[:eb], js))
    L.soap_destroy(h)
    return outs


def test_noalloc_matches_batch_entry_point():
    import torch
    from paper_2609_05709_amd.soap import load_library
    L = load_library()
    # first call: 2000 centers of the 3000-atom water cluster (25 MB of float32
    # scratch in the mixed mode)
    wl = workloads.WATER1000
    print("[noalloc] water1000 centers [500, 2500)", flush=True)
    a, b = _run_pair(L, wl, wl.structure(), 500, 2000)
    for x, y in zip(a, b):
        assert not torch.isnan(x).any()
        assert torch.equal(x, y)
    # second call, smaller: the 64-water cluster, every center
    wl = workloads.WATER64
    print("[noalloc] water64 all centers", flush=True)
    a, b = _run_pair(L, wl, wl.structure(), 0, 192)
    for x, y in zip(a, b):
        assert not torch.isnan(x).any()
        assert torch.equal(x, y)


def test_noalloc_refuses_batches_above_the_static_scratch():
    import torch
    from paper_2609_05709_amd.soap import RBF_CODES, SOAP_ECAPACITY, SOAP_OK, load_library
    L = load_library()
    wl = workloads.CHNO4096
    st = wl.structure()
    z = np.ascontiguousarray(sorted(wl.species), dtype=np.int32)
    h = ctypes.c_void_p()
    assert L.soap_create(z.ctypes.data, len(z), wl.r_cut, wl.n_max, wl.l_max, wl.sigma, RBF_CODES[wl.rbf],
                         ctypes.byref(h)) == SOAP_OK
    pos, Z = torch.from_numpy(st.pos).cuda(), torch.from_numpy(st.Z).cuda()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    E = ctypes.c_int64()
    assert L.soap_build_neighbors(h, st.n_atoms, pos.data_ptr(), Z.data_ptr(), st.n_atoms, None, ctypes.byref(E),
                                  stream) == SOAP_OK
    # 4096 centers need 317 MB of float32 coefficient scratch (16 S n L bytes
    # per center, S = 4, n = 10, L = 121): above the 64 MiB array
    desc = torch.empty(1, device="cuda")
    assert L.soap_derivatives_batch_noalloc(h, 0, st.n_atoms, desc.data_ptr(), desc.data_ptr(), desc.data_ptr(),
                                            stream) == SOAP_ECAPACITY
    assert b"static" in L.soap_last_error(h)
    L.soap_destroy(h)
