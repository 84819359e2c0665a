"""Python binding of libsoap.so (include/soap.h): argument marshalling only.

Every step of the descriptor and Jacobian runs in the library's HIP kernels;
torch provides device memory and the current stream.  If the library is not
built this module raises on use: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsoap.so")

SOAP_OK, SOAP_EINVAL, SOAP_ESPECIES, SOAP_ENOMEM, SOAP_EHIP, SOAP_ECAPACITY, SOAP_ESTATE = 0, -1, -2, -3, -4, -5, -6
SOAP_RBF_GTO, SOAP_RBF_POLYNOMIAL, SOAP_RBF_POLYNOMIAL_LAPLACE = 0, 1, 2
RBF_CODES = {"gto": SOAP_RBF_GTO, "polynomial": SOAP_RBF_POLYNOMIAL,
             "polynomial-laplace": SOAP_RBF_POLYNOMIAL_LAPLACE}
SOAP_FP32, SOAP_FP64 = 0, 1
SOAP_AVERAGE_INNER, SOAP_AVERAGE_OUTER = 1, 2
SOAP_ARITH_MIXED, SOAP_ARITH_FP64 = 0, 1
ARITH_CODES = {"mixed": SOAP_ARITH_MIXED, "fp64": SOAP_ARITH_FP64}
SOAP_BATCH_DESCRIPTOR, SOAP_BATCH_DERIVATIVES = 0, 1
MAX_DEGREE = 2048

# every entry point declared in include/soap.h
ABI_SYMBOLS = ("soap_create", "soap_set_option", "soap_get_option", "soap_num_features", "soap_num_edge_features",
               "soap_feature_labels", "soap_feature_map", "soap_build_neighbors", "soap_get_neighbors",
               "soap_set_cell", "soap_get_neighbor_images",
               "soap_compute", "soap_coefficients", "soap_coefficient_derivatives", "soap_compute_averaged",
               "soap_derivatives", "soap_compute_batch", "soap_derivatives_batch", "soap_derivatives_batch_noalloc",
               "soap_plan_batches",
               "soap_scatter_dense", "soap_timing",
               "soap_last_error", "soap_destroy")

_STATUS = {SOAP_EINVAL: "EINVAL", SOAP_ESPECIES: "ESPECIES", SOAP_ENOMEM: "ENOMEM", SOAP_EHIP: "EHIP",
           SOAP_ECAPACITY: "ECAPACITY", SOAP_ESTATE: "ESTATE"}


class SoapError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_STATUS.get(code, code)}: {msg}")
        self.code = code


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libsoap.so and declare the C ABI; raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library {path} is not built (run __graft_entry__.build())")
    L = ctypes.CDLL(path)
    vp, i32, i64, dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    L.soap_create.restype = ctypes.c_int
    L.soap_create.argtypes = [vp, i32, dbl, i32, i32, dbl, i32, ctypes.POINTER(vp)]
    L.soap_set_option.restype = ctypes.c_int
    L.soap_set_option.argtypes = [vp, ctypes.c_char_p, i64]
    L.soap_get_option.restype = ctypes.c_int
    L.soap_get_option.argtypes = [vp, ctypes.c_char_p, ctypes.POINTER(i64)]
    L.soap_num_features.restype = i64
    L.soap_num_features.argtypes = [vp]
    L.soap_num_edge_features.restype = i64
    L.soap_num_edge_features.argtypes = [vp]
    L.soap_feature_labels.restype = ctypes.c_int
    L.soap_feature_labels.argtypes = [vp, vp]
    L.soap_feature_map.restype = ctypes.c_int
    L.soap_feature_map.argtypes = [vp, i32, vp]
    L.soap_build_neighbors.restype = ctypes.c_int
    L.soap_build_neighbors.argtypes = [vp, i64, vp, vp, i64, vp, ctypes.POINTER(i64), vp]
    L.soap_get_neighbors.restype = ctypes.c_int
    L.soap_get_neighbors.argtypes = [vp, vp, vp, vp]
    L.soap_compute.restype = ctypes.c_int
    L.soap_compute.argtypes = [vp, vp, vp]
    L.soap_coefficients.restype = ctypes.c_int
    L.soap_coefficients.argtypes = [vp, vp, vp]
    L.soap_derivatives.restype = ctypes.c_int
    L.soap_derivatives.argtypes = [vp, vp, vp, vp, vp]
    L.soap_compute_batch.restype = ctypes.c_int
    L.soap_compute_batch.argtypes = [vp, i64, i64, vp, vp]
    L.soap_derivatives_batch.restype = ctypes.c_int
    L.soap_derivatives_batch.argtypes = [vp, i64, i64, vp, vp, vp, vp]
    L.soap_derivatives_batch_noalloc.restype = ctypes.c_int
    L.soap_derivatives_batch_noalloc.argtypes = [vp, i64, i64, vp, vp, vp, vp]
    L.soap_plan_batches.restype = ctypes.c_int
    L.soap_plan_batches.argtypes = [vp, i32, i64, i64, vp, vp, ctypes.POINTER(i64)]
    L.soap_scatter_dense.restype = ctypes.c_int
    L.soap_scatter_dense.argtypes = [vp, vp, vp, vp, vp]
    L.soap_set_cell.restype = ctypes.c_int
    L.soap_set_cell.argtypes = [vp, vp, vp]
    L.soap_get_neighbor_images.restype = ctypes.c_int
    L.soap_get_neighbor_images.argtypes = [vp, vp, vp]
    L.soap_coefficient_derivatives.restype = ctypes.c_int
    L.soap_coefficient_derivatives.argtypes = [vp, vp, vp, vp, vp]
    L.soap_compute_averaged.restype = ctypes.c_int
    L.soap_compute_averaged.argtypes = [vp, i32, vp, vp]
    L.soap_timing.restype = ctypes.c_int
    L.soap_timing.argtypes = [vp, vp, vp, i32]
    L.soap_last_error.restype = ctypes.c_char_p
    L.soap_last_error.argtypes = [vp]
    L.soap_destroy.restype = None
    L.soap_destroy.argtypes = [vp]
    _lib = L
    return L


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


class Soap:
    """One library context: species, r_cut, n_max, l_max, sigma, rbf
    ("gto" | "polynomial" | "polynomial-laplace"), dtype ("float32" | "float64"),
    arith ("mixed" | "fp64": the float32 mode's internal arithmetic), device
    (made current before soap_create; None = the current device)."""

    def __init__(self, species, r_cut, n_max, l_max, sigma, rbf="gto", dtype="float32", quad_n=None,
                 arith="mixed", device=None):
        import numpy as np
        import torch
        self._L = load_library()
        if not torch.cuda.is_available():
            raise RuntimeError("no HIP device available")
        if device is not None:
            # the context lives on the device current at soap_create
            torch.cuda.set_device(torch.device(device))
        self.species = sorted(int(z) for z in species)
        self.r_cut, self.n_max, self.l_max, self.sigma = float(r_cut), int(n_max), int(l_max), float(sigma)
        if rbf not in RBF_CODES:
            raise ValueError(f"unknown rbf {rbf!r}; expected one of {sorted(RBF_CODES)}")
        self.rbf = rbf
        self.dtype = torch.float64 if dtype in ("float64", torch.float64) else torch.float32
        z = np.ascontiguousarray(self.species, dtype=np.int32)
        h = ctypes.c_void_p()
        code = self._L.soap_create(z.ctypes.data, len(z), self.r_cut, self.n_max, self.l_max, self.sigma,
                                   RBF_CODES[rbf], ctypes.byref(h))
        if code != SOAP_OK:
            raise SoapError(code, "soap_create: " + self._L.soap_last_error(None).decode())
        self._h = h
        if self.dtype == torch.float64:
            self._check(self._L.soap_set_option(self._h, b"dtype", SOAP_FP64))
        if quad_n is not None:
            self._check(self._L.soap_set_option(self._h, b"quad_n", int(quad_n)))
        if arith not in ARITH_CODES:
            raise ValueError(f"unknown arith {arith!r}; expected one of {sorted(ARITH_CODES)}")
        if arith != "mixed":
            self._check(self._L.soap_set_option(self._h, b"arith", ARITH_CODES[arith]))
        self.n_features = int(self._L.soap_num_features(self._h))
        self.n_edge_features = int(self._L.soap_num_edge_features(self._h))
        self.E = None
        self.n_centers = None
        self._keep = ()

    # -- helpers -------------------------------------------------------------
    def _check(self, code):
        if code != SOAP_OK:
            raise SoapError(code, self._L.soap_last_error(self._h).decode())

    def close(self):
        if getattr(self, "_h", None):
            self._L.soap_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_timing(self, on: bool):
        self._check(self._L.soap_set_option(self._h, b"timing", 1 if on else 0))

    def get_option(self, key: str) -> int:
        v = ctypes.c_int64()
        self._check(self._L.soap_get_option(self._h, key.encode(), ctypes.byref(v)))
        return int(v.value)

    def set_option(self, key: str, value: int):
        self._check(self._L.soap_set_option(self._h, key.encode(), int(value)))

    def timing(self, reset: bool = True):
        """(ms[3], counts[3]) summed over timed calls: neighbour search, density
        kernel, edge Jacobian kernel."""
        import numpy as np
        ms = np.zeros(3)
        cnt = np.zeros(3, dtype=np.int64)
        self._check(self._L.soap_timing(self._h, ms.ctypes.data, cnt.ctypes.data, 1 if reset else 0))
        return ms, cnt

    def feature_labels(self):
        import numpy as np
        out = np.empty((self.n_features, 5), dtype=np.int32)
        self._check(self._L.soap_feature_labels(self._h, out.ctypes.data))
        return out

    def feature_map(self, species_index: int):
        import numpy as np
        out = np.empty(self.n_edge_features, dtype=np.int32)
        self._check(self._L.soap_feature_map(self._h, int(species_index), out.ctypes.data))
        return out

    # -- neighbour rows --------------------------------------------------------
    def build_neighbors(self, pos, Z, centers=None) -> int:
        """pos: (N, 3) device tensor of self.dtype; Z: (N,) int32 device tensor;
        centers: optional (n_centers,) int32 device tensor."""
        import torch
        if pos.dtype != self.dtype or not pos.is_cuda or pos.dim() != 2 or pos.shape[1] != 3:
            raise ValueError("pos must be a (N, 3) device tensor of the context dtype")
        if Z.dtype != torch.int32 or not Z.is_cuda or Z.shape[0] != pos.shape[0]:
            raise ValueError("Z must be an (N,) int32 device tensor")
        pos, Z = pos.contiguous(), Z.contiguous()
        nc = pos.shape[0]
        cptr = None
        if centers is not None:
            if centers.dtype != torch.int32 or not centers.is_cuda:
                raise ValueError("centers must be an int32 device tensor")
            centers = centers.contiguous()
            nc = centers.shape[0]
            cptr = centers.data_ptr()
        E = ctypes.c_int64()
        self.E = self.n_centers = None
        self._check(self._L.soap_build_neighbors(self._h, pos.shape[0], pos.data_ptr(), Z.data_ptr(), nc, cptr,
                                                 ctypes.byref(E), _stream()))
        self._keep = (pos, Z, centers)  # the library reads these in later calls
        self.E, self.n_centers, self.n_atoms = int(E.value), int(nc), int(pos.shape[0])
        return self.E

    def set_cell(self, cell=None, pbc=(True, True, True)):
        """Periodic cell (3 x 3, lattice vectors as rows, angstrom) and periodic
        directions for the next build_neighbors; None = open boundaries."""
        import numpy as np
        self.E = self.n_centers = None
        if cell is None:
            self._check(self._L.soap_set_cell(self._h, None, None))
            return
        c = np.ascontiguousarray(np.asarray(cell, dtype=np.float64).reshape(9))
        p = np.ascontiguousarray(np.asarray(pbc, dtype=np.int32).reshape(3))
        self._check(self._L.soap_set_cell(self._h, c.ctypes.data, p.ctypes.data))

    def neighbor_images(self):
        """(E, 3) int32 image index of every edge of the last build."""
        import torch
        if self.E is None:
            raise SoapError(SOAP_ESTATE, "no neighbour list: call build_neighbors first")
        img = torch.empty((max(self.E, 1), 3), dtype=torch.int32, device="cuda")
        self._check(self._L.soap_get_neighbor_images(self._h, img.data_ptr(), _stream()))
        return img[: self.E]

    def neighbors(self):
        import torch
        if self.E is None:
            raise SoapError(SOAP_ESTATE, "no neighbour list: call build_neighbors first")
        row = torch.empty(self.n_centers + 1, dtype=torch.int64, device="cuda")
        cols = torch.empty(max(self.E, 1), dtype=torch.int32, device="cuda")
        self._check(self._L.soap_get_neighbors(self._h, row.data_ptr(), cols.data_ptr(), _stream()))
        return row, cols[: self.E]

    # -- outputs ----------------------------------------------------------------
    def _out(self, t, shape):
        import torch
        if self.E is None:
            raise SoapError(SOAP_ESTATE, "no neighbour list: call build_neighbors first")
        if t is None:
            return torch.empty(shape, dtype=self.dtype, device="cuda")
        if tuple(t.shape) != tuple(shape) or t.dtype != self.dtype or not t.is_contiguous():
            raise ValueError(f"output must be a contiguous {self.dtype} tensor of shape {shape}")
        return t

    def compute(self, out=None):
        desc = self._out(out, (self.n_centers, self.n_features))
        self._check(self._L.soap_compute(self._h, desc.data_ptr(), _stream()))
        return desc

    def coefficients(self, out=None):
        S, L = len(self.species), (self.l_max + 1) ** 2
        c = self._out(out, (self.n_centers, S, self.n_max, L))
        self._check(self._L.soap_coefficients(self._h, c.data_ptr(), _stream()))
        return c

    def coefficient_derivatives(self, c=None, jc_edge=None, jc_self=None):
        """The "cc" mode: coefficients c (n_c, S, n_max, L), their edge
        gradients jc_edge (E, 3, n_max, L) = d c^{species(j)}(i) / d r_j and the
        center blocks jc_self (n_c, 3, S, n_max, L)."""
        S, L = len(self.species), (self.l_max + 1) ** 2
        c = self._out(c, (self.n_centers, S, self.n_max, L))
        jc_edge = self._out(jc_edge, (self.E, 3, self.n_max, L))
        jc_self = self._out(jc_self, (self.n_centers, 3, S, self.n_max, L))
        self._check(self._L.soap_coefficient_derivatives(self._h, c.data_ptr(), jc_edge.data_ptr() if self.E else None,
                                                         jc_self.data_ptr(), _stream()))
        return c, jc_edge, jc_self

    def compute_averaged(self, mode, out=None):
        """Density-averaged descriptor (n_features,): mode "outer" (mean power
        spectrum) or "inner" (power spectrum of the mean coefficients)."""
        code = {"inner": SOAP_AVERAGE_INNER, "outer": SOAP_AVERAGE_OUTER}.get(mode)
        if code is None:
            raise ValueError("mode must be 'inner' or 'outer'")
        desc = self._out(out, (self.n_features,))
        self._check(self._L.soap_compute_averaged(self._h, code, desc.data_ptr(), _stream()))
        return desc

    def derivatives(self, desc=None, jac_edge=None, jac_self=None):
        desc = self._out(desc, (self.n_centers, self.n_features))
        jac_edge = self._out(jac_edge, (self.E, 3, self.n_edge_features))
        jac_self = self._out(jac_self, (self.n_centers, 3, self.n_features))
        self._check(self._L.soap_derivatives(self._h, desc.data_ptr(), jac_edge.data_ptr() if self.E else None,
                                             jac_self.data_ptr(), _stream()))
        return desc, jac_edge, jac_self

    # -- center batches ---------------------------------------------------------
    def plan_batches(self, budget_bytes: int, jacobian: bool = True):
        """Consecutive center batches whose outputs (and, with the Jacobian,
        the library's scratch) fit budget_bytes: (center_first, edge_first),
        each of length B + 1."""
        import numpy as np
        if self.E is None:
            raise SoapError(SOAP_ESTATE, "no neighbour list: call build_neighbors first")
        what = SOAP_BATCH_DERIVATIVES if jacobian else SOAP_BATCH_DESCRIPTOR
        nb = ctypes.c_int64()
        self._check(self._L.soap_plan_batches(self._h, what, int(budget_bytes), 0, None, None, ctypes.byref(nb)))
        cf = np.empty(nb.value + 1, dtype=np.int64)
        ef = np.empty(nb.value + 1, dtype=np.int64)
        self._check(self._L.soap_plan_batches(self._h, what, int(budget_bytes), nb.value, cf.ctypes.data,
                                              ef.ctypes.data, ctypes.byref(nb)))
        return cf, ef

    def compute_batch(self, first: int, count: int, out=None):
        desc = self._out(out, (count, self.n_features))
        self._check(self._L.soap_compute_batch(self._h, int(first), int(count), desc.data_ptr(), _stream()))
        return desc

    def derivatives_batch(self, first: int, count: int, n_edges: int, desc=None, jac_edge=None, jac_self=None):
        """Descriptor and Jacobian of centers [first, first + count); n_edges =
        the edges of their rows (edge_first[k + 1] - edge_first[k])."""
        desc = self._out(desc, (count, self.n_features))
        jac_edge = self._out(jac_edge, (n_edges, 3, self.n_edge_features))
        jac_self = self._out(jac_self, (count, 3, self.n_features))
        self._check(self._L.soap_derivatives_batch(self._h, int(first), int(count), desc.data_ptr(),
                                                   jac_edge.data_ptr() if n_edges else None, jac_self.data_ptr(),
                                                   _stream()))
        return desc, jac_edge, jac_self

    def scatter_dense(self, jac_edge, jac_self, out=None):
        dense = self._out(out, (self.n_centers, self.n_atoms, 3, self.n_features))
        self._check(self._L.soap_scatter_dense(self._h, jac_edge.data_ptr() if self.E else None,
                                               jac_self.data_ptr(), dense.data_ptr(), _stream()))
        return dense
