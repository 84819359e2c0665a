"""SOAP oracle: plain, slow, float64 CPU reference of the descriptor and its
analytic Jacobian, written from the paper's equations (Secs. 2.1-2.3, 3.1).

TEST INFRASTRUCTURE ONLY.  Only tests/, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of bench.py may import this package.  It shares no code
with the HIP path: its constants come from 50-digit mpmath (constants.py) and
its arithmetic from soap_oracle.c.

Output conventions (so results can be compared with any implementation):
* features: species pairs mu <= nu over the species sorted by Z, then n, then
  n' (n' >= n when mu == nu), then l innermost;
* descriptor: (n_centers, F);
* Jacobian: for each center i, blocks for every neighbour j (|r_ij| < r_cut,
  j != i) and for i itself, in ascending atom index; block = d p_i / d r_j,
  shape (3, F).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import constants

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "soap_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")


def build(force: bool = False) -> str:
    """Compile the oracle (gcc, OpenMP, no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-std=gnu11", "-fopenmp", "-ffp-contract=off",
                               "-o", tmp, _SRC, "-lquadmath", "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Params(ctypes.Structure):
    _fields_ = [("S", ctypes.c_int32), ("n", ctypes.c_int32), ("lmax", ctypes.c_int32), ("rbf", ctypes.c_int32),
                ("rc", ctypes.c_double), ("sigma", ctypes.c_double),
                ("alpha_hi", ctypes.c_void_p), ("alpha_lo", ctypes.c_void_p),
                ("beta_hi", ctypes.c_void_p), ("beta_lo", ctypes.c_void_p),
                ("Q", ctypes.c_int32),
                ("G_hi", ctypes.c_void_p), ("G_lo", ctypes.c_void_p),
                ("rq_hi", ctypes.c_void_p), ("rq_lo", ctypes.c_void_p),
                ("sh_lmax", ctypes.c_int32),
                ("sh_ptr", ctypes.c_void_p), ("sh_exp", ctypes.c_void_p),
                ("sh_c_hi", ctypes.c_void_p), ("sh_c_lo", ctypes.c_void_p),
                ("wn_hi", ctypes.c_void_p), ("wn_lo", ctypes.c_void_p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        path = _LIB if os.path.exists(_LIB) else build()
        L = ctypes.CDLL(path)
        vp, i64, i32, dbl = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double
        L.oracle_neighbors.restype = i64
        L.oracle_neighbors.argtypes = [i64, vp, dbl, vp, i64, vp, vp, i64]
        L.oracle_neighbors_periodic.restype = i64
        L.oracle_neighbors_periodic.argtypes = [i64, vp, dbl, vp, vp, ctypes.c_int, vp, i64, vp, vp, vp, i64]
        L.oracle_neighbors_grid.restype = i64
        L.oracle_neighbors_grid.argtypes = [i64, vp, dbl, vp, vp, i64]
        L.oracle_solid_harmonics.restype = None
        L.oracle_solid_harmonics.argtypes = [vp, ctypes.c_int, vp, vp, vp]
        L.oracle_bessel_il.restype = None
        L.oracle_bessel_il.argtypes = [ctypes.c_int, dbl, vp]
        L.oracle_radial.restype = None
        L.oracle_radial.argtypes = [vp, dbl, vp, vp, vp]
        L.oracle_num_features.restype = i64
        L.oracle_num_features.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
        L.oracle_soap.restype = ctypes.c_int
        L.oracle_soap.argtypes = [vp, i64, vp, vp, vp, i64, vp, vp, vp, vp, ctypes.c_int, vp, vp, vp, vp]
        L.oracle_threads.restype = ctypes.c_int
        L.oracle_threads.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


def threads(n: int = 0) -> int:
    """Worker threads of the per-center loop (OpenMP): n > 0 sets them;
    returns the count the next compute() uses."""
    return int(lib().oracle_threads(int(n)))


def _ptr(a):
    return None if a is None else a.ctypes.data


def bessel_il(l_max: int, x: float) -> np.ndarray:
    """Modified spherical Bessel functions i_l(x), l = 0..l_max (unscaled)."""
    out = np.empty(l_max + 1)
    lib().oracle_bessel_il(l_max, float(x), out.ctypes.data)
    return out


def neighbors(pos64: np.ndarray, r_cut: float, centers=None):
    """All-pairs neighbour rows (ascending j) for the given centers."""
    pos64 = np.ascontiguousarray(pos64, dtype=np.float64)
    n = pos64.shape[0]
    cen = None if centers is None else np.ascontiguousarray(centers, dtype=np.int64)
    nc = n if cen is None else len(cen)
    row = np.zeros(nc + 1, dtype=np.int64)
    E = lib().oracle_neighbors(n, _ptr(pos64), r_cut, _ptr(cen), nc, _ptr(row), None, 0)
    cols = np.empty(max(E, 1), dtype=np.int32)
    lib().oracle_neighbors(n, _ptr(pos64), r_cut, _ptr(cen), nc, _ptr(row), _ptr(cols), E)
    return row, cols[:E]


def image_bounds(pos64, r_cut, cell, pbc):
    """Largest image index per direction that can reach the cutoff: the
    interplanar spacing d_k = V / |b x c| (and cyclic) bounds how far an image
    moves along each reciprocal direction; the spread of the fractional
    coordinates adds to it."""
    cell = np.asarray(cell, dtype=np.float64).reshape(3, 3)
    frac = np.asarray(pos64, dtype=np.float64) @ np.linalg.inv(cell)
    vol = abs(np.linalg.det(cell))
    out = np.zeros(3, dtype=np.int32)
    for k in range(3):
        if pbc[k]:
            cr = np.cross(cell[(k + 1) % 3], cell[(k + 2) % 3])
            d = vol / np.linalg.norm(cr)
            spread = frac[:, k].max() - frac[:, k].min() if len(frac) else 0.0
            out[k] = int(np.ceil(r_cut / d + spread)) + 1
    return out


def neighbors_periodic(pos64, r_cut, cell, pbc, centers=None, f32=True):
    """Brute-force periodic neighbour rows: (row, cols, img) with img[e] the
    integer image (n_a, n_b, n_c) of atom cols[e]; ascending j, then n."""
    pos64 = np.ascontiguousarray(pos64, dtype=np.float64)
    cellv = np.ascontiguousarray(np.asarray(cell, dtype=np.float64).reshape(9))
    nimg = np.ascontiguousarray(image_bounds(pos64, r_cut, cell, pbc))
    n = pos64.shape[0]
    cen = None if centers is None else np.ascontiguousarray(centers, dtype=np.int64)
    nc = n if cen is None else len(cen)
    row = np.zeros(nc + 1, dtype=np.int64)
    args = (n, _ptr(pos64), r_cut, _ptr(cellv), _ptr(nimg), 1 if f32 else 0, _ptr(cen), nc, _ptr(row))
    E = lib().oracle_neighbors_periodic(*args, None, None, 0)
    cols = np.empty(max(E, 1), dtype=np.int32)
    img = np.empty((max(E, 1), 3), dtype=np.int32)
    lib().oracle_neighbors_periodic(*args, _ptr(cols), _ptr(img), E)
    return row, cols[:E], img[:E]


def image_position(pos64, cell, j, n, f32=True):
    """r_j + ((n_a a + n_b b) + n_c c), float64, rounded to float32 if f32."""
    cell = np.asarray(cell, dtype=np.float64).reshape(3, 3)
    s = float(n[0]) * cell[0] + float(n[1]) * cell[1]
    s = s + float(n[2]) * cell[2]
    v = np.asarray(pos64[j], dtype=np.float64) + s
    return v.astype(np.float32).astype(np.float64) if f32 else v


def neighbors_grid(pos64: np.ndarray, r_cut: float):
    """Uniform-grid neighbour rows for every atom (ascending j)."""
    pos64 = np.ascontiguousarray(pos64, dtype=np.float64)
    n = pos64.shape[0]
    row = np.zeros(n + 1, dtype=np.int64)
    E = lib().oracle_neighbors_grid(n, _ptr(pos64), r_cut, _ptr(row), None, 0)
    cols = np.empty(max(E, 1), dtype=np.int32)
    lib().oracle_neighbors_grid(n, _ptr(pos64), r_cut, _ptr(row), _ptr(cols), E)
    return row, cols[:E]


class OracleSOAP:
    """Reference SOAP for species (list of Z), r_cut, n_max, l_max, sigma, rbf."""

    def __init__(self, species, r_cut: float, n_max: int, l_max: int, sigma: float, rbf: str = "gto",
                 quad_n: int = 64):
        if rbf not in ("gto", "polynomial", "polynomial-laplace"):
            raise ValueError("rbf must be 'gto', 'polynomial' or 'polynomial-laplace'")
        if n_max < 1 or l_max < 0 or sigma <= 0:
            raise ValueError("bad basis size or sigma")
        if rbf == "gto" and r_cut <= 1.0:
            raise ValueError("GTO basis needs r_cut > 1 A")
        self.species = sorted(int(z) for z in species)
        self.S = len(self.species)
        self.r_cut, self.n_max, self.l_max, self.sigma, self.rbf, self.quad_n = \
            float(r_cut), int(n_max), int(l_max), float(sigma), rbf, int(quad_n)
        self._keep = []
        p = _Params()
        p.S, p.n, p.lmax, p.rbf = self.S, self.n_max, self.l_max, {"gto": 0, "polynomial": 1}.get(rbf, 2)
        p.rc, p.sigma = self.r_cut, self.sigma
        if rbf == "gto":
            g = constants.gto_arrays(self.r_cut, self.n_max, self.l_max)
            for k in ("alpha_hi", "alpha_lo", "beta_hi", "beta_lo"):
                setattr(p, k, self._hold(g[k]))
        else:
            g = constants.poly_arrays(self.r_cut, self.n_max, self.quad_n)
            p.Q = self.quad_n
            for k in ("G_hi", "G_lo", "rq_hi", "rq_lo"):
                setattr(p, k, self._hold(g[k]))
            if rbf == "polynomial-laplace":
                wl = constants.poly_laplace_arrays(self.r_cut, self.n_max)
                for k in ("wn_hi", "wn_lo"):
                    setattr(p, k, self._hold(wl[k]))
        sh = constants.solid_harmonic_arrays(self.l_max + 1)
        p.sh_lmax = self.l_max + 1
        for k in ("sh_ptr", "sh_exp", "sh_c_hi", "sh_c_lo"):
            setattr(p, k, self._hold(sh[k]))
        self._p = p
        self.n_features = int(lib().oracle_num_features(self.S, self.n_max, self.l_max))

    def _hold(self, a):
        a = np.ascontiguousarray(a)
        self._keep.append(a)
        return a.ctypes.data

    def features(self):
        """List of (mu, nu, n, n', l) in output order."""
        out = []
        for mu in range(self.S):
            for nu in range(mu, self.S):
                for a in range(self.n_max):
                    for b in range(a if mu == nu else 0, self.n_max):
                        for l in range(self.l_max + 1):
                            out.append((mu, nu, a, b, l))
        return out

    def species_index(self, Z):
        lut = {z: k for k, z in enumerate(self.species)}
        try:
            return np.array([lut[int(z)] for z in Z], dtype=np.int32)
        except KeyError as e:
            raise ValueError("atomic number %s not in species list" % e) from None

    def solid_harmonics(self, v, l_max=None):
        lm = self.l_max + 1 if l_max is None else l_max
        L = (lm + 1) ** 2
        Y = np.empty(L)
        G = np.empty(3 * L)
        v = np.ascontiguousarray(v, dtype=np.float64)
        lib().oracle_solid_harmonics(ctypes.byref(self._p), lm, v.ctypes.data, Y.ctypes.data, G.ctypes.data)
        return Y, G.reshape(3, L)

    def radial(self, r: float):
        """Radial parts at distance r: (R[n][l], dR/dr[n][l], on-site c0[n]).
        GTO: c_nlm = R r^l Y_lm; polynomial: c_nlm = R Y_lm (R = f_nl)."""
        R = np.empty((self.n_max, self.l_max + 1))
        dR = np.empty_like(R)
        c0 = np.empty(self.n_max)
        lib().oracle_radial(ctypes.byref(self._p), float(r), R.ctypes.data, dR.ctypes.data, c0.ctypes.data)
        return R, dR, c0

    def compute(self, pos64, Z, centers=None, jacobian=False, coefficients=False, nb=None,
                coefficient_jacobian=False):
        """Descriptor (and Jacobian blocks, coefficients) for the given centers.

        Returns a dict with desc (nc, F); if jacobian: blk_ptr (nc+1), blk_j,
        jac (nblocks, 3, F); if coefficients: c (nc, S, n_max, (l_max+1)^2);
        if coefficient_jacobian: dc (E, 3, n_max, (l_max+1)^2), for the e-th
        neighbour edge (i, j) of the rows, d c^{species(j)}(i) / d r_j (Eqs.
        gto-derivative, poly-cartesian-derivative; the other species blocks
        of c do not depend on r_j), and dc_self (nc, 3, S, n_max, L) =
        d c(i) / d r_i = - sum_j of the edge blocks (translational
        invariance); always: row_ptr, cols (the neighbour rows used)."""
        pos64 = np.ascontiguousarray(pos64, dtype=np.float64)
        spec = self.species_index(Z)
        n = pos64.shape[0]
        cen = None if centers is None else np.ascontiguousarray(centers, dtype=np.int64)
        nc = n if cen is None else len(cen)
        row, cols = neighbors(pos64, self.r_cut, cen) if nb is None else nb
        F = self.n_features
        L = (self.l_max + 1) ** 2
        desc = np.empty((nc, F))
        cout = np.empty((nc, self.S, self.n_max, L)) if coefficients else None
        out = dict(desc=desc, row_ptr=row, cols=cols)
        blk_ptr = blk_j = jac = None
        dcout = np.empty((int(row[-1]), 3, self.n_max, L)) if coefficient_jacobian else None
        if jacobian:
            deg = np.diff(row)
            blk_ptr = np.zeros(nc + 1, dtype=np.int64)
            blk_ptr[1:] = np.cumsum(deg + 1)
            nblk = int(blk_ptr[-1])
            blk_j = np.empty(nblk, dtype=np.int32)
            jac = np.empty((nblk, 3, F))
            out.update(blk_ptr=blk_ptr, blk_j=blk_j, jac=jac)
        rc = lib().oracle_soap(ctypes.byref(self._p), n, _ptr(pos64), _ptr(spec), _ptr(cen), nc, _ptr(row),
                               _ptr(cols), _ptr(desc), _ptr(cout), 1 if jacobian else 0, _ptr(blk_ptr),
                               _ptr(blk_j), _ptr(jac), _ptr(dcout))
        if rc != 0:
            raise MemoryError("oracle allocation failed")
        if coefficients:
            out["c"] = cout
        if coefficient_jacobian:
            out["dc"] = dcout
            spec_j = spec[cols]
            dself = np.zeros((nc, 3, self.S, self.n_max, L))
            for c in range(nc):
                for e in range(int(row[c]), int(row[c + 1])):
                    dself[c, :, spec_j[e]] -= dcout[e]
            out["dc_self"] = dself
        return out

    def compute_periodic(self, pos64, Z, cell, pbc, centers=None, f32=True, **kw):
        """compute() for a periodic structure: every neighbour image becomes an
        atom of an extended structure (the home atoms, then one entry per edge
        at its image position), whose neighbour rows are the periodic rows.
        Returns compute()'s dict plus img_atom / img_shift, the atom and image
        of every extended index (home atoms: their own index, image 0)."""
        pos64 = np.asarray(pos64, dtype=np.float64)
        n = pos64.shape[0]
        row, cols, img = neighbors_periodic(pos64, self.r_cut, cell, pbc, centers, f32)
        E = len(cols)
        ext = np.concatenate([pos64, np.array([image_position(pos64, cell, int(j), m, f32)
                                               for j, m in zip(cols, img)]).reshape(E, 3)])
        Zx = np.concatenate([np.asarray(Z), np.asarray(Z)[cols]])
        out = self.compute(ext, Zx, centers=np.arange(n) if centers is None else centers,
                           nb=(row, np.arange(n, n + E, dtype=np.int32)), **kw)
        out["img_atom"] = np.concatenate([np.arange(n), cols]).astype(np.int64)
        out["img_shift"] = np.concatenate([np.zeros((n, 3), dtype=np.int32), img])
        return out

    def power_spectrum(self, c):
        """Eq. (powerspectrum) of one coefficient set c (S, n_max, L), in the
        output feature order: pi sqrt(8/(2l+1)) sum_m c^mu_nlm c^nu_n'lm."""
        out = []
        for mu, nu, a, b, l in self.features():
            m = slice(l * l, (l + 1) * (l + 1))
            out.append(np.pi * np.sqrt(8.0 / (2 * l + 1)) * float(np.dot(c[mu, a, m], c[nu, b, m])))
        return np.array(out)

    def averaged(self, pos64, Z, mode, centers=None):
        """The density-averaged descriptors of the paper's averaging modes:
        "outer" = mean over the centers of the power spectrum, "inner" = the
        power spectrum of the mean over the centers of the coefficients."""
        r = self.compute(pos64, Z, centers=centers, coefficients=True)
        if mode == "outer":
            return r["desc"].mean(axis=0)
        if mode == "inner":
            return self.power_spectrum(r["c"].mean(axis=0))
        raise ValueError("mode must be 'inner' or 'outer'")
