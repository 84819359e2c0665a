"""Seeded synthetic structures for the SOAP descriptor + Jacobian workloads.

Input generation only (no SOAP arithmetic).  The HIP path and the CPU oracle
both consume exactly these arrays: positions are generated in float64, rounded
once to float32, and that float32 array (or its exact float64 upcast) is what
every consumer sees.

The workloads stand in for the water clusters (H2O)_n of the paper's results
section (Sec. 4: GTO basis, average "off"), whose construction the paper does
not describe, plus a four-species condensed phase:

* water clusters: liquid density 0.0334 molecules/A^3, O-O >= 2.6 A, rigid
  molecules (O-H 0.9572 A, H-O-H 104.52 deg) in uniform random orientations;
* a CHNO sphere: 4096 atoms, Z = 1, 6, 7, 8 in ratio 4:2:1:1, uniform in a
  35 A ball with minimum pair distance 0.9 A.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "csrc", "workloads.c")
_LIB = os.path.join(_HERE, "libsoapgen.so")

WATER_DENSITY = 0.0334  # molecules per A^3
OO_MIN = 2.6            # A


def build_generator(force: bool = False) -> str:
    """Compile the generator shared library (plain C, host only)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-std=gnu11", "-ffp-contract=off",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _gen():
    global _lib
    if _lib is None:
        path = _LIB if os.path.exists(_LIB) else build_generator()
        lib = ctypes.CDLL(path)
        lib.soapgen_water.restype = ctypes.c_int64
        lib.soapgen_water.argtypes = [ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_double,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)]
        lib.soapgen_multispecies.restype = ctypes.c_int64
        lib.soapgen_multispecies.argtypes = [ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_double,
                                             ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                             ctypes.c_void_p, ctypes.c_void_p]
        lib.soapgen_splitmix_stream.restype = None
        lib.soapgen_splitmix_stream.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p]
        _lib = lib
    return _lib


def splitmix_stream(seed: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.uint64)
    _gen().soapgen_splitmix_stream(seed, n, out.ctypes.data)
    return out


@dataclass
class Structure:
    pos: np.ndarray          # (N, 3) float32: the only positions any consumer sees
    Z: np.ndarray            # (N,) int32
    radius: float            # radius of the generating ball, A
    draws: int               # rejection-sampling draws used
    recipe: dict = field(default_factory=dict)

    @property
    def n_atoms(self) -> int:
        return int(self.pos.shape[0])

    @property
    def pos64(self) -> np.ndarray:
        """Exact float64 upcast of the float32 positions."""
        return self.pos.astype(np.float64)


def water_cluster(n_mol: int, seed: int) -> Structure:
    pos = np.empty((3 * n_mol, 3), dtype=np.float64)
    Z = np.empty(3 * n_mol, dtype=np.int32)
    R = ctypes.c_double(0.0)
    draws = _gen().soapgen_water(n_mol, seed, WATER_DENSITY, OO_MIN, pos.ctypes.data, Z.ctypes.data,
                                 ctypes.byref(R))
    if draws < 0:
        raise RuntimeError("water generator failed")
    return Structure(pos.astype(np.float32), Z, R.value, int(draws),
                     dict(kind="water", n_mol=n_mol, seed=seed, density=WATER_DENSITY, oo_min=OO_MIN))


def multispecies_sphere(n: int, seed: int, radius: float, dmin: float, composition: dict) -> Structure:
    zl = np.array(sorted(composition), dtype=np.int32)
    zc = np.array([composition[z] for z in sorted(composition)], dtype=np.int64)
    pos = np.empty((n, 3), dtype=np.float64)
    Z = np.empty(n, dtype=np.int32)
    draws = _gen().soapgen_multispecies(n, seed, radius, dmin, zl.ctypes.data, zc.ctypes.data, len(zl),
                                        pos.ctypes.data, Z.ctypes.data)
    if draws < 0:
        raise RuntimeError("multi-species generator failed")
    return Structure(pos.astype(np.float32), Z, radius, int(draws),
                     dict(kind="multispecies", n=n, seed=seed, radius=radius, dmin=dmin,
                          composition=dict(composition)))


def random_small(n: int, seed: int, box: float, species=(1, 8), dmin: float = 0.7) -> Structure:
    """Tiny random structures for fuzzing: n atoms in a ball sized from `box`."""
    comp = {}
    for k in range(n):
        z = species[k % len(species)]
        comp[z] = comp.get(z, 0) + 1
    return multispecies_sphere(n, seed, box, dmin, comp)


# --- the five workloads ------------------------------------------------------

@dataclass(frozen=True)
class Workload:
    name: str
    species: tuple
    rbf: str
    r_cut: float
    sigma: float
    n_max: int
    l_max: int
    jacobian: bool
    make: tuple  # ("water", n_mol, seed) or ("multi", n, seed, R, dmin, composition-tuple)

    def structure(self) -> Structure:
        if self.make[0] == "water":
            return water_cluster(self.make[1], self.make[2])
        _, n, seed, R, dmin, comp = self.make
        return multispecies_sphere(n, seed, R, dmin, dict(comp))

    def with_basis(self, n_max: int, l_max: int, rbf: str | None = None) -> "Workload":
        rbf = rbf or self.rbf
        return Workload(f"{self.name.split('_')[0]}_{rbf}_n{n_max}l{l_max}", self.species, rbf,
                        self.r_cut, self.sigma, n_max, l_max, self.jacobian, self.make)


WATER64 = Workload("water64_gto_n4l4", (1, 8), "gto", 5.0, 0.5, 4, 4, True, ("water", 64, 0))
WATER1000 = Workload("water1000_gto_n8l6", (1, 8), "gto", 6.0, 0.5, 8, 6, True, ("water", 1000, 1))
CHNO4096 = Workload("chno4096_poly_n10l10", (1, 6, 7, 8), "polynomial", 5.0, 0.4, 10, 10, True,
                    ("multi", 4096, 3, 35.0, 0.9, ((1, 2048), (6, 1024), (7, 512), (8, 512))))
WATER1M = Workload("water333334_gto_n8l6_desc", (1, 8), "gto", 5.0, 0.5, 8, 6, False, ("water", 333334, 4))

GRID_NL = (2, 4, 6, 8, 10, 12)


def hyperparameter_grid():
    """The 3000-atom water cluster over n_max, l_max in {2..12}^2: GTO, and the
    polynomial basis in its quadrature and Laplace forms."""
    out = []
    for rbf in ("gto", "polynomial", "polynomial-laplace"):
        for n in GRID_NL:
            for l in GRID_NL:
                out.append(WATER1000.with_basis(n, l, rbf))
    return out


WORKLOADS = {0: WATER64, 1: WATER1000, 3: CHNO4096, 4: WATER1M}
