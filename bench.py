"""Benchmark of the SOAP descriptor + analytic Jacobian hot path on one MI355X.

One step = one pass of the whole path over the structure: neighbour search
(soap_build_neighbors), then descriptor + Jacobian (soap_derivatives), or the
descriptor alone (soap_compute) for descriptor-only workloads.  Inputs are
resident in HBM before the timed region; output buffers are allocated once.

Default workload: the 3000-atom water cluster (1000 H2O), GTO basis,
r_cut 6 A, sigma 0.5 A, n_max 8, l_max 6, descriptor + Jacobian, float32
outputs.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--dtype float32|float64] [--arith mixed|fp64]
                  [--mode derivatives|cc|inner|outer] [--periodic] [--grid OUT.jsonl] [--no-cpu-baseline]

Without --workload the line also carries, under "configs", the same headline
with float64 internal arithmetic, the 64-water cluster (GTO n4 l4), the CHNO
condensed phase (polynomial n10 l10) and the 1,000,002-atom water descriptor
(GTO n8 l6), each with its ms/step, atoms/s, kernel and step roofline
fractions and (unless --no-cpu-baseline) the oracle's baseline.

--mode picks the output of a Jacobian workload: the descriptor + Jacobian
(default), the coefficients and their Jacobian ("cc"), or one averaged
descriptor row ("inner", "outer").  --periodic puts the structure in an
orthorhombic periodic cell 1.6 A wider than its extent (images across the
faces become neighbours).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SOAP atoms/s (desc+Jacobian), 3000-atom water, per (n_max,l_max); % roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP64_PEAK_TFLOPS = 78.6        # MI355X FP64 vector


def workload_by_name(name):
    from paper_2609_05709_amd import workloads as w
    table = {"water64": w.WATER64, "water1000": w.WATER1000, "chno4096": w.CHNO4096, "water1m": w.WATER1M}
    if name in table:
        return table[name]
    # water1000_<rbf>_n<N>l<L>, e.g. water1000_polynomial_n12l12
    parts = name.split("_")
    if parts[0] == "water1000" and len(parts) == 3:
        nl = parts[2]
        n, l = nl[1:].split("l")
        return w.WATER1000.with_basis(int(n), int(l), parts[1])
    raise SystemExit(f"unknown workload {name}")


def algorithmic(wl, st_n, E, F, Fe, out_bytes, jac):
    """Algorithmic HBM bytes per step and per kernel launch: the outputs the
    method must write (descriptor rows, the center blocks and the neighbour
    blocks restricted to the species pairs that can be non-zero)."""
    desc = st_n * F * out_bytes
    self_blocks = st_n * 3 * F * out_bytes if jac else 0
    edge_blocks = E * 3 * Fe * out_bytes if jac else 0
    return dict(step=desc + self_blocks + edge_blocks, density=desc + self_blocks, jacobian=edge_blocks)


def density_flops(wl, E, n_centers, F):
    """Algorithmic float64 operations of the descriptor-only density kernel
    (GTO), per step: per edge, the real solid harmonics (about 3 flops per
    (l, m)), the radial factors B_nl = sum_k beta C exp(-a' r^2) (2 n^2 (l+1)
    flops plus n (l+1) exponentials, each counted as 1), and the projection
    c += B Y (2 n L flops); per center, the power spectrum (2 (2l+1) flops per
    feature)."""
    n, l = wl.n_max, wl.l_max
    L = (l + 1) ** 2
    per_edge = 3 * L + 2 * n * n * (l + 1) + n * (l + 1) + 2 * n * L
    per_center = sum(2 * (2 * ll + 1) for ll in range(l + 1)) * (F // (l + 1))
    return E * per_edge + n_centers * per_center


def step_work(wl, nc, E, F, Fe, out_bytes, jac, quad_n=64):
    """Algorithmic work of one step (the method's own work, no structural
    zeros): float64-equivalent operations and HBM bytes.  Per edge: real
    solid harmonics (~3 flops per (l, m); ~12 with gradients), the radial
    factors (GTO: 2 n^2 (l+1) flops per factor and n (l+1) exponentials;
    polynomial quadrature: 2 n Q (l+1) per factor and Q (l+2) Bessel values
    plus 2 Q exponentials; Laplace form: 8 n (n+3) Clenshaw flops and ~10 per
    (n, l)), the projection 2 n L; with the Jacobian the radial factor's
    derivative (the radial flops again), the precontraction 8 S n L, the
    assembly 12 (F_e + F_ss) and the center block 3 F_e.  Per center: the
    power spectrum, 2 (2l+1) flops per feature.  Bytes: the outputs."""
    n, l, S = wl.n_max, wl.l_max, len(wl.species)
    L = (l + 1) ** 2
    if wl.rbf == "gto":
        radial = 2 * n * n * (l + 1) + n * (l + 1)
    elif wl.rbf == "polynomial":
        radial = 2 * n * quad_n * (l + 1) + quad_n * (l + 2) + 2 * quad_n
    else:
        radial = 8 * n * (n + 3) + 10 * n * (l + 1)
    if jac:
        F_ss = (l + 1) * n * (n + 1) // 2
        per_edge = 12 * L + 2 * radial + 2 * n * L + 8 * S * n * L + 12 * (Fe + F_ss) + 3 * Fe
    else:
        per_edge = 3 * L + radial + 2 * n * L
    per_center = sum(2 * (2 * ll + 1) for ll in range(l + 1)) * (F // (l + 1))
    flops = E * per_edge + nc * per_center
    nbytes = (nc * F + (3 * nc * F + 3 * E * Fe if jac else 0)) * out_bytes
    return flops, nbytes


def step_roofline(flops, nbytes, ms_step):
    """The binding roofline of the whole step: floor = max(bytes / HBM peak,
    flops / FP64 peak); frac = floor / measured step time."""
    t_hbm = nbytes / (HBM_PEAK_GBS * 1e9)
    t_alu = flops / (FP64_PEAK_TFLOPS * 1e12)
    floor = max(t_hbm, t_alu)
    return {"bound": "hbm" if t_hbm >= t_alu else "alu", "floor_ms": floor * 1e3, "alg_flops": flops,
            "alg_bytes": nbytes, "frac": floor / (ms_step * 1e-3)}


def measured_traffic(workload_name, kernel, output):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    runs (FETCH_SIZE, WRITE_SIZE, each scaled by the reading of a plain copy of
    known size), or None if absent, taken at another output precision or on
    different kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        doc = json.load(open(path))[workload_name]
        sha = kernels_source_sha()
        if doc["kernels_source_sha256_16"] != sha or doc["output"] != output:
            return None
        k = doc["per_launch"][kernel]
        return k["fetch_bytes"] + k["write_bytes"]
    except (OSError, KeyError, ValueError):
        return None


KERNEL_SOURCES = ("soap_device.h", "soap_kernels.hip", "density_streamed.hip", "jacobian_fixed.hip", "soap_internal.h")


def kernels_source_sha():
    """sha256 (16 hex digits) of the descriptor kernels' sources: counter
    readings taken on other sources do not describe these kernels."""
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2609_05709_amd", "csrc", name), "rb").read())
    return h.hexdigest()[:16]


def copy_calibration():
    """A plain device copy of 1 GiB, three times: the reference reading for
    scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    n = 256 * 1024 * 1024
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "repeats": 3}))


def _oracle_rate(o, wl, st, budget_s):
    """Centers per second of the oracle over seeded random batches of 128
    centers until ~budget_s of wall time; (rate, centers done, seconds)."""
    rng = np.random.default_rng(12345)
    order = rng.permutation(st.n_atoms)
    done, t0 = 0, time.perf_counter()
    while done < st.n_atoms and time.perf_counter() - t0 < budget_s:
        batch = np.sort(order[done:done + 128])
        o.compute(st.pos64, st.Z, centers=batch, jacobian=wl.jacobian)
        done += len(batch)
    dt = time.perf_counter() - t0
    return done / dt, done, dt


def _cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


LARGE_SAMPLE = 20000  # centers timed for the oracle on structures above LARGE_ATOMS
LARGE_ATOMS = 100000


def _cpu_baseline_large(o, wl, st, threads):
    """Large structures: the oracle's uniform-grid neighbour search over all
    atoms (timed whole), then the descriptor of a seeded sample of centers
    on those rows, scaled linearly to every center (each center's work is
    independent given its row)."""
    import oracle
    t0 = time.perf_counter()
    row, cols = oracle.neighbors_grid(st.pos64, wl.r_cut)
    t_nb = time.perf_counter() - t0
    rng = np.random.default_rng(12345)
    idx = np.sort(rng.choice(st.n_atoms, size=min(LARGE_SAMPLE, st.n_atoms), replace=False))
    deg = row[idx + 1] - row[idx]
    rs = np.zeros(len(idx) + 1, dtype=np.int64)
    rs[1:] = np.cumsum(deg)
    cs = np.concatenate([cols[row[i]:row[i + 1]] for i in idx])
    t0 = time.perf_counter()
    o.compute(st.pos64, st.Z, centers=idx, nb=(rs, cs), jacobian=wl.jacobian)
    t_c = time.perf_counter() - t0
    total = t_nb + t_c * st.n_atoms / len(idx)
    return {"value": st.n_atoms / total, "unit": "atoms/s", "cores": threads, "kind": "oracle",
            "sample": f"uniform-grid neighbour search over all {st.n_atoms} atoms ({t_nb:.1f} s), then the "
                      f"{'descriptor + Jacobian' if wl.jacobian else 'descriptor'} of {len(idx)} seeded random "
                      f"centers ({t_c:.1f} s) scaled linearly to all centers: {total:.0f} s estimated; "
                      f"{threads} threads of {_cpu_model()} ({os.cpu_count()} logical CPUs)"}


def cpu_baseline(wl, st, budget_s=12.0, one_thread=False):
    """The oracle as it stands, on the host cores, over a bounded sample of
    centers; with one_thread, also a sample on a single thread."""
    import oracle
    o = oracle.OracleSOAP(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf)
    threads = oracle.threads()
    if st.n_atoms > LARGE_ATOMS:
        return _cpu_baseline_large(o, wl, st, threads)
    what = "descriptor + Jacobian" if wl.jacobian else "descriptor"
    rate, done, dt = _oracle_rate(o, wl, st, budget_s)
    out = {"value": rate, "unit": "atoms/s", "cores": threads, "kind": "oracle",
           "sample": f"{done} of {st.n_atoms} centers (seeded random), neighbour search + {what}, "
                     f"{dt:.1f} s on {threads} threads of {_cpu_model()} ({os.cpu_count()} logical CPUs)"}
    if one_thread:
        oracle.threads(1)
        try:
            rate1, done1, dt1 = _oracle_rate(o, wl, st, budget_s * 0.75)
        finally:
            oracle.threads(threads)
        out["one_thread"] = {"value": rate1, "unit": "atoms/s", "cores": 1,
                             "sample": f"{done1} of {st.n_atoms} centers, {dt1:.1f} s"}
    return out


def cc_bytes(sp, wl, nc, E, out_bytes):
    """Algorithmic bytes of the coefficient-Jacobian outputs: c, the edge
    gradients (neighbour's species block) and the center blocks."""
    nL = wl.n_max * (wl.l_max + 1) ** 2
    S = len(wl.species)
    return (nc * S * nL + E * 3 * nL + nc * 3 * S * nL) * out_bytes


# what the timed path computes in, per output precision and internal arithmetic
DTYPE_LABEL = {
    ("float32", "mixed"): "mixed: f64 geometry/radial sums/accumulation/MFMA, f32 staged operands and final assembly",
    ("float32", "fp64"): "f64 (outputs rounded to f32)",
    ("float64", "mixed"): "f64",
    ("float64", "fp64"): "f64",
}


def run(wl, steps, warmup, dtype, with_cpu=True, quiet=False, mode="derivatives", periodic=False, arith="mixed",
        cpu_budget_s=12.0, desc_tile=0, pipeline=None, pipeline_density_wg=None, djac_tile=None, batches=0,
        options=()):
    import torch
    from paper_2609_05709_amd.soap import Soap
    st = wl.structure()
    tdt = torch.float64 if dtype == "float64" else torch.float32
    out_bytes = 8 if dtype == "float64" else 4
    dev = torch.device("cuda:0")
    sp = Soap(wl.species, wl.r_cut, wl.n_max, wl.l_max, wl.sigma, wl.rbf, dtype=dtype, arith=arith)
    if desc_tile:
        sp._check(sp._L.soap_set_option(sp._h, b"desc_tile", int(desc_tile)))
    if djac_tile is not None:
        sp._check(sp._L.soap_set_option(sp._h, b"djac_tile", int(djac_tile)))
    if pipeline is not None:
        sp._check(sp._L.soap_set_option(sp._h, b"pipeline", int(pipeline)))
    for key, value in options:
        sp._check(sp._L.soap_set_option(sp._h, key.encode(), int(value)))
    if pipeline_density_wg is not None:
        sp._check(sp._L.soap_set_option(sp._h, b"pipeline_density_wg", int(pipeline_density_wg)))
    if periodic:
        lo = st.pos.min(axis=0) - np.float32(0.8)
        st = type(st)((st.pos - lo).astype(np.float32), st.Z, st.radius, st.draws, dict(st.recipe, periodic=True))
        sp.set_cell(np.diag((st.pos.max(axis=0) + 0.8).astype(np.float64)), (1, 1, 1))
    pos = torch.from_numpy(st.pos.astype(np.float64) if dtype == "float64" else st.pos).to(dev, tdt)
    Z = torch.from_numpy(st.Z).to(dev)
    E = sp.build_neighbors(pos, Z)
    nc = st.n_atoms
    S, L = len(wl.species), (wl.l_max + 1) ** 2
    if mode == "cc":
        cc = torch.empty((nc, S, wl.n_max, L), dtype=tdt, device=dev)
        jce = torch.empty((E, 3, wl.n_max, L), dtype=tdt, device=dev)
        jcs = torch.empty((nc, 3, S, wl.n_max, L), dtype=tdt, device=dev)
    elif mode in ("inner", "outer"):
        avg = torch.empty(sp.n_features, dtype=tdt, device=dev)
    elif batches:
        # the structure streamed in batches sized by a memory budget: buffers
        # for the largest batch, reused by every batch
        per_center = sp.n_features * out_bytes * (4 if wl.jacobian else 1)
        total = nc * per_center + (E * 3 * sp.n_edge_features * out_bytes if wl.jacobian else 0)
        cf, ef = sp.plan_batches(total // batches + 1, jacobian=wl.jacobian)
        bmax, emax = int(np.diff(cf).max()), int(np.diff(ef).max())
        desc = torch.empty((bmax, sp.n_features), dtype=tdt, device=dev)
        if wl.jacobian:
            jedge = torch.empty((max(emax, 1), 3, sp.n_edge_features), dtype=tdt, device=dev)
            jself = torch.empty((bmax, 3, sp.n_features), dtype=tdt, device=dev)
    else:
        desc = torch.empty((nc, sp.n_features), dtype=tdt, device=dev)
        if wl.jacobian:
            jedge = torch.empty((E, 3, sp.n_edge_features), dtype=tdt, device=dev)
            jself = torch.empty((nc, 3, sp.n_features), dtype=tdt, device=dev)

    def step():
        sp.build_neighbors(pos, Z)
        if batches:
            for k in range(len(cf) - 1):
                a, n_c, n_e = int(cf[k]), int(cf[k + 1] - cf[k]), int(ef[k + 1] - ef[k])
                if wl.jacobian:
                    sp.derivatives_batch(a, n_c, n_e, desc[:n_c], jedge[:max(n_e, 1)] if n_e else jedge[:0],
                                         jself[:n_c])
                else:
                    sp.compute_batch(a, n_c, desc[:n_c])
        elif mode == "cc":
            sp.coefficient_derivatives(cc, jce, jcs)
        elif mode in ("inner", "outer"):
            sp.compute_averaged(mode, avg)
        elif wl.jacobian:
            sp.derivatives(desc, jedge, jself)
        else:
            sp.compute(desc)

    for _ in range(warmup):
        step()
    # timed region 1: the K steps, nothing but the path on the stream
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record()
    for _ in range(steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / steps
    # timed region 2: the same K steps with HIP events around each segment
    # (neighbours, density + outputs, Jacobian) on the library's stream; the
    # events cost about 30 us per step between kernels, so they stay out of
    # region 1
    sp.timing(reset=True)
    sp.set_timing(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    seg_ms, seg_n = sp.timing(reset=True)
    sp.set_timing(False)

    jac = wl.jacobian and mode == "derivatives"
    alg = algorithmic(wl, nc, E, sp.n_features, sp.n_edge_features, out_bytes, jac)
    # the kernels the library's plan chose for this basis
    desc_kernel = "k_desc" if sp.get_option("descriptor_kernel") else "k_density"
    dens_kernel = ("k_density", "k_djac", "k_djs")[int(sp.get_option("jacobian_density_kernel"))]
    # per step (a pipelined step launches its kernels once per center chunk;
    # the chunks' Jacobian launches then overlap the density launches)
    kern = {"neighbors": seg_ms[0] / steps, "density": seg_ms[1] / steps, "jacobian": seg_ms[2] / steps,
            "launches_per_step": {"neighbors": int(seg_n[0]) // steps, "density": int(seg_n[1]) // steps,
                                  "jacobian": int(seg_n[2]) // steps}}
    if mode == "cc":
        # the density kernel's gradient stores dominate: HBM-bound
        b = cc_bytes(sp, wl, nc, E, out_bytes)
        alg = dict(step=b, density=b, jacobian=0)
        t = kern["density"] * 1e-3
        roof = {"kernel": "k_density", "bound": "hbm", "achieved": b / t / 1e9, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "traffic": None, "alg_bytes_per_launch": b}
    elif jac:
        # the edge-block writes dominate: HBM-bound kernel
        t = kern["jacobian"] * 1e-3
        roof = {"kernel": "k_jacobian", "bound": "hbm", "achieved": alg["jacobian"] / t / 1e9, "peak": HBM_PEAK_GBS,
                "unit": "GB/s",
                # the counters were taken on the default (mixed-arithmetic) kernels
                "traffic": None if periodic or arith != "mixed" else measured_traffic(wl.name, "k_jacobian", dtype),
                "alg_bytes_per_launch": alg["jacobian"]}
    else:
        fl = density_flops(wl, E, nc, sp.n_features)
        t = kern["density"] * 1e-3
        roof = {"kernel": desc_kernel, "bound": "alu", "achieved": fl / t / 1e12, "peak": FP64_PEAK_TFLOPS,
                "unit": "TFLOP/s",
                "traffic": None if arith != "mixed" else measured_traffic(
                    wl.name + ("" if mode == "derivatives" else "_" + mode), desc_kernel, dtype),
                "alg_flops_per_launch": fl}
    roof["frac"] = roof["achieved"] / roof["peak"]
    line = {
        "metric": METRIC,
        "value": nc * steps / (ms_total * 1e-3),
        "unit": "atoms/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE_LABEL[(dtype, arith)],
        "data": "synthetic",
        "config": {"workload": wl.name + ("" if mode == "derivatives" else "_" + mode) + ("_periodic" if periodic else "")
                   + (f"_batches{len(cf) - 1}" if batches else ""),
                   "n_atoms": nc, "edges": E, "rbf": wl.rbf, "n_max": wl.n_max,
                   "l_max": wl.l_max, "r_cut": wl.r_cut, "sigma": wl.sigma, "species": list(wl.species),
                   "output": dtype, "arith": arith, "jacobian": jac or mode == "cc", "mode": mode,
                   "features": sp.n_features,
                   "edge_features": sp.n_edge_features},
        "kernel_ms": kern,
        "kernels": {"descriptor": desc_kernel, "jacobian_density": dens_kernel},
        "plan": {k: sp.get_option(k) for k in ("jacobian_l_groups", "jacobian_density_tile", "jacobian_density_lds",
                                                "jacobian_tile", "jacobian_lds", "output_kernel_rows", "output_lds")},
        "kernel_timing": "HIP events per segment, on the stream each kernel runs on, over a second pass of the "
                         "K steps; per-step sums",
        "step_alg_bytes": alg["step"],
        "step_hbm_fraction": alg["step"] / (ms_step * 1e-3) / (HBM_PEAK_GBS * 1e9),
        "wall_s": wall,
        "roofline": roof,
    }
    if mode == "derivatives":
        fl, nb = step_work(wl, nc, E, sp.n_features, sp.n_edge_features, out_bytes, jac)
        line["step_roofline"] = step_roofline(fl, nb, ms_step)
    sp.close()
    if with_cpu and mode == "derivatives" and not periodic:
        line["cpu_baseline"] = cpu_baseline(wl, st, budget_s=cpu_budget_s, one_thread=wl.name in (
            workload_by_name("water64").name, workload_by_name("water1000").name))
    return line


# the other workloads of the default line: the 64-water cluster, the CHNO
# condensed phase (polynomial basis) and the million-atom water descriptor
EXTRA_WORKLOADS = ("water64", "chno4096", "water1m")


def summary(line):
    """The per-workload figures carried in the default line's "configs"."""
    keep = ("value", "unit", "ms_per_step", "dtype", "config", "kernel_ms", "roofline", "step_roofline",
            "cpu_baseline", "steps", "warmup")
    return {k: line[k] for k in keep if k in line}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None,
                    help="one workload only (default: the 3000-atom water headline, plus the other workloads and "
                         "the float64-arithmetic headline in the line's \"configs\")")
    ap.add_argument("--dtype", default="float32", choices=["float32", "float64"])
    ap.add_argument("--arith", default="mixed", choices=["mixed", "fp64"],
                    help="internal arithmetic of the float32 mode: float32 staging and assembly, or float64 throughout")
    ap.add_argument("--mode", default="derivatives", choices=["derivatives", "cc", "inner", "outer"])
    ap.add_argument("--periodic", action="store_true")
    ap.add_argument("--grid", default=None, help="sweep n_max, l_max in {2..12}^2 for every radial basis; write JSONL here")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--batches", type=int, default=0,
                    help="stream the structure through about this many center batches sized by a memory budget "
                         "(one neighbour search per step, outputs in buffers of the largest batch)")
    ap.add_argument("--pipeline", type=int, default=None, help="center chunks of a pipelined derivatives call")
    ap.add_argument("--pipeline-density-wg", type=int, default=None,
                    help="density workgroups per CU while pipelined (0 = as planned)")
    ap.add_argument("--djac-tile", type=int, default=None, choices=[0, -1, 32, 64],
                    help="Jacobian path's density step (GTO): 0 automatic, -1 the shared density kernel, else chunk")
    ap.add_argument("--desc-tile", type=int, default=0, choices=[0, -1, 16, 32, 64],
                    help="GTO descriptor kernel: 0 automatic, -1 the shared density kernel, else edges per chunk")
    ap.add_argument("--option", action="append", default=[], metavar="KEY=VALUE",
                    help="any soap_set_option tuning knob (e.g. out_rows=0, djs_tile=32); repeatable")
    ap.add_argument("--copy-calibration", action="store_true", help="run only a 1 GiB device copy (counter scaling)")
    a = ap.parse_args()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the SOAP path here is built and timed on a single MI355X "
              "(centers shard across GPUs without communication)", file=sys.stderr)
        sys.exit(2)
    if a.copy_calibration:
        copy_calibration()
        return
    if a.grid:
        from paper_2609_05709_amd import workloads as w
        with open(a.grid, "w") as f:
            for wl in w.hyperparameter_grid():
                line = run(wl, max(3, a.steps // 4), 2, a.dtype, with_cpu=False)
                f.write(json.dumps(line) + "\n")
                f.flush()
                print(f"{wl.name}: {line['value']:.4g} atoms/s, {line['ms_per_step']:.3f} ms, "
                      f"jac {line['roofline']['frac']:.3f} of HBM", flush=True)
        return
    wl = workload_by_name(a.workload or "water1000")
    line = run(wl, a.steps, a.warmup, a.dtype, with_cpu=not a.no_cpu_baseline, mode=a.mode, periodic=a.periodic,
               arith=a.arith, desc_tile=a.desc_tile, pipeline=a.pipeline, pipeline_density_wg=a.pipeline_density_wg,
               djac_tile=a.djac_tile, batches=a.batches,
               options=[tuple(o.split("=", 1)) for o in a.option])
    if a.workload is None and a.mode == "derivatives" and not a.periodic:
        # the same headline in the paper's arithmetic (float64 internally,
        # float32 outputs), and the other workloads, each with its own
        # roofline fraction and oracle baseline
        extra = {}
        if a.dtype == "float32" and a.arith == "mixed":
            extra[wl.name + "_arith_fp64"] = summary(run(wl, a.steps, a.warmup, a.dtype, with_cpu=False,
                                                         arith="fp64"))
        for name in EXTRA_WORKLOADS:
            xl = workload_by_name(name)
            extra[xl.name] = summary(run(xl, a.steps, a.warmup, a.dtype, with_cpu=not a.no_cpu_baseline,
                                         arith=a.arith, cpu_budget_s=8.0))
            print(f"[bench] {xl.name}: {extra[xl.name]['ms_per_step']:.3f} ms/step", file=sys.stderr, flush=True)
        line["configs"] = extra
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
