#!/usr/bin/env python3
"""Throughput of the compressed se_a descriptor (DP Compress, arXiv:2107.02103).

One step = one forward (T, D) plus one backward (dE/dR~) pass of the HIP
kernels over the whole workload, inputs resident in HBM.  Default workload:
Cu-like fcc 64^3 supercell, 1,048,576 atoms, r_c 8.0 A, sel 512, embedding
1->25->50->100, M' = 16, float64.

Prints one JSON line: neighbour pairs/s (whole job), the fraction of the
FP64 vector FMA peak reached with the algorithmic FLOP count
(5,400 per valid pair + 12,800 per atom), the roofline of the dominant kernel
(HIP events on the launch stream) and the plain C oracle timed on this host's
cores on a bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "neighbor-pairs/s fwd+bwd compressed se_a (fp64) + % of FP64 vector FMA peak"
PEAK_TFLOPS = {"f64": 78.6, "f32": 157.3, "f32acc64": 157.3}   # MI355X vector peaks
FLOP_PAIR_FWD, FLOP_PAIR_BWD, FLOP_ATOM = 1800.0, 3600.0, 12800.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash(kernel="se_a"):
    src = ("dpc_descriptor.hip" if kernel.startswith("descriptor") else
           "dpc_env.hip" if kernel in ("env_mat_kernel", "force_kernel", "reverse_kernel") else
           "dpc_se_a.hip")
    p = os.path.join(ROOT, "paper_2107_02103_amd", "csrc", src)
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


def stored_profile(cfg_name, kernel, dtype="f64"):
    """The committed rocprofv3 --pmc summary of this kernel and workload
    (HBM bytes per launch from FETCH_SIZE and WRITE_SIZE, calibrated by a
    plain copy; the shader clock from GRBM_GUI_ACTIVE where taken) and its
    file name, if it was taken on the current kernel source; else (None,
    None).  These counters cannot be read in the same process as the timing,
    so the values are stored measurements, not this run's."""
    suffix = "" if dtype == "f64" else "_" + dtype
    rel = os.path.join("profiles", f"pmc_{kernel}_{cfg_name}{suffix}.json")
    p = os.path.join(ROOT, rel)
    if not os.path.exists(p):
        return None, None
    d = json.load(open(p))
    if d.get("kernel_source_sha256_16") != kernel_source_hash(kernel):
        return None, None
    return d, rel


def hbm_traffic(cfg_name, kernel, dtype="f64"):
    d, rel = stored_profile(cfg_name, kernel, dtype)
    return (d.get("hbm_bytes_per_launch"), rel) if d else (None, None)


def library_record():
    """Which library this run loaded, and a hash of the sources it is built from."""
    from paper_2107_02103_amd import binding as B
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2107_02103_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        h.update(f.encode())
        h.update(open(os.path.join(csrc, f), "rb").read())
    return {"path": os.path.relpath(B.LIB_PATH, ROOT), "csrc_sha256_16": h.hexdigest()[:16]}


def roofline_entry(bound, kernel, achieved, peak, unit, cfg_name, dtype="f64", stored=True):
    d, src = stored_profile(cfg_name, kernel, dtype) if stored else (None, None)
    e = {"bound": bound, "kernel": kernel, "achieved": achieved, "peak": peak, "unit": unit,
         "frac": achieved / peak, "traffic": d.get("hbm_bytes_per_launch") if d else None,
         "traffic_source": src}
    if d and d.get("shader_clock_ghz"):
        # the peak is quoted at 2.4 GHz; the kernel ran at this clock under load
        e["sclk_ghz"] = d["shader_clock_ghz"]
    return e


def cpu_baseline(x, seconds, dtype="f64", atoms=None):
    """The C oracle (plain loops, OpenMP over atoms; float64 arithmetic on the
    mode's inputs, float32-rounded for the float32 modes) on the first atoms
    of the workload, in chunks, until `seconds` of wall time are used.  When
    one pass over the whole workload takes under a third of that, the whole
    workload is run three times and the median is reported."""
    import numpy as np
    from oracle import cref
    from oracle.table import build_tables
    c = x.cfg
    n = x.nlist.shape[0] if atoms is None else atoms
    tabs, em, dT = build_tables(x), x.em[:n], x.dT[:n]
    if dtype != "f64":
        tabs = [t.rounded(np.float32) for t in tabs]
        em = em.astype(np.float32).astype(np.float64)
        dT = dT.astype(np.float32).astype(np.float64)
    pb = cref.Problem(em, x.nlist[:n], x.atype[:n], tabs, c.sel, c.m2)
    chunk = 512

    def run(limit):
        done, pairs = 0, 0
        t0 = time.perf_counter()
        while done < n and time.perf_counter() - t0 < limit:
            i1 = min(n, done + chunk)
            pb.forward(done, i1)
            pb.backward(dT[done:i1], done, i1)
            pairs += int((x.nlist[done:i1] >= 0).sum())
            done = i1
        return done, pairs, time.perf_counter() - t0

    done, pairs, dt = run(seconds)
    how = "1 run"
    if done == n and dt < seconds / 3:
        times = [dt] + [run(float("inf"))[2] for _ in range(2)]
        dt = float(np.median(times))
        how = "median of 3 runs"
    cpu = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": pairs / dt, "unit": "pairs/s", "cores": cref.num_threads(), "kind": "oracle",
            "sample": f"atoms 0..{done - 1} of {n} ({pairs} valid pairs), fwd+bwd, {how}, "
                      f"{dt:.2f} s, {cpu}"}


def copy_probe(mib):
    """Device-to-device copy of `mib` MiB, three times (counter calibration)."""
    import torch
    n = mib * (1 << 20) // 8
    a = torch.ones(n, dtype=torch.float64, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n * 8, "launches": 3}), flush=True)


def bench_descriptor_bwd(args):
    """dpc_descriptor_bwd (dE/dT from dE/dD and T) over the configuration's
    atoms with M = 100, M' = 16: seeded standard-normal T and dE/dD resident
    in HBM, HIP events around each launch on the launch stream.  The kernel
    is bound by HBM bandwidth: 8 (4 M + M M' + 4 M) bytes per atom in float64."""
    import numpy as np
    import torch
    import paper_2107_02103_amd as P
    from synth.configs import get_config
    from synth.system import random_grad
    from oracle.se_a import descriptor_backward

    key = int(args.config) if args.config.isdigit() else args.config
    cfg = get_config(key)
    n, m1, m2 = cfg.natoms, cfg.m1, cfg.m2
    log(f"[bench] descriptor backward: generating T and dE/dD for {n} atoms")
    rng = np.random.default_rng([2107_02103, 77, 3])
    T = random_grad(rng, n, m1)
    dD = random_grad(rng, n, m1, width=m2)
    Tg, Dg = torch.from_numpy(T).cuda(), torch.from_numpy(dD).cuda()
    out = torch.empty_like(Tg)
    s = torch.cuda.Stream()
    run = lambda: P.dpc_descriptor_bwd(s, P.DPC_F64, n, m1, m2, Tg, Dg, out)
    with torch.cuda.stream(s):
        for _ in range(args.warmup):
            run()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        t0 = time.perf_counter()
        for e0, e1 in evs:
            e0.record(s)
            run()
            e1.record(s)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    nbytes = 8.0 * (4 * m1 + m1 * m2 + 4 * m1) * n
    achieved = nbytes / (ms * 1e-3) / 1e9
    res = {
        "metric": "descriptor backward dE/dT from dE/dD (fp64), atoms/s + % of HBM bandwidth",
        "value": n * args.steps / wall, "unit": "atoms/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": wall / args.steps * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{cfg.name} descriptor: {n} atoms, M {m1}, M2 {m2}, "
                               "T and dE/dD standard normal", "atoms": n},
        "kernel_ms": ms,
        "roofline": roofline_entry("hbm", "descriptor_bwd_m16_kernel", achieved, 8000.0, "GB/s", cfg.name),
        "library": library_record(),
    }
    del Tg, Dg, out
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        # the oracle (plain Python loops, one core) on the first atoms for ~cpu_seconds
        t0, done = time.perf_counter(), 0
        while done < n and time.perf_counter() - t0 < args.cpu_seconds:
            descriptor_backward(T[done:done + 16], dD[done:done + 16])
            done += 16
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": done / dt, "unit": "atoms/s", "cores": 1, "kind": "oracle",
                               "sample": f"atoms 0..{done - 1} of {n}, {dt:.1f} s"}
    print(json.dumps(res), flush=True)


def bench_env_force(args):
    """The steps on either side of the descriptor: dpc_env_mat_a (positions ->
    R~) and dpc_force_a (dE/dR~ -> forces, virials) over the configuration,
    with the reverse slots built once (as a neighbour list is).  dE/dR~ is
    seeded standard normal on valid slots.  Both kernels are bound by HBM:
    env 4 B (nlist) + 32 B (R~) per slot; force 4 + 4 (nlist, reverse slot)
    + 32 (own dE/dR~ row) per slot + 32 (the reverse row) per valid slot +
    96 B (F, V) per atom, float64."""
    import numpy as np
    import torch
    import paper_2107_02103_amd as P
    from synth import make_inputs
    from synth.configs import get_config
    from synth.system import random_grad

    key = int(args.config) if args.config.isdigit() else args.config
    cfg = get_config(key)
    log(f"[bench] env/force: generating {cfg.name}")
    x = make_inputs(cfg, with_grad=False)
    n, nnei, pairs = cfg.natoms, cfg.nnei, x.n_valid
    st = x.stats
    coord = torch.from_numpy(x.coords).cuda()
    at = torch.from_numpy(x.atype).cuda()
    nl = torch.from_numpy(x.nlist).cuda()
    em = torch.empty((n, nnei, 4), dtype=torch.float64, device="cuda")
    rev = torch.empty((n, nnei), dtype=torch.int32, device="cuda")
    lam = random_grad(np.random.default_rng([2107_02103, 88, 9]), n, nnei) * (x.nlist >= 0)[..., None]
    dem = torch.from_numpy(lam).cuda()
    del lam
    F = torch.empty((n, 3), dtype=torch.float64, device="cuda")
    V = torch.empty((n, 9), dtype=torch.float64, device="cuda")
    s = torch.cuda.Stream()
    env = lambda: P.dpc_env_mat_a(s, P.DPC_F64, n, cfg.ntypes, nnei, cfg.box, cfg.rc, cfg.rcs,
                                  st["mean"], st["sigma"], st["sigma_all"], coord, at, nl, em)
    force = lambda: P.dpc_force_a(s, P.DPC_F64, n, cfg.ntypes, nnei, cfg.box, cfg.rc, cfg.rcs,
                                  st["sigma"], st["sigma_all"], coord, at, nl, rev, dem, F, V)
    with torch.cuda.stream(s):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        P.dpc_nlist_reverse(s, n, cfg.ntypes, cfg.sel, cfg.box, coord, at, nl, rev)
        e1.record(s)
        for _ in range(args.warmup):
            env(); force()
        torch.cuda.synchronize()
        rev_ms = e0.elapsed_time(e1)
        evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(args.steps)]
        t0 = time.perf_counter()
        for a, b, c in evs:
            a.record(s); env(); b.record(s); force(); c.record(s)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    env_ms = float(np.mean([a.elapsed_time(b) for a, b, _ in evs]))
    force_ms = float(np.mean([b.elapsed_time(c) for _, b, c in evs]))
    env_bytes = 36.0 * n * nnei
    force_bytes = 40.0 * n * nnei + 32.0 * pairs + 96.0 * n
    dom, dom_ms, dom_bytes = ("force_kernel", force_ms, force_bytes) if force_ms >= env_ms else \
        ("env_mat_kernel", env_ms, env_bytes)
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    res = {
        "metric": "environment matrix + force/virial assembly (fp64), neighbour pairs/s + % of HBM bandwidth",
        "value": pairs * args.steps / wall, "unit": "pairs/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": wall / args.steps * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {n} atoms, sel {list(cfg.sel)}, rc {cfg.rc}, rcs {cfg.rcs}; "
                               "dE/dR~ standard normal on valid slots", "atoms": n, "valid_pairs": pairs},
        "env_ms": env_ms, "force_ms": force_ms, "reverse_ms_once": rev_ms,
        "env_GBps": env_bytes / (env_ms * 1e-3) / 1e9, "force_GBps": force_bytes / (force_ms * 1e-3) / 1e9,
        "roofline": roofline_entry("hbm", dom, achieved, 8000.0, "GB/s", cfg.name),
        "library": library_record(),
    }
    print(json.dumps(res), flush=True)


def _fitting_setup(n, m1, m2, width=240):
    """A seeded random fitting net on the device, its workspace and a rocBLAS handle."""
    import numpy as np
    import torch
    import paper_2107_02103_amd as P
    from synth.system import random_fitting_net
    net = random_fitting_net(np.random.default_rng([2107_02103, 66, 1]), m1 * m2, (width,) * 3)
    keep = [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in net["W"] + net["b"] + [net["w_out"]]]
    c = P.dpc_fitting_net()
    c.n_in, c.width, c.b_out = m1 * m2, width, net["b_out"]
    for l in range(3):
        c.W[l] = keep[l].data_ptr()
        c.b[l] = keep[3 + l].data_ptr()
    c.w_out = keep[6].data_ptr()
    nb = P.dpc_fitting_workspace_bytes(n, width)
    ws = torch.empty(nb // 8, dtype=torch.float64, device="cuda")
    return c, keep, ws, nb, P.RocblasHandle()


def bench_fitting(args):
    """dpc_fitting_fwd_bwd (energy and dE/dD) over the configuration's atoms:
    M = 100, M' = 16 descriptors (seeded standard normal), widths 240; its
    GEMMs run on the matrix cores through rocBLAS.  FLOP per atom:
    4 (1600 x 240 + 2 x 240 x 240) (forward and data gradient)."""
    import numpy as np
    import torch
    import paper_2107_02103_amd as P
    from synth.configs import get_config
    from synth.system import random_grad
    key = int(args.config) if args.config.isdigit() else args.config
    cfg = get_config(key)
    n, m1, m2 = cfg.natoms, cfg.m1, cfg.m2
    log(f"[bench] fitting net: {n} atoms")
    D = torch.from_numpy(random_grad(np.random.default_rng([2107_02103, 77, 8]), n, m1, width=m2)).cuda()
    net, keep, ws, nb, h = _fitting_setup(n, m1, m2)
    E = torch.empty(n, dtype=torch.float64, device="cuda")
    G = torch.empty_like(D)
    s = torch.cuda.Stream()
    run = lambda: P.dpc_fitting_fwd_bwd(s, h.value, n, net, D, ws, nb, E, G)
    with torch.cuda.stream(s):
        for _ in range(args.warmup):
            run()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        t0 = time.perf_counter()
        for a, b in evs:
            a.record(s); run(); b.record(s)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    flop = 4.0 * n * (m1 * m2 * 240 + 2 * 240 * 240)
    res = {"metric": "fitting net energy + dE/dD (fp64), atoms/s + % of FP64 matrix peak",
           "value": n * args.steps / wall, "unit": "atoms/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": wall / args.steps * 1e3, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
           "config": {"workload": f"{cfg.name} fitting net: {n} atoms, input {m1 * m2}, widths 240-240-240, "
                                  "descriptors standard normal", "atoms": n},
           "ms": ms,
           "roofline": {"bound": "mfma", "kernel": "rocBLAS dgemm + fitting kernels", "achieved": flop / (ms * 1e-3) / 1e12,
                        "peak": 78.6, "unit": "TFLOP/s", "frac": flop / (ms * 1e-3) / 1e12 / 78.6, "traffic": None}}
    h.close()
    print(json.dumps(res), flush=True)


def bench_chain(args):
    """Positions to energies and forces: dpc_env_mat_a (R~), dpc_se_a_tab_fwd
    (T, D), dpc_fitting_fwd_bwd (E, dE/dD; seeded random fitting net),
    dpc_se_a_tab_bwd_from_dD (dE/dT formed inside the backward, then dE/dR~)
    and dpc_force_a, one call each per step on one stream.  The neighbour
    list (dpc_nlist_build) and its reverse slots are built once from the
    positions, as an MD code does every few steps; the descriptor backward
    and the backward as two calls are timed once beside the fused call.
    float64."""
    import numpy as np
    import torch
    import paper_2107_02103_amd as P
    from synth import make_inputs
    from synth.configs import get_config
    from synth.system import random_grad

    key = int(args.config) if args.config.isdigit() else args.config
    cfg = get_config(key)
    log(f"[bench] chain: generating {cfg.name}")
    x = make_inputs(cfg, with_grad=False)
    n, nnei, m1, m2, pairs = cfg.natoms, cfg.nnei, cfg.m1, cfg.m2, x.n_valid
    st = x.stats
    op = P.SeATab(x.nets, x.lo, x.L1, x.L2, cfg.d1, cfg.d2, cfg.sel, m2)
    coord = torch.from_numpy(x.coords).cuda()
    at = torch.from_numpy(x.atype).cuda()
    nl = torch.empty((n, nnei), dtype=torch.int32, device="cuda")
    nlb = P.dpc_nlist_workspace_bytes(n, cfg.box, cfg.rc)
    nlws = torch.empty(nlb, dtype=torch.uint8, device="cuda")
    fnet, keep, ws, nb, hblas = _fitting_setup(n, m1, m2)
    Ea = torch.empty(n, dtype=torch.float64, device="cuda")
    dD = torch.empty((n, m1, m2), dtype=torch.float64, device="cuda")
    em = torch.empty((n, nnei, 4), dtype=torch.float64, device="cuda")
    T = torch.empty((n, m1, 4), dtype=torch.float64, device="cuda")
    D = torch.empty((n, m1, m2), dtype=torch.float64, device="cuda")
    dT = torch.empty_like(T)
    dR = torch.empty_like(em)
    rev = torch.empty((n, nnei), dtype=torch.int32, device="cuda")
    F = torch.empty((n, 3), dtype=torch.float64, device="cuda")
    V = torch.empty((n, 9), dtype=torch.float64, device="cuda")
    s = torch.cuda.Stream()
    names = ["env", "fwd", "fitting", "bwd_from_dD", "force"]

    def step(evs=None):
        calls = [
            lambda: P.dpc_env_mat_a(s, P.DPC_F64, n, cfg.ntypes, nnei, cfg.box, cfg.rc, cfg.rcs, st["mean"],
                                    st["sigma"], st["sigma_all"], coord, at, nl, em),
            lambda: op.forward(em, nl, at, T, D, stream=s),
            lambda: P.dpc_fitting_fwd_bwd(s, hblas.value, n, fnet, D, ws, nb, Ea, dD),
            lambda: op.backward_from_dD(em, nl, at, T, dD, dR, stream=s),
            lambda: P.dpc_force_a(s, P.DPC_F64, n, cfg.ntypes, nnei, cfg.box, cfg.rc, cfg.rcs, st["sigma"],
                                  st["sigma_all"], coord, at, nl, rev, dR, F, V),
        ]
        for k, c in enumerate(calls):
            if evs is not None:
                evs[k].record(s)
            c()
        if evs is not None:
            evs[-1].record(s)

    once = {}
    with torch.cuda.stream(s):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record(s)
        P.dpc_nlist_build(s, n, cfg.ntypes, cfg.sel, cfg.box, cfg.rc, coord, at, nlws, nlb, nl, wait=False)
        ev[1].record(s)
        P.dpc_nlist_reverse(s, n, cfg.ntypes, cfg.sel, cfg.box, coord, at, nl, rev)
        ev[2].record(s)
        torch.cuda.synchronize()
        status = nlws[:8].view(torch.int32).cpu().tolist()
        if status != [0, 0]:
            raise RuntimeError(f"neighbour list status {status} (truncated, over capacity)")
        once["nlist"] = ev[0].elapsed_time(ev[1])
        once["reverse"] = ev[1].elapsed_time(ev[2])
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        # the same backward as two calls, for comparison
        ev2 = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev2[0].record(s)
        op.descriptor_backward(T, dD, dT, stream=s)
        ev2[1].record(s)
        op.backward(em, nl, at, dT, dR, stream=s)
        ev2[2].record(s)
        torch.cuda.synchronize()
        once["descriptor_bwd (two-call path)"] = ev2[0].elapsed_time(ev2[1])
        once["bwd (two-call path)"] = ev2[1].elapsed_time(ev2[2])
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(args.steps)]
        t0 = time.perf_counter()
        for e in evs:
            step(e)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    per = {nm: float(np.mean([e[k].elapsed_time(e[k + 1]) for e in evs])) for k, nm in enumerate(names)}
    res = {
        "metric": "positions to energies and forces (fp64), neighbour pairs/s",
        "value": pairs * args.steps / wall, "unit": "pairs/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": wall / args.steps * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {n} atoms, sel {list(cfg.sel)}; random fitting net 240-240-240",
                   "atoms": n, "valid_pairs": pairs},
        "kernel_ms": per, "once_ms": once, "library": library_record(),
    }
    print(json.dumps(res), flush=True)


def bench_nlist(args):
    """dpc_nlist_build over the configuration's positions (cell list, then one
    wavefront per atom ranking its candidates).  Algorithmic bytes: the
    positions and types in (28 B per atom) and the list out (4 B per slot)."""
    import numpy as np
    import torch
    import paper_2107_02103_amd as P
    from synth import make_inputs
    from synth.configs import get_config
    key = int(args.config) if args.config.isdigit() else args.config
    cfg = get_config(key)
    log(f"[bench] neighbour list: generating {cfg.name}")
    x = make_inputs(cfg, with_grad=False)
    n, nnei = cfg.natoms, cfg.nnei
    coord = torch.from_numpy(x.coords).cuda()
    at = torch.from_numpy(x.atype).cuda()
    nl = torch.empty((n, nnei), dtype=torch.int32, device="cuda")
    nb = P.dpc_nlist_workspace_bytes(n, cfg.box, cfg.rc)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    s = torch.cuda.Stream()
    run = lambda: P.dpc_nlist_build(s, n, cfg.ntypes, cfg.sel, cfg.box, cfg.rc, coord, at, ws, nb, nl,
                                    wait=False)
    with torch.cuda.stream(s):
        for _ in range(args.warmup):
            run()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        t0 = time.perf_counter()
        for a, b in evs:
            a.record(s); run(); b.record(s)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    same = bool(np.array_equal(nl.cpu().numpy(), x.nlist))
    nbytes = 28.0 * n + 4.0 * n * nnei
    achieved = nbytes / (ms * 1e-3) / 1e9
    res = {"metric": "neighbour list build (cell list, type-then-distance order), atoms/s",
           "value": n * args.steps / wall, "unit": "atoms/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": wall / args.steps * 1e3, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
           "config": {"workload": f"{cfg.name}: {n} atoms, box {cfg.box:.3f}, rc {cfg.rc}, sel {list(cfg.sel)}",
                      "atoms": n, "workspace_bytes": nb},
           "ms": ms, "equals_generator_lists": same,
           "roofline": roofline_entry("hbm", "nl_list_kernel", achieved, 8000.0, "GB/s", cfg.name),
           "library": library_record()}
    if not args.no_cpu_baseline:
        from oracle import nlist as onl
        t0, done, chunk = time.perf_counter(), 0, 64
        while done < n and time.perf_counter() - t0 < args.cpu_seconds:
            onl.neighbour_list(x.coords, x.atype, cfg.sel, cfg.box, cfg.rc,
                               centres=np.arange(done, min(n, done + chunk)))
            done = min(n, done + chunk)
        dt = time.perf_counter() - t0
        from oracle import cref
        res["cpu_baseline"] = {"value": done / dt, "unit": "atoms/s", "cores": cref.num_threads(),
                               "kind": "oracle", "sample": f"atoms 0..{done - 1} of {n} (brute force "
                               f"over all atoms), {dt:.1f} s"}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="3", help="workload index 0..4 or name (default 3: cu1m)")
    ap.add_argument("--dtype", default=None, choices=[None, "f64", "f32", "f32acc64"])
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--stride", type=float, default=None,
                    help="table stride d1 on the observed range (band stride 10 x d1; default: the "
                         "workload's 0.01 / 0.1), for the stride study")
    ap.add_argument("--chain", action="store_true",
                    help="time positions -> R~ -> T, D -> E, dE/dD -> dE/dT -> dE/dR~ -> forces")
    ap.add_argument("--fitting", action="store_true", help="time the fitting net (energy and dE/dD)")
    ap.add_argument("--nlist", action="store_true", help="time the neighbour-list build")
    ap.add_argument("--env-force", action="store_true",
                    help="time the environment matrix and the force / virial assembly instead")
    ap.add_argument("--descriptor-bwd", action="store_true",
                    help="time the descriptor backward (dE/dT from dE/dD) instead of the se_a step")
    ap.add_argument("--shard", type=int, default=1,
                    help="time one GPU's share when the workload is split by contiguous atom ranges "
                         "over this many GPUs: atoms 0 .. natoms/K - 1 (the kernels need no exchange)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (3 times), the known-size "
                         "kernel that calibrates the HBM byte counters, and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): the descriptor kernel "
              "shards by atoms with no exchange, so multi-GPU throughput is not measured here.",
              file=sys.stderr)
        sys.exit(2)

    if args.copy_probe_mib:
        copy_probe(args.copy_probe_mib)
        return
    if args.descriptor_bwd:
        bench_descriptor_bwd(args)
        return
    if args.env_force:
        bench_env_force(args)
        return
    if args.chain:
        bench_chain(args)
        return
    if args.fitting:
        bench_fitting(args)
        return
    if args.nlist:
        bench_nlist(args)
        return

    import numpy as np
    import torch
    import paper_2107_02103_amd as P
    from synth import make_inputs
    from synth.configs import get_config

    key = int(args.config) if args.config.isdigit() else args.config
    cfg = get_config(key)
    if args.stride:
        cfg = cfg.with_(d1=args.stride, d2=10 * args.stride)
    dtype = args.dtype or cfg.dtype
    mode = {"f64": P.DPC_F64, "f32": P.DPC_F32, "f32acc64": P.DPC_F32_ACC64}[dtype]
    store = np.float64 if dtype == "f64" else np.float32

    t = time.perf_counter()
    log(f"[bench] generating {cfg.name} ({cfg.natoms} atoms, sel {cfg.sel})")
    x = make_inputs(cfg)
    atoms, pairs = cfg.natoms, x.n_valid
    if args.shard > 1:
        # the table and the neighbour lists stay those of the whole system;
        # this GPU's atoms are a contiguous range of rows
        atoms = cfg.natoms // args.shard
        pairs = int(np.count_nonzero(x.nlist[:atoms] >= 0))
    log(f"[bench] inputs ready in {time.perf_counter() - t:.1f} s: {pairs} valid pairs")

    op = P.SeATab(x.nets, x.lo, x.L1, x.L2, cfg.d1, cfg.d2, cfg.sel, cfg.m2, dtype=mode)
    em = torch.from_numpy(x.em[:atoms].astype(store, copy=False)).cuda()
    nl = torch.from_numpy(x.nlist[:atoms]).cuda()
    at = torch.from_numpy(x.atype[:atoms]).cuda()
    dT = torch.from_numpy(x.dT[:atoms].astype(store, copy=False)).cuda()
    tacc = torch.float32 if dtype == "f32" else torch.float64
    T = torch.empty((atoms, cfg.m1, 4), dtype=tacc, device="cuda")
    D = torch.empty((atoms, cfg.m1, cfg.m2), dtype=tacc, device="cuda")
    dR = torch.empty((atoms, cfg.nnei, 4), dtype=tacc, device="cuda")
    torch.cuda.synchronize()
    log(f"[bench] resident on {torch.cuda.get_device_name(0)}")

    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        for _ in range(args.warmup):
            op.forward(em, nl, at, T, D, stream=s)
            op.backward(em, nl, at, dT, dR, stream=s)
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
                torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        t0 = time.perf_counter()
        for e0, e1, e2 in evs:
            e0.record(s)
            op.forward(em, nl, at, T, D, stream=s)
            e1.record(s)
            op.backward(em, nl, at, dT, dR, stream=s)
            e2.record(s)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    fwd_ms = float(np.mean([a.elapsed_time(b) for a, b, _ in evs]))
    bwd_ms = float(np.mean([b.elapsed_time(c) for _, b, c in evs]))
    log(f"[bench] {args.steps} steps in {wall:.3f} s: fwd {fwd_ms:.3f} ms, bwd {bwd_ms:.3f} ms")

    flop_fwd = FLOP_PAIR_FWD * pairs + FLOP_ATOM * atoms
    flop_bwd = FLOP_PAIR_BWD * pairs
    step_s = wall / args.steps
    peak = PEAK_TFLOPS[dtype]
    tflops = (flop_fwd + flop_bwd) / step_s / 1e12
    # backward passes that accumulate in float64 (float64 and the mixed mode)
    # with M1 <= 128 run on the matrix-core kernel (the library's rule), in
    # float64 MFMA: its peak is the FP64 matrix peak, 78.6 TFLOP/s, as the
    # FP64 vector peak
    bwd_mfma = dtype in ("f64", "f32acc64") and cfg.widths[-1] <= 128
    bwd_name = "se_a_bwd_mfma_kernel" if bwd_mfma else "se_a_bwd_kernel"
    dom = bwd_name if bwd_ms >= fwd_ms else "se_a_fwd_kernel"
    bound = "mfma" if dom == "se_a_bwd_mfma_kernel" else "alu"
    dom_peak = PEAK_TFLOPS["f64"] if bound == "mfma" else peak
    dom_ms = max(bwd_ms, fwd_ms)
    dom_flop = flop_bwd if bwd_ms >= fwd_ms else flop_fwd
    achieved = dom_flop / (dom_ms * 1e-3) / 1e12
    out = {
        "metric": METRIC,
        "value": pairs * args.steps / wall,
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.kind} {cfg.ncell}^3 cells, {atoms} atoms, "
                               f"rc {cfg.rc}, rcs {cfg.rcs}, sel {list(cfg.sel)}, "
                               f"embedding {'-'.join(map(str, cfg.widths))}, M2 {cfg.m2}, "
                               f"table stride {cfg.d1}/{cfg.d2}"
                               + (f"; one GPU's share of {args.shard}: atoms 0..{atoms - 1}" if args.shard > 1 else ""),
                   "atoms": atoms, "valid_pairs": pairs, "nnei": cfg.nnei,
                   "table_bytes": int(op.coeff.numel() * op.coeff.element_size())},
        "tflops_algorithmic": tflops,
        "frac_vector_peak": tflops / peak,
        "fwd_ms": fwd_ms,
        "bwd_ms": bwd_ms,
        "roofline": roofline_entry(bound, dom, achieved, dom_peak, "TFLOP/s", cfg.name, dtype,
                                   stored=not (args.stride or args.shard > 1)),
        "library": library_record(),
    }
    del T, D, dR, em, dT
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log(f"[bench] cpu baseline (oracle) for ~{args.cpu_seconds:.0f} s")
        out["cpu_baseline"] = cpu_baseline(x, args.cpu_seconds, dtype, atoms)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
