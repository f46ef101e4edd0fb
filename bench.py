"""Benchmark: the 1.5-SPSA probe regenerate-and-apply sweeps on one MI355X.

A step is Algorithm 1 on one device with the forward passes replaced by synthetic losses:
for each of K probes zo_perturb(+eps), zo_perturb(-2 eps), zo_perturb(+eps); then
zo_probe_coeffs on the host; then one fused zo_update. Weights are one flat bf16 buffer
shaped like OPT-13B (12,853,473,280 parameters, ~N(0, 0.02)), resident in HBM before the
timed region starts; K = 16, eps = lr = 1e-3.

Prints one JSON line. `value` is the metric's own quantity: the fused update's effective
HBM bandwidth, algorithmic bytes (one read and one write of every weight) over the median
duration of its launches in the timed steps, with its params-probes rate beside it;
`roofline` is that kernel's. The whole step's rate is `step_gbps` (3K + 1 sweeps).
`fused_schedule` times the same step in 2K + 1 sweeps (zo_perturb2 merges the restore of
probe k with the +eps of probe k + 1, zo_update_restore merges the last restore with the
update) over the same number of steps; `roofline_update_restore` is the kernel it ends
with. `graph_fused_schedule` replays the fused step captured once into a HIP graph.
Per-kernel durations come from HIP events recorded around every launch on the stream the
kernels run on (medians; mean, min and max beside them). `opt30b` repeats the update, the
update with restore and a few steps of both schedules on an OPT-30B shaped buffer at K = 8
and K = 32 (run after the OPT-13B buffer is freed).
"""

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fused probe-update effective HBM GB/s + params·probes/s (OPT-13B shape, K=16)"
HBM_PEAK_GBPS = 8000.0
# VALU issue peak: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz (a wave64 instruction takes 4 cycles).
VALU_PEAK_TLANEOPS = 256 * 64 * 2.4e9 / 1e12
# LDS: 128 bytes per clock per CU = 32 conflict-free 4-byte table reads per clock; uniform random
# bytes into a 256-entry table on 32 banks cost 6.31 cycles per 64-lane read instead of 2.
LDS_PEAK_GLOOKUPS = 256 * 32 * 2.4  # 1e9 lookups/s
LDS_RANDOM_GLOOKUPS = 256 * 64 / 6.31 * 2.4


def workloads_names():
    import workloads
    return workloads.WORKLOADS.keys()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


SWEEP_SOURCES = ("zo_sweep.hip", "zo_stream.h", "zo_plan.h", "zo_plan.cpp")  # the kernels, their loops and launch shapes


def sweep_source_digest():
    """SHA-256 over the sources that decide which kernels run and how (the sweep kernels and
    the launch planner), in this order."""
    import hashlib
    h = hashlib.sha256()
    for name in SWEEP_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2609_38095_amd", "csrc", name), "rb").read())
    return h.hexdigest()


def measured_counters(workload, K, dtype, layout="flat"):
    """Per-launch HBM bytes (FETCH_SIZE and WRITE_SIZE, each scaled by a plain copy of known
    size) and VALU instruction counts (SQ_INSTS_VALU) from the committed rocprofv3 summaries,
    keyed by kernel; {} when none matches this workload or the sweep sources have changed since
    the counters were taken."""
    import glob
    digest = sweep_source_digest()
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        for line in open(path):
            if line.startswith("counters-json:"):
                d = json.loads(line.split(":", 1)[1])
                key = (d.get("workload"), d.get("K"), d.get("dtype"), d.get("layout", "flat"), d.get("source_sha256"))
                if key == (workload, K, dtype, layout, digest):
                    return d
    return {}


def binding_unit(hbm_frac, lds_busy=None, valu_busy=None):
    """The unit that bounds a kernel: the highest of its HBM fraction, LDS busy share and VALU
    busy share ("hbm", "lds" or "alu"); a share not measured (None) is left out."""
    use = {"hbm": hbm_frac, "lds": lds_busy, "alu": valu_busy}
    return max((u for u in use if use[u] is not None), key=lambda u: use[u])


_CPU = {}


def _oracle_window(off):
    """One full oracle step over the shared window at global offset `off` (a pool task)."""
    import oracle
    c = _CPU
    oracle.full_step(c["theta"], c["dtype"], off, 2024, 0, c["eps"], c["lr"], c["lp"], c["lm"], c["l0"])
    return 3 * c["K"] + 1


def cpu_baseline(w, K, budget_s=12.0, procs=1):
    """The oracle on the host: full steps (3K perturbs + one update) over windows of the
    workload at random offsets, in one process or in `procs` forked worker processes that
    each run whole windows. Must run before the GPU is touched (the workers are forked)."""
    import multiprocessing

    import numpy as np

    import workloads

    m = 1 << 16
    lp, lm, l0 = workloads.synthetic_losses(K, 0)
    _CPU.update(theta=workloads.normal_bf16_bits(m, 0) if w.dtype == "bf16" else workloads.normal_f32(m, 0),
                dtype=w.dtype, eps=w.eps, lr=w.lr, lp=lp, lm=lm, l0=l0, K=K)
    rng = np.random.default_rng(1)
    offsets = [int(rng.integers(0, w.n - m)) for _ in range(1024)]
    windows, sweeps = 0, 0
    t0 = time.perf_counter()
    if procs == 1:
        while time.perf_counter() - t0 < budget_s and windows < len(offsets):
            sweeps += _oracle_window(offsets[windows])
            windows += 1
    else:
        with multiprocessing.get_context("fork").Pool(procs) as pool:
            while time.perf_counter() - t0 < budget_s and windows + procs <= len(offsets):
                sweeps += sum(pool.map(_oracle_window, offsets[windows:windows + procs], chunksize=1))
                windows += procs
    t_total = time.perf_counter() - t0
    b = 2 if w.dtype == "bf16" else 4
    gbps = sweeps * 2 * b * m / t_total / 1e9
    how = "single-threaded numpy" if procs == 1 else f"{procs} worker processes (one window each), numpy"
    return {"value": round(gbps, 4), "unit": "GB/s", "cores": procs, "kind": "oracle",
            "sample": f"{windows} full steps (3K+1 = {3 * K + 1} sweeps) over windows of {m} weights at random "
                      f"offsets of the {w.name} buffer, {how}, {t_total:.1f} s wall; "
                      f"host {platform.processor() or platform.machine()}, os.cpu_count()={os.cpu_count()}"}


class Timer:
    """HIP events recorded around launches on one stream, per kernel name."""

    def __init__(self, stream):
        self.stream = stream
        self.ev = {}

    def __call__(self, kind, fn):
        import torch
        a = torch.cuda.Event(enable_timing=True)
        z = torch.cuda.Event(enable_timing=True)
        a.record(self.stream)
        fn()
        z.record(self.stream)
        self.ev.setdefault(kind, []).append((a, z))

    def ms(self):
        """{kind: array of per-launch milliseconds} (after a synchronisation)."""
        import numpy as np
        return {k: np.array([a.elapsed_time(z) for a, z in v]) for k, v in self.ev.items()}


def launch_stats(d):
    import numpy as np
    return {"median_ms": round(float(np.median(d)), 4), "avg_ms": round(float(d.mean()), 4),
            "min_ms": round(float(d.min()), 4), "max_ms": round(float(d.max()), 4), "launches": int(d.size)}


def roofline(kernel, d, n, b, K, counters, ceil_gbps=None, per_call=None):
    """The roofline object of one sweep kernel from its per-launch durations d (ms): achieved
    algorithmic GB/s over the median launch, against 8 TB/s, with the measured VALU, integer
    and LDS shares from the committed counters, and the unit that binds."""
    import numpy as np
    sweep_bytes = 2.0 * b * n
    med = float(np.median(d))
    gb = sweep_bytes / (med * 1e-3) / 1e9
    hbm_frac = gb / HBM_PEAK_GBPS
    r = {"kernel": kernel, "bound": "hbm", "achieved": round(gb, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
         "frac": round(hbm_frac, 4),
         "traffic": counters.get("traffic_bytes_per_launch", {}).get(kernel), **launch_stats(d),
         "bytes_per_launch": sweep_bytes, "hbm_frac": round(hbm_frac, 4),
         "frac_of_rmw_ceiling": round(gb / ceil_gbps, 4) if ceil_gbps else None}
    if per_call:
        r["per_sweep"] = per_call
    if kernel.startswith("zo_update"):
        r["params_probes_per_s"] = float(f"{n * K / (med * 1e-3):.4e}")
    valu = counters.get("valu_instructions_per_launch", {}).get(kernel)
    alu = valu * 64 / (med * 1e-3) / 1e12 if valu else None
    valu_busy = counters.get("valu_busy", {}).get(kernel)
    ints = counters.get("int_instructions_per_launch", {}).get(kernel)
    if alu is not None:
        r["valu_tlaneops"] = round(alu, 2)
        r["alu_frac"] = round(alu / VALU_PEAK_TLANEOPS, 4)
    if valu_busy is not None:
        r["valu_busy"] = valu_busy
    if ints is not None:
        it = ints * 64 / (med * 1e-3) / 1e12
        r["int32_int64_tlaneops"] = round(it, 2)
        r["int32_int64_frac"] = round(it / VALU_PEAK_TLANEOPS, 4)
    lds = counters.get("lds_per_launch", {}).get(kernel)
    lds_busy = lds["lds_busy"] if lds is not None else None
    glk = None
    if kernel.startswith("zo_update"):
        # one table lookup per element and probe group
        glk = n * ((K + 7) // 8) / (med * 1e-3) / 1e9
        r["table_glookups_per_s"] = round(glk, 1)
        if lds_busy is not None:
            r["lds_busy"] = lds_busy
    bound = binding_unit(hbm_frac, lds_busy if glk is not None else None,
                         valu_busy if valu_busy is not None else r.get("alu_frac"))
    if bound == "lds":
        r.update(bound="lds", achieved=round(glk, 1), peak=round(LDS_PEAK_GLOOKUPS, 1),
                 unit="G lookups/s", frac=round(glk / LDS_PEAK_GLOOKUPS, 4),
                 peak_random_index=round(LDS_RANDOM_GLOOKUPS, 1),
                 frac_of_random_index_peak=round(glk / LDS_RANDOM_GLOOKUPS, 4))
    elif bound == "alu":
        r.update(bound="alu", achieved=round(alu, 2), peak=round(VALU_PEAK_TLANEOPS, 2), unit="Tlane-op/s",
                 frac=round(alu / VALU_PEAK_TLANEOPS, 4))
    return r


class Sweeps:
    """The library calls of one workload on one device, flat buffer or separate tensors."""

    def __init__(self, w, layout, dev, seed=2024):
        import torch

        import paper_2609_38095_amd as zo
        import workloads
        self.zo, self.w, self.seed = zo, w, seed
        self.stream = torch.cuda.current_stream(dev)
        self.cur = self.stream  # the stream the sweeps are issued on (the capture stream while capturing)
        dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        if layout == "flat":
            self.theta = torch.empty(w.n, dtype=dt, device=dev)
            if w.hidden:
                workloads.fill_model_buffer_device(self.theta, w)
            else:
                self.theta.copy_(torch.from_numpy(workloads.tiny_theta(w.n)))
            self.tensors = None
            self.n_tensors = 1
        else:
            spans = workloads.tensor_offsets(w)
            self.tensors = [torch.empty(sz, dtype=dt, device=dev) for _, _, sz in spans]
            self.offs = [o for _, o, _ in spans]
            workloads.fill_model_tensors_device(self.tensors, w)
            self.n_tensors = len(self.tensors)
        torch.cuda.synchronize()

    def perturb(self, k, e, step):
        if self.tensors is None:
            self.zo.zo_perturb(self.theta, k, e, self.seed, step, stream=self.cur)
        else:
            self.zo.zo_perturb_segments(self.tensors, self.offs, k, e, 0, 0.0, self.seed, step, stream=self.cur)

    def perturb2(self, ka, ea, kb, eb, step):
        if self.tensors is None:
            self.zo.zo_perturb2(self.theta, ka, ea, kb, eb, self.seed, step, stream=self.cur)
        else:
            self.zo.zo_perturb_segments(self.tensors, self.offs, ka, ea, kb, eb, self.seed, step, stream=self.cur)

    def update(self, c, step):
        if self.tensors is None:
            self.zo.zo_update(self.theta, c, self.w.lr, self.seed, step, stream=self.cur)
        else:
            self.zo.zo_update_segments(self.tensors, self.offs, c, self.w.lr, self.seed, step, stream=self.cur)

    def update_restore(self, c, step, kr, er):
        if self.tensors is None:
            self.zo.zo_update_restore(self.theta, c, self.w.lr, self.seed, step, kr, er, stream=self.cur)
        else:
            self.zo.zo_update_segments(self.tensors, self.offs, c, self.w.lr, self.seed, step, kr, er,
                                       stream=self.cur)

    def one_step(self, K, step, timer=None):
        """Algorithm 1's sequential schedule: 3K perturbs, the coefficients, one update."""
        import workloads
        w = self.w
        run = timer or (lambda kind, fn: fn())
        lp, lm, l0 = workloads.synthetic_losses(K, step)
        for k in range(K):
            for e in (w.eps, -2.0 * w.eps, w.eps):
                run("zo_perturb", lambda: self.perturb(k, e, step))
        c = self.zo.zo_probe_coeffs(lp, lm, l0, w.eps)
        run("zo_update", lambda: self.update(c, step))

    def fused_step(self, K, step, timer=None):
        """The fused schedule: 2K + 1 sweeps (restore of probe k merged with +eps of probe
        k + 1, the last restore merged with the update)."""
        import workloads
        w = self.w
        run = timer or (lambda kind, fn: fn())
        lp, lm, l0 = workloads.synthetic_losses(K, step)
        run("zo_perturb_fused", lambda: self.perturb(0, w.eps, step))
        for k in range(K):
            run("zo_perturb_fused", lambda: self.perturb(k, -2.0 * w.eps, step))
            if k + 1 < K:
                run("zo_perturb2", lambda: self.perturb2(k, w.eps, k + 1, w.eps, step))
        c = self.zo.zo_probe_coeffs(lp, lm, l0, w.eps)
        run("zo_update_restore", lambda: self.update_restore(c, step, K - 1, w.eps))


def rmw_ceiling(sw, b, launches=6):
    """The plain in-place read-modify-write ceiling of the flat buffer: the fastest of the
    XOR sweep's eight shapes (the sweeps' own streaming loop, grid-stride or one chunk per
    wave, unpaced or paced, two or three row groups in flight), each timed over `launches`
    launches (an even number of XOR passes leaves the weights as they were)."""
    import ctypes

    import numpy as np
    import torch
    calib = ctypes.CDLL(os.path.join(os.path.dirname(sw.zo.LIB_PATH), "libzo_calib.so"))
    calib.zo_calib_rmw_shape.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                                         ctypes.c_void_p]
    sptr = ctypes.c_void_p(sw.stream.cuda_stream)
    buf_bytes = sw.w.n * b - (sw.w.n * b) % 16
    base = {0: "grid-stride", 1: "one chunk per wave", 2: "grid-stride, paced", 3: "one chunk per wave, paced"}
    names = {flags | ahead: name + (", three ahead" if ahead else "") for ahead in (0, 4) for flags, name in base.items()}
    shapes = {}
    for shape, name in names.items():
        def rmw():
            rc = calib.zo_calib_rmw_shape(ctypes.c_void_p(sw.theta.data_ptr()), buf_bytes, 0x5A5A5A5A, shape, sptr)
            if rc != 0:
                raise RuntimeError(f"zo_calib_rmw_shape failed ({rc})")
        rmw()
        rmw()
        t = Timer(sw.stream)
        for _ in range(launches):
            t("rmw", rmw)
        torch.cuda.synchronize()
        med = float(np.median(t.ms()["rmw"]))
        shapes[name] = {"gbps": round(2.0 * buf_bytes / (med * 1e-3) / 1e9, 1), "median_ms": round(med, 4)}
    best = max(shapes, key=lambda k: shapes[k]["gbps"])
    return {"gbps": shapes[best]["gbps"], "shape": best, "shapes": shapes, "launches_per_shape": launches,
            "kernel": "plain in-place 16-byte XOR sweep of the same buffer (libzo_calib.so) by the sweeps' own "
                      "streaming loop and launch shapes, no probe work; the fastest shape"}


def opt30b_legs(dev, Ks=(8, 32), alone=10, steps=2):
    """The OPT-30B shaped buffer at each K: the update and the update with restore timed
    alone (`alone` launches each), then one warmup step and `steps` timed steps of the
    sequential and of the fused schedule with every launch timed."""
    import numpy as np
    import torch

    import workloads
    w = workloads.WORKLOADS["opt30b"]
    log(f"workload opt30b: n={w.n}, {w.n * 2 / 1e9:.2f} GB of weights")
    sw = Sweeps(w, "flat", dev)
    out = {}
    for K in Ks:
        counters = measured_counters(w.name, K, w.dtype)
        lp, lm, l0 = workloads.synthetic_losses(K, 77)
        c = sw.zo.zo_probe_coeffs(lp, lm, l0, w.eps)
        t = Timer(sw.stream)
        sw.update(c, 77)
        for _ in range(alone):
            t("zo_update", lambda: sw.update(c, 77))
        sw.update_restore(c, 77, K - 1, w.eps)
        for _ in range(alone):
            t("zo_update_restore", lambda: sw.update_restore(c, 77, K - 1, w.eps))
        sw.one_step(K, 100)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(steps):
            sw.one_step(K, 101 + s, t)
        torch.cuda.synchronize()
        seq = (time.perf_counter() - t0) / steps
        t0 = time.perf_counter()
        for s in range(steps):
            sw.fused_step(K, 201 + s, t)
        torch.cuda.synchronize()
        fused = (time.perf_counter() - t0) / steps
        ms = t.ms()
        sweep_bytes = 2.0 * 2 * w.n
        out[f"K{K}"] = {
            "K": K,
            "roofline_update": roofline("zo_update", ms["zo_update"], w.n, 2, K, counters),
            "roofline_update_restore": roofline("zo_update_restore", ms["zo_update_restore"], w.n, 2, K, counters),
            "roofline_perturb": roofline("zo_perturb", ms["zo_perturb"], w.n, 2, K, counters),
            "step_ms": round(seq * 1e3, 3), "step_gbps": round((3 * K + 1) * sweep_bytes / seq / 1e9, 1),
            "fused_step_ms": round(fused * 1e3, 3),
            "fused_step_gbps": round((2 * K + 1) * sweep_bytes / fused / 1e9, 1),
            "how": f"update and update with restore timed alone ({alone} launches each, medians; the update's "
                   f"launches inside the steps too), then {steps} timed steps of each schedule",
        }
        log(f"opt30b K={K}: update {out[f'K{K}']['roofline_update']['median_ms']} ms, "
            f"step {out[f'K{K}']['step_ms']} ms, fused {out[f'K{K}']['fused_step_ms']} ms")
    del sw
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="opt13b", choices=sorted(workloads_names()),
                    help="tiny, opt125m, opt1.3b, opt13b, opt30b, qwen3-1.7b or qwen3-8b")
    ap.add_argument("--K", type=int, default=0, help="probes per step (default: the workload's first)")
    ap.add_argument("--layout", default="flat", choices=["flat", "tensors"],
                    help="flat: one contiguous buffer (zo_perturb, zo_update); tensors: every OPT tensor "
                         "allocated separately, swept with zo_perturb_segments / zo_update_segments")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-opt30b", action="store_true",
                    help="skip the OPT-30B legs (run by default after the default OPT-13B flat workload)")
    ap.add_argument("--no-graph", action="store_true", help="skip the HIP graph replay of the fused step")
    ap.add_argument("--calib-copy-gib", type=float, default=0.0,
                    help="before warmup, run one plain device copy of this many GiB (calibrates HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the library has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import workloads

    w = workloads.WORKLOADS[args.workload]
    K = args.K or w.K[0]
    if args.layout == "tensors" and not w.hidden:
        print(f"--layout tensors needs a model-shaped workload ({w.name} is one flat vector)", file=sys.stderr)
        sys.exit(2)
    run_opt30b = not args.no_opt30b and args.workload == "opt13b" and args.layout == "flat"
    baselines = {}
    if not args.no_cpu_baseline:
        # before torch touches the GPU: the all-cores leg forks worker processes
        log("timing the CPU oracle baseline (one process, then all cores)")
        baselines["cpu_baseline"] = cpu_baseline(w, K)
        baselines["cpu_baseline_all_cores"] = cpu_baseline(w, K, procs=min(16, os.cpu_count() or 1))

    import numpy as np
    import torch

    import paper_2609_38095_amd as zo

    n, b = w.n, (2 if w.dtype == "bf16" else 4)
    dev = torch.device("cuda:0")
    zo.library()
    log(f"workload {w.name}: n={n} dtype={w.dtype} K={K} eps={w.eps} lr={w.lr}; {n * b / 1e9:.2f} GB of weights")
    sw = Sweeps(w, args.layout, dev)
    if args.layout == "tensors":
        log(f"per-tensor layout: {sw.n_tensors} separately allocated tensors")
    if args.calib_copy_gib > 0:
        nb = int(args.calib_copy_gib * 2 ** 30)
        src = torch.ones(nb, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {nb} bytes read, {nb} bytes written")
        del src, dst
        torch.cuda.empty_cache()

    timer = Timer(sw.stream)
    for s in range(args.warmup):
        sw.one_step(K, s)
        torch.cuda.synchronize()
        log(f"warmup step {s} done")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        sw.one_step(K, args.warmup + s, timer)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    log(f"timed {args.steps} steps in {elapsed:.3f} s")

    sw.fused_step(K, args.warmup + args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        sw.fused_step(K, args.warmup + args.steps + 1 + s, timer)
    torch.cuda.synchronize()
    fused_elapsed = time.perf_counter() - t0
    log(f"timed {args.steps} fused-schedule steps in {fused_elapsed:.3f} s")

    graph_elapsed = None
    if not args.no_graph:
        # The fused step captured once into a HIP graph and replayed: every replay applies the
        # captured step (its probes and coefficients) again, with no host launches in between.
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream(dev)
        side.wait_stream(sw.stream)
        torch.cuda.synchronize()
        sw.cur = side
        with torch.cuda.graph(graph, stream=side):
            sw.fused_step(K, args.warmup + 2 * args.steps + 1)
        sw.cur = sw.stream
        graph.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            graph.replay()
        torch.cuda.synchronize()
        graph_elapsed = time.perf_counter() - t0
        log(f"timed {args.steps} graph replays of the fused step in {graph_elapsed:.3f} s")

    # Plain in-place read-modify-write ceiling of the flat buffer. Not measured for the
    # per-tensor layout, where a plain sweep would need one launch per tensor.
    ceiling = rmw_ceiling(sw, b) if args.layout == "flat" else None
    ceil_gbps = ceiling["gbps"] if ceiling else None
    if ceiling:
        log(f"plain read-modify-write ceiling of this buffer: {ceil_gbps:.1f} GB/s ({ceiling['shape']})")

    ms = timer.ms()
    t_step = elapsed / args.steps
    t_fused = fused_elapsed / args.steps
    sweep_bytes = 2.0 * b * n
    step_gbps = (3 * K + 1) * sweep_bytes / t_step / 1e9
    counters = measured_counters(w.name, K, w.dtype, args.layout)
    per_call = (f"one call covers {sw.n_tensors} tensors in {-(-sw.n_tensors // 64)} launches; times are per call"
                if args.layout == "tensors" else None)
    roof = {k: roofline(k, ms[k], n, b, K, counters, ceil_gbps, per_call)
            for k in ("zo_update", "zo_update_restore", "zo_perturb", "zo_perturb2") if k in ms}
    upd = roof["zo_update"]
    n_tensors = sw.n_tensors
    del sw
    torch.cuda.empty_cache()

    out = {
        "metric": METRIC,
        "value": upd["achieved"] if upd["unit"] == "GB/s" else round(sweep_bytes / (upd["median_ms"] * 1e-3) / 1e9, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_step * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded OPT-shaped weights ~N(0,0.02), losses ~N(2.0,0.05))",
        "config": {"workload": (f"{w.name}-shaped flat {w.dtype} parameter set, fused update inside full "
                                f"1.5-SPSA steps" if args.layout == "flat" else
                                f"{w.name}-shaped {w.dtype} parameter set as {n_tensors} separately allocated "
                                f"tensors, fused update inside full 1.5-SPSA steps"),
                   "layout": args.layout, "n_tensors": n_tensors,
                   "n_params": n, "K": K, "eps": w.eps, "lr": w.lr, "sweeps_per_step": 3 * K + 1,
                   "parallelism": "single GPU"},
        "value_is": "zo_update: algorithmic bytes (2 x bytes of the weights) / median launch duration "
                    f"over the {args.steps} timed steps",
        "update_gbps": round(sweep_bytes / (upd["median_ms"] * 1e-3) / 1e9, 1),
        "update_params_probes_per_s": upd["params_probes_per_s"],
        "update_restore_gbps": round(sweep_bytes / (roof["zo_update_restore"]["median_ms"] * 1e-3) / 1e9, 1),
        "perturb_gbps": round(sweep_bytes / (roof["zo_perturb"]["median_ms"] * 1e-3) / 1e9, 1),
        "step_gbps": round(step_gbps, 1),
        "step_params_probes_per_s": float(f"{n * 4 * K / t_step:.4e}"),
        "roofline": upd,
        "roofline_update_restore": roof["zo_update_restore"],
        "roofline_perturb": roof["zo_perturb"],
        "roofline_perturb2": roof.get("zo_perturb2"),
        "rmw_ceiling": None if ceiling is None else {**ceiling, "step_frac_of_ceiling": round(step_gbps / ceil_gbps, 4)},
        "fused_schedule": {
            "ms_per_step": round(t_fused * 1e3, 3),
            "sweeps_per_step": 2 * K + 1,
            "effective_gbps": round((2 * K + 1) * sweep_bytes / t_fused / 1e9, 1),
            "speedup_vs_sequential": round(elapsed / fused_elapsed, 3),
            "step_params_probes_per_s": float(f"{n * 4 * K / t_fused:.4e}"),
        },
        "graph_fused_schedule": None if graph_elapsed is None else {
            "ms_per_step": round(graph_elapsed / args.steps * 1e3, 3),
            "effective_gbps": round((2 * K + 1) * sweep_bytes / (graph_elapsed / args.steps) / 1e9, 1),
            "speedup_vs_eager_fused": round(fused_elapsed / graph_elapsed, 3),
            "how": "the fused step captured once into a HIP graph (torch.cuda.CUDAGraph) and replayed; "
                   "each replay re-applies the captured step",
        },
    }
    if run_opt30b:
        out["opt30b"] = opt30b_legs(dev)
    out.update(baselines)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
