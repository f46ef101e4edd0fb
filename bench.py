"""Benchmark: one 1.5-SPSA step of probe regenerate-and-apply sweeps on one MI355X.

A step is Algorithm 1 on one device with the forward passes replaced by synthetic losses:
for each of K probes zo_perturb(+eps), zo_perturb(-2 eps), zo_perturb(+eps); then
zo_probe_coeffs on the host; then one fused zo_update. Weights are one flat bf16 buffer
shaped like OPT-13B (12,853,473,280 parameters, ~N(0, 0.02)), resident in HBM before the
timed region starts; K = 16, eps = lr = 1e-3.

Prints one JSON line. `value` is the step's effective HBM bandwidth: algorithmic bytes
(one read and one write of every weight per sweep, 3K + 1 sweeps) over the step time.
`fused_schedule` times the same step in 2K + 1 sweeps (zo_perturb2 merges the restore of
probe k with the +eps of probe k + 1, zo_update_restore merges the last restore with the
update) over the same number of steps.
`graph_fused_schedule` replays the fused step captured once into a HIP graph (no host
launches between kernels; each replay re-applies the captured step).
Per-kernel durations come from HIP events recorded around every launch on the stream the
kernels run on; `roofline` is the dominant kernel's (zo_perturb: 3K of the 3K + 1 sweeps)
and `roofline_update` the fused update's.
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


def measured_counters(workload, K, dtype, layout="flat"):
    """Per-launch HBM bytes (FETCH_SIZE and WRITE_SIZE, each scaled by a plain copy of known
    size) and VALU instruction counts (SQ_INSTS_VALU) from the committed rocprofv3 summaries,
    keyed by kernel; {} when none matches this workload or the sweep source has changed since
    the counters were taken."""
    import glob
    import hashlib
    src = os.path.join(ROOT, "paper_2609_38095_amd", "csrc", "zo_sweep.hip")
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
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


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="opt13b", choices=sorted(workloads_names()),
                    help="tiny, opt125m, opt1.3b, opt13b, opt30b, qwen3-1.7b or qwen3-8b")
    ap.add_argument("--K", type=int, default=0, help="probes per step (default: the workload's first)")
    ap.add_argument("--layout", default="flat", choices=["flat", "tensors"],
                    help="flat: one contiguous buffer (zo_perturb, zo_update); tensors: every OPT tensor "
                         "allocated separately, swept with zo_perturb_segments / zo_update_segments")
    ap.add_argument("--no-cpu-baseline", action="store_true")
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
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    dev = torch.device("cuda:0")
    zo.library()
    log(f"workload {w.name}: n={n} dtype={w.dtype} K={K} eps={w.eps} lr={w.lr}; {n * b / 1e9:.2f} GB of weights")

    seed = 2024
    stream = torch.cuda.current_stream(dev)
    cur = {"s": stream}  # the stream the sweeps are issued on (the capture stream while capturing)
    if args.layout == "flat":
        theta = torch.empty(n, dtype=dt, device=dev)
        if w.hidden:
            workloads.fill_model_buffer_device(theta, w)
        else:
            theta.copy_(torch.from_numpy(workloads.tiny_theta(n)))
        n_tensors = 1
        perturb = lambda k, e, step: zo.zo_perturb(theta, k, e, seed, step, stream=cur["s"])
        perturb2 = lambda ka, ea, kb, eb, step: zo.zo_perturb2(theta, ka, ea, kb, eb, seed, step, stream=cur["s"])
        update = lambda c, step: zo.zo_update(theta, c, w.lr, seed, step, stream=cur["s"])
        update_restore = lambda c, step, kr, er: zo.zo_update_restore(theta, c, w.lr, seed, step, kr, er,
                                                                      stream=cur["s"])
    else:
        spans = workloads.tensor_offsets(w)
        tensors = [torch.empty(sz, dtype=dt, device=dev) for _, _, sz in spans]
        offs = [o for _, o, _ in spans]
        workloads.fill_model_tensors_device(tensors, w)
        n_tensors = len(tensors)
        perturb = lambda k, e, step: zo.zo_perturb_segments(tensors, offs, k, e, 0, 0.0, seed, step,
                                                            stream=cur["s"])
        perturb2 = lambda ka, ea, kb, eb, step: zo.zo_perturb_segments(tensors, offs, ka, ea, kb, eb, seed, step,
                                                                       stream=cur["s"])
        update = lambda c, step: zo.zo_update_segments(tensors, offs, c, w.lr, seed, step, stream=cur["s"])
        update_restore = lambda c, step, kr, er: zo.zo_update_segments(tensors, offs, c, w.lr, seed, step, kr, er,
                                                                       stream=cur["s"])
        log(f"per-tensor layout: {n_tensors} separately allocated tensors")
    torch.cuda.synchronize()
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

    ev = {"perturb": [], "update": []}

    def timed(kind, fn):
        a = torch.cuda.Event(enable_timing=True)
        z = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        fn()
        z.record(stream)
        ev[kind].append((a, z))

    def one_step(step, record):
        lp, lm, l0 = workloads.synthetic_losses(K, step)
        for k in range(K):
            for e in (w.eps, -2.0 * w.eps, w.eps):
                if record:
                    timed("perturb", lambda: perturb(k, e, step))
                else:
                    perturb(k, e, step)
        c = zo.zo_probe_coeffs(lp, lm, l0, w.eps)
        if record:
            timed("update", lambda: update(c, step))
        else:
            update(c, step)

    def fused_step(step):
        lp, lm, l0 = workloads.synthetic_losses(K, step)
        perturb(0, w.eps, step)
        for k in range(K):
            perturb(k, -2.0 * w.eps, step)
            if k + 1 < K:
                perturb2(k, w.eps, k + 1, w.eps, step)
        c = zo.zo_probe_coeffs(lp, lm, l0, w.eps)
        update_restore(c, step, K - 1, w.eps)

    for s in range(args.warmup):
        one_step(s, False)
        torch.cuda.synchronize()
        log(f"warmup step {s} done")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        one_step(args.warmup + s, True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    log(f"timed {args.steps} steps in {elapsed:.3f} s")

    fused_step(args.warmup + args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        fused_step(args.warmup + args.steps + 1 + s)
    torch.cuda.synchronize()
    fused_elapsed = time.perf_counter() - t0
    log(f"timed {args.steps} fused-schedule steps in {fused_elapsed:.3f} s")

    # The fused step captured once into a HIP graph and replayed: every replay applies the
    # captured step (its probes and coefficients) again, with no host launches in between.
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream(dev)
    side.wait_stream(stream)
    torch.cuda.synchronize()
    cur["s"] = side
    with torch.cuda.graph(graph, stream=side):
        fused_step(args.warmup + 2 * args.steps + 1)
    cur["s"] = stream
    graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    graph_elapsed = time.perf_counter() - t0
    log(f"timed {args.steps} graph replays of the fused step in {graph_elapsed:.3f} s")

    # Plain in-place read-modify-write ceiling of the flat buffer (an even number of XOR passes
    # leaves the weights as they were). Not measured for the per-tensor layout, where a plain
    # sweep would need one launch per tensor.
    ceil_gbps = ceil_ms = None
    ceil_launches = 6
    if args.layout == "flat":
        import ctypes
        calib = ctypes.CDLL(os.path.join(os.path.dirname(zo.LIB_PATH), "libzo_calib.so"))
        calib.zo_calib_rmw.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p]
        sptr = ctypes.c_void_p(stream.cuda_stream)
        buf_bytes = n * b - (n * b) % 16

        def rmw():
            rc = calib.zo_calib_rmw(ctypes.c_void_p(theta.data_ptr()), buf_bytes, 0x5A5A5A5A, sptr)
            if rc != 0:
                raise RuntimeError(f"zo_calib_rmw failed ({rc})")

        rmw()
        rmw()
        ceil_ev = []
        for _ in range(ceil_launches):
            a = torch.cuda.Event(enable_timing=True)
            z = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            rmw()
            z.record(stream)
            ceil_ev.append((a, z))
        torch.cuda.synchronize()
        ceil_ms = float(np.mean([a.elapsed_time(z) for a, z in ceil_ev]))
        ceil_gbps = 2.0 * buf_bytes / (ceil_ms * 1e-3) / 1e9
        log(f"plain read-modify-write ceiling of this buffer: {ceil_gbps:.1f} GB/s")

    ms = {k: np.array([a.elapsed_time(z) for a, z in v]) for k, v in ev.items()}
    t_step = elapsed / args.steps
    sweep_bytes = 2.0 * b * n
    step_bytes = (3 * K + 1) * sweep_bytes
    gbps = step_bytes / t_step / 1e9
    p_ms, u_ms = float(ms["perturb"].mean()), float(ms["update"].mean())
    p_gbps, u_gbps = sweep_bytes / (p_ms * 1e-3) / 1e9, sweep_bytes / (u_ms * 1e-3) / 1e9

    counters = measured_counters(w.name, K, w.dtype, args.layout)

    def roof(kernel, avg_ms, gb):
        d = ms["perturb" if kernel == "zo_perturb" else "update"]
        hbm_frac = gb / HBM_PEAK_GBPS
        valu = counters.get("valu_instructions_per_launch", {}).get(kernel)
        alu = valu * 64 / (avg_ms * 1e-3) / 1e12 if valu else None
        r = {"kernel": kernel, "bound": "hbm", "achieved": round(gb, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
             "frac": round(hbm_frac, 4), "traffic": counters.get("traffic_bytes_per_launch", {}).get(kernel),
             "avg_ms": round(avg_ms, 4), "min_ms": round(float(d.min()), 4), "max_ms": round(float(d.max()), 4),
             "launches": int(d.size), "bytes_per_launch": sweep_bytes, "hbm_frac": round(hbm_frac, 4),
             "frac_of_rmw_ceiling": round(gb / ceil_gbps, 4) if ceil_gbps else None}
        if args.layout == "tensors":
            r["per_sweep"] = (f"one call covers {n_tensors} tensors in {-(-n_tensors // 64)} launches; "
                              "times are per call")
        # VALU: issued lane-ops against the 2.4 GHz issue peak, and the measured busy share of
        # the CUs' VALU issue capacity at the clock the GPU actually ran (SQ_ACTIVE_INST_VALU)
        valu_busy = counters.get("valu_busy", {}).get(kernel)
        ints = counters.get("int_instructions_per_launch", {}).get(kernel)
        if alu is not None:
            r["valu_tlaneops"] = round(alu, 2)
            r["alu_frac"] = round(alu / VALU_PEAK_TLANEOPS, 4)
        if valu_busy is not None:
            r["valu_busy"] = valu_busy
        if ints is not None:
            it = ints * 64 / (avg_ms * 1e-3) / 1e12
            r["int32_int64_tlaneops"] = round(it, 2)
            r["int32_int64_frac"] = round(it / VALU_PEAK_TLANEOPS, 4)
        lds = counters.get("lds_per_launch", {}).get(kernel)
        lds_busy = lds["lds_busy"] if lds is not None and kernel == "zo_update" else None
        if kernel == "zo_update":
            # one table lookup per element and probe group
            glk = n * ((K + 7) // 8) / (avg_ms * 1e-3) / 1e9
            r["table_glookups_per_s"] = round(glk, 1)
            if lds_busy is not None:
                r["lds_busy"] = lds_busy
        bound = binding_unit(hbm_frac, lds_busy, valu_busy if valu_busy is not None else r.get("alu_frac"))
        if bound == "lds":
            r.update(bound="lds", achieved=round(glk, 1), peak=round(LDS_PEAK_GLOOKUPS, 1),
                     unit="G lookups/s", frac=round(glk / LDS_PEAK_GLOOKUPS, 4),
                     peak_random_index=round(LDS_RANDOM_GLOOKUPS, 1),
                     frac_of_random_index_peak=round(glk / LDS_RANDOM_GLOOKUPS, 4))
        elif bound == "alu":
            r.update(bound="alu", achieved=round(alu, 2), peak=round(VALU_PEAK_TLANEOPS, 2), unit="Tlane-op/s",
                     frac=round(alu / VALU_PEAK_TLANEOPS, 4))
        return r

    out = {
        "metric": METRIC,
        "value": round(gbps, 1),
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
        "config": {"workload": (f"{w.name}-shaped flat {w.dtype} parameter set, full 1.5-SPSA step"
                                if args.layout == "flat" else
                                f"{w.name}-shaped {w.dtype} parameter set as {n_tensors} separately allocated "
                                f"tensors, full 1.5-SPSA step"),
                   "layout": args.layout, "n_tensors": n_tensors,
                   "n_params": n, "K": K, "eps": w.eps, "lr": w.lr, "sweeps_per_step": 3 * K + 1,
                   "parallelism": "single GPU"},
        "update_gbps": round(u_gbps, 1),
        "update_params_probes_per_s": float(f"{n * K / (u_ms * 1e-3):.4e}"),
        "perturb_gbps": round(p_gbps, 1),
        "step_params_probes_per_s": float(f"{n * 4 * K / t_step:.4e}"),
        "roofline": roof("zo_perturb", p_ms, p_gbps),
        "roofline_update": roof("zo_update", u_ms, u_gbps),
        "rmw_ceiling": None if ceil_gbps is None else {
            "gbps": round(ceil_gbps, 1), "avg_ms": round(ceil_ms, 4), "launches": ceil_launches,
            "kernel": "plain in-place 16-byte XOR sweep of the same buffer (libzo_calib.so), "
                      "same memory shape as the sweeps, no probe work",
            "step_frac_of_ceiling": round(gbps / ceil_gbps, 4)},
        "fused_schedule": {
            "ms_per_step": round(fused_elapsed / args.steps * 1e3, 3),
            "sweeps_per_step": 2 * K + 1,
            "effective_gbps": round((2 * K + 1) * sweep_bytes / (fused_elapsed / args.steps) / 1e9, 1),
            "speedup_vs_sequential": round(elapsed / fused_elapsed, 3),
            "step_params_probes_per_s": float(f"{n * 4 * K / (fused_elapsed / args.steps):.4e}"),
        },
        "graph_fused_schedule": {
            "ms_per_step": round(graph_elapsed / args.steps * 1e3, 3),
            "effective_gbps": round((2 * K + 1) * sweep_bytes / (graph_elapsed / args.steps) / 1e9, 1),
            "speedup_vs_eager_fused": round(fused_elapsed / graph_elapsed, 3),
            "how": "the fused step captured once into a HIP graph (torch.cuda.CUDAGraph) and replayed; "
                   "each replay re-applies the captured step",
        },
    }
    out.update(baselines)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
