"""Benchmark of one training step of a workload on one MI355X.

A step of a dense workload (c1-c5) is one ``dlvm_gradient`` call (the forward
recomputed from the original inputs, then the whole adjoint) followed, for
workloads with an SGD update, by one ``dlvm_sgd_step`` call. A step of a
recurrent workload (r1) is ``dlvm_rnn_forward`` over its T steps,
``dlvm_rnn_backward`` seeded with fixed output adjoints, and the update. Inputs
are seeded, synthetic and resident in device memory before the timed region
starts.

Prints one JSON line. ``value`` is steps per second of the whole job on one
GPU. ``roofline`` describes the kernel that takes the most time in a step: its
algorithmic flops (or bytes) per launch, divided by its average launch
duration measured with HIP events on the launch stream during the timed steps.
``cpu_baseline`` times the float64 oracle on the host cores on a bounded sample
of the same workload.

With no --workload the step is the deep bf16 network's training step (c5:
4096 -> 8 x 4096 relu -> 1000, softmax cross-entropy, batch 16384, gradient and
fused SGD), the largest configuration of the metric; the others are selected
with --workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c5]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads  # noqa: E402

METRIC = "MLP fwd+grad steps/s, TFLOP/s (% MFMA peak); fused elementwise GB/s"
# MI355X published peaks: dense MFMA per dtype, and HBM3E bandwidth.
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}
PEAK_HBM_GBS = 8000.0
PEAK_VALU_F32_TFLOPS = 157.3  # float32 vector FMA rate of the whole chip


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default="c5",
                    choices=sorted(workloads.WORKLOADS) + sorted(workloads.RNN_WORKLOADS) +
                    sorted(workloads.CHAIN_WORKLOADS) + ["ce5"])
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="budget of the oracle CPU baseline (0 disables it)")
    ap.add_argument("--entry", default="gradient", choices=["gradient", "vjp"],
                    help="gradient: dlvm_gradient (+ dlvm_sgd_step); vjp: the seedable gradient "
                         "of the logits (dlvm_vjp) with a fixed random seed, timed on its own "
                         "(no per-launch roofline)")
    ap.add_argument("--graph", action="store_true",
                    help="replay a captured step graph instead of enqueueing every step's "
                         "launches from the host")
    ap.add_argument("--checkpoint", type=int, default=1, metavar="K",
                    help="keep only every K-th hidden layer output and recompute the rest in "
                         "the adjoint sweep (1: keep all); the rate still counts the "
                         "algorithmic flops only")
    ap.add_argument("--chain-in-epilogue", action="store_true",
                    help="c4: run the eight-operator chain in the dense product's epilogue "
                         "instead of the standalone chain kernel")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (5 times) and exit: the "
                         "reference kernel for scaling the FETCH_SIZE / WRITE_SIZE counters")
    return ap.parse_args()


def kernel_source_hash() -> str:
    """Hash of the library's device sources, the .hip and .hpp files (a traffic
    record is valid only for them; the host planner's choices are part of the
    launch name a record is matched on)."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1711_03016_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if not name.endswith((".hip", ".hpp")):
            continue
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def traffic_record(workload: str, dom: dict) -> float | None:
    """HBM bytes per launch of the dominant kernel, from a committed counter summary.

    profiles/*.md may hold a line ``TRAFFIC_RECORD {json}`` written from two
    rocprofv3 --pmc passes (FETCH_SIZE, WRITE_SIZE) scaled by the same counters
    on a plain copy of known size. It is used only when its workload, launch
    name and shape match and it was taken on the current kernel sources.
    """
    pdir = os.path.join(ROOT, "profiles")
    if not os.path.isdir(pdir):
        return None
    want = kernel_source_hash()
    for name in sorted(os.listdir(pdir)):
        if not name.endswith(".md"):
            continue
        with open(os.path.join(pdir, name)) as f:
            for line in f:
                if not line.startswith("TRAFFIC_RECORD "):
                    continue
                r = json.loads(line[len("TRAFFIC_RECORD "):])
                if (r.get("workload") == workload and r.get("kernel") == dom["name"]
                        and [r.get("M"), r.get("N"), r.get("K")] == [dom["M"], dom["N"], dom["K"]]
                        and r.get("source_hash") == want):
                    return float(r["bytes_per_launch"])
    return None


def copy_calibration(mib: int) -> None:
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 5}))


def default_steps(wl) -> tuple[int, int]:
    flops = wl.flops()
    if flops > 1e12:
        return 30, 5
    if flops > 1e10:
        return 200, 20
    return 2000, 100


def host_facts() -> dict:
    """What the oracle baseline ran on: logical CPUs, the cores this process
    may run on (affinity mask) and the CPU model."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "affinity_cores": len(os.sched_getaffinity(0)),
            "cpu_model": model}


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        return max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - threadpoolctl is optional
        return os.cpu_count() or 1


def single_thread(fn):
    """Run fn() with the BLAS limited to one thread and the calling thread
    pinned to one core of the affinity mask."""
    from threadpoolctl import threadpool_limits
    old = os.sched_getaffinity(0)
    os.sched_setaffinity(0, {min(old)})
    try:
        with threadpool_limits(limits=1):
            return fn()
    finally:
        os.sched_setaffinity(0, old)


def cpu_baseline(wl, budget_s: float) -> dict | None:
    """Time the oracle (as it stands) on the host on a bounded sample: with
    the BLAS on all its threads, then on one thread pinned to one core.

    A workload whose whole batch is cheap is timed at full size. Otherwise
    the gradient is timed on a rows and on b = 4a, 16a, ... rows of the batch
    (after one untimed call), b growing until the rows' share of the time is
    at least half the time on a rows or the budget is spent, and the time is
    fitted through the two as fixed + per_row * rows (the fixed part, e.g.
    rounding every parameter to bf16, does not grow with the rows; every
    product does) and evaluated at the full batch; the update is timed once
    as it is (it does not depend on the rows)."""
    if budget_s <= 0:
        return None
    import oracle
    spec = oracle.MlpSpec(wl.widths, wl.acts, wl.loss, wl.dtype)

    def update(params, grads):
        for (W, b), (dW, db) in zip(params, grads):
            oracle.sgd_f32(W, dW, wl.lr)
            oracle.sgd_f32(b, db, wl.lr)

    def run(cap_flops: float, budget: float):
        if wl.flops(wl.batch) <= cap_flops:
            x, params, y = workloads.make_inputs(wl)
            n, el = 0, 0.0
            while True:
                t0 = time.perf_counter()
                _, grads, _ = oracle.mlp_gradient(spec, x, params, y, wrt_x=wl.wrt_x)
                if wl.sgd:
                    update(params, grads)
                el += time.perf_counter() - t0
                n += 1
                if el >= budget or el * (n + 1) / n > 2 * budget:
                    break
            return n / el, (f"{n} oracle steps (float64 gradient{' + SGD' if wl.sgd else ''}) "
                            f"on the whole batch of {wl.batch} rows in {el:.1f} s")
        a = wl.batch
        while a > 1 and wl.flops(2 * a) > cap_flops:
            a //= 2
        x, params, y = workloads.make_inputs(wl, batch=wl.batch)

        def timed(rows):
            t0 = time.perf_counter()
            _, g, _ = oracle.mlp_gradient(spec, x[:rows], params, y[:rows], wrt_x=wl.wrt_x)
            return time.perf_counter() - t0, g

        # one untimed call first: the first touch of the oracle's large
        # temporaries (every parameter in float64) costs several times a step
        t0 = time.perf_counter()
        timed(a)
        spent = time.perf_counter() - t0
        ta, grads = timed(a)
        spent += ta
        b, tb = a, ta
        while 4 * b <= wl.batch:
            nb = 4 * b
            per_row_est = max((tb - ta) / (b - a), 0.0) if b > a else 0.0
            est = ta + (nb - a) * per_row_est
            if b > a and spent + est > budget:
                break
            b = nb
            tb, grads = timed(b)
            spent += tb
            if tb - ta >= 0.5 * ta:
                break
        per_row = max((tb - ta) / (b - a), 0.0) if b > a else 0.0
        fixed = max(ta - per_row * a, 0.0)
        t_sgd = 0.0
        if wl.sgd:
            t0 = time.perf_counter()
            update(params, grads)
            t_sgd = time.perf_counter() - t0
        per_step = fixed + per_row * wl.batch + t_sgd
        sample = (f"float64 oracle gradient on {a} rows ({ta:.2f} s) and {b} rows "
                  f"({tb:.2f} s) of the {wl.batch}, fitted as {fixed:.2f} s + "
                  f"{per_row * 1e3:.3f} ms per row and evaluated at {wl.batch} rows"
                  + (f", plus one SGD update over all parameters ({t_sgd:.2f} s)" if wl.sgd else ""))
        return 1.0 / per_step, sample

    threads = blas_threads()
    value, sample = run(1.1e11, budget_s / 2)
    one_value, one_sample = single_thread(lambda: run(2.6e10, budget_s / 2))
    return {"value": value, "unit": "steps/s", "cores": int(threads), "kind": "oracle",
            "sample": sample,
            "single_thread": {"value": one_value, "unit": "steps/s", "cores": 1,
                              "sample": one_sample + "; BLAS limited to one thread, pinned "
                                                     "to one core"},
            "host": host_facts()}


def vjp_bench(args, wl, m, P, xd, dP, dx, ws, stream, steps, warmup):
    """Steps of the seedable gradient of the logits (dlvm_vjp) only."""
    import torch
    if wl.loss != "softmax_ce":
        raise SystemExit("--entry vjp needs a softmax workload")
    B, C = wl.batch, wl.widths[-1]
    g = torch.Generator(device="cpu").manual_seed(7)
    seed = (torch.randn((B, C), generator=g) / B).to("cuda:0")
    for _ in range(warmup):
        m.vjp(P, xd, seed, B, dP, dx, ws, stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        m.vjp(P, xd, seed, B, dP, dx, ws, stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    sps = steps / elapsed
    # the output layer's own product is dead in the seedable gradient
    flops = wl.flops() - 2 * B * wl.widths[-2] * C
    print(json.dumps({"metric": METRIC, "entry": "vjp", "value": round(sps, 3), "unit": "steps/s",
                      "n_gpus": 1, "steps": steps, "warmup": warmup,
                      "ms_per_step": round(elapsed / steps * 1e3, 4), "higher_is_better": True,
                      "dtype": wl.dtype, "data": "synthetic",
                      "config": {"workload": f"{wl.name}: {wl.title}", "global_batch": B},
                      "tflops": round(flops * sps / 1e12, 3),
                      "mfma_frac": round(flops * sps / 1e12 / PEAK_TFLOPS[wl.dtype], 4)}), flush=True)


def measure(m, wl, step, eager_step, steps, warmup, with_sgd, flags_ws=None,
            bound_by_intensity=False):
    """Warm up, find the launch position that takes the most time, time `steps`
    whole steps, then time the dominant launch on its stream over as many steps.

    Returns (steps/s, seconds, roofline dict, per-group microseconds per step).
    """
    import torch

    import paper_1711_03016_amd as dl

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    if flags_ws is not None and m.check(flags_ws) != dl.OK:
        raise RuntimeError("device flags raised during warm-up")

    # find the launch that takes the most time (outside the timed region)
    B = getattr(wl, "batch", 1)
    plan = m.plan(B)
    if not with_sgd:
        plan = plan[:-1]
    probe_steps = 20  # (a few steps let one slow dispatch pick the wrong launch)
    m.probe_arm(-1, probe_steps * len(plan) + 8)
    for _ in range(probe_steps):
        eager_step()
    torch.cuda.synchronize()
    times = []
    for e in plan:
        n, ms = m.probe_read(e["index"])
        times.append(ms / max(n, 1))
    dom = plan[int(np.argmax(times))]
    m.probe_disarm()
    groups: dict = {}
    for e, ms in zip(plan, times):
        key = e["name"].split(" ")[0]
        groups[key] = round(groups.get(key, 0.0) + ms * 1e3, 2)

    # timed region: whole steps, nothing else on the stream
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    sps = steps / elapsed

    # the same number of steps again, the dominant launch timed by events that
    # its own dispatch packet records on its stream (begin and end on the GPU)
    m.probe_arm(dom["index"], steps)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(steps):
        eager_step()
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    n_dom, ms_dom = m.probe_read(dom["index"])
    m.probe_disarm()
    avg_s = ms_dom / max(n_dom, 1) / 1e3

    ridge = PEAK_TFLOPS[wl.dtype] * 1e12 / (PEAK_HBM_GBS * 1e9)  # flop per byte
    mfma = dom["flops"] > 0 and (not bound_by_intensity or dom["flops"] >= ridge * dom["bytes"])
    if dom["name"].startswith("small_step"):
        # one workgroup of plain float32 fused multiply-adds (no matrix cores):
        # priced against the chip's float32 vector rate (256 CUs x 2.4 GHz)
        achieved = dom["flops"] / avg_s / 1e12
        roof = {"bound": "alu", "achieved": round(achieved, 4), "peak": PEAK_VALU_F32_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_VALU_F32_TFLOPS, 6)}
    elif mfma:
        achieved = dom["flops"] / avg_s / 1e12
        peak = PEAK_TFLOPS[wl.dtype]
        roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak,
                "unit": "TFLOP/s", "frac": round(achieved / peak, 4)}
    else:
        achieved = dom["bytes"] / avg_s / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof["traffic"] = traffic_record(wl.name, dom)
    roof["kernel"] = (f"{dom['name']} M={dom['M']} N={dom['N']} K={dom['K']} "
                      f"(launch {dom['index']} of {len(plan)}, {n_dom} timed launches, "
                      f"avg {avg_s * 1e6:.2f} us)")
    roof["probe_ms_per_step"] = round((t3 - t2) / steps * 1e3, 4)
    return sps, elapsed, roof, groups


def result_line(wl, sps, elapsed, steps, warmup, roof, config, step_flops=None, **extra) -> dict:
    tflops = (wl.flops() if step_flops is None else step_flops) * sps / 1e12
    out = {
        "metric": METRIC,
        "value": round(sps, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(elapsed / steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": config,
    }
    out.update(extra)
    out["tflops"] = round(tflops, 3)
    out["mfma_frac"] = round(tflops / PEAK_TFLOPS[wl.dtype], 4)
    out["roofline"] = roof
    return out


def rnn_main(args, wl) -> None:
    """A step of a recurrent workload: dlvm_rnn_forward over the T steps,
    dlvm_rnn_backward seeded with fixed output adjoints, and the fused SGD."""
    import torch

    import paper_1711_03016_amd as dl

    steps, warmup = default_steps(wl)
    steps = args.steps if args.steps is not None else steps
    warmup = args.warmup if args.warmup is not None else warmup
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    tdt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    B, T, Kx, H = wl.batch, wl.steps, wl.in_width, wl.hidden
    xs, h0, W, U, b, dhs = workloads.make_rnn_inputs(wl)
    m = dl.Rnn(T, Kx, H, wl.act, wl.dtype, wl.wrt_x, wl.wrt_h0, B)
    P = m.pack_cell(W, U, b, dev, tdt)
    master = m.pack_cell(W, U, b, dev, torch.float32) if wl.dtype == "bf16" else None
    xd = torch.from_numpy(xs).to(dev).to(tdt)
    hs = torch.empty((T + 1, B, H), dtype=tdt, device=dev)
    hs[0] = torch.from_numpy(h0).to(dev).to(tdt)
    dhd = torch.from_numpy(dhs).to(dev).to(tdt)
    del xs, dhs
    dP = torch.empty(m.param_count(), device=dev)
    dxs = torch.empty((T, B, Kx), device=dev) if wl.wrt_x else None
    dh0 = torch.empty((B, H), device=dev) if wl.wrt_h0 else None
    ws = torch.empty(m.workspace_bytes(B), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        m.forward(P, xd, B, hs, ws, stream)
        m.backward(P, xd, hs, dhd, B, dP, dxs, dh0, ws, stream)
        if wl.sgd:
            m.sgd_step(P, master, dP, wl.lr, stream)

    sps, elapsed, roof, groups = measure(m, wl, step, step, steps, warmup, wl.sgd)
    config = {"workload": f"{wl.name}: {wl.title}", "global_batch": B, "steps_T": T,
              "in_width": Kx, "hidden": H, "act": wl.act, "parallelism": "none"}
    out = result_line(wl, sps, elapsed, steps, warmup, roof, config, launch="eager",
                      workspace_bytes=int(ws.numel()), launch_groups_us=groups)
    del P, master, xd, hs, dhd, ws, dP, dxs, dh0
    out["cpu_baseline"] = rnn_cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def rnn_cpu_baseline(wl, budget_s: float) -> dict | None:
    """The oracle's forward + seedable gradient (+ SGD) on a slice of the rows."""
    if budget_s <= 0:
        return None
    import oracle
    threads = blas_threads()
    rows = wl.batch
    while rows > 4 and wl.flops(rows) > 4e10:
        rows //= 2
    xs, h0, W, U, b, dhs = workloads.make_rnn_inputs(wl, batch=rows)
    spec = oracle.RnnSpec(wl.steps, wl.in_width, wl.hidden, wl.act, wl.dtype)
    n = 0
    t_grad = t_sgd = 0.0
    while True:
        t0 = time.perf_counter()
        oracle.rnn_forward(spec, xs, h0, W, U, b)
        dW, dU, db, _, _ = oracle.rnn_vjp(spec, xs, h0, W, U, b, dhs, wl.wrt_x, wl.wrt_h0)
        t1 = time.perf_counter()
        if wl.sgd:
            for p_, g_ in ((W, dW), (U, dU), (b, db)):
                oracle.sgd_f32(p_, g_, wl.lr)
        t2 = time.perf_counter()
        t_grad += t1 - t0
        t_sgd += t2 - t1
        n += 1
        el = t_grad + t_sgd
        if el >= budget_s or el * (n + 1) / n > 2 * budget_s:
            break
    per_step = (t_grad / n) * (wl.batch / rows) + t_sgd / n
    sample = (f"{n} oracle steps (float64 forward + seedable gradient"
              f"{' + SGD' if wl.sgd else ''}) on {rows} of {wl.batch} rows in {el:.1f} s")
    if rows != wl.batch:
        sample += (f"; forward and gradient time scaled by {wl.batch}/{rows} rows (linear in "
                   "the rows), update time taken as measured")
    return {"value": 1.0 / per_step, "unit": "steps/s", "cores": int(threads),
            "kind": "oracle", "sample": sample, "host": host_facts()}


def chain_main(args, wl) -> None:
    """A step of a chain workload: one dlvm_chain_run of the chain in its
    optimal order. Also timed: the same chain left to right (what it costs
    without reordering)."""
    import torch

    import paper_1711_03016_amd as dl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    tdt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    dims, n = list(wl.dims), wl.n
    mats = [torch.from_numpy(a).to(dev).to(tdt).contiguous() for a in workloads.make_chain_inputs(dims)]
    out = torch.empty((dims[0], dims[-1]), device=dev)
    cost, split = dl.chain_order(dims)
    l2r = [[(j - 1 if j > i else -1) for j in range(n)] for i in range(n)]
    l2r_cost = sum(dims[0] * dims[k + 1] * dims[k + 2] for k in range(n - 1))
    m = dl.Chain(wl.dtype, dims)
    m_l2r = dl.Chain(wl.dtype, dims, l2r)
    ws = torch.empty(max(m.workspace_bytes(1), m_l2r.workspace_bytes(1)), dtype=torch.uint8,
                     device=dev)
    steps = args.steps if args.steps is not None else 200
    warmup = args.warmup if args.warmup is not None else 20
    stream = torch.cuda.current_stream()

    def step():
        m.run(mats, out, ws, stream)

    def step_l2r():
        m_l2r.run(mats, out, ws, stream)

    for _ in range(warmup):
        step_l2r()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step_l2r()
    torch.cuda.synchronize()
    elapsed_l2r = time.perf_counter() - t0

    sps, elapsed, roof, groups = measure(m, wl, step, step, steps, warmup, False,
                                         bound_by_intensity=True)
    config = {"workload": f"{wl.name}: {wl.title}", "dims": dims,
              "order": oracle_free_order(split), "parallelism": "none"}
    out_line = result_line(wl, sps, elapsed, steps, warmup, roof, config, step_flops=2 * cost,
                           launch="eager",
                           workspace_bytes=int(ws.numel()), launch_groups_us=groups,
                           multiply_adds=cost, left_to_right_multiply_adds=l2r_cost,
                           left_to_right_steps_per_s=round(steps / elapsed_l2r, 3))
    del mats, out, ws
    out_line["cpu_baseline"] = chain_cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out_line), flush=True)


def oracle_free_order(split, i=0, j=None) -> str:
    """The order of a split table as text (written here so that the timed
    path does not need the oracle)."""
    if j is None:
        j = len(split) - 1
    if i == j:
        return f"A{i}"
    k = split[i][j]
    return "(" + oracle_free_order(split, i, k) + oracle_free_order(split, k + 1, j) + ")"


def chain_cpu_baseline(wl, budget_s: float) -> dict | None:
    """The oracle's chain product (float64, left to right as it stands) on the
    first rows of A_0; the work is linear in those rows."""
    if budget_s <= 0:
        return None
    import oracle
    threads = blas_threads()
    mats = workloads.make_chain_inputs(wl.dims)
    rows = wl.dims[0]
    while rows > 16 and rows * sum(wl.dims[k + 1] * wl.dims[k + 2] for k in range(wl.n - 1)) > 2e9:
        rows //= 2
    sample = [mats[0][:rows]] + mats[1:]
    n, el = 0, 0.0
    while True:
        t0 = time.perf_counter()
        oracle.chain_product(sample, wl.dtype)
        el += time.perf_counter() - t0
        n += 1
        if el >= budget_s or el * (n + 1) / n > 2 * budget_s:
            break
    per = el / n * wl.dims[0] / rows
    return {"value": 1.0 / per, "unit": "steps/s", "cores": int(threads), "kind": "oracle",
            "host": host_facts(), "sample": f"{n} oracle chain products (float64, left to right) on {rows} of "
                      f"{wl.dims[0]} rows of A_0 in {el:.1f} s, scaled by {wl.dims[0]}/{rows}"}


def ce_main(args) -> None:
    """The loss step of the deep bf16 network on its own: softmax
    cross-entropy of 16384 x 1000 float32 logits with bf16 dlogits and the
    loss (dlvm_softmax_xent: the loss kernel, then the one-block loss
    finalisation). Its algorithmic bytes, 98,369,536 per call (logits read,
    dlogits written, labels read), fit the 256 MB Infinity Cache, so the calls
    rotate over 8 sets of logits and dlogits (786 MB together): each call
    reads logits that the previous 7 calls have pushed out of the cache, and
    the rate is that of HBM. The same calls on one resident set are timed
    beside it."""
    import torch

    import paper_1711_03016_amd as dl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    rows, C, R = 16384, 1000, 8
    g = torch.Generator(device="cpu").manual_seed(5)
    logits = [(torch.randn((rows, C), generator=g) * 3).to(dev) for _ in range(R)]
    labels = torch.randint(0, C, (rows,), generator=g, dtype=torch.int32).to(dev)
    dz = [torch.empty((rows, C), dtype=torch.bfloat16, device=dev) for _ in range(R)]
    ws = torch.zeros(dl.softmax_xent_ws_bytes(rows), dtype=torch.uint8, device=dev)
    loss = torch.empty(1, device=dev)
    steps = args.steps if args.steps is not None else 200
    warmup = args.warmup if args.warmup is not None else 16
    nbytes = rows * C * (4 + 2) + rows * 4

    def run(n, rotate):
        for i in range(n):
            k = i % R if rotate else 0
            dl.softmax_xent("bf16", rows, C, logits[k], labels, 1.0 / rows, dz[k], loss, ws)

    out = {}
    for rotate in (True, False):
        run(warmup, rotate)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run(steps, rotate)
        e1.record()
        torch.cuda.synchronize()
        out[rotate] = e0.elapsed_time(e1) / steps / 1e3
    t = out[True]
    achieved = nbytes / t / 1e9
    print(json.dumps({
        "metric": "fused softmax cross-entropy GB/s (logits from HBM)", "value": round(achieved, 1),
        "unit": "GB/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": round(t * 1e3, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "ce5: softmax cross-entropy of 16384 x 1000 float32 logits, bf16 "
                               "dlogits, 8 rotated buffers", "rows": rows, "classes": C},
        "bytes_per_call": nbytes,
        "resident_ms_per_call": round(out[False] * 1e3, 4),
        "resident_gbs": round(nbytes / out[False] / 1e9, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None,
                     "kernel": "softmax_xent call (loss kernel + one-block finalisation), "
                               "rotated buffers"}}), flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the workloads "
              "here are single-GPU and no multi-GPU path is built", file=sys.stderr)
        sys.exit(2)
    if args.workload == "ce5":
        return ce_main(args)
    if args.workload in workloads.RNN_WORKLOADS:
        return rnn_main(args, workloads.RNN_WORKLOADS[args.workload])
    if args.workload in workloads.CHAIN_WORKLOADS:
        return chain_main(args, workloads.CHAIN_WORKLOADS[args.workload])
    import torch

    import paper_1711_03016_amd as dl

    wl = workloads.WORKLOADS[args.workload]
    steps, warmup = default_steps(wl)
    steps = args.steps if args.steps is not None else steps
    warmup = args.warmup if args.warmup is not None else warmup
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    tdt = torch.float32 if wl.dtype == "f32" else torch.bfloat16

    # inputs, resident in device memory before timing
    x, params, y = workloads.make_inputs(wl)
    B = wl.batch
    m = dl.Model(wl.widths, wl.acts, wl.dtype, wl.loss, wl.wrt_x, B,
                 checkpoint_every=args.checkpoint, chain_in_epilogue=args.chain_in_epilogue)
    P = m.pack(params, dev, tdt)
    master = m.pack(params, dev, torch.float32) if wl.dtype == "bf16" and wl.sgd else None
    del params
    xd = torch.from_numpy(x).to(dev).to(tdt)
    yd = None if y is None else torch.from_numpy(y).to(dev)
    del x
    ws = torch.empty(m.workspace_bytes(B), dtype=torch.uint8, device=dev)
    loss = torch.empty(1, device=dev)
    dP = torch.empty(m.param_count(), device=dev)
    dx = torch.empty((B, wl.widths[0]), device=dev) if wl.wrt_x else None
    stream = torch.cuda.current_stream()

    def eager_step():
        m.gradient(P, xd, yd, B, loss, dP, dx, ws, stream)
        if wl.sgd:
            m.sgd_step(P, master, dP, wl.lr, stream)

    if args.entry == "vjp":
        return vjp_bench(args, wl, m, P, xd, dP, dx, ws, stream, steps, warmup)

    # A step is the same launches either way; with --graph they are captured
    # once into a HIP graph and replayed.
    graph = None if not args.graph else m.step_graph(P, master, xd, yd, B, loss, dP, dx, ws,
                                                 update=wl.sgd, lr=wl.lr)
    step = eager_step if graph is None else (lambda: graph.launch(stream))
    sps, elapsed, roof, groups = measure(m, wl, step, eager_step, steps, warmup, wl.sgd,
                                         flags_ws=ws)
    config = {"workload": f"{wl.name}: {wl.title}", "global_batch": B,
              "widths": list(wl.widths), "loss": wl.loss, "parallelism": "none",
              **({"checkpoint_every": args.checkpoint} if args.checkpoint > 1 else {}),
              **({"chain": "in_epilogue"} if args.chain_in_epilogue and wl.loss == "chain8" else {})}
    out = result_line(wl, sps, elapsed, steps, warmup, roof, config,
                      launch="eager" if graph is None else "hip_graph",
                      workspace_bytes=int(ws.numel()), launch_groups_us=groups)
    del graph, P, master, xd, ws, dP, dx
    out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
