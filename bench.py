"""FrameFT adapter hot-path benchmark (one GPU).

A step is the whole adapter hot path over one batch: forward (y_a) then
backward (dX and dC on the support) of one adapted layer, inputs already in
HBM.  Default workload: Llama-2-7B q_proj (4096 x 4096, frames k = 64,
rho = 64 on both sides, 10,000 coefficients) on 8 x 512 = 4096 bf16 tokens.

Prints ONE JSON line.  `roofline` describes the dominant kernel (the one with
the longest average duration) as algorithmic HBM bytes per launch divided by
its average duration, measured with HIP events recorded around that kernel on
its stream during the timed steps.  `cpu_baseline` times the fp64 oracle on
this machine's host on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E peak, GB/s
METRIC = "FrameFT adapter fwd+bwd tokens/s @Llama-7B shapes; % of HBM roofline"
CSRC = os.path.join(ROOT, "paper_2608_26430_amd", "csrc")


def kernel_hash() -> str:
    """Hash of every library source: identifies the kernels a profile or counter file belongs to."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(T, n, m, nnz, esz):
    """Bytes each kernel must move at minimum (activations once, coefficients once)."""
    fwd = T * esz * (n + m) + 4 * nnz                  # read x, write y_a; read c
    bwd = T * esz * (m + 2 * n) + 4 * nnz              # read g, read x, write dX; read c
    red = 4 * nnz                                       # write dC
    return fwd, bwd, red


_CPU = {}   # oracle inputs shared with the forked CPU-baseline workers


def _oracle_tokens(span):
    """Oracle forward + backward (dX, dC) on tokens [lo, hi) of the benchmark workload, one thread."""
    from threadpoolctl import threadpool_limits
    from oracle import frameft_oracle as O
    lo, hi = span
    c = _CPU
    d = c["data"]
    with threadpool_limits(limits=1):
        O.adapter_fwd(c["P_in"], c["P_out"], d.rows, d.cols, d.vals, d.scale, d.X[lo:hi])
        _, dc = O.adapter_bwd(c["P_in"], c["P_out"], d.rows, d.cols, d.vals, d.scale, d.X[lo:hi], d.G[lo:hi])
    return dc


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, ad, data, budget_s=12.0):
    """The fp64 oracle's forward + backward on the benchmark workload, on the host cores.

    Runs before anything touches the GPU, so that worker processes can be forked.  The tokens are
    split over one single-threaded worker process per core (at most 16, the host share of one
    GPU); each runs the oracle unchanged on its share, and the dC parts are summed.  The sample is
    the whole token batch, repeated while the budget allows; a single-thread figure on a prefix
    is reported next to it."""
    import multiprocessing as mp
    from oracle import frameft_oracle as O
    t0 = time.perf_counter()
    P_in = O.tight_fusion_frame(ad.k_in, ad.rho_in, ad.d_in)
    P_out = P_in if (ad.k_out, ad.rho_out, ad.d_out) == (ad.k_in, ad.rho_in, ad.d_in) else \
        O.tight_fusion_frame(ad.k_out, ad.rho_out, ad.d_out)
    setup = time.perf_counter() - t0
    _CPU.update(P_in=P_in, P_out=P_out, data=data)
    T = wl.tokens
    # one thread on a prefix
    S = min(T, 256)
    t0 = time.perf_counter()
    _oracle_tokens((0, S))
    one = S / (time.perf_counter() - t0)
    cores = max(1, min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()))
    spans = [(T * i // cores, T * (i + 1) // cores) for i in range(cores)]
    with mp.get_context("fork").Pool(cores) as pool:
        pool.map(_oracle_tokens, [(0, 1)] * cores)        # workers started before the clock
        reps, t0 = 0, time.perf_counter()
        while True:
            parts = pool.map(_oracle_tokens, spans)
            reps += 1
            elapsed = time.perf_counter() - t0
            if elapsed >= budget_s / 2 or reps >= 8:
                break
    dc = np.sum(parts, axis=0)
    assert dc.shape == (ad.nnz,) and np.all(np.isfinite(dc))
    return {"value": round(reps * T / elapsed, 2), "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"all {T} tokens x {reps}, fp64 scipy-sparse oracle fwd+bwd (dX, dC) split over {cores} "
                      f"single-threaded processes; frame construction ({setup:.1f} s) excluded",
            "seconds": round(elapsed, 3), "cpu_model": _cpu_model(),
            "single_thread": {"value": round(one, 2), "sample": f"first {S} tokens, 1 thread"}}


def bench_stack(args, torch, ff, inputs, dev):
    """The whole adapter step of a multi-layer workload (the 32-layer x 7-projection Llama-2-7B
    stack): adapters of one shape share a plan (the support is shared across layers) and run as
    one batched forward and one batched backward launch per shape.  Activations, upstream
    gradients and coefficients are seeded device draws (a timing workload; the stack's parity is
    tested on its first and last layers)."""
    wl = inputs.WORKLOADS[args.workload]
    T, L = wl.tokens, wl.layers
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    esz = 2 if wl.dtype == "bf16" else 4
    gen = torch.Generator(device=dev)
    gen.manual_seed(wl.seed)
    shapes = {}
    for ad in wl.adapters:
        shapes.setdefault((ad.d_in, ad.d_out, ad.rho_in, ad.rho_out, ad.nnz), []).append(ad)
    frames, groups = {}, []
    t0 = time.perf_counter()
    for gi, ((n, m, rn, rm, nnz), ads) in enumerate(shapes.items()):
        for d, r in ((n, rn), (m, rm)):
            if (d, r) not in frames:
                frames[(d, r)] = ff.framegen(d, d // r, r)
        count = L * len(ads)
        if args.per_layer_masks:   # every adapter its own random support: a plan group per shape
            plans = [ff.plan_create(frames[(n, rn)], frames[(m, rm)],
                                    *inputs.support(inputs.rng(wl.seed + 10 * gi + 1000 * (i + 1)), m, n, nnz),
                                    max_tokens=T) for i in range(count)]
            plan = ff.plan_group(plans)
        else:                      # one support shared by the layers (Sec. 3.3)
            rows, cols = inputs.support(inputs.rng(wl.seed + 10 * gi), m, n, nnz)
            plans = [ff.plan_create(frames[(n, rn)], frames[(m, rm)], rows, cols, max_tokens=T, max_batch=count)]
            plan = plans[0]
        Xs = [torch.randn((T, n), generator=gen, device=dev).to(tdt) for _ in range(count)]
        Gs = [torch.randn((T, m), generator=gen, device=dev).to(tdt) for _ in range(count)]
        cs = []
        for i in range(count):
            pl = plans[i % len(plans)]
            order = torch.from_numpy(pl.order).to(dev)
            v = torch.randn((nnz,), generator=gen, device=dev) * 0.02
            c = torch.zeros((pl.coef_slots,), device=dev)
            c[order >= 0] = v[order[order >= 0]]
            cs.append(c)
        Ys = [torch.empty((T, m), dtype=tdt, device=dev) for _ in range(count)]
        dXs = [torch.empty((T, n), dtype=tdt, device=dev) for _ in range(count)]
        dCs = [torch.empty((plans[i % len(plans)].coef_slots,), device=dev) for i in range(count)]
        pa = ff.binding.pointer_array
        groups.append(dict(name="+".join(a.name for a in ads), n=n, m=m, nnz=nnz, count=count, plan=plan, plans=plans,
                           scale=inputs.scale_for(wl, ads[0]), X=Xs, G=Gs, Y=Ys, dX=dXs, dC=dCs, c=cs,
                           fptr=(pa(Xs, dev), pa(cs, dev), pa(Ys, dev)),
                           bptr=(pa(Xs, dev), pa(Gs, dev), pa(cs, dev), pa(dXs, dev), pa(dCs, dev))))
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t0

    def step(evs=None):
        for i, g in enumerate(groups):
            fwd, bwd = ((ff.adapter_fwd_group, ff.adapter_bwd_group) if args.per_layer_masks else
                        (ff.adapter_fwd_batched, ff.adapter_bwd_batched))
            if evs is not None:
                ff.binding.time_next_kernel(evs[i][0], evs[i][1])
            fwd(g["plan"], g["X"], g["c"], g["scale"], g["Y"], ptrs=g["fptr"])
            if evs is not None:
                ff.binding.time_next_kernel(evs[i][2], evs[i][3])
            bwd(g["plan"], g["X"], g["G"], g["c"], g["scale"], g["dX"], g["dC"], ptrs=g["bptr"])

    for _ in range(args.warmup):
        step()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    start.record()
    for _ in range(args.steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - w0) * 1e3
    ms_per_step = start.elapsed_time(stop) / args.steps
    evs = [[[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in groups] for _ in range(args.steps)]
    for e in evs:
        step(e)
    torch.cuda.synchronize()
    kernels, step_bytes, dom = {}, 0, None
    for i, g in enumerate(groups):
        b_fwd, b_bwd, b_red = algorithmic_bytes(T, g["n"], g["m"], g["nnz"], esz)
        step_bytes += g["count"] * (b_fwd + b_bwd + b_red)
        for j, (lab, b) in enumerate((("fwd", b_fwd), ("bwd", b_bwd))):
            us = 1e3 * float(np.mean([e[i][2 * j].elapsed_time(e[i][2 * j + 1]) for e in evs]))
            key = f"{lab}_kernel[{g['name']} x{g['count']}]"
            kernels[key] = round(us, 2)
            if dom is None or us > dom[1]:
                dom = (key, us, g["count"] * b)
    achieved = dom[2] / (dom[1] * 1e-6) / 1e9
    out = {
        "metric": METRIC, "value": round(T / (ms_per_step * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {L} layers x {len(wl.adapters)} projections "
                               f"({', '.join(a.name for a in wl.adapters)}), {T} tokens, batched fwd+bwd(dX,dC) "
                               f"per projection shape"
                               + (", a random support per adapter (plan groups)" if args.per_layer_masks else
                                  ", one support per projection shape shared by the layers"),
                   "tokens": T, "adapters": L * len(wl.adapters), "per_layer_masks": bool(args.per_layer_masks)},
        "roofline": {"bound": "hbm", "kernel": dom[0], "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "algorithmic_bytes_per_launch": dom[2], "avg_us": round(dom[1], 3)},
        "step_roofline": {"bytes_per_step": step_bytes,
                          "frac": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "kernel_us": kernels},
        "context": {"setup_s": round(setup_s, 3), "wall_ms_timed": round(wall_ms, 3), "kernel_hash": kernel_hash()},
    }
    print(json.dumps(out), flush=True)


def bench_merge(args, torch, ff, inputs, dev):
    """Merge into the frozen weight (Algorithm 1 steps 5-6): W = W + s P_out C P_in^T in place on
    a bf16 m x n weight, alternating +s and -s (merge, then unmerge: the hot swap of Sec. 3.4, "Storage efficiency").

    Algorithmic bytes per merge: read and write W (4 m n B for bf16) plus the coefficients
    (4 B each); the contraction is nnz (2 k_out) (2 k_in) multiply-adds, which the bf16-weight
    merge runs as three bf16 MFMA products per term (split operands).  The roofline line takes
    whichever bound is longer: HBM at 8 TB/s or those MFMA flops at the bf16 dense peak of
    2.5 PFLOP/s.  W0 is drawn on the device (seeded); this mode times the kernel and checks nothing.
    """
    wl = inputs.WORKLOADS[args.workload]
    ad = wl.adapters[args.adapter]
    data = inputs.adapter_data(wl, ad, tokens=1)
    n, m, nnz = ad.d_in, ad.d_out, ad.nnz
    f_in = ff.framegen(n, ad.k_in, ad.rho_in)
    f_out = f_in if (m, ad.k_out, ad.rho_out) == (n, ad.k_in, ad.rho_in) else ff.framegen(m, ad.k_out, ad.rho_out)
    plan = ff.plan_create(f_in, f_out, data.rows, data.cols, max_tokens=1)
    c = torch.from_numpy(plan.to_plan(data.vals)).to(dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(wl.seed)
    W = (torch.randn((m, n), generator=gen, device=dev) * (1.0 / np.sqrt(n))).to(torch.bfloat16)
    for i in range(args.warmup):
        ff.merge_delta(plan, c, data.scale if i % 2 == 0 else -data.scale, W, beta=1.0)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(args.steps):
        ff.merge_delta(plan, c, data.scale if i % 2 == 0 else -data.scale, W, beta=1.0)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for i, (e0, e1) in enumerate(evs):
        ff.binding.time_next_kernel(e0, e1)
        ff.merge_delta(plan, c, data.scale if i % 2 == 0 else -data.scale, W, beta=1.0)
    torch.cuda.synchronize()
    avg_us = float(np.mean([e0.elapsed_time(e1) for e0, e1 in evs])) * 1e3
    nbytes = 4 * m * n + 4 * nnz
    fma = nnz * (2 * ad.k_out) * (2 * ad.k_in)
    ach = nbytes / (avg_us * 1e-6) / 1e9
    tflops = 3 * 2 * fma / (avg_us * 1e-6) / 1e12     # bf16 MFMA flops (three products per term)
    mfma_bound = 3 * 2 * fma / 2500e12 > nbytes / 8e12
    roof = ({"bound": "mfma", "achieved": round(tflops, 2), "peak": 2500.0, "unit": "TFLOP/s",
             "frac": round(tflops / 2500.0, 4)} if mfma_bound else
            {"bound": "hbm", "achieved": round(ach, 1), "peak": 8000.0, "unit": "GB/s", "frac": round(ach / 8000.0, 4)})
    roof.update({"kernel": "merge_kernel", "traffic": None, "algorithmic_bytes_per_launch": nbytes,
                 "algorithmic_flops_per_launch": 2 * fma, "avg_us": round(avg_us, 3)})
    print(json.dumps({
        "metric": "FrameFT merge W += s P_out C P_in^T into a bf16 weight (HBM GB/s)", "value": round(ach, 1),
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "dtype": "bf16 split products, f32 accumulation, bf16 weight", "data": "synthetic",
        "config": {"workload": f"{args.workload}: merge of {ad.name} {n}->{m}, nnz={nnz}, frames "
                               f"(k={ad.k_in}, rho={ad.rho_in}) -> (k={ad.k_out}, rho={ad.rho_out})"},
        "roofline": roof,
        "context": {"rank1_fma": fma, "bf16_mfma_tflops": round(tflops, 2), "hbm_gbs": round(ach, 1),
                    "kernel_hash": kernel_hash()}}))


# Query and value projections (d_in -> d_out) of the models whose frame construction time the
# paper reports on an A100 (Appendix, basis generation time: Spectral Tetris rows, seconds).
FRAMEGEN_MODELS = {
    "Llama-2-7B": ([(4096, 4096), (4096, 4096)], 0.09),
    "Gemma-2-9B": ([(3584, 4096), (3584, 2048)], 0.21),
    "Llama-3.1-8B": ([(4096, 4096), (4096, 1024)], 0.11),
}


def bench_framegen(torch, ff, rho=64, reps=5):
    """Wall time of building every distinct frame one model's adapted projections need.

    Frames depend only on (d, k, rho) and are shared across layers (Sec. 3.4, "Memory Overhead"), so a model needs one
    frame per distinct dimension.  The paper's instruction-tuning runs use rho = 2 (a single dense
    block of width d per frame), which the GPU path does not take; rho = 64 is timed instead.
    """
    out = {}
    for name, (projs, paper_s) in FRAMEGEN_MODELS.items():
        dims = sorted({d for p in projs for d in p})
        times = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            frames = [ff.framegen(d, d // rho, rho) for d in dims]
            torch.cuda.synchronize()
            times.append(time.perf_counter() - t0)
            del frames
        out[name] = {"dims": dims, "rho": rho, "median_s": round(float(np.median(times)), 5),
                     "paper_s_a100_spectral_tetris": paper_s}
    print(json.dumps({"metric": "frame construction time (ff_framegen: host construction, "
                                "exact tightness checks, upload)", "unit": "s",
                      "higher_is_better": False, "models": out,
                      "note": "paper's times are an A100 PyTorch run at rho = 2; context, not a target"}))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="cfg2_llama7b_qproj")
    ap.add_argument("--adapter", type=int, default=0, help="adapter of a multi-adapter workload (one layer)")
    ap.add_argument("--stack", action="store_true",
                    help="time every adapter of every layer of the workload (the 7B stack) as batched calls")
    ap.add_argument("--per-layer-masks", action="store_true",
                    help="with --stack: a random support per adapter (plan groups) instead of one per shape")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sets", type=int, default=0,
                    help="buffer sets rotated over the steps (0: enough to exceed 512 MiB; 1: one set, "
                         "which may stay in the last-level cache)")
    ap.add_argument("--merge", action="store_true",
                    help="time the merge W += s P_out C P_in^T into the workload adapter's bf16 weight "
                         "(alternating +s and -s, the hot swap) instead of the training step")
    ap.add_argument("--framegen", action="store_true",
                    help="time frame construction (ff_framegen, host build and upload) for the adapted "
                         "projections of the models in the paper's basis-generation-time table")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="first run 3 device-to-device copies of this many MiB (a known-size kernel "
                         "that calibrates the HBM byte counters of a --pmc profile)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (the adapter shards "
              "over tokens with one dC all-reduce, see the design notes); run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    from paper_2608_26430_amd import inputs
    cpu = None
    if not (args.stack or args.framegen or args.merge or args.no_cpu_baseline):
        wl = inputs.WORKLOADS[args.workload]
        cpu = cpu_baseline(wl, wl.adapters[args.adapter], inputs.adapter_data(wl, wl.adapters[args.adapter]))

    import torch
    import paper_2608_26430_amd as ff

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    if args.copy_probe_mib > 0:
        src = torch.ones(args.copy_probe_mib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.stack:
        bench_stack(args, torch, ff, inputs, dev)
        return
    if args.framegen:
        bench_framegen(torch, ff)
        return
    if args.merge:
        bench_merge(args, torch, ff, inputs, dev)
        return
    wl = inputs.WORKLOADS[args.workload]
    ad = wl.adapters[args.adapter]
    data = inputs.adapter_data(wl, ad)
    T, n, m, nnz = wl.tokens, ad.d_in, ad.d_out, ad.nnz
    esz = 2 if wl.dtype == "bf16" else 4
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32

    t0 = time.perf_counter()
    f_in = ff.framegen(n, ad.k_in, ad.rho_in)
    f_out = f_in if (m, ad.k_out, ad.rho_out) == (n, ad.k_in, ad.rho_in) else ff.framegen(m, ad.k_out, ad.rho_out)
    plan = ff.plan_create(f_in, f_out, data.rows, data.cols, max_tokens=T)
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t0

    # Buffer sets (X, G, Y, dX, c, dC and the saved copy) rotated from step to step, enough of them
    # that the working set is well beyond the 256 MB last-level cache (Infinity Cache): each
    # timed step then streams its activations from HBM, as a step over fresh data would.
    set_bytes = esz * T * (2 * n + 2 * m)
    nsets = 1 if args.sets == 1 else max(2, min(8, -(-(512 << 20) // set_bytes))) if args.sets == 0 else args.sets
    X0 = torch.from_numpy(data.X).to(dev, tdt)
    G0 = torch.from_numpy(data.G).to(dev, tdt)
    c0 = torch.from_numpy(plan.to_plan(data.vals)).to(dev)      # plan layout (padded)
    sets = [dict(X=X0.clone(), G=G0.clone(), c=c0.clone(), Y=torch.empty((T, m), dtype=tdt, device=dev),
                 dX=torch.empty((T, n), dtype=tdt, device=dev),
                 dC=torch.empty((plan.coef_slots,), dtype=torch.float32, device=dev),
                 # a training step: the forward also leaves the coefficients in the backward's order
                 saved=plan.new_saved(dev)) for _ in range(nsets)]
    del X0, G0

    def step(i, evs=None):
        b = sets[i % nsets]
        if evs is not None:
            ff.binding.time_next_kernel(evs[0], evs[1])
        ff.adapter_fwd(plan, b["X"], b["c"], data.scale, Y=b["Y"], save=b["saved"])
        if evs is not None:
            ff.binding.time_next_kernel(evs[2], evs[3])
        ff.adapter_bwd(plan, b["X"], b["G"], b["c"], data.scale, dX=b["dX"], dC=b["dC"], saved=b["saved"])

    def timed(steps, first):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        start.record()
        for i in range(steps):
            step(first(i))
        stop.record()
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / steps, (time.perf_counter() - w0) * 1e3

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    # timed region: K whole steps over the rotated sets, no per-kernel events (step time)
    ms_per_step, wall_ms = timed(args.steps, lambda i: i)
    # context: the same steps on one set, whose 128 MB may stay partly in the last-level cache
    ms_warm, _ = timed(args.steps, lambda i: 0)

    # per-kernel durations: the same rotated steps with events around the fused kernels
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for i, e in enumerate(evs):
        step(i, e)
    torch.cuda.synchronize()
    fwd_us = 1e3 * float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    bwd_us = 1e3 * float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    # spread of single steps: events between consecutive rotated steps, median and CoV
    sev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    sev[0].record()
    for i in range(args.steps):
        step(i)
        sev[i + 1].record()
    torch.cuda.synchronize()
    per_step = np.array([1e3 * sev[i].elapsed_time(sev[i + 1]) for i in range(args.steps)])

    # a plain device copy of 256 MiB (read + write), the achievable HBM rate beside the 8 TB/s peak
    csrc = torch.empty(64 << 20, dtype=torch.float32, device=dev)
    cdst = torch.empty_like(csrc)
    cdst.copy_(csrc)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(5):
        cdst.copy_(csrc)
    c1.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * csrc.numel() * 4 * 5 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del csrc, cdst

    b_fwd, b_bwd, b_red = algorithmic_bytes(T, n, m, nnz, esz)
    if bwd_us >= fwd_us:
        dom, dom_us, dom_bytes = "bwd_kernel", bwd_us, b_bwd
    else:
        dom, dom_us, dom_bytes = "fwd_kernel", fwd_us, b_fwd
    achieved = dom_bytes / (dom_us * 1e-6) / 1e9
    traffic = None
    tfile = os.path.join(ROOT, "profiles", f"traffic_{args.workload}.json")
    if os.path.exists(tfile):
        tr = json.load(open(tfile))
        if tr.get("kernel_hash") == kernel_hash() and dom in tr.get("bytes_per_launch", {}):
            traffic = tr["bytes_per_launch"][dom]
    step_bytes = b_fwd + b_bwd + b_red
    value = T / (ms_per_step * 1e-3)

    # context: the frozen W0 GEMM of this layer through the vendor BLAS (not part of the step)
    W0 = torch.randn((m, n), device=dev, dtype=tdt)
    Xg = sets[0]["X"]
    for _ in range(3):
        torch.matmul(Xg, W0.t())
    torch.cuda.synchronize()
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g0.record()
    for _ in range(10):
        torch.matmul(Xg, W0.t())
    g1.record()
    torch.cuda.synchronize()
    gemm_us = 1e3 * g0.elapsed_time(g1) / 10

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {ad.name} {n}->{m}, frames (k={ad.k_in}, rho={ad.rho_in}) -> "
                               f"(k={ad.k_out}, rho={ad.rho_out}), nnz={nnz}, {T} tokens, fwd+bwd(dX,dC)",
                   "tokens": T, "d_in": n, "d_out": m, "nnz": nnz},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": dom_bytes, "avg_us": round(dom_us, 3)},
        "step_roofline": {"bytes_per_step": step_bytes, "frac": round(step_bytes / (ms_per_step * 1e-3) / 1e9
                                                                       / HBM_PEAK_GBS, 4),
                          "fwd_kernel_us": round(fwd_us, 3), "bwd_kernel_us": round(bwd_us, 3)},
        "context": {"step_us_median": round(float(np.median(per_step)), 3),
                    "step_us_cov": round(float(np.std(per_step) / np.mean(per_step)), 4),
                    "copy_256mib_gbs": round(copy_gbs, 1),
                    "w0_gemm_us": round(gemm_us, 2), "setup_s": round(setup_s, 3),
                    "wall_ms_timed": round(wall_ms, 3), "buffer_sets": nsets,
                    "buffer_set_mb": round(set_bytes / 1e6, 1),
                    "one_set_ms_per_step": round(ms_warm, 5),
                    "one_set_tokens_per_s": round(T / (ms_warm * 1e-3), 1),
                    "tile_tokens": plan.tile_tokens(wl.dtype), "input_chunks": plan.gen_chunks,
                    "chunk_tile_tokens": plan.gen_tile_tokens(wl.dtype), "kernel_hash": kernel_hash()},
    }
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
