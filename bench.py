"""PD-scan benchmark on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 2]

One step = dictionary preparation (pdssm_prepare), one forward scan
(pdssm_scan_fwd: y, h_final, saved chunk states) and one backward scan
(pdssm_scan_bwd: dD, db, dc, dh0) over one batch of seeded synthetic inputs
already resident in HBM.  A 512 MiB buffer is rewritten between steps (not
timed) so that no input of a step is still cached.  The default 200 untimed
steps, preceded by at least 0.3 s of the same step (clock_settle in the line;
also with a short --warmup), let the GPU clocks settle: the compute-heavier
workloads run up to 20% slower during the first ~100 ms of load.  Then 50
steps are timed.  Prints ONE JSON line.

value = state updates (B*L*H*N) per second of the whole step (mean step
time; every call also reports its median).
roofline = the dominant kernel's algorithmic bytes (each tensor of the method
read or written once: 24 + 8/N bytes per state update forward, 48 + 8/N
backward, in complex64) over its average duration, measured with HIP events
on the stream the kernels are launched on, against the 8 TB/s HBM peak;
traffic = the HBM bytes per launch that rocprofv3 counters measured for the
same kernel source (profiles/), else null.  The chunk-entering states handed
from the forward to the backward are reported apart (design_bytes).
markov_manyone = with the default workload, the many-to-one workload of the
same shape (L=2048, d=1024 as 16 heads of 64, Markov-chain map choices),
timed the same way in the same run.
cpu_baseline = the float64 oracle timed on this host: whole passes over every
sequence of the workload on the 16-core CPU share of a one-GPU machine.

--ste times the straight-through training step instead (Sec. 3.1 Prop. 2):
prepare, forward, the backward with the scaled states (pdssm_scan_bwd_ste),
the candidate-map scores and the dictionary gradient (pdssm_ste_grads) and
the two tempered-softmax products (routing logits, dense dictionary); the
line then carries an "ste" object with each call's time and roofline.  It
combines with --real (real rows) and --bf16 (bf16 pairs, z complex64).

--decode times single-step decode instead (pdssm_decode_step: one recurrence
step per sequence, state updated in place), back to back on the workload's
B, H, N, K; value = state updates (B*H*N) per second, with its bytes per step.
"""
import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_FP32_PEAK_TFS = 157.3
FLUSH_BYTES = 512 << 20
SETTLE_S = 0.3  # untimed sustained load before the warm-up steps (clock ramp)
METRIC = "PD-scan state-updates/s (B*L*H*N) fwd and fwd+bwd; achieved HBM GB/s vs peak"


def alg_bytes(w, C, op, esz=8, ssz=8):
    """Algorithmic HBM bytes of one call: every tensor of the method read or
    written once.  Forward: idx, D, b, c and the dictionary in; y and h_final
    out (24 + 8/N bytes per state update in complex64).  Backward: idx, dy,
    D, b, c and the dictionary in; dD, db, dc and dh0 out (48 + 8/N).  The
    chunk-entering states that the forward hands to the backward are this
    design's own intermediate, not the method's, and are counted apart
    (design_bytes).  esz = bytes per entry of D, b, c, dD, db, dc (8 for
    complex64, 4 for bf16 pairs or the real model); ssz = bytes per state
    entry of h_final and dh0 (8, or 4 for the real model, whose states are
    real; the library keeps h_final and dh0 as complex64 and the saved states
    as fp32); y and dy are fp32."""
    B, L, H, N, K = w.B, w.L, w.H, w.N, w.K
    steps = B * L * H
    su = steps * N
    dict_b = H * K * N * 4
    if op == "fwd":
        return steps * 4 + 3 * su * esz + dict_b + steps * 4 + B * H * N * ssz
    return steps * 8 + 3 * su * esz + dict_b + 3 * su * esz + B * H * N * ssz


def saved_bytes(w, C, ssz=8):
    """The chunk-entering states: written once by the forward, read once by
    the backward (ssz bytes per entry, C chunks per sequence)."""
    return w.B * w.H * C * w.N * ssz


def ste_bytes(w, C, real=False, bf16=False):
    """Algorithmic bytes and flops of the straight-through calls (real: the
    real-valued model, 4-byte rows and real states; bf16: 4-byte rows, z
    complex64)."""
    B, L, H, N, K = w.B, w.L, w.H, w.N, w.K
    steps = B * L * H
    su = steps * N
    esz = 4 if (real or bf16) else 8
    ssz = 4 if real else 8
    zsz = 4 if real else 8
    return {
        # the plain backward, plus z [B,L,H,N] written
        "bwd_ste": alg_bytes(w, C, "bwd", esz, ssz) + su * zsz,
        # idx, pi, g (= db) and z read once, q [B,L,H,K] and G [H,K,N,N] f32 written once
        "ste_grads": steps * 4 + H * K * N * 4 + su * (esz + zsz) + steps * K * 4 + H * K * N * N * 4,
        # per step and (i, j): Re(g_i conj z_j) = two real multiply-adds (one when real)
        "ste_grads_flops": (2 if real else 4) * steps * N * N,
        # logits and q in, d logits out; M and G in, dM out
        "softmax": 3 * steps * K * 4 + 3 * H * K * N * N * 4,
    }


def host_cpu():
    """What the host offers: nproc (the cores this process may run on), the
    machine's logical CPU count and the CPU model."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count() or 1
    return {"nproc": nproc, "logical_cpus": os.cpu_count(), "model": model}


# A one-GPU machine grants its job a 16-core share of the host, whatever nproc
# shows; the oracle's thread pool uses that share.
CPU_SHARE = 16


def cpu_baseline(w, inp, target_s=12.0):
    """Time the float64 oracle (fwd + bwd, one whole sequence per task) on
    this host: whole passes over every sequence of the workload on a pool of
    threads (the oracle's C loops run without the GIL), repeated until about
    target_s seconds have passed; the median pass gives the rate.  Then the
    same oracle on one thread, whole sequences one after another (median
    sequence time)."""
    from concurrent.futures import ThreadPoolExecutor

    from oracle import oracle_bwd, oracle_fwd
    from paper_2605_19150_amd.inputs import sub_sequence
    seqs = [(bb, hh) for bb in range(w.B) for hh in range(w.H)]
    subs = []
    for bb, hh in seqs:
        sub = sub_sequence(inp, bb, hh)
        for k in ("D", "b", "c"):
            sub[k] = sub[k].astype(np.complex128)
        sub["dy"] = sub["dy"].astype(np.float64)
        subs.append(sub)
    host = host_cpu()
    threads = max(1, min(CPU_SHARE, host["nproc"]))

    def one(sub):
        oracle_fwd(sub["idx"], sub["pi"], sub["D"], sub["b"], sub["c"])
        oracle_bwd(sub["idx"], sub["pi"], sub["D"], sub["b"], sub["c"], sub["dy"])
        return w.L * w.N

    passes = []
    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=threads) as pool:
        while True:
            t = time.perf_counter()
            done = sum(pool.map(one, subs))
            passes.append(time.perf_counter() - t)
            if time.perf_counter() - t0 >= target_s and len(passes) >= 3:
                break
    wall = time.perf_counter() - t0
    med = float(np.median(passes))
    # the same oracle on one thread: whole sequences one after another
    per_seq = []
    t1 = time.perf_counter()
    while time.perf_counter() - t1 < target_s / 4 or len(per_seq) < 3:
        t = time.perf_counter()
        one(subs[len(per_seq) % len(subs)])
        per_seq.append(time.perf_counter() - t)
    one_med = float(np.median(per_seq))
    return {"value": done / med, "unit": "state-updates/s", "cores": threads, "kind": "oracle",
            "sample": "fwd+bwd float64 oracle on all %d sequences of the workload (L=%d, N=%d) per pass, "
                      "%d passes on %d threads (median pass %.3f s), %.1f s wall"
                      % (len(subs), w.L, w.N, len(passes), threads, med, wall),
            "host": host,
            "note": "thread pool = the %d-core CPU share of a one-GPU box (nproc %d)"
                    % (CPU_SHARE, host["nproc"]),
            "single_thread": {"value": w.L * w.N / one_med, "unit": "state-updates/s",
                              "sample": "%d whole sequences one after another on one thread "
                                        "(median %.4f s per sequence)" % (len(per_seq), one_med)}}


def traffic_from_profiles(kernel, workload_name):
    """HBM bytes per launch of `kernel` on this workload from the committed
    counter summary, or None when there is none or the kernel sources have
    changed since the counters were taken."""
    from paper_2605_19150_amd.profiling import read_traffic_summary
    return read_traffic_summary(os.path.join(ROOT, "profiles"), kernel, workload_name)


def decode_bench(args, w, dev):
    """Single-step decode: steps of one token for every (batch, head)
    sequence, in place, back to back (launch cost included)."""
    import torch
    from paper_2605_19150_amd import pdssm
    from paper_2605_19150_amd.inputs import make_inputs

    T = 64  # distinct tokens cycled through
    inp = make_inputs(w.B, T, w.H, w.N, w.K, seed=0, pi_kind=w.pi_kind, dmag=w.dmag, bc_var=w.bc_var,
                      idx_kind=w.idx_kind, with_h0=True)
    tok = [{k: torch.from_numpy(np.ascontiguousarray(inp[k][:, t])).to(dev) for k in ("idx", "D", "b", "c")}
           for t in range(T)]
    pi = torch.from_numpy(inp["pi"]).to(dev)
    h = torch.from_numpy(inp["h0"]).to(dev)
    y = torch.empty((w.B, w.H), dtype=torch.float32, device=dev)
    L = pdssm.load()
    d = pdssm.desc(w.B, 1, w.H, w.N, w.K)
    st = pdssm._stream(None)
    args_of = [[ctypes.byref(d), pdssm._p(x["idx"]), pdssm._p(pi), pdssm._p(x["D"]), pdssm._p(x["b"]),
                pdssm._p(x["c"]), pdssm._p(h), pdssm._p(h), pdssm._p(y), None, st] for x in tok]

    def run(n):
        for i in range(n):
            rc = L.pdssm_decode_step(*args_of[i % T])
            if rc != pdssm.OK:
                raise pdssm.PdssmError(rc, "pdssm_decode_step")

    steps = max(args.steps, 1) * 20
    run(max(args.warmup, 1) * 5)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    run(steps)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    nseq = w.B * w.H
    nbytes = nseq * (4 + 4 + 5 * w.N * 8) + w.H * w.K * w.N * 4  # idx, y; D, b, c, h in, h out; dictionary
    print(json.dumps({
        "metric": "PD-scan single-step decode state-updates/s (B*H*N per step)",
        "value": nseq * w.N / (ms * 1e-3), "unit": "state-updates/s", "n_gpus": 1, "steps": steps,
        "warmup": max(args.warmup, 1) * 5, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic (seeded, shapes and distributions of the named workload)",
        "config": {"workload": w.name + " decode", "B": w.B, "H": w.H, "N": w.N, "K": w.K, "step": "decode",
                   "parallelism": "single-gpu"},
        "decode": {"kernel": "k_decode", "alg_bytes": nbytes, "alg_GBps": nbytes / (ms * 1e-3) / 1e9,
                   "note": "back-to-back launches, one per token: launch-bound at these sizes"},
        "device": torch.cuda.get_device_name(dev),
    }), flush=True)


def front_bench(args, w, dev):
    """Selection front end and token projections for the workload's layer:
    the maps of a dense dictionary [H,K,N,N] (pdssm_dict_argmax), the routing
    of every token with d_model = H*N (pdssm_route: bf16 product on the
    matrix cores, fp32 logits written, argmax fused), and the whole
    projection (pdssm_project: routing, b, c and the diagonal generator in one
    product, u read once)."""
    import torch
    from paper_2605_19150_amd import pdssm

    Dm, T = w.H * w.N, w.B * w.L
    g = torch.Generator(device="cpu").manual_seed(0)
    u = torch.randn((w.B, w.L, Dm), generator=g).to(torch.bfloat16).to(dev)
    S = (torch.randn((w.H, w.K, Dm), generator=g) / Dm ** 0.5).to(torch.bfloat16).to(dev)
    Wp = [(torch.randn((w.H, 2 * w.N, Dm), generator=g) / Dm ** 0.5).to(torch.bfloat16).to(dev) for _ in range(3)]
    M = torch.randn((w.H, w.K, w.N, w.N), generator=g).to(dev)
    lg = torch.empty((w.B, w.L, w.H, w.K), dtype=torch.float32, device=dev)
    idx = torch.empty((w.B, w.L, w.H), dtype=torch.int32, device=dev)
    pi = torch.empty((w.H, w.K, w.N), dtype=torch.int32, device=dev)
    outs = [torch.empty((w.B, w.L, w.H, w.N), dtype=torch.complex64, device=dev) for _ in range(3)]
    L = pdssm.load()
    st = pdssm._stream(None)
    flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)
    P = pdssm._p

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        assert L.pdssm_dict_argmax(w.H, w.K, w.N, P(M), P(pi), st) == pdssm.OK
        if ev is not None:
            ev[1].record()
        assert L.pdssm_route(T, Dm, w.H, w.K, P(u), P(S), P(lg), P(idx), st) == pdssm.OK
        if ev is not None:
            ev[2].record()
        assert L.pdssm_project(T, Dm, w.H, w.K, w.N, P(u), P(S), P(Wp[0]), P(Wp[1]), P(Wp[2]), P(lg), P(idx),
                               P(outs[0]), P(outs[1]), P(outs[2]), st) == pdssm.OK
        if ev is not None:
            ev[3].record()

    t_settle = time.perf_counter()
    while time.perf_counter() - t_settle < SETTLE_S:
        flush.fill_(1.0)
        step()
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        flush.fill_(1.0)
        step()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        flush.fill_(float(i))
        step(evs[i])
    torch.cuda.synchronize()
    am_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    rt_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    pj_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    rt_bytes = T * Dm * 2 + w.H * w.K * Dm * 2 + T * w.H * w.K * 4 + T * w.H * 4
    rt_flops = 2.0 * T * w.H * w.K * Dm
    cols = w.H * w.K + 3 * 2 * w.H * w.N
    pj_flops = 2.0 * T * cols * Dm
    pj_bytes = T * Dm * 2 + cols * Dm * 2 + T * w.H * w.K * 4 + T * w.H * 4 + 3 * T * w.H * w.N * 8
    am_bytes = w.H * w.K * w.N * w.N * 4 + w.H * w.K * w.N * 4
    tf = pj_flops / (pj_ms * 1e-3) / 1e12
    print(json.dumps({
        "metric": "PD-SSM layer projections TFLOP/s (routing, b, c and the diagonal generator in one product)",
        "value": tf, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": am_ms + rt_ms + pj_ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16 operands, f32 accumulation", "data": "synthetic (seeded)",
        "config": {"workload": w.name + " layer front end", "tokens": T, "d_model": Dm, "H": w.H, "K": w.K,
                   "N": w.N, "step": "dict_argmax+route+project", "parallelism": "single-gpu"},
        "roofline": {"bound": "mfma", "kernel": "k_project_dma", "achieved": tf, "peak": 2500.0,
                     "unit": "TFLOP/s", "frac": tf / 2500.0, "traffic": None},
        "project": {"kernel": "k_project_dma", "ms": pj_ms, "flops": pj_flops, "TFLOPs": tf,
                    "frac_mfma_bf16": tf / 2500.0, "alg_bytes": pj_bytes,
                    "alg_GBps": pj_bytes / (pj_ms * 1e-3) / 1e9, "columns": cols},
        "route": {"kernel": "k_project_dma (routing tiles only)", "ms": rt_ms, "alg_bytes": rt_bytes,
                  "alg_GBps": rt_bytes / (rt_ms * 1e-3) / 1e9, "flops": rt_flops,
                  "TFLOPs": rt_flops / (rt_ms * 1e-3) / 1e12,
                  "frac_mfma_bf16": rt_flops / (rt_ms * 1e-3) / 1e12 / 2500.0},
        "dict_argmax": {"kernel": "k_dict_argmax", "ms": am_ms, "alg_bytes": am_bytes,
                        "alg_GBps": am_bytes / (am_ms * 1e-3) / 1e9},
        "device": torch.cuda.get_device_name(dev),
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=200,
                    help="untimed steps first: the GPU clocks ramp up over the first ~100 ms of load")
    ap.add_argument("--workload", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-second-leg", action="store_true",
                    help="with the default workload, skip timing the many-to-one workload of the same shape")
    ap.add_argument("--only", choices=["fwd", "bwd", "both"], default="both",
                    help="profiling aid: launch only one call per step")
    ap.add_argument("--ste", action="store_true",
                    help="time the straight-through step (scores, dictionary gradient, softmax products)")
    ap.add_argument("--temp", type=float, default=1.0, help="softmax temperature of --ste")
    ap.add_argument("--decode", action="store_true", help="time single-step decode instead")
    ap.add_argument("--front", action="store_true",
                    help="time the selection front end (dictionary argmax, routing product + argmax) instead")
    ap.add_argument("--bf16", action="store_true",
                    help="bf16 (re, im) pairs for D, b, c and the gradients (fp32 arithmetic)")
    ap.add_argument("--real", action="store_true",
                    help="the real-valued model: real fp32 D, b, c and gradients")
    ap.add_argument("--chunk", type=int, default=0,
                    help="scan chunk length (4, 8 or 16 steps; 0: the library's default)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="profiling aid: time a plain 1 GiB device copy instead")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: runs on exactly one GPU; --gpus %d is not supported "
              "(the PD scan shards by sequence without communication)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2605_19150_amd import pdssm
    from paper_2605_19150_amd.inputs import WORKLOADS, workload_inputs

    dev = torch.device("cuda:0")
    if args.copy_calibration:
        n = 1 << 30
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(args.warmup):
            dst.copy_(src)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        print(json.dumps({"copy_bytes": 2 * n, "ms": ms, "GBps": 2 * n / ms / 1e6}))
        return

    w = WORKLOADS[args.workload]
    if args.decode:
        decode_bench(args, w, dev)
        return
    if args.front:
        front_bench(args, w, dev)
        return
    if args.real and args.bf16:
        sys.exit("bench.py: --real and --bf16 do not combine (one row format at a time)")
    # Written between timed steps so that no input is still in L2 / MALL.
    flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)
    res, inp = time_scan(args, args.workload, dev, flush)
    out = scan_line(args, w, res)
    out["device"] = torch.cuda.get_device_name(dev)
    plain = args.only == "both" and not args.ste and not args.bf16 and not args.real
    if plain and args.workload == 2 and not args.no_second_leg:
        # the second workload of the same shape (L=2048, d=1024 as 16 heads
        # of 64): many-to-one maps chosen by a Markov chain, timed the same way
        w3 = WORKLOADS[3]
        del inp
        res3, inp = time_scan(args, 3, dev, flush)
        leg = scan_line(args, w3, res3)
        out["markov_manyone"] = {k: leg[k] for k in ("ms_per_step", "ms_per_step_median", "value", "prepare",
                                                      "fwd", "bwd", "fwd_bwd")}
        out["markov_manyone"]["workload"] = w3.name
        out["markov_manyone"]["chunk"] = leg["config"]["chunk"]
        if not args.no_cpu_baseline:
            inp = None
    if not args.no_cpu_baseline and plain:
        if inp is None:
            from paper_2605_19150_amd.inputs import workload_inputs
            inp = workload_inputs(args.workload, seed=0)
        print("bench: timing the oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w, inp)
    print(json.dumps(out), flush=True)


def time_scan(args, wi, dev, flush):
    """Time args.steps steps of workload wi after args.warmup untimed ones;
    every call bracketed by HIP events on the stream the kernels run on.
    Returns (per-call times and the Scan, the host inputs)."""
    import torch
    from paper_2605_19150_amd import pdssm
    from paper_2605_19150_amd.inputs import WORKLOADS, workload_inputs

    w = WORKLOADS[wi]
    print("bench: workload %d (%s): generating inputs" % (wi, w.name), file=sys.stderr, flush=True)
    inp = workload_inputs(wi, seed=0, real=args.real)
    T = {k: torch.from_numpy(v).to(dev) for k, v in inp.items()}
    if args.bf16:
        for k in ("D", "b", "c"):
            T[k] = torch.view_as_real(T[k]).to(torch.bfloat16).contiguous()
    s = pdssm.Scan(w.B, w.L, w.H, w.N, w.K, args.chunk, ste=args.ste, bf16=args.bf16, real=args.real)
    if args.ste:
        from paper_2605_19150_amd.inputs import selection_inputs
        logits, M = selection_inputs(inp["idx"], inp["pi"], seed=0)
        T["logits"], T["M"] = torch.from_numpy(logits).to(dev), torch.from_numpy(M).to(dev)
        dlogits, dM = torch.empty_like(T["logits"]), torch.empty_like(T["M"])
    stream = torch.cuda.current_stream()

    def step(ev=None):
        rec = (lambda i: ev[i].record(stream)) if ev is not None else (lambda i: None)
        rec(0)
        s.prepare(T["pi"])
        rec(1)
        if args.only in ("fwd", "both"):
            s.fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"])
        rec(2)
        if args.only in ("bwd", "both"):
            if args.ste:
                s.bwd_ste(T["idx"], T["pi"], T["D"], T["b"], T["c"], T["dy"])
            else:
                s.bwd(T["idx"], T["pi"], T["D"], T["b"], T["c"], T["dy"])
        rec(3)
        if args.ste:
            s.ste_grads(T["idx"], T["pi"])
            rec(4)
            pdssm.softmax_vjp(T["logits"], s.q, 3, args.temp, out=dlogits)
            pdssm.softmax_vjp(T["M"], s.G, 2, args.temp, out=dM)
            rec(5)

    if args.only == "bwd":
        s.prepare(T["pi"])
        s.fwd(T["idx"], T["pi"], T["D"], T["b"], T["c"])
    # The GPU clocks ramp up over the first ~100 ms of sustained load: the
    # same step runs for at least SETTLE_S seconds before the W warm-up steps
    # (untimed; the timed region is the K steps below either way).
    settle, t_settle = 0, time.perf_counter()
    while True:
        flush.fill_(1.0)
        step()
        settle += 1
        if settle % 8 == 0:
            torch.cuda.synchronize()
            if time.perf_counter() - t_settle >= SETTLE_S:
                break
    settle_s = time.perf_counter() - t_settle
    for _ in range(args.warmup):
        flush.fill_(1.0)
        step()
    torch.cuda.synchronize()
    s.check_status()
    print("bench: timing %d steps" % args.steps, file=sys.stderr, flush=True)

    nev = 6 if args.ste else 4
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        flush.fill_(float(i))
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    s.check_status()
    ms = lambda a, b: np.array([e[a].elapsed_time(e[b]) for e in evs])  # noqa: E731
    res = {"scan": s, "wall": wall, "prepare": ms(0, 1), "fwd": ms(1, 2), "bwd": ms(2, 3),
           "step": ms(0, nev - 1), "settle": {"steps": settle, "s": settle_s}}
    if args.ste:
        res["ste_grads"] = ms(3, 4)
        res["softmax"] = ms(4, 5)
    return res, inp


def scan_line(args, w, res):
    """The bench line of one timed workload: means (the roofline's kernel
    durations) and medians of every call, algorithmic bytes and fractions of
    the HBM peak."""
    s = res["scan"]
    mean = lambda k: float(np.mean(res[k]))  # noqa: E731
    med = lambda k: float(np.median(res[k]))  # noqa: E731
    su = w.state_updates
    esz = 4 if (args.bf16 or args.real) else 8
    ssz = 4 if args.real else 8
    fwd_b, bwd_b = alg_bytes(w, s.C, "fwd", esz, ssz), alg_bytes(w, s.C, "bwd", esz, ssz)
    sv_b = saved_bytes(w, s.C, ssz)
    fused = s.fused
    kern = {"fwd": "k_fwd_fused" if fused else "k_fwd_*(chunked)",
            "bwd": "k_bwd_fused" if fused else "k_bwd_*(chunked)"}
    fwd_ms, bwd_ms = mean("fwd"), mean("bwd")
    dom = "bwd" if (bwd_ms >= fwd_ms and args.only != "fwd") else "fwd"
    dom_ms, dom_b = (bwd_ms, bwd_b) if dom == "bwd" else (fwd_ms, fwd_b)
    achieved = dom_b / (dom_ms * 1e-3) / 1e9
    suffix = "_bf16" if args.bf16 else ("_real" if args.real else "")
    traffic = traffic_from_profiles(kern[dom] + suffix, w.name) if fused else None

    def call(k, nbytes):
        m, d = mean(k), med(k)
        return {"kernel": kern[k], "ms": m, "ms_median": d, "state_updates_per_s": su / (m * 1e-3),
                "alg_bytes": nbytes, "alg_GBps": nbytes / (m * 1e-3) / 1e9,
                "frac": nbytes / (m * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "frac_median": nbytes / (d * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "design_bytes": nbytes + sv_b}

    ms_step, ms_step_med = mean("step"), med("step")
    fb_ms, fb_med = fwd_ms + bwd_ms, med("fwd") + med("bwd")
    out = {
        "metric": METRIC,
        "value": su / (ms_step * 1e-3),
        "unit": "state-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_median": ms_step_med,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16-io/f32" if args.bf16 else ("f32-real" if args.real else "f32"),
        "data": "synthetic (seeded, shapes and distributions of the named workload)",
        "config": {"workload": w.name + (" (real-valued model)" if args.real else ""), "B": w.B, "L": w.L,
                   "H": w.H, "N": w.N, "K": w.K, "chunk": s.chunk, "segments": s.segments,
                   "step": ("prepare+fwd+bwd_ste+ste_grads+softmax_vjp" if args.ste else "prepare+fwd+bwd")
                   if args.only == "both" else args.only,
                   "global_batch": w.B, "seq_len": w.L, "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "kernel": kern[dom],
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "bytes": "algorithmic: %s (%.1f + 8/N bytes per state update)"
                              % ("idx, dy, D, b, c in; dD, db, dc, dh0 out" if dom == "bwd"
                                 else "idx, D, b, c in; y, h_final out", (48.0 if dom == "bwd" else 24.0) * esz / 8)},
        "prepare": {"ms": mean("prepare"), "ms_median": med("prepare")},
        "fwd": call("fwd", fwd_b),
        "bwd": call("bwd", bwd_b),
        "fwd_bwd": {"ms": fb_ms, "ms_median": fb_med, "alg_bytes": fwd_b + bwd_b,
                    "state_updates_per_s": su / (fb_ms * 1e-3),
                    "frac": (fwd_b + bwd_b) / (fb_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                    "frac_median": (fwd_b + bwd_b) / (fb_med * 1e-3) / 1e9 / HBM_PEAK_GBS},
        "design_bytes": {"saved_states": sv_b,
                         "note": "chunk-entering states written by the forward and read by the backward; "
                                 "part of each call's traffic, not of its algorithmic bytes"},
        "wall_s_timed": res["wall"],
        "clock_settle": res["settle"],
    }
    if args.ste:
        sb = ste_bytes(w, s.C, real=args.real, bf16=args.bf16)
        out["fwd_bwd"] = None
        out["bwd"]["alg_bytes"] = sb["bwd_ste"]
        out["bwd"]["kernel"] = kern["bwd"] + " (+ z)"
        out["bwd"]["alg_GBps"] = sb["bwd_ste"] / (bwd_ms * 1e-3) / 1e9
        out["bwd"]["frac"] = out["bwd"]["alg_GBps"] / HBM_PEAK_GBS
        out["bwd"]["frac_median"] = sb["bwd_ste"] / (med("bwd") * 1e-3) / 1e9 / HBM_PEAK_GBS
        out["roofline"]["achieved"] = out["bwd"]["alg_GBps"] if dom == "bwd" else achieved
        out["roofline"]["frac"] = out["roofline"]["achieved"] / HBM_PEAK_GBS
        out["roofline"]["traffic"] = traffic_from_profiles("k_bwd_fused_ste" + suffix, w.name) if fused else None
        out["roofline"]["kernel"] = kern[dom] + (" (+ z)" if dom == "bwd" else "")
        if dom == "bwd":
            out["roofline"]["bytes"] = ("algorithmic: idx, dy, D, b, c in; dD, db, dc, z, dh0 out "
                                        "(%.1f + 8/N bytes per state update)"
                                        % (48.0 * esz / 8 + (4 if args.real else 8)))
        dg_ms, sm_ms = mean("ste_grads"), mean("softmax")
        gbps = sb["ste_grads"] / (dg_ms * 1e-3) / 1e9
        tfs = sb["ste_grads_flops"] / (dg_ms * 1e-3) / 1e12
        out["ste"] = {
            "temp": args.temp,
            "ste_grads": {"ms": dg_ms, "ms_median": med("ste_grads"), "alg_bytes": sb["ste_grads"],
                          "alg_GBps": gbps, "frac_hbm": gbps / HBM_PEAK_GBS, "flops": sb["ste_grads_flops"],
                          "TFLOPs": tfs, "frac_mfma_fp32": tfs / MFMA_FP32_PEAK_TFS,
                          "traffic": traffic_from_profiles("k_ste_gemm" + suffix, w.name)},
            "softmax_vjp": {"ms": sm_ms, "ms_median": med("softmax"), "alg_bytes": sb["softmax"],
                            "alg_GBps": sb["softmax"] / (sm_ms * 1e-3) / 1e9},
        }
    return out


if __name__ == "__main__":
    main()
