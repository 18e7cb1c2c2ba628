"""Benchmark: chunkwise Q-Delta on one MI355X.

The default workload (``--workload train``) is the training-step layer shape
(B=4, T=4096, H=16, d_k=d_v=128, chunk 64, bf16 activations, fp32 gates and
states).  A step is the chunk forward (writing the per-chunk saved context)
followed by the chunk backward.  Inputs are resident in HBM before the timed
region.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K=100] [--warmup W=20] [--gate G2] [--no-cpu]
                    [--workload train|fwd|long|decode|varlen|tiny]

The other workloads are the layer's other shapes: ``fwd`` (forward only,
B=8 T=2048 H=8 d=128), ``long`` (forward only, B=1 T=65536 H=16 d=128),
``decode`` (1024 successive single-token steps of 64 sequences, H=16 d=128;
a step of the benchmark is all 1024 of them), ``varlen`` (packed 32768 tokens,
lognormal lengths, H=32 d_k=128 d_v=256, forward + backward) and ``tiny``
(fp32 forward, B=1 T=256 H=2 d=64).

Timing: untimed steps for --settle-ms (GPU clock ramp-up), W warm-up steps,
then exactly K steps between two synchronisations with nothing else
recorded (`ms_per_step`, `value`); then K more steps with the library's HIP
events around every kernel launch on the launch stream, which give each
kernel's average launch duration.

Bytes: `step_alg_bytes` and every `alg_bytes_per_launch` count only the
mandated streams (inputs read once, outputs written once, per-chunk entry
states priced as fp32 through HBM; hand-offs between kernels excluded): 4900 B
per token-head for the training step at d = 128.  `roofline` is the kernel
with the largest share of the step; `traffic` is its HBM bytes per launch from
the committed FETCH_SIZE/WRITE_SIZE counter summary (null once the kernel
sources changed since it was taken).  `cpu_baseline` times the fp64 CPU oracle
on a bounded sample of the same workload on this host's cores; `parity`
compares the GPU outputs of the last timed step with that oracle run.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2606_08804_amd import qdelta, synth  # noqa: E402

HBM_PEAK = 8.0e12          # B/s, MI355X HBM3E
VALU_F32_PEAK = 157.3e12   # flop/s, MI355X fp32 vector (256 CUs x 2.4 GHz)
MFMA_BF16_PEAK = 2.5e15    # flop/s, dense bf16 MFMA
MFMA_F32_PEAK = 157.3e12   # flop/s, dense fp32 MFMA
C = 64
# committed FETCH_SIZE / WRITE_SIZE summaries, one per workload
TRAFFIC_FILES = {w: os.path.join(ROOT, "profiles", f"traffic_{w}.json")
                 for w in ("train", "fwd", "long", "decode", "varlen", "tiny", "recurrent")}


def fwd_flops_per_token_head(Dk, Dv):
    """Algorithmic forward flops per token and head: the three state-sized
    products (W S^T, Q S^T, D^T Kbar), the Gram and WY products and the causal
    halves of the chunk-local C x C work."""
    return 6 * Dk * Dv + C * (3 * Dk + 2 * Dv) + C * C / 3


def bwd_flops_per_token_head(Dk, Dv):
    return 2.5 * fwd_flops_per_token_head(Dk, Dv)


def alg_bytes_per_token_head(Dk, Dv, e, with_bwd, saved=True):
    """Algorithmic HBM bytes per token-head of a whole step: only the mandated
    streams, each counted once -- inputs read once, outputs written once, and
    the per-chunk entry states priced as fp32 going through HBM (written by the
    forward, read by the backward).  Hand-offs between kernels (the chunk
    factors T, P, M, the new values D, the exit-state gradients) are not
    algorithmic.  At Dk = Dv = 128 in bf16 this is 2060 B forward and
    2840 B backward, 4900 B per token-head in all."""
    qkv = (2 * Dk + Dv) * e
    gates = 3 * 4
    states = Dv * Dk * 4 / C
    fwd = qkv + gates + Dv * e + (states if saved else 0)
    if not with_bwd:
        return fwd
    bwd = qkv + Dv * e + gates + states + (2 * Dk + Dv) * e + gates
    return fwd + bwd


def kernel_alg_bytes_per_token_head(stage, Dk, Dv, e, saved=True):
    """The algorithmic streams of the per-step count that one kernel reads or
    writes itself (a stream that several kernels read counts for each of
    them; the gate block the preparation writes stands for the gates).
    Hand-offs are excluded as in alg_bytes_per_token_head."""
    qk = 2 * Dk * e
    v = Dv * e
    gates = 3 * 4
    states = Dv * Dk * 4 / C
    if stage in ("prep_fwd", "prep_bwd"):   # q, k, gates
        return qk + gates
    if stage == "scan_fwd":                 # q, k, v, gates -> o, entry states
        return qk + v + gates + v + (states if saved else 0)
    if stage == "scan_bwd":                 # q, k, dO, gates -> dv
        return qk + v + gates + v
    if stage == "intra":                    # q, k, v, dO, gates, entry states -> dq, dk, dgates
        return qk + 2 * v + gates + states + qk + gates
    if stage == "seg_maps":                 # q, k, v, gates (segment maps: hand-offs)
        return qk + v + gates
    if stage == "seg_out":                  # q, k, v, gates -> o
        return qk + v + gates + v
    if stage == "seg_compose":              # hand-offs only
        return 0
    raise KeyError(stage)


def kernel_state_io_bytes_per_seq(stage, Dk, Dv, has_s0):
    """Per (sequence, head) fp32 states a kernel moves once: the forward scan
    reads the initial state (when there is one) and writes the final state;
    the backward scan writes the initial-state gradient (the benchmark
    passes no final-state gradient)."""
    st = Dv * Dk * 4
    if stage == "scan_fwd":
        return (2 if has_s0 else 1) * st
    if stage == "scan_bwd":
        return st
    if stage == "seg_compose":              # reads the initial state
        return st if has_s0 else 0
    if stage == "seg_out":                  # writes the final state
        return st
    return 0


def handoff_bytes_per_unit(stage, Dk, Dv, e, saved=True):
    """Every byte a kernel moves per (chunk, head) unit, hand-offs included
    (activations e bytes, gates and states 4 bytes, hand-offs in their stored
    precision): the figure to compare with counter traffic."""
    act_qk = C * Dk * e
    act_v = C * Dv * e
    gates = C * 4
    state = Dv * Dk * 4
    cc_e = 10 * 256 * e          # C x C operators stored as their ten lower 16 x 16 blocks
    if stage in ("prep_fwd", "prep_bwd"):
        # q, k, 3 gates -> gate block, P, T (and M when the context is kept)
        return 2 * act_qk + 3 * gates + 3 * gates + (3 if saved else 2) * cc_e
    if stage == "scan_fwd":
        # gate block, q, k, P, T, v -> o (and the entry state in the
        # activation dtype and D when the context is kept)
        b = 3 * gates + 2 * act_qk + 2 * cc_e + act_v + act_v
        return b + (state * e // 4 + act_v if saved else 0)
    if stage == "scan_bwd":      # gate block, P, M, k, q, dO -> dS' (dtype), dv
        return 3 * gates + 2 * cc_e + 2 * act_qk + act_v + state * e // 4 + act_v
    if stage == "intra":         # gate block, S, dS' (dtype), D, dO, v, q, k, P, M
        #                          -> dq, dk, dbeta, dlam, dlog_alpha
        return 3 * gates + 2 * state * e // 4 + 3 * act_v + 2 * act_qk + 2 * cc_e + 2 * act_qk + 3 * gates
    if stage in ("seg_maps", "seg_out", "seg_compose"):
        return 0                 # per-segment figures, not per unit
    raise KeyError(stage)


# Sources of the kernels whose counters are stored: the kernel files and the
# workspace layout.  A stored summary applies only while they hash to the
# digest stored with it.
KERNEL_SOURCES = ("qd_api.hip", "qd_bwd.hip", "qd_common.h", "qd_fwd.hip", "qd_rec_bwd.hip", "qd_step.hip")


def strip_comments(src):
    """C++ source without its comments, trailing blanks and empty lines (string
    and character literals kept whole), so that editing a comment does not
    change the digest."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    lines = (l.rstrip() for l in "".join(out).split("\n"))
    return "\n".join(l for l in lines if l)


def source_digest():
    """Digest of the kernel sources' code (comments left out), to tell whether
    stored counters still apply."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_08804_amd", "csrc")
    for f in KERNEL_SOURCES:
        with open(os.path.join(csrc, f), encoding="utf-8") as fh:
            h.update(f.encode())
            h.update(strip_comments(fh.read()).encode())
    return h.hexdigest()[:16]


def stored_traffic(workload, stage):
    """HBM bytes per launch of a stage from the committed rocprofv3 counter
    summary of a workload, or None when there is none or the kernels changed
    since it was taken."""
    try:
        with open(TRAFFIC_FILES[workload]) as f:
            t = json.load(f)
    except (KeyError, OSError, ValueError):
        return None
    if t.get("source_digest") != source_digest():
        return None
    s = t.get("stages", {}).get(stage)
    return None if s is None else s.get("hbm_bytes_per_launch")


def host_info():
    """CPU count, the CPUs this process may run on, and the CPU model."""
    try:
        aff = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        aff = os.cpu_count()
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "affinity_cpus": aff, "cpu_model": model}


def cpu_baseline(d, heads, with_bwd, tokens_per_unit_run, min_seconds=10.0):
    """Time the fp64 oracle (forward, plus the BPTT backward when `with_bwd`)
    on the (sequence, head) units of `heads` over the full sequences, repeated
    until about `min_seconds` have been timed; scaled to tokens/s of the
    whole workload (every (sequence, head) unit costs the same per token).
    Also returns the oracle's outputs of the last pass, against which the
    benchmark checks the GPU's timed result."""
    from oracle import build as obuild
    from oracle import recurrent
    obuild.build(force=False)
    H = d["q"].shape[2]
    f = synth.to_f64
    sl = lambda x: None if x is None else x[:, :, heads].contiguous()
    pk = (lambda x: x) if d["cu_seqlens"] is None else (lambda x: None if x is None else x[0])
    q, k, v = pk(f(sl(d["q"]))), pk(f(sl(d["k"]))), pk(f(sl(d["v"])))
    beta, lam, la = pk(f(sl(d["beta"]))), pk(f(sl(d["lam"]))), pk(f(sl(d["log_alpha"])))
    S0 = None if d["initial_state"] is None else f(d["initial_state"][:, heads].contiguous())
    dO = pk(f(sl(d["d_o"]))) if with_bwd else None
    cu = None if d["cu_seqlens"] is None else d["cu_seqlens"].numpy()
    # the oracle's own thread count: one per CPU of this process, at most 16
    # (the host share of one GPU on the measurement machines)
    threads = recurrent.default_threads()
    reps, t0 = 0, time.perf_counter()
    while True:
        o_ref, S_ref = recurrent.fwd(q, k, v, beta, lam, la, S0, cu_seqlens=cu, nthreads=threads)
        g_ref = None
        if with_bwd:
            g_ref = recurrent.bwd(q, k, v, beta, lam, la, S0, d_o=dO, cu_seqlens=cu, nthreads=threads)
        reps += 1
        total = time.perf_counter() - t0
        if total >= min_seconds or reps >= 30:
            break
    dt = total / reps
    frac = len(heads) / H
    tokens_per_s = tokens_per_unit_run / (dt / frac)
    what = "forward + BPTT backward" if with_bwd else "forward"
    out = {"value": tokens_per_s, "unit": "tokens/s", "cores": threads, "kind": "oracle",
           "sample": f"fp64 recurrence {what} of {len(heads)} of {H} heads (all sequences, all tokens), "
                     f"{reps} passes in {total:.1f} s ({dt:.2f} s each), scaled to all heads",
           "threads_note": "one oracle thread per CPU available to this process, capped at 16 "
                           "(the host CPU share of one GPU)"}
    out.update(host_info())
    return out, {"o": o_ref, "final_state": S_ref, "grads": g_ref}


def normwise(got, ref):
    """max|got - ref| / max|ref| (absolute when the reference is all zero)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.abs(ref).max() if ref.size else 0.0
    err = np.abs(got - ref).max() if ref.size else 0.0
    return float(err / scale if scale > 0 else err)


def same_run_parity(d, heads, ref, got, dtype):
    """Compares the GPU outputs of the last timed step, restricted to `heads`,
    with the oracle outputs of the CPU baseline's last pass (normwise max
    error per tensor, the tolerance of the activation dtype)."""
    f = synth.to_f64
    packed = d["cu_seqlens"] is not None
    tol = 2e-2 if dtype == "bf16" else 1e-4

    def act(x):       # [B, T, H, ...] device tensor -> sampled heads as fp64
        x = x[:, :, heads].cpu()
        return f(x[0] if packed else x)

    errs = {"o": normwise(act(got["o"]), ref["o"]),
            "final_state": normwise(f(got["final_state"][:, heads].cpu()), ref["final_state"])}
    if ref["grads"] is not None:
        g = got["grads"]
        for key in ("dq", "dk", "dv", "dbeta", "dlam", "dlog_alpha"):
            if g.get(key) is not None:
                errs[key] = normwise(act(g[key]), ref["grads"][key])
        errs["d_initial_state"] = normwise(f(g["d_initial_state"][:, heads].cpu()),
                                           ref["grads"]["d_initial_state"])
    return {"heads": list(heads), "tolerance": tol, "max_err": max(errs.values()),
            "ok": all(v <= tol for v in errs.values()), "errors": errs}


def chunk_units(d, H):
    """(chunk, head) units the chunk kernels process."""
    if d["cu_seqlens"] is None:
        B, T = d["q"].shape[:2]
        return B * ((T + C - 1) // C) * H
    return sum((L + C - 1) // C for L in d["lengths"]) * H


def token_heads(d):
    return d["q"].shape[0] * d["q"].shape[1] * d["q"].shape[2]


def kernel_rooflines(stages, d, Dk, Dv, e, saved):
    """Per kernel: average launch duration (HIP events on the launch stream)
    and the HBM roofline of its algorithmic bytes (the mandated streams it
    touches, states priced as fp32); the hand-off-inclusive byte count is
    given beside it."""
    H = d["q"].shape[2]
    units = chunk_units(d, H)
    th = token_heads(d)
    nseq = (d["q"].shape[0] if d["cu_seqlens"] is None else len(d["lengths"])) * H
    has_s0 = d["initial_state"] is not None
    out = {}
    for s, (tot_ms, launches) in stages.items():
        if not launches:
            continue
        avg_s = tot_ms / launches / 1e3
        b = (kernel_alg_bytes_per_token_head(s, Dk, Dv, e, saved) * th
             + kernel_state_io_bytes_per_seq(s, Dk, Dv, has_s0) * nseq)
        bh = handoff_bytes_per_unit(s, Dk, Dv, e, saved) * units + kernel_state_io_bytes_per_seq(s, Dk, Dv, has_s0) * nseq
        out[s] = {"avg_launch_us": avg_s * 1e6, "alg_bytes_per_launch": int(b),
                  "achieved_GBps": b / avg_s / 1e9, "frac": b / avg_s / HBM_PEAK,
                  "bytes_incl_handoffs_per_launch": int(bh),
                  "GBps_incl_handoffs": bh / avg_s / 1e9}
    return out


def roofline_of(kern, dom, traffic):
    k = kern[dom]
    return {"bound": "hbm", "kernel": dom, "achieved": k["achieved_GBps"], "peak": HBM_PEAK / 1e9,
            "unit": "GB/s", "frac": k["frac"], "traffic": traffic,
            "alg_bytes_per_launch": k["alg_bytes_per_launch"], "avg_launch_us": k["avg_launch_us"]}


def settle(step, min_ms):
    """Untimed steps until `min_ms` of wall time have passed: the GPU's clocks
    ramp up over the first milliseconds of sustained work."""
    if min_ms <= 0:
        return 0
    n, t0 = 0, time.perf_counter()
    while True:
        step()
        n += 1
        if n % 4 == 0:
            torch.cuda.synchronize()
            if (time.perf_counter() - t0) * 1e3 >= min_ms:
                return n


def timed(step, steps, warmup, settle_ms):
    """Headline timing: W warm-up steps, then exactly K steps between two
    synchronisations, timed with events on the launch stream and no other
    instrumentation.  Then K more steps with the library's HIP events around
    every kernel launch, for the per-kernel durations."""
    n_settle = settle(step, settle_ms)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        step()
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    qdelta.profile_begin()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    stages = qdelta.profile_end()
    return ms, stages, n_settle


def run_chunk(args, wid, with_bwd):
    """Chunk forward (+ backward) workloads."""
    w = synth.WORKLOADS[wid]
    d = synth.make_workload(wid, args.gate)
    dev = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in d.items()}
    B, T, H, Dk, Dv = d["q"].shape[0], d["q"].shape[1], w.H, w.Dk, w.Dv
    cu = dev["cu_seqlens"]
    n_seqs = 0 if cu is None else len(d["lengths"])
    dt = qdelta.QDELTA_BF16 if w.dtype == "bf16" else qdelta.QDELTA_F32
    e = 2 if w.dtype == "bf16" else 4
    wsf = torch.empty(max(1, qdelta.workspace_bytes(B, T, H, Dk, Dv, dt, n_seqs, False)), dtype=torch.uint8,
                      device="cuda")
    wsb = torch.empty(max(1, qdelta.workspace_bytes(B, T, H, Dk, Dv, dt, n_seqs, True)), dtype=torch.uint8,
                      device="cuda")
    args_in = (dev["q"], dev["k"], dev["v"], dev["beta"], dev["lam"], dev["log_alpha"], dev["initial_state"])
    last = {}

    # forward-only dense batches run the segment-parallel form when the
    # library suggests more than one segment (long sequences, few heads)
    n_seg = 1 if (with_bwd or cu is not None) else qdelta.suggest_segments(B, T, H, Dk, Dv, dt)
    single_ms = None
    if with_bwd:
        def step():
            o, Sf, saved = qdelta.chunk_fwd(*args_in, cu_seqlens=cu, save_states=True, workspace=wsf)
            g = qdelta.chunk_bwd(*args_in, saved, dev["d_o"], cu_seqlens=cu, workspace=wsb)
            last.update(o=o, final_state=Sf, grads=g)
    elif n_seg > 1:
        wss = torch.empty(qdelta.segmented_workspace_bytes(B, T, H, Dk, Dv, dt, n_seg), dtype=torch.uint8,
                          device="cuda")

        def step():
            o, Sf, _ = qdelta.chunk_fwd_segmented(*args_in, n_segments=n_seg, workspace=wss)
            last.update(o=o, final_state=Sf)

        single_ms, _, _ = timed(lambda: qdelta.chunk_fwd(*args_in, save_states=False, workspace=wsf),
                                args.steps, args.warmup, args.settle_ms)
    else:
        def step():
            o, Sf, _ = qdelta.chunk_fwd(*args_in, cu_seqlens=cu, save_states=False, workspace=wsf)
            last.update(o=o, final_state=Sf)

    ms, stages, n_settle = timed(step, args.steps, args.warmup, args.settle_ms)
    tokens = B * T
    th = tokens * H
    value = tokens / (ms / 1e3)
    kern = kernel_rooflines(stages, d, Dk, Dv, e, with_bwd)
    dom = max(kern, key=lambda s: kern[s]["avg_launch_us"])
    wname = {v: k for k, v in WORKLOAD_IDS.items()}[wid]
    traffic = stored_traffic(wname, dom)
    fl = fwd_flops_per_token_head(Dk, Dv) + (bwd_flops_per_token_head(Dk, Dv) if with_bwd else 0)
    peak = MFMA_BF16_PEAK if w.dtype == "bf16" else MFMA_F32_PEAK
    nseq = (B if n_seqs == 0 else n_seqs) * H
    has_s0 = d["initial_state"] is not None
    state_io = sum(kernel_state_io_bytes_per_seq(s, Dk, Dv, has_s0) for s in ("scan_fwd", "scan_bwd")
                   if with_bwd or s == "scan_fwd") * nseq
    bpth = alg_bytes_per_token_head(Dk, Dv, e, with_bwd, saved=with_bwd)
    step_bytes = bpth * th + state_io
    what = "fwd+bwd" if with_bwd else "fwd"
    shape = (f"T={T},H={H},d={Dk},bf16" if wid == 3 else
             f"{w.name.split(' ', 1)[1]}")
    metric = ("Q-Delta chunk fwd+bwd tokens/s (T=4096,H=16,d=128,bf16); % MFMA peak" if wid == 3 else
              f"Q-Delta chunk {what} tokens/s ({shape})")
    cfg = {"workload": w.name, "B": B, "T": T, "H": H, "Dk": Dk, "Dv": Dv, "chunk": C,
           "gate_mode": args.gate, "parallelism": "single GPU"}
    if n_seqs:
        cfg["n_seqs"] = n_seqs
    if n_seg > 1:
        cfg["segments"] = n_seg
    step_traffic = None
    per = [stored_traffic(wname, s) for s in kern]
    if all(x is not None for x in per):
        step_traffic = int(sum(x * stages[s][1] / args.steps for x, s in zip(per, kern)))
    out = {
        "metric": metric, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic", "config": cfg,
        "clock_settle_steps": n_settle,
        "single_pass_ms_per_step": single_ms,
        "mfma_frac_step": th * fl / (ms / 1e3) / peak,
        "step_alg_bytes": {"per_token_head": bpth, "state_io": state_io, "total": int(step_bytes),
                           "GBps": step_bytes / (ms / 1e3) / 1e9,
                           "hbm_frac": step_bytes / (ms / 1e3) / HBM_PEAK,
                           "counter_traffic": step_traffic,
                           "traffic_over_alg": None if step_traffic is None else step_traffic / step_bytes},
        "kernel_avg_us": {s: round(k["avg_launch_us"], 2) for s, k in kern.items()},
        "kernels": kern,
        "roofline": roofline_of(kern, dom, traffic),
    }
    if not args.no_cpu:
        nh = H if wid in (1, 4) else max(1, min(H, args.cpu_units // max(1, B if n_seqs == 0 else 1)))
        if wid == 5:
            nh = 2
        heads = list(range(nh))
        cb, ref = cpu_baseline(d, heads, with_bwd, tokens)
        out["cpu_baseline"] = cb
        out["parity"] = same_run_parity(d, heads, ref, last, w.dtype)
    return out


def run_layer(args):
    """The autograd layer (gate and q/k/v/output projections + the chunk
    kernels) forward and backward at the training shape: B=4, T=4096,
    d_model = H*d = 2048, H=16, d=128, bf16 parameters and activations."""
    from paper_2606_08804_amd import layer
    B, T, H, d = 4, 4096, 16, 128
    torch.manual_seed(0)
    m = layer.QDeltaLayer(d_model=H * d, n_heads=H, head_dk=d, head_dv=d).to(torch.bfloat16).cuda()
    g = torch.Generator(device="cuda").manual_seed(1)
    h = torch.randn(B, T, H * d, device="cuda", generator=g).to(torch.bfloat16).requires_grad_()
    dy = torch.randn(B, T, H * d, device="cuda", generator=g).to(torch.bfloat16)

    def step():
        m.zero_grad(set_to_none=True)
        h.grad = None
        m(h).backward(dy)

    ms, stages, n_settle = timed(step, args.steps, args.warmup, args.settle_ms)
    tokens = B * T
    dd = {"q": torch.empty(B, T, H, 0), "cu_seqlens": None, "initial_state": None}
    kern = kernel_rooflines(stages, dd, d, d, 2, True)
    dom = max(kern, key=lambda s: kern[s]["avg_launch_us"])
    core_ms = sum(k["avg_launch_us"] * stages[s][1] for s, k in kern.items()) / 1e3 / args.steps
    D = H * d
    gemm_flops = 3 * 2 * tokens * D * (H * (3 * d) + 3 * H + H * d)   # fwd + two bwd products
    return {
        "metric": f"Q-Delta layer fwd+bwd tokens/s (B={B},T={T},d_model={D},H={H},d={d},bf16)",
        "value": tokens / (ms / 1e3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"layer bf16 B={B} T={T} d_model={D} H={H} d={d} (decay on)",
                   "parallelism": "single GPU"},
        "clock_settle_steps": n_settle,
        "qdelta_kernels_ms_per_step": core_ms,
        "other_ms_per_step": ms - core_ms,
        "projection_gemm_tflops_per_step": gemm_flops / 1e12,
        "kernel_avg_us": {s: round(k["avg_launch_us"], 2) for s, k in kern.items()},
        "kernels": kern,
        # counters were taken on the chunk-kernel benchmark, not on this workload
        "roofline": roofline_of(kern, dom, None),
    }


def run_recurrent(args):
    """The fully recurrent form on short continuing sequences (64 sequences
    from a carried state, H=16, d=128, bf16) at T = 16 tokens: forward, and
    forward + backward as a training step, each with the chunkwise form on
    the same input timed beside it; both again at T = 4 and T = 64 to show
    where the two forms cross over."""
    B, H, d, T_main = 64, 16, 128, 16
    by_T = {}
    main = None
    for T in (4, 16, 64):
        dd = synth.make(B, T, H, d, d, "bf16", args.gate, seed=20260007, s0=True, with_do=True)
        g = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in dd.items()}
        ins = (g["q"], g["k"], g["v"], g["beta"], g["lam"], g["log_alpha"], g["initial_state"])
        wsf = torch.empty(max(1, qdelta.workspace_bytes(B, T, H, d, d, qdelta.QDELTA_BF16, 0, False)),
                          dtype=torch.uint8, device="cuda")
        wsb = torch.empty(max(1, qdelta.workspace_bytes(B, T, H, d, d, qdelta.QDELTA_BF16, 0, True)),
                          dtype=torch.uint8, device="cuda")
        wsr = torch.empty(qdelta.recurrent_workspace_bytes(B, T, H, d, d), dtype=torch.uint8, device="cuda")

        def rec_train():
            qdelta.recurrent_fwd(*ins)
            qdelta.recurrent_bwd(*ins, g["d_o"], workspace=wsr)

        def chunk_train():
            _, _, saved = qdelta.chunk_fwd(*ins, save_states=True, workspace=wsf)
            qdelta.chunk_bwd(*ins, saved, g["d_o"], workspace=wsb)

        ms, stages, _ = timed(lambda: qdelta.recurrent_fwd(*ins), args.steps, args.warmup, args.settle_ms)
        ms_chunk, _, _ = timed(lambda: qdelta.chunk_fwd(*ins, save_states=False, workspace=wsf),
                               args.steps, args.warmup, 0)
        ms_tr, st_tr, _ = timed(rec_train, args.steps, args.warmup, 0)
        ms_ctr, _, _ = timed(chunk_train, args.steps, args.warmup, 0)
        by_T[T] = {"recurrent_fwd_ms": ms, "chunk_fwd_ms": ms_chunk,
                   "recurrent_fwd_bwd_ms": ms_tr, "chunk_fwd_bwd_ms": ms_ctr,
                   "recurrent_bwd_kernel_us": st_tr["rec_bwd"][0] / st_tr["rec_bwd"][1] * 1e3}
        if T == T_main:
            tot, launches = stages["rec_fwd"]
            btot, blaunch = st_tr["rec_bwd"]
            main = (ms, tot / launches / 1e3, ms_chunk, ms_tr, btot / blaunch / 1e3, ms_ctr)
    ms, avg_s, ms_chunk, ms_tr, avg_b, ms_ctr = main
    T = T_main
    # ALU roofline: forward 6 Dk Dv flops per token-head (S x and S q dot
    # products, rank-1 update); backward 22 Dk Dv (three sweeps: 6 + 8 + 8)
    flops = B * T * H * 6 * d * d
    bflops = B * T * H * 22 * d * d
    kern = {"rec_fwd": {"avg_launch_us": avg_s * 1e6, "alg_flops_per_launch": flops,
                        "achieved_TFLOPs": flops / avg_s / 1e12, "frac": flops / avg_s / VALU_F32_PEAK},
            "rec_bwd": {"avg_launch_us": avg_b * 1e6, "alg_flops_per_launch": bflops,
                        "achieved_TFLOPs": bflops / avg_b / 1e12, "frac": bflops / avg_b / VALU_F32_PEAK}}
    return {
        "metric": f"Q-Delta recurrent fwd tokens/s (B={B},T={T},H={H},d={d},bf16, carried state)",
        "value": B * T / (ms / 1e3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"recurrent fwd bf16 B={B} T={T} H={H} d={d} with initial state",
                   "gate_mode": args.gate, "parallelism": "single GPU"},
        "chunk_fwd_ms_same_input": ms_chunk,
        "recurrent_fwd_bwd_tokens_per_s": B * T / (ms_tr / 1e3), "recurrent_fwd_bwd_ms": ms_tr,
        "chunk_fwd_bwd_ms_same_input": ms_ctr,
        "by_T": by_T,
        "kernel_avg_us": {k: round(v["avg_launch_us"], 2) for k, v in kern.items()},
        "kernels": kern,
        "roofline": {"bound": "alu", "kernel": "rec_fwd", "achieved": flops / avg_s / 1e12,
                     "peak": VALU_F32_PEAK / 1e12, "unit": "TFLOP/s", "frac": flops / avg_s / VALU_F32_PEAK,
                     "traffic": None, "avg_launch_us": avg_s * 1e6},
    }


def run_decode(args):
    """1024 successive single-token updates of 64 sequences (H=16, d=128)."""
    wl = synth.WORKLOADS[4]
    N, steps_dec = wl.extra["decode_N"], wl.extra["decode_steps"]
    H, D = wl.H, wl.Dk
    d = synth.make_decode(N, H, D, steps_dec, gate_mode=args.gate)
    q, k, v = d["q"].cuda(), d["k"].cuda(), d["v"].cuda()
    beta, lam = d["beta"].cuda(), d["lam"].cuda()
    la = d["log_alpha"].cuda() if d["log_alpha"] is not None else None
    S0 = d["initial_state"].cuda()
    S = S0.clone()
    outs = torch.empty((steps_dec, N, H, D), dtype=torch.bfloat16, device="cuda")

    def decode_all():
        for s in range(steps_dec):
            qdelta.recurrent_step(q[s], k[s], v[s], beta[s], lam[s], None if la is None else la[s], S,
                                  out=outs[s])

    def eager_step():
        S.copy_(S0)
        decode_all()

    # the 1024 launches of a step captured once into a HIP graph (a serving
    # loop's form: no host launch per token); the state reset stays outside
    # the graph as ordinary stream work
    torch.cuda.synchronize()
    S.copy_(S0)
    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        decode_all()                      # one eager pass on the capture stream before capturing
        torch.cuda.synchronize()
        S.copy_(S0)
        with torch.cuda.graph(graph, stream=cap):
            decode_all()
    torch.cuda.current_stream().wait_stream(cap)
    torch.cuda.synchronize()

    def graph_step():
        S.copy_(S0)
        graph.replay()

    # a benchmark step here is 1024 decode steps (tens of milliseconds)
    ms, stages, n_settle = timed(eager_step, min(args.steps, 10), min(args.warmup, 3), args.settle_ms)
    ms_graph, _, _ = timed(graph_step, min(args.steps, 10), min(args.warmup, 3), 0)
    tokens = N * steps_dec
    tot_ms, launches = stages["step"]
    avg_s = tot_ms / launches / 1e3
    b = N * H * (2 * D * D * 4 + 4 * D * 2 + 3 * 4)
    kern = {"step": {"avg_launch_us": avg_s * 1e6, "alg_bytes_per_launch": b,
                     "achieved_GBps": b / avg_s / 1e9, "frac": b / avg_s / HBM_PEAK}}
    out = {
        "metric": "Q-Delta recurrent decode tokens/s (64 seqs x 1024 steps, H=16, d=128, bf16)",
        "value": tokens / (ms / 1e3), "unit": "tokens/s", "n_gpus": 1, "steps": min(args.steps, 10),
        "warmup": min(args.warmup, 3), "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "decode 64 seqs x 1024 steps H16 d128", "N": N, "H": H, "Dk": D, "Dv": D,
                   "decode_steps": steps_dec, "gate_mode": args.gate, "parallelism": "single GPU",
                   "note": "a benchmark step is all 1024 decode steps (one launch each) plus one state reset "
                           "copy; graph_* is the same step replayed from a captured HIP graph"},
        "clock_settle_steps": n_settle,
        "us_per_decode_step": ms * 1e3 / steps_dec,
        "graph_ms_per_step": ms_graph,
        "graph_us_per_decode_step": ms_graph * 1e3 / steps_dec,
        "kernel_avg_us": {"step": round(avg_s * 1e6, 2)},
        "kernels": kern,
        "roofline": roofline_of(kern, "step", stored_traffic("decode", "step")),
    }
    if not args.no_cpu:
        from oracle import build as obuild
        from oracle import recurrent
        obuild.build(force=False)
        f = synth.to_f64
        nseq = 16
        ref = {key: f(d[key][:, :nseq].transpose(0, 1).contiguous()) for key in ("q", "k", "v", "beta", "lam")}
        lar = None if d["log_alpha"] is None else f(d["log_alpha"][:, :nseq].transpose(0, 1).contiguous())
        S0r = f(d["initial_state"][:nseq])
        threads = recurrent.default_threads()
        reps, t0 = 0, time.perf_counter()
        while True:
            o_ref, S_ref = recurrent.fwd(ref["q"], ref["k"], ref["v"], ref["beta"], ref["lam"], lar, S0r,
                                         nthreads=threads)
            reps += 1
            total = time.perf_counter() - t0
            if total >= 10.0 or reps >= 30:
                break
        dt = total / reps
        out["cpu_baseline"] = {
            "value": nseq * steps_dec / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"fp64 recurrence over the same 1024 tokens for {nseq} of {N} sequences (all {H} heads), "
                      f"{reps} passes in {total:.1f} s ({dt:.2f} s each)",
            "threads_note": "one oracle thread per CPU available to this process, capped at 16 "
                            "(the host CPU share of one GPU)"}
        out["cpu_baseline"].update(host_info())
        # the timed steps' outputs (every step recomputes the same 1024 tokens from S0)
        errs = {"o": normwise(f(outs[:, :nseq].transpose(0, 1).cpu()), o_ref),
                "final_state": normwise(f(S[:nseq].cpu()), S_ref)}
        out["parity"] = {"sequences": list(range(nseq)), "tolerance": 2e-2, "max_err": max(errs.values()),
                         "ok": all(x <= 2e-2 for x in errs.values()), "errors": errs}
    return out


def run_segments(args):
    """The segment-parallel forward against the single pass on long
    sequences: B=1, T=65536, d=128, bf16, at H = 16 (the long-context
    workload), 4 and 2, for 1 (the single pass), 2, 4, 8 and 16 segments;
    `value` is the long-context workload with the library's suggested
    segment count."""
    T, d = 65536, 128
    out_by_H = {}
    main = None
    for H in (16, 4, 2):
        dd = synth.make(1, T, H, d, d, "bf16", args.gate, seed=20260004, s0=True)
        g = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in dd.items()}
        ins = (g["q"], g["k"], g["v"], g["beta"], g["lam"], g["log_alpha"], g["initial_state"])
        sugg = qdelta.suggest_segments(1, T, H, d, d)
        res = {}
        for G in (1, 2, 4, 8, 16):
            ws = torch.empty(qdelta.segmented_workspace_bytes(1, T, H, d, d, qdelta.QDELTA_BF16, G),
                             dtype=torch.uint8, device="cuda")
            ms, _, _ = timed(lambda: qdelta.chunk_fwd_segmented(*ins, n_segments=G, workspace=ws),
                             args.steps, args.warmup, args.settle_ms if G == 1 else 0)
            res[G] = ms
        out_by_H[H] = {"ms_by_segments": res, "suggested": sugg, "best": min(res, key=res.get)}
        if H == 16:
            main = (res[sugg], sugg)
    ms, sugg = main
    return {
        "metric": "Q-Delta chunk fwd tokens/s (B=1,T=65536,H=16,d=128,bf16), suggested segments",
        "value": T / (ms / 1e3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "long-context forward B1 T65536 d128, H 16 / 4 / 2, segment sweep",
                   "gate_mode": args.gate, "parallelism": "single GPU", "segments_used": sugg},
        "by_heads": out_by_H,
    }


WORKLOAD_IDS = {"train": 3, "fwd": 2, "long": 4, "varlen": 5, "tiny": 1}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # the GPU's clocks settle over the first few milliseconds of work: 20
    # warm-up steps, then 100 timed steps (about 60 ms at the training shape)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--gate", default="G2", choices=["G1", "G2", "G3"])
    ap.add_argument("--workload", default="train",
                    choices=["train", "fwd", "long", "decode", "varlen", "tiny", "layer", "recurrent", "segments"])
    ap.add_argument("--no-cpu", action="store_true",
                    help="skip the CPU oracle baseline (and with it the same-run parity check)")
    ap.add_argument("--settle-ms", type=float, default=200.0,
                    help="untimed steps for this long before the warm-up steps (GPU clock ramp-up)")
    ap.add_argument("--cpu-units", type=int, default=64)
    ap.add_argument("--calib-copy", type=int, default=0, metavar="MIB",
                    help="after the run, copy a MIB-MiB device buffer three times (outside the timed "
                         "region) so that a counter profile holds a plain copy of known size")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the layer shards over (sequence, head) units with no exchange)", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)

    if args.workload == "decode":
        out = run_decode(args)
    elif args.workload == "layer":
        out = run_layer(args)
    elif args.workload == "recurrent":
        out = run_recurrent(args)
    elif args.workload == "segments":
        out = run_segments(args)
    else:
        wid = WORKLOAD_IDS[args.workload]
        out = run_chunk(args, wid, synth.WORKLOADS[wid].bwd)
    if args.calib_copy > 0:
        src = torch.ones(args.calib_copy << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = args.calib_copy << 20
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
