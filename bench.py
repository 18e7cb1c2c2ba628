"""Benchmark: chunkwise Q-Delta forward + backward on one MI355X.

A step is one pass of the whole hot path over one synthetic batch of the
training-step layer shape (B=4, T=4096, H=16, d_k=d_v=128, chunk 64, bf16
activations, fp32 gates and states): the chunk forward (writing the per-chunk
states) followed by the chunk backward.  Inputs are resident in HBM before the
timed region.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--gate G2] [--no-cpu]

`roofline` describes the kernel with the largest share of the step time; its
duration is measured live with HIP events recorded around each of its
launches on the launch stream.  `cpu_baseline` times the fp64 CPU oracle on a
bounded sample of the same workload on this host's cores.
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
MFMA_BF16_PEAK = 2.5e15    # flop/s, dense bf16 MFMA
METRIC = "Q-Delta chunk fwd+bwd tokens/s (T=4096,H=16,d=128,bf16); % MFMA peak"
C = 64


def fwd_flops_per_token_head(Dk, Dv):
    """Algorithmic forward flops per token and head: the three state-sized
    products (W S^T, Q S^T, D^T Kbar), the Gram and WY products and the causal
    halves of the chunk-local C x C work."""
    return 6 * Dk * Dv + C * (3 * Dk + 2 * Dv) + C * C / 3


def bwd_flops_per_token_head(Dk, Dv):
    return 2.5 * fwd_flops_per_token_head(Dk, Dv)


def stage_bytes_per_unit(stage, Dk, Dv, e):
    """Bytes one (chunk, head) unit of a kernel stage must move: every tensor
    it consumes or produces, counted once (activations e bytes, gates and
    states 4 bytes, workspace hand-offs in their stored precision)."""
    act_qk = C * Dk * e
    act_v = C * Dv * e
    gates = C * 4
    state = Dv * Dk * 4
    cc_e = C * C * e
    if stage in ("prep_fwd", "prep_bwd"):   # q, k, 3 gates -> gate block, P, M, T
        return 2 * act_qk + 3 * gates + 3 * gates + 3 * cc_e
    if stage == "scan_fwd":      # gate block, q, k, P, T, v -> o, state (dtype), D
        return 3 * gates + 2 * act_qk + 2 * cc_e + act_v + act_v + state * e // 4 + act_v
    if stage == "scan_bwd":      # gate block, P, M, k, q, dO -> dS' (dtype), dD, dv
        return 3 * gates + 2 * cc_e + 2 * act_qk + act_v + state * e // 4 + act_v + act_v
    if stage == "intra":         # gate block, S, dS' (dtype), D, dD, dO, v, q, k, M
        #                          -> dq, dk, dbeta, dlam, dlog_alpha
        return 3 * gates + 2 * state * e // 4 + 4 * act_v + 2 * act_qk + cc_e + 2 * act_qk + 3 * gates
    raise KeyError(stage)


def source_digest():
    """Digest of the kernel sources, to tell whether stored counters still apply."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_08804_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic(stage):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when there is none or the kernels changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "traffic_train_bf16_B4_T4096_H16_d128.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_digest") != source_digest():
        return None
    s = t.get("stages", {}).get(stage)
    return None if s is None else s.get("hbm_bytes_per_launch")


def cpu_baseline(d, units_sample, min_seconds=10.0):
    """Time the fp64 oracle (forward + backward) on a sample of the workload's
    (sequence, head) units, over the full sequence length."""
    from oracle import build as obuild
    from oracle import recurrent
    obuild.build(force=False)
    B, T, H = d["q"].shape[:3]
    heads = list(range(min(H, max(1, units_sample // B))))
    f = synth.to_f64
    sl = lambda x: None if x is None else x[:, :, heads].contiguous()
    q, k, v = f(sl(d["q"])), f(sl(d["k"])), f(sl(d["v"]))
    beta, lam, la = f(sl(d["beta"])), f(sl(d["lam"])), f(sl(d["log_alpha"]))
    S0 = None if d["initial_state"] is None else f(d["initial_state"][:, heads].contiguous())
    dO = f(sl(d["d_o"]))
    threads = recurrent.default_threads()
    # repeat the sample until about 10 s of CPU work have been timed
    reps, t0 = 0, time.perf_counter()
    while True:
        recurrent.fwd(q, k, v, beta, lam, la, S0, nthreads=threads)
        recurrent.bwd(q, k, v, beta, lam, la, S0, d_o=dO, nthreads=threads)
        reps += 1
        total = time.perf_counter() - t0
        if total >= min_seconds or reps >= 30:
            break
    dt = total / reps
    units = B * len(heads)
    tokens_per_s = (B * T) / (dt * (B * H) / units)
    return {"value": tokens_per_s, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"fp64 recurrence forward + BPTT backward of {units} of {B * H} (sequence, head) "
                      f"units over T={T}, {reps} passes in {total:.1f} s ({dt:.2f} s each), scaled to all units"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--gate", default="G2", choices=["G1", "G2", "G3"])
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
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

    w = synth.WORKLOADS[3]
    d = synth.make_workload(3, args.gate)
    dev = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in d.items()}
    B, T, H, Dk, Dv = w.B, w.T, w.H, w.Dk, w.Dv
    dt = qdelta.QDELTA_BF16
    wsf = torch.empty(qdelta.workspace_bytes(B, T, H, Dk, Dv, dt, 0, False), dtype=torch.uint8, device="cuda")
    wsb = torch.empty(qdelta.workspace_bytes(B, T, H, Dk, Dv, dt, 0, True), dtype=torch.uint8, device="cuda")
    args_in = (dev["q"], dev["k"], dev["v"], dev["beta"], dev["lam"], dev["log_alpha"], dev["initial_state"])

    def step():
        o, Sf, saved = qdelta.chunk_fwd(*args_in, save_states=True, workspace=wsf)
        g = qdelta.chunk_bwd(*args_in, saved, dev["d_o"], workspace=wsb)
        return o, g

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    qdelta.profile_begin()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        step()
    end.record()
    torch.cuda.synchronize()
    stages = qdelta.profile_end()
    ms = start.elapsed_time(end) / args.steps
    tokens = B * T
    value = tokens / (ms / 1e3)

    # dominant kernel and its roofline
    dom = max(stages, key=lambda s: stages[s][0])
    tot_ms, launches = stages[dom]
    avg_s = tot_ms / launches / 1e3
    units = qdelta.saved_state_slots(B, T) * H
    alg_bytes = stage_bytes_per_unit(dom, Dk, Dv, 2) * units
    achieved = alg_bytes / avg_s / 1e9
    traffic = stored_traffic(dom)
    roof = {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK / 1e9, "unit": "GB/s",
            "frac": achieved / (HBM_PEAK / 1e9), "traffic": traffic,
            "alg_bytes_per_launch": alg_bytes, "avg_launch_us": avg_s * 1e6}
    step_flops = tokens * H * (fwd_flops_per_token_head(Dk, Dv) + bwd_flops_per_token_head(Dk, Dv))
    breakdown = {s: round(v[0] / max(1, v[1]) * 1e3, 2) for s, v in stages.items() if v[1]}

    out = {
        "metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "B": B, "T": T, "H": H, "Dk": Dk, "Dv": Dv, "chunk": C,
                   "gate_mode": args.gate, "parallelism": "single GPU"},
        "mfma_frac_step": step_flops / (ms / 1e3) / MFMA_BF16_PEAK,
        "kernel_avg_us": breakdown,
        "roofline": roof,
    }
    if args.calib_copy > 0:
        src = torch.ones(args.calib_copy << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = args.calib_copy << 20
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(d, args.cpu_units)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
