"""Seeded synthetic inputs for the Q-Delta layer workloads.

This module only draws random numbers and casts them; it holds none of the
method's arithmetic, so both the GPU path and the CPU oracle may consume its
output.  Distributions follow the workload definitions used for parity and
measurement (language-model and long-context layer shapes):

* q, k ~ N(0, 1), L2-normalised over the head dimension, then cast.
* v ~ N(0, 1).
* beta = sigmoid(N(0, 1)) and lambda = sigmoid(N(0, 1)), per token per head, fp32.
* decay alpha per gate mode: "G1" alpha = 1 (log_alpha = None),
  "G2" alpha = sigmoid(N(0, 1)), "G3" alpha = sigmoid(N(4, 1)); handed over as
  fp32 log(alpha).
* initial state ~ N(0, 0.02^2) fp32 when requested, else None (zero).
* upstream dO ~ N(0, 1) in the activation dtype when requested.
* packed variable-length batches: lengths clip(round(exp(N(ln 1024, 1))), 64, 8192)
  drawn until they cover the token budget; the last length is the remainder,
  merged into the previous sequence when shorter than 64.

Every tensor comes from its own stream spawned from one SeedSequence in the
fixed order q, k, v, beta, lam, alpha, S0, dO, lengths, so adding a tensor never
shifts the others.
"""
from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

STREAMS = ("q", "k", "v", "beta", "lam", "alpha", "S0", "dO", "lengths")


@dataclass
class Workload:
    name: str
    B: int
    T: int
    H: int
    Dk: int
    Dv: int
    dtype: str                  # "f32" or "bf16"
    chunk: int = 64
    s0: bool = False
    bwd: bool = False
    varlen_tokens: int = 0      # > 0: packed variable-length batch of this many tokens
    seed: int = 0
    extra: dict = field(default_factory=dict)


# The five workloads (sizes as named by the benchmark definition).
WORKLOADS = {
    1: Workload("tiny-fp32 B1 T256 H2 d64", 1, 256, 2, 64, 64, "f32", seed=20260001),
    2: Workload("fwd-bf16 B8 T2048 H8 d128", 8, 2048, 8, 128, 128, "bf16", s0=True, seed=20260002),
    3: Workload("train-bf16 B4 T4096 H16 d128", 4, 4096, 16, 128, 128, "bf16", s0=True, bwd=True,
                seed=20260003),
    4: Workload("long-bf16 B1 T65536 H16 d128", 1, 65536, 16, 128, 128, "bf16", s0=True,
                seed=20260004, extra=dict(decode_N=64, decode_steps=1024)),
    5: Workload("varlen-bf16 32768 tok H32 dk128 dv256", 1, 32768, 32, 128, 256, "bf16", bwd=True,
                varlen_tokens=32768, seed=20260005),
}


def torch_dtype(name: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def _rngs(seed: int):
    ss = np.random.SeedSequence(seed)
    return {name: np.random.default_rng(s) for name, s in zip(STREAMS, ss.spawn(len(STREAMS)))}


def _unit(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _sigmoid(z: np.ndarray) -> np.ndarray:
    return 1.0 / (1.0 + np.exp(-z))


def varlen_lengths(rng: np.random.Generator, total: int, median: float = 1024.0,
                   sigma: float = 1.0, lo: int = 64, hi: int = 8192) -> list:
    lens = []
    acc = 0
    while acc < total:
        L = int(np.clip(np.round(np.exp(rng.normal(np.log(median), sigma))), lo, hi))
        if acc + L >= total:
            L = total - acc
        lens.append(L)
        acc += L
    if len(lens) > 1 and lens[-1] < lo:
        lens[-2] += lens.pop()
    return lens


def make(B: int, T: int, H: int, Dk: int, Dv: int, dtype: str = "bf16", gate_mode: str = "G2",
         seed: int = 0, s0: bool = False, with_do: bool = False, lengths: Optional[list] = None,
         varlen_tokens: int = 0, s0_std: float = 0.02) -> dict:
    """Draw one batch.

    Dense batches are ``[B, T, H, D]``.  When ``lengths`` is given, or
    ``varlen_tokens`` > 0 (lengths drawn from the lognormal recipe), the batch
    is packed as ``[1, Ttot, H, D]`` with ``cu_seqlens`` (int32, N+1).
    Returns a dict of CPU torch tensors (activations in ``dtype``, gates and
    states fp32) plus ``cu_seqlens`` and ``lengths`` (None when dense).
    """
    r = _rngs(seed)
    if varlen_tokens and lengths is None:
        lengths = varlen_lengths(r["lengths"], varlen_tokens)
    if lengths is not None:
        lengths = [int(x) for x in lengths]
        B, T = 1, int(sum(lengths))
    N = len(lengths) if lengths is not None else B
    td = torch_dtype(dtype)
    q = _unit(r["q"].standard_normal((B, T, H, Dk)).astype(np.float32))
    k = _unit(r["k"].standard_normal((B, T, H, Dk)).astype(np.float32))
    v = r["v"].standard_normal((B, T, H, Dv)).astype(np.float32)
    beta = _sigmoid(r["beta"].standard_normal((B, T, H))).astype(np.float32)
    lam = _sigmoid(r["lam"].standard_normal((B, T, H))).astype(np.float32)
    if gate_mode == "G1":
        log_alpha = None
    else:
        mean = {"G2": 0.0, "G3": 4.0}[gate_mode]
        z = r["alpha"].normal(mean, 1.0, (B, T, H))
        log_alpha = (-np.logaddexp(0.0, -z)).astype(np.float32)   # log sigmoid(z)
    S0 = (r["S0"].normal(0.0, s0_std, (N, H, Dv, Dk)).astype(np.float32) if s0 else None)
    dO = r["dO"].standard_normal((B, T, H, Dv)).astype(np.float32) if with_do else None
    out = dict(
        q=torch.from_numpy(q).to(td), k=torch.from_numpy(k).to(td), v=torch.from_numpy(v).to(td),
        beta=torch.from_numpy(beta), lam=torch.from_numpy(lam),
        log_alpha=None if log_alpha is None else torch.from_numpy(log_alpha),
        initial_state=None if S0 is None else torch.from_numpy(S0),
        d_o=None if dO is None else torch.from_numpy(dO).to(td),
        cu_seqlens=None, lengths=lengths,
    )
    if lengths is not None:
        cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
        out["cu_seqlens"] = torch.from_numpy(cu)
    return out


def make_workload(i: int, gate_mode: str = "G2") -> dict:
    w = WORKLOADS[i]
    return make(w.B, w.T, w.H, w.Dk, w.Dv, w.dtype, gate_mode, seed=w.seed, s0=w.s0,
                with_do=w.bwd, varlen_tokens=w.varlen_tokens)


def make_decode(N: int = 64, H: int = 16, D: int = 128, steps: int = 1024, dtype: str = "bf16",
                gate_mode: str = "G2", seed: int = 20260014, s0_std: float = 0.02) -> dict:
    """Inputs for `steps` successive single-token updates of N sequences."""
    d = make(steps, N, H, D, D, dtype, gate_mode, seed=seed, s0=False)
    r = _rngs(seed)
    S0 = r["S0"].normal(0.0, s0_std, (N, H, D, D)).astype(np.float32)
    d["initial_state"] = torch.from_numpy(S0)
    return d   # activations are [steps, N, H, D]: step s uses index s


def to_f64(t):
    """Exact widening of a CPU tensor to a float64 numpy array (None passes)."""
    return None if t is None else t.to(torch.float64).numpy()
