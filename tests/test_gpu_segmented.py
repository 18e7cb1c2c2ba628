"""The segment-parallel forward (qdelta_chunk_fwd_segmented) against the
fp64 oracle and against the single-pass forward: several segment counts
including ones that do not divide the chunk count, a ragged last chunk,
every gate mode, fp32 and bf16, a saved context that the backward accepts,
and the long-context workload at full size (sampled heads)."""
import pytest
import torch

from paper_2606_08804_amd import qdelta, synth
from tests.gpu_helpers import (TOL, bwd_errors, dev, f64, fwd_errors, gpu_bwd, gpu_fwd, normwise,
                               oracle_fwd, select_heads)

pytestmark = pytest.mark.gpu


def seg_fwd(d, n_segments, save_states=False):
    o, Sf, saved = qdelta.chunk_fwd_segmented(dev(d["q"]), dev(d["k"]), dev(d["v"]), dev(d["beta"]),
                                              dev(d["lam"]), dev(d["log_alpha"]), dev(d["initial_state"]),
                                              n_segments=n_segments, save_states=save_states)
    torch.cuda.synchronize()
    return o, Sf, saved


@pytest.mark.parametrize("gate", ["G1", "G2", "G3"])
@pytest.mark.parametrize("G", [2, 3, 5, 16])
def test_segmented_bf16(gate, G):
    d = synth.make(2, 1000, 2, 128, 128, "bf16", gate, seed=170, s0=True)   # 16 chunks, the last ragged
    o, Sf, _ = seg_fwd(d, G)
    e = fwd_errors(d, o, Sf)
    assert all(v <= TOL["bf16"] for v in e.values()), (G, e)
    o1, Sf1, _ = gpu_fwd(d)
    assert normwise(f64(o.cpu()), f64(o1.cpu())) <= TOL["bf16"]


@pytest.mark.parametrize("Dv", [64, 128, 256])
def test_segmented_fp32(Dv):
    d = synth.make(1, 700, 2, 64, Dv, "f32", "G3", seed=171, s0=True)
    o, Sf, _ = seg_fwd(d, 4)
    e = fwd_errors(d, o, Sf)
    assert all(v <= TOL["f32"] for v in e.values()), (Dv, e)


@pytest.mark.parametrize("Dk,Dv", [(64, 64), (64, 256), (128, 64), (128, 256)])
def test_segmented_bf16_dims(Dk, Dv):
    d = synth.make(1, 900, 2, Dk, Dv, "bf16", "G3", seed=172, s0=True)
    o, Sf, _ = seg_fwd(d, 4)
    e = fwd_errors(d, o, Sf)
    assert all(v <= TOL["bf16"] for v in e.values()), (Dk, Dv, e)


def test_segmented_one_segment_is_the_single_pass():
    d = synth.make(2, 300, 2, 128, 128, "bf16", "G2", seed=173, s0=True)
    o, Sf, _ = seg_fwd(d, 1)
    o1, Sf1, _ = gpu_fwd(d)
    assert torch.equal(o, o1) and torch.equal(Sf, Sf1)


def test_segmented_saved_context_feeds_the_backward():
    d = synth.make(1, 800, 2, 128, 128, "bf16", "G3", seed=174, s0=True, with_do=True)
    o, Sf, saved = seg_fwd(d, 4, save_states=True)
    g = gpu_bwd(d, saved)
    e = bwd_errors(d, g)
    assert all(v <= TOL["bf16"] for v in e.values()), e


@pytest.mark.parametrize("gate", ["G1", "G2"])
def test_segmented_long_context_full(gate):
    """B=1, T=65536, H=16, d=128: four segments of 256 chunks; sampled heads
    against the oracle over all 65536 tokens."""
    d = synth.make_workload(4, gate)
    o, Sf, _ = seg_fwd(d, 4)
    heads = [0, 9]
    ds = select_heads(d, heads)
    o_ref, S_ref = oracle_fwd(ds)
    assert normwise(f64(o[:, :, heads].cpu()), o_ref) <= TOL["bf16"]
    assert normwise(f64(Sf[:, heads].cpu()), S_ref) <= TOL["bf16"]


def test_segmented_empty_inputs():
    """T = 0 passes the initial state through; B = 0 launches nothing."""
    d = synth.make(2, 0, 2, 128, 128, "bf16", "G2", seed=175, s0=True)
    o, Sf, _ = seg_fwd(d, 4)
    assert o.shape == (2, 0, 2, 128)
    assert torch.equal(Sf.cpu(), d["initial_state"])
    d0 = synth.make(0, 128, 2, 128, 128, "bf16", "G2", seed=176, s0=False)
    o0, Sf0, _ = seg_fwd(d0, 4)
    assert o0.shape == (0, 128, 2, 128) and Sf0.shape == (0, 2, 128, 128)
