"""GPU parity of the fully recurrent forward (token by token, one launch)
against the fp64 oracle, and against the chunkwise forward on the same
inputs.  Tolerances as the chunk path: normwise 1e-4 (fp32), 2e-2 (bf16)."""
import pytest
import torch

from paper_2606_08804_amd import qdelta, synth
from tests.gpu_helpers import TOL, dev, f64, fwd_errors, gpu_fwd, normwise

pytestmark = pytest.mark.gpu


def rec_fwd(d, output_final_state=True):
    o, Sf = qdelta.recurrent_fwd(dev(d["q"]), dev(d["k"]), dev(d["v"]), dev(d["beta"]),
                                 dev(d["lam"]), dev(d["log_alpha"]), dev(d["initial_state"]),
                                 cu_seqlens=dev(d["cu_seqlens"]),
                                 output_final_state=output_final_state)
    torch.cuda.synchronize()
    return o, Sf


def _check(errs, tol, what):
    bad = {k: v for k, v in errs.items() if not (v <= tol)}
    assert not bad, f"{what}: {errs}"


@pytest.mark.parametrize("gate", ["G1", "G2", "G3"])
@pytest.mark.parametrize("dt,Dk,Dv", [("bf16", 128, 128), ("bf16", 128, 256), ("bf16", 64, 40),
                                      ("f32", 64, 64), ("f32", 128, 96)])
def test_recurrent_fwd_matches_oracle(gate, dt, Dk, Dv):
    d = synth.make(2, 150, 3, Dk, Dv, dt, gate, seed=141, s0=True)
    o, Sf = rec_fwd(d)
    _check(fwd_errors(d, o, Sf), TOL[dt], f"recurrent fwd {dt} {gate} Dk={Dk} Dv={Dv}")


def test_recurrent_fwd_varlen_and_optional_arguments():
    """Packed sequences with empty and one-token members, lambda == 0 (NULL),
    no decay, zero initial state, and no final state requested."""
    d = synth.make(1, 0, 2, 128, 128, "bf16", "G1", seed=142, lengths=[5, 0, 1, 130, 64])
    o, Sf = rec_fwd(d)
    _check(fwd_errors(d, o, Sf), TOL["bf16"], "recurrent fwd varlen")
    dn = dict(d, lam=None)
    o2, Sf2 = rec_fwd(dn, output_final_state=False)
    assert Sf2 is None
    d0 = dict(d, lam=torch.zeros_like(d["lam"]))
    o_ref = fwd_errors(d0, o2, torch.zeros(5, 2, 128, 128))["o"]
    assert o_ref <= TOL["bf16"]


def test_recurrent_fwd_equals_chunk_fwd():
    """Two GPU algorithms for the same recurrence (Sec. 3.3): token by token
    and chunkwise agree on a training-like shape."""
    d = synth.make(2, 1000, 4, 128, 128, "bf16", "G3", seed=143, s0=True)
    o_r, S_r = rec_fwd(d)
    o_c, S_c, _ = gpu_fwd(d)
    assert normwise(f64(o_r.cpu()), f64(o_c.cpu())) <= TOL["bf16"]
    assert normwise(f64(S_r.cpu()), f64(S_c.cpu())) <= TOL["bf16"]


def test_recurrent_fwd_empty_sequences_pass_state_through():
    d = synth.make(2, 0, 2, 64, 64, "bf16", "G2", seed=144, s0=True)
    o, Sf = rec_fwd(d)
    assert o.shape == (2, 0, 2, 64)
    assert torch.equal(Sf.cpu(), d["initial_state"])


def test_recurrent_fwd_at_training_shape():
    """B=4, T=4096, H=16, d=128, bf16, decay on, carried state: the
    recurrent forward equals the oracle on sampled heads and the chunk
    forward on every output."""
    from tests.gpu_helpers import select_heads
    d = synth.make(4, 4096, 16, 128, 128, "bf16", "G2", seed=145, s0=True)
    o_r, S_r = rec_fwd(d)
    o_c, S_c, _ = gpu_fwd(d)
    assert normwise(f64(o_r.cpu()), f64(o_c.cpu())) <= TOL["bf16"]
    assert normwise(f64(S_r.cpu()), f64(S_c.cpu())) <= TOL["bf16"]
    heads = [0, 11]
    ds = select_heads(d, heads)
    errs = fwd_errors(ds, o_r[:, :, heads].contiguous(), S_r[:, heads].contiguous())
    _check(errs, TOL["bf16"], "recurrent fwd at training shape (heads 0, 11)")


def test_recurrent_fwd_at_varlen_workload_size():
    """The packed workload (32768 tokens, lognormal lengths up to 8192, H=32,
    dk=128, dv=256, bf16): token by token equals chunkwise on every output."""
    d = synth.make(1, 0, 32, 128, 256, "bf16", "G2", seed=146, varlen_tokens=32768)
    o_r, S_r = rec_fwd(d)
    o_c, S_c, _ = gpu_fwd(d)
    assert normwise(f64(o_r.cpu()), f64(o_c.cpu())) <= TOL["bf16"]
    assert normwise(f64(S_r.cpu()), f64(S_c.cpu())) <= TOL["bf16"]
