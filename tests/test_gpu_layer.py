"""The autograd layer on the GPU (bf16 parameters and activations, HIP
recurrence) against the same layer in fp64 on the CPU with the recurrence
computed by the oracle: output and the gradients of the input and of every
parameter, normwise (max|got-ref|/max|ref|) within the bf16 tolerance; the
scalar gate-bias gradient, a sum over every (token, head), relative to the
sum of its summands' magnitudes."""
import copy

import pytest
import torch

from paper_2606_08804_amd import layer
from tests import oracle_binding
from tests.gpu_helpers import TOL, normwise

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("use_decay,varlen,fixed_lambda", [(True, False, None), (False, True, None),
                                                          (True, False, 0.0), (True, True, 0.5)])
def test_layer_matches_oracle_layer(monkeypatch, use_decay, varlen, fixed_lambda):
    torch.manual_seed(41)
    m = layer.QDeltaLayer(d_model=256, n_heads=2, head_dk=128, head_dv=128, use_decay=use_decay,
                          fixed_lambda=fixed_lambda)
    m = m.to(torch.bfloat16)
    ref = copy.deepcopy(m).double()
    g = torch.Generator().manual_seed(42)
    B, T = (1, 270) if varlen else (2, 150)
    h = torch.randn(B, T, 256, generator=g).to(torch.bfloat16)
    dy = torch.randn(B, T, 256, generator=g).to(torch.bfloat16)
    cu = torch.tensor([0, 70, 71, 270], dtype=torch.int32) if varlen else None

    mg = m.cuda()
    hg = h.cuda().requires_grad_()
    y = mg(hg, cu_seqlens=None if cu is None else cu.cuda())
    y.backward(dy.cuda())
    torch.cuda.synchronize()

    monkeypatch.setattr(layer, "_binding", oracle_binding)
    # the reference's lambda bias, broadcast to one copy per (token, head), so
    # that its gradient holds the summands of the scalar bias gradient
    if fixed_lambda is None:
        ref.lambda_bias = torch.nn.Parameter(ref.lambda_bias.detach().expand(B, T, ref.H).clone())
    hr = h.double().requires_grad_()
    yr = ref(hr, cu_seqlens=cu)
    yr.backward(dy.double())

    tol = TOL["bf16"]
    assert normwise(y.detach().cpu().double().numpy(), yr.detach().numpy()) <= tol
    assert normwise(hg.grad.cpu().double().numpy(), hr.grad.numpy()) <= tol
    for (name, p), (_, pr) in zip(mg.named_parameters(), ref.named_parameters()):
        if name == "lambda_bias":
            # a sum over every (token, head) with cancellation: its error is
            # measured against the sum of the summands' magnitudes
            terms = pr.grad
            err = abs(float(p.grad) - float(terms.sum())) / float(terms.abs().sum())
        else:
            err = normwise(p.grad.cpu().double().numpy(), pr.grad.numpy())
        assert err <= tol, (name, err)


def test_layer_continuation_with_carried_state():
    """Running a sequence in two calls, the second from the first's final
    state, equals one call over the whole sequence (output and final state)."""
    torch.manual_seed(43)
    m = layer.QDeltaLayer(d_model=256, n_heads=2, head_dk=128, head_dv=128).to(torch.bfloat16).cuda()
    g = torch.Generator().manual_seed(44)
    h = torch.randn(2, 200, 256, generator=g).to(torch.bfloat16).cuda()
    with torch.no_grad():
        y, S = m(h, output_final_state=True)
        y1, S1 = m(h[:, :77].contiguous(), output_final_state=True)
        y2, S2 = m(h[:, 77:].contiguous(), initial_state=S1, output_final_state=True)
    torch.cuda.synchronize()
    tol = TOL["bf16"]
    assert normwise(torch.cat([y1, y2], 1).float().cpu().numpy(), y.float().cpu().numpy()) <= tol
    assert normwise(S2.cpu().numpy(), S.cpu().numpy()) <= tol


@pytest.mark.parametrize("dt,D", [(torch.bfloat16, 128), (torch.bfloat16, 64), (torch.float32, 128),
                                  (torch.float32, 64)])
def test_l2norm_kernels_match_normalize(dt, D):
    """Row normalisation of a strided slice of a fused projection (1001 rows,
    one of them zero, so clamped) against F.normalize and its gradient in fp64."""
    from paper_2606_08804_amd import qdelta
    g = torch.Generator().manual_seed(45)
    fused = torch.randn(7, 11, 13, 2 * D + 64, generator=g)
    fused[3, 4, 5] = 0.0
    fused = fused.to(dt)
    dy = torch.randn(7, 11, 13, D, generator=g).to(dt)
    x_cpu = fused[..., D:2 * D]                         # the k slice: strided rows
    xr = x_cpu.double().requires_grad_()
    yr = torch.nn.functional.normalize(xr, dim=-1, eps=1e-12)
    yr.backward(dy.double())
    x = fused.cuda()[..., D:2 * D]
    y, rn = qdelta.l2norm_fwd(x)
    dx = qdelta.l2norm_bwd(y, rn, dy.cuda())
    torch.cuda.synchronize()
    tol = TOL["bf16"] if dt == torch.bfloat16 else TOL["f32"]
    assert normwise(y.double().cpu().numpy(), yr.detach().numpy()) <= tol
    assert normwise(dx.double().cpu().numpy(), xr.grad.numpy()) <= tol
    assert float(rn[3, 4, 5]) < 0 and torch.all(y[3, 4, 5] == 0)
