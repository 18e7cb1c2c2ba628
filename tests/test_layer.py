"""The autograd layer's wiring, on the CPU, with the library binding replaced
by the fp64 oracle (tests/oracle_binding.py): torch.autograd.gradcheck
compares the layer's analytic gradients (oracle backward + the chain rule
through projections, L2 norms and gate nonlinearities) with central
differences of its forward.  The GPU layer itself is tested in
tests/test_gpu_layer.py."""
import math

import pytest
import torch

from paper_2606_08804_amd import layer
from tests import oracle_binding


@pytest.fixture
def oracle_core(monkeypatch):
    monkeypatch.setattr(layer, "_binding", oracle_binding)


def _inputs(B, T, H, dk, dv, seed, with_lam=True, with_decay=True, s0=True):
    g = torch.Generator().manual_seed(seed)
    q = torch.nn.functional.normalize(torch.randn(B, T, H, dk, generator=g, dtype=torch.float64), dim=-1)
    k = torch.nn.functional.normalize(torch.randn(B, T, H, dk, generator=g, dtype=torch.float64), dim=-1)
    v = torch.randn(B, T, H, dv, generator=g, dtype=torch.float64)
    beta = torch.sigmoid(torch.randn(B, T, H, generator=g, dtype=torch.float64))
    lam = torch.sigmoid(torch.randn(B, T, H, generator=g, dtype=torch.float64)) if with_lam else None
    la = torch.nn.functional.logsigmoid(torch.randn(B, T, H, generator=g, dtype=torch.float64) + 2) \
        if with_decay else None
    S0 = 0.1 * torch.randn(B, H, dv, dk, generator=g, dtype=torch.float64) if s0 else None
    return [q, k, v, beta, lam, la, S0]


@pytest.mark.parametrize("with_lam,with_decay", [(True, True), (False, True), (True, False)])
def test_function_gradcheck(oracle_core, with_lam, with_decay):
    xs = _inputs(1, 7, 2, 3, 4, seed=1, with_lam=with_lam, with_decay=with_decay)
    xs = [None if x is None else x.requires_grad_() for x in xs]
    live = [i for i, x in enumerate(xs) if x is not None]

    def f(*args):
        full = list(xs)
        for i, a in zip(live, args):
            full[i] = a
        o, Sf = layer.qdelta_chunk(*full)
        return o, Sf

    assert torch.autograd.gradcheck(f, [xs[i] for i in live], eps=1e-6, atol=1e-7, rtol=1e-6)


def test_function_gradcheck_varlen(oracle_core):
    xs = _inputs(1, 9, 1, 3, 3, seed=2)
    xs[6] = 0.1 * torch.randn(3, 1, 3, 3, dtype=torch.float64)
    cu = torch.tensor([0, 4, 4, 9], dtype=torch.int32)
    xs = [x.requires_grad_() for x in xs]

    def f(*args):
        return layer.qdelta_chunk(*args, cu_seqlens=cu)

    assert torch.autograd.gradcheck(f, xs, eps=1e-6, atol=1e-7, rtol=1e-6)


@pytest.mark.parametrize("use_decay,fixed_lambda", [(True, None), (False, None), (True, 0.5), (True, 0.0)])
def test_layer_gradcheck(oracle_core, use_decay, fixed_lambda):
    torch.manual_seed(3)
    m = layer.QDeltaLayer(d_model=6, n_heads=2, head_dk=3, head_dv=4, use_decay=use_decay,
                          fixed_lambda=fixed_lambda).double()
    h = torch.randn(2, 5, 6, dtype=torch.float64, requires_grad=True)
    params = list(m.parameters())

    names = [n for n, _ in m.named_parameters()]

    def f(h, *ps):
        return torch.func.functional_call(m, dict(zip(names, ps)), (h,))

    assert torch.autograd.gradcheck(f, [h] + [p.detach().clone().requires_grad_() for p in params],
                                    eps=1e-6, atol=1e-7, rtol=1e-6)


def test_lambda_gate_at_initialisation():
    """lambda = sigmoid(W_lambda h + b), b a scalar initialised to -0.8: at
    h = 0 every head's lambda is sigmoid(-0.8); beta = 1/2; alpha = 1/2."""
    m = layer.QDeltaLayer(d_model=8, n_heads=4, head_dk=4, head_dv=4)
    beta, lam, log_alpha = m.gates(torch.zeros(1, 3, 8))
    assert torch.allclose(lam, torch.full_like(lam, 1 / (1 + math.exp(0.8))))
    assert torch.allclose(beta, torch.full_like(beta, 0.5))
    assert torch.allclose(log_alpha, torch.full_like(log_alpha, math.log(0.5)))


def test_layer_has_no_cpu_path():
    """The product layer never computes the recurrence on the CPU."""
    m = layer.QDeltaLayer(d_model=8, n_heads=2, head_dk=64, head_dv=64)
    with pytest.raises((ValueError, OSError, RuntimeError)):
        m(torch.randn(1, 4, 8))


def test_fixed_lambda_variants():
    """The paper's ablations as layer settings: a constant lambda is handed
    to the kernels as a number (no lambda tensor; 0 is the gated delta rule),
    and no decay as a NULL log alpha; the gate projection has one block per
    learned gate."""
    h = torch.randn(1, 3, 8)
    m = layer.QDeltaLayer(d_model=8, n_heads=2, head_dk=4, head_dv=4, fixed_lambda=0.8)
    beta, lam, la = m.gates(h)
    assert lam == 0.8 and isinstance(lam, float) and la is not None
    assert m.w_gates.out_features == 4 and not hasattr(m, "lambda_bias")
    m0 = layer.QDeltaLayer(d_model=8, n_heads=2, head_dk=4, head_dv=4, fixed_lambda=0, use_decay=False)
    beta, lam, la = m0.gates(h)
    assert lam == 0.0 and la is None and m0.w_gates.out_features == 2


def test_function_constant_lambda_gradcheck(oracle_core):
    """A constant lambda given as a number: gradients of every tensor input
    through the autograd function, and equal outputs to the same constant
    given as a filled tensor."""
    xs = _inputs(1, 6, 2, 3, 4, seed=5)
    lam_c = 0.5
    o_t, S_t = layer.qdelta_chunk(*xs[:4], torch.full_like(xs[3], lam_c), *xs[5:])
    o_c, S_c = layer.qdelta_chunk(*xs[:4], lam_c, *xs[5:])
    assert torch.equal(o_t, o_c) and torch.equal(S_t, S_c)
    ts = [x.requires_grad_() for i, x in enumerate(xs) if i != 4]

    def f(q, k, v, beta, la, S0):
        return layer.qdelta_chunk(q, k, v, beta, lam_c, la, S0)

    assert torch.autograd.gradcheck(f, ts, eps=1e-6, atol=1e-7, rtol=1e-6)
