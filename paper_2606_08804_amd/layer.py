"""Q-Delta as a trainable PyTorch layer: an autograd function over the HIP
chunk forward and backward, and a module with the gate projections.

``qdelta_chunk(q, k, v, beta, lam, log_alpha, initial_state, cu_seqlens)``
    differentiable in every tensor argument; the forward saves the per-chunk
    context (``chunk_fwd(save_states=True)``) and the backward hands it to
    ``chunk_bwd``.  Returns ``(o, final_state)``.

``QDeltaLayer(d_model, n_heads, head_dk, head_dv)``
    h [B, T, d_model] -> y [B, T, d_model].  Per head, from the hidden state:
    q, k, v by one fused projection (q and k L2-normalised per head, the
    condition under which the update is contractive, Sec. 3.4 Lemma 1);
    beta = sigmoid(W_beta h); alpha = sigmoid(W_alpha h), passed as its log;
    lambda = sigmoid(W_lambda h + b) with one scalar bias b initialised to
    -0.8 (App. "Query-Feedback Coefficient"); then the recurrence and an output
    projection.  The short convolutions, output gate and normalisation of the
    paper's block appear only in its architecture figure (Fig. 1b) and are not
    part of this layer.

The projections are ordinary library GEMMs; the q/k normalisation and the
recurrence are the library's kernels.  There is no CPU path: without the built library every call raises.
"""
import math

import torch
import torch.nn.functional as F

from . import qdelta as _binding


class QDeltaFunction(torch.autograd.Function):
    """Autograd wrapper of the chunkwise forward (Sec. 3.3) and its exact
    backward.  lam is a per-token tensor, a number (one constant lambda, no
    gradient taken) or None (lambda == 0); log_alpha None means alpha == 1."""

    @staticmethod
    def forward(ctx, q, k, v, beta, lam, log_alpha, initial_state, cu_seqlens):
        need = any(ctx.needs_input_grad[:7])
        o, final_state, saved = _binding.chunk_fwd(
            q, k, v, beta, lam, log_alpha, initial_state, cu_seqlens=cu_seqlens,
            output_final_state=True, save_states=need)
        ctx.lam_const = None if isinstance(lam, torch.Tensor) else lam
        lam_t = lam if isinstance(lam, torch.Tensor) else None
        ctx.save_for_backward(q, k, v, beta, lam_t, log_alpha, initial_state, cu_seqlens, saved)
        return o, final_state

    @staticmethod
    def backward(ctx, d_o, d_final_state):
        q, k, v, beta, lam_t, log_alpha, initial_state, cu_seqlens, saved = ctx.saved_tensors
        # a constant lambda is not differentiated here: passing it as None
        # would mean lambda == 0, so hand the number over and drop its gradient
        lam = lam_t if lam_t is not None else ctx.lam_const
        if d_o is None:
            d_o = torch.zeros(v.shape, dtype=v.dtype, device=v.device)
        dSf = None if d_final_state is None else d_final_state.contiguous()
        need_dS0 = initial_state is not None and ctx.needs_input_grad[6]
        g = _binding.chunk_bwd(q, k, v, beta, lam, log_alpha, initial_state, saved,
                               d_o.contiguous(), d_final_state=dSf, cu_seqlens=cu_seqlens,
                               need_d_initial_state=need_dS0)
        dlam = g["dlam"] if lam_t is not None else None
        return (g["dq"], g["dk"], g["dv"], g["dbeta"], dlam, g["dlog_alpha"],
                g["d_initial_state"], None)


class L2NormFunction(torch.autograd.Function):
    """Row L2 normalisation over the last dim in one HIP pass each way
    (strided rows read in place)."""

    @staticmethod
    def forward(ctx, x):
        y, rn = _binding.l2norm_fwd(x)
        ctx.save_for_backward(y, rn)
        return y

    @staticmethod
    def backward(ctx, dy):
        y, rn = ctx.saved_tensors
        return _binding.l2norm_bwd(y, rn, dy.contiguous())


def qdelta_chunk(q, k, v, beta, lam=None, log_alpha=None, initial_state=None, cu_seqlens=None):
    """Differentiable chunkwise Q-Delta.  Layouts as the C ABI: q, k [B,T,H,Dk],
    v [B,T,H,Dv] (bf16 or fp32), gates [B,T,H] fp32, states [N,H,Dv,Dk] fp32."""
    return QDeltaFunction.apply(q, k, v, beta, lam, log_alpha, initial_state, cu_seqlens)


class QDeltaLayer(torch.nn.Module):
    """Token mixer of a Q-Delta block: projections, gates, recurrence, output.

    Parameters live in the module's dtype (``.to(torch.bfloat16)`` runs the
    recurrence on bf16 activations); gates are formed in fp32 (or wider), the
    q and k L2 norms by the library's row-normalisation kernels."""

    def __init__(self, d_model, n_heads, head_dk=128, head_dv=128, use_decay=True, qk_norm=True,
                 lambda_bias=-0.8, fixed_lambda=None):
        """fixed_lambda: None for the learned gate lambda_t = sigmoid(W h + b);
        a number for a constant lambda (the paper's ablations: scalar 0.2, 0.5,
        0.8, and 1.0 for "no gating"), handed to the kernels as a scalar, so no
        lambda tensor is formed or read; 0 gives the gated delta rule.
        use_decay=False gives alpha == 1 ("no state decay")."""
        super().__init__()
        self.d_model, self.H, self.dk, self.dv = d_model, n_heads, head_dk, head_dv
        self.use_decay, self.qk_norm = use_decay, qk_norm
        self.fixed_lambda = None if fixed_lambda is None else float(fixed_lambda)
        self.w_qkv = torch.nn.Linear(d_model, n_heads * (2 * head_dk + head_dv), bias=False)
        # beta (, lambda) (, alpha)
        n_gates = 1 + (self.fixed_lambda is None) + bool(use_decay)
        self.w_gates = torch.nn.Linear(d_model, n_gates * n_heads, bias=False)
        if self.fixed_lambda is None:
            self.lambda_bias = torch.nn.Parameter(torch.tensor(float(lambda_bias)))
        self.w_out = torch.nn.Linear(n_heads * head_dv, d_model, bias=False)
        self.reset_parameters()

    def reset_parameters(self):
        for lin in (self.w_qkv, self.w_gates, self.w_out):
            torch.nn.init.normal_(lin.weight, std=1.0 / math.sqrt(lin.in_features))

    def gates(self, h):
        """beta, lambda, log alpha ([..., H] fp32 or wider; lambda a number
        when fixed, log alpha None without decay)."""
        acc = torch.promote_types(h.dtype, torch.float32)
        g = self.w_gates(h).to(acc)
        H = self.H
        beta = torch.sigmoid(g[..., :H])
        nxt = H
        if self.fixed_lambda is None:
            lam = torch.sigmoid(g[..., H:2 * H] + self.lambda_bias.to(acc))
            nxt = 2 * H
        else:
            lam = self.fixed_lambda
        log_alpha = F.logsigmoid(g[..., nxt:]) if self.use_decay else None
        return beta, lam, log_alpha

    def forward(self, h, initial_state=None, cu_seqlens=None, output_final_state=False):
        B, T, _ = h.shape
        H, dk, dv = self.H, self.dk, self.dv
        qkv = self.w_qkv(h).view(B, T, H, 2 * dk + dv)
        q, k, v = qkv.split([dk, dk, dv], dim=-1)
        if self.qk_norm:
            q = L2NormFunction.apply(q)
            k = L2NormFunction.apply(k)
        beta, lam, log_alpha = self.gates(h)
        o, final_state = qdelta_chunk(q.contiguous(), k.contiguous(), v.contiguous(),
                                      beta.contiguous(), lam.contiguous() if isinstance(lam, torch.Tensor) else lam,
                                      None if log_alpha is None else log_alpha.contiguous(),
                                      initial_state, cu_seqlens)
        y = self.w_out(o.reshape(B, T, H * dv))
        return (y, final_state) if output_final_state else y
