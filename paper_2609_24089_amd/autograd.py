"""Differentiable attention whose double backward is the exact BoB path.

`attention(q, k, v, scale, causal)` returns O = softmax(scale q k^T + mask) v
(eq. 1) and supports two levels of reverse-mode differentiation:

* first backward (eqs. 2-3): `attn_bwd` gives dQ, dK, dV;
* backward of that backward (Sec. 3.1, eqs. 4-5): for cotangents
  (U_Q, U_K, U_V) on (dQ, dK, dV), BoB Pass 1 and Pass 2 give the gradients
  (Qt, Kt, Vt, dOt) of Phi = <dQ,U_Q> + <dK,U_K> + <dV,U_V> with respect to
  Q, K, V and the upstream gradient dO.

This is how the method is used for Hessian-vector products: differentiate a
loss once with create_graph=True, contract the gradient with a direction,
and differentiate again; the second call routes through the two BoB passes
(Sec. 4, the replacement of the attention double backward).

Qt, Kt, Vt are total derivatives of Phi: they already account for the
dependence of O (through D) and of the row statistics L on Q, K, V, so the
first-backward node reports no gradient for its O and L inputs.  dOt flows
into whatever produced dO, which carries the loss curvature in O.

Every step runs in the HIP kernels of libflashbob.so; the tensors must be
contiguous [B, H, N, d] bf16 or fp32 on the ROCm device.  k and v may have
fewer heads than q (grouped-query attention: query head h uses key/value
head h // (H / Hkv)); their gradients then sum over each group.
"""
import torch

from . import attn_bob_pass1_rows, attn_bob_pass2_cols, attn_bwd, attn_fwd_lse


class _AttentionFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, scale, causal):
        O, L = attn_fwd_lse(q, k, v, scale, causal=causal)
        ctx.save_for_backward(q, k, v, O, L)
        ctx.scale, ctx.causal = scale, causal
        return O

    @staticmethod
    def backward(ctx, dO):
        q, k, v, O, L = ctx.saved_tensors
        dq, dk, dv = _AttentionBackwardFn.apply(q, k, v, O, L, dO.contiguous(), ctx.scale, ctx.causal)
        return dq, dk, dv, None, None


class _AttentionBackwardFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, O, L, dO, scale, causal):
        dq, dk, dv, D = attn_bwd(q, k, v, O, dO, L, scale, causal=causal)
        ctx.save_for_backward(q, k, v, O, L, dO, D, dq)
        ctx.scale, ctx.causal = scale, causal
        return dq, dk, dv

    @staticmethod
    def backward(ctx, gdq, gdk, gdv):
        q, k, v, O, L, dO, D, dq = ctx.saved_tensors
        cot = [torch.zeros_like(x) if g is None else g.contiguous() for g, x in ((gdq, q), (gdk, k), (gdv, v))]
        Qt, dOt, alpha, E = attn_bob_pass1_rows(q, k, v, O, dO, *cot, L, D, ctx.scale, causal=ctx.causal, dQ=dq)
        Kt, Vt = attn_bob_pass2_cols(q, k, v, dO, *cot, L, D, alpha, E, ctx.scale, causal=ctx.causal)
        return Qt, Kt, Vt, None, None, dOt, None, None


def attention(q, k, v, scale=None, causal=False):
    """Softmax attention O = softmax(scale q k^T + mask) v with first and
    second derivatives on the HIP path.  scale defaults to 1/sqrt(d)."""
    if scale is None:
        scale = q.shape[-1] ** -0.5
    return _AttentionFn.apply(q, k, v, float(scale), bool(causal))
