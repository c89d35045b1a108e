"""Drop-in torch modules over libdyad.

* ``DyadLinear``: one Dyad layer, y = W x + b with W = BlockDiag(W1) +
  BlockTrans(W2) in the IT / OT / DT form (paper Sec. 3, Eqs. 1-16), a
  replacement for ``torch.nn.Linear``.
* ``DyadFF``: the feed-forward block fc1 -> GELU -> fc2 with both layers Dyad.
  The forward writes GELU(fc1) and stashes fc1's pre-activation in the same
  epilogue; the backward applies GELU' inside fc2's input-gradient epilogue,
  so the activation gradient is never a separate pass.

Autograd runs every pass through the C-ABI (forward, input gradient, weight and
bias gradient); there is no torch fallback and CPU tensors are rejected.
Leading input dimensions are flattened into the token dimension.  Weights
are stored as [n_dyad, out/n_dyad, in/n_dyad] tensors, W1 the BlockDiag and W2
the BlockTrans component.
"""
from __future__ import annotations

import math

import torch

from . import backward_dw, backward_dx, forward

__all__ = ["DyadLinear", "DyadFF", "dyad_linear", "dyad_ff"]


def _tokens(x: torch.Tensor) -> torch.Tensor:
    return x.reshape(-1, x.shape[-1]).contiguous()


class _DyadLinearFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w1, w2, bias, variant):
        ctx.variant = variant
        ctx.has_bias = bias is not None
        ctx.save_for_backward(x, w1, w2)
        return forward(x, w1, w2, bias, variant)

    @staticmethod
    def backward(ctx, dy):
        x, w1, w2 = ctx.saved_tensors
        dy = dy.contiguous()
        dx = backward_dx(dy, w1, w2, ctx.variant) if ctx.needs_input_grad[0] else None
        dw1 = dw2 = db = None
        if any(ctx.needs_input_grad[1:4]):
            dw1, dw2, db = backward_dw(dy, x, w1.shape[0], ctx.variant, want_db=ctx.has_bias)
        return dx, dw1, dw2, db, None


class _DyadFFFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w1a, w2a, ba, w1b, w2b, bb, variant):
        a, h = forward(x, w1a, w2a, ba, variant, act="gelu", stash_h=True)
        y = forward(a, w1b, w2b, bb, variant)
        ctx.variant = variant
        ctx.bias = (ba is not None, bb is not None)
        ctx.save_for_backward(x, h, a, w1a, w2a, w1b, w2b)
        return y

    @staticmethod
    def backward(ctx, dy):
        x, h, a, w1a, w2a, w1b, w2b = ctx.saved_tensors
        v = ctx.variant
        dy = dy.contiguous()
        # fc2: input gradient times GELU'(fc1 pre-activation), then its weights
        dz1 = backward_dx(dy, w1b, w2b, v, act_in="gelu", h_in=h)
        dw1b, dw2b, dbb = backward_dw(dy, a, w1b.shape[0], v, want_db=ctx.bias[1])
        # fc1
        dx = backward_dx(dz1, w1a, w2a, v) if ctx.needs_input_grad[0] else None
        dw1a, dw2a, dba = backward_dw(dz1, x, w1a.shape[0], v, want_db=ctx.bias[0])
        return dx, dw1a, dw2a, dba, dw1b, dw2b, dbb, None


def dyad_linear(x, w1, w2, bias=None, variant="IT"):
    """Functional form of ``DyadLinear``: x [..., n_in] -> [..., n_out]."""
    D, bo, _ = w1.shape
    y = _DyadLinearFn.apply(_tokens(x), w1, w2, bias, variant)
    return y.reshape(*x.shape[:-1], D * bo)


def dyad_ff(x, fc1, fc2, variant="IT"):
    """Functional form of ``DyadFF``; fc1 / fc2 are (W1, W2, bias) triples."""
    D, bo, _ = fc2[0].shape
    y = _DyadFFFn.apply(_tokens(x), *fc1, *fc2, variant)
    return y.reshape(*x.shape[:-1], D * bo)


class DyadLinear(torch.nn.Module):
    """Dyad replacement for ``torch.nn.Linear(in_features, out_features)``.

    ``n_dyad`` must divide both widths.  Initialisation (a convenience, not part
    of the method): uniform in +-1/sqrt(2 * in_features / n_dyad), the fan-in of
    one output feature (two components of in_features / n_dyad inputs each).
    """

    def __init__(self, in_features, out_features, n_dyad, variant="IT", bias=True, device=None,
                 dtype=torch.bfloat16):
        super().__init__()
        if in_features % n_dyad or out_features % n_dyad:
            raise ValueError("n_dyad must divide in_features and out_features")
        if variant not in ("IT", "OT", "DT"):
            raise ValueError("variant is one of IT, OT, DT")
        self.in_features, self.out_features, self.n_dyad, self.variant = in_features, out_features, n_dyad, variant
        shape = (n_dyad, out_features // n_dyad, in_features // n_dyad)
        kw = {"device": device, "dtype": dtype}
        self.w1 = torch.nn.Parameter(torch.empty(shape, **kw))
        self.w2 = torch.nn.Parameter(torch.empty(shape, **kw))
        self.bias = torch.nn.Parameter(torch.empty(out_features, **kw)) if bias else None
        self.reset_parameters()

    def reset_parameters(self):
        bound = 1.0 / math.sqrt(2 * self.in_features / self.n_dyad)
        with torch.no_grad():
            for p in (self.w1, self.w2, self.bias):
                if p is not None:
                    p.uniform_(-bound, bound)

    def forward(self, x):
        return dyad_linear(x, self.w1, self.w2, self.bias, self.variant)

    def extra_repr(self):
        return (f"in_features={self.in_features}, out_features={self.out_features}, "
                f"n_dyad={self.n_dyad}, variant={self.variant}, bias={self.bias is not None}")


class DyadFF(torch.nn.Module):
    """Feed-forward block fc1 (d -> ffn) -> GELU -> fc2 (ffn -> d), both Dyad layers."""

    def __init__(self, d, ffn, n_dyad, variant="IT", bias=True, device=None, dtype=torch.bfloat16):
        super().__init__()
        self.fc1 = DyadLinear(d, ffn, n_dyad, variant, bias, device, dtype)
        self.fc2 = DyadLinear(ffn, d, n_dyad, variant, bias, device, dtype)
        self.variant = variant

    def forward(self, x):
        return dyad_ff(x, (self.fc1.w1, self.fc1.w2, self.fc1.bias),
                       (self.fc2.w1, self.fc2.w2, self.fc2.bias), self.variant)
