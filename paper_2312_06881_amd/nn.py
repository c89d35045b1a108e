"""Drop-in torch modules over libdyad.

* ``DyadLinear``: one Dyad layer, y = W x + b with W = BlockDiag(W1) +
  BlockTrans(W2) in the IT / OT / DT form (paper Sec. 2.2-2.4, Eqs. 1-16), a
  replacement for ``torch.nn.Linear``.
* ``DyadFF``: the feed-forward block fc1 -> GELU -> fc2 with both layers Dyad,
  each with its own variant if wanted (a heterogeneous mix, Sec. 4).  Unfused,
  the forward writes GELU(fc1) and stashes fc1's pre-activation in the same
  epilogue; fused, fc1 writes only the pre-activation and fc2's forward and
  weight-gradient kernels apply GELU as they stage it.  Either way the backward
  applies GELU' inside fc2's input-gradient epilogue, so the activation
  gradient is never a separate pass.

Autograd runs every pass through the C-ABI (forward, input gradient, weight and
bias gradient); there is no torch fallback and CPU tensors are rejected.
Leading input dimensions are flattened into the token dimension.  Weights
are stored as [n_dyad, ceil(out/n_dyad), ceil(in/n_dyad)] tensors, W1 the
BlockDiag and W2 the BlockTrans component; widths that n_dyad does not divide
are zero-padded (appendix, caveat on rectangular W).
"""
from __future__ import annotations

import math

import torch

from . import DyadError, backward_dw, backward_dx, forward

__all__ = ["DyadLinear", "DyadFF", "dyad_linear", "dyad_ff"]


def _tokens(x: torch.Tensor) -> torch.Tensor:
    return x.reshape(-1, x.shape[-1]).contiguous()


class _DyadLinearFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w1, w2, bias, variant, n_out):
        ctx.variant = variant
        ctx.has_bias = bias is not None
        ctx.save_for_backward(x, w1, w2)
        return forward(x, w1, w2, bias, variant, n_out=n_out)

    @staticmethod
    def backward(ctx, dy):
        x, w1, w2 = ctx.saved_tensors
        dy = dy.contiguous()
        dx = None
        if ctx.needs_input_grad[0]:
            dx = backward_dx(dy, w1, w2, ctx.variant, n_in=x.shape[1])
        dw1 = dw2 = db = None
        if any(ctx.needs_input_grad[1:4]):
            dw1, dw2, db = backward_dw(dy, x, w1.shape[0], ctx.variant, want_db=ctx.has_bias)
        return dx, dw1, dw2, db, None, None


_REFUSED = (-2, -4)   # DYAD_ERR_SHAPE, DYAD_ERR_DTYPE: no fused kernel for this layer


class _DyadFFFn(torch.autograd.Function):
    """fc1 -> GELU -> fc2.  Unfused: fc1's epilogue writes GELU(h) and stashes h.  Fused:
    fc1 writes only its pre-activation h; fc2's forward and weight-gradient kernels apply
    GELU to h as they stage it (dyad_forward_ex / dyad_backward_dw_ex), so GELU(h) is never
    written.  Both: fc2's input-gradient epilogue multiplies by GELU'(h).  A layer the fused
    kernels refuse runs unfused."""

    @staticmethod
    def forward(ctx, x, w1a, w2a, ba, w1b, w2b, bb, variants, ffn, d_out, fused):
        va, vb = variants
        y = None
        if fused:
            h = forward(x, w1a, w2a, ba, va, n_out=ffn)
            try:
                y = forward(h, w1b, w2b, bb, vb, n_out=d_out, act_in="gelu")
                a = None
            except DyadError as e:
                if e.status not in _REFUSED:
                    raise
        if y is None:
            a, h = forward(x, w1a, w2a, ba, va, act="gelu", stash_h=True, n_out=ffn)
            y = forward(a, w1b, w2b, bb, vb, n_out=d_out)
        ctx.variants = variants
        ctx.bias = (ba is not None, bb is not None)
        ctx.fused = a is None
        ctx.save_for_backward(x, h, a, w1a, w2a, ba, w1b, w2b)
        return y

    @staticmethod
    def backward(ctx, dy):
        x, h, a, w1a, w2a, ba, w1b, w2b = ctx.saved_tensors
        va, vb = ctx.variants
        dy = dy.contiguous()
        # fc2: input gradient times GELU'(fc1 pre-activation), then its weights
        dz1 = backward_dx(dy, w1b, w2b, vb, act_in="gelu", h_in=h)
        dwb = None
        if ctx.fused:
            try:
                dwb = backward_dw(dy, h, w1b.shape[0], vb, want_db=ctx.bias[1], act_in="gelu")
            except DyadError as e:
                if e.status not in _REFUSED:
                    raise
                # this weight gradient has no fused kernel: recompute GELU(h) through fc1
                a, _ = forward(x, w1a, w2a, ba, va, act="gelu", stash_h=True, n_out=h.shape[1])
        if dwb is None:
            dwb = backward_dw(dy, a, w1b.shape[0], vb, want_db=ctx.bias[1])
        dw1b, dw2b, dbb = dwb
        # fc1
        dx = backward_dx(dz1, w1a, w2a, va, n_in=x.shape[1]) if ctx.needs_input_grad[0] else None
        dw1a, dw2a, dba = backward_dw(dz1, x, w1a.shape[0], va, want_db=ctx.bias[0])
        return dx, dw1a, dw2a, dba, dw1b, dw2b, dbb, None, None, None, None


def _variant_pair(variant):
    pair = (variant, variant) if isinstance(variant, str) else tuple(variant)
    if len(pair) != 2 or any(v not in ("IT", "OT", "DT") for v in pair):
        raise ValueError("variant is one of IT, OT, DT, or an (fc1, fc2) pair of them")
    return pair


def dyad_linear(x, w1, w2, bias=None, variant="IT", out_features=None):
    """Functional form of ``DyadLinear``: x [..., n_in] -> [..., n_out], where n_out is
    out_features, else bias's length, else n_dyad * bo."""
    D, bo, _ = w1.shape
    if out_features is None:
        out_features = bias.shape[0] if bias is not None else D * bo
    y = _DyadLinearFn.apply(_tokens(x), w1, w2, bias, variant, out_features)
    return y.reshape(*x.shape[:-1], out_features)


def dyad_ff(x, fc1, fc2, variant="IT", ffn=None, fused=False):
    """Functional form of ``DyadFF``; fc1 / fc2 are (W1, W2, bias) triples; variant is one
    variant or an (fc1, fc2) pair; ffn is the hidden width (default n_dyad * fc1's bo).
    The output width is x's, as the block is d -> ffn -> d.  fused: GELU applied inside
    fc2's kernels, the activation never written (see _DyadFFFn)."""
    d = x.shape[-1]
    if ffn is None:
        ffn = fc1[0].shape[0] * fc1[0].shape[1]
    y = _DyadFFFn.apply(_tokens(x), *fc1, *fc2, _variant_pair(variant), ffn, d, bool(fused))
    return y.reshape(*x.shape[:-1], d)


class DyadLinear(torch.nn.Module):
    """Dyad replacement for ``torch.nn.Linear(in_features, out_features)``.

    A width that ``n_dyad`` does not divide is zero-padded up to the next multiple
    (appendix, caveat on rectangular W); such layers run on the library's general
    kernels rather than the matrix-core ones.  Initialisation (a convenience, not
    part of the method): uniform in +-1/sqrt(2 * in_features / n_dyad), the
    fan-in of one output feature (two components of in_features / n_dyad inputs each).
    """

    def __init__(self, in_features, out_features, n_dyad, variant="IT", bias=True, device=None,
                 dtype=torch.bfloat16):
        super().__init__()
        if min(in_features, out_features, n_dyad) <= 0:
            raise ValueError("widths and n_dyad must be positive")
        if variant not in ("IT", "OT", "DT"):
            raise ValueError("variant is one of IT, OT, DT")
        self.in_features, self.out_features, self.n_dyad, self.variant = in_features, out_features, n_dyad, variant
        shape = (n_dyad, -(-out_features // n_dyad), -(-in_features // n_dyad))
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
        return dyad_linear(x, self.w1, self.w2, self.bias, self.variant, self.out_features)

    def extra_repr(self):
        return (f"in_features={self.in_features}, out_features={self.out_features}, "
                f"n_dyad={self.n_dyad}, variant={self.variant}, bias={self.bias is not None}")


class DyadFF(torch.nn.Module):
    """Feed-forward block fc1 (d -> ffn) -> GELU -> fc2 (ffn -> d), both Dyad layers.

    ``variant`` is one of IT / OT / DT for both layers, or an (fc1, fc2) pair for a
    heterogeneous mix; ``n_dyad`` likewise may be one value or a pair.  ``fused``: fc1
    writes only its pre-activation and fc2's kernels apply GELU as they stage it."""

    def __init__(self, d, ffn, n_dyad, variant="IT", bias=True, device=None, dtype=torch.bfloat16,
                 fused=False):
        super().__init__()
        self.fused = fused
        va, vb = _variant_pair(variant)
        da, db = (n_dyad, n_dyad) if isinstance(n_dyad, int) else tuple(n_dyad)
        self.fc1 = DyadLinear(d, ffn, da, va, bias, device, dtype)
        self.fc2 = DyadLinear(ffn, d, db, vb, bias, device, dtype)
        self.variant = (va, vb)
        self.ffn = ffn

    def forward(self, x):
        return dyad_ff(x, (self.fc1.w1, self.fc1.w2, self.fc1.bias),
                       (self.fc2.w1, self.fc2.w2, self.fc2.bias), self.variant, self.ffn, self.fused)
