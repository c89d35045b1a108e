"""GPU parity of the large-batch path for n_dyad 8 and 16 with a transpose.

Forward and input gradient: input de-interleaved once, component 2 as a
per-block GEMM into an fp32 slice, component 1 as a per-block GEMM whose
epilogue adds that slice (read at the permuted place of each column under an
output transpose).  They take it from 2048 tokens with reduction blocks of at
least 256 (n_dyad 16; 128 with an output transpose, 64 for the input gradient
under one from 8192 tokens) or 512 (n_dyad 8); the other passes of these
shapes run on the fused tiles and are checked the same way.  Shapes cover the
three per-block tile widths (blocks of 256, 128 and 64 columns), token counts
that leave a ragged tile, and a wide layer whose slice does not fit the
workspace at once, so the tokens run in chunks (checked on sampled rows, the
chunk boundaries among them).

Weight gradients take it from 2048 tokens at n_dyad 16 and 8192 at n_dyad 8
(the n_dyad 8 case here: 8200 tokens): component 2's strided operands
de-interleaved into block-ordered copies, both components on the plain tiles.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2312_06881_amd as dy
from workloads import draw, layer_inputs
from tests.parity_util import assert_close

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
VARIANTS = ("IT", "OT", "DT")


def gpu(t):
    return None if t is None else t.to(DEV)


def banner(*what):
    print("CASE", *what, flush=True)


def case_id(c):
    return "x".join(map(str, c))


SHAPES = [  # (n_in, n_out, n_dyad, tokens); which pass takes the path, and its tile
    (4096, 1024, 16, 2100),   # forward, blocks of 64
    (1024, 4096, 16, 2049),   # input gradient, blocks of 64
    (4096, 2048, 16, 2100),   # forward (blocks of 128); input gradient of IT / DT (256)
    (2048, 2048, 16, 2049),   # OT / DT forward, IT / DT input gradient, blocks of 128
    (4096, 2048, 8, 2300),    # n_dyad 8 forward, blocks of 256
    (4096, 512, 8, 2048),     # n_dyad 8 forward, blocks of 64
    (2048, 4096, 8, 2051),    # n_dyad 8 input gradient, blocks of 256
]


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", SHAPES, ids=case_id)
def test_forward_and_dx_full(shape, variant):
    """GELU forward with the pre-activations kept, and the GELU' input
    gradient, element by element."""
    n_in, n_out, D, M = shape
    banner("permuted", shape, variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=5)
    y, h = dy.forward(gpu(L.X), gpu(L.W1), gpu(L.W2), gpu(L.bias), variant=variant, act="gelu", stash_h=True)
    dx = dy.backward_dx(gpu(L.dZ), gpu(L.W1), gpu(L.W2), variant=variant, act_in="gelu", h_in=gpu(L.H_in))
    torch.cuda.synchronize()
    ry, rh = oracle.forward(variant, n_in, n_out, D, L.f64("X"), L.f64("W1"), L.f64("W2"), L.f64("bias"),
                            act=oracle.ACT_GELU, want_h=True)
    rdx = oracle.backward_dx(variant, n_in, n_out, D, L.f64("dZ"), L.f64("W1"), L.f64("W2"),
                             act_in=oracle.ACT_GELU, H_in=L.f64("H_in"))
    assert_close(y, ry, "bf16", "Y")
    assert_close(h, rh, "bf16", "H")
    assert_close(dx, rdx, "bf16", "dX")


def test_no_bias_plain_forward():
    """Forward without bias or activation (the reduction's plain store)."""
    n_in, n_out, D, M = 2048, 2048, 16, 2049
    banner("permuted_nobias")
    L = layer_inputs(n_in, n_out, D, M, "bf16", bias="none", seed_offset=6)
    y = dy.forward(gpu(L.X), gpu(L.W1), gpu(L.W2), None, variant="DT")
    torch.cuda.synchronize()
    ry = oracle.forward("DT", n_in, n_out, D, L.f64("X"), L.f64("W1"), L.f64("W2"), None)
    assert_close(y, ry, "bf16", "Y")


def _draw(name, shape, std):
    return draw(name, shape, std, "bf16")


@pytest.mark.parametrize("variant", VARIANTS)
def test_wide_forward_chunked_sampled(variant):
    """Wide layer 8192 -> 32768 at n_dyad 16 with 16640 tokens: the forward's
    fp32 slice (and under an input transpose the de-interleaved input) exceeds
    the 2 GiB workspace, so its tokens run in chunks (16384 tokens for
    Dyad-OT, 14336 for Dyad-IT and -DT); rows on both sides of either boundary
    are checked."""
    n_in, n_out, D, M = 8192, 32768, 16, 16640
    banner("permuted_wide", variant)
    X = _draw("X", (M, n_in), 1.0)
    W1 = _draw("W1", (D, n_out // D, n_in // D), 0.02)
    W2 = _draw("W2", (D, n_out // D, n_in // D), 0.02)
    b = _draw("bias", (n_out,), 0.02)
    y = dy.forward(gpu(X), gpu(W1), gpu(W2), gpu(b), variant=variant)
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    rows = set(rng.choice(M, size=12, replace=False).tolist())
    rows |= {0, 14335, 14336, 16383, 16384, M - 1}
    rows = np.array(sorted(rows))
    f64 = lambda t: t.to(torch.float64).numpy()  # noqa: E731
    ry = oracle.forward(variant, n_in, n_out, D, f64(X[rows]), f64(W1), f64(W2), f64(b))
    assert_close(y[rows], ry, "bf16", "Y rows")


DW_SHAPES = [  # (n_in, n_out, n_dyad, tokens)
    (1024, 4096, 16, 2100),
    (4096, 2048, 16, 2049),
    (1024, 2048, 8, 8200),
]


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", DW_SHAPES, ids=case_id)
def test_backward_dw_full(shape, variant):
    """Weight and bias gradients on the large-batch path (n_dyad 16 from 2048
    tokens, n_dyad 8 from 8192): component 2's strided operands
    de-interleaved into block-ordered copies, both components on the plain
    tiles; element by element."""
    n_in, n_out, D, M = shape
    banner("permuted_dw", shape, variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=8)
    dw1, dw2, db = dy.backward_dw(gpu(L.dZ), gpu(L.X), D, variant=variant)
    torch.cuda.synchronize()
    r1, r2, rb = oracle.backward_dw(variant, n_in, n_out, D, L.f64("dZ"), L.f64("X"))
    assert_close(dw1, r1, "bf16", "dW1")
    assert_close(dw2, r2, "bf16", "dW2")
    assert_close(db, rb, "bf16", "db")


@pytest.mark.parametrize("variant", VARIANTS)
def test_wide_blocks_few_hundred_tokens(variant):
    """Blocks of 512 at n_dyad 16 with 300 tokens (the large-batch path from
    256 tokens on such blocks: 128-token tiles, a ragged last one): forward
    with GELU, input gradient with GELU', weight gradients, element by
    element."""
    n_in, n_out, D, M = 8192, 8192, 16, 300
    banner("permuted_few_hundred", variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=9)
    y, h = dy.forward(gpu(L.X), gpu(L.W1), gpu(L.W2), gpu(L.bias), variant=variant, act="gelu", stash_h=True)
    dx = dy.backward_dx(gpu(L.dZ), gpu(L.W1), gpu(L.W2), variant=variant, act_in="gelu", h_in=gpu(L.H_in))
    dw1, dw2, db = dy.backward_dw(gpu(L.dZ), gpu(L.X), D, variant=variant)
    torch.cuda.synchronize()
    W1, W2 = L.f64("W1"), L.f64("W2")
    ry, rh = oracle.forward(variant, n_in, n_out, D, L.f64("X"), W1, W2, L.f64("bias"), act=oracle.ACT_GELU,
                            want_h=True)
    rdx = oracle.backward_dx(variant, n_in, n_out, D, L.f64("dZ"), W1, W2, act_in=oracle.ACT_GELU,
                             H_in=L.f64("H_in"))
    r1, r2, rb = oracle.backward_dw(variant, n_in, n_out, D, L.f64("dZ"), L.f64("X"))
    assert_close(y, ry, "bf16", "Y")
    assert_close(h, rh, "bf16", "H")
    assert_close(dx, rdx, "bf16", "dX")
    assert_close(dw1, r1, "bf16", "dW1")
    assert_close(dw2, r2, "bf16", "dW2")
    assert_close(db, rb, "bf16", "db")


@pytest.mark.parametrize("variant", VARIANTS)
def test_wide_blocks_1030_tokens_sampled(variant):
    """The same layer with 1030 tokens (256-token tiles from 1025 tokens),
    forward and input gradient on sampled rows."""
    n_in, n_out, D, M = 8192, 8192, 16, 1030
    banner("permuted_1030", variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=10)
    y = dy.forward(gpu(L.X), gpu(L.W1), gpu(L.W2), gpu(L.bias), variant=variant)
    dx = dy.backward_dx(gpu(L.dZ), gpu(L.W1), gpu(L.W2), variant=variant)
    torch.cuda.synchronize()
    rows = np.array(sorted({0, 1, 255, 256, 511, 767, 768, 1023, 1024, M - 1}))
    W1, W2 = L.f64("W1"), L.f64("W2")
    ry = oracle.forward(variant, n_in, n_out, D, L.X[rows].to(torch.float64).numpy(), W1, W2, L.f64("bias"))
    rdx = oracle.backward_dx(variant, n_in, n_out, D, L.dZ[rows].to(torch.float64).numpy(), W1, W2)
    assert_close(y[rows], ry, "bf16", "Y rows")
    assert_close(dx[rows], rdx, "bf16", "dX rows")


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("layer", [(8192, 32768), (32768, 8192)], ids=["fc1", "fc2"])
def test_wide_layer_256_tokens_split_sampled(layer, variant):
    """The wide layer 8192 <-> 32768 at n_dyad 16 with 256 tokens: the passes
    whose reduction blocks are 2048 wide (fc2 forward, fc1 input gradient)
    split the reduction of both components in two, each part its own fp32
    slice, added in order by the split reduction.  Forward with GELU, input
    gradient with GELU', on sampled rows."""
    n_in, n_out = layer
    D, M = 16, 256
    banner("permuted_split256", layer, variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=11)
    y, h = dy.forward(gpu(L.X), gpu(L.W1), gpu(L.W2), gpu(L.bias), variant=variant, act="gelu", stash_h=True)
    dx = dy.backward_dx(gpu(L.dZ), gpu(L.W1), gpu(L.W2), variant=variant, act_in="gelu", h_in=gpu(L.H_in))
    torch.cuda.synchronize()
    rows = np.array([0, 1, 63, 64, 127, 128, 200, M - 1])
    W1, W2 = L.f64("W1"), L.f64("W2")
    ry, rh = oracle.forward(variant, n_in, n_out, D, L.X[rows].to(torch.float64).numpy(), W1, W2, L.f64("bias"),
                            act=oracle.ACT_GELU, want_h=True)
    rdx = oracle.backward_dx(variant, n_in, n_out, D, L.dZ[rows].to(torch.float64).numpy(), W1, W2,
                             act_in=oracle.ACT_GELU, H_in=L.H_in[rows].to(torch.float64).numpy())
    assert_close(y[rows], ry, "bf16", "Y rows")
    assert_close(h[rows], rh, "bf16", "H rows")
    assert_close(dx[rows], rdx, "bf16", "dX rows")
