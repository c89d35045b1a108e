"""GPU parity of the small-batch paths (up to 256 tokens): forward, input
gradient and weight / bias gradients through the C-ABI against the CPU
oracle, element by element.

Shapes are chosen so that every form of that path runs: block slabs and
gathered residues (n_dyad 2, 3, 4, 8, 16), untransposed and transposed
weights, 128-column row units that fill a workgroup or leave waves idle,
reductions split across waves and across workgroups, and token counts that
leave a ragged 16-token tile.  Passes the path declines (block widths that
128 does not divide) run through the tiled kernels and are checked the same
way.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2312_06881_amd as dy
from workloads import layer_inputs
from tests.parity_util import assert_close

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
VARIANTS = ("IT", "OT", "DT")
ACT = {"none": oracle.ACT_NONE, "gelu": oracle.ACT_GELU}

SHAPES = [  # (n_in, n_out, n_dyad)
    (512, 512, 1),
    (512, 1024, 2),
    (512, 1024, 4),
    (768, 1536, 3),     # odd n_dyad: residues k*3 + b gathered element by element
    (1536, 512, 4),     # input-gradient blocks of 384 columns: three strips
    (768, 3072, 4),     # OPT-125m fc1: forward on this path, input gradient tiled
    (1024, 2048, 8),
    (2048, 8192, 16),
    (4096, 2048, 16),   # long reduction in the input gradient: split
]
TOKENS = [1, 7, 16, 17, 32]


def gpu(t):
    return None if t is None else t.to(DEV)


def banner(*what):
    print("CASE", *what, flush=True)


def case_id(c):
    return "x".join(map(str, c))


@pytest.mark.parametrize("M", TOKENS)
@pytest.mark.parametrize("act", ["none", "gelu"])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", SHAPES, ids=case_id)
def test_forward_few_tokens(shape, variant, act, M):
    n_in, n_out, D = shape
    banner("forward", shape, variant, act, M)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=M)
    y, h = dy.forward(gpu(L.X), gpu(L.W1), gpu(L.W2), gpu(L.bias), variant=variant, act=act, stash_h=True)
    torch.cuda.synchronize()
    ry, rh = oracle.forward(variant, n_in, n_out, D, L.f64("X"), L.f64("W1"), L.f64("W2"),
                            L.f64("bias"), act=ACT[act], want_h=True)
    assert_close(y, ry, "bf16", "Y")
    if act == "gelu":
        assert_close(h, rh, "bf16", "H")


@pytest.mark.parametrize("M", TOKENS)
@pytest.mark.parametrize("act_in", ["none", "gelu"])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", SHAPES, ids=case_id)
def test_backward_dx_few_tokens(shape, variant, act_in, M):
    n_in, n_out, D = shape
    banner("backward_dx", shape, variant, act_in, M)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=M)
    h_in = gpu(L.H_in) if act_in == "gelu" else None
    dx = dy.backward_dx(gpu(L.dZ), gpu(L.W1), gpu(L.W2), variant=variant, act_in=act_in, h_in=h_in)
    torch.cuda.synchronize()
    ref = oracle.backward_dx(variant, n_in, n_out, D, L.f64("dZ"), L.f64("W1"), L.f64("W2"),
                             act_in=ACT[act_in], H_in=L.f64("H_in") if act_in == "gelu" else None)
    assert_close(dx, ref, "bf16", "dX")


@pytest.mark.parametrize("M", TOKENS)
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", SHAPES, ids=case_id)
def test_backward_dw_few_tokens(shape, variant, M):
    """Weight and bias gradients with at most 32 tokens: one token split, the
    tiles storing bf16 results directly."""
    n_in, n_out, D = shape
    banner("backward_dw", shape, variant, M)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=M)
    dw1, dw2, db = dy.backward_dw(gpu(L.dZ), gpu(L.X), D, variant=variant)
    torch.cuda.synchronize()
    r1, r2, rb = oracle.backward_dw(variant, n_in, n_out, D, L.f64("dZ"), L.f64("X"))
    assert_close(dw1, r1, "bf16", "dW1")
    assert_close(dw2, r2, "bf16", "dW2")
    assert_close(db, rb, "bf16", "db")


MID_SHAPES = [(512, 1024, 4), (768, 1536, 3), (1536, 512, 4), (2048, 8192, 16), (4096, 2048, 16)]
MID_TOKENS = [33, 100, 256]


@pytest.mark.parametrize("M", MID_TOKENS)
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", MID_SHAPES, ids=case_id)
def test_forward_and_dx_up_to_256_tokens(shape, variant, M):
    """Batches of 33-256 tokens (GELU forward with stash, GELU' input gradient).
    At n_dyad 16 the output-transposed input gradients take the small-batch
    path, its waves splitting the tokens 32 at a time and looping over chunks
    of the reduction (at 256 tokens with reduction blocks of 512 or more, the
    large-batch path instead); the other passes run on the tiled kernels."""
    n_in, n_out, D = shape
    banner("mid", shape, variant, M)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=M)
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


@pytest.mark.parametrize("variant", VARIANTS)
def test_few_tokens_repeatable(variant):
    """Split reductions are added in a fixed order: two calls give identical bits."""
    n_in, n_out, D, M = 4096, 2048, 16, 16
    banner("repeat", variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16")
    X, W1, W2, b, dZ = gpu(L.X), gpu(L.W1), gpu(L.W2), gpu(L.bias), gpu(L.dZ)
    y1 = dy.forward(X, W1, W2, b, variant=variant)
    y2 = dy.forward(X, W1, W2, b, variant=variant)
    d1 = dy.backward_dx(dZ, W1, W2, variant=variant)
    d2 = dy.backward_dx(dZ, W1, W2, variant=variant)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2) and torch.equal(d1, d2)


@pytest.mark.parametrize("variant", VARIANTS)
def test_wide_few_tokens_all_passes(variant):
    """Wide layer 8192 -> 32768 at n_dyad 16 with 16 tokens: forward and input
    gradient in full (the tokens of a decode step)."""
    n_in, n_out, D, M = 8192, 32768, 16, 16
    banner("wide_few", variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16")
    y = dy.forward(gpu(L.X), gpu(L.W1), gpu(L.W2), gpu(L.bias), variant=variant)
    dx = dy.backward_dx(gpu(L.dZ), gpu(L.W1), gpu(L.W2), variant=variant)
    torch.cuda.synchronize()
    ry = oracle.forward(variant, n_in, n_out, D, L.f64("X"), L.f64("W1"), L.f64("W2"), L.f64("bias"))
    rdx = oracle.backward_dx(variant, n_in, n_out, D, L.f64("dZ"), L.f64("W1"), L.f64("W2"))
    assert_close(y, ry, "bf16", "Y")
    assert_close(dx, rdx, "bf16", "dX")
    assert np.isfinite(y.float().cpu().numpy()).all()


def test_two_streams_keep_their_workspaces():
    """Split sums live in one workspace per stream: passes queued on two
    streams at once give bitwise the results of the same passes run one after
    the other."""
    banner("two_streams")
    n_in, n_out, D, M = 8192, 32768, 16, 16
    La = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=1)
    Lb = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=2)
    a = [gpu(t) for t in (La.X, La.W1, La.W2, La.bias, La.dZ)]
    b = [gpu(t) for t in (Lb.X, Lb.W1, Lb.W2, Lb.bias, Lb.dZ)]
    ref = []
    for X, W1, W2, bias, dZ in (a, b):
        ref.append((dy.forward(X, W1, W2, bias, variant="DT"), dy.backward_dx(dZ, W1, W2, variant="DT")))
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    got = []
    for _ in range(3):
        outs = []
        for st, (X, W1, W2, bias, dZ) in ((s1, a), (s2, b)):
            with torch.cuda.stream(st):
                outs.append((dy.forward(X, W1, W2, bias, variant="DT"), dy.backward_dx(dZ, W1, W2, variant="DT")))
        got.append(outs)
    torch.cuda.synchronize()
    for outs in got:
        for (y, dx), (ry, rdx) in zip(outs, ref):
            assert torch.equal(y, ry) and torch.equal(dx, rdx)
