"""GPU parity: libdyad (through its C-ABI) against the CPU oracle, element by element.

Small cases span several tiles and a ragged token tail and run every pass in full;
the named full-size workloads are checked on sampled tokens and sampled
weight-gradient entries (each one a full sum over all tokens).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2312_06881_amd as dy
from workloads import OPT125M, OPT350M, TINY, layer_inputs
from workloads import draw as _draw
from tests.parity_util import assert_close, to64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
VARIANTS = ("IT", "OT", "DT")
ACT = {"none": oracle.ACT_NONE, "gelu": oracle.ACT_GELU}

SMALL = [  # (n_in, n_out, n_dyad, M)
    (256, 512, 4, 300),
    (512, 256, 4, 200),
    (768, 3072, 4, 130),
    (3072, 768, 4, 65),
    (1024, 512, 8, 129),
    (512, 2048, 16, 77),
    (256, 256, 2, 100),
    (256, 256, 1, 100),
    (1024, 1024, 8, 129),
    (4096, 4096, 16, 70),
    (1024, 4096, 16, 100),  # input gradient under an output transpose, 64-column blocks:
    (4096, 1024, 16, 100),  #   components apart; the same for the forward pass
    (512, 1024, 8, 90),
    (192, 96, 3, 50),     # odd n_dyad, block widths 64 and 32
    (40, 24, 8, 33),      # block widths 5 and 3
]


def workloads_draw(name, shape, std):
    return _draw(name, shape, std, "bf16")


def case_id(c):
    return "x".join(map(str, c))


def gpu(t):
    return None if t is None else t.to(DEV)


def banner(*what):
    print("CASE", *what, flush=True)


@pytest.mark.parametrize("act", ["none", "gelu"])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", SMALL, ids=case_id)
def test_forward_small(shape, variant, act):
    n_in, n_out, D, M = shape
    banner("forward", shape, variant, act)
    L = layer_inputs(n_in, n_out, D, M, "bf16")
    y, h = dy.forward(gpu(L.X), gpu(L.W1), gpu(L.W2), gpu(L.bias), variant=variant, act=act,
                      stash_h=True)
    torch.cuda.synchronize()
    ry, rh = oracle.forward(variant, n_in, n_out, D, L.f64("X"), L.f64("W1"), L.f64("W2"),
                            L.f64("bias"), act=ACT[act], want_h=True)
    assert_close(y, ry, "bf16", "Y")
    if act == "gelu":
        assert_close(h, rh, "bf16", "H")


@pytest.mark.parametrize("act_in", ["none", "gelu"])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", SMALL, ids=case_id)
def test_backward_dx_small(shape, variant, act_in):
    n_in, n_out, D, M = shape
    banner("backward_dx", shape, variant, act_in)
    L = layer_inputs(n_in, n_out, D, M, "bf16")
    h_in = gpu(L.H_in) if act_in == "gelu" else None
    dx = dy.backward_dx(gpu(L.dZ), gpu(L.W1), gpu(L.W2), variant=variant, act_in=act_in, h_in=h_in)
    torch.cuda.synchronize()
    ref = oracle.backward_dx(variant, n_in, n_out, D, L.f64("dZ"), L.f64("W1"), L.f64("W2"),
                             act_in=ACT[act_in], H_in=L.f64("H_in") if act_in == "gelu" else None)
    assert_close(dx, ref, "bf16", "dX")


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", SMALL, ids=case_id)
def test_backward_dw_small(shape, variant):
    n_in, n_out, D, M = shape
    banner("backward_dw", shape, variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16")
    dw1, dw2, db = dy.backward_dw(gpu(L.dZ), gpu(L.X), D, variant=variant)
    torch.cuda.synchronize()
    r1, r2, rb = oracle.backward_dw(variant, n_in, n_out, D, L.f64("dZ"), L.f64("X"))
    assert_close(dw1, r1, "bf16", "dW1")
    assert_close(dw2, r2, "bf16", "dW2")
    assert_close(db, rb, "bf16", "db")


@pytest.mark.parametrize("variant", VARIANTS)
def test_tiny_fp32_all_passes(variant):
    """n_in=64, n_out=256, n_dyad=4, M=128, fp32, bias 0; also against the dense W the oracle spans."""
    (_, n_in, n_out), = TINY.layers
    D, M = TINY.n_dyad, TINY.M
    banner("tiny_fp32", variant)
    L = layer_inputs(n_in, n_out, D, M, "f32", bias="zero")
    x, w1, w2, b, dz = (gpu(t) for t in (L.X, L.W1, L.W2, L.bias, L.dZ))
    y = dy.forward(x, w1, w2, b, variant=variant)
    dx = dy.backward_dx(dz, w1, w2, variant=variant)
    dw1, dw2, db = dy.backward_dw(dz, x, D, variant=variant)
    torch.cuda.synchronize()
    X, W1, W2, dZ = L.f64("X"), L.f64("W1"), L.f64("W2"), L.f64("dZ")
    ry = oracle.forward(variant, n_in, n_out, D, X, W1, W2, L.f64("bias"))
    assert_close(y, ry, "f32", "Y")
    W = oracle.forward(variant, n_in, n_out, D, np.eye(n_in), W1, W2).T   # dense W, n_out x n_in
    assert_close(y, X @ W.T, "f32", "Y vs dense W")
    assert_close(dx, oracle.backward_dx(variant, n_in, n_out, D, dZ, W1, W2), "f32", "dX")
    assert_close(dx, dZ @ W, "f32", "dX vs dense W")
    r1, r2, rb = oracle.backward_dw(variant, n_in, n_out, D, dZ, X)
    assert_close(dw1, r1, "f32", "dW1")
    assert_close(dw2, r2, "f32", "dW2")
    assert_close(db, rb, "f32", "db")


@pytest.mark.parametrize("variant", VARIANTS)
def test_fp32_larger(variant):
    n_in, n_out, D, M = 384, 768, 4, 150
    banner("fp32_larger", variant)
    L = layer_inputs(n_in, n_out, D, M, "f32")
    x, w1, w2, b, dz, h = (gpu(t) for t in (L.X, L.W1, L.W2, L.bias, L.dZ, L.H_in))
    y = dy.forward(x, w1, w2, b, variant=variant, act="gelu")
    dx = dy.backward_dx(dz, w1, w2, variant=variant, act_in="gelu", h_in=h)
    dw1, dw2, db = dy.backward_dw(dz, x, D, variant=variant)
    torch.cuda.synchronize()
    X, W1, W2, dZ = L.f64("X"), L.f64("W1"), L.f64("W2"), L.f64("dZ")
    assert_close(y, oracle.forward(variant, n_in, n_out, D, X, W1, W2, L.f64("bias"),
                                   act=oracle.ACT_GELU), "f32", "Y")
    assert_close(dx, oracle.backward_dx(variant, n_in, n_out, D, dZ, W1, W2,
                                        act_in=oracle.ACT_GELU, H_in=L.f64("H_in")), "f32", "dX")
    r1, r2, rb = oracle.backward_dw(variant, n_in, n_out, D, dZ, X)
    assert_close(dw1, r1, "f32", "dW1")
    assert_close(dw2, r2, "f32", "dW2")
    assert_close(db, rb, "f32", "db")


def test_empty_batch():
    banner("empty")
    L = layer_inputs(256, 512, 4, 1, "bf16")
    x = torch.empty((0, 256), dtype=torch.bfloat16, device=DEV)
    y = dy.forward(x, gpu(L.W1), gpu(L.W2), gpu(L.bias), variant="DT")
    assert y.shape == (0, 512)
    dz = torch.empty((0, 512), dtype=torch.bfloat16, device=DEV)
    dx = dy.backward_dx(dz, gpu(L.W1), gpu(L.W2), variant="IT")
    assert dx.shape == (0, 256)
    dw1, dw2, db = dy.backward_dw(dz, x, 4, variant="OT")
    torch.cuda.synchronize()
    assert not dw1.float().abs().sum() and not dw2.float().abs().sum() and not db.float().abs().sum()


@pytest.mark.parametrize("variant", VARIANTS)
def test_single_token_no_bias(variant):
    banner("single_token", variant)
    n_in, n_out, D = 768, 3072, 4
    L = layer_inputs(n_in, n_out, D, 1, "bf16", bias="none")
    y = dy.forward(gpu(L.X), gpu(L.W1), gpu(L.W2), None, variant=variant)
    torch.cuda.synchronize()
    assert_close(y, oracle.forward(variant, n_in, n_out, D, L.f64("X"), L.f64("W1"), L.f64("W2")),
                 "bf16", "Y")


def test_dw_is_deterministic():
    banner("determinism")
    n_in, n_out, D, M = 768, 3072, 4, 4099
    L = layer_inputs(n_in, n_out, D, M, "bf16")
    dz, x = gpu(L.dZ), gpu(L.X)
    a = dy.backward_dw(dz, x, D, variant="DT")
    b = dy.backward_dw(dz, x, D, variant="DT")
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)


@pytest.mark.parametrize("variant", VARIANTS)
def test_ff_chain(variant):
    """fc1 (GELU, pre-activation stashed) -> fc2, then the backward chain, end to end."""
    d, ffn, D, M = 256, 1024, 4, 130
    banner("ff_chain", variant)
    L1 = layer_inputs(d, ffn, D, M, "bf16")
    L2 = layer_inputs(ffn, d, D, M, "bf16", seed_offset=100)
    x, w11, w12, b1 = (gpu(t) for t in (L1.X, L1.W1, L1.W2, L1.bias))
    w21, w22, b2, dy2 = (gpu(t) for t in (L2.W1, L2.W2, L2.bias, L2.dZ))
    a1, h1 = dy.forward(x, w11, w12, b1, variant=variant, act="gelu", stash_h=True)
    y2 = dy.forward(a1, w21, w22, b2, variant=variant)
    dh1 = dy.backward_dx(dy2, w21, w22, variant=variant, act_in="gelu", h_in=h1)
    g21, g22, gb2 = dy.backward_dw(dy2, a1, D, variant=variant)
    dx = dy.backward_dx(dh1, w11, w12, variant=variant)
    g11, g12, gb1 = dy.backward_dw(dh1, x, D, variant=variant)
    torch.cuda.synchronize()
    X = L1.f64("X")
    ra1, rh1 = oracle.forward(variant, d, ffn, D, X, L1.f64("W1"), L1.f64("W2"), L1.f64("bias"),
                              act=oracle.ACT_GELU, want_h=True)
    ry2 = oracle.forward(variant, ffn, d, D, ra1, L2.f64("W1"), L2.f64("W2"), L2.f64("bias"))
    rdh1 = oracle.backward_dx(variant, ffn, d, D, L2.f64("dZ"), L2.f64("W1"), L2.f64("W2"),
                              act_in=oracle.ACT_GELU, H_in=rh1)
    r21, r22, rb2 = oracle.backward_dw(variant, ffn, d, D, L2.f64("dZ"), ra1)
    rdx = oracle.backward_dx(variant, d, ffn, D, rdh1, L1.f64("W1"), L1.f64("W2"))
    r11, r12, rb1 = oracle.backward_dw(variant, d, ffn, D, rdh1, X)
    for got, ref, what in ((a1, ra1, "a1"), (h1, rh1, "h1"), (y2, ry2, "y2"), (dh1, rdh1, "dh1"),
                           (g21, r21, "dW21"), (g22, r22, "dW22"), (gb2, rb2, "db2"),
                           (dx, rdx, "dx"), (g11, r11, "dW11"), (g12, r12, "dW12"),
                           (gb1, rb1, "db1")):
        # each layer rounds its output to bf16 before the next consumes it, so the
        # chain is held to the max-norm bar only, not the per-layer elementwise bound
        g = to64(got)
        err = float(np.abs(g - ref).max() / np.abs(ref).max())
        assert err <= 2e-2, (what, err)


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", [(256, 768, 4, 16461), (384, 768, 4, 16400), (768, 768, 4, 16384)],
                         ids=case_id)
def test_forward_bias_large_batch_full(shape, variant):
    """Forward with a bias epilogue at batches that fill the GPU with 256 x 192 tiles (the
    path that keeps two stages of loads in flight), every output checked: two, three and
    twelve stages per component, and a ragged last token tile."""
    n_in, n_out, D, M = shape
    banner("forward_large", shape, variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16")
    y = dy.forward(gpu(L.X), gpu(L.W1), gpu(L.W2), gpu(L.bias), variant=variant)
    torch.cuda.synchronize()
    ry = oracle.forward(variant, n_in, n_out, D, L.f64("X"), L.f64("W1"), L.f64("W2"), L.f64("bias"))
    assert_close(y, ry, "bf16", "Y")


# ---- widths that n_dyad does not divide: zero-padded layers -------------------

PADDED = [  # (n_in, n_out, n_dyad, M)
    (6, 7, 2, 5),          # the appendix's 7 x 6 weight at n_dyad 2
    (250, 510, 4, 77),
    (768, 3072, 5, 96),    # OPT-125m fc1 widths at n_dyad 5: blocks of 154 and 615
    (3072, 768, 5, 40),
    (100, 36, 8, 33),      # blocks of 13 and 5
    (5, 9, 8, 17),         # n_dyad above n_in: three groups see only padding
    (250, 510, 4, 1100),   # enough tokens to split the weight gradient (ragged last split)
    (768, 3072, 5, 600),
    (768, 3072, 3, 700),   # n_dyad 3 divides both widths, not the blocks (256, 1024)
    (768, 3072, 6, 300),   # blocks of 128 and 512
    (1536, 384, 6, 257),   # blocks of 256 and 64
    (384, 1536, 3, 2100),  # enough tokens for the de-interleaved forms of every pass
    # from 512 tokens, shapes no fused tile takes run on zero-padded block copies:
    (640, 1280, 5, 700),   # n_dyad 5 dividing both widths (blocks 128 / 256)
    (896, 448, 7, 520),    # n_dyad 7 (blocks 128 / 64)
    (776, 1544, 8, 600),   # blocks of 97 and 193, padded to 128 / 256
    (768, 3072, 12, 512),  # n_dyad 12
]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", PADDED, ids=case_id)
def test_padded_all_passes(shape, variant, dtype):
    """Forward (GELU, H stash), input gradient (GELU'), weight and bias gradients of a
    zero-padded layer; outputs are written through the C-ABI into buffers with a guard
    tail that must stay untouched (no write lands past n_out or n_in)."""
    n_in, n_out, D, M = shape
    banner("padded", shape, variant, dtype)
    L = layer_inputs(n_in, n_out, D, M, dtype)
    tdt = L.X.dtype
    code = dy.BF16 if dtype == "bf16" else dy.F32
    v = dy.VARIANTS[variant]
    x, w1, w2, b, dz, hin = (gpu(t) for t in (L.X, L.W1, L.W2, L.bias, L.dZ, L.H_in))
    guard = 64
    sentinel = -1536.0   # exact in bf16

    def guarded(n):
        return torch.full((n + guard,), sentinel, dtype=tdt, device=DEV)

    y, h, dx = guarded(M * n_out), guarded(M * n_out), guarded(M * n_in)
    bo, bi = w1.shape[1], w1.shape[2]
    dw1, dw2, db = guarded(D * bo * bi), guarded(D * bo * bi), guarded(n_out)
    s = torch.cuda.current_stream().cuda_stream
    assert dy.dyad_forward(v, n_in, n_out, D, M, code, x.data_ptr(), w1.data_ptr(), w2.data_ptr(),
                           b.data_ptr(), dy.ACT_GELU, y.data_ptr(), h.data_ptr(), s) == 0
    assert dy.dyad_backward_dx(v, n_in, n_out, D, M, code, dz.data_ptr(), w1.data_ptr(),
                               w2.data_ptr(), dy.ACT_GELU, hin.data_ptr(), dx.data_ptr(), s) == 0
    need = dy.dyad_dw_workspace_bytes(v, n_in, n_out, D, M, code)
    ws = torch.empty((max(need, 16),), dtype=torch.uint8, device=DEV)
    if need:   # a call without the workspace is refused before any launch
        assert dy.dyad_backward_dw(v, n_in, n_out, D, M, code, dz.data_ptr(), x.data_ptr(), dw1.data_ptr(),
                                   dw2.data_ptr(), db.data_ptr(), None, 0, s) == -5
    assert dy.dyad_backward_dw(v, n_in, n_out, D, M, code, dz.data_ptr(), x.data_ptr(),
                               dw1.data_ptr(), dw2.data_ptr(), db.data_ptr(), ws.data_ptr(), need, s) == 0
    torch.cuda.synchronize()
    for t in (y, h, dx, dw1, dw2, db):
        assert bool((t[-guard:] == sentinel).all()), "write past the end of an output"
    ry, rh = oracle.forward(variant, n_in, n_out, D, L.f64("X"), L.f64("W1"), L.f64("W2"),
                            L.f64("bias"), act=oracle.ACT_GELU, want_h=True)
    rdx = oracle.backward_dx(variant, n_in, n_out, D, L.f64("dZ"), L.f64("W1"), L.f64("W2"),
                             act_in=oracle.ACT_GELU, H_in=L.f64("H_in"))
    r1, r2, rb = oracle.backward_dw(variant, n_in, n_out, D, L.f64("dZ"), L.f64("X"))
    assert_close(y[:-guard].view(M, n_out), ry, dtype, "Y")
    assert_close(h[:-guard].view(M, n_out), rh, dtype, "H")
    assert_close(dx[:-guard].view(M, n_in), rdx, dtype, "dX")
    assert_close(dw1[:-guard].view(D, bo, bi), r1, dtype, "dW1")
    assert_close(dw2[:-guard].view(D, bo, bi), r2, dtype, "dW2")
    assert_close(db[:-guard], rb, dtype, "db")
    # entries that touch only padding get exactly zero
    assert bool((dw1[:-guard].view(D, bo, bi)[torch.from_numpy(r1 == 0).to(DEV)] == 0).all())
    assert bool((dw2[:-guard].view(D, bo, bi)[torch.from_numpy(r2 == 0).to(DEV)] == 0).all())


# ---- full-size named workloads, sampled ---------------------------------------

def sample_rows(M, n, seed):
    rng = np.random.default_rng(seed)
    rows = set(rng.choice(M, size=min(n, M), replace=False).tolist())
    rows |= {0, M - 1, M - 2} & set(range(M))
    return np.array(sorted(rows))


def _f64_rows(t, lo, hi):
    return t[lo:hi].to(torch.float64).numpy()


def oracle_dw_sampled(variant, n_in, n_out, D, dZ, X, comp, i, j, k, chunk=4096):
    """Sampled dW entries and the full db from the oracle, the token sum taken in chunks of
    `chunk` tokens (each entry is linear in the tokens, so the chunk results add up to the
    whole sum) to keep the fp64 copies of very large dZ / X bounded."""
    M = dZ.shape[0]
    ent = np.zeros(len(comp), np.float64)
    db = np.zeros(n_out, np.float64)
    for lo in range(0, M, chunk):
        hi = min(M, lo + chunk)
        z, x = _f64_rows(dZ, lo, hi), _f64_rows(X, lo, hi)
        ent += oracle.backward_dw_entries(variant, n_in, n_out, D, z, x, comp, i, j, k)
        db += oracle.bias_grad(z)
    return ent, db


def check_full_layer(n_in, n_out, D, M, variant, fwd_act="none", dx_act="none", seed_offset=0):
    """One layer at full size, every pass as the bench calls it: forward with `fwd_act`
    (GELU with the pre-activation stashed when "gelu"), input gradient with `dx_act`
    (GELU' of H_in when "gelu"), weight and bias gradients.  Checked on 40 sampled tokens
    (plus the first and last two) and 300 sampled dW entries (corners included), each
    entry a full sum over all M tokens."""
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=seed_offset)
    x, w1, w2, b, dz = (gpu(t) for t in (L.X, L.W1, L.W2, L.bias, L.dZ))
    h_in = gpu(L.H_in) if dx_act == "gelu" else None
    if fwd_act == "gelu":
        y, h = dy.forward(x, w1, w2, b, variant=variant, act="gelu", stash_h=True, n_out=n_out)
    else:
        y, h = dy.forward(x, w1, w2, b, variant=variant, n_out=n_out), None
    dx = dy.backward_dx(dz, w1, w2, variant=variant, act_in=dx_act, h_in=h_in, n_in=n_in)
    dw1, dw2, db = dy.backward_dw(dz, x, D, variant=variant)
    torch.cuda.synchronize()
    del x, dz, h_in
    rows = sample_rows(M, 40, 7)
    W1, W2 = L.f64("W1"), L.f64("W2")
    Xs = L.X[rows].to(torch.float64).numpy()
    ry, rh = oracle.forward(variant, n_in, n_out, D, Xs, W1, W2, L.f64("bias"), act=ACT[fwd_act],
                            want_h=True)
    assert_close(y[rows], ry, "bf16", "Y rows")
    if fwd_act == "gelu":
        assert_close(h[rows], rh, "bf16", "H rows")
    del y, h
    dZs = L.dZ[rows].to(torch.float64).numpy()
    Hs = L.H_in[rows].to(torch.float64).numpy() if dx_act == "gelu" else None
    rdx = oracle.backward_dx(variant, n_in, n_out, D, dZs, W1, W2, act_in=ACT[dx_act], H_in=Hs)
    assert_close(dx[rows], rdx, "bf16", "dX rows")
    del dx
    rng = np.random.default_rng(11)
    n = 300
    bo, bi = -(-n_out // D), -(-n_in // D)   # zero-padded blocks where D does not divide
    comp = rng.integers(1, 3, n)
    i, j, k = rng.integers(0, D, n), rng.integers(0, bo, n), rng.integers(0, bi, n)
    comp[:4], i[:4], j[:4], k[:4] = [1, 2, 1, 2], [0, 0, D - 1, D - 1], [0, 0, bo - 1, bo - 1], [0, 0, bi - 1, bi - 1]
    ref, rdb = oracle_dw_sampled(variant, n_in, n_out, D, L.dZ, L.X, comp, i, j, k)
    ti, tj, tk = (torch.as_tensor(a, device=DEV) for a in (i, j, k))
    got = np.where(comp == 1, to64(dw1[ti, tj, tk]), to64(dw2[ti, tj, tk]))
    # sampled entries: compare against the scale of the whole sampled set
    assert_close(got, ref, "bf16", "dW entries")
    assert_close(db, rdb, "bf16", "db")


# The feed-forward block as the bench runs it: fc1 forward with GELU and the
# pre-activation stash, fc1 input gradient plain; fc2 forward plain, fc2 input
# gradient with GELU' of fc1's pre-activation.
FF_ACTS = {"fc1": ("gelu", "none"), "fc2": ("none", "gelu")}


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("wl", [OPT125M, OPT350M], ids=lambda w: w.name)
def test_full_size_ff_sampled(wl, variant):
    for li, (name, n_in, n_out) in enumerate(wl.layers):
        banner("full", wl.name, name, variant)
        fa, da = FF_ACTS[name]
        check_full_layer(n_in, n_out, wl.n_dyad, wl.M, variant, fa, da, seed_offset=li)


# OPT-125m feed-forward widths at n_dyad 3 and 6 (blocks 256 / 1024 and 128 /
# 512, which n_dyad does not divide: the forward pass under an output
# transpose runs its components apart) and 5 (zero-padded blocks of 154 / 615).
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("D", [3, 5, 6])
def test_full_size_odd_dyad_sampled(D, variant):
    for li, (name, n_in, n_out) in enumerate(OPT125M.layers):
        banner("full odd", D, name, variant)
        fa, da = FF_ACTS[name]
        check_full_layer(n_in, n_out, D, OPT125M.M, variant, fa, da, seed_offset=li)


# The zero-padded forms take the tokens in chunks that keep their copies and
# slice within 2 GiB: with 16360 outputs at n_dyad 5 (blocks of 154 / 3272,
# padded to 160 / 3328) a chunk under an output transpose holds about 31500
# tokens, so 40000 tokens run as two, the second ragged.
@pytest.mark.parametrize("variant", VARIANTS)
def test_padded_forms_token_chunks_sampled(variant):
    banner("padded chunks", variant)
    check_full_layer(768, 16360, 5, 40000, variant, "gelu", "none", seed_offset=3)


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", [(768, 3072, 4, 5000), (3072, 768, 4, 3001), (1024, 1024, 16, 2049)],
                         ids=case_id)
def test_backward_dw_many_splits(shape, variant):
    """Token counts that spread over many splits, with a ragged last split."""
    n_in, n_out, D, M = shape
    banner("backward_dw_splits", shape, variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=3)
    dw1, dw2, db = dy.backward_dw(gpu(L.dZ), gpu(L.X), D, variant=variant)
    torch.cuda.synchronize()
    r1, r2, rb = oracle.backward_dw(variant, n_in, n_out, D, L.f64("dZ"), L.f64("X"))
    assert_close(dw1, r1, "bf16", "dW1")
    assert_close(dw2, r2, "bf16", "dW2")
    assert_close(db, rb, "bf16", "db")


# ---- width/block sweep and the wide layer, full size, sampled ---------------------

SWEEP_POINTS = [(d, D) for d in (1024, 2048, 4096, 8192) for D in (2, 4, 8, 16)]


@pytest.mark.parametrize("layer", ["fc1", "fc2"])
@pytest.mark.parametrize("d,D", SWEEP_POINTS, ids=lambda v: str(v))
def test_sweep_dt_sampled(d, D, layer):
    """Dyad-DT feed-forward at every width/block sweep point, M = 16384: fc1 d -> 4d (forward
    with GELU and stash), fc2 4d -> d (input gradient with GELU'), each pass as benched."""
    n_in, n_out = (d, 4 * d) if layer == "fc1" else (4 * d, d)
    banner("sweep", d, D, layer)
    fa, da = FF_ACTS[layer]
    check_full_layer(n_in, n_out, D, 16384, "DT", fa, da, seed_offset=0 if layer == "fc1" else 1)


@pytest.mark.parametrize("M", [16, 256, 32768])
def test_wide_it_forward(M):
    """Wide layer 8192 -> 32768, n_dyad 16, Dyad-IT forward; small-M rows checked in full."""
    n_in, n_out, D = 8192, 32768, 16
    banner("wide_forward", M)
    X = workloads_draw("X", (M, n_in), 1.0)
    W1 = workloads_draw("W1", (D, n_out // D, n_in // D), 0.02)
    W2 = workloads_draw("W2", (D, n_out // D, n_in // D), 0.02)
    b = workloads_draw("bias", (n_out,), 0.02)
    y = dy.forward(gpu(X), gpu(W1), gpu(W2), gpu(b), variant="IT")
    torch.cuda.synchronize()
    rows = sample_rows(M, 24, 5) if M > 256 else np.arange(M)
    f64 = lambda t: t.to(torch.float64).numpy()  # noqa: E731
    ref = oracle.forward("IT", n_in, n_out, D, X[rows].to(torch.float64).numpy(), f64(W1), f64(W2), f64(b))
    assert_close(y[rows], ref, "bf16", "Y rows")


@pytest.mark.parametrize("M", [4096, 32768])
def test_wide_it_backward_sampled(M):
    """Wide layer 8192 -> 32768, n_dyad 16, Dyad-IT forward, dX and dW, sampled; 32768 tokens
    is the wide configuration's fwd+bwd batch."""
    banner("wide_backward", M)
    check_full_layer(8192, 32768, 16, M, "IT")
