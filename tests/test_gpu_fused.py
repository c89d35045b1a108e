"""GPU parity of the fused feed-forward path: a layer whose input is GELU(H), with the
activation applied inside the kernels as the input operand is staged
(dyad_forward_ex / dyad_backward_dw_ex with act_in = GELU), so GELU(H) never exists
in memory.

The oracle's reference input is GELU(H) in fp64 rounded once to bf16 (RNE), the value
the unfused chain stores between fc1 and fc2 and the one the kernels round their fp32
GELU to before the multiply."""
import numpy as np
import pytest
import torch

import oracle
import paper_2312_06881_amd as dy
from paper_2312_06881_amd.nn import DyadFF
from workloads import OPT125M, layer_inputs
from tests.parity_util import assert_close, to64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
VARIANTS = ("IT", "OT", "DT")


def banner(*what):
    print("CASE", *what, flush=True)


def gpu(t):
    return None if t is None else t.to(DEV)


def gelu_bf16(H):
    """Reference activated input: exact GELU of the bf16 pre-activation, rounded to bf16."""
    g = oracle.gelu_array(H.to(torch.float64).numpy())
    return torch.from_numpy(g).to(torch.bfloat16).to(torch.float64).numpy()


SHAPES = [  # (n_in, n_out, n_dyad, M): several tiles, ragged token tails
    (3072, 768, 4, 700),
    (1024, 512, 4, 300),
    (768, 3072, 4, 130),
    (512, 512, 2, 257),
    (256, 256, 1, 100),
    (2048, 1024, 8, 129),
]


@pytest.mark.parametrize("act", ["none", "gelu"])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda c: "x".join(map(str, c)))
def test_forward_gelu_in(shape, variant, act):
    n_in, n_out, D, M = shape
    if D > 4 and variant != "IT":
        pytest.skip("no fused tile for an output transpose above n_dyad 4 (refusal tested below)")
    banner("forward_gelu_in", shape, variant, act)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=40)
    h_in = L.H_in   # the previous layer's pre-activation, [M, n_in]
    y, h = dy.forward(gpu(h_in), gpu(L.W1), gpu(L.W2), gpu(L.bias), variant=variant, act=act,
                      stash_h=True, act_in="gelu")
    torch.cuda.synchronize()
    ry, rh = oracle.forward(variant, n_in, n_out, D, gelu_bf16(h_in), L.f64("W1"), L.f64("W2"),
                            L.f64("bias"), act=oracle.ACT_GELU if act == "gelu" else oracle.ACT_NONE,
                            want_h=True)
    assert_close(y, ry, "bf16", "Y")
    if act == "gelu":
        assert_close(h, rh, "bf16", "H")


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda c: "x".join(map(str, c)))
def test_backward_dw_gelu_in(shape, variant):
    n_in, n_out, D, M = shape
    banner("backward_dw_gelu_in", shape, variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=41)
    dw1, dw2, db = dy.backward_dw(gpu(L.dZ), gpu(L.H_in), D, variant=variant, act_in="gelu")
    torch.cuda.synchronize()
    r1, r2, rb = oracle.backward_dw(variant, n_in, n_out, D, L.f64("dZ"), gelu_bf16(L.H_in))
    assert_close(dw1, r1, "bf16", "dW1")
    assert_close(dw2, r2, "bf16", "dW2")
    assert_close(db, rb, "bf16", "db")


@pytest.mark.parametrize("variant", VARIANTS)
def test_act_in_none_is_the_plain_call(variant):
    """act_in = NONE runs exactly dyad_forward / dyad_backward_dw: bitwise equal outputs."""
    n_in, n_out, D, M = 768, 3072, 4, 333
    banner("act_in_none", variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=42)
    x, w1, w2, b, dz = (gpu(t) for t in (L.X, L.W1, L.W2, L.bias, L.dZ))
    assert torch.equal(dy.forward(x, w1, w2, b, variant=variant),
                       dy.forward(x, w1, w2, b, variant=variant, act_in="none"))
    v = dy.VARIANTS[variant]
    y = torch.empty((M, n_out), dtype=torch.bfloat16, device=DEV)
    s = torch.cuda.current_stream().cuda_stream
    assert dy.dyad_forward_ex(v, n_in, n_out, D, M, dy.BF16, dy.ACT_NONE, x.data_ptr(), w1.data_ptr(),
                              w2.data_ptr(), b.data_ptr(), dy.ACT_NONE, y.data_ptr(), None, s) == 0
    assert torch.equal(y, dy.forward(x, w1, w2, b, variant=variant))
    assert (dy.dyad_dw_workspace_bytes_ex(v, n_in, n_out, D, M, dy.BF16, dy.ACT_NONE) ==
            dy.dyad_dw_workspace_bytes(v, n_in, n_out, D, M, dy.BF16))
    a = dy.backward_dw(dz, x, D, variant=variant)
    torch.cuda.synchronize()
    for u, w in zip(a, dy.backward_dw(dz, x, D, variant=variant, act_in="none")):
        assert torch.equal(u, w)


def test_refusals_before_any_launch():
    """Shapes and dtypes without a fused kernel are refused (no output is touched)."""
    s = torch.cuda.current_stream().cuda_stream
    sentinel = -1536.0

    def fwd(variant, n_in, n_out, D, M, dtype=torch.bfloat16):
        code = dy.BF16 if dtype == torch.bfloat16 else dy.F32
        x = torch.randn((M, n_in), device=DEV).to(dtype)
        w = torch.zeros((D, -(-n_out // D), -(-n_in // D)), device=DEV, dtype=dtype)
        y = torch.full((M, n_out), sentinel, device=DEV, dtype=dtype)
        rc = dy.dyad_forward_ex(dy.VARIANTS[variant], n_in, n_out, D, M, code, dy.ACT_GELU, x.data_ptr(),
                                w.data_ptr(), w.data_ptr(), None, dy.ACT_NONE, y.data_ptr(), None, s)
        torch.cuda.synchronize()
        assert bool((y == sentinel).all())
        return rc

    assert fwd("IT", 768, 3072, 4, 64, torch.float32) == -4    # fp32
    assert fwd("IT", 770, 3072, 4, 64) == -2                   # zero-padded width
    assert fwd("OT", 2048, 1024, 16, 64) == -2                 # output transpose at n_dyad 16
    assert fwd("IT", 768, 3072, 3, 64) == -2                   # n_dyad 3
    z = torch.zeros((64, 96), device=DEV, dtype=torch.bfloat16)
    x = torch.zeros((64, 96), device=DEV, dtype=torch.bfloat16)
    w = torch.empty((4, 24, 24), device=DEV, dtype=torch.bfloat16)
    assert dy.dyad_backward_dw_ex(0, 96, 96, 4, 64, dy.BF16, dy.ACT_GELU, z.data_ptr(), x.data_ptr(), w.data_ptr(),
                                  w.data_ptr(), None, None, 0, s) == -2   # blocks of 24
    assert dy.dyad_dw_workspace_bytes_ex(0, 96, 96, 4, 64, dy.BF16, dy.ACT_GELU) == 0


def sample_rows(M, n, seed):
    rng = np.random.default_rng(seed)
    return np.array(sorted(set(rng.choice(M, size=n, replace=False).tolist()) | {0, M - 1}))


@pytest.mark.parametrize("variant", VARIANTS)
def test_opt125m_fc2_fused_full_size_sampled(variant):
    """OPT-125m fc2 (3072 -> 768, n_dyad 4, 16384 tokens) as the fused block runs it:
    forward on GELU(h) and the weight gradient on GELU(h); sampled tokens and entries."""
    (_, _, _), (_, n_in, n_out) = OPT125M.layers
    D, M = OPT125M.n_dyad, OPT125M.M
    banner("opt125m_fc2_fused", variant)
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=1)
    h = gpu(L.H_in)
    y = dy.forward(h, gpu(L.W1), gpu(L.W2), gpu(L.bias), variant=variant, act_in="gelu")
    dw1, dw2, db = dy.backward_dw(gpu(L.dZ), h, D, variant=variant, act_in="gelu")
    torch.cuda.synchronize()
    rows = sample_rows(M, 40, 9)
    ry = oracle.forward(variant, n_in, n_out, D, gelu_bf16(L.H_in[rows]), L.f64("W1"), L.f64("W2"),
                        L.f64("bias"))
    assert_close(y[rows], ry, "bf16", "Y rows")
    rng = np.random.default_rng(12)
    n = 200
    comp = rng.integers(1, 3, n)
    i, j, k = rng.integers(0, D, n), rng.integers(0, n_out // D, n), rng.integers(0, n_in // D, n)
    ref = np.zeros(n)
    rdb = np.zeros(n_out)
    for lo in range(0, M, 4096):
        z = L.dZ[lo:lo + 4096].to(torch.float64).numpy()
        ref += oracle.backward_dw_entries(variant, n_in, n_out, D, z, gelu_bf16(L.H_in[lo:lo + 4096]),
                                          comp, i, j, k)
        rdb += oracle.bias_grad(z)
    ti, tj, tk = (torch.as_tensor(a, device=DEV) for a in (i, j, k))
    got = np.where(comp == 1, to64(dw1[ti, tj, tk]), to64(dw2[ti, tj, tk]))
    assert_close(got, ref, "bf16", "dW entries")
    assert_close(db, rdb, "bf16", "db")


@pytest.mark.parametrize("variant", VARIANTS)
def test_fused_ff_module_against_oracle_chain(variant):
    """DyadFF(fused=True) forward and backward against the oracle chain (fc1 pre-activation,
    GELU, fc2; GELU' on fc2's input gradient), and against DyadFF(fused=False)."""
    d, ffn, D, M = 512, 2048, 4, 300
    banner("fused_ff", variant)
    torch.manual_seed(5)
    ff = DyadFF(d, ffn, D, variant, device=DEV, fused=True)
    ref_ff = DyadFF(d, ffn, D, variant, device=DEV, fused=False)
    ref_ff.load_state_dict(ff.state_dict())
    x = torch.randn((M, d), device=DEV).bfloat16()
    g = torch.randn((M, d), device=DEV).bfloat16()
    xa = x.clone().requires_grad_(True)
    y = ff(xa)
    y.backward(g)
    xb = x.clone().requires_grad_(True)
    y0 = ref_ff(xb)
    y0.backward(g)
    torch.cuda.synchronize()
    W = lambda p: p.detach().to(torch.float64).cpu().numpy()  # noqa: E731
    X = to64(x)
    rh = oracle.forward(variant, d, ffn, D, X, W(ff.fc1.w1), W(ff.fc1.w2), W(ff.fc1.bias))
    ra = oracle.gelu_array(rh)
    ry = oracle.forward(variant, ffn, d, D, ra, W(ff.fc2.w1), W(ff.fc2.w2), W(ff.fc2.bias))
    G = to64(g)
    rdh = oracle.backward_dx(variant, ffn, d, D, G, W(ff.fc2.w1), W(ff.fc2.w2), act_in=oracle.ACT_GELU, H_in=rh)
    rw21, rw22, rb2 = oracle.backward_dw(variant, ffn, d, D, G, ra)
    rdx = oracle.backward_dx(variant, d, ffn, D, rdh, W(ff.fc1.w1), W(ff.fc1.w2))
    rw11, rw12, rb1 = oracle.backward_dw(variant, d, ffn, D, rdh, X)
    # a chain of bf16 layers: the max-norm bar (each layer rounds its output before the next)
    for got, ref, what in ((y, ry, "y"), (xa.grad, rdx, "dx"), (ff.fc2.w1.grad, rw21, "dW21"),
                           (ff.fc2.w2.grad, rw22, "dW22"), (ff.fc2.bias.grad, rb2, "db2"),
                           (ff.fc1.w1.grad, rw11, "dW11"), (ff.fc1.w2.grad, rw12, "dW12"),
                           (ff.fc1.bias.grad, rb1, "db1")):
        err = float(np.abs(to64(got) - ref).max() / np.abs(ref).max())
        assert err <= 2e-2, (what, err)
    # the fused and unfused blocks round the same values: their outputs agree closely
    assert float((y.float() - y0.float()).abs().max() / y0.float().abs().max()) <= 1e-2
    for p, q in zip(ff.parameters(), ref_ff.parameters()):
        assert float((p.grad.float() - q.grad.float()).abs().max() / q.grad.float().abs().max()) <= 1e-2
