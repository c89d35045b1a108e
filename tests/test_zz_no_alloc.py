"""dyad_forward_noalloc through the C-ABI: its outputs against dyad_forward's on the
same inputs (the bf16 bar of the parity tests), on two calls in a row with the second
smaller, for plans whose split buffer fits the fixed scratch array and for one whose
buffer would not (which then runs a plan that needs none); and no device memory is
taken by the call, where dyad_forward on a new stream takes its pool buffer."""
import numpy as np
import pytest
import torch

import oracle
import paper_2312_06881_amd as dy
from workloads import layer_inputs
from tests.parity_util import assert_close, maxnorm_rel, to64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def banner(*what):
    print("CASE", *what, flush=True)


def assert_close_gpu(got, other, what):
    """Two bf16 results of the same fp32 sums taken in different orders: the bar of the
    parity tests (max-norm 2e-2) and, elementwise, one bf16 ulp (each side is within half
    an ulp of its own fp32 sum) plus 2^-10 of the max-norm for the order of the sums."""
    g, r = to64(got), to64(other)
    assert maxnorm_rel(g, r) <= 2e-2, what
    bound = 2.0 ** -7 * np.abs(r) + 2.0 ** -10 * float(np.abs(r).max())
    bad = np.abs(g - r) > bound
    assert not bad.any(), f"{what}: {int(bad.sum())} elements apart by more than one ulp"


def run(fn, variant, L, act, stream):
    n_in, n_out, D, M = L.n_in, L.n_out, L.n_dyad, L.M
    x, w1, w2, b = (t.to(DEV) for t in (L.X, L.W1, L.W2, L.bias))
    y = torch.empty((M, n_out), dtype=torch.bfloat16, device=DEV)
    h = torch.empty_like(y) if act == dy.ACT_GELU else None
    rc = fn(dy.VARIANTS[variant], n_in, n_out, D, M, dy.BF16, x.data_ptr(), w1.data_ptr(), w2.data_ptr(),
            b.data_ptr(), act, y.data_ptr(), None if h is None else h.data_ptr(), stream.cuda_stream)
    assert rc == 0, dy.dyad_strerror(rc)
    stream.synchronize()
    return y, h


# (n_in, n_out, n_dyad, [M of the first call, M of the second]): small batches on the
# split-reduction paths (buffers of a few MiB), n_dyad 16 with 64-column blocks at a
# batch whose two fp32 component slices (512 MiB) exceed the array, and zero-padded
# blocks (n_dyad 5) on the padded forms, whose copies and slice (15 MiB) fit it
CASES = [
    (8192, 8192, 16, (32, 16)),
    (768, 3072, 4, (32, 9)),
    (3072, 768, 4, (200, 17)),
    (4096, 1024, 16, (16384, 2100)),
    (768, 3072, 5, (1000, 600)),
]


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}x{c[1]}xD{c[2]}")
def test_noalloc_matches_forward_two_calls(case, variant):
    n_in, n_out, D, Ms = case
    s = torch.cuda.Stream(DEV)
    for k, M in enumerate(Ms):
        banner("noalloc", n_in, n_out, D, M, variant)
        act = dy.ACT_GELU if k == 0 else dy.ACT_NONE
        L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=20 + k)
        y0, h0 = run(dy.dyad_forward, variant, L, act, s)
        y1, h1 = run(dy.dyad_forward_noalloc, variant, L, act, s)
        assert_close_gpu(y1, y0, "Y noalloc vs forward")
        if h0 is not None:
            assert_close_gpu(h1, h0, "H noalloc vs forward")
        # and the oracle on (sampled) tokens, at the parity tests' bar
        rows = np.arange(M) if M <= 256 else np.unique(np.r_[0:8, M - 8:M, np.linspace(0, M - 1, 40).astype(int)])
        ry, rh = oracle.forward(variant, n_in, n_out, D, L.X[rows].to(torch.float64).numpy(), L.f64("W1"),
                                L.f64("W2"), L.f64("bias"), act=act, want_h=True)
        assert_close(y1[rows], ry, "bf16", "Y noalloc vs oracle")
        if h1 is not None:
            assert_close(h1[rows], rh, "bf16", "H noalloc vs oracle")


def test_noalloc_takes_no_device_memory():
    n_in, n_out, D, M = 8192, 8192, 16, 32
    banner("noalloc_memory")
    L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=30)
    s = torch.cuda.Stream(DEV)
    run(dy.dyad_forward_noalloc, "IT", L, dy.ACT_NONE, s)      # scratch address looked up
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info(DEV)[0]
    run(dy.dyad_forward_noalloc, "IT", L, dy.ACT_NONE, s)
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info(DEV)[0] == free0
    # dyad_forward on a stream it has not seen takes a pool buffer (at least 1 MiB)
    s2 = torch.cuda.Stream(DEV)
    run(dy.dyad_forward, "IT", L, dy.ACT_NONE, s2)
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info(DEV)[0] < free0


def test_noalloc_rejects_bad_arguments_like_forward():
    FAKE = 1 << 20
    a = dict(variant=0, n_in=64, n_out=256, n_dyad=4, M=8, dtype=1, X=FAKE, W1=FAKE, W2=FAKE, bias=None,
             act=0, Y=FAKE, H=None, stream=None)
    for bad, code in ((dict(variant=3), -1), (dict(dtype=7), -4), (dict(X=FAKE + 8), -3), (dict(Y=None), -1)):
        b = {**a, **bad}
        assert dy.dyad_forward_noalloc(**b) == code == dy.dyad_forward(**b)
