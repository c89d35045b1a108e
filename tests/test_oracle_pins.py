"""Pins of the CPU oracle against things other than itself (all CPU-only).

Each test fixes the oracle to an independent statement of the paper:
  * a dense weight assembled from ``scipy.linalg.block_diag`` (Sec. 2.2.1, Eq. 2)
    and the explicit permutation matrix P of Eq. 5 (Sec. 2.2.2), composed as the
    paper's Eq. 6 / Eq. 13 / Eq. 16 compose it;
  * a gather / batched-product / scatter form built from the index definitions
    (Eq. 3 and the strided view of Eq. 9 as explicit index arrays, the output
    map of Sec. 2.4 as an explicit scatter);
  * special cases: n_dyad = 1 collapses to one dense matrix W1+W2; W2 = 0 gives a
    textbook batched GEMM; linearity;
  * structural counts: each component stores n_in*n_out/n_dyad distinct dense
    positions, and the OPT-125m parameter counts printed in the paper's appendix;
  * the backward pass against central finite differences of the forward pass
    and against the dense gradient pushed through P;
  * GELU against scipy's normal CDF and its own finite differences.
"""
import math
import os

import numpy as np
import pytest
import scipy.linalg
import scipy.stats

import oracle
from oracle import ACT_GELU, ACT_NONE

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

SHAPES = [  # (n_in, n_out, D): square and rectangular blocks, D | b and D does not divide b
    (16, 16, 4),      # the figure case: blocks 4x4, n_dyad 4
    (8, 12, 2),
    (12, 18, 3),      # bi=4, bo=6: D divides neither block size
    (64, 256, 4),
    (24, 40, 8),      # bi=3, bo=5
    (32, 16, 16),     # bi=2, bo=1
    (10, 6, 1),       # dense
]


def perm_eq5(D, b):
    """Permutation matrix of Eq. 5 for n_dyad=D and block size b: P[a, c] = 1 iff c = D*(a % b) + a // b."""
    n = D * b
    P = np.zeros((n, n))
    for a in range(n):
        P[a, D * (a % b) + a // b] = 1.0
    return P


def dense_weight(variant, n_in, n_out, D, W1, W2):
    """Dense W from the two components, composed through P (Eq. 6 reading: BlockTrans X-view = P X)."""
    bi, bo = n_in // D, n_out // D
    B1 = scipy.linalg.block_diag(*W1)
    B2 = scipy.linalg.block_diag(*W2)
    P_in, P_out = perm_eq5(D, bi), perm_eq5(D, bo)
    if variant == "IT":      # Y2 = W2' (P X)
        W2d = B2 @ P_in
    elif variant == "OT":    # Y2 = P^T (W2' X), Eq. 13
        W2d = P_out.T @ B2
    else:                    # Y2 = P2^T W2' (P1 X), Eq. 16
        W2d = P_out.T @ B2 @ P_in
    return B1 + W2d


def rand_case(n_in, n_out, D, M, seed):
    rng = np.random.default_rng(seed)
    bi, bo = n_in // D, n_out // D
    return (rng.standard_normal((M, n_in)), rng.standard_normal((D, bo, bi)),
            rng.standard_normal((D, bo, bi)), rng.standard_normal(n_out))


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
@pytest.mark.parametrize("shape", SHAPES)
def test_forward_matches_dense_through_permutation(variant, shape):
    n_in, n_out, D = shape
    X, W1, W2, b = rand_case(n_in, n_out, D, 5, 7)
    W = dense_weight(variant, n_in, n_out, D, W1, W2)
    Y = oracle.forward(variant, n_in, n_out, D, X, W1, W2, b)
    np.testing.assert_allclose(Y, X @ W.T + b, rtol=1e-12, atol=1e-12)


def gathered_block_forward(variant, n_in, n_out, D, X, W1, W2, b):
    """Forward from the definitions, in gather / batched-product / scatter form:
    block i of component 1 reads input features i*bi + k (Eq. 3); component 2
    reads features k*D + i under an input transpose (the strided view of Eq. 9,
    as an explicit index array) and writes output j*D + i under an output
    transpose (Sec. 2.4, as an explicit scatter), else i*bo + j."""
    bi, bo = n_in // D, n_out // D
    i_idx = np.arange(D)[:, None]
    blk_in = i_idx * bi + np.arange(bi)[None, :]          # [D, bi]: i*bi + k
    str_in = np.arange(bi)[None, :] * D + i_idx           # [D, bi]: k*D + i
    blk_out = i_idx * bo + np.arange(bo)[None, :]         # [D, bo]: i*bo + j
    str_out = np.arange(bo)[None, :] * D + i_idx          # [D, bo]: j*D + i
    in2 = str_in if variant in ("IT", "DT") else blk_in
    out2 = str_out if variant in ("OT", "DT") else blk_out
    Y = np.tile(b, (X.shape[0], 1)).astype(np.float64)
    for W, cols, rows in ((W1, blk_in, blk_out), (W2, in2, out2)):
        G = X[:, cols]                                    # [M, D, bi] gathered input blocks
        Z = np.einsum("ijk,mik->mij", W, G)               # [M, D, bo] block products
        np.add.at(Y, (slice(None), rows), Z)              # scatter to the output features
    return Y


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
@pytest.mark.parametrize("shape", SHAPES)
def test_forward_matches_gathered_block_form(variant, shape):
    n_in, n_out, D = shape
    X, W1, W2, b = rand_case(n_in, n_out, D, 6, 11)
    Y = oracle.forward(variant, n_in, n_out, D, X, W1, W2, b)
    np.testing.assert_allclose(Y, gathered_block_forward(variant, n_in, n_out, D, X, W1, W2, b),
                               rtol=1e-12, atol=1e-12)


def test_eq9_view_is_P_x_not_PT_x():
    """The strided view of Eq. 9 equals P X for Eq. 5's P; P^T X agrees only when block size == n_dyad."""
    for (bi, D) in [(16, 4), (3, 2), (4, 4)]:
        n = bi * D
        x = np.arange(n, dtype=float)
        view = x.reshape(bi, D).T.reshape(-1)
        P = perm_eq5(D, bi)
        assert np.array_equal(view, P @ x)
        assert np.array_equal(view, P.T @ x) == (bi == D)


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
def test_ndyad_1_is_dense(variant):
    n_in, n_out = 9, 7
    X, W1, W2, b = rand_case(n_in, n_out, 1, 4, 3)
    Y = oracle.forward(variant, n_in, n_out, 1, X, W1, W2, b)
    np.testing.assert_allclose(Y, X @ (W1[0] + W2[0]).T + b, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shape", SHAPES)
def test_w2_zero_is_batched_gemm(shape):
    n_in, n_out, D = shape
    X, W1, _, b = rand_case(n_in, n_out, D, 4, 5)
    W2 = np.zeros_like(W1)
    ref = np.einsum("mik,ijk->mij", X.reshape(4, D, n_in // D), W1).reshape(4, n_out) + b
    for v in ("IT", "OT", "DT"):
        np.testing.assert_allclose(oracle.forward(v, n_in, n_out, D, X, W1, W2, b), ref,
                                   rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
def test_linearity(variant):
    n_in, n_out, D = 24, 40, 4
    Xa, W1a, W2a, _ = rand_case(n_in, n_out, D, 3, 1)
    Xb, W1b, W2b, _ = rand_case(n_in, n_out, D, 3, 2)
    f = lambda X, W1, W2: oracle.forward(variant, n_in, n_out, D, X, W1, W2)  # noqa: E731
    np.testing.assert_allclose(f(2 * Xa - Xb, W1a, W2a), 2 * f(Xa, W1a, W2a) - f(Xb, W1a, W2a),
                               rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(f(Xa, W1a + W1b, W2a - 3 * W2b),
                               f(Xa, W1a, W2a) + f(Xa, W1b, -3 * W2b), rtol=1e-10, atol=1e-10)


def materialise(variant, n_in, n_out, D, W1, W2):
    """Dense W read back from the oracle by feeding the identity as the tokens."""
    return oracle.forward(variant, n_in, n_out, D, np.eye(n_in), W1, W2).T


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
@pytest.mark.parametrize("shape", SHAPES)
def test_support_counts(variant, shape):
    """Each component covers n_in*n_out/D distinct positions; the overlap is n_in*n_out/D^2 when D | bi, bo."""
    n_in, n_out, D = shape
    bi, bo = n_in // D, n_out // D
    rng = np.random.default_rng(0)
    W1 = rng.uniform(1, 2, (D, bo, bi))
    W2 = rng.uniform(1, 2, (D, bo, bi))
    s1 = materialise(variant, n_in, n_out, D, W1, np.zeros_like(W2)) != 0
    s2 = materialise(variant, n_in, n_out, D, np.zeros_like(W1), W2) != 0
    assert s1.sum() == n_in * n_out // D
    assert s2.sum() == n_in * n_out // D
    assert s1.sum() + s2.sum() == 2 * n_in * n_out // D
    if bi % D == 0 and bo % D == 0:
        assert (s1 & s2).sum() == n_in * n_out // (D * D)
    both = materialise(variant, n_in, n_out, D, W1, W2) != 0
    assert np.array_equal(both, s1 | s2)


def test_overlap_when_ndyad_does_not_divide_blocks():
    """IT at n_in=12, n_out=18, D=3: the components share 36 positions (the D^2 formula would say 24)."""
    rng = np.random.default_rng(1)
    W = rng.uniform(1, 2, (3, 6, 4))
    s1 = materialise("IT", 12, 18, 3, W, 0 * W) != 0
    s2 = materialise("IT", 12, 18, 3, 0 * W, W) != 0
    assert (s1 & s2).sum() == 36


def _read_param_table():
    rows = []
    with open(os.path.join(GOLDEN, "opt125m_params.txt")) as fh:
        for line in fh:
            if line.strip() and not line.startswith("#"):
                name, kind, D, p = line.split()
                rows.append((name, kind, int(D), float(p)))
    return rows


def test_opt125m_parameter_counts_match_paper():
    """OPT-125m: 12 decoder layers of width 768, FF 3072, learned positions 2050 x 768."""
    d, ffn, L, n_pos = 768, 3072, 12, 2050
    attn = 4 * (d * d + d)
    norms = 2 * 2 * d
    rng = np.random.default_rng(0)
    for name, kind, D, printed in _read_param_table():
        if kind == "dense":
            ff = 2 * d * ffn + ffn + d
        else:
            ff = 0
            for n_in, n_out in ((d, ffn), (ffn, d)):
                W1 = np.zeros((D, n_out // D, n_in // D))
                W2 = np.zeros((D, n_out // D, n_in // D))
                # the oracle accepts exactly these component shapes, and rejects others
                oracle.forward("IT", n_in, n_out, D, rng.standard_normal((1, n_in)), W1, W2)
                with pytest.raises(ValueError):
                    oracle.forward("IT", n_in, n_out, D, rng.standard_normal((1, n_in)),
                                   W1[:, :-1], W2)
                ff += W1.size + W2.size + n_out
        total = L * (attn + norms + ff) + 2 * d + n_pos * d
        assert round(total / 1e6, 2) == printed, name


def flat_loss(variant, n_in, n_out, D, X, W1, W2, b, G, act):
    Y = oracle.forward(variant, n_in, n_out, D, X, W1, W2, b, act=act)
    return float((Y * G).sum())


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
@pytest.mark.parametrize("shape", [(8, 12, 2), (12, 18, 3), (16, 8, 4)])
def test_backward_matches_finite_differences(variant, shape):
    n_in, n_out, D = shape
    M = 3
    X, W1, W2, b = rand_case(n_in, n_out, D, M, 21)
    G = np.random.default_rng(22).standard_normal((M, n_out))
    dX = oracle.backward_dx(variant, n_in, n_out, D, G, W1, W2)
    dW1, dW2, db = oracle.backward_dw(variant, n_in, n_out, D, G, X)
    eps = 1e-6
    L = lambda X_, W1_, W2_, b_: flat_loss(variant, n_in, n_out, D, X_, W1_, W2_, b_, G, ACT_NONE)  # noqa
    for arr, grad, idx in ((X, dX, 0), (W1, dW1, 1), (W2, dW2, 2), (b, db, 3)):
        num = np.zeros_like(arr)
        for pos in np.ndindex(arr.shape):
            args_p = [X.copy(), W1.copy(), W2.copy(), b.copy()]
            args_m = [X.copy(), W1.copy(), W2.copy(), b.copy()]
            args_p[idx][pos] += eps
            args_m[idx][pos] -= eps
            num[pos] = (L(*args_p) - L(*args_m)) / (2 * eps)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
def test_gelu_chain_finite_differences(variant):
    """X = GELU(H_in): dL/dH_in = dX(act_in=GELU); Y = GELU(W X + b): H stash is the pre-activation."""
    n_in, n_out, D, M = 12, 8, 4, 2
    H_in, W1, W2, b = rand_case(n_in, n_out, D, M, 31)
    G = np.random.default_rng(32).standard_normal((M, n_out))
    gelu_v = np.vectorize(oracle.gelu)
    X = gelu_v(H_in)
    dH = oracle.backward_dx(variant, n_in, n_out, D, G, W1, W2, act_in=ACT_GELU, H_in=H_in)
    eps = 1e-6
    num = np.zeros_like(H_in)
    for pos in np.ndindex(H_in.shape):
        hp, hm = H_in.copy(), H_in.copy()
        hp[pos] += eps
        hm[pos] -= eps
        num[pos] = (flat_loss(variant, n_in, n_out, D, gelu_v(hp), W1, W2, b, G, ACT_NONE) -
                    flat_loss(variant, n_in, n_out, D, gelu_v(hm), W1, W2, b, G, ACT_NONE)) / (2 * eps)
    np.testing.assert_allclose(dH, num, rtol=1e-6, atol=1e-8)
    Y, H = oracle.forward(variant, n_in, n_out, D, X, W1, W2, b, act=ACT_GELU, want_h=True)
    W = dense_weight(variant, n_in, n_out, D, W1, W2)
    np.testing.assert_allclose(H, X @ W.T + b, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(Y, gelu_v(H), rtol=0, atol=0)


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
@pytest.mark.parametrize("shape", SHAPES)
def test_backward_matches_dense_gradient(variant, shape):
    """dX = dZ W; dW_c is dL/dW_c of L = <dZ, X W^T>, pushed through block_diag and P."""
    n_in, n_out, D = shape
    bi, bo = n_in // D, n_out // D
    M = 7
    X, W1, W2, _ = rand_case(n_in, n_out, D, M, 41)
    dZ = np.random.default_rng(42).standard_normal((M, n_out))
    W = dense_weight(variant, n_in, n_out, D, W1, W2)
    np.testing.assert_allclose(oracle.backward_dx(variant, n_in, n_out, D, dZ, W1, W2), dZ @ W,
                               rtol=1e-12, atol=1e-12)
    G = dZ.T @ X                                          # dL/dW, dense n_out x n_in
    P_in, P_out = perm_eq5(D, bi), perm_eq5(D, bo)
    G2 = {"IT": G @ P_in.T, "OT": P_out @ G, "DT": P_out @ G @ P_in.T}[variant]

    def blocks(A):
        return np.stack([A[i * bo:(i + 1) * bo, i * bi:(i + 1) * bi] for i in range(D)])

    dW1, dW2, db = oracle.backward_dw(variant, n_in, n_out, D, dZ, X)
    np.testing.assert_allclose(dW1, blocks(G), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW2, blocks(G2), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, dZ.sum(0), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("fwd,bwd", [("IT", "OT"), ("OT", "IT"), ("DT", "DT")])
def test_transpose_symmetry(fwd, bwd):
    """W_IT(W1,W2)^T = W_OT(W1^T,W2^T) and W_DT^T = W_DT(.^T): dX of one variant is the other's forward."""
    n_in, n_out, D = 24, 40, 4
    _, W1, W2, _ = rand_case(n_in, n_out, D, 1, 51)
    dZ = np.random.default_rng(52).standard_normal((6, n_out))
    dX = oracle.backward_dx(fwd, n_in, n_out, D, dZ, W1, W2)
    Y = oracle.forward(bwd, n_out, n_in, D, dZ, W1.transpose(0, 2, 1), W2.transpose(0, 2, 1))
    np.testing.assert_allclose(dX, Y, rtol=1e-12, atol=1e-12)


def test_dw_entries_agree_with_full_dw():
    n_in, n_out, D = 24, 40, 4
    for v in ("IT", "OT", "DT"):
        X, _, _, _ = rand_case(n_in, n_out, D, 9, 61)
        dZ = np.random.default_rng(62).standard_normal((9, n_out))
        dW1, dW2, _ = oracle.backward_dw(v, n_in, n_out, D, dZ, X)
        rng = np.random.default_rng(63)
        n = 50
        comp = rng.integers(1, 3, n)
        i, j, k = rng.integers(0, D, n), rng.integers(0, n_out // D, n), rng.integers(0, n_in // D, n)
        got = oracle.backward_dw_entries(v, n_in, n_out, D, dZ, X, comp, i, j, k)
        ref = np.where(comp == 1, dW1[i, j, k], dW2[i, j, k])
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_empty_token_batch():
    n_in, n_out, D = 8, 12, 2
    _, W1, W2, b = rand_case(n_in, n_out, D, 1, 71)
    assert oracle.forward("IT", n_in, n_out, D, np.zeros((0, n_in)), W1, W2, b).shape == (0, n_out)
    dW1, dW2, db = oracle.backward_dw("DT", n_in, n_out, D, np.zeros((0, n_out)), np.zeros((0, n_in)))
    assert not dW1.any() and not dW2.any() and not db.any()


def test_gelu_against_normal_cdf():
    for x in (-6.0, -2.5, -1.0, -0.3, 0.0, 0.4, 1.0, 3.0, 8.0):
        assert oracle.gelu(x) == pytest.approx(x * scipy.stats.norm.cdf(x), rel=1e-14, abs=1e-300)
        assert oracle.gelu(x) - oracle.gelu(-x) == pytest.approx(x, rel=1e-14, abs=1e-15)
        h = 1e-5
        fd = (oracle.gelu(x + h) - oracle.gelu(x - h)) / (2 * h)
        assert oracle.gelu_grad(x) == pytest.approx(fd, rel=1e-8, abs=1e-10)
    assert oracle.gelu_grad(0.0) == 0.5
    assert oracle.gelu(1.0) == pytest.approx(0.8413447460685429, rel=1e-15)  # Phi(1)
    assert math.isclose(oracle.gelu_grad(30.0), 1.0)


def test_gelu_array_against_normal_cdf():
    """The elementwise form used for a layer whose input is GELU(H): scipy's normal CDF,
    any shape, and the scalar form bit for bit."""
    x = np.random.default_rng(3).standard_normal((37, 11)) * 4.0
    g = oracle.gelu_array(x)
    assert g.shape == x.shape
    np.testing.assert_allclose(g, x * scipy.stats.norm.cdf(x), rtol=1e-13, atol=1e-300)
    assert all(g.flat[i] == oracle.gelu(x.flat[i]) for i in range(0, x.size, 7))


# ---- widths that n_dyad does not divide: zero-padding (appendix, caveat on rectangular W) ----

PADDED = [  # (n_in, n_out, D) with D dividing at most one width
    (6, 7, 2),        # the appendix's 7 x 6 weight: one zero row makes n_dyad 2 possible
    (10, 13, 4),
    (30, 17, 3),
    (5, 9, 8),        # bi = 1, bo = 2: most entries touch padding
    (12, 10, 4),      # n_in divisible, n_out not
]


def padded_blocks(n_in, n_out, D):
    return -(-n_in // D), -(-n_out // D)


def padded_dense(variant, n_in, n_out, D, W1, W2):
    """Dense weight of the zero-padded layer: the divisible layer of widths D*bi -> D*bo
    (assembled through block_diag and P), restricted to its first n_out rows and n_in columns."""
    bi, bo = padded_blocks(n_in, n_out, D)
    return dense_weight(variant, D * bi, D * bo, D, W1, W2)[:n_out, :n_in]


def padded_case(n_in, n_out, D, M, seed):
    rng = np.random.default_rng(seed)
    bi, bo = padded_blocks(n_in, n_out, D)
    return (rng.standard_normal((M, n_in)), rng.standard_normal((D, bo, bi)),
            rng.standard_normal((D, bo, bi)), rng.standard_normal(n_out))


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
@pytest.mark.parametrize("shape", PADDED)
def test_padded_forward_is_cropped_dense(variant, shape):
    n_in, n_out, D = shape
    X, W1, W2, b = padded_case(n_in, n_out, D, 5, 81)
    Y = oracle.forward(variant, n_in, n_out, D, X, W1, W2, b)
    W = padded_dense(variant, n_in, n_out, D, W1, W2)
    np.testing.assert_allclose(Y, X @ W.T + b, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
@pytest.mark.parametrize("shape", PADDED)
def test_padded_layer_is_divisible_layer_on_zero_padded_input(variant, shape):
    """The caveat's recipe taken literally: append zero input features, run the layer whose
    widths n_dyad divides, keep the first n_out outputs.  GELU and the H stash follow."""
    n_in, n_out, D = shape
    bi, bo = padded_blocks(n_in, n_out, D)
    X, W1, W2, b = padded_case(n_in, n_out, D, 4, 82)
    Xp = np.zeros((4, D * bi))
    Xp[:, :n_in] = X
    bp = np.concatenate([b, np.random.default_rng(83).standard_normal(D * bo - n_out)])
    Yp, Hp = oracle.forward(variant, D * bi, D * bo, D, Xp, W1, W2, bp, act=ACT_GELU, want_h=True)
    Y, H = oracle.forward(variant, n_in, n_out, D, X, W1, W2, b, act=ACT_GELU, want_h=True)
    np.testing.assert_array_equal(Y, Yp[:, :n_out])
    np.testing.assert_array_equal(H, Hp[:, :n_out])


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
@pytest.mark.parametrize("shape", PADDED)
def test_padded_backward_matches_dense_gradient(variant, shape):
    """dX = dZ W over the cropped dense W; dW_c is the padded layer's dense gradient (dZ and X
    with zero columns appended) gathered through block_diag and P, so entries that touch
    padding get exactly zero."""
    n_in, n_out, D = shape
    bi, bo = padded_blocks(n_in, n_out, D)
    M = 6
    X, W1, W2, _ = padded_case(n_in, n_out, D, M, 84)
    dZ = np.random.default_rng(85).standard_normal((M, n_out))
    W = padded_dense(variant, n_in, n_out, D, W1, W2)
    np.testing.assert_allclose(oracle.backward_dx(variant, n_in, n_out, D, dZ, W1, W2), dZ @ W,
                               rtol=1e-12, atol=1e-12)
    Xp = np.zeros((M, D * bi))
    Xp[:, :n_in] = X
    dZp = np.zeros((M, D * bo))
    dZp[:, :n_out] = dZ
    G = dZp.T @ Xp
    P_in, P_out = perm_eq5(D, bi), perm_eq5(D, bo)
    G2 = {"IT": G @ P_in.T, "OT": P_out @ G, "DT": P_out @ G @ P_in.T}[variant]

    def blocks(A):
        return np.stack([A[i * bo:(i + 1) * bo, i * bi:(i + 1) * bi] for i in range(D)])

    dW1, dW2, db = oracle.backward_dw(variant, n_in, n_out, D, dZ, X)
    np.testing.assert_allclose(dW1, blocks(G), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW2, blocks(G2), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, dZ.sum(0), rtol=1e-12, atol=1e-12)
    comp = np.repeat([1, 2], D * bo * bi)
    i, j, k = (a.ravel() for a in np.meshgrid(np.arange(D), np.arange(bo), np.arange(bi), indexing="ij"))
    i, j, k = np.tile(i, 2), np.tile(j, 2), np.tile(k, 2)
    got = oracle.backward_dw_entries(variant, n_in, n_out, D, dZ, X, comp, i, j, k)
    np.testing.assert_allclose(got, np.concatenate([dW1.ravel(), dW2.ravel()]), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("variant", ["IT", "OT", "DT"])
def test_padded_backward_finite_differences(variant):
    n_in, n_out, D = 6, 7, 2
    M = 2
    X, W1, W2, b = padded_case(n_in, n_out, D, M, 86)
    G = np.random.default_rng(87).standard_normal((M, n_out))
    dX = oracle.backward_dx(variant, n_in, n_out, D, G, W1, W2)
    dW1, dW2, db = oracle.backward_dw(variant, n_in, n_out, D, G, X)
    eps = 1e-6
    L = lambda X_, W1_, W2_, b_: flat_loss(variant, n_in, n_out, D, X_, W1_, W2_, b_, G, ACT_NONE)  # noqa
    for arr, grad, idx in ((X, dX, 0), (W1, dW1, 1), (W2, dW2, 2), (b, db, 3)):
        num = np.zeros_like(arr)
        for pos in np.ndindex(arr.shape):
            args_p = [X.copy(), W1.copy(), W2.copy(), b.copy()]
            args_m = [X.copy(), W1.copy(), W2.copy(), b.copy()]
            args_p[idx][pos] += eps
            args_m[idx][pos] -= eps
            num[pos] = (L(*args_p) - L(*args_m)) / (2 * eps)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-7)


def test_appendix_7x6_example_live_entries():
    """The appendix's 7 x 6 weight with n_dyad 2: one zero row pads it to 8 x 6, blocks 4 x 3.
    Of the 2 * 8 * 6 / 2 = 48 stored entries, the 3 + 3 that sit in the padded row (W1 block 1,
    row 3 and its BlockTrans partner) do not reach the 7 x 6 weight; the other 42 each do."""
    n_in, n_out, D = 6, 7, 2
    for v in ("IT", "OT", "DT"):
        live = 0
        for c in (1, 2):
            for idx in np.ndindex(D, 4, 3):
                W1 = np.zeros((D, 4, 3))
                W2 = np.zeros((D, 4, 3))
                (W1 if c == 1 else W2)[idx] = 1.0
                Wd = oracle.forward(v, n_in, n_out, D, np.eye(n_in), W1, W2).T   # column e = W e
                live += int(np.count_nonzero(Wd) == 1)
                assert np.count_nonzero(Wd) <= 1
        assert live == 42, v
