"""Pins of the oracle to facts other than itself (CPU only).

Each test checks the oracle against something the paper or mathematics fixes:
a hand-derived worked example, closed forms, library routines on special
cases, brute force on tiny inputs, or invariants.  Together they are chosen
so that a dropped term, a wrong sign or index, a transposed operand or a
wrong permutation direction anywhere in the oracle fails at least one.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

HERE = os.path.dirname(os.path.abspath(__file__))


def torch_conv64(x, w, stride, pad):
    """Library convolution in float64 (the textbook definition of Eq. 7 with p = 0)."""
    return F.conv2d(torch.from_numpy(np.asarray(x, np.float64)),
                    torch.from_numpy(np.asarray(w, np.float64)),
                    stride=stride, padding=pad).numpy()


def dense_from_bsr(P, I, D, n, m):
    """Re-assemble the dense masked weight from (P, I, D) with numpy indexing."""
    t, N, h, wd = D.shape
    G = len(P) - 1
    W = np.zeros((G * N, m, h, wd))
    for g in range(G):
        for z in range(P[g], P[g + 1]):
            W[g * N:(g + 1) * N, I[z]] = D[z]
    return W[:n]


# ---------------------------------------------------------------------------
# Worked example with the Fig. 1 shape (8 x 6 x 3 x 3, N = 4), derived by hand.
# ---------------------------------------------------------------------------

def _golden():
    with open(os.path.join(HERE, "golden", "fig1_8x6x3x3_n4.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("mode", ["plain", "rearranged"])
def test_golden_fig1_shape(oracle_lib, mode):
    g = _golden()
    a = np.array(g["a"], np.float64)
    w = a[:, :, None, None] * np.ones((1, 1, 3, 3))
    exp = g[mode]
    pr = oracle_lib.prune(w, g["N"], g["p"], rearrange=(mode == "rearranged"))
    np.testing.assert_array_equal(pr.perm, exp["perm"])
    S = oracle_lib.block_scores(pr.wt, g["N"])
    np.testing.assert_array_equal(S, 9.0 * np.array(exp["scores_div9"], np.float64))
    assert pr.t == exp["t"]
    np.testing.assert_array_equal(pr.T, exp["T"])
    np.testing.assert_array_equal(pr.P, exp["P"])
    np.testing.assert_array_equal(pr.I, exp["I"])
    # D[z][i] = a[perm[4g + i]][I[z]] * ones(3, 3)
    perm = np.array(exp["perm"])
    for gi in range(2):
        for z in range(exp["P"][gi], exp["P"][gi + 1]):
            for i in range(4):
                np.testing.assert_array_equal(pr.D[z, i], a[perm[4 * gi + i], exp["I"][z]] * np.ones((3, 3)))
    # The convolution with the hand-masked weight, by the library routine.
    T = np.array(exp["T"])
    wbar = a[perm][:, :, None, None] * np.ones((1, 1, 3, 3))
    for j in range(8):
        for k in range(6):
            if not T[k, j // 4]:
                wbar[j, k] = 0.0
    np.testing.assert_array_equal(pr.wbar, wbar)
    x = np.arange(2 * 6 * 5 * 5, dtype=np.float64).reshape(2, 6, 5, 5) % 7
    np.testing.assert_array_equal(oracle_lib.conv2d(x, pr.wbar, (1, 1), (1, 1)),
                                  torch_conv64(x, wbar, 1, 1))
    np.testing.assert_array_equal(oracle_lib.decode(x, pr.P, pr.I, pr.D, 8, (1, 1), (1, 1)),
                                  torch_conv64(x, wbar, 1, 1))


# ---------------------------------------------------------------------------
# Eq. 7 with p = 0 is the ordinary convolution (library routine).
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("k,stride,pad,B,cin,cout,H,W", [
    (1, 1, 0, 2, 5, 7, 6, 5),
    (1, 2, 0, 2, 4, 6, 7, 7),
    (3, 1, 1, 1, 6, 8, 9, 8),
    (3, 2, 1, 2, 3, 5, 9, 10),
    (7, 2, 3, 1, 3, 4, 15, 13),
    (3, 1, 0, 1, 2, 3, 5, 6),
])
def test_conv_p0_is_library_conv(oracle_lib, k, stride, pad, B, cin, cout, H, W):
    rng = np.random.default_rng(1)
    w = rng.standard_normal((cout, cin, k, k))
    x = rng.standard_normal((B, cin, H, W))
    pr = oracle_lib.prune(w, 4, 0.0, rearrange=False)
    assert pr.t == cin * -(-cout // 4)
    np.testing.assert_array_equal(pr.wbar, w)
    y = oracle_lib.conv2d(x, pr.wbar, (stride, stride), (pad, pad))
    np.testing.assert_allclose(y, torch_conv64(x, w, stride, pad), rtol=1e-12, atol=1e-12)
    # With rearrangement and p = 0 the output channels are the permuted ones.
    pr2 = oracle_lib.prune(w, 4, 0.0, rearrange=True)
    y2 = oracle_lib.conv2d(x, pr2.wbar, (stride, stride), (pad, pad))
    np.testing.assert_allclose(y2, torch_conv64(x, w, stride, pad)[:, pr2.perm], rtol=1e-12,
                               atol=1e-12)


def test_conv_p1_is_zero(oracle_lib):
    rng = np.random.default_rng(2)
    w = rng.standard_normal((8, 5, 3, 3))
    x = rng.standard_normal((2, 5, 6, 6))
    pr = oracle_lib.prune(w, 4, 1.0, rearrange=True)
    assert pr.t == 0 and pr.T.sum() == 0
    assert np.all(pr.P == 0)
    assert not np.any(oracle_lib.conv2d(x, pr.wbar, (1, 1), (1, 1)))
    assert not np.any(oracle_lib.decode(x, pr.P, pr.I, pr.D, 8, (1, 1), (1, 1)))


def test_conv_at_matches_full(oracle_lib):
    rng = np.random.default_rng(3)
    w = rng.standard_normal((10, 6, 3, 3))
    x = rng.standard_normal((2, 6, 9, 7))
    pr = oracle_lib.prune(w, 4, 0.5, rearrange=True)
    y = oracle_lib.conv2d(x, pr.wbar, (2, 2), (1, 1))
    idx = rng.choice(y.size, 50, replace=False)
    np.testing.assert_array_equal(oracle_lib.conv2d_at(x, pr.wbar, idx, (2, 2), (1, 1)),
                                  y.reshape(-1)[idx])


# ---------------------------------------------------------------------------
# Eq. 8 (block-wise decode over the BSR) equals Eq. 7 (dense masked weight).
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n,m,k,N,p,stride,pad", [
    (16, 9, 1, 4, 0.5, 1, 0),
    (24, 7, 3, 16, 0.3, 1, 1),    # ragged last col-group (24 = 16 + 8)
    (20, 5, 3, 8, 0.7, 2, 1),     # ragged (20 = 8 + 8 + 4), stride 2
    (12, 3, 7, 32, 0.0, 2, 3),    # one ragged col-group, 7x7
    (8, 6, 1, 1, 0.5, 1, 0),
])
def test_decode_equals_dense(oracle_lib, n, m, k, N, p, stride, pad):
    rng = np.random.default_rng(4)
    w = rng.standard_normal((n, m, k, k))
    x = rng.standard_normal((2, m, 11, 10))
    pr = oracle_lib.prune(w, N, p, rearrange=True)
    yd = oracle_lib.conv2d(x, pr.wbar, (stride, stride), (pad, pad))
    ye = oracle_lib.decode(x, pr.P, pr.I, pr.D, n, (stride, stride), (pad, pad))
    np.testing.assert_allclose(ye, yd, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(yd, torch_conv64(x, pr.wbar, stride, pad), rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# Sec. 3.3: permuting this layer's outputs and the next layer's inputs by the
# same perm leaves the two-layer composite unchanged.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("p", [0.0, 0.5])
def test_composite_permutation_invariance(oracle_lib, p):
    gen = torch.Generator().manual_seed(5)
    w1 = torch.randint(-3, 4, (12, 5, 3, 3), generator=gen).double().numpy()
    w2 = torch.randint(-3, 4, (7, 12, 1, 1), generator=gen).double().numpy()
    x = torch.randint(0, 4, (2, 5, 8, 8), generator=gen).double().numpy()
    pr = oracle_lib.prune(w1, 4, p, rearrange=True)
    assert sorted(pr.perm.tolist()) == list(range(12))
    assert len(set(pr.perm.tolist())) == 12 and not np.array_equal(pr.perm, np.arange(12))
    # Rearranged network: layer 1 uses Omega-bar (rearranged order), layer 2 its
    # input channels permuted the same way.
    h1 = np.maximum(oracle_lib.conv2d(x, pr.wbar, (1, 1), (1, 1)), 0.0)
    y_re = oracle_lib.conv2d(h1, w2[:, pr.perm], (1, 1), (0, 0))
    # Original order: filter perm[j'] of layer 1 is Omega-bar's filter j'.
    w1_orig = np.empty_like(pr.wbar)
    w1_orig[pr.perm] = pr.wbar
    h1o = np.maximum(torch_conv64(x, w1_orig, 1, 1), 0.0)
    y_orig = torch_conv64(h1o, w2, 1, 0)
    np.testing.assert_array_equal(y_re, y_orig)
    if p == 0.0:
        np.testing.assert_array_equal(w1_orig, w1)


# ---------------------------------------------------------------------------
# The epilogue after a convolution: folded batch norm (or bias) and ReLU/ReLU6.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("act", ["none", "relu", "relu6"])
def test_epilogue_equals_torch_batch_norm_and_activation(oracle_lib, act):
    """Inference batch norm (torch's routine, fp64) folds into scale = gamma /
    sqrt(var + eps) and bias = beta - mean * scale; the oracle's per-channel
    affine map plus activation must give torch's batch_norm + relu/relu6."""
    gen = torch.Generator().manual_seed(21)
    y = torch.randn((3, 7, 5, 4), generator=gen, dtype=torch.float64) * 4
    gamma = torch.randn(7, generator=gen, dtype=torch.float64)
    beta = torch.randn(7, generator=gen, dtype=torch.float64)
    mean = torch.randn(7, generator=gen, dtype=torch.float64)
    var = torch.rand(7, generator=gen, dtype=torch.float64) + 0.5
    eps = 1e-5
    ref = torch.nn.functional.batch_norm(y, mean, var, gamma, beta, False, 0.0, eps)
    ref = {"none": ref, "relu": torch.relu(ref), "relu6": torch.nn.functional.relu6(ref)}[act]
    scale = gamma / torch.sqrt(var + eps)
    bias = beta - mean * scale
    got = oracle_lib.epilogue(y.numpy(), scale.numpy(), bias.numpy(), act)
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-13, atol=1e-13)
    # Either parameter absent: scale 1 / bias 0.
    np.testing.assert_array_equal(oracle_lib.epilogue(y.numpy(), None, bias.numpy()),
                                  (y + bias[None, :, None, None]).numpy())
    np.testing.assert_array_equal(oracle_lib.epilogue(y.numpy(), scale.numpy(), None),
                                  (y * scale[None, :, None, None]).numpy())
    np.testing.assert_array_equal(oracle_lib.epilogue(y.numpy()), y.numpy())


def test_composite_with_epilogue_permutation_invariance(oracle_lib):
    """Sec. 3.3: with layer 1's filters rearranged, its per-channel scale and
    bias taken in the same order and layer 2's input channels permuted, the
    two-layer network (conv -> folded BN -> ReLU6 -> pruned conv) is unchanged."""
    gen = torch.Generator().manual_seed(8)
    w1 = torch.randint(-3, 4, (16, 6, 3, 3), generator=gen).double().numpy()
    w2 = torch.randint(-2, 3, (12, 16, 1, 1), generator=gen).double().numpy()
    x = torch.randint(0, 4, (2, 6, 7, 9), generator=gen).double().numpy()
    scale = torch.randint(-2, 3, (16,), generator=gen).double().numpy()
    bias = torch.randint(-9, 10, (16,), generator=gen).double().numpy()
    pr1 = oracle_lib.prune(w1, 4, 0.5, rearrange=True)
    assert not np.array_equal(pr1.perm, np.arange(16))
    pr2 = oracle_lib.prune(w2[:, pr1.perm], 4, 0.5, rearrange=False)
    h = oracle_lib.epilogue(oracle_lib.conv2d(x, pr1.wbar, (1, 1), (1, 1)), scale[pr1.perm],
                            bias[pr1.perm], "relu6")
    y_re = oracle_lib.conv2d(h, pr2.wbar, (1, 1), (0, 0))
    # The same network in the original channel order, through torch's conv.
    w1o = np.empty_like(pr1.wbar)
    w1o[pr1.perm] = pr1.wbar
    w2o = np.empty_like(pr2.wbar)
    w2o[:, pr1.perm] = pr2.wbar
    ho = torch_conv64(x, w1o, 1, 1) * scale[None, :, None, None] + bias[None, :, None, None]
    ho = np.clip(ho, 0.0, 6.0)
    np.testing.assert_array_equal(y_re, torch_conv64(ho, w2o, 1, 0))


# ---------------------------------------------------------------------------
# Closed forms for the l1 scores and the rearrangement.
# ---------------------------------------------------------------------------

def test_filter_perm_closed_form(oracle_lib):
    c = np.array([0.5, 3.0, -2.0, 3.0, 1.0, 0.0, 2.0])
    w = c[:, None, None, None] * np.ones((7, 4, 3, 3))
    # norm_j = 36 |c_j|: 3.0 (j1), 3.0 (j3), -2 and 2 (j2, j6), 1.0, 0.5, 0.0
    np.testing.assert_array_equal(oracle_lib.filter_norms(w), 36 * np.abs(c))
    np.testing.assert_array_equal(oracle_lib.filter_perm(w, True), [1, 3, 2, 6, 4, 0, 5])
    np.testing.assert_array_equal(oracle_lib.filter_perm(w, False), np.arange(7))
    # All-equal filters: a stable sort leaves the order alone.
    np.testing.assert_array_equal(oracle_lib.filter_perm(np.ones((9, 2, 1, 1)), True), np.arange(9))


@pytest.mark.parametrize("n,N", [(16, 4), (20, 8), (5, 4), (6, 16), (7, 1)])
def test_block_scores_closed_form(oracle_lib, n, N):
    rng = np.random.default_rng(6)
    m, kh, kw = 5, 3, 2
    a = rng.integers(-9, 10, size=(n, m)).astype(np.float64)
    wt = a[:, :, None, None] * np.ones((1, 1, kh, kw))
    G = -(-n // N)
    expect = np.zeros((m, G))
    for k in range(m):
        for g in range(G):
            expect[k, g] = kh * kw * np.abs(a[g * N:min(n, (g + 1) * N), k]).sum()
    np.testing.assert_array_equal(oracle_lib.block_scores(wt, N), expect)


# ---------------------------------------------------------------------------
# Selection: Eq. 1 count, the argmax of Eq. 5, tie rule, special cases.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("K,p,t", [
    (1024, 0.5, 512), (8192, 0.5, 4096), (384, 0.3, 269), (131072, 0.7, 39322),
    (10, 0.0, 10), (10, 1.0, 0), (4, 0.625, 1), (4, 0.375, 2), (0, 0.5, 0), (7, 0.5, 3),
])
def test_kept_count(oracle_lib, K, p, t):
    assert oracle_lib.kept_count(K, p) == t


@pytest.mark.parametrize("seed", range(6))
def test_selection_is_argmax_brute_force(oracle_lib, seed):
    rng = np.random.default_rng(100 + seed)
    m, n, N = [(3, 8, 2), (2, 12, 4), (4, 6, 2), (3, 10, 3), (2, 9, 4), (5, 3, 1)][seed]
    w = rng.standard_normal((n, m, 2, 2))
    p = [0.5, 0.3, 0.7, 0.5, 0.4, 0.6][seed]
    pr = oracle_lib.prune(w, N, p, rearrange=bool(seed % 2))
    S = oracle_lib.block_scores(pr.wt, N).reshape(-1)
    K = S.size
    assert K <= 16
    t = K - int(np.floor(p * K + 0.5))
    assert pr.t == t
    best, arg = -1.0, None
    for comb in itertools.combinations(range(K), t):
        v = S[list(comb)].sum()
        if v > best:
            best, arg = v, comb
    T = np.zeros(K, np.uint8)
    T[list(arg)] = 1
    np.testing.assert_array_equal(pr.T.reshape(-1), T)


def test_selection_invariants(oracle_lib):
    rng = np.random.default_rng(7)
    w = rng.standard_normal((48, 40, 3, 3))
    for N, p in [(4, 0.5), (16, 0.3), (8, 0.7), (32, 0.5)]:
        pr = oracle_lib.prune(w, N, p, rearrange=True)
        S = oracle_lib.block_scores(pr.wt, N)
        assert pr.T.sum() == pr.t == oracle_lib.kept_count(S.size, p)
        kept, pruned = S[pr.T == 1], S[pr.T == 0]
        assert kept.min() >= pruned.max()


def test_tie_rule_all_equal(oracle_lib):
    w = np.ones((8, 6, 3, 3))
    pr = oracle_lib.prune(w, 4, 0.5, rearrange=True)
    np.testing.assert_array_equal(pr.perm, np.arange(8))
    flat = pr.T.reshape(-1)
    np.testing.assert_array_equal(flat, [1] * 6 + [0] * 6)


def test_n1_is_weight_pruning(oracle_lib):
    """N = 1 with 1x1 kernels is element-wise magnitude pruning (Sec. 3.2)."""
    rng = np.random.default_rng(8)
    n, m, p = 9, 7, 0.4
    w = rng.standard_normal((n, m, 1, 1))
    pr = oracle_lib.prune(w, 1, p, rearrange=False)
    t = n * m - int(np.floor(p * n * m + 0.5))
    mag = np.abs(w[:, :, 0, 0]).T.reshape(-1)       # row-major by input channel k
    keep = np.argsort(-mag, kind="stable")[:t]
    T = np.zeros(n * m, np.uint8)
    T[keep] = 1
    np.testing.assert_array_equal(pr.T.reshape(-1), T)
    np.testing.assert_array_equal(pr.wbar[:, :, 0, 0] != 0, T.reshape(m, n).T.astype(bool))


def test_n_equals_n_is_row_pruning(oracle_lib):
    """N = n: a block is a whole row of Omega, i.e. one input channel of every filter."""
    rng = np.random.default_rng(9)
    n, m, p = 6, 10, 0.3
    w = rng.standard_normal((n, m, 3, 3))
    pr = oracle_lib.prune(w, n, p, rearrange=False)
    row = np.abs(w).sum(axis=(0, 2, 3))
    t = m - int(np.floor(p * m + 0.5))
    keep = np.sort(np.argsort(-row, kind="stable")[:t])
    np.testing.assert_array_equal(np.nonzero(pr.T[:, 0])[0], keep)
    np.testing.assert_array_equal(pr.I, keep)
    assert np.all(pr.wbar[:, np.setdiff1d(np.arange(m), keep)] == 0)


# ---------------------------------------------------------------------------
# BSR invariants (Sec. 3.4).
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n,m,k,N,p", [(32, 20, 1, 16, 0.5), (24, 9, 3, 16, 0.3),
                                       (20, 11, 3, 8, 0.7), (10, 4, 7, 4, 0.5),
                                       (8, 6, 1, 32, 0.2)])
def test_pack_invariants(oracle_lib, n, m, k, N, p):
    rng = np.random.default_rng(10)
    w = rng.standard_normal((n, m, k, k))
    pr = oracle_lib.prune(w, N, p, rearrange=True)
    G = -(-n // N)
    assert pr.P[0] == 0 and pr.P[-1] == pr.t and len(pr.P) == G + 1
    assert np.all(np.diff(pr.P) >= 0)
    assert len(pr.I) == pr.t and pr.D.shape == (pr.t, N, k, k)
    for g in range(G):
        seg = pr.I[pr.P[g]:pr.P[g + 1]]
        assert np.all(np.diff(seg) > 0)
        np.testing.assert_array_equal(seg, np.nonzero(pr.T[:, g])[0])
    np.testing.assert_array_equal(dense_from_bsr(pr.P, pr.I, pr.D, n, m), pr.wbar)
    if n % N:
        assert not np.any(pr.D[pr.P[G - 1]:, n % N:])


# ---------------------------------------------------------------------------
# Backward of Eq. 7 (fine-tuning with the 1xN pattern fixed).
# ---------------------------------------------------------------------------

BWD_SHAPES = [  # (n, m, k, stride, pad, B, H, W, N)
    (12, 5, 1, 1, 0, 2, 6, 5, 4),
    (10, 7, 3, 1, 1, 2, 7, 6, 4),      # ragged last col-group
    (16, 3, 3, 2, 1, 1, 9, 8, 8),
    (8, 3, 7, 2, 3, 1, 11, 10, 4),
    (9, 6, 1, 2, 0, 2, 7, 7, 2),
]


@pytest.mark.parametrize("shape", BWD_SHAPES, ids=lambda s: "n%d_m%d_k%d_s%d_p%d" % s[:5])
def test_bwd_equals_torch_conv_gradients(oracle_lib, shape):
    """dX equals torch's conv2d_input with the masked weight; dW equals torch's
    conv2d_weight times the 1xN mask (fp64 library routines)."""
    n, m, k, s, pd, B, H, W, N = shape
    rng = np.random.default_rng(n * m + k)
    w = rng.standard_normal((n, m, k, k))
    x = rng.standard_normal((B, m, H, W))
    pr = oracle_lib.prune(w, N, 0.5, True)
    Ho, Wo = (H + 2 * pd - k) // s + 1, (W + 2 * pd - k) // s + 1
    dy = rng.standard_normal((B, n, Ho, Wo))
    dx = oracle_lib.conv2d_bwd_data(dy, pr.wbar, (H, W), (s, s), (pd, pd))
    ref_dx = torch.nn.grad.conv2d_input((B, m, H, W), torch.from_numpy(pr.wbar), torch.from_numpy(dy),
                                        stride=s, padding=pd)
    np.testing.assert_allclose(dx, ref_dx.numpy(), rtol=1e-12, atol=1e-12)
    dw = oracle_lib.conv2d_bwd_weight(x, dy, pr.T, N, (k, k), (s, s), (pd, pd))
    ref_dw = torch.nn.grad.conv2d_weight(torch.from_numpy(x), (n, m, k, k), torch.from_numpy(dy),
                                         stride=s, padding=pd).numpy()
    keep = np.repeat(pr.T.T, N, axis=0)[:n][:, :, None, None]     # [n][m] kept-block mask
    np.testing.assert_allclose(dw, ref_dw * keep, rtol=1e-12, atol=1e-12)
    assert np.all(dw[keep[:, :, 0, 0] == 0] == 0)


@pytest.mark.parametrize("shape", BWD_SHAPES, ids=lambda s: "n%d_m%d_k%d_s%d_p%d" % s[:5])
def test_bwd_adjoint_identities(oracle_lib, shape):
    """Eq. 7 is bilinear in (X, Wbar), so with integer data, exactly:
    <conv(X, Wbar), dY> = <X, dX>  and  <conv(X, V), dY> = <dW, V> for any V
    with the same 1xN mask (no library routine involved)."""
    n, m, k, s, pd, B, H, W, N = shape
    rng = np.random.default_rng(7 * n + m)
    w = rng.integers(-3, 4, (n, m, k, k)).astype(np.float64)
    x = rng.integers(-2, 3, (B, m, H, W)).astype(np.float64)
    pr = oracle_lib.prune(w, N, 0.5, True)
    y = oracle_lib.conv2d(x, pr.wbar, (s, s), (pd, pd))
    dy = rng.integers(-2, 3, y.shape).astype(np.float64)
    dx = oracle_lib.conv2d_bwd_data(dy, pr.wbar, (H, W), (s, s), (pd, pd))
    assert np.sum(y * dy) == np.sum(x * dx)
    v = oracle_lib.masked_weight(rng.integers(-3, 4, (n, m, k, k)).astype(np.float64), pr.T, N)
    dw = oracle_lib.conv2d_bwd_weight(x, dy, pr.T, N, (k, k), (s, s), (pd, pd))
    assert np.sum(oracle_lib.conv2d(x, v, (s, s), (pd, pd)) * dy) == np.sum(dw * v)


def test_bwd_with_everything_pruned_is_zero(oracle_lib):
    rng = np.random.default_rng(3)
    w = rng.standard_normal((8, 4, 3, 3))
    x = rng.standard_normal((1, 4, 5, 5))
    pr = oracle_lib.prune(w, 4, 1.0, False)
    dy = rng.standard_normal((1, 8, 5, 5))
    assert np.all(oracle_lib.conv2d_bwd_data(dy, pr.wbar, (5, 5), (1, 1), (1, 1)) == 0)
    assert np.all(oracle_lib.conv2d_bwd_weight(x, dy, pr.T, 4, (3, 3), (1, 1), (1, 1)) == 0)
