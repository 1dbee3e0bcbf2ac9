"""Pins of the fp64 direct conv / matmul oracle (CPU only).

The oracle is the plain definition of a conv / FC layer on masked weights
(Sec. 4.2: layer weights W_i and bias b_i; pruning zeroes weights).  It is
checked against a pure-Python brute force, against library routines at rate 1
(torch conv2d and numpy matmul in fp64), against hand-worked examples and
against properties of convolution (linearity, zero input, shift equivariance,
1x1 conv = matmul, whole-matrix row pruning leaves only the bias).
"""

import json
import os

import numpy as np
import pytest
import torch

from oracle import brute
from oracle import prune as P

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


def test_golden_conv_examples(oracle_direct):
    g = GOLD["conv_plus_3x3"]
    x = np.array(g["x"], dtype=np.float64).reshape(1, 1, 3, 3)
    w = np.array(g["w"], dtype=np.float64).reshape(1, 1, 3, 3)
    assert oracle_direct.conv2d(x, w, None, (1, 1), (1, 1))[0, 0].tolist() == g["y_stride1_pad1"]
    assert oracle_direct.conv2d(x, w, None, (2, 2), (1, 1))[0, 0].tolist() == g["y_stride2_pad1"]
    m = np.array(g["col_whole_rate3"]["mask"], dtype=np.float64).reshape(1, 1, 3, 3)
    assert oracle_direct.conv2d(x, w * m, None, (1, 1), (1, 1))[0, 0].tolist() == \
        g["col_whole_rate3"]["y_stride1_pad1"]


def test_golden_linear_example(oracle_direct):
    g = GOLD["matrix_4x8"]
    ex = g["col_2x4_rate2"]
    W = np.array(g["W"], dtype=np.float64) * np.array(ex["mask"], dtype=np.float64)
    x = np.array(ex["x_feature_major"], dtype=np.float64)
    assert oracle_direct.linear(x, W).tolist() == ex["y"]


def _rand(rng, shape):
    return rng.standard_normal(shape)


@pytest.mark.parametrize("trial", range(12))
def test_matches_python_brute_force(oracle_direct, trial):
    rng = np.random.default_rng(100 + trial)
    N, C, O = int(rng.integers(1, 3)), int(rng.integers(1, 6)), int(rng.integers(1, 5))
    H, W = int(rng.integers(1, 7)), int(rng.integers(1, 7))
    k = int(rng.choice([1, 3]))
    s = int(rng.integers(1, 3))
    p = int(rng.integers(0, 2))
    if H + 2 * p < k or W + 2 * p < k:
        p = k
    x, w, b = _rand(rng, (N, C, H, W)), _rand(rng, (O, C, k, k)), _rand(rng, (O,))
    relu = bool(trial % 2)
    y = oracle_direct.conv2d(x, w, b, (s, s), (p, p), relu=relu)
    yb = np.array(brute.conv2d(x.tolist(), w.tolist(), b.tolist(), (s, s), (p, p), relu=relu))
    assert y.shape == yb.shape
    np.testing.assert_allclose(y, yb, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("trial", range(6))
def test_linear_matches_python_brute_force(oracle_direct, trial):
    rng = np.random.default_rng(200 + trial)
    K, B, O = int(rng.integers(1, 20)), int(rng.integers(1, 6)), int(rng.integers(1, 9))
    x, w, b = _rand(rng, (K, B)), _rand(rng, (O, K)), _rand(rng, (O,))
    y = oracle_direct.linear(x, w, b, relu=bool(trial % 2))
    yb = np.array(brute.linear(x.tolist(), w.tolist(), b.tolist(), relu=bool(trial % 2)))
    np.testing.assert_allclose(y, yb, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("N,C,H,W,O,k,s,p", [
    (2, 16, 12, 12, 24, 3, 1, 1), (2, 8, 13, 11, 8, 3, 2, 1), (1, 3, 23, 23, 16, 7, 2, 3),
    (3, 32, 7, 7, 40, 1, 1, 0), (2, 16, 14, 14, 32, 1, 2, 0), (1, 4, 5, 9, 6, 5, 1, 2)])
def test_rate_one_equals_library_conv(oracle_direct, N, C, H, W, O, k, s, p):
    rng = np.random.default_rng(N * 1000 + C * 10 + k)
    x, w, b = _rand(rng, (N, C, H, W)), _rand(rng, (O, C, k, k)), _rand(rng, (O,))
    m = P.prune_mask(P.gemm_form(w), 16, 16, P.COL, 1).reshape(w.shape)
    assert m.all()
    y = oracle_direct.conv2d(x, w * m, b, (s, s), (p, p))
    ref = torch.nn.functional.conv2d(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b),
                                     stride=s, padding=p).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-11)


def test_1x1_conv_is_matmul(oracle_direct):
    rng = np.random.default_rng(9)
    x, w = _rand(rng, (3, 24, 5, 6)), _rand(rng, (10, 24, 1, 1))
    y = oracle_direct.conv2d(x, w, None, (1, 1), (0, 0))
    ref = np.matmul(w[:, :, 0, 0], x.reshape(3, 24, 30)).reshape(3, 10, 5, 6)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)
    # the linear entry point is the same product on feature-major data
    xf = x.transpose(1, 0, 2, 3).reshape(24, -1)
    yl = oracle_direct.linear(xf, w[:, :, 0, 0])
    np.testing.assert_allclose(yl, y.transpose(1, 0, 2, 3).reshape(10, -1), rtol=1e-12, atol=1e-12)


def test_linearity_in_weights_and_inputs(oracle_direct):
    rng = np.random.default_rng(12)
    x1, x2 = _rand(rng, (2, 6, 9, 9)), _rand(rng, (2, 6, 9, 9))
    w1, w2 = _rand(rng, (5, 6, 3, 3)), _rand(rng, (5, 6, 3, 3))
    f = lambda x, w: oracle_direct.conv2d(x, w, None, (1, 1), (1, 1))
    np.testing.assert_allclose(f(x1 + 2 * x2, w1), f(x1, w1) + 2 * f(x2, w1), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(f(x1, w1 - 3 * w2), f(x1, w1) - 3 * f(x1, w2), rtol=1e-10, atol=1e-10)


def test_zero_input_gives_bias(oracle_direct):
    rng = np.random.default_rng(13)
    w, b = _rand(rng, (7, 4, 3, 3)), _rand(rng, (7,))
    y = oracle_direct.conv2d(np.zeros((2, 4, 6, 6)), w, b, (1, 1), (1, 1))
    assert np.array_equal(y, np.broadcast_to(b[None, :, None, None], y.shape))
    yr = oracle_direct.conv2d(np.zeros((2, 4, 6, 6)), w, b, (1, 1), (1, 1), relu=True)
    assert np.array_equal(yr, np.maximum(y, 0))


def test_shift_equivariance_away_from_borders(oracle_direct):
    rng = np.random.default_rng(14)
    x = _rand(rng, (1, 3, 12, 12))
    w = _rand(rng, (4, 3, 3, 3))
    xs = np.zeros_like(x)
    xs[:, :, 2:, 1:] = x[:, :, :-2, :-1]
    y = oracle_direct.conv2d(x, w, None, (1, 1), (0, 0))
    ys = oracle_direct.conv2d(xs, w, None, (1, 1), (0, 0))
    np.testing.assert_allclose(ys[:, :, 2:, 1:], y[:, :, :-2, :-1], rtol=1e-12, atol=1e-12)


def test_whole_matrix_row_pruning_leaves_bias_on_pruned_filters(oracle_direct):
    rng = np.random.default_rng(15)
    x, w, b = _rand(rng, (2, 8, 7, 7)), _rand(rng, (12, 8, 3, 3)), _rand(rng, (12,))
    m = P.prune_mask(P.gemm_form(w), 0, 0, P.ROW, 4).reshape(w.shape)
    pruned = np.nonzero(m.reshape(12, -1)[:, 0] == 0)[0]
    assert len(pruned) == 9
    y = oracle_direct.conv2d(x, w * m, b, (1, 1), (1, 1))
    for o in pruned:
        assert np.all(y[:, o] == b[o])


# ------------------------------------------------------------- maxpool glue ---
def _f(v):
    return float(v) if not isinstance(v, str) else float(v.replace("inf", "inf"))


def _maxpool_brute(x):
    """2x2 / stride 2 / floor max pooling by plain loops; NaN propagates."""
    N, C, H, W = x.shape
    out = np.empty((N, C, H // 2, W // 2))
    for n in range(N):
        for c in range(C):
            for i in range(H // 2):
                for j in range(W // 2):
                    vals = [float(x[n, c, 2 * i + a, 2 * j + b]) for a in (0, 1) for b in (0, 1)]
                    out[n, c, i, j] = float("nan") if any(v != v for v in vals) else max(vals)
    return out


def test_maxpool_golden_example():
    from oracle import glue
    g = GOLD["maxpool_2x2"]
    x = np.vectorize(_f)(np.array(g["x"], dtype=object)).astype(np.float64)
    want = np.vectorize(_f)(np.array(g["y"], dtype=object)).astype(np.float64)
    got = glue.maxpool2x2(x)
    assert got.shape == want.shape == (1, 2, 2, 2)
    assert np.array_equal(got, want, equal_nan=True)


@pytest.mark.parametrize("shape", [(2, 3, 4, 4), (1, 2, 5, 7), (3, 1, 9, 2), (1, 1, 1, 6)])
def test_maxpool_matches_brute_force_with_nonfinite_values(shape):
    from oracle import glue
    rng = np.random.default_rng(sum(shape))
    x = rng.integers(-3, 4, size=shape).astype(np.float64)       # many ties
    flat = x.reshape(-1)
    idx = rng.permutation(flat.size)
    flat[idx[: max(1, flat.size // 10)]] = -np.inf
    flat[idx[max(1, flat.size // 10): max(2, flat.size // 7)]] = np.nan
    assert np.array_equal(glue.maxpool2x2(x), _maxpool_brute(x), equal_nan=True)
