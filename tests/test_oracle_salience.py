"""Pins for the oracle's salience (Sec. 3.1 attention, Sec. 3.2 Eq. (4)) and pooling."""
import math
from fractions import Fraction

import numpy as np
import pytest

from golden_io import fracs, read_blocks


def brute_salience(K, Qw, H):
    """Independent NumPy implementation: full causal score matrix, row softmax, average."""
    n, G, d = K.shape
    w = Qw.shape[0]
    N = n - w
    acc = np.zeros(n)
    for h in range(H):
        g = (h * G) // H                      # consecutive GQA grouping
        logits = Qw[:, h, :].astype(np.float64) @ K[:, g, :].astype(np.float64).T / math.sqrt(d)
        pos = np.arange(n)[None, :]
        qpos = (n - w + np.arange(w))[:, None]
        logits = np.where(pos <= qpos, logits, -np.inf)
        logits -= logits.max(axis=1, keepdims=True)
        p = np.exp(logits)
        p /= p.sum(axis=1, keepdims=True)
        acc += p.sum(axis=0)
    return acc[:N] / (w * H)


@pytest.mark.parametrize("n,G,H,w,seed", [(64, 2, 4, 8, 0), (40, 1, 3, 5, 1), (97, 4, 8, 16, 2)])
def test_salience_matches_brute_force(oracle_lib, n, G, H, w, seed):
    rng = np.random.default_rng(seed)
    d = 16
    K = rng.standard_normal((n, G, d)).astype(np.float32) * 2
    Qw = rng.standard_normal((w, H, d)).astype(np.float32) * 2
    s = oracle_lib.salience(K, Qw, H)
    np.testing.assert_allclose(s, brute_salience(K, Qw, H), rtol=1e-12, atol=1e-15)


def test_salience_tiny_config_matches_brute_force(oracle_lib):
    from workloads import CONFIGS, make_layer
    li = make_layer(CONFIGS["tiny"], with_basis=False)
    s = oracle_lib.salience(li.K, li.Qw, 2)
    np.testing.assert_allclose(s, brute_salience(li.K, li.Qw, 2), rtol=1e-11, atol=1e-18)


def test_salience_zero_query_closed_form(oracle_lib):
    """q = 0 makes attention uniform over the visible prefix: query i at position n-w+i
    gives every visible key weight 1/(n-w+i+1), so s_t = (1/w) sum_i 1/(n-w+i+1)."""
    n, G, H, w, d = 50, 2, 4, 6, 8
    K = np.random.default_rng(3).standard_normal((n, G, d)).astype(np.float32)
    Qw = np.zeros((w, H, d), np.float32)
    s = oracle_lib.salience(K, Qw, H)
    expect = sum(1.0 / (n - w + i + 1) for i in range(w)) / w
    np.testing.assert_allclose(s, np.full(n - w, expect), rtol=1e-14)


def test_salience_two_key_logistic(oracle_lib):
    """n = 2, w = 1: the single window query sits at position 1 and sees keys 0 and 1, so
    s_0 = sigmoid(x_0 - x_1) with x_t = <q, k_t> / sqrt(d)."""
    d = 4
    K = np.array([[[1.0, 0.5, 0.0, 2.0]], [[0.0, -1.0, 1.0, 0.5]]], np.float32)
    Qw = np.array([[[0.3, -0.2, 0.7, 1.1]]], np.float32)
    s = oracle_lib.salience(K, Qw, 1)
    x0 = float(np.dot(Qw[0, 0].astype(np.float64), K[0, 0])) / 2.0
    x1 = float(np.dot(Qw[0, 0].astype(np.float64), K[1, 0])) / 2.0
    assert s.shape == (1,)
    assert s[0] == pytest.approx(1.0 / (1.0 + math.exp(x1 - x0)), rel=1e-14)


def test_salience_equivariant_under_coded_permutation(oracle_lib):
    """Every coded token is visible to every window query, so permuting coded keys
    permutes s (a position-dependent indexing mistake would break this)."""
    rng = np.random.default_rng(4)
    n, G, H, w, d = 60, 2, 4, 7, 8
    K = rng.standard_normal((n, G, d)).astype(np.float32)
    Qw = rng.standard_normal((w, H, d)).astype(np.float32)
    perm = rng.permutation(n - w)
    K2 = K.copy()
    K2[: n - w] = K[perm]
    s1 = oracle_lib.salience(K, Qw, H)
    s2 = oracle_lib.salience(K2, Qw, H)
    np.testing.assert_allclose(s2, s1[perm], rtol=1e-12)


def test_salience_gqa_grouping(oracle_lib):
    """Heads 0..H/G-1 read KV head 0.  Make KV head 1 carry a needle that only head
    group 1 can see: s must equal the average of the two groups' separate attention."""
    n, w, d = 20, 2, 4
    K = np.zeros((n, 2, d), np.float32)
    K[5, 1, 0] = 8.0                      # needle in KV head 1 only
    Qw = np.zeros((w, 4, d), np.float32)
    Qw[:, 2:, 0] = 4.0                    # heads 2,3 (group 1) look along channel 0
    s = oracle_lib.salience(K, Qw, 4)
    # group 0 heads: uniform over the prefix; group 1 heads: needle has logit 16
    expect = np.zeros(n - w)
    for i in range(w):
        p = n - w + i
        uni = np.full(p + 1, 1.0 / (p + 1))
        x = np.zeros(p + 1)
        x[5] = 16.0
        e = np.exp(x - x.max())
        e /= e.sum()
        expect += 2 * uni[: n - w] + 2 * e[: n - w]
    expect /= w * 4
    np.testing.assert_allclose(s, expect, rtol=1e-13)


def test_pool_handworked(oracle_lib):
    blk = read_blocks("pool_handworked.txt")[0]
    s = np.array([float(x) for x in blk["s"]])
    want = np.array([float(x) for x in fracs(blk["sbar"])], np.float32)
    got = oracle_lib.pool(s)
    assert got.dtype == np.float32
    np.testing.assert_array_equal(got, want)


def test_pool_constant_edges(oracle_lib):
    """Constant input: interior keeps the constant, the first/last two tokens see 3/5, 4/5
    of it (zero padding, always divided by 5)."""
    c = 0.125
    got = oracle_lib.pool(np.full(9, c))
    want = np.array([3, 4, 5, 5, 5, 5, 5, 4, 3], np.float64) * c / 5
    np.testing.assert_array_equal(got, want.astype(np.float32))


def test_pool_short_inputs(oracle_lib):
    got = oracle_lib.pool(np.array([1.0, 2.0]))
    np.testing.assert_array_equal(got, np.array([0.6, 0.6], np.float32))
    got = oracle_lib.pool(np.array([5.0]))
    np.testing.assert_array_equal(got, np.array([1.0], np.float32))


def test_weights_min_max_integerisation(oracle_lib):
    sb = np.array([0.25, 0.75, 0.5, 0.25, 1.25], np.float32)
    u = oracle_lib.weights(sb)
    assert list(u) == [1, 8388609, 4194305, 1, 16777217]


def test_weights_constant_signal_is_uniform(oracle_lib):
    u = oracle_lib.weights(np.full(7, 0.3, np.float32))
    assert len(set(u.tolist())) == 1 and u[0] >= 1


def test_weights_monotone_and_bounded(oracle_lib):
    rng = np.random.default_rng(5)
    sb = rng.random(1000).astype(np.float32) ** 3
    u = oracle_lib.weights(sb)
    assert u.min() == 1 and u.max() == (1 << 24) + 1
    order = np.argsort(sb, kind="stable")
    assert np.all(np.diff(u[order].astype(np.int64)) >= 0)
    # exact: u = 1 + floor(2^24 (s - min)/(max - min)) evaluated with exact rationals,
    # allowing the single fp64 rounding of the quotient to move an integer boundary
    mn, mx = Fraction(float(sb.min())), Fraction(float(sb.max()))
    for t in range(0, 1000, 37):
        exact = 1 + math.floor((Fraction(float(sb[t])) - mn) / (mx - mn) * (1 << 24))
        assert abs(int(u[t]) - exact) <= 1
