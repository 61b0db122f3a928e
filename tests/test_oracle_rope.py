"""Pins for the oracle's rotary-key path (Sec. 3.1 "Joint per-token vector"; Algorithm 1,
first step: keys un-rotated to pre-RoPE before coding; last step: the reconstruction
re-rotated to post-RoPE).  The rotation is the rotate-half form of rotary position
embedding: pair i = coordinates (i, i + d/2), turned by position * theta_i."""
import math

import numpy as np
import pytest


def brute_attention(K, V, q, H):
    T, G, d = K.shape
    out = np.zeros((H, d))
    for h in range(H):
        g = (h * G) // H
        x = K[:, g, :].astype(np.float64) @ q[h].astype(np.float64) / math.sqrt(d)
        a = np.exp(x - x.max())
        a /= a.sum()
        out[h] = a @ V[:, g, :].astype(np.float64)
    return out


def _x(seed, n=5, G=2, d=128):
    return np.random.default_rng(seed).standard_normal((n, G, d)).astype(np.float32)


def test_quarter_and_half_turns_are_rotate_half(oracle_lib):
    """Textbook form: RoPE(x) = x cos + rotate_half(x) sin with rotate_half(x) =
    [-x_{d/2:}, x_{:d/2}].  A quarter turn is rotate_half itself, a half turn is -x."""
    X = _x(1)
    theta = np.full(64, np.pi / 2, np.float32)
    rh = np.concatenate([-X[..., 64:], X[..., :64]], axis=-1)
    np.testing.assert_allclose(oracle_lib.rope(X, 1, theta), rh, atol=1e-6)
    np.testing.assert_allclose(oracle_lib.rope(X, 2, theta), -X, atol=1e-6)
    np.testing.assert_array_equal(oracle_lib.rope(X, 0, theta), X.astype(np.float64))


def test_matches_complex_multiplication(oracle_lib):
    """Pair i as the complex number x_i + i x_{i+d/2}, multiplied by exp(i p theta_i)."""
    from workloads import rope_theta
    X = _x(2, n=7)
    theta = rope_theta("llama3")
    pos = np.array([0, 1, 17, 255, 4096, 32767, 131071])
    Y = oracle_lib.rope(X, pos, theta)
    z = X[..., :64].astype(np.float64) + 1j * X[..., 64:].astype(np.float64)
    z = z * np.exp(1j * pos[:, None, None] * theta.astype(np.float64)[None, None, :])
    np.testing.assert_allclose(Y[..., :64], z.real, atol=1e-9)
    np.testing.assert_allclose(Y[..., 64:], z.imag, atol=1e-9)


def test_inverse_norm_and_relative_position(oracle_lib):
    """Rotations: the sign -1 undoes +1, norms are kept, and the score between a query at s
    and a key at t depends on t - s only."""
    from workloads import rope_theta
    theta = rope_theta("llama3")
    X = _x(3, n=4)
    pos = np.array([3, 100, 9000, 70000])
    Y = oracle_lib.rope(X, pos, theta).astype(np.float32)
    np.testing.assert_allclose(oracle_lib.rope(Y, pos, theta, -1), X, atol=1e-5)
    np.testing.assert_allclose(np.linalg.norm(Y, axis=-1), np.linalg.norm(X, axis=-1), rtol=1e-6)
    q, k = _x(4, n=1, G=1)[0, 0], _x(5, n=1, G=1)[0, 0]
    for s, t in ((0, 5), (1000, 1005), (50000, 50005), (7, 3)):
        qs = oracle_lib.rope(q[None, None], s, theta)[0, 0]
        kt = oracle_lib.rope(k[None, None], t, theta)[0, 0]
        kr = oracle_lib.rope(k[None, None], t - s, theta)[0, 0]
        assert abs(qs @ kt - q.astype(np.float64) @ kr) < 1e-9 * (1 + abs(q @ k))


def test_zero_frequencies_equal_the_plain_codec(oracle_lib):
    """theta = 0: the rotation is the identity, so compression and decode are those of the
    rotation-free codec, bit for bit."""
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["tiny"]
    li = make_layer(cfg, n_queries=1)
    z = np.zeros(64, np.float32)
    a = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], 20, 16, "f32")
    b = oracle_lib.compress_rope(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], 20, 16, "f32", z)
    np.testing.assert_array_equal(a.alloc.rank, b.alloc.rank)
    np.testing.assert_array_equal(a.coefK, b.coefK)
    np.testing.assert_array_equal(oracle_lib.decode(a.coefK, a.coefV, a.alloc.rank, a.Kx, a.Vx, li.PK, li.PV,
                                                    li.q[0], cfg["H"]),
                                  oracle_lib.decode_rope(b, li.PK, li.PV, li.q[0], cfg["H"], z))


def test_full_budget_is_attention_over_the_rotated_cache(oracle_lib):
    """kappa = 100: every coded token at full rank (fp32 storage), so un-rotate, project,
    reconstruct and re-rotate give back each post-RoPE key; the decode equals plain attention
    over the cache as the model holds it."""
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["tiny_rope"]
    li = make_layer(cfg, n_queries=2)
    c = oracle_lib.compress_rope(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], 100, 16, "f32", li.theta)
    assert np.all(c.alloc.rank == 128)
    for qi in range(2):
        got = oracle_lib.decode_rope(c, li.PK, li.PV, li.q[qi], cfg["H"], li.theta)
        ref = brute_attention(li.K, li.V, li.q[qi], cfg["H"])
        np.testing.assert_allclose(got, ref, rtol=0, atol=2e-5 * np.abs(ref).max())


def test_exact_low_rank_pre_rope_keys(oracle_lib):
    """Pre-RoPE keys and values in the span of the first 16 basis rows: with r_min = 16 every
    coded token is rebuilt exactly at any budget, but only if each key is un-rotated and
    re-rotated at its own position (a shifted position leaves the span)."""
    from workloads import CONFIGS, make_layer, rope_theta
    cfg = CONFIGS["tiny_rope"]
    li = make_layer(cfg, n_queries=1)
    n, G, d = li.K.shape
    rng = np.random.default_rng(9)
    theta = rope_theta("llama3")
    Kp = np.einsum("tgj,gjd->tgd", rng.standard_normal((n, G, 16)), li.PK[:, :16, :].astype(np.float64))
    Vp = np.einsum("tgj,gjd->tgd", rng.standard_normal((n, G, 16)), li.PV[:, :16, :].astype(np.float64))
    K = oracle_lib.rope(Kp.astype(np.float32), np.arange(n), theta).astype(np.float32)
    V = Vp.astype(np.float32)
    c = oracle_lib.compress_rope(K, V, li.Qw, li.PK, li.PV, cfg["H"], 20, 16, "f32", theta)
    got = oracle_lib.decode_rope(c, li.PK, li.PV, li.q[0], cfg["H"], theta)
    ref = brute_attention(K, V, li.q[0], cfg["H"])
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-4 * np.abs(ref).max())
    # the same cache un-rotated one position late is not in the span: coefficients past 16
    Kl = oracle_lib.rope(K[:n - cfg["w"]], np.arange(1, n - cfg["w"] + 1), theta, -1)
    tail = np.einsum("tgd,gjd->tgj", Kl, li.PK[:, 16:, :].astype(np.float64))
    assert np.abs(tail).max() > 1e-2


def test_salience_stays_spiky_with_rope(oracle_lib):
    """The workload keeps its structure under rotation: the planted 5% of tokens draw most
    of the observation window's attention."""
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["tiny_rope"]
    li = make_layer(cfg)
    s = oracle_lib.salience(li.K, li.Qw, cfg["H"])
    assert s[li.planted[0]].sum() > 0.8 * s.sum()
