"""Pins for the oracle's shared cross-head basis (Sec. 3.1 Eq. (1) "Joint per-token vector"
and "Shared basis"; Eq. (3) in joint units; Eq. (6) with z_t = [k_t (all heads); v_t (all
heads)])."""
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


def _cfg(**kw):
    from workloads import CONFIGS
    c = dict(CONFIGS["tiny_joint"])
    c.update(kw)
    return c


def test_budget_in_joint_units(oracle_lib):
    """Eq. (3) with D = 2 G d: a token at rank r costs r scalars of z; the ranks spend B
    exactly, each between r_min and R."""
    from workloads import make_layer
    cfg = _cfg(G=2, H=4, seed=31, joint_R=384)
    li = make_layer(cfg)
    for kappa in (10, 20, 40):
        jc = oracle_lib.compress_joint(li.K, li.V, li.Qw, li.W, 4, kappa, 16, "f32")
        Dz = 2 * 2 * 128
        assert jc.B == (kappa * 512 * Dz) // 100 - 32 * Dz
        assert int(jc.alloc.rank.sum()) == jc.B
        assert jc.alloc.rank.min() >= 16 and jc.alloc.rank.max() <= 384


def test_rank_space_form(oracle_lib):
    """The reconstruct-in-place decode equals its rank-space form: score = <W_K,g q, m . c>
    (W_K,g = the columns of head g's keys), output = W_V,g^T sum_t a_t (m . c_t) plus the
    exact rows; written here with numpy from the block layout of z."""
    rng = np.random.default_rng(3)
    G, H, d, R, N, nx = 2, 4, 128, 320, 90, 5
    W = np.linalg.qr(rng.standard_normal((2 * G * d, R)))[0].T.astype(np.float32)
    rank = rng.integers(1, R + 1, N).astype(np.int32)
    coef = rng.standard_normal((N, R)).astype(np.float32)
    coef[np.arange(R)[None, :] >= rank[:, None]] = 0
    Kx = rng.standard_normal((nx, G, d)).astype(np.float32)
    Vx = rng.standard_normal((nx, G, d)).astype(np.float32)
    q = rng.standard_normal((H, d)).astype(np.float32)
    got = oracle_lib.decode_joint(coef, rank, Kx, Vx, W, q, H)
    C, Wd = coef.astype(np.float64), W.astype(np.float64)
    for h in range(H):
        g = h // (H // G)
        qp = Wd[:, g * d:(g + 1) * d] @ q[h]
        x = np.concatenate([C @ qp, Kx[:, g, :].astype(np.float64) @ q[h]]) / math.sqrt(d)
        a = np.exp(x - x.max())
        a /= a.sum()
        acc = a[:N] @ C
        o = Wd[:, (G + g) * d:(G + g + 1) * d].T @ acc + a[N:] @ Vx[:, g, :]
        np.testing.assert_allclose(got[h], o, rtol=0, atol=1e-12 * np.abs(o).max())


def test_full_rank_square_basis_is_attention(oracle_lib):
    """R = D (G = 1: D = 256) and kappa = 100: every coded token at full rank of an
    orthonormal square basis, so the decode is attention over the original cache."""
    from workloads import make_layer
    cfg = _cfg()
    li = make_layer(cfg, n_queries=2)
    jc = oracle_lib.compress_joint(li.K, li.V, li.Qw, li.W, 2, 100, 16, "f32")
    assert np.all(jc.alloc.rank == 256)
    for i in range(2):
        got = oracle_lib.decode_joint(jc.coef, jc.alloc.rank, jc.Kx, jc.Vx, li.W, li.q[i], 2)
        ref = brute_attention(li.K, li.V, li.q[i], 2)
        np.testing.assert_allclose(got, ref, rtol=0, atol=2e-5 * np.abs(ref).max())


def test_exact_low_rank_joint_vectors(oracle_lib):
    """Joint vectors in the span of the first 16 basis rows with r_min = 16: every token is
    rebuilt exactly at any budget, for every head, although R < D."""
    from workloads import make_layer
    cfg = _cfg(G=2, H=4, seed=33, joint_R=384)
    li = make_layer(cfg, n_queries=1)
    n, G, d = li.K.shape
    rng = np.random.default_rng(5)
    Z = rng.standard_normal((n, 16)) @ li.W[:16].astype(np.float64)
    K = Z[:, :G * d].reshape(n, G, d).astype(np.float32)
    V = Z[:, G * d:].reshape(n, G, d).astype(np.float32)
    jc = oracle_lib.compress_joint(K, V, li.Qw, li.W, 4, 20, 16, "f32")
    got = oracle_lib.decode_joint(jc.coef, jc.alloc.rank, jc.Kx, jc.Vx, li.W, li.q[0], 4)
    ref = brute_attention(K, V, li.q[0], 4)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-5 * np.abs(ref).max())


def test_projection_is_nested_and_parseval(oracle_lib):
    """Eq. (6) with orthonormal rows: the coefficients are W z, truncation keeps a prefix,
    and ||z||^2 = ||W z||^2 + ||z - W^T W z||^2 (Parseval on the span plus its complement)."""
    from workloads import make_layer
    cfg = _cfg(G=2, H=4, seed=34, joint_R=384)
    li = make_layer(cfg)
    n, G, d = li.K.shape
    full = oracle_lib.project_joint(li.K[:8], li.V[:8], li.W, np.full(8, 384, np.int32), "f32")
    part = oracle_lib.project_joint(li.K[:8], li.V[:8], li.W, np.arange(8, dtype=np.int32) * 40, "f32")
    for t in range(8):
        np.testing.assert_array_equal(part[t, :40 * t], full[t, :40 * t])
        assert np.all(part[t, 40 * t:] == 0)
    z = np.concatenate([li.K[:8].reshape(8, -1), li.V[:8].reshape(8, -1)], axis=1).astype(np.float64)
    c = full.astype(np.float64)
    resid = z - c @ li.W.astype(np.float64)
    np.testing.assert_allclose((z ** 2).sum(1), (c ** 2).sum(1) + (resid ** 2).sum(1), rtol=1e-5)


def test_generator_joint_basis_is_orthonormal_and_ordered():
    """The shared basis the workloads draw: orthonormal rows in descending order of the
    calibration second moment's eigenvalues."""
    from workloads import make_layer
    li = make_layer(_cfg(G=2, H=4, seed=35, joint_R=384))
    W = li.W.astype(np.float64)
    np.testing.assert_allclose(W @ W.T, np.eye(384), atol=1e-5)
