"""Pins for the oracle's projection/truncation (Sec. 3.3 Eq. (6)) and reconstruct-in-place
decode (Sec. 4.4 "Cost"), plus the end-to-end oracle on the tiny workload."""
import math

import numpy as np
import pytest


def brute_attention(K, V, q, H):
    """Independent full-KV attention: K,V [T][G][d], q [H][d] -> [H][d] (fp64)."""
    T, G, d = K.shape
    out = np.zeros((H, d))
    for h in range(H):
        g = (h * G) // H
        x = K[:, g, :].astype(np.float64) @ q[h].astype(np.float64) / math.sqrt(d)
        a = np.exp(x - x.max())
        a /= a.sum()
        out[h] = a @ V[:, g, :].astype(np.float64)
    return out


def signed_permutation(rng, d):
    P = np.zeros((d, d), np.float32)
    P[np.arange(d), rng.permutation(d)] = rng.choice([-1.0, 1.0], d)
    return P


def test_basis_orthonormal():
    from workloads import CONFIGS, make_layer
    li = make_layer(CONFIGS["tiny"])
    for P in (li.PK[0], li.PV[0]):
        P = P.astype(np.float64)
        np.testing.assert_allclose(P @ P.T, np.eye(128), atol=2e-6)


def test_projection_full_rank_is_exact_and_parseval(oracle_lib):
    """Orthonormal P: full rank reproduces x; the truncation error at rank r equals the
    energy of the dropped coefficients (Parseval) and never grows with r."""
    from workloads import CONFIGS, make_layer
    li = make_layer(CONFIGS["tiny"])
    X = li.K[:40]
    P = li.PK
    x = X[:, 0, :].astype(np.float64)
    full = oracle_lib.project(X, P, np.full(40, 128, np.int32), "f32")[:, 0, :].astype(np.float64)
    Pd = P[0].astype(np.float64)
    np.testing.assert_allclose(full @ Pd, x, atol=1e-5 * np.abs(x).max())
    prev = None
    for r in (1, 8, 16, 33, 64, 100, 128):
        c = oracle_lib.project(X, P, np.full(40, r, np.int32), "f32")[:, 0, :].astype(np.float64)
        assert np.all(c[:, r:] == 0)
        np.testing.assert_allclose(c[:, :r], full[:, :r], rtol=0, atol=0)
        err = np.sum((x - c @ Pd) ** 2, axis=1)
        dropped = np.sum(full[:, r:] ** 2, axis=1)
        np.testing.assert_allclose(err, dropped, rtol=1e-4, atol=1e-8)
        if prev is not None:
            assert np.all(err <= prev + 1e-9)
        prev = err


def test_projection_storage_rounding_is_nearest_bf16(oracle_lib):
    """bf16 storage keeps the coefficient nearest to the exact projection (8 significant
    bits, ties to even): check against torch's bfloat16 rounding of the fp32 value where
    the fp64 and fp32 values round identically."""
    import torch
    rng = np.random.default_rng(11)
    X = rng.standard_normal((64, 2, 128)).astype(np.float32)
    P = np.stack([signed_permutation(rng, 128), signed_permutation(rng, 128)])
    P[1] *= np.float32(0.7)              # non-trivial products
    r = np.full(64, 128, np.int32)
    c32 = oracle_lib.project(X, P, r, "f32")
    cbf = oracle_lib.project(X, P, r, "bf16")
    ref = torch.from_numpy(c32).to(torch.bfloat16).float().numpy()
    np.testing.assert_array_equal(cbf, ref)


def test_decode_full_rank_equals_full_attention(oracle_lib):
    """Budget B = N R keeps every coded token at full rank; with an exactly orthogonal basis
    (signed permutation) reconstruct-in-place is exact and decode is plain attention."""
    rng = np.random.default_rng(12)
    n, w, G, H, d = 300, 20, 2, 6, 128
    K = rng.standard_normal((n, G, d)).astype(np.float32)
    V = rng.standard_normal((n, G, d)).astype(np.float32)
    PK = np.stack([signed_permutation(rng, d) for _ in range(G)])
    PV = np.stack([signed_permutation(rng, d) for _ in range(G)])
    N = n - w
    rank = np.full(N, d, np.int32)
    cK = oracle_lib.project(K[:N], PK, rank, "f32")
    cV = oracle_lib.project(V[:N], PV, rank, "f32")
    q = rng.standard_normal((H, d)).astype(np.float32)
    o = oracle_lib.decode(cK, cV, rank, K[N:], V[N:], PK, PV, q, H)
    np.testing.assert_allclose(o, brute_attention(K, V, q, H), rtol=1e-12, atol=1e-13)


def test_decode_exact_low_rank_data(oracle_lib):
    """Keys/values supported on the first 16 basis directions: every rank >= r_min = 16
    reproduces them exactly, so the compressed cache decodes like the full one."""
    from workloads import CONFIGS, make_layer
    li = make_layer(CONFIGS["tiny"])
    rng = np.random.default_rng(13)
    n, w, d = 512, 32, 128
    PK, PV = li.PK.astype(np.float64), li.PV.astype(np.float64)
    K = (rng.standard_normal((n, 1, 16)) @ PK[0, :16]).astype(np.float32)
    V = (rng.standard_normal((n, 1, 16)) @ PV[0, :16]).astype(np.float32)
    c = oracle_lib.compress(K, V, li.Qw, li.PK, li.PV, 2, 20, 16, "f32")
    assert c.alloc.rank.min() >= 16
    o = oracle_lib.decode(c.coefK, c.coefV, c.alloc.rank, c.Kx, c.Vx, li.PK, li.PV, li.q[0], 2)
    np.testing.assert_allclose(o, brute_attention(K, V, li.q[0], 2), rtol=2e-5, atol=2e-6)


def test_decode_rank_space_identity(oracle_lib):
    """<q, P^T (m.c)> = <P q, m.c> and sum_t a_t P^T (m.c_t) = P^T sum_t a_t (m.c_t): the
    rank-space evaluation (what a fused kernel computes) equals reconstruct-in-place."""
    from workloads import CONFIGS, make_layer
    li = make_layer(CONFIGS["tiny"])
    c = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, 2, 20, 16, "f32")
    o = oracle_lib.decode(c.coefK, c.coefV, c.alloc.rank, c.Kx, c.Vx, li.PK, li.PV, li.q[0], 2)
    PK, PV = li.PK[0].astype(np.float64), li.PV[0].astype(np.float64)
    cK, cV = c.coefK[:, 0].astype(np.float64), c.coefV[:, 0].astype(np.float64)
    for h in range(2):
        q = li.q[0, h].astype(np.float64)
        qr = PK @ q
        xs = np.concatenate([cK @ qr, c.Kx[:, 0].astype(np.float64) @ q]) / math.sqrt(128)
        a = np.exp(xs - xs.max())
        a /= a.sum()
        N = cK.shape[0]
        o_h = PV.T @ (a[:N] @ cV) + a[N:] @ c.Vx[:, 0].astype(np.float64)
        np.testing.assert_allclose(o[h], o_h, rtol=1e-10, atol=1e-13)


def test_decode_appended_exact_tokens(oracle_lib):
    """Tokens appended after compression stay exact and join the softmax."""
    rng = np.random.default_rng(14)
    n, w, G, H, d = 200, 10, 1, 2, 128
    K = rng.standard_normal((n + 5, G, d)).astype(np.float32)
    V = rng.standard_normal((n + 5, G, d)).astype(np.float32)
    P = np.stack([signed_permutation(rng, d)])
    N = n - w
    rank = np.full(N, d, np.int32)
    cK = oracle_lib.project(K[:N], P, rank, "f32")
    cV = oracle_lib.project(V[:N], P, rank, "f32")
    q = rng.standard_normal((H, d)).astype(np.float32)
    o = oracle_lib.decode(cK, cV, rank, K[N:], V[N:], P, P, q, H)
    np.testing.assert_allclose(o, brute_attention(K, V, q, H), rtol=1e-12, atol=1e-13)


def test_tiny_end_to_end_error_falls_with_budget(oracle_lib):
    """Directional check (not a parity pin): decode error vs full attention shrinks as the
    budget grows, and full budget is exact up to the fp32 basis."""
    from workloads import CONFIGS, make_layer
    li = make_layer(CONFIGS["tiny"], n_queries=4)
    ref = [brute_attention(li.K, li.V, li.q[i], 2) for i in range(4)]
    errs = []
    r_min = 4                             # fixed floor: the floor itself moves the error
    for kappa in (13, 20, 40, 100):
        c = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, 2, kappa, r_min, "f32")
        e = 0.0
        for i in range(4):
            o = oracle_lib.decode(c.coefK, c.coefV, c.alloc.rank, c.Kx, c.Vx, li.PK, li.PV,
                                  li.q[i], 2)
            e = max(e, np.abs(o - ref[i]).max() / np.abs(ref[i]).max())
        errs.append(e)
    assert errs[0] >= errs[1] >= errs[2] >= errs[3]
    assert errs[3] < 1e-5
