"""Pins for the oracle's residual codec (Sec. 3.1 "Residual codec", Eq. (2); Algorithm 1:
strided anchors and the window exact, the other tokens coded as residuals to the mean of
their c nearest anchors; Eq. (3) with n_ref = |E|)."""
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


@pytest.mark.parametrize("delta,c", [(16, 4), (8, 2), (5, 1), (16, 1)])
def test_nearest_anchors_match_brute_force(oracle_lib, delta, c):
    rng = np.random.default_rng(delta * 10 + c)
    N, G, d = 300, 2, 128
    K = rng.standard_normal((N + 8, G, d)).astype(np.float32)
    V = rng.standard_normal((N + 8, G, d)).astype(np.float32)
    nn, dist = oracle_lib.anchor_nearest(K, V, N, delta, c)
    anchors = np.arange(0, N, delta)
    Z = np.concatenate([K[:N].reshape(N, -1), V[:N].reshape(N, -1)], axis=1).astype(np.float64)
    for t in range(N):
        if t % delta == 0:
            assert np.all(nn[t] == -1)
            continue
        dd = ((Z[anchors] - Z[t]) ** 2).sum(axis=1)
        order = np.argsort(dd, kind="stable")[:c]
        assert list(nn[t]) == list(order), t
        np.testing.assert_allclose(dist[t], dd[order], rtol=1e-12)


def test_duplicate_of_an_anchor_has_zero_residual(oracle_lib):
    """With c = 1, a token equal to an anchor has that anchor as its reference and a zero
    residual: every coefficient is 0 and decode rebuilds it exactly."""
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["tiny"]
    li = make_layer(cfg, n_queries=1)
    K, V = li.K.copy(), li.V.copy()
    for t in (5, 77, 130):
        K[t], V[t] = K[48], V[48]          # anchor number 3 (token 48)
    ac = oracle_lib.compress_anchor(K, V, li.Qw, li.PK, li.PV, cfg["H"], 30, 16, "f32", delta=16, c=1)
    for t in (5, 77, 130):
        i = int(np.searchsorted(ac.coded, t))
        assert ac.coded[i] == t and ac.nn[i, 0] == 3
        assert np.all(ac.resK[i] == 0) and np.all(ac.coefK[i] == 0) and np.all(ac.coefV[i] == 0)


def test_budget_counts_the_anchors(oracle_lib):
    """Eq. (3): B = kappa n d - |E| d with E = anchors + window, in whole coefficients; the
    allocation spends exactly B over the coded tokens."""
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["tiny"]
    li = make_layer(cfg)
    for kappa in (30, 50, 100):
        ac = oracle_lib.compress_anchor(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], kappa, 16, "f32")
        n, w, d = cfg["n"], cfg["w"], 128
        na = len(ac.anchors)
        assert na == (n - w + 15) // 16 and len(ac.coded) == n - w - na
        assert ac.B == (kappa * n * d) // 100 - (na + w) * d
        assert int(ac.alloc.rank.sum()) == ac.B
        assert ac.alloc.rank.min() >= 16 and ac.alloc.rank.max() <= 128


def test_full_budget_decode_is_plain_attention(oracle_lib):
    """kappa = 100 keeps every coded token at full rank: anchor mean + full projection of
    the residual rebuild each key and value exactly (orthonormal basis, fp32 storage), so the
    decode equals attention over the original cache."""
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["tiny"]
    li = make_layer(cfg, n_queries=2)
    ac = oracle_lib.compress_anchor(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], 100, 16, "f32")
    assert np.all(ac.alloc.rank == 128)
    for i in range(2):
        o = oracle_lib.decode_anchor(ac, li.PK, li.PV, li.q[i], cfg["H"])
        ref = brute_attention(li.K, li.V, li.q[i], cfg["H"])
        np.testing.assert_allclose(o, ref, atol=2e-5 * np.abs(ref).max())


def test_rank_space_form_with_anchor_means(oracle_lib):
    """The rank-space form a fused decode computes: score = mean of the c anchor scores +
    <P_K q, m . c^K> / sqrt(d), value = mean of the anchor values + P_V^T (m . c^V); an
    independent numpy implementation of it agrees with the oracle's reconstruct-in-place
    decode to fp64 rounding."""
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["tiny"]
    li = make_layer(cfg, n_queries=1)
    H = cfg["H"]
    ac = oracle_lib.compress_anchor(li.K, li.V, li.Qw, li.PK, li.PV, H, 30, 16, "f32")
    o = oracle_lib.decode_anchor(ac, li.PK, li.PV, li.q[0], H)
    G, d = 1, 128
    q = li.q[0].astype(np.float64)
    r = ac.alloc.rank
    mask = (np.arange(d)[None, :] < r[:, None]).astype(np.float64)
    for h in range(H):
        g = h * G // H
        PKg, PVg = li.PK[g].astype(np.float64), li.PV[g].astype(np.float64)
        xa = ac.Ka[:, g, :].astype(np.float64) @ q[h] / math.sqrt(d)                  # anchors
        xc = xa[ac.nn].mean(axis=1) + (ac.coefK[:, g, :] * mask) @ (PKg @ q[h]) / math.sqrt(d)
        xe = ac.Kx[:, g, :].astype(np.float64) @ q[h] / math.sqrt(d)
        x = np.concatenate([xc, xa, xe])
        p = np.exp(x - x.max())
        p /= p.sum()
        Nc, na = len(xc), len(xa)
        pc, pa, pe = p[:Nc], p[Nc:Nc + na], p[Nc + na:]
        # anchors collect their own weight and a 1/c share of every coded token that uses them
        wa = pa.copy()
        np.add.at(wa, ac.nn.reshape(-1), np.repeat(pc / ac.nn.shape[1], ac.nn.shape[1]))
        acc = (pc[:, None] * ac.coefV[:, g, :] * mask).sum(axis=0)
        out = acc @ PVg + wa @ ac.Va[:, g, :] + pe @ ac.Vx[:, g, :]
        np.testing.assert_allclose(out, o[h], rtol=0, atol=1e-12 * np.abs(o[h]).max() + 1e-15)


def test_residual_lowers_the_coded_energy(oracle_lib):
    """The codec's premise: on the Llama-shaped draws the residual to the anchor mean is
    smaller than the token itself on average (so the same rank loses less)."""
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k"])
    cfg.update(n=2048, G=2, H=8)
    li = make_layer(cfg)
    ac = oracle_lib.compress_anchor(li.K, li.V, li.Qw, li.PK, li.PV, 8, 30, 16, "bf16")
    e = np.linalg.norm(ac.resV.astype(np.float64), axis=-1).mean()
    z = np.linalg.norm(li.V[ac.coded].astype(np.float64), axis=-1).mean()
    assert e < z
