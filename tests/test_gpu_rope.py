"""GPU parity of the rotary-key path (Sec. 3.1 "Joint per-token vector"; Algorithm 1, first
and last steps) against the fp64 oracle, through the C ABI.

Compress un-rotates each coded key at its position (hardware sine and cosine of the exact
fraction of a turn, fp32 rotation, rounded to the storage type) before the Eq. (6)
projection; decode rebuilds each coded key from its coefficients by MFMA, turns it to its
position and scores it against the post-RoPE query.  Bars: layout bit-exact; coefficients
within a per-coordinate bound that adds the rotation's error to the plain projection's;
decode within 2e-2 of max |o| per (sequence, query, head) in bf16 (fp32 layers: 1e-4)."""
import math

import numpy as np
import pytest

from test_gpu_parity import (DEC_TOL_BF16, decode_err, dev, expected_layout, host, layer, rel_err, say,
                             unpack)

pytestmark = pytest.mark.gpu

DEC_TOL_ROPE_F32 = 1e-4
TRIG_EPS = 2.0 ** -17      # allowance for the kernel's rotation per unit of |x_i| + |x_{i+64}|


@pytest.fixture(scope="module")
def vr():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible MI355X")
    import paper_2607_15498_amd as vr
    vr.library()
    return vr


def rope_shape(vr, cfg, theta, n=None, kappa=None, r_min=None, G=None, H=None):
    return vr.Shape(n=cfg["n"] if n is None else n, G=cfg["G"] if G is None else G,
                    H=cfg["H"] if H is None else H, w=cfg["w"], r_min=cfg["r_min"] if r_min is None else r_min,
                    kappa_pct=cfg["kappa"] if kappa is None else kappa, dtype=cfg["dtype"],
                    rope_theta=tuple(float(x) for x in theta))


def compress_gpu(vr, shape, li, sbar=None, cap=None, K=None, V=None):
    import torch
    dt = shape.torch_dtype
    K = li.K if K is None else K
    V = li.V if V is None else V
    Kd, Vd, Qw = dev(K, dt), dev(V, dt), dev(li.Qw, dt)
    PK, PV = dev(li.PK, torch.float32), dev(li.PV, torch.float32)
    if sbar is None:
        cache = vr.compress(shape, Kd, Vd, Qw, PK, PV, cap=cap)
    else:
        cache = vr.new_cache(shape, cap)
        vr.allocate(shape, dev(sbar, torch.float32), cache)
        vr.project(shape, Kd, Vd, PK, PV, cache)
    torch.cuda.synchronize()
    return cache, PK, PV


_OC = {}


def oracle_rope(oracle_lib, name, li, kappa=None, r_min=None):
    from workloads import CONFIGS
    cfg = CONFIGS[name]
    key = (name, kappa, r_min, li.q.shape[0])
    if key not in _OC:
        _OC[key] = oracle_lib.compress_rope(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"],
                                            cfg["kappa"] if kappa is None else kappa,
                                            cfg["r_min"] if r_min is None else r_min, cfg["dtype"], li.theta)
    return _OC[key]


def _ulp(x, storage):
    """Spacing of the storage type's values at |x| (bf16: 8 significant bits)."""
    a = np.maximum(np.abs(x), 1e-38)
    e = np.floor(np.log2(a))
    return 2.0 ** (e - (7 if storage == "bf16" else 23))


@pytest.mark.parametrize("name", ["tiny_rope", "llama_32k_rope"])
def test_rope_projection(vr, oracle_lib, name):
    from workloads import CONFIGS
    cfg = CONFIGS[name]
    say(f"[rope project] {name}")
    li = layer(name)
    oc = oracle_rope(oracle_lib, name, li)
    shape = rope_shape(vr, cfg, li.theta)
    cache, _, _ = compress_gpu(vr, shape, li, sbar=oc.sbar)
    N = shape.N
    rank = oc.alloc.rank.astype(np.int64)
    srank, sidx, chunk_off = expected_layout(rank, N)
    assert np.array_equal(host(cache.sidx).astype(np.int64), sidx)
    assert np.array_equal(host(cache.chunk_off).astype(np.int64), chunk_off)
    st = cfg["dtype"]
    # the oracle's un-rotated keys (fp64) and their rounding to the storage type
    Ku64 = oracle_lib.rope(li.K[:N], np.arange(N), li.theta, -1)
    for kind, ref in (("K", oc.coefK), ("V", oc.coefV)):
        got = unpack(host(cache.coef_k if kind == "K" else cache.coef_v), srank, sidx, chunk_off, N, kind)
        err = np.abs(got - ref)
        P = li.PK if kind == "K" else li.PV
        X = oracle_lib.round_storage(Ku64, st) if kind == "K" else li.V[:N]
        Xa = np.abs(X.astype(np.float64))
        # plain projection bound (as for position-free keys): 2^-15 S_j plus storage rounding
        S = np.stack([Xa[:, g, :] @ np.abs(P[g].astype(np.float64)).T for g in range(X.shape[1])], axis=1)
        bound = np.abs(ref) * (2.0 ** -7 if st == "bf16" else 2.0 ** -23) + 2.0 ** -15 * S
        if kind == "K":
            # the kernel's rotation errs by at most TRIG_EPS (|x_i| + |x_{i+64}|) per coordinate
            # before its rounding to the storage type, which can then land one unit away
            K0 = np.abs(li.K[:N].astype(np.float64))
            pair = K0[..., :64] + K0[..., 64:]
            amb = TRIG_EPS * np.concatenate([pair, pair], axis=-1) + _ulp(Ku64, st)
            bound = bound + np.stack([amb[:, g, :] @ np.abs(P[g].astype(np.float64)).T for g in range(X.shape[1])],
                                     axis=1)
        ok = err <= bound
        say(f"  {kind}: max rel {rel_err(got, ref):.3e}, max err / bound {float((err / bound).max()):.3e}, "
            f"identical {float((err == 0).mean()):.4f}")
        assert ok.all()
    # the window stays exact and post-RoPE
    w = shape.w
    assert np.array_equal(host(cache.k_exact)[:, :w].transpose(1, 0, 2), li.K[N:])


@pytest.mark.parametrize("name", ["tiny_rope", "llama_32k_rope"])
def test_rope_decode_same_ranks(vr, oracle_lib, name):
    import torch
    from workloads import CONFIGS
    cfg = CONFIGS[name]
    say(f"[rope decode] {name}")
    li = layer(name, n_queries=2)
    oc = oracle_rope(oracle_lib, name, li)
    shape = rope_shape(vr, cfg, li.theta)
    cache, PK, PV = compress_gpu(vr, shape, li, sbar=oc.sbar)
    assert np.array_equal(host(cache.rank).astype(np.int64), oc.alloc.rank)
    out = host(vr.decode(shape, [cache], dev(li.q, shape.torch_dtype), PK, PV))
    torch.cuda.synchronize()
    tol = DEC_TOL_ROPE_F32 if cfg["dtype"] == "f32" else DEC_TOL_BF16
    for i in range(li.q.shape[0]):
        o_or = oracle_lib.decode_rope(oc, li.PK, li.PV, li.q[i], cfg["H"], li.theta)
        e = decode_err(out[i], o_or)
        say(f"  query {i}: decode max rel err {e:.3e}")
        assert e <= tol


def test_rope_end_to_end(vr, oracle_lib):
    """GPU salience on the post-RoPE cache feeds the GPU allocation; the oracle runs the
    whole rotary path independently."""
    import torch
    from workloads import CONFIGS
    name = "llama_32k_rope"
    cfg = CONFIGS[name]
    say(f"[rope end-to-end] {name}")
    li = layer(name, n_queries=2)
    oc = oracle_rope(oracle_lib, name, li)
    shape = rope_shape(vr, cfg, li.theta)
    cache, PK, PV = compress_gpu(vr, shape, li)
    mism = int((host(cache.rank).astype(np.int64) != oc.alloc.rank).sum())
    out = host(vr.decode(shape, [cache], dev(li.q, torch.bfloat16), PK, PV))
    torch.cuda.synchronize()
    errs = [decode_err(out[i], oracle_lib.decode_rope(oc, li.PK, li.PV, li.q[i], cfg["H"], li.theta))
            for i in range(2)]
    say(f"  rank mismatches {mism} of {shape.N}; decode max rel err {max(errs):.3e}")
    assert mism <= max(8, shape.N // 1000)
    assert max(errs) <= DEC_TOL_BF16


def test_rope_full_budget_is_attention(vr):
    """kappa = 100: every token at full rank, so decode equals attention over the post-RoPE
    bf16 cache (up to the rounding of the un-rotated keys and of the coefficients)."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k_rope"])
    cfg.update(n=3000, G=2, H=8, seed=15)
    li = make_layer(cfg, n_queries=1)
    shape = rope_shape(vr, cfg, li.theta, kappa=100)
    cache, PK, PV = compress_gpu(vr, shape, li)
    assert int(host(cache.rank).min()) == 128
    out = host(vr.decode(shape, [cache], dev(li.q, torch.bfloat16), PK, PV))[0]
    ref = np.zeros((8, 128))
    for h in range(8):
        g = h // 4
        x = li.K[:, g, :].astype(np.float64) @ li.q[0, h].astype(np.float64) / math.sqrt(128)
        a = np.exp(x - x.max())
        a /= a.sum()
        ref[h] = a @ li.V[:, g, :]
    e = decode_err(out, ref)
    say(f"[rope full budget] err vs attention {e:.3e}")
    assert e <= DEC_TOL_BF16


def test_rope_multi_sequence_appended(vr, oracle_lib):
    """S = 3 sequences, Q = 5 queries (20 rows per KV head: two row tiles), a ragged last
    chunk and 3 post-RoPE exact tokens appended after compression."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k_rope"])
    cfg.update(n=1300, G=2, H=8, seed=78)
    Q, extra, n = 5, 3, 1300
    caches, qs, refs = [], [], []
    for s in range(3):
        li = make_layer(cfg, seq=s, n_queries=Q, n=n + extra)
        shape = rope_shape(vr, cfg, li.theta, n=n)
        Kc, Vc = li.K[:n], li.V[:n]
        # the window queries of a prompt of n tokens sit at n - w .. n - 1: redraw them for n
        li_n = make_layer(cfg, seq=s, n_queries=Q, n=n)
        oc = oracle_lib.compress_rope(Kc, Vc, li_n.Qw, li.PK, li.PV, 8, 20, 16, "bf16", li.theta)
        cache, PK, PV = compress_gpu(vr, shape, li_n, sbar=oc.sbar, cap=32 + extra, K=Kc, V=Vc)
        for e in range(extra):
            vr.append_exact(shape, cache, dev(li.K[n + e], torch.bfloat16), dev(li.V[n + e], torch.bfloat16))
        caches.append(cache)
        qs.append(li.q)
        ocx = type(oc)(oc.s, oc.sbar, oc.u, oc.alloc, oc.B, oc.coefK, oc.coefV,
                       np.concatenate([oc.Kx, li.K[n:]]), np.concatenate([oc.Vx, li.V[n:]]))
        refs.append([oracle_lib.decode_rope(ocx, li.PK, li.PV, li.q[i], 8, li.theta) for i in range(Q)])
    out = host(vr.decode(shape, caches, dev(np.stack(qs), torch.bfloat16), PK, PV))
    torch.cuda.synchronize()
    worst = max(decode_err(out[s][i], refs[s][i]) for s in range(3) for i in range(Q))
    say(f"[rope multi] worst decode rel err {worst:.3e}")
    assert worst <= DEC_TOL_BF16


def test_rope_zero_frequencies_match_the_plain_path(vr):
    """theta = 0: the rotary path computes the plain codec (ranks and coefficients bit for
    bit; decode through the reconstruction within rounding of the rank-space decode)."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k"])
    cfg.update(n=2600, G=2, H=8, seed=21)
    li = make_layer(cfg, n_queries=1)
    plain = vr.Shape(n=2600, G=2, H=8, w=32, r_min=16, kappa_pct=20, dtype="bf16")
    rot = rope_shape(vr, cfg, np.zeros(64), n=2600, G=2, H=8)
    c0, PK, PV = compress_gpu(vr, plain, li)
    c1, _, _ = compress_gpu(vr, rot, li)
    assert torch.equal(c0.rank, c1.rank) and torch.equal(c0.coef_k, c1.coef_k) and torch.equal(c0.coef_v, c1.coef_v)
    q = dev(li.q, torch.bfloat16)
    o0 = host(vr.decode(plain, [c0], q, PK, PV))[0]
    o1 = host(vr.decode(rot, [c1], q, PK, PV))[0]
    e = decode_err(o1, o0)
    say(f"[rope theta=0] rotary vs rank-space decode {e:.3e}")
    assert e <= 2e-3
