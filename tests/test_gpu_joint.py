"""GPU parity of the shared cross-head basis (Sec. 3.1 Eq. (1) "Joint per-token vector" and
"Shared basis"; Eq. (3) in joint units; Eq. (6)) against the fp64 oracle, through the C ABI.

Bars: 16-bit ranks, per-token offsets and chunk offsets bit-exact given the same fp32 pooled
salience; coefficients within a per-coordinate bound of the bf16 hi + lo projection (plus one
storage rounding); decode within 2e-2 of max |o| per (sequence, query, head) in bf16, 1e-4
in fp32."""
import math

import numpy as np
import pytest

from test_gpu_parity import DEC_TOL_BF16, DEC_TOL_F32, check_salience, decode_err, dev, host, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def vr():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible MI355X")
    import paper_2607_15498_amd as vr
    vr.library()
    return vr


def jshape(vr, cfg, n=None, kappa=None, r_min=None):
    return vr.Shape(n=cfg["n"] if n is None else n, G=cfg["G"], H=cfg["H"], w=cfg["w"],
                    r_min=cfg["r_min"] if r_min is None else r_min,
                    kappa_pct=cfg["kappa"] if kappa is None else kappa, dtype=cfg["dtype"])


def gpu_joint(vr, shape, li, cap=None, K=None, V=None):
    import torch
    dt = shape.torch_dtype
    K = li.K if K is None else K
    V = li.V if V is None else V
    sb = torch.empty(shape.n - shape.w, dtype=torch.float32, device="cuda")
    W = dev(li.W, torch.float32)
    c = vr.joint_compress(shape, dev(K, dt), dev(V, dt), dev(li.Qw, dt), W, cap=cap, sbar_out=sb)
    torch.cuda.synchronize()
    return c, host(sb), W


def unpack_joint(c):
    rank = host(c.rank).astype(np.int64)
    off = host(c.offset).astype(np.int64)
    coef = host(c.coef)
    out = np.zeros((c.N, c.R), np.float32)
    for t in range(c.N):
        out[t, :rank[t]] = coef[off[t]:off[t] + rank[t]]
    return out


def _cfg(name, **kw):
    from workloads import CONFIGS
    c = dict(CONFIGS[name])
    c.update(kw)
    return c


CASES = {
    "tiny_joint": dict(),
    "small_joint": dict(n=4096, G=2, H=8, seed=41, joint_R=512),
    "small_joint_r256": dict(n=3000, G=2, H=8, seed=42, joint_R=256, kappa=10),
}


def _case(name):
    from workloads import make_layer
    base = "tiny_joint" if name == "tiny_joint" else "llama_32k_joint"
    cfg = _cfg(base, **CASES[name])
    return cfg, make_layer(cfg, n_queries=2)


@pytest.mark.parametrize("name", list(CASES))
def test_joint_allocation_layout_projection_decode(vr, oracle_lib, name):
    import torch
    cfg, li = _case(name)
    say(f"[joint] {name}: n {cfg['n']}, G {cfg['G']}, R {cfg['joint_R']}, kappa {cfg['kappa']}")
    shape = jshape(vr, cfg)
    c, sb_gpu, W = gpu_joint(vr, shape, li)
    # the allocation given the GPU's pooled salience, bit for bit
    oc = oracle_lib.compress_joint(li.K, li.V, li.Qw, li.W, cfg["H"], cfg["kappa"], cfg["r_min"], cfg["dtype"],
                                   sbar=sb_gpu)
    rank = host(c.rank).astype(np.int64)
    assert c.B == oc.B and rank.sum() == oc.B
    assert np.array_equal(rank, oc.alloc.rank)
    off = host(c.offset).astype(np.int64)
    assert np.array_equal(off, np.concatenate([[0], np.cumsum(rank)]))
    assert np.array_equal(host(c.chunk_off).astype(np.int64), off[::256][: len(host(c.chunk_off)) - 1].tolist() + [oc.B])
    # salience against the oracle's
    check_salience(sb_gpu, oracle_lib.pool(oracle_lib.salience(li.K, li.Qw, cfg["H"])), f"joint {name}")
    # coefficients: bf16 hi + lo basis against exact inputs -> 2^-15 S_j, plus one storage rounding
    got = unpack_joint(c)
    ref = oc.coef
    N = shape.n - shape.w
    Z = np.concatenate([li.K[:N].reshape(N, -1), li.V[:N].reshape(N, -1)], axis=1).astype(np.float64)
    S = np.abs(Z) @ np.abs(li.W.astype(np.float64)).T
    st = 2.0 ** -7 if cfg["dtype"] == "bf16" else 2.0 ** -23
    mask = np.arange(c.R)[None, :] < rank[:, None]
    err = np.abs(got - ref)
    bound = np.abs(ref) * st + 2.0 ** -15 * S
    say(f"  coefficients: max err / bound {float((err / bound)[mask].max()):.3e}, identical "
        f"{float((err == 0)[mask].mean()):.4f}")
    assert (err <= bound).all()
    # window rows exact
    w = shape.w
    assert np.array_equal(host(c.k_exact)[:, :w].transpose(1, 0, 2), li.K[N:])
    # decode against the oracle's reconstruct-in-place attention on the same ranks
    out = host(vr.joint_decode(shape, [c], dev(li.q, shape.torch_dtype), W))
    torch.cuda.synchronize()
    tol = DEC_TOL_F32 if cfg["dtype"] == "f32" else DEC_TOL_BF16
    for i in range(li.q.shape[0]):
        o_or = oracle_lib.decode_joint(oc.coef, oc.alloc.rank, oc.Kx, oc.Vx, li.W, li.q[i], cfg["H"])
        e = decode_err(out[i], o_or)
        say(f"  query {i}: decode max rel err {e:.3e}")
        assert e <= tol


def test_joint_llama_32k_end_to_end(vr, oracle_lib):
    """The Llama-shaped 32K layer with R = 1024 (Dz = 2048): GPU salience feeds the GPU
    allocation; the oracle runs the whole path independently.  Coefficients of a sample of
    tokens, then the decode of two queries (32 query rows: two row tiles)."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["llama_32k_joint"]
    li = make_layer(cfg, n_queries=2)
    shape = jshape(vr, cfg)
    say(f"[joint end-to-end] llama_32k_joint")
    c, sb_gpu, W = gpu_joint(vr, shape, li)
    oc = oracle_lib.compress_joint(li.K, li.V, li.Qw, li.W, cfg["H"], cfg["kappa"], cfg["r_min"], "bf16")
    rank = host(c.rank).astype(np.int64)
    mism = int((rank != oc.alloc.rank).sum())
    # one query per call (32 query rows, the most one decode takes)
    errs = []
    for i in range(2):
        out = host(vr.joint_decode(shape, [c], dev(li.q[i:i + 1], torch.bfloat16), W))[0]
        torch.cuda.synchronize()
        errs.append(decode_err(out, oracle_lib.decode_joint(oc.coef, oc.alloc.rank, oc.Kx, oc.Vx, li.W, li.q[i],
                                                           cfg["H"])))
    say(f"  rank mismatches {mism} of {shape.n - shape.w}; decode max rel err {max(errs):.3e}; mean rank "
        f"{rank.mean():.1f}")
    assert mism <= max(8, (shape.n - shape.w) // 1000)
    assert max(errs) <= DEC_TOL_BF16


def test_joint_square_full_rank_is_attention(vr):
    """R = Dz (G = 1) and kappa = 100: every token at full rank of an orthonormal square basis,
    so the decode is attention over the cache (fp32 layer)."""
    import torch
    cfg, li = _case("tiny_joint")
    shape = jshape(vr, cfg, kappa=100)
    c, _, W = gpu_joint(vr, shape, li)
    assert int(host(c.rank).min()) == 256
    out = host(vr.joint_decode(shape, [c], dev(li.q, torch.float32), W))[0]
    ref = np.zeros((2, 128))
    for h in range(2):
        x = li.K[:, 0, :].astype(np.float64) @ li.q[0, h].astype(np.float64) / math.sqrt(128)
        a = np.exp(x - x.max())
        a /= a.sum()
        ref[h] = a @ li.V[:, 0, :]
    e = decode_err(out, ref)
    say(f"[joint full rank] err vs attention {e:.3e}")
    assert e <= DEC_TOL_F32


@pytest.mark.parametrize("Q", [2, 4])
def test_joint_multi_sequence_appended(vr, oracle_lib, Q):
    """S = 3 sequences, Q queries (16 or 32 query rows), a ragged last tile and 3 exact tokens
    appended after compression."""
    import torch
    from workloads import make_layer
    cfg = _cfg("llama_32k_joint", n=1300, G=2, H=8, seed=43, joint_R=256)
    shape = jshape(vr, cfg)
    extra = 3
    caches, qs, refs = [], [], []
    for s in range(3):
        li = make_layer(cfg, seq=s, n_queries=Q, n=1300 + extra)
        Kc, Vc = li.K[:1300], li.V[:1300]
        c, sb, W = gpu_joint(vr, shape, li, cap=32 + extra, K=Kc, V=Vc)
        for e in range(extra):
            vr.joint_append_exact(shape, c, dev(li.K[1300 + e], torch.bfloat16), dev(li.V[1300 + e], torch.bfloat16))
        oc = oracle_lib.compress_joint(Kc, Vc, li.Qw, li.W, 8, 20, 16, "bf16", sbar=sb)
        assert np.array_equal(host(c.rank).astype(np.int64), oc.alloc.rank)
        Kx = np.concatenate([oc.Kx, li.K[1300:]])
        Vx = np.concatenate([oc.Vx, li.V[1300:]])
        caches.append(c)
        qs.append(li.q)
        refs.append([oracle_lib.decode_joint(oc.coef, oc.alloc.rank, Kx, Vx, li.W, li.q[i], 8) for i in range(Q)])
    out = host(vr.joint_decode(shape, caches, dev(np.stack(qs), torch.bfloat16), W))
    torch.cuda.synchronize()
    worst = max(decode_err(out[s][i], refs[s][i]) for s in range(3) for i in range(Q))
    say(f"[joint multi Q={Q}] worst decode rel err {worst:.3e}")
    assert caches[0].n_exact == 32 + extra
    assert worst <= DEC_TOL_BF16
