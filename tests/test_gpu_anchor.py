"""GPU parity of the residual codec (Sec. 3.1 "Residual codec", Eq. (2); Algorithm 1: strided
exact anchors, each other prefix token coded as its residual to the mean of its 4 nearest
anchors), through the C ABI, against the fp64 CPU oracle.

* Nearest anchors are an argmin over floating-point distances: the GPU ranks by fp32 keys
  ||z_a||^2 - 2 <z_a, z_t> (exact bf16 products, fp32 sums), the oracle by exact fp64
  distances.  Where they pick different anchors, the GPU's picks must lie within the fp32
  error bound of the oracle's 4th nearest distance (a valid choice); the count is reported.
* Given the oracle's salience and nearest anchors, ranks, storage order and anchor lists are
  bit-exact, anchors and window rows exact, coefficients within the bound derived below.
* Decode over the compressed cache within 2e-2 of max |o| per (sequence, query, head)."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

DEC_TOL_BF16 = 2e-2
DELTA = 16


def say(*a):
    import os
    print(*a, file=sys.stderr, flush=True)
    path = os.environ.get("VARRATE_PARITY_LOG")
    if path:
        with open(path, "a") as fh:
            print(*a, file=fh)


@pytest.fixture(scope="module")
def vr():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible MI355X")
    import paper_2607_15498_amd as vr
    vr.library()
    return vr


def dev(a, dt):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(dt).cuda()


def host(t):
    import torch
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy()


CASES = {
    # name: (base config, overrides, kappa, r_min)
    "llama_8k": ("llama_32k", dict(n=8192, seed=61), 20, 16),
    "qwen_16k": ("qwen_16k_stack", dict(), 25, 16),
    "llama_ragged": ("llama_32k", dict(n=1300, G=2, H=8, seed=62), 30, 16),
}
_PREP = {}


def prepared(vr, oracle_lib, name, n_queries=1):
    import torch
    from workloads import CONFIGS, make_layer
    key = (name, n_queries)
    if key in _PREP:
        return _PREP[key]
    base, over, kappa, r_min = CASES[name]
    cfg = dict(CONFIGS[base])
    cfg.update(over)
    li = make_layer(cfg, n_queries=n_queries)
    ac = oracle_lib.compress_anchor(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], kappa, r_min, "bf16", delta=DELTA)
    shape = vr.Shape(n=cfg["n"], G=cfg["G"], H=cfg["H"], w=cfg["w"], r_min=r_min, kappa_pct=kappa,
                     dtype="bf16", anchor_stride=DELTA)
    _PREP[key] = (cfg, li, ac, shape)
    return _PREP[key]


def zdist(li, t, anchors_tok):
    """Exact squared distances over the joint vector of token t to the given anchor tokens."""
    z = lambda i: np.concatenate([li.K[i].reshape(-1), li.V[i].reshape(-1)]).astype(np.float64)
    zt = z(t)
    return np.array([((z(a) - zt) ** 2).sum() for a in anchors_tok]), (zt ** 2).sum()


@pytest.mark.parametrize("name", ["llama_8k", "qwen_16k", "llama_ragged"])
def test_anchor_search(vr, oracle_lib, name):
    import torch
    cfg, li, ac, shape = prepared(vr, oracle_lib, name)
    say(f"[anchor search] {name}: N={shape.N} coded, {shape.na} anchors, z of {2 * cfg['G'] * 128}")
    nn = host(vr.anchor_search(shape, dev(li.K, torch.bfloat16), dev(li.V, torch.bfloat16))).astype(np.int64)
    torch.cuda.synchronize()
    want = ac.nn.astype(np.int64)
    assert nn.shape == want.shape
    diff = np.nonzero(np.any(nn != want, axis=1))[0]
    za2 = np.array([(np.concatenate([li.K[a].reshape(-1), li.V[a].reshape(-1)]).astype(np.float64) ** 2).sum()
                    for a in ac.anchors])
    for i in diff:
        t = int(ac.coded[i])
        d_gpu, zt2 = zdist(li, t, ac.anchors[nn[i]])
        # fp32 keys: each of the 2 G d products is exact, the sums round at 2^-24 per add, so
        # a key is within about 2^-24 * 2 G d * (|z_a|^2 + |z_t|^2) of exact; be generous
        eps = 2.0 ** -12 * (zt2 + za2.max())
        assert len(set(nn[i].tolist())) == 4, i
        assert np.all(d_gpu <= ac.dist[i, 3] + eps), (i, d_gpu, ac.dist[i])
        assert np.all(np.sort(d_gpu) <= ac.dist[i] + eps), (i, d_gpu, ac.dist[i])
    say(f"  tokens whose anchor set differs from the oracle's: {len(diff)} of {len(want)} (all within the fp32 bound)")
    assert len(diff) <= max(4, len(want) // 1000)


def layout(rank, N):
    srank = np.empty(N, np.int64)
    sidx = np.empty(N, np.int64)
    nch = (N + 255) // 256
    chunk_off = np.zeros(nch + 1, np.int64)
    for c in range(nch):
        t = np.arange(c * 256, min(N, c * 256 + 256))
        order = np.lexsort((t, -rank[t]))
        sidx[t] = t[order]
        srank[t] = rank[t][order]
        chunk_off[c + 1] = chunk_off[c] + 16 * srank[t][::16].sum()
    return srank, sidx, chunk_off


def encode_with_oracle_inputs(vr, oracle_lib, name, n_queries=1, cap=None):
    import torch
    cfg, li, ac, shape = prepared(vr, oracle_lib, name, n_queries)
    PK, PV = dev(li.PK, torch.float32), dev(li.PV, torch.float32)
    cache = vr.anchor_encode(shape, dev(li.K, torch.bfloat16), dev(li.V, torch.bfloat16), dev(ac.sbar, torch.float32),
                             dev(ac.nn.astype(np.int16), torch.int16), PK, PV, cap=cap)
    torch.cuda.synchronize()
    return cfg, li, ac, shape, cache, PK, PV


@pytest.mark.parametrize("name", ["llama_8k", "qwen_16k", "llama_ragged"])
def test_anchor_encode_given_oracle_salience_and_anchors(vr, oracle_lib, name):
    from test_gpu_parity import unpack
    cfg, li, ac, shape, cache, PK, PV = encode_with_oracle_inputs(vr, oracle_lib, name)
    N = shape.N
    say(f"[anchor encode] {name}: B={cache.B} over {N} coded tokens")
    rank = host(cache.rank).astype(np.int64)
    assert np.array_equal(rank, ac.alloc.rank) and cache.B == ac.B and int(rank.sum()) == ac.B
    srank, sidx, chunk_off = layout(rank, N)
    assert np.array_equal(host(cache.sidx).astype(np.int64), sidx)
    assert np.array_equal(host(cache.chunk_off).astype(np.int64), chunk_off)
    # exact rows: anchors and window
    assert np.array_equal(host(cache.k_anchor), ac.Ka) and np.array_equal(host(cache.v_anchor), ac.Va)
    assert np.array_equal(host(cache.k_exact)[:, :shape.w].transpose(1, 0, 2), ac.Kx)
    # anchors of each stored position, and the inverse lists
    snn = host(cache.snn).astype(np.int64)
    assert np.array_equal(snn, ac.nn[sidx].astype(np.int64))
    off = host(cache.inv_off).astype(np.int64)
    pos = host(cache.inv_pos).astype(np.int64)
    assert off[0] == 0 and off[-1] == 4 * N
    for a in range(shape.na):
        got = np.sort(pos[off[a]:off[a + 1]])
        want = np.sort(np.nonzero(np.any(snn == a, axis=1))[0])
        assert np.array_equal(got, want), a
    # coefficients of the residuals: the kernel forms the anchor mean in fp32 and rounds the
    # residual to bf16, which may land one bf16 unit (2^-8 relative) from the oracle's rounding
    # of the exact residual; the projection then adds at most 2^-15 S_j and bf16 storage one
    # more unit of the result: |c - c_or| <= 2^-7 |c_or| + 2^-7 S_j, S_j = sum_i |P_ji e_i|.
    for kind, ref, res, P in (("K", ac.coefK, ac.resK, li.PK), ("V", ac.coefV, ac.resV, li.PV)):
        got = unpack(host(cache.coef_k if kind == "K" else cache.coef_v), srank, sidx, chunk_off, N, kind)
        ea = np.abs(res.astype(np.float64))
        S = np.stack([ea[:, g, :] @ np.abs(P[g].astype(np.float64)).T for g in range(shape.G)], axis=1)
        err = np.abs(got - ref)
        ok = err <= 2.0 ** -7 * np.abs(ref) + 2.0 ** -7 * S
        say(f"  {kind}: beyond-bound {int((~ok).sum())}, identical {float((err == 0).mean()):.4f}, "
            f"max err / S_j {float((err / np.maximum(S, 1e-30)).max()):.3e}")
        assert ok.all()


def decode_err(o_gpu, o_or):
    return max(np.abs(o_gpu[h] - o_or[h]).max() / np.abs(o_or[h]).max() for h in range(o_or.shape[0]))


@pytest.mark.parametrize("name,nq", [("llama_8k", 1), ("qwen_16k", 1), ("llama_ragged", 4)])
def test_anchor_decode(vr, oracle_lib, name, nq):
    """Decode over the residual-coded cache (anchor-mean score terms, anchor value weights
    merged by log-sum-exp) against the oracle's reconstruct-in-place decode, the cache built
    from the oracle's salience and nearest anchors."""
    import torch
    cfg, li, ac, shape, cache, PK, PV = encode_with_oracle_inputs(vr, oracle_lib, name, n_queries=nq)
    out = host(vr.decode(shape, [cache], dev(li.q, torch.bfloat16), PK, PV))
    torch.cuda.synchronize()
    worst = max(decode_err(out[i], oracle_lib.decode_anchor(ac, li.PK, li.PV, li.q[i], cfg["H"])) for i in range(nq))
    say(f"[anchor decode] {name} queries={nq}: worst rel err {worst:.3e}")
    assert worst <= DEC_TOL_BF16


def test_anchor_decode_multi_sequence_appended_and_quantised(vr, oracle_lib):
    """S = 3 sequences x Q = 5 queries (two row tiles), two tokens appended after compression,
    then the same caches with 4-bit coefficient codes."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k"])
    cfg.update(n=1300, G=2, H=8, seed=277)
    shape = vr.Shape(n=1300, G=2, H=8, w=32, r_min=16, kappa_pct=30, dtype="bf16", anchor_stride=DELTA)
    Q, extra = 5, 2
    caches, acs, qs, lis = [], [], [], []
    for s in range(3):
        li = make_layer(cfg, seq=s, n_queries=Q, n=1300 + extra)
        Kc, Vc = li.K[:1300], li.V[:1300]
        ac = oracle_lib.compress_anchor(Kc, Vc, li.Qw, li.PK, li.PV, 8, 30, 16, "bf16", delta=DELTA)
        PK, PV = dev(li.PK, torch.float32), dev(li.PV, torch.float32)
        cache = vr.anchor_encode(shape, dev(Kc, torch.bfloat16), dev(Vc, torch.bfloat16), dev(ac.sbar, torch.float32),
                                 dev(ac.nn.astype(np.int16), torch.int16), PK, PV, cap=32 + extra)
        for e in range(extra):
            vr.append_exact(shape, cache, dev(li.K[1300 + e], torch.bfloat16), dev(li.V[1300 + e], torch.bfloat16))
        caches.append(cache)
        acs.append(ac)
        qs.append(li.q)
        lis.append(li)
    q = dev(np.stack(qs), torch.bfloat16)
    out = host(vr.decode(shape, caches, q, PK, PV))
    qcs = [vr.quantize(shape, c, 4) for c in caches]
    outq = host(vr.decode_q(shape, caches, qcs, q, PK, PV))
    torch.cuda.synchronize()
    worst = worst_q = 0.0
    for s in range(3):
        li, ac = lis[s], acs[s]
        Kx = np.concatenate([ac.Kx, li.K[1300:]])
        Vx = np.concatenate([ac.Vx, li.V[1300:]])
        qk = oracle_lib.quantize(ac.coefK, ac.alloc.rank, 4)
        qv = oracle_lib.quantize(ac.coefV, ac.alloc.rank, 4)
        import dataclasses
        acq = dataclasses.replace(ac, coefK=qk.deq, coefV=qv.deq)
        for i in range(Q):
            worst = max(worst, decode_err(out[s][i], oracle_lib.decode_anchor(ac, li.PK, li.PV, li.q[i], 8, Kx, Vx)))
            worst_q = max(worst_q, decode_err(outq[s][i], oracle_lib.decode_anchor(acq, li.PK, li.PV, li.q[i], 8, Kx, Vx)))
    say(f"[anchor decode multi] worst rel err {worst:.3e}; 4-bit codes {worst_q:.3e}")
    assert worst <= DEC_TOL_BF16 and worst_q <= DEC_TOL_BF16


@pytest.mark.parametrize("name", ["llama_8k", "qwen_16k"])
def test_anchor_end_to_end(vr, oracle_lib, name):
    """GPU compress of the residual codec (salience, anchor search, encode) and decode, against
    the oracle's own pipeline, fully independent."""
    import torch
    cfg, li, ac, shape = prepared(vr, oracle_lib, name, n_queries=2)
    PK, PV = dev(li.PK, torch.float32), dev(li.PV, torch.float32)
    sb = torch.empty(shape.n - shape.w, dtype=torch.float32, device="cuda")
    cache = vr.compress(shape, dev(li.K, torch.bfloat16), dev(li.V, torch.bfloat16), dev(li.Qw, torch.bfloat16),
                        PK, PV, sbar_out=sb)
    out = host(vr.decode(shape, [cache], dev(li.q, torch.bfloat16), PK, PV))
    torch.cuda.synchronize()
    from test_gpu_parity import check_salience
    check_salience(host(sb), ac.sbar, f"anchor {name}")
    mism = int((host(cache.rank).astype(np.int64) != ac.alloc.rank).sum())
    worst = max(decode_err(out[i], oracle_lib.decode_anchor(ac, li.PK, li.PV, li.q[i], cfg["H"])) for i in range(2))
    say(f"[anchor end-to-end] {name}: rank mismatches {mism} of {shape.N}; worst decode rel err {worst:.3e}")
    assert mism <= max(8, shape.N // 1000)
    assert worst <= DEC_TOL_BF16
