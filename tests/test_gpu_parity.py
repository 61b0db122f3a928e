"""GPU parity of the HIP codec (through the C ABI) against the fp64 CPU oracle.

Tolerances (from the workload definition): ranks, offsets and layout bit-exact given the
same fp32 pooled salience; salience within 1e-3 relative (entries below 1e-6 of the max are
an underflow floor, reported separately); decode within 2e-2 of max |o| per (sequence,
query, head) in bf16.  The fp32 tiny workload is also held to a tighter decode bound."""
import math
import os
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

SAL_RTOL = 1e-3
DEC_TOL_BF16 = 2e-2
DEC_TOL_F32 = 1e-4


def say(*a):
    """Progress and observed errors: stderr, and appended to the file named by
    VARRATE_PARITY_LOG when that variable is set (so a run keeps its measured errors)."""
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


def shape_of(vr, cfg, n=None, kappa=None, r_min=None, w=None):
    return vr.Shape(n=cfg["n"] if n is None else n, G=cfg["G"], H=cfg["H"], w=cfg["w"] if w is None else w,
                    r_min=cfg["r_min"] if r_min is None else r_min,
                    kappa_pct=cfg["kappa"] if kappa is None else kappa, dtype=cfg["dtype"])


def expected_layout(rank, N):
    """Storage order and chunk offsets of the tile-rectangle layout (the header's contract):
    chunks of 256 tokens stored by (rank descending, index ascending); tile h of a chunk (its
    stored slots 16h .. 16h + 15) takes 16 * m_h elements, m_h = its first slot's rank."""
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


def unpack(coef, srank, sidx, chunk_off, N, kind, d=128):
    """GPU streams [G][stride] -> [N][G][d] (zeros past each rank).  Tile h of chunk c sits at
    chunk_off[c] + 16 * (sum of the chunk's earlier tile maxima): for K, 16 rows of m_h
    coordinates; for V, m_h coordinate rows of 16 slots.  Asserts that every element past a
    slot's rank (and every element of an absent slot) is zero."""
    G = coef.shape[0]
    out = np.zeros((N, G, d), np.float32)
    nch = (N + 255) // 256
    for c in range(nch):
        t0 = c * 256
        T = min(256, N - t0)
        base = int(chunk_off[c])
        for h in range(16):
            if 16 * h >= T:
                break
            m = int(srank[t0 + 16 * h])
            blk = coef[:, base:base + 16 * m].astype(np.float32)
            blk = blk.reshape(G, 16, m) if kind == "K" else blk.reshape(G, m, 16).transpose(0, 2, 1)
            for i in range(16):
                slot = t0 + 16 * h + i
                r = int(srank[slot]) if 16 * h + i < T else 0
                assert np.all(blk[:, i, r:] == 0), (kind, c, h, i)
                if r:
                    out[sidx[slot], :, :r] = blk[:, i, :r]
            base += 16 * m
        assert base == chunk_off[c + 1]
    return out


def rel_err(got, ref):
    return np.abs(got - ref).max() / max(np.abs(ref).max(), 1e-30)


def decode_err(o_gpu, o_or):
    """max over heads of ||d||_inf / ||o||_inf."""
    return max(np.abs(o_gpu[h] - o_or[h]).max() / np.abs(o_or[h]).max() for h in range(o_or.shape[0]))


_LAYERS = {}


def layer(name, **kw):
    from workloads import CONFIGS, make_layer
    key = (name, tuple(sorted(kw.items())))
    if key not in _LAYERS:
        _LAYERS[key] = make_layer(CONFIGS[name], **kw)
    return _LAYERS[key]


_ORACLE = {}


def oracle_compress(oracle_lib, name, li, kappa, r_min, sbar=None, tag=""):
    from workloads import CONFIGS
    cfg = CONFIGS[name]
    key = (name, kappa, r_min, tag)
    if key not in _ORACLE:
        _ORACLE[key] = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], kappa, r_min,
                                           cfg["dtype"], sbar=sbar)
    return _ORACLE[key]


def gpu_compress(vr, shape, li, sbar=None, cap=None):
    import torch
    dt = shape.torch_dtype
    K, V, Qw = dev(li.K, dt), dev(li.V, dt), dev(li.Qw, dt)
    PK, PV = dev(li.PK, torch.float32), dev(li.PV, torch.float32)
    if sbar is None:
        sb = torch.empty(shape.N, dtype=torch.float32, device="cuda")
        cache = vr.compress(shape, K, V, Qw, PK, PV, cap=cap, sbar_out=sb)
    else:
        sb = dev(sbar, torch.float32)
        cache = vr.new_cache(shape, cap)
        vr.allocate(shape, sb, cache)
        vr.project(shape, K, V, PK, PV, cache)
    torch.cuda.synchronize()
    return cache, sb, PK, PV


# ---------------------------------------------------------------------------------------
def check_salience(got, want, label):
    """Elementwise relative error <= SAL_RTOL on entries at or above 1e-6 of the largest
    (the underflow floor); below it the absolute error stays under SAL_RTOL x the floor."""
    g = np.asarray(got, np.float64)
    o = np.asarray(want, np.float64)
    floor = 1e-6 * o.max()
    big = o >= floor
    rel = np.abs(g[big] - o[big]) / o[big]
    small = np.abs(g[~big] - o[~big]).max() if (~big).any() else 0.0
    say(f"  {label}: salience max rel {rel.max():.3e} over {big.sum()} entries; "
        f"{(~big).sum()} below floor, max abs there {small:.3e}")
    assert rel.max() <= SAL_RTOL, label
    assert small <= SAL_RTOL * floor, label


# Window rows per KV head ((H/G) w): tiny 64, llama 128, qwen 224 (the second row tile of
# waves 0-5), and a small synthetic layer at the 256-row maximum.
SALIENCE_CASES = {
    "tiny": None,
    "llama_32k": None,
    "qwen_16k_stack": None,
    "rows256": dict(base="llama_32k", n=3000, G=1, H=8, w=32, seed=31),
}


@pytest.mark.parametrize("name", list(SALIENCE_CASES))
def test_salience_parity(vr, oracle_lib, name):
    from workloads import CONFIGS, make_layer
    over = SALIENCE_CASES[name]
    if over is None:
        cfg = CONFIGS[name]
        li = layer(name)
    else:
        cfg = dict(CONFIGS[over["base"]])
        cfg.update({k: v for k, v in over.items() if k != "base"})
        li = make_layer(cfg)
    say(f"[salience] {name}: n={cfg['n']} G={cfg['G']} H={cfg['H']} w={cfg['w']} "
        f"({cfg['H'] // cfg['G'] * cfg['w']} window rows per KV head)")
    sbar_or = oracle_lib.pool(oracle_lib.salience(li.K, li.Qw, cfg["H"]))
    shape = shape_of(vr, cfg)
    _, sb, _, _ = gpu_compress(vr, shape, li)
    check_salience(host(sb), sbar_or, name)
    # the salience entry point alone (pooling launch) gives the same bits as compress
    import torch
    sb2 = vr.salience(shape, dev(li.K, shape.torch_dtype), dev(li.Qw, shape.torch_dtype))
    torch.cuda.synchronize()
    assert np.array_equal(host(sb2), host(sb)), name


def sbar_cases(N, oracle_sbar):
    rng = np.random.default_rng(123)
    cases = {
        "oracle": oracle_sbar,
        "constant": np.full(N, 0.37, np.float32),
        "ties": rng.integers(0, 4, N).astype(np.float32) / 7,
        # about N/24 and N/160 tokens per weight: the threshold's digit bucket then holds
        # several hundred to a few thousand candidates (the LDS narrowing, and the direct
        # ranking with one slice per candidate)
        "ties24": rng.integers(0, 24, N).astype(np.float32) / 23,
        "ties160": rng.integers(0, 160, N).astype(np.float32) / 159,
        "one_hot": np.where(np.arange(N) == N // 3, 1.0, 0.0).astype(np.float32),
        "random": rng.random(N).astype(np.float32),
        "spiky": (rng.random(N) ** 12).astype(np.float32),
    }
    return cases


@pytest.mark.parametrize("name,kappa,r_min", [("tiny", 20, 16), ("tiny", 13, 0), ("tiny", 100, 16),
                                              ("llama_32k", 20, 16), ("llama_32k", 10, 8),
                                              ("llama_32k", 40, 16), ("llama_32k", 13, 16)])
def test_allocation_bit_exact(vr, oracle_lib, name, kappa, r_min):
    from workloads import CONFIGS
    cfg = CONFIGS[name]
    li = layer(name)
    base = oracle_compress(oracle_lib, name, li, cfg["kappa"], cfg["r_min"])
    N = cfg["n"] - cfg["w"]
    shape = shape_of(vr, cfg, kappa=kappa, r_min=r_min)
    B = oracle_lib.budget(cfg["n"], 128, cfg["w"], kappa)
    import torch
    for case, sb in sbar_cases(N, base.sbar).items():
        say(f"[allocate] {name} kappa={kappa} r_min={r_min} case={case}")
        want = oracle_lib.allocate(oracle_lib.weights(sb), B, r_min, 128).rank
        cache = vr.new_cache(shape)
        vr.allocate(shape, dev(sb, torch.float32), cache)
        torch.cuda.synchronize()
        got = host(cache.rank).astype(np.int64)
        mism = int((got != want).sum())
        assert mism == 0, f"{case}: {mism} rank mismatches"
        srank, sidx, chunk_off = expected_layout(want.astype(np.int64), N)
        assert np.array_equal(host(cache.chunk_off).astype(np.int64), chunk_off), case
        assert np.array_equal(host(cache.srank).astype(np.int64), srank), case
        assert np.array_equal(host(cache.sidx).astype(np.int64), sidx), case
        assert cache.B == B and got.sum() == B


@pytest.mark.parametrize("n,kappa,r_min", [(40000, 20, 16), (40000, 10, 8), (32800, 40, 16)])
def test_allocation_bit_exact_grid_passes(vr, oracle_lib, n, kappa, r_min):
    """Coded lengths other than the workloads' (39968 tokens: 40 workgroups of 1024 with a
    ragged last one; 32768: exactly 32): the synthetic sbar cases, ranks, storage order and
    chunk table bit-exact against the oracle."""
    import torch
    from workloads import CONFIGS
    cfg = CONFIGS["llama_32k"]
    N = n - cfg["w"]
    shape = shape_of(vr, cfg, n=n, kappa=kappa, r_min=r_min)
    B = oracle_lib.budget(n, 128, cfg["w"], kappa)
    for case, sb in sbar_cases(N, None).items():
        if sb is None:
            continue
        say(f"[allocate] n={n} kappa={kappa} r_min={r_min} case={case}")
        want = oracle_lib.allocate(oracle_lib.weights(sb), B, r_min, 128).rank
        cache = vr.new_cache(shape)
        vr.allocate(shape, dev(sb, torch.float32), cache)
        torch.cuda.synchronize()
        got = host(cache.rank).astype(np.int64)
        mism = int((got != want).sum())
        assert mism == 0, f"{case}: {mism} rank mismatches"
        srank, sidx, chunk_off = expected_layout(want.astype(np.int64), N)
        assert np.array_equal(host(cache.chunk_off).astype(np.int64), chunk_off), case
        assert np.array_equal(host(cache.srank).astype(np.int64), srank), case
        assert np.array_equal(host(cache.sidx).astype(np.int64), sidx), case
        assert got.sum() == B


@pytest.mark.parametrize("name", ["tiny", "llama_32k"])
def test_layout_and_projection(vr, oracle_lib, name):
    from workloads import CONFIGS
    cfg = CONFIGS[name]
    say(f"[project] {name}")
    li = layer(name)
    oc = oracle_compress(oracle_lib, name, li, cfg["kappa"], cfg["r_min"])
    shape = shape_of(vr, cfg)
    cache, _, _, _ = gpu_compress(vr, shape, li, sbar=oc.sbar)
    N = shape.N
    rank = oc.alloc.rank.astype(np.int64)
    srank, sidx, chunk_off = expected_layout(rank, N)
    assert np.array_equal(host(cache.srank).astype(np.int64), srank)
    assert np.array_equal(host(cache.sidx).astype(np.int64), sidx)
    assert np.array_equal(host(cache.chunk_off).astype(np.int64), chunk_off)
    for kind, ref, X in (("K", oc.coefK, li.K), ("V", oc.coefV, li.V)):
        got = unpack(host(cache.coef_k if kind == "K" else cache.coef_v), srank, sidx, chunk_off, N, kind)
        err = np.abs(got - ref)
        # The kernel forms P x from bf16 hi + lo parts of P (x too when it is fp32): each
        # product is within 3 x 2^-18 |P_ji x_i| of exact (the dropped lo x lo term and the
        # two split residuals), and the fp32 MFMA accumulation of 128 such terms (12 rounded
        # accumulator updates at most, each <= 2^-24 of the running sum) adds under
        # 2^-19 sum_i |P_ji x_i|.  So |c_kernel - c| <= 2^-15 S_j with S_j = sum_i |P_ji x_i|
        # (<= ||x_t||, as basis rows have unit norm).  bf16 storage then rounds the kernel's
        # value, which lands at most one unit (<= 2^-7 |ref|) from the rounding of the exact
        # value.  A projection that dropped the basis lo part would err by up to 2^-9 S_j.
        G = X.shape[1]
        P = li.PK if kind == "K" else li.PV
        Xa = np.abs(X[:N].astype(np.float64))
        S = np.stack([Xa[:, g, :] @ np.abs(P[g].astype(np.float64)).T for g in range(G)], axis=1)
        if cfg["dtype"] == "bf16":
            ok = err <= np.abs(ref) * 2.0 ** -7 + 2.0 ** -15 * S
        else:
            ok = err <= np.abs(ref) * 2.0 ** -23 + 2.0 ** -15 * S
        frac = float((err / np.maximum(S, 1e-30)).max())
        say(f"  {kind}: max rel {rel_err(got, ref):.3e}, max err / S_j {frac:.3e}, beyond-bound "
            f"{int((~ok).sum())}, identical {float((err == 0).mean()):.4f}")
        assert ok.all()
    # exact window rows are copied verbatim
    w = shape.w
    assert np.array_equal(host(cache.k_exact)[:, :w].transpose(1, 0, 2), li.K[N:])
    assert np.array_equal(host(cache.v_exact)[:, :w].transpose(1, 0, 2), li.V[N:])
    assert cache.n_exact == w


@pytest.mark.parametrize("name", ["tiny", "llama_32k"])
def test_decode_parity_same_ranks(vr, oracle_lib, name):
    import torch
    from workloads import CONFIGS
    cfg = CONFIGS[name]
    say(f"[decode] {name}")
    li = layer(name, n_queries=2)
    oc = oracle_compress(oracle_lib, name, li, cfg["kappa"], cfg["r_min"], tag="q2")
    shape = shape_of(vr, cfg)
    cache, _, PK, PV = gpu_compress(vr, shape, li, sbar=oc.sbar)
    assert np.array_equal(host(cache.rank).astype(np.int64), oc.alloc.rank)
    q = dev(li.q, shape.torch_dtype)
    out = vr.decode(shape, [cache], q, PK, PV)
    torch.cuda.synchronize()
    o_gpu = host(out)
    tol = DEC_TOL_F32 if cfg["dtype"] == "f32" else DEC_TOL_BF16
    for i in range(li.q.shape[0]):
        o_or = oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV, li.q[i], cfg["H"])
        e = decode_err(o_gpu[i], o_or)
        say(f"  query {i}: decode max rel err {e:.3e}")
        assert e <= tol


@pytest.mark.parametrize("name,Q,law,check", [("llama_32k", 1, "aware", 1),       # 4 rows per KV head
                                                ("qwen_16k_stack", 1, "aware", 1),  # 7 rows
                                                ("llama_32k", 4, "aware", 4),       # 16 rows
                                                ("agnostic_32k", 64, "agnostic", 6)])  # 256 rows
def test_decode_row_tiles(vr, oracle_lib, name, Q, law, check):
    """Decode at full size in each query-row grouping the kernel has: row tiles of at most
    4 rows (four 16-position tiles per MFMA group), at most 8 (two), and 16-row tiles (one
    each; 16 row tiles for 64 queries).  `check` queries, spread over the batch, are compared
    with the oracle one by one."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS[name]
    say(f"[decode rows] {name} Q={Q} ({law})")
    li = make_layer(cfg, n_queries=Q, query_law=law)
    oc = oracle_compress(oracle_lib, name, li, cfg["kappa"], cfg["r_min"], tag=f"rows{Q}{law}")
    shape = shape_of(vr, cfg)
    cache, _, PK, PV = gpu_compress(vr, shape, li, sbar=oc.sbar)
    assert np.array_equal(host(cache.rank).astype(np.int64), oc.alloc.rank)
    out = host(vr.decode(shape, [cache], dev(li.q, shape.torch_dtype), PK, PV))
    torch.cuda.synchronize()
    worst = 0.0
    for i in np.linspace(0, Q - 1, check).astype(int):
        o_or = oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV, li.q[i], cfg["H"])
        worst = max(worst, decode_err(out[i], o_or))
    say(f"  worst decode rel err {worst:.3e} over {check} queries")
    assert worst <= DEC_TOL_BF16


def test_llama_128k_layer(vr, oracle_lib):
    """One layer of the Llama-3.1-8B-shaped 128K stack at full size (n = 131072, 8 KV x 32
    query heads): salience, bit-exact ranks on the oracle's pooled salience, and decode."""
    import torch
    from workloads import CONFIGS
    name = "llama_128k_stack"
    cfg = CONFIGS[name]
    say(f"[128k] drawing layer 0 (n={cfg['n']})")
    li = layer(name, n_queries=1)
    oc = oracle_compress(oracle_lib, name, li, cfg["kappa"], cfg["r_min"])
    shape = shape_of(vr, cfg)
    _, sb, _, _ = gpu_compress(vr, shape, li)
    g, o = host(sb).astype(np.float64), oc.sbar.astype(np.float64)
    big = o >= 1e-6 * o.max()
    sal = float((np.abs(g[big] - o[big]) / o[big]).max())
    cache, _, PK, PV = gpu_compress(vr, shape, li, sbar=oc.sbar)
    mism = int((host(cache.rank).astype(np.int64) != oc.alloc.rank).sum())
    out = host(vr.decode(shape, [cache], dev(li.q, shape.torch_dtype), PK, PV))
    torch.cuda.synchronize()
    o_or = oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV, li.q[0], cfg["H"])
    e = decode_err(out[0], o_or)
    say(f"  salience max rel {sal:.2e}; rank mismatches {mism}; decode err {e:.3e}")
    assert sal <= SAL_RTOL and mism == 0 and e <= DEC_TOL_BF16


def test_qwen_stack_batch8(vr, oracle_lib):
    """Qwen2.5-7B-shaped stack (4 KV x 28 query heads, n = 16384): the first and last of its
    28 layers for all 8 independent sequences, decoded as one batch of 8 caches per layer
    (7 query rows per KV head), every sequence against the oracle."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["qwen_16k_stack"]
    shape = shape_of(vr, cfg)
    for lyr in (0, cfg["layers"] - 1):
        caches, qs, refs = [], [], []
        for sq in range(cfg["batch"]):
            li = make_layer(cfg, layer=lyr, seq=sq, n_queries=1)
            oc = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], cfg["kappa"], cfg["r_min"], "bf16")
            cache, _, PK, PV = gpu_compress(vr, shape, li, sbar=oc.sbar)
            assert np.array_equal(host(cache.rank).astype(np.int64), oc.alloc.rank), (lyr, sq)
            caches.append(cache)
            qs.append(li.q)
            refs.append(oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV,
                                          li.q[0], cfg["H"]))
        out = host(vr.decode(shape, caches, dev(np.stack(qs), torch.bfloat16), PK, PV))
        torch.cuda.synchronize()
        worst = max(decode_err(out[sq][0], refs[sq]) for sq in range(cfg["batch"]))
        say(f"[qwen stack] layer {lyr}: worst decode err over {cfg['batch']} sequences {worst:.3e}")
        assert worst <= DEC_TOL_BF16


@pytest.mark.parametrize("name", ["tiny", "llama_32k"])
def test_end_to_end(vr, oracle_lib, name):
    """GPU salience feeds the GPU allocation; the oracle runs independently throughout."""
    import torch
    from workloads import CONFIGS
    cfg = CONFIGS[name]
    say(f"[end-to-end] {name}")
    li = layer(name, n_queries=2)
    oc = oracle_compress(oracle_lib, name, li, cfg["kappa"], cfg["r_min"], tag="q2")
    shape = shape_of(vr, cfg)
    cache, _, PK, PV = gpu_compress(vr, shape, li)
    mism = int((host(cache.rank).astype(np.int64) != oc.alloc.rank).sum())
    out = host(vr.decode(shape, [cache], dev(li.q, shape.torch_dtype), PK, PV))
    torch.cuda.synchronize()
    errs = []
    for i in range(li.q.shape[0]):
        o_or = oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV, li.q[i], cfg["H"])
        errs.append(decode_err(out[i], o_or))
    say(f"  rank mismatches {mism} of {shape.N}; decode max rel err {max(errs):.3e}")
    assert mism <= max(8, shape.N // 1000)
    assert max(errs) <= DEC_TOL_BF16


@pytest.mark.parametrize("Q", [8, 9, 13])
def test_decode_row_tile_pairs(vr, oracle_lib, Q):
    """Batches of query rows decode two row tiles per wave: Q = 8 (32 rows per KV head, one
    pair of full row tiles), 9 (36 rows: a pair, then a row tile whose partner is past the
    last) and 13 (52 rows: two pairs, the second one's partner holding 4 rows), two sequences;
    every query against the oracle."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k"])
    cfg.update(n=1300, G=2, H=8, seed=91)
    shape = vr.Shape(n=1300, G=2, H=8, w=32, r_min=16, kappa_pct=20, dtype="bf16")
    say(f"[row tile pairs] Q={Q}")
    caches, qs, refs = [], [], []
    for s in range(2):
        li = make_layer(cfg, seq=s, n_queries=Q, n=1300)
        oc = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, 8, 20, 16, "bf16")
        cache, _, PK, PV = gpu_compress(vr, shape, li, sbar=oc.sbar)
        caches.append(cache)
        qs.append(li.q)
        refs.append([oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV, li.q[i], 8)
                     for i in range(Q)])
    out = host(vr.decode(shape, caches, dev(np.stack(qs), torch.bfloat16), PK, PV))
    torch.cuda.synchronize()
    worst = max(decode_err(out[s][i], refs[s][i]) for s in range(2) for i in range(Q))
    say(f"  worst decode rel err {worst:.3e}")
    assert worst <= DEC_TOL_BF16


def test_decode_multi_sequence_many_queries_appended(vr, oracle_lib):
    """S = 3 independent sequences, Q = 5 queries each (20 query rows per KV head: two row
    tiles), ragged last chunk, and 3 exact tokens appended after compression."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k"])
    cfg.update(n=1300, G=2, H=8, seed=77)
    shape = vr.Shape(n=1300, G=2, H=8, w=32, r_min=16, kappa_pct=20, dtype="bf16")
    Q, extra = 5, 3
    caches, qs, refs = [], [], []
    for s in range(3):
        li = make_layer(cfg, seq=s, n_queries=Q, n=1300 + extra)
        Kc, Vc = li.K[:1300], li.V[:1300]
        oc = oracle_lib.compress(Kc, Vc, li.Qw, li.PK, li.PV, 8, 20, 16, "bf16")
        li2 = type(li)(Kc, Vc, li.Qw, li.q, li.PK, li.PV, li.planted, cfg)
        cache, _, PK, PV = gpu_compress(vr, shape, li2, sbar=oc.sbar, cap=32 + extra)
        for e in range(extra):
            vr.append_exact(shape, cache, dev(li.K[1300 + e], torch.bfloat16), dev(li.V[1300 + e], torch.bfloat16))
        caches.append(cache)
        qs.append(li.q)
        Kx = np.concatenate([oc.Kx, li.K[1300:]])
        Vx = np.concatenate([oc.Vx, li.V[1300:]])
        refs.append([oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, Kx, Vx, li.PK, li.PV, li.q[i], 8)
                     for i in range(Q)])
    q = dev(np.stack(qs), torch.bfloat16)
    out = host(vr.decode(shape, caches, q, PK, PV))
    torch.cuda.synchronize()
    worst = max(decode_err(out[s][i], refs[s][i]) for s in range(3) for i in range(Q))
    say(f"[multi] worst decode rel err {worst:.3e}")
    assert caches[0].n_exact == 32 + extra
    assert worst <= DEC_TOL_BF16


def test_decode_more_sequences_than_one_launch(vr, oracle_lib):
    """S = 20 sequences in one call: more than the 16 a launch carries, so the call splits
    into two launch pairs with their own records; every sequence against the oracle."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k"])
    cfg.update(n=700, G=2, H=8, seed=19)
    shape = vr.Shape(n=700, G=2, H=8, w=32, r_min=16, kappa_pct=25, dtype="bf16")
    caches, qs, refs = [], [], []
    for sq in range(20):
        li = make_layer(cfg, seq=sq, n_queries=1)
        oc = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, 8, 25, 16, "bf16")
        cache, _, PK, PV = gpu_compress(vr, shape, li, sbar=oc.sbar)
        caches.append(cache)
        qs.append(li.q)
        refs.append(oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV, li.q[0], 8))
    out = host(vr.decode(shape, caches, dev(np.stack(qs), torch.bfloat16), PK, PV))
    torch.cuda.synchronize()
    worst = max(decode_err(out[sq][0], refs[sq]) for sq in range(20))
    say(f"[20 sequences] worst decode rel err {worst:.3e}")
    assert worst <= DEC_TOL_BF16


@pytest.mark.parametrize("name", ["tiny", "qwen_16k_stack", "llama_32k"])
def test_compress_equals_the_three_entry_points(vr, name):
    """varrate_compress pools the salience inside the allocation's first pass; its outputs
    must equal those of varrate_salience -> varrate_allocate -> varrate_project bit for bit."""
    import torch
    from workloads import CONFIGS
    say(f"[compress = steps] {name}")
    li = layer(name)
    shape = shape_of(vr, CONFIGS[name])
    dt = shape.torch_dtype
    K, V, Qw = dev(li.K, dt), dev(li.V, dt), dev(li.Qw, dt)
    PK, PV = dev(li.PK, torch.float32), dev(li.PV, torch.float32)
    sb1 = vr.salience(shape, K, Qw)
    c1 = vr.new_cache(shape)
    vr.allocate(shape, sb1, c1)
    vr.project(shape, K, V, PK, PV, c1)
    sb2 = torch.empty(shape.N, dtype=torch.float32, device="cuda")
    c2 = vr.compress(shape, K, V, Qw, PK, PV, sbar_out=sb2)
    torch.cuda.synchronize()
    assert np.array_equal(host(sb1), host(sb2))
    for f in ("rank", "srank", "sidx", "chunk_off", "coef_k", "coef_v", "k_exact", "v_exact"):
        assert np.array_equal(host(getattr(c1, f)), host(getattr(c2, f))), f


@pytest.mark.parametrize("n,w,kappa,r_min", [(33, 32, 100, 16), (40, 32, 90, 0), (287, 32, 50, 16),
                                             (289, 32, 25, 4), (600, 1, 30, 16), (2080, 32, 100, 16)])
def test_ragged_and_degenerate(vr, oracle_lib, n, w, kappa, r_min):
    """One coded token, chunks of 255 / 1 tokens, window of 1, floor 0, full budget."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k"])
    cfg.update(n=n, w=w, G=2, H=4, seed=91)
    say(f"[ragged] n={n} w={w} kappa={kappa} r_min={r_min}")
    li = make_layer(cfg, n_queries=1)
    shape = vr.Shape(n=n, G=2, H=4, w=w, r_min=r_min, kappa_pct=kappa, dtype="bf16")
    B = oracle_lib.budget(n, 128, w, kappa)
    if B < (n - w) * r_min or B > (n - w) * 128:
        pytest.skip("infeasible budget for this shape")
    oc = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, 4, kappa, r_min, "bf16")
    cache, sb, PK, PV = gpu_compress(vr, shape, li)
    s = host(sb)
    got_rank = host(cache.rank).astype(np.int64)
    cache2, _, _, _ = gpu_compress(vr, shape, li, sbar=oc.sbar)
    assert np.array_equal(host(cache2.rank).astype(np.int64), oc.alloc.rank)
    out = host(vr.decode(shape, [cache2], dev(li.q, torch.bfloat16), PK, PV))
    torch.cuda.synchronize()
    o_or = oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV, li.q[0], 4)
    e = decode_err(out[0], o_or)
    mism = int((got_rank != oc.alloc.rank).sum())
    say(f"  decode err {e:.3e}; e2e rank mismatches {mism} of {n - w}")
    check_salience(s, oc.sbar, f"ragged n={n} w={w}")
    assert mism <= max(8, (n - w) // 1000)
    assert e <= DEC_TOL_BF16


def test_full_budget_is_attention(vr):
    """kappa = 100 keeps every token at full rank: decode equals attention over the bf16
    cache up to coefficient storage rounding."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k"])
    cfg.update(n=3000, G=2, H=8, seed=5)
    li = make_layer(cfg, n_queries=1)
    shape = vr.Shape(n=3000, G=2, H=8, w=32, r_min=16, kappa_pct=100, dtype="bf16")
    cache, _, PK, PV = gpu_compress(vr, shape, li)
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
    say(f"[full budget] err vs attention {e:.3e}")
    assert e <= DEC_TOL_BF16


def test_run_twice_bitwise_identical(vr):
    import torch
    li = layer("llama_32k", n_queries=2)
    from workloads import CONFIGS
    shape = shape_of(vr, CONFIGS["llama_32k"])
    outs = []
    for _ in range(2):
        cache, sb, PK, PV = gpu_compress(vr, shape, li)
        o = vr.decode(shape, [cache], dev(li.q, torch.bfloat16), PK, PV)
        torch.cuda.synchronize()
        outs.append((host(sb), host(cache.rank), host(cache.coef_k), host(cache.coef_v), host(o)))
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


def test_read_probe_runs_clean(vr):
    """The measurement probe reads the bytes it is given and leaves the sink alone (the fold
    of an all-ones buffer is zero, never the sink's trigger value); errors come back as codes."""
    import torch
    say("read probe: 1 MiB + ragged 48 B tail")
    buf = torch.ones(((1 << 20) + 48) // 4, dtype=torch.int32, device="cuda")
    sink = torch.zeros(vr.PROBE_WGS, dtype=torch.int32, device="cuda")
    vr.read_probe(buf, (1 << 20) + 48, sink)
    vr.read_probe(buf, 16, sink)
    torch.cuda.synchronize()
    assert int(sink.abs().sum()) == 0
    with pytest.raises(vr.VarRateError):
        vr.read_probe(buf[1:], 16, sink)          # misaligned source
    with pytest.raises(vr.VarRateError):
        vr.read_probe(buf, 4 * buf.numel() + 16, sink)
