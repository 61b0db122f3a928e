"""GPU parity of the group-wise b-bit coefficient quantiser and of decode over quantised
coefficients (Sec. 3.3 "Composability"), through the C ABI, against the fp64 CPU oracle.

* Codes and binary16 scales are integer/bit results: given the same stored coefficients
  (the oracle's, packed into the layer's layout here) they must match the oracle exactly.
* Decode over quantised coefficients is compared with the oracle's reconstruct-in-place
  decode of the dequantised coefficients, within 2e-2 of max |o| per (sequence, query, head).
* End to end (GPU compress -> quantise -> decode against the oracle's own pipeline) the same
  decode bound holds."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

DEC_TOL_BF16 = 2e-2


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


def pack(coef, srank, sidx, chunk_off, N, kind, stride):
    """[N][G][d] coefficients (bf16 values) -> the layer's [G][stride] tile-rectangle stream."""
    import torch
    G = coef.shape[1]
    out = np.zeros((G, stride), np.float32)
    for c in range((N + 255) // 256):
        t0, T = c * 256, min(256, N - c * 256)
        base = int(chunk_off[c])
        for h in range(16):
            if 16 * h >= T:
                break
            m = int(srank[t0 + 16 * h])
            blk = np.zeros((G, 16, m), np.float32)
            for i in range(16):
                if 16 * h + i < T:
                    slot = t0 + 16 * h + i
                    r = int(srank[slot])
                    blk[:, i, :r] = coef[sidx[slot], :, :r]
            flat = blk.reshape(G, 16 * m) if kind == "K" else blk.transpose(0, 2, 1).reshape(G, 16 * m)
            out[:, base:base + 16 * m] = flat
            base += 16 * m
    return torch.from_numpy(out).to(torch.bfloat16)


def q_tile_bytes(m, b):
    return 0 if m == 0 else 2 * ((m + 7) // 8 * 8) * b + 32 * ((m + 31) // 32)


def unpack_codes(stream, qchunk_off, srank, sidx, N, kind, b):
    """GPU code stream [G][q_stride] bytes -> codes [N][G][128] int, scales [N][G][4] fp32."""
    G = stream.shape[0]
    codes = np.zeros((N, G, 128), np.int64)
    scales = np.zeros((N, G, 4), np.float32)
    for c in range((N + 255) // 256):
        t0, T = c * 256, min(256, N - c * 256)
        base = int(qchunk_off[c])
        for h in range(16):
            if 16 * h >= T:
                break
            m = int(srank[t0 + 16 * h])
            mq, ks = (m + 7) // 8 * 8, (m + 31) // 32
            nb = 2 * mq * b
            raw = stream[:, base:base + nb]
            bits = np.unpackbits(raw, axis=1, bitorder="little").reshape(G, 16 * mq, b)
            val = (bits * (1 << np.arange(b))).sum(axis=-1)
            val = np.where(val >= (1 << (b - 1)), val - (1 << b), val)
            val = val.reshape(G, 16, mq) if kind == "K" else val.reshape(G, mq, 16).transpose(0, 2, 1)
            sc = stream[:, base + nb:base + nb + 32 * ks].copy().view(np.float16).astype(np.float32)
            sc = sc.reshape(G, ks, 16)
            for i in range(16):
                if 16 * h + i >= T:
                    assert np.all(val[:, i] == 0) and np.all(sc[:, :, i] == 0), (kind, c, h, i)
                    continue
                slot = t0 + 16 * h + i
                r = int(srank[slot])
                assert np.all(val[:, i, r:] == 0), (kind, c, h, i)
                codes[sidx[slot], :, :mq] = val[:, i]
                scales[sidx[slot], :, :ks] = sc[:, :, i]
            base += q_tile_bytes(m, b)
        assert base == int(qchunk_off[c + 1])
    return codes, scales


_CASES = {}


def prepared(vr, oracle_lib, name, n=None, G=None, H=None, n_queries=1):
    """Oracle compress of a bf16 layer, and a GPU cache holding the oracle's own stored
    coefficients (ranks from the GPU allocation on the oracle's pooled salience, which is
    bit-exact; the coefficient streams packed from the oracle's values)."""
    import torch
    from workloads import CONFIGS, make_layer
    key = (name, n, G, H, n_queries)
    if key in _CASES:
        return _CASES[key]
    cfg = dict(CONFIGS[name])
    if n is not None:
        cfg.update(n=n, G=G, H=H, seed=1000 + n)
    li = make_layer(cfg, n_queries=n_queries)
    oc = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], cfg["kappa"], cfg["r_min"], "bf16")
    shape = vr.Shape(n=cfg["n"], G=cfg["G"], H=cfg["H"], w=cfg["w"], r_min=cfg["r_min"],
                     kappa_pct=cfg["kappa"], dtype="bf16")
    PK, PV = dev(li.PK, torch.float32), dev(li.PV, torch.float32)
    cache = vr.new_cache(shape)
    vr.allocate(shape, dev(oc.sbar, torch.float32), cache)
    vr.project(shape, dev(li.K, torch.bfloat16), dev(li.V, torch.bfloat16), PK, PV, cache)
    torch.cuda.synchronize()
    N = shape.N
    rank = oc.alloc.rank.astype(np.int64)
    assert np.array_equal(cache.rank.cpu().numpy().astype(np.int64), rank)
    srank, sidx, chunk_off = layout(rank, N)
    cache.coef_k.copy_(pack(oc.coefK, srank, sidx, chunk_off, N, "K", cache.coef_stride).cuda())
    cache.coef_v.copy_(pack(oc.coefV, srank, sidx, chunk_off, N, "V", cache.coef_stride).cuda())
    torch.cuda.synchronize()
    _CASES[key] = (cfg, li, oc, shape, cache, PK, PV, (srank, sidx, chunk_off))
    return _CASES[key]


QCASES = [("llama_32k", None, None, None), ("ragged", 1300, 2, 8)]


@pytest.mark.parametrize("bits", [3, 4, 8])
@pytest.mark.parametrize("case", QCASES, ids=lambda c: c[0])
def test_codes_and_scales_bit_exact(vr, oracle_lib, case, bits):
    import torch
    name, n, G, H = case
    cfg, li, oc, shape, cache, PK, PV, (srank, sidx, _) = prepared(vr, oracle_lib, "llama_32k" if name == "ragged" else name, n, G, H)
    say(f"[quantise] {name} bits={bits}")
    qc = vr.quantize(shape, cache, bits)
    torch.cuda.synchronize()
    N = shape.N
    qoff = qc.qchunk_off.cpu().numpy().astype(np.int64)
    want_off = np.zeros_like(qoff)
    for c in range(len(qoff) - 1):
        want_off[c + 1] = want_off[c] + sum(q_tile_bytes(int(srank[i]), bits)
                                             for i in range(c * 256, min(N, c * 256 + 256), 16))
    assert np.array_equal(qoff, want_off)
    rank = oc.alloc.rank
    for kind, coef, stream in (("K", oc.coefK, qc.code_k), ("V", oc.coefV, qc.code_v)):
        want = oracle_lib.quantize(coef, rank, bits)
        codes, scales = unpack_codes(stream.cpu().numpy(), qoff, srank, sidx, N, kind, bits)
        mism_c = int((codes != want.codes).sum())
        mism_s = int((scales != want.scales).sum())
        say(f"  {kind}: code mismatches {mism_c} of {codes.size}, scale mismatches {mism_s}")
        assert mism_c == 0 and mism_s == 0


def decode_err(o_gpu, o_or):
    return max(np.abs(o_gpu[h] - o_or[h]).max() / np.abs(o_or[h]).max() for h in range(o_or.shape[0]))


@pytest.mark.parametrize("bits", [3, 4, 8])
@pytest.mark.parametrize("nq", [1, 4])
def test_decode_over_codes(vr, oracle_lib, bits, nq):
    """Quantised decode of the Llama-shaped 32K layer (4 and 16 query rows per KV head)
    against the oracle's decode of the dequantised coefficients, same codes."""
    import torch
    cfg, li, oc, shape, cache, PK, PV, _ = prepared(vr, oracle_lib, "llama_32k", n_queries=4)
    qc = vr.quantize(shape, cache, bits)
    q = li.q[:nq]
    out = vr.decode_q(shape, [cache], [qc], dev(q, torch.bfloat16), PK, PV)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy()
    qk = oracle_lib.quantize(oc.coefK, oc.alloc.rank, bits)
    qv = oracle_lib.quantize(oc.coefV, oc.alloc.rank, bits)
    worst = 0.0
    for i in range(nq):
        ref = oracle_lib.decode(qk.deq, qv.deq, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV, q[i], cfg["H"])
        worst = max(worst, decode_err(o[i], ref))
    say(f"[decode q] bits={bits} queries={nq}: worst rel err {worst:.3e}")
    assert worst <= DEC_TOL_BF16


def test_decode_over_codes_multi_sequence_appended(vr, oracle_lib):
    """S = 3 sequences, Q = 5 queries (20 rows: two row tiles), a ragged last chunk, two
    exact tokens appended after compression, 4-bit codes, every sequence against the oracle."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k"])
    cfg.update(n=1300, G=2, H=8, seed=177)
    shape = vr.Shape(n=1300, G=2, H=8, w=32, r_min=16, kappa_pct=20, dtype="bf16")
    Q, extra, bits = 5, 2, 4
    caches, qcs, qs, refs = [], [], [], []
    for s in range(3):
        li = make_layer(cfg, seq=s, n_queries=Q, n=1300 + extra)
        Kc, Vc = li.K[:1300], li.V[:1300]
        oc = oracle_lib.compress(Kc, Vc, li.Qw, li.PK, li.PV, 8, 20, 16, "bf16")
        PK, PV = dev(li.PK, torch.float32), dev(li.PV, torch.float32)
        cache = vr.new_cache(shape, cap=32 + extra)
        vr.allocate(shape, dev(oc.sbar, torch.float32), cache)
        vr.project(shape, dev(Kc, torch.bfloat16), dev(Vc, torch.bfloat16), PK, PV, cache)
        torch.cuda.synchronize()
        srank, sidx, chunk_off = layout(oc.alloc.rank.astype(np.int64), shape.N)
        cache.coef_k.copy_(pack(oc.coefK, srank, sidx, chunk_off, shape.N, "K", cache.coef_stride).cuda())
        cache.coef_v.copy_(pack(oc.coefV, srank, sidx, chunk_off, shape.N, "V", cache.coef_stride).cuda())
        for e in range(extra):
            vr.append_exact(shape, cache, dev(li.K[1300 + e], torch.bfloat16), dev(li.V[1300 + e], torch.bfloat16))
        qcs.append(vr.quantize(shape, cache, bits))
        caches.append(cache)
        qs.append(li.q)
        qk = oracle_lib.quantize(oc.coefK, oc.alloc.rank, bits)
        qv = oracle_lib.quantize(oc.coefV, oc.alloc.rank, bits)
        Kx = np.concatenate([oc.Kx, li.K[1300:]])
        Vx = np.concatenate([oc.Vx, li.V[1300:]])
        refs.append([oracle_lib.decode(qk.deq, qv.deq, oc.alloc.rank, Kx, Vx, li.PK, li.PV, li.q[i], 8)
                     for i in range(Q)])
    out = vr.decode_q(shape, caches, qcs, dev(np.stack(qs), torch.bfloat16), PK, PV)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy()
    worst = max(decode_err(o[s][i], refs[s][i]) for s in range(3) for i in range(Q))
    say(f"[decode q multi] worst rel err {worst:.3e}")
    assert worst <= DEC_TOL_BF16


@pytest.mark.parametrize("bits", [3, 4])
def test_quantised_end_to_end(vr, oracle_lib, bits):
    """GPU compress -> GPU quantise -> GPU decode against the oracle's compress -> quantise
    -> decode, fully independent (Llama-shaped 32K layer, two queries)."""
    import torch
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["llama_32k"]
    li = make_layer(cfg, n_queries=2)
    shape = vr.Shape(n=cfg["n"], G=cfg["G"], H=cfg["H"], w=cfg["w"], r_min=cfg["r_min"],
                     kappa_pct=cfg["kappa"], dtype="bf16")
    PK, PV = dev(li.PK, torch.float32), dev(li.PV, torch.float32)
    cache = vr.compress(shape, dev(li.K, torch.bfloat16), dev(li.V, torch.bfloat16), dev(li.Qw, torch.bfloat16), PK, PV)
    qc = vr.quantize(shape, cache, bits)
    out = vr.decode_q(shape, [cache], [qc], dev(li.q, torch.bfloat16), PK, PV)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy()
    oc = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, cfg["H"], cfg["kappa"], cfg["r_min"], "bf16")
    qk = oracle_lib.quantize(oc.coefK, oc.alloc.rank, bits)
    qv = oracle_lib.quantize(oc.coefV, oc.alloc.rank, bits)
    worst = max(decode_err(o[i], oracle_lib.decode(qk.deq, qv.deq, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV,
                                                   li.q[i], cfg["H"])) for i in range(2))
    say(f"[quantised end-to-end] bits={bits}: worst rel err {worst:.3e}")
    assert worst <= DEC_TOL_BF16
