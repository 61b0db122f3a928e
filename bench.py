"""Benchmark of the variable-rank KV codec's hot path on one MI355X.

A step is one pass of the whole path over one synthetic layer of the Llama-3.1-8B-shaped
workload (8 KV heads x 32 query heads, d 128, 32768 cached tokens, bf16, budget 20%,
floor 16, window 32): salience -> allocation -> projection (compress), then one decode
query in rank space.  Inputs are device-resident before timing.  To keep the 256 MB
Infinity Cache from serving repeated reads, steps rotate over several copies of the
layer's K/V (compress reads) and over many cache slots: a step decodes the slot that
was compressed half a rotation earlier, so decode never reads what it just wrote.

Timed launches are replayed from captured HIP graphs (one per stage, one for whole
steps), so the GPU is never waiting on host-side Python between launches.

Prints one JSON line.  `value` is the decode attention throughput (algorithmic decode
bytes / average decode launch time); compress time per 32K tokens, per-stage times, the
decode kernel's roofline and the CPU oracle baseline are reported beside it.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
N_INPUT_COPIES = 4             # 4 x 134 MB of K/V (537 MB > the 256 MB Infinity Cache)
N_CACHE_SLOTS = 24             # 24 x 28 MB of compressed caches


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=48)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="llama_32k",
                    choices=("llama_32k", "llama_128k_stack", "qwen_16k_stack", "agnostic_32k"),
                    help="llama_32k: the headline layer (default).  The others are the model-stack "
                         "and query-agnostic workloads, reported in their own JSON line")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-stack", action="store_true",
                    help="default run only: skip the 32-layer 128K stack that the line also reports")
    ap.add_argument("--mode", choices=("bench", "pmc"), default="bench",
                    help="pmc: a short run for hardware-counter passes (eager decodes on distinct "
                         "cache slots, then plain 64 MiB device copies that calibrate the byte counters; "
                         "with --config agnostic_32k: eight eager batch-64 decodes of the 20%% cache)")
    return ap.parse_args()


def decode_bytes(shape, cache, n_queries=1):
    """Algorithmic bytes one decode must move: packed coefficients, exact slots, the stored
    ranks and chunk offsets, both fp32 bases, queries and outputs."""
    es = 2 if shape.dtype == "bf16" else 4
    G, H, d = shape.G, shape.H, 128
    coef = 2 * G * cache.B * es
    exact = 2 * G * cache.n_exact * d * es
    meta = cache.N + (cache.chunk_off.numel()) * 4
    bases = 2 * G * d * d * 4
    qo = 2 * n_queries * H * d * es
    return coef + exact + meta + bases + qo


def decode_bytes_q(shape, cache, bits, rank, n_queries=1):
    """Algorithmic bytes of a decode over b-bit codes: the codes of every coefficient, one
    binary16 scale per 32-coordinate group, plus what decode_bytes counts besides the
    coefficients (exact slots, ranks and chunk offsets, bases, queries and outputs)."""
    es = 2
    groups = int(((rank.astype(np.int64) + 31) // 32).sum())
    codes = 2 * shape.G * (cache.B * bits // 8 + 2 * groups)
    return decode_bytes(shape, cache, n_queries) - 2 * shape.G * cache.B * es + codes


def footprint_pct(shape, cache, coef_bytes):
    """Stored bytes of the compressed layer (coefficients or codes + scales, exact rows,
    ranks) as a percentage of the full bf16 K/V cache."""
    full = 2 * shape.n * shape.G * 128 * 2
    exact = 2 * shape.G * shape.w * 128 * 2
    return 100.0 * (coef_bytes + exact + cache.N) / full


def compress_bytes(shape, cache):
    """Minimum bytes of one compress: K and V read once, window queries and bases read,
    packed coefficients, ranks, layout tables and exact rows written."""
    es = 2 if shape.dtype == "bf16" else 4
    G, H, d, n, w = shape.G, shape.H, 128, shape.n, shape.w
    read = 2 * n * G * d * es + w * H * d * es + 2 * G * d * d * 4
    write = 2 * G * cache.B * es + 2 * G * w * d * es + cache.N * (1 + 1 + 4) + cache.chunk_off.numel() * 4
    return read + write


def _median_time(fn, reps):
    ts, out = [], None
    for _ in range(reps):
        t0 = time.perf_counter()
        out = fn()
        ts.append(time.perf_counter() - t0)
    return float(np.median(ts)), out


def _oracle_layer(oracle, cfg, li, reps=1, decode_reps=1):
    """The oracle's stages on one layer, timed one by one (median of `reps` runs each), then
    `decode_reps` decodes of the first query (median).  Returns seconds per stage."""
    H, n, w, r_min = cfg["H"], cfg["n"], cfg["w"], cfg["r_min"]
    N = n - w
    st = {}
    st["salience"], s = _median_time(lambda: oracle.salience(li.K, li.Qw, H), reps)
    st["pool"], sb = _median_time(lambda: oracle.pool(s), reps)
    st["weights"], u = _median_time(lambda: oracle.weights(sb), reps)
    B = oracle.budget(n, 128, w, cfg["kappa"])
    st["allocate"], al = _median_time(lambda: oracle.allocate(u, B, r_min, 128), reps)
    st["project"], (cK, cV) = _median_time(
        lambda: (oracle.project(li.K[:N], li.PK, al.rank, cfg["dtype"]),
                 oracle.project(li.V[:N], li.PV, al.rank, cfg["dtype"])), reps)
    st["compress"] = sum(st[k] for k in ("salience", "pool", "weights", "allocate", "project"))
    Kx, Vx = np.ascontiguousarray(li.K[N:]), np.ascontiguousarray(li.V[N:])
    dec = lambda: oracle.decode(cK, cV, al.rank, Kx, Vx, li.PK, li.PV, li.q[0], H)
    st["decode"], _ = _median_time(dec, decode_reps)
    return st, dec


def cpu_baseline(cfg, li, dbytes, gpu, decode_reps=24, qwen_layers=4, llama128_layers=2):
    """The fp64 oracle (as it stands) on the host cores, on bounded samples of the workloads:
    the Llama 32K layer stage by stage (median of 3 compresses, median of `decode_reps`
    decodes; one decode again on one thread), `qwen_layers` layers of one of the 8 Qwen
    sequences scaled to the 28-layer x 8-sequence stack, and `llama128_layers` of the 32
    layers of the 128K stack scaled to 32.  `gpu` holds the GPU figures for the ratios."""
    import oracle
    from workloads import CONFIGS, make_layer
    cores = oracle.threads()
    t0 = time.perf_counter()
    st, dec = _oracle_layer(oracle, cfg, li, reps=3, decode_reps=decode_reps)
    oracle.set_threads(1)
    try:
        t1thr, _ = _median_time(dec, 1)
    finally:
        oracle.set_threads(cores)
    ms = {k: round(v * 1e3, 2) for k, v in st.items()}
    out = {
        "value": round(dbytes / st["decode"] / 1e9, 4),
        "unit": "GB/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"llama_32k: one full layer ({cfg['n']} tokens), fp64 stages timed one by one "
                  f"(median of 3), decode of one query median of {decode_reps} "
                  f"(reconstruct-in-place); value = decode bytes / decode time",
        "stage_ms": ms,
        "compress_ms_per_32k_tokens": round(st["compress"] * 1e3 * 32768 / cfg["n"], 1),
        "decode_GBps_1_thread": round(dbytes / t1thr / 1e9, 5),
        "gpu_over_cpu": {"decode": round(st["decode"] * 1e3 / gpu["decode_ms"], 1),
                         "compress": round(st["compress"] * 1e3 / gpu["compress_ms"], 1)},
    }
    # Qwen2.5-7B-shaped stack: `qwen_layers` of 28 layers, sequence 0 of 8, scaled x (28/L) x 8
    qc = CONFIGS["qwen_16k_stack"]
    acc = {"compress": 0.0, "decode": 0.0}
    for lyr in range(qwen_layers):
        qli = make_layer(qc, layer=lyr, seq=0, n_queries=1)
        qst, _ = _oracle_layer(oracle, qc, qli)
        acc["compress"] += qst["compress"]
        acc["decode"] += qst["decode"]
    sc = qc["layers"] / qwen_layers * qc["batch"]
    out["qwen_16k_stack_scaled"] = {
        "sample": f"layers 0..{qwen_layers - 1} of sequence 0 (of 28 layers x 8 sequences), scaled x{sc:g}",
        "compress_ms_stack": round(acc["compress"] * 1e3 * sc, 1),
        "decode_ms_per_step": round(acc["decode"] * 1e3 * sc, 1),
        "decode_tokens_per_s": round(qc["batch"] / (acc["decode"] * sc), 3),
    }
    # Llama-3.1-8B-shaped 128K stack: `llama128_layers` of 32 layers, scaled x 32/L
    lc = CONFIGS["llama_128k_stack"]
    acc = {"compress": 0.0, "decode": 0.0}
    for lyr in range(llama128_layers):
        lli = make_layer(lc, layer=lyr, n_queries=1)
        lst, _ = _oracle_layer(oracle, lc, lli)
        acc["compress"] += lst["compress"]
        acc["decode"] += lst["decode"]
    sc = lc["layers"] / llama128_layers
    out["llama_128k_stack_scaled"] = {
        "sample": f"layers 0..{llama128_layers - 1} of 32 (host draws), scaled x{sc:g}",
        "compress_ms_per_32k_tokens": round(acc["compress"] * 1e3 * sc * 32768 / (lc["n"] * lc["layers"]), 1),
        "decode_ms_per_step": round(acc["decode"] * 1e3 * sc, 1),
        "decode_tokens_per_s": round(1.0 / (acc["decode"] * sc), 4),
    }
    out["wall_s"] = round(time.perf_counter() - t0, 1)
    return out


# HBM bytes of one decode call (both launches), from the FETCH_SIZE and WRITE_SIZE counter
# passes of `bench.py --mode pmc`, scaled by a 64 MiB copy kernel (FETCH x 2.0, WRITE x 1.0).
# They hold for the decode source they were taken on (SHA-256 prefix of the files below);
# after any change to it, traffic is reported as null until the counters are taken again.
DECODE_TRAFFIC = {"source_sha256": "7bfcb5b3f285c259", "bytes": 31487296}
DECODE_SOURCES = ("paper_2607_15498_amd/csrc/decode.hip", "paper_2607_15498_amd/csrc/vr_device.h")


def decode_source_sha():
    import hashlib
    h = hashlib.sha256()
    for f in DECODE_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def decode_traffic():
    if DECODE_TRAFFIC["bytes"] is None or decode_source_sha() != DECODE_TRAFFIC["source_sha256"]:
        return None
    return DECODE_TRAFFIC["bytes"]


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this codec has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    if args.config in ("llama_128k_stack", "qwen_16k_stack"):
        return bench_stack(args)
    if args.config == "agnostic_32k":
        return bench_agnostic(args)
    import torch

    import paper_2607_15498_amd as vr
    from workloads import CONFIGS, make_layer

    cfg = CONFIGS[args.config]
    dev = torch.device("cuda:0")
    li = make_layer(cfg, n_queries=1)
    shape = vr.Shape(n=cfg["n"], G=cfg["G"], H=cfg["H"], w=cfg["w"], r_min=cfg["r_min"],
                     kappa_pct=cfg["kappa"], dtype=cfg["dtype"])
    dt = shape.torch_dtype
    up = lambda a, t=dt: torch.from_numpy(np.ascontiguousarray(a)).to(t).to(dev)
    Ks = [up(li.K) for _ in range(N_INPUT_COPIES)]
    Vs = [up(li.V) for _ in range(N_INPUT_COPIES)]
    Qw, q = up(li.Qw), up(li.q)
    PK, PV = up(li.PK, torch.float32), up(li.PV, torch.float32)
    slots = [vr.new_cache(shape, device=dev) for _ in range(N_CACHE_SLOTS)]
    sbars = [torch.empty(shape.N, dtype=torch.float32, device=dev) for _ in range(N_INPUT_COPIES)]
    out = torch.empty_like(q)
    ws_c = torch.zeros(vr.library().varrate_compress_workspace_bytes(__import__("ctypes").byref(shape.c())),
                       dtype=torch.uint8, device=dev)
    ws_d = vr.decode_workspace(shape, 1, 1, dev)

    # fill every slot once (untimed) so each decode reads a real compressed cache
    for i, c in enumerate(slots):
        j = i % N_INPUT_COPIES
        vr.compress(shape, Ks[j], Vs[j], Qw, PK, PV, cache=c, sbar_out=sbars[j], workspace=ws_c)
    torch.cuda.synchronize()

    if args.mode == "pmc":
        # Counter passes: one eager decode per slot (the slots differ, so no decode re-reads what
        # an earlier one left in the caches), then copies of a known size: 64 MiB read + 64 MiB
        # written per copy, the scale for FETCH_SIZE / WRITE_SIZE.
        for i in range(8):
            vr.decode(shape, [slots[i]], q, PK, PV, out=out, workspace=ws_d)
        torch.cuda.synchronize()
        src = torch.empty(32 << 20, dtype=torch.bfloat16, device=dev).fill_(1.0)
        dsts = [torch.empty_like(src) for _ in range(2)]
        for i in range(4):
            dsts[i % 2].copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "pmc", "decode_launches": 8, "decode_bytes": int(decode_bytes(shape, slots[0])),
                          "copy_launches": 4, "copy_bytes_each_way": src.numel() * 2}), flush=True)
        return

    # Every timed launch is replayed from a captured HIP graph, so host-side Python does not
    # gap the GPU: one graph per stage (one launch per cache slot) and one for whole steps.
    def stage_fns(i):
        j = i % N_INPUT_COPIES
        c = slots[i % N_CACHE_SLOTS]
        d = slots[(i + N_CACHE_SLOTS // 2) % N_CACHE_SLOTS]
        return {
            "salience": lambda: vr.salience(shape, Ks[j], Qw, sbars[j], workspace=ws_c),
            "allocate": lambda: vr.allocate(shape, sbars[j], c, workspace=ws_c),
            "project": lambda: vr.project(shape, Ks[j], Vs[j], PK, PV, c, workspace=ws_c),
            "compress": lambda: vr.compress(shape, Ks[j], Vs[j], Qw, PK, PV, cache=c, sbar_out=sbars[j],
                                            workspace=ws_c),
            "decode": lambda: vr.decode(shape, [d], q, PK, PV, out=out, workspace=ws_d),
        }

    def step(i):
        # one pass of the hot path as a caller runs it: compress (the single entry point),
        # then decode
        fns = stage_fns(i)
        fns["compress"]()
        fns["decode"]()

    for i in range(max(args.warmup, 1)):
        step(i)
    torch.cuda.synchronize()
    cap_stream = torch.cuda.Stream()
    graphs = {}
    for name in ("salience", "allocate", "project", "compress", "decode"):
        g_ = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_, stream=cap_stream):
            for i in range(N_CACHE_SLOTS):
                stage_fns(i)[name]()
        graphs[name] = g_
    step_graphs = []
    for i in range(N_CACHE_SLOTS):
        g_ = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_, stream=cap_stream):
            step(i)
        step_graphs.append(g_)
    torch.cuda.synchronize()

    ev = lambda: torch.cuda.Event(enable_timing=True)

    # per stage: median (p10, p90) over replays of its graph, per launch
    stage_st = {name: _replay_stats(g_, 8, N_CACHE_SLOTS) for name, g_ in graphs.items()}
    stage = {name: st["p50"] for name, st in stage_st.items()}

    # timed region: exactly `steps` whole steps (compress + decode)
    steps = args.steps
    for i in range(args.warmup):
        step_graphs[i % N_CACHE_SLOTS].replay()
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    t0 = time.perf_counter()
    e0.record()
    for i in range(steps):
        step_graphs[(args.warmup + i) % N_CACHE_SLOTS].replay()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step_events = e0.elapsed_time(e1) / steps

    ms_dec = stage["decode"]
    ms_comp = stage["compress"]
    dbytes = decode_bytes(shape, slots[0])
    cbytes = compress_bytes(shape, slots[0])
    dec_gbs = dbytes / (ms_dec * 1e-3) / 1e9
    result = {
        "metric": "compressed decode attn GB/s (% HBM peak) + compress ms per 32K tokens, 1 GPU",
        "value": round(dec_gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / steps, 4),
        "ms_per_step_gpu_events": round(ms_step_events, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg["dtype"] == "bf16" else "f32",
        "data": "synthetic (seeded keys/values/queries with planted salient tokens; "
                "offline PCA bases from disjoint calibration draws)",
        "config": {"workload": f"{args.config}: 1 layer, {cfg['G']} KV x {cfg['H']} q heads, d 128, "
                               f"n {cfg['n']}, w {cfg['w']}, budget {cfg['kappa']}%, r_min {cfg['r_min']}",
                   "decode_batch": 1, "coded_budget_B": slots[0].B},
        "pct_hbm_peak": round(100 * dec_gbs / HBM_PEAK_GBS, 2),
        "compress_ms_per_32k_tokens": round(ms_comp * 32768 / cfg["n"], 4),
        "compress_GBps_algorithmic": round(cbytes / (ms_comp * 1e-3) / 1e9, 1),
        "stage_ms": {k: round(v, 4) for k, v in stage.items()},
        "stage_ms_p10_p90": {k: [round(st["p10"], 4), round(st["p90"], 4)] for k, st in stage_st.items()},
        "timing": "medians over 8 replays of a graph of 24 launches on distinct inputs/caches "
                  "(HIP events on the launching stream); p10/p90 beside them",
        "roofline": {"kernel": "decode_ring_kernel + decode_merge_kernel (rank-space decode attention)", "bound": "hbm",
                     "achieved": round(dbytes / (ms_dec * 1e-3) / 1e9, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(dbytes / (ms_dec * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": decode_traffic(), "bytes_per_launch": int(dbytes)},
    }
    # quantised coefficients (Sec. 3.3 "Composability"): every slot quantised, then decodes
    # over the codes timed like the plain decode (24 slots per replay, medians)
    rank_host = slots[0].rank.cpu().numpy()
    qrows = {}
    for bits in (4, 3):
        qslots = [vr.quantize(shape, c, bits) for c in slots]
        torch.cuda.synchronize()
        gq, gz = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
        with torch.cuda.graph(gq, stream=cap_stream):
            for i in range(N_CACHE_SLOTS):
                j = (i + N_CACHE_SLOTS // 2) % N_CACHE_SLOTS
                vr.decode_q(shape, [slots[j]], [qslots[j]], q, PK, PV, out=out, workspace=ws_d)
        with torch.cuda.graph(gz, stream=cap_stream):
            for i in range(N_CACHE_SLOTS):
                vr.quantize(shape, slots[i], bits, qslots[i])
        torch.cuda.synchronize()
        stq = _replay_stats(gq, 8, N_CACHE_SLOTS)
        stz = _replay_stats(gz, 4, N_CACHE_SLOTS)
        qbytes = decode_bytes_q(shape, slots[0], bits, rank_host)
        coefq = 2 * shape.G * (slots[0].B * bits // 8 + 2 * int(((rank_host.astype(np.int64) + 31) // 32).sum()))
        qrows[f"{bits}bit"] = {
            "decode_ms": round(stq["p50"], 4), "decode_ms_p10_p90": [round(stq["p10"], 4), round(stq["p90"], 4)],
            "decode_GBps": round(qbytes / (stq["p50"] * 1e-3) / 1e9, 2),
            "frac": round(qbytes / (stq["p50"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "decode_bytes": int(qbytes),
            "quantize_ms": round(stz["p50"], 4),
            "footprint_pct_of_full_kv": round(footprint_pct(shape, slots[0], coefq), 2),
        }
        del gq, gz, qslots
    result["quantized_coefficients"] = dict(
        qrows, footprint_pct_bf16_coefficients=round(footprint_pct(shape, slots[0], 2 * shape.G * slots[0].B * 2), 2),
        note="group-wise symmetric codes, 32-coordinate groups, binary16 scales; decode_bytes counts "
             "codes + scales + exact rows + metadata + bases; same 32K layer and batch 1")
    # residual codec (Sec. 3.1 Eq. 2): anchors every 16 tokens kept exact, the other tokens
    # coded as residuals to their 4 nearest anchors' mean; same layer, budget and floor
    result["residual_codec"] = bench_anchor(args, shape, Ks, Vs, Qw, q, PK, PV, out, cap_stream)
    # rotary keys: a 32K layer of the same geometry whose cache is post-RoPE
    result["rotary_keys"] = bench_rope(args, cap_stream)
    # shared cross-head basis: one R = 1024 coefficient row per token for all heads and K, V
    result["shared_basis"] = bench_joint(args, cap_stream)
    if not args.no_stack:
        # the 128K end of the 32K-128K target range: the 32-layer Llama stack, decode at batch 1
        del graphs, step_graphs, slots, Ks, Vs, sbars
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        stk = bench_stack(args, "llama_128k_stack", emit=False, quant_bits=4)
        result["llama_128k_stack"] = {
            "workload": stk["config"]["workload"],
            "decode_GBps": stk["value"], "pct_hbm_peak": stk["pct_hbm_peak"],
            "frac": round(stk["value"] / HBM_PEAK_GBS, 4),
            "decode_ms_per_step": stk["ms_per_step"], "decode_ms_per_step_p10_p90": stk["ms_per_step_p10_p90"],
            "decode_us_per_layer": round(stk["ms_per_step"] * 1e3 / 32, 2),
            "decode_tokens_per_s": stk["decode_tokens_per_s"],
            "decode_bytes_per_step": stk["decode_bytes_per_step"],
            "compress_ms_per_32k_tokens": stk["compress_ms_per_32k_tokens"],
            "compress_ms_per_32k_tokens_all_layers": stk["compress_ms_per_32k_tokens_all_layers"],
            "decode_4bit": stk["decode_4bit"],
        }
    # measured read ceiling for the same byte counts: the decode's time over the probe's
    probe_sizes = [int(dbytes)]
    if "llama_128k_stack" in result:
        probe_sizes.append(int(result["llama_128k_stack"]["decode_bytes_per_step"]) // 32)
    probe = bench_read_probe(cap_stream, probe_sizes)
    dec_us = [ms_dec * 1e3] + ([result["llama_128k_stack"]["decode_us_per_layer"]] if len(probe_sizes) > 1 else [])
    for (k, row), us in zip(probe.items(), dec_us):
        row["decode_us"] = round(us, 2)
        row["decode_over_probe_with_second_launch"] = round(us / row["with_second_launch"]["us"], 3)
    result["read_probe"] = dict(probe, note="varrate_read_probe over 8 rotating windows (no last-level cache "
                                            "reuse), graphs of 24 launches like the decode's, medians; keys are the byte counts of the "
                                            "32K decode call and of one 128K layer's decode")
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg, li, dbytes, {"decode_ms": ms_dec, "compress_ms": ms_comp})
    print(json.dumps(result), flush=True)


def bench_read_probe(cap_stream, sizes, n_windows=8, per_graph=N_CACHE_SLOTS):
    """Measured read ceiling: the library's streaming-read probe over `nbytes` (each size in
    `sizes`), replayed from a graph of `per_graph` launches (as many as the decode graphs hold)
    that cycles through `n_windows` distinct windows so that no launch finds its bytes in the
    256 MB last-level cache, alone and followed by a one-element fill (a second dependent
    launch, the shape of a decode call: streaming kernel + merge)."""
    import torch

    import paper_2607_15498_amd as vr
    dev = torch.device("cuda:0")
    span = max(sizes)
    span = (span + 4095) // 4096 * 4096
    buf = torch.ones(n_windows * span // 4, dtype=torch.int32, device=dev)
    sink = torch.zeros(vr.PROBE_WGS, dtype=torch.int32, device=dev)
    tiny = torch.zeros(1, dtype=torch.int32, device=dev)
    res = {}
    for nb in sizes:
        nb = nb // 16 * 16
        row = {}
        for label, second in (("alone", False), ("with_second_launch", True)):
            g_ = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_, stream=cap_stream):
                for i in range(per_graph):
                    vr.read_probe(buf[(i % n_windows) * span // 4:], nb, sink)
                    if second:
                        tiny.fill_(i)
            torch.cuda.synchronize()
            st = _replay_stats(g_, 8, per_graph)
            row[label] = {"us": round(st["p50"] * 1e3, 2),
                          "GBps": round(nb / (st["p50"] * 1e-3) / 1e9, 1),
                          "frac": round(nb / (st["p50"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        res[str(nb)] = row
    del buf
    return res


def bench_rope(args, cap_stream, n_slots=12):
    """Rotary keys (Sec. 3.1 "Joint per-token vector"; Algorithm 1 first and last steps) on a
    32K layer of the same geometry with Llama-3.1 frequencies: compress (salience on the
    post-RoPE cache, un-rotation, allocation, projection) and decode (keys rebuilt by MFMA and
    rotated to their positions), each replayed from a graph over `n_slots` caches."""
    import ctypes
    import torch

    import paper_2607_15498_amd as vr
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["llama_32k_rope"]
    li = make_layer(cfg, n_queries=1)
    sh = vr.Shape(n=cfg["n"], G=cfg["G"], H=cfg["H"], w=cfg["w"], r_min=cfg["r_min"], kappa_pct=cfg["kappa"],
                  dtype=cfg["dtype"], rope_theta=tuple(float(x) for x in li.theta))
    dev = torch.device("cuda:0")
    up = lambda a, t=torch.bfloat16: torch.from_numpy(np.ascontiguousarray(a)).to(t).to(dev)
    Ks = [up(li.K) for _ in range(N_INPUT_COPIES)]
    Vs = [up(li.V) for _ in range(N_INPUT_COPIES)]
    Qw, q = up(li.Qw), up(li.q)
    PK, PV = up(li.PK, torch.float32), up(li.PV, torch.float32)
    out = torch.empty_like(q)
    slots = [vr.new_cache(sh, device=dev) for _ in range(n_slots)]
    wsc = torch.zeros(vr.library().varrate_compress_workspace_bytes(ctypes.byref(sh.c())), dtype=torch.uint8,
                      device=dev)
    wsd = vr.decode_workspace(sh, 1, 1, dev)
    for i, c in enumerate(slots):
        vr.compress(sh, Ks[i % len(Ks)], Vs[i % len(Vs)], Qw, PK, PV, cache=c, workspace=wsc)
    torch.cuda.synchronize()
    gc, gd = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(gc, stream=cap_stream):
        for i, c in enumerate(slots):
            vr.compress(sh, Ks[i % len(Ks)], Vs[i % len(Vs)], Qw, PK, PV, cache=c, workspace=wsc)
    with torch.cuda.graph(gd, stream=cap_stream):
        for i in range(n_slots):
            vr.decode(sh, [slots[(i + n_slots // 2) % n_slots]], q, PK, PV, out=out, workspace=wsd)
    torch.cuda.synchronize()
    stc = _replay_stats(gc, 3, n_slots)
    std = _replay_stats(gd, 8, n_slots)
    # the plain decode's bytes plus each stored position's token index (read once per KV head)
    by = decode_bytes(sh, slots[0]) + sh.G * slots[0].N * 4
    flops = 2.0 * sh.G * 128 * int(slots[0].rank[:slots[0].N].to(torch.int64).sum()) + 2.0 * sh.H * slots[0].N * 128
    res = {
        "config": f"llama_32k_rope: 1 layer, 8 KV x 32 q heads, n {sh.n}, w {sh.w}, budget {sh.kappa_pct}%, "
                  f"r_min {sh.r_min}, Llama-3.1 rotary frequencies (base 500000, scaling 8)",
        "compress_ms_per_32k_tokens": round(stc["p50"] * 32768 / sh.n, 4),
        "compress_ms_p10_p90": [round(stc["p10"], 4), round(stc["p90"], 4)],
        "decode_ms": round(std["p50"], 4), "decode_ms_p10_p90": [round(std["p10"], 4), round(std["p90"], 4)],
        "decode_GBps": round(by / (std["p50"] * 1e-3) / 1e9, 2),
        "frac": round(by / (std["p50"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "decode_bytes": int(by),
        "decode_key_rebuild_GFLOP": round(flops / 1e9, 3),
    }
    del gc, gd, slots, Ks, Vs
    return res


def bench_joint(args, cap_stream, n_slots=12):
    """Shared cross-head basis (Sec. 3.1 Eq. (1) "Joint per-token vector", "Shared basis") on
    a 32K layer of the Llama geometry with R = 1024 (Dz = 2048): compress (salience, joint
    water-filling, projection onto W) and decode, each replayed from a graph over `n_slots`
    caches."""
    import ctypes
    import torch

    import paper_2607_15498_amd as vr
    from workloads import CONFIGS, make_layer
    cfg = CONFIGS["llama_32k_joint"]
    li = make_layer(cfg, n_queries=1)
    R = cfg["joint_R"]
    sh = vr.Shape(n=cfg["n"], G=cfg["G"], H=cfg["H"], w=cfg["w"], r_min=cfg["r_min"], kappa_pct=cfg["kappa"],
                  dtype=cfg["dtype"])
    dev = torch.device("cuda:0")
    up = lambda a, t=torch.bfloat16: torch.from_numpy(np.ascontiguousarray(a)).to(t).to(dev)
    Ks = [up(li.K) for _ in range(N_INPUT_COPIES)]
    Vs = [up(li.V) for _ in range(N_INPUT_COPIES)]
    Qw, q = up(li.Qw), up(li.q)
    W = up(li.W, torch.float32)
    out = torch.empty_like(q)
    slots = [vr.new_jcache(sh, R, device=dev) for _ in range(n_slots)]
    wsc = torch.zeros(vr.library().varrate_joint_compress_workspace_bytes(ctypes.byref(sh.c()), R),
                      dtype=torch.uint8, device=dev)
    wsd = vr.joint_decode_workspace(sh, R, 1, 1, dev)
    for i, c in enumerate(slots):
        vr.joint_compress(sh, Ks[i % len(Ks)], Vs[i % len(Vs)], Qw, W, cache=c, workspace=wsc)
    torch.cuda.synchronize()
    gc, gd = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(gc, stream=cap_stream):
        for i, c in enumerate(slots):
            vr.joint_compress(sh, Ks[i % len(Ks)], Vs[i % len(Vs)], Qw, W, cache=c, workspace=wsc)
    with torch.cuda.graph(gd, stream=cap_stream):
        for i in range(n_slots):
            vr.joint_decode(sh, [slots[(i + n_slots // 2) % n_slots]], q, W, out=out, workspace=wsd)
    torch.cuda.synchronize()
    stc = _replay_stats(gc, 3, n_slots)
    std = _replay_stats(gd, 8, n_slots)
    c0 = slots[0]
    rank_sum = int(c0.rank.to(torch.int64).sum())
    Dz = 2 * sh.G * 128
    # coefficients, exact rows, ranks and offsets, the basis's key and value columns (fp32),
    # queries and outputs
    by = 2 * c0.B + 2 * sh.G * c0.n_exact * 128 * 2 + c0.N * 6 + R * Dz * 4 + 2 * sh.H * 128 * 2
    proj_flop = 2.0 * rank_sum * Dz
    res = {
        "config": f"llama_32k_joint: 1 layer, 8 KV x 32 q heads, n {sh.n}, w {sh.w}, budget {sh.kappa_pct}%, "
                  f"r_min {sh.r_min}, R {R}, Dz {Dz}, B {c0.B} (mean rank {rank_sum / c0.N:.1f})",
        "compress_ms_per_32k_tokens": round(stc["p50"] * 32768 / sh.n, 4),
        "compress_ms_p10_p90": [round(stc["p10"], 4), round(stc["p90"], 4)],
        "projection_GFLOP_kept_coefficients": round(proj_flop / 1e9, 1),
        "decode_ms": round(std["p50"], 4), "decode_ms_p10_p90": [round(std["p10"], 4), round(std["p90"], 4)],
        "decode_GBps": round(by / (std["p50"] * 1e-3) / 1e9, 2),
        "frac": round(by / (std["p50"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "decode_bytes": int(by),
        "footprint_pct_of_full_kv": round(100.0 * (2 * c0.B + 2 * sh.G * sh.w * 128 * 2 + c0.N * 2)
                                          / (2 * sh.n * sh.G * 128 * 2), 2),
    }
    del gc, gd, slots, Ks, Vs
    return res


def decode_bytes_anchor(shape, cache, n_queries=1):
    """Algorithmic bytes of a decode over the residual codec: the coded tokens' coefficients,
    the exact anchor and window rows, ranks, chunk offsets, each stored position's anchors and
    the anchors' inverse lists, both bases, queries and outputs."""
    es = 2
    G, H, d = shape.G, shape.H, 128
    coef = 2 * G * cache.B * es
    exact = 2 * G * (cache.n_exact + cache.na) * d * es
    meta = cache.N + cache.chunk_off.numel() * 4 + cache.N * 8 + cache.N * 16 + (cache.na + 1) * 4
    return coef + exact + meta + 2 * G * d * d * 4 + 2 * n_queries * H * d * es


def bench_anchor(args, shape0, Ks, Vs, Qw, q, PK, PV, out, cap_stream, n_slots=12):
    """The residual codec on the bench layer: compress (salience, nearest-anchor search,
    encode) and decode, each replayed from a graph over `n_slots` caches (medians)."""
    import ctypes
    import torch

    import paper_2607_15498_amd as vr
    ash = vr.Shape(n=shape0.n, G=shape0.G, H=shape0.H, w=shape0.w, r_min=shape0.r_min,
                   kappa_pct=shape0.kappa_pct, dtype=shape0.dtype, anchor_stride=16)
    dev = Ks[0].device
    slots = [vr.new_cache(ash, device=dev) for _ in range(n_slots)]
    wsa = torch.zeros(vr.library().varrate_compress_workspace_bytes(ctypes.byref(ash.c())), dtype=torch.uint8,
                      device=dev)
    wsd = vr.decode_workspace(ash, 1, 1, dev)
    for i, c in enumerate(slots):
        vr.compress(ash, Ks[i % len(Ks)], Vs[i % len(Vs)], Qw, PK, PV, cache=c, workspace=wsa)
    torch.cuda.synchronize()
    gc, gd, gs = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(gc, stream=cap_stream):
        for i, c in enumerate(slots):
            vr.compress(ash, Ks[i % len(Ks)], Vs[i % len(Vs)], Qw, PK, PV, cache=c, workspace=wsa)
    with torch.cuda.graph(gd, stream=cap_stream):
        for i in range(n_slots):
            vr.decode(ash, [slots[(i + n_slots // 2) % n_slots]], q, PK, PV, out=out, workspace=wsd)
    with torch.cuda.graph(gs, stream=cap_stream):
        for i in range(n_slots):
            vr.anchor_search(ash, Ks[i % len(Ks)], Vs[i % len(Vs)], workspace=wsa)
    torch.cuda.synchronize()
    stc = _replay_stats(gc, 3, n_slots)
    std = _replay_stats(gd, 8, n_slots)
    sts = _replay_stats(gs, 3, n_slots)
    by = decode_bytes_anchor(ash, slots[0])
    full = 2 * ash.n * ash.G * 128 * 2
    stored = 2 * ash.G * slots[0].B * 2 + 2 * ash.G * (ash.w + slots[0].na) * 128 * 2 + slots[0].N * 9
    res = {
        "config": f"anchors every 16 prefix tokens ({slots[0].na}), {slots[0].N} coded tokens, B {slots[0].B}, "
                  f"budget {ash.kappa_pct}%, r_min {ash.r_min}",
        "compress_ms_per_32k_tokens": round(stc["p50"] * 32768 / ash.n, 4),
        "anchor_search_ms": round(sts["p50"], 4),
        "anchor_search_TFLOPs": round(2.0 * slots[0].N * slots[0].na * 2 * ash.G * 128 / (sts["p50"] * 1e-3) / 1e12, 1),
        "decode_ms": round(std["p50"], 4), "decode_ms_p10_p90": [round(std["p10"], 4), round(std["p90"], 4)],
        "decode_GBps": round(by / (std["p50"] * 1e-3) / 1e9, 2),
        "frac": round(by / (std["p50"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "decode_bytes": int(by),
        "footprint_pct_of_full_kv": round(100.0 * stored / full, 2),
    }
    del gc, gd, gs, slots
    return res


def _graph_ms(g_, reps):
    """Median ms of one replay of a captured graph over `reps` replays (events on the
    current stream, which the replays run on)."""
    return _replay_stats(g_, reps)["p50"]


def _replay_stats(g_, reps, per=1):
    """Per-replay durations of a captured graph (HIP events on the current stream around
    each replay, back to back), divided by `per` launches per replay: median, p10, p90, mean
    in ms."""
    import torch
    g_.replay()
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    evs[0].record()
    for i in range(reps):
        g_.replay()
        evs[i + 1].record()
    torch.cuda.synchronize()
    t = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(reps)]) / per
    return {"p50": float(np.median(t)), "p10": float(np.percentile(t, 10)),
            "p90": float(np.percentile(t, 90)), "mean": float(t.mean()), "n": int(reps)}


def _pct(st, nd=4):
    return {k: (round(v, nd) if isinstance(v, float) else v) for k, v in st.items()}


def bench_stack(args, config=None, emit=True, quant_bits=None):
    """Whole model stack: every layer (and sequence) drawn on the device, compressed, then
    decode steps of one query per sequence over all layers (one decode call per layer, the
    batch's caches in that call).  Compress and decode are timed from captured graphs.  The
    Qwen batch decodes with 128 tokens appended to every exact tail (the middle of its 256
    steps); the Llama 128K stack decodes right after the prompt."""
    import torch

    import paper_2607_15498_amd as vr
    from workloads import CONFIGS, make_head_model
    from workloads.synth_gpu import make_layer_device

    name = config or args.config
    cfg = CONFIGS[name]
    L, S, n, w = cfg["layers"], cfg["batch"], cfg["n"], cfg["w"]
    extra = 128 if S > 1 else 0
    dev = torch.device("cuda:0")
    shape = vr.Shape(n=n, G=cfg["G"], H=cfg["H"], w=w, r_min=cfg["r_min"], kappa_pct=cfg["kappa"],
                     dtype=cfg["dtype"])
    dt = shape.torch_dtype
    up = lambda a, t=dt: torch.from_numpy(np.ascontiguousarray(a)).to(t).to(dev)
    t0 = time.perf_counter()
    inputs, caches, bases, qs = [], [], [], []
    for l in range(L):
        hms = [make_head_model(cfg["seed"], l, g, cfg["d"]) for g in range(cfg["G"])]
        row, qrow = [], []
        for sq in range(S):
            dl = make_layer_device(cfg, layer=l, seq=sq, head_models=hms, with_basis=(sq == 0), device=dev)
            if sq == 0:
                bases.append((up(dl.PK, torch.float32), up(dl.PV, torch.float32)))
            row.append((dl.K, dl.V, up(dl.Qw)))
            qrow.append(dl.q)
        inputs.append(row)
        caches.append([vr.new_cache(shape, cap=w + 2 * extra + 8, device=dev) for _ in range(S)])
        qs.append(up(np.stack(qrow)))
    torch.cuda.synchronize()
    t_draw = time.perf_counter() - t0
    ws_c = torch.zeros(vr.library().varrate_compress_workspace_bytes(__import__("ctypes").byref(shape.c())),
                       dtype=torch.uint8, device=dev)
    ws_d = vr.decode_workspace(shape, S, 1, dev)

    def compress_all(into=None):
        for l in range(L):
            for sq in range(S):
                K, V, Qw = inputs[l][sq]
                c = caches[l][sq] if into is None else into[(l * S + sq) % len(into)]
                vr.compress(shape, K, V, Qw, bases[l][0], bases[l][1], cache=c, workspace=ws_c)
    compress_all()
    torch.cuda.synchronize()
    if extra:
        gen = torch.Generator(device=dev)
        gen.manual_seed(cfg["seed"])
        for l in range(L):
            for sq in range(S):
                for _ in range(extra):
                    kv = torch.randn((2, cfg["G"], cfg["d"]), generator=gen, device=dev).to(dt)
                    vr.append_exact(shape, caches[l][sq], kv[0], kv[1])
        torch.cuda.synchronize()
    outs = [torch.empty_like(qs[l]) for l in range(L)]

    def step():
        for l in range(L):
            vr.decode(shape, caches[l], qs[l], bases[l][0], bases[l][1], out=outs[l], workspace=ws_d)
    step()
    torch.cuda.synchronize()
    cap = torch.cuda.Stream()
    g_step, g_comp = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_step, stream=cap):
        step()
    # re-compressing would reset the decode caches' exact tails (appended tokens): with a tail,
    # the timed compress writes two spare caches in turn instead (the same work per call)
    spare = [vr.new_cache(shape, cap=w + 2 * extra + 8, device=dev) for _ in range(2)] if extra else None
    with torch.cuda.graph(g_comp, stream=cap):
        compress_all(spare)
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        g_step.replay()
    torch.cuda.synchronize()
    st_step = _replay_stats(g_step, max(args.steps, 1))
    ms_step = st_step["p50"]
    ms_comp = _replay_stats(g_comp, 3)["p50"]
    dbytes = sum(decode_bytes(shape, c) for row in caches for c in row)
    gbs = dbytes / (ms_step * 1e-3) / 1e9
    result = {
        "metric": "compressed decode attn GB/s (% HBM peak) + compress ms per 32K tokens, 1 GPU",
        "value": round(gbs, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4), "ms_per_step_p10_p90": [round(st_step["p10"], 4), round(st_step["p90"], 4)],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg["dtype"], "data": "synthetic, drawn on the device (same recipe as the parity inputs, "
                                        "device Philox draws per layer/head/sequence)",
        "config": {"workload": f"{name}: {L} layers, {cfg['G']} KV x {cfg['H']} q heads, d 128, "
                               f"n {n}, w {w}, budget {cfg['kappa']}%, r_min {cfg['r_min']}, "
                               f"batch {S} independent sequences, decode exact tail w + {extra}",
                   "decode_calls_per_step": L},
        "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "decode_tokens_per_s": round(S / (ms_step * 1e-3), 1),
        "decode_bytes_per_step": int(dbytes),
        # per 32K tokens of one layer (the single-layer workload's unit), and of the whole stack
        "compress_ms_per_32k_tokens": round(ms_comp * 32768 / (n * S * L), 4),
        "compress_ms_per_32k_tokens_all_layers": round(ms_comp * 32768 / (n * S), 4),
        "compress_timing": "graph replay" + (" (into two spare caches in turn)" if extra else ""),
        "compress_ms_total": round(ms_comp, 3),
        "draw_s": round(t_draw, 1),
    }
    if quant_bits:
        # every layer's coefficients quantised to b-bit codes, then the same decode step over them
        qcs = [[vr.quantize(shape, c, quant_bits) for c in row] for row in caches]
        torch.cuda.synchronize()
        g_q = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_q, stream=cap):
            for l in range(L):
                vr.decode_q(shape, caches[l], qcs[l], qs[l], bases[l][0], bases[l][1], out=outs[l], workspace=ws_d)
        torch.cuda.synchronize()
        st_q = _replay_stats(g_q, max(args.steps, 1))
        qbytes = sum(decode_bytes_q(shape, c, quant_bits, c.rank.cpu().numpy()) for row in caches for c in row)
        result[f"decode_{quant_bits}bit"] = {
            "ms_per_step": round(st_q["p50"], 4), "ms_per_step_p10_p90": [round(st_q["p10"], 4), round(st_q["p90"], 4)],
            "decode_GBps": round(qbytes / (st_q["p50"] * 1e-3) / 1e9, 2),
            "frac": round(qbytes / (st_q["p50"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "decode_tokens_per_s": round(S / (st_q["p50"] * 1e-3), 1),
            "decode_bytes_per_step": int(qbytes),
        }
    if emit:
        print(json.dumps(result), flush=True)
    return result


def bench_agnostic(args):
    """Query-agnostic reuse: one 32K prefix compressed once per budget (10/20/40%; r_min 8 at
    10%, where 16 is infeasible in per-head units), then 64 fresh Gaussian queries decoded as
    one batch.  Reports decode GB/s per budget and the error of VarRate and of the uniform
    ("flat") allocation at the same budget against full-KV attention over the uncompressed
    bf16 cache (fp32 reference on the device)."""
    import torch

    import paper_2607_15498_amd as vr
    from workloads import CONFIGS
    from workloads.synth_gpu import make_layer_device

    cfg = CONFIGS[args.config]
    Qn, n, w, G, H = cfg["queries"], cfg["n"], cfg["w"], cfg["G"], cfg["H"]
    dev = torch.device("cuda:0")
    dl = make_layer_device(cfg, n_queries=Qn, query_law="agnostic", device=dev)
    up = lambda a, t=torch.bfloat16: torch.from_numpy(np.ascontiguousarray(a)).to(t).to(dev)
    PK, PV, Qw, q = up(dl.PK, torch.float32), up(dl.PV, torch.float32), up(dl.Qw), up(dl.q)
    # full-KV attention reference (fp32), [Q][H][d]
    hpg = H // G
    ref = torch.empty((Qn, H, 128), dtype=torch.float32, device=dev)
    for h in range(H):
        g = h // hpg
        sc = (q[:, h].float() @ dl.K[:, g].float().T) / np.sqrt(128.0)
        ref[:, h] = torch.softmax(sc, dim=-1) @ dl.V[:, g].float()

    def rel_l2(out):
        e = (out.float() - ref).norm(dim=-1) / ref.norm(dim=-1)
        e = e.flatten().cpu().numpy()
        return {"mean": round(float(e.mean()), 5), "p95": round(float(np.percentile(e, 95)), 5),
                "max": round(float(e.max()), 5)}

    if args.mode == "pmc":
        # Counter passes: the 20% cache decoded eagerly 8 times as one batch of 64 queries.
        kappa, r_min = next(b for b in cfg["budgets"] if b[0] == 20)
        shape = vr.Shape(n=n, G=G, H=H, w=w, r_min=r_min, kappa_pct=kappa, dtype="bf16")
        cache = vr.compress(shape, dl.K, dl.V, Qw, PK, PV)
        ws = vr.decode_workspace(shape, 1, Qn, dev)
        out = torch.empty_like(q)
        for _ in range(8):
            vr.decode(shape, [cache], q, PK, PV, out=out, workspace=ws)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "pmc", "config": args.config, "decode_launches": 8,
                          "decode_bytes": int(decode_bytes(shape, cache, Qn))}), flush=True)
        return

    rows = []
    for kappa, r_min in cfg["budgets"]:
        shape = vr.Shape(n=n, G=G, H=H, w=w, r_min=r_min, kappa_pct=kappa, dtype="bf16")
        cache = vr.compress(shape, dl.K, dl.V, Qw, PK, PV)
        flat = vr.new_cache(shape, device=dev)
        vr.allocate(shape, torch.full((shape.N,), 0.5, dtype=torch.float32, device=dev), flat)
        vr.project(shape, dl.K, dl.V, PK, PV, flat)
        ws = vr.decode_workspace(shape, 1, Qn, dev)
        out = torch.empty_like(q)
        vr.decode(shape, [cache], q, PK, PV, out=out, workspace=ws)
        torch.cuda.synchronize()
        err_v = rel_l2(out)
        vr.decode(shape, [flat], q, PK, PV, out=out, workspace=ws)
        torch.cuda.synchronize()
        err_f = rel_l2(out)
        g_ = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        with torch.cuda.graph(g_, stream=cap):
            vr.decode(shape, [cache], q, PK, PV, out=out, workspace=ws)
        ms = _graph_ms(g_, 20)
        by = decode_bytes(shape, cache, Qn)
        # the call's binding roof: min over HBM (its bytes at 8 TB/s) and bf16 MFMA (score and
        # value products of every query row against every kept coefficient, 2.5 PFLOP/s)
        rsum = int(cache.rank.to(torch.int64).sum())
        flop = 2.0 * 2 * (Qn * hpg) * G * rsum
        t_hbm = by / (HBM_PEAK_GBS * 1e9)
        t_mfma = flop / 2.5e15
        rows.append({"budget_pct": kappa, "r_min": r_min, "decode_ms": round(ms, 4),
                     "decode_GBps": round(by / (ms * 1e-3) / 1e9, 1), "decode_bytes": int(by),
                     "decode_GFLOP": round(flop / 1e9, 2),
                     "binding_roof": "hbm" if t_hbm >= t_mfma else "mfma",
                     "frac_of_binding_roof": round(max(t_hbm, t_mfma) / (ms * 1e-3), 4),
                     "rel_l2_err_varrate": err_v, "rel_l2_err_flat": err_f})
    main_row = next(r for r in rows if r["budget_pct"] == 20)
    result = {
        "metric": "compressed decode attn GB/s (% HBM peak), batch of 64 query-agnostic queries, 1 GPU",
        "value": main_row["decode_GBps"], "unit": "GB/s", "n_gpus": 1, "steps": 20, "warmup": 1,
        "ms_per_step": main_row["decode_ms"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (device draws, fresh Gaussian decode queries independent of the window)",
        "config": {"workload": f"agnostic_32k: 1 layer, {G} KV x {H} q heads, d 128, n {n}, w {w}, "
                               f"{Qn} queries per call"},
        "budgets": rows,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
