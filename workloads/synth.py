"""Seeded synthetic KV caches shaped like the paper's models (no trained weights here).

Recipe (one per layer x KV head x sequence):
  * keys      k_t = M_g (sigma * xi_t), xi ~ N(0, I_128), sigma_j = 1/j, M_g a seeded random
              orthogonal matrix; two seeded outlier channels are then scaled by 10.  A seeded
              5% subset of the coded tokens is "planted": k_t += a_t u_g with u_g a seeded unit
              vector per KV head and a_t ~ U(6, 10), so planted logits sit 6..10 nats above the
              background and attention is spiky (a few needle tokens draw almost all of it).
  * queries   q = sqrt(d) u_g + N(0, 0.1^2 I) for the observation window and for query-aware
              decode; query-agnostic decode draws q ~ N(0, s^2 I) with s set for logit std ~2.
  * values    low-rank plus noise  v = A_g eta + 0.1 eps  (A_g in R^{128x32}, entries
              N(0, 1/32)), or, for the tiny config, the key law without planting.
  * RoPE      (configs with rope="llama3") the drawn keys are pre-RoPE; the cache holds them
              rotated at their positions 0..n-1 in the rotate-half layout with Llama-3.1's
              frequencies (base 500000, long-context scaling factor 8), the window queries at
              n-w..n-1 and the decode queries at n.  The planted direction u_g then lives on
              the 16 slowest pairs, so planted tokens stay salient across the context.
  * basis     per (layer, KV head, K|V): eigenvectors of the uncentred second moment of 8192
              calibration draws from a disjoint seed, rows in descending-eigenvalue order,
              each row's largest-magnitude entry made positive.  The basis is an input to the
              codec (offline calibration), not part of the path under test.

Storage rounding of the inputs themselves (bf16 configs) is done here so that every consumer
sees identical values.  Nothing in this module computes salience, ranks, projections or
attention.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

MASK64 = (1 << 64) - 1

# Workload shapes: the paper's Llama-3.1-8B / Qwen2.5-7B attention geometry with synthetic
# contents (n = total cached prompt tokens, w = exact window = observation window).
CONFIGS: Dict[str, dict] = {
    "tiny": dict(layers=1, G=1, H=2, d=128, n=512, w=32, kappa=20, r_min=16,
                 dtype="f32", seed=0, values="keys", batch=1),
    "llama_32k": dict(layers=1, G=8, H=32, d=128, n=32768, w=32, kappa=20, r_min=16,
                      dtype="bf16", seed=1, values="lowrank", batch=1),
    "qwen_16k_stack": dict(layers=28, G=4, H=28, d=128, n=16384, w=32, kappa=20, r_min=16,
                           dtype="bf16", seed=2, values="lowrank", batch=8, steps=256),
    "llama_128k_stack": dict(layers=32, G=8, H=32, d=128, n=131072, w=32, kappa=20, r_min=16,
                             dtype="bf16", seed=3, values="lowrank", batch=1),
    "tiny_rope": dict(layers=1, G=1, H=2, d=128, n=512, w=32, kappa=20, r_min=16,
                      dtype="f32", seed=6, values="keys", batch=1, rope="llama3"),
    "llama_32k_rope": dict(layers=1, G=8, H=32, d=128, n=32768, w=32, kappa=20, r_min=16,
                           dtype="bf16", seed=7, values="lowrank", batch=1, rope="llama3"),
    "tiny_joint": dict(layers=1, G=1, H=2, d=128, n=512, w=32, kappa=20, r_min=16,
                       dtype="f32", seed=8, values="keys", batch=1, joint_R=256),
    "llama_32k_joint": dict(layers=1, G=8, H=32, d=128, n=32768, w=32, kappa=20, r_min=16,
                            dtype="bf16", seed=9, values="lowrank", batch=1, joint_R=1024),
    "agnostic_32k": dict(layers=1, G=8, H=32, d=128, n=32768, w=32, kappa=20, r_min=16,
                         dtype="bf16", seed=4, values="lowrank", batch=1, queries=64,
                         budgets=((10, 8), (20, 16), (40, 16))),
}

PLANT_FRACTION = 0.05
PLANT_LOGIT_LO, PLANT_LOGIT_HI = 6.0, 10.0
QUERY_NOISE = 0.1
OUTLIER_SCALE = 10.0
VALUE_RANK = 32
VALUE_NOISE = 0.1
CALIB_DRAWS = 8192
CALIB_SEED_OFFSET = 10 ** 6

# stream tags keep the per-purpose generators disjoint
_S_HEAD, _S_KEYS, _S_VALS, _S_QWIN, _S_QDEC, _S_VHEAD = 1, 2, 3, 4, 5, 6


def splitmix64(x: int) -> int:
    """SplitMix64 finaliser (Steele, Lea, Flood 2014)."""
    x = (x + 0x9E3779B97F4A7C15) & MASK64
    z = x
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def seed_for(base: int, layer: int = 0, head: int = 0, seq: int = 0, stream: int = 0) -> int:
    return splitmix64((base ^ (layer << 16) ^ (head << 8) ^ seq ^ (stream << 40)) & MASK64)


def _rng(*args) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed_for(*args)))


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    if not np.all(np.isfinite(a)):
        raise ValueError("bf16_round expects finite inputs")
    bits = a.view(np.uint32)
    out = bits + (np.uint32(0x7FFF) + ((bits >> np.uint32(16)) & np.uint32(1)))
    out &= np.uint32(0xFFFF0000)
    return out.view(np.float32).reshape(a.shape)


def _orthogonal(rng: np.random.Generator, d: int) -> np.ndarray:
    z = rng.standard_normal((d, d))
    q, r = np.linalg.qr(z)
    return q * np.sign(np.diag(r))[None, :]


@dataclasses.dataclass
class HeadModel:
    M: np.ndarray          # [d, d] orthogonal mixing of the decaying spectrum
    outliers: np.ndarray   # [2] outlier channel indices
    u: np.ndarray          # [d] planted / query direction (unit)
    A: np.ndarray          # [d, VALUE_RANK] value loading matrix
    Mv: np.ndarray         # [d, d] mixing for the key-law values (tiny config)
    outliers_v: np.ndarray


def rope_theta(kind: str, d: int = 128) -> np.ndarray:
    """Per-pair rotary frequencies (radians per position), float32 [d/2].  "llama3": base
    500000 with Llama-3.1's long-context scaling (factor 8, low/high frequency factors 1
    and 4, original context 8192): slow pairs divided by 8, fast pairs kept, a linear blend
    of the two in between."""
    if kind != "llama3":
        raise ValueError(kind)
    inv = 500000.0 ** (-np.arange(0, d, 2, dtype=np.float64) / d)
    factor, lo_f, hi_f, old = 8.0, 1.0, 4.0, 8192.0
    wavelen = 2.0 * np.pi / inv
    smooth = np.clip((old / wavelen - lo_f) / (hi_f - lo_f), 0.0, 1.0)
    out = (1.0 - smooth) * inv / factor + smooth * inv
    return out.astype(np.float32)


def _rotate(x: np.ndarray, pos: np.ndarray, theta: np.ndarray) -> np.ndarray:
    """x [m, ..., d] rotated at positions pos [m] (rotate-half pairs i, i + d/2), fp64."""
    h = x.shape[-1] // 2
    a = pos.astype(np.float64)[:, None] * theta.astype(np.float64)[None, :]
    shape = (len(pos),) + (1,) * (x.ndim - 2) + (h,)
    c, s = np.cos(a).reshape(shape), np.sin(a).reshape(shape)
    x0, x1 = x[..., :h], x[..., h:]
    return np.concatenate([x0 * c - x1 * s, x0 * s + x1 * c], axis=-1)


ROPE_SLOW_PAIRS = 16


def make_head_model(base: int, layer: int, head: int, d: int = 128, rope: bool = False) -> HeadModel:
    rng = _rng(base, layer, head, 0, _S_HEAD)
    M = _orthogonal(rng, d)
    outliers = rng.choice(d, size=2, replace=False)
    u = rng.standard_normal(d)
    if rope:      # only the slowest pairs: planted logits survive the relative rotation
        keep = np.zeros(d, bool)
        keep[d // 2 - ROPE_SLOW_PAIRS:d // 2] = True
        keep[d - ROPE_SLOW_PAIRS:] = True
        u = np.where(keep, u, 0.0)
    u /= np.linalg.norm(u)
    A = rng.standard_normal((d, VALUE_RANK)) / np.sqrt(VALUE_RANK)
    rv = _rng(base, layer, head, 0, _S_VHEAD)
    Mv = _orthogonal(rv, d)
    outliers_v = rv.choice(d, size=2, replace=False)
    return HeadModel(M, outliers, u, A, Mv, outliers_v)


def _spectrum(d: int) -> np.ndarray:
    return 1.0 / np.arange(1, d + 1, dtype=np.float64)


def _draw_keys(rng, hm: HeadModel, n_tok: int, n_coded: int, d: int):
    xi = rng.standard_normal((n_tok, d))
    k = (xi * _spectrum(d)[None, :]) @ hm.M.T
    k[:, hm.outliers] *= OUTLIER_SCALE
    n_plant = int(round(PLANT_FRACTION * n_coded))
    planted = np.sort(rng.choice(n_coded, size=n_plant, replace=False)) if n_plant else \
        np.zeros(0, dtype=np.int64)
    a = rng.uniform(PLANT_LOGIT_LO, PLANT_LOGIT_HI, size=n_plant)
    k[planted] += a[:, None] * hm.u[None, :]
    return k, planted


def _draw_values(rng, hm: HeadModel, n_tok: int, d: int, law: str):
    if law == "lowrank":
        eta = rng.standard_normal((n_tok, VALUE_RANK))
        eps = rng.standard_normal((n_tok, d))
        return eta @ hm.A.T + VALUE_NOISE * eps
    if law == "keys":
        xi = rng.standard_normal((n_tok, d))
        v = (xi * _spectrum(d)[None, :]) @ hm.Mv.T
        v[:, hm.outliers_v] *= OUTLIER_SCALE
        return v
    raise ValueError(law)


def _window_law_queries(rng, hm_of_head, n_q: int, H: int, d: int) -> np.ndarray:
    q = np.empty((n_q, H, d))
    for h in range(H):
        q[:, h, :] = np.sqrt(d) * hm_of_head[h].u[None, :] + \
            QUERY_NOISE * rng.standard_normal((n_q, d))
    return q


def calibration_basis(base: int, layer: int, head: int, hm: HeadModel, d: int,
                      values_law: str):
    """Offline PCA bases (P_K, P_V), each [d, d] float32, rows = directions, descending."""
    out = []
    for kind in ("k", "v"):
        rng = _rng(base + CALIB_SEED_OFFSET, layer, head, 0, _S_KEYS if kind == "k" else _S_VALS)
        if kind == "k":
            x, _ = _draw_keys(rng, hm, CALIB_DRAWS, CALIB_DRAWS, d)
        else:
            x = _draw_values(rng, hm, CALIB_DRAWS, d, values_law)
        c = x.T @ x / CALIB_DRAWS
        evals, evecs = np.linalg.eigh(c)
        order = np.argsort(-evals, kind="stable")
        P = evecs[:, order].T.copy()
        for j in range(d):
            i = int(np.argmax(np.abs(P[j])))
            if P[j, i] < 0:
                P[j] = -P[j]
        out.append(P.astype(np.float32))
    return out[0], out[1]


def joint_calibration_basis(cfg: dict, layer: int, head_models, R: int) -> np.ndarray:
    """Offline shared basis (Sec. 3.1 "Shared basis"): the top-R eigenvectors of the uncentred
    second moment of 8192 calibration joint vectors z = [k (all heads); v (all heads)], drawn
    from the same disjoint seeds as the per-head bases; rows in descending-eigenvalue order,
    each row's largest-magnitude entry positive.  float32 [R][2 G d]."""
    G, d = cfg["G"], cfg["d"]
    base = cfg["seed"]
    Z = np.empty((CALIB_DRAWS, 2 * G * d))
    for g in range(G):
        hm = head_models[g]
        rk = _rng(base + CALIB_SEED_OFFSET, layer, g, 0, _S_KEYS)
        rv = _rng(base + CALIB_SEED_OFFSET, layer, g, 0, _S_VALS)
        Z[:, g * d:(g + 1) * d], _ = _draw_keys(rk, hm, CALIB_DRAWS, CALIB_DRAWS, d)
        Z[:, (G + g) * d:(G + g + 1) * d] = _draw_values(rv, hm, CALIB_DRAWS, d, cfg["values"])
    c = Z.T @ Z / CALIB_DRAWS
    evals, evecs = np.linalg.eigh(c)
    order = np.argsort(-evals, kind="stable")[:R]
    W = evecs[:, order].T.copy()
    for j in range(R):
        i = int(np.argmax(np.abs(W[j])))
        if W[j, i] < 0:
            W[j] = -W[j]
    return W.astype(np.float32)


@dataclasses.dataclass
class LayerInputs:
    K: np.ndarray      # [n, G, d] float32 (values exactly representable in the storage dtype)
    V: np.ndarray      # [n, G, d]
    Qw: np.ndarray     # [w, H, d] observation-window queries
    q: np.ndarray      # [Q, H, d] decode queries
    PK: np.ndarray     # [G, d, d] float32, rows = basis directions
    PV: np.ndarray     # [G, d, d]
    planted: list      # per KV head: planted coded-token indices
    cfg: dict
    theta: Optional[np.ndarray] = None   # rotary frequencies [d/2] (RoPE configs), else None
    W: Optional[np.ndarray] = None       # shared cross-head basis [R][2 G d] (joint configs), else None


def decode_queries(cfg: dict, layer: int, seq: int, n_q: int, law: str,
                   head_models, K: Optional[np.ndarray] = None) -> np.ndarray:
    G, H, d = cfg["G"], cfg["H"], cfg["d"]
    rng = _rng(cfg["seed"], layer, 0, seq, _S_QDEC)
    hm_of_head = [head_models[h // (H // G)] for h in range(H)]
    if law == "aware":
        q = _window_law_queries(rng, hm_of_head, n_q, H, d)
    elif law == "agnostic":
        assert K is not None
        rms = float(np.sqrt(np.mean(np.sum(K.astype(np.float64) ** 2, axis=-1))))
        s = 2.0 * np.sqrt(d) / rms
        q = s * rng.standard_normal((n_q, H, d))
    else:
        raise ValueError(law)
    return q


def make_layer(cfg: dict, layer: int = 0, seq: int = 0, n_queries: int = 1,
               query_law: str = "aware", n: Optional[int] = None,
               with_basis: bool = True) -> LayerInputs:
    """Draw one layer of one sequence.  ``n`` overrides the config's prompt length.  Configs
    with ``joint_R`` also carry the shared cross-head basis of that many rows."""
    G, H, d, w = cfg["G"], cfg["H"], cfg["d"], cfg["w"]
    n = cfg["n"] if n is None else n
    base = cfg["seed"]
    N = n - w
    rope = cfg.get("rope")
    hms = [make_head_model(base, layer, g, d, rope=bool(rope)) for g in range(G)]
    K = np.empty((n, G, d))
    V = np.empty((n, G, d))
    planted = []
    for g in range(G):
        k, p = _draw_keys(_rng(base, layer, g, seq, _S_KEYS), hms[g], n, max(N, 0), d)
        K[:, g, :] = k
        planted.append(p)
        V[:, g, :] = _draw_values(_rng(base, layer, g, seq, _S_VALS), hms[g], n, d, cfg["values"])
    hm_of_head = [hms[h // (H // G)] for h in range(H)]
    Qw = _window_law_queries(_rng(base, layer, 0, seq, _S_QWIN), hm_of_head, w, H, d)
    q = decode_queries(cfg, layer, seq, n_queries, query_law, hms, K)
    theta = None
    if rope:
        theta = rope_theta(rope, d)
        K = _rotate(K, np.arange(n), theta)
        Qw = _rotate(Qw, np.arange(N, n), theta)
        q = _rotate(q, np.full(q.shape[0], n), theta)
    rnd = bf16_round if cfg["dtype"] == "bf16" else (lambda a: a.astype(np.float32))
    K, V, Qw, q = (rnd(a.astype(np.float32)) for a in (K, V, Qw, q))
    if with_basis:
        PK = np.empty((G, d, d), np.float32)
        PV = np.empty((G, d, d), np.float32)
        for g in range(G):
            PK[g], PV[g] = calibration_basis(base, layer, g, hms[g], d, cfg["values"])
    else:
        PK = PV = None
    W = joint_calibration_basis(cfg, layer, hms, cfg["joint_R"]) if with_basis and cfg.get("joint_R") else None
    return LayerInputs(K, V, Qw, q, PK, PV, planted, cfg, theta, W)
