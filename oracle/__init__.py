"""VarRate CPU oracle -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg may import
this package.  The product path (``paper_2607_15498_amd``) never imports it and shares no
code with it.

Thin ctypes wrapper over ``varrate_oracle.c`` (plain C, fp64, OpenMP over independent
rows/tokens).  Each wrapper names the passage of the paper its C function follows; the
readings of open points are documented beside the C functions.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "varrate_oracle.c")
_LIB = os.path.join(_HERE, "libvarrate_oracle.so")

_f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
_u32p = np.ctypeslib.ndpointer(np.uint32, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS")
_i64 = ctypes.c_int64
_int = ctypes.c_int


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no fast-math, no fp contraction, OpenMP)."""
    if force or not os.path.exists(_LIB):
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
               "-fno-fast-math", "-fvisibility=hidden", "-Wall", "-o", _LIB, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        L.vro_budget.restype = _i64
        L.vro_budget.argtypes = [_i64, _i64, _i64, _i64]
        L.vro_threads.restype = _int
        L.vro_set_threads.restype = None
        L.vro_set_threads.argtypes = [_int]
        L.vro_salience.restype = None
        L.vro_salience.argtypes = [_i64, _int, _int, _int, _int, _f32p, _f32p, _f64p]
        L.vro_pool.restype = None
        L.vro_pool.argtypes = [_f64p, _i64, _f32p]
        L.vro_weights.restype = None
        L.vro_weights.argtypes = [_f32p, _i64, _u32p]
        L.vro_allocate.restype = _int
        L.vro_allocate.argtypes = [_u32p, _i64, _i64, _int, _int, _i32p,
                                   ctypes.POINTER(_i64), ctypes.POINTER(_i64),
                                   ctypes.POINTER(_i64)]
        L.vro_project.restype = None
        L.vro_project.argtypes = [_i64, _int, _int, _f32p, _f32p, _i32p, _int, _f32p]
        L.vro_half_round.restype = ctypes.c_float
        L.vro_half_round.argtypes = [ctypes.c_float]
        L.vro_quantize.restype = None
        L.vro_quantize.argtypes = [_i64, _int, _int, _f32p, _i32p, _int,
                                   np.ctypeslib.ndpointer(np.int8, flags="C_CONTIGUOUS"), _f32p, _f32p]
        L.vro_anchor_nearest.restype = None
        L.vro_anchor_nearest.argtypes = [_i64, _int, _int, _int, _int, _f32p, _f32p, _i32p, _f64p]
        L.vro_decode_anchor.restype = None
        L.vro_decode_anchor.argtypes = [_i64, _i64, _i64, _int, _int, _int, _int, _f32p, _f32p, _i32p, _i32p,
                                        _f32p, _f32p, _f32p, _f32p, _f32p, _f32p, _f32p, _f64p]
        L.vro_decode.restype = None
        L.vro_decode.argtypes = [_i64, _i64, _int, _int, _int, _f32p, _f32p, _i32p,
                                 _f32p, _f32p, _f32p, _f32p, _f32p, _f64p]
        L.vro_project_joint.restype = None
        L.vro_project_joint.argtypes = [_i64, _int, _int, _int, _f32p, _f32p, _f32p, _i32p, _int, _f32p]
        L.vro_decode_joint.restype = None
        L.vro_decode_joint.argtypes = [_i64, _i64, _int, _int, _int, _int, _f32p, _i32p, _f32p, _f32p,
                                       _f32p, _f32p, _f64p]
        L.vro_rope.restype = None
        L.vro_rope.argtypes = [_i64, _int, _int, _f32p, _i64p, _f32p, _int, _f64p]
        L.vro_decode_rope.restype = None
        L.vro_decode_rope.argtypes = [_i64, _i64, _int, _int, _int, _f32p, _f32p, _i32p,
                                      _f32p, _f32p, _f32p, _f32p, _f32p, _i64p, _f32p, _f64p]
        _lib = L
    return _lib


def threads() -> int:
    return int(lib().vro_threads())


def set_threads(n: int) -> None:
    """Thread count of the oracle's OpenMP loops from now on."""
    lib().vro_set_threads(int(n))


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def budget(n: int, d: int, w: int, kappa_pct: int) -> int:
    """Eq. (3), integer form: floor(kappa n d / 100) - w d."""
    return int(lib().vro_budget(n, d, w, kappa_pct))


def salience(K: np.ndarray, Qw: np.ndarray, H: int) -> np.ndarray:
    """Eq. (4): s_t for the coded tokens t < n - w.  K [n][G][d], Qw [w][H][d]."""
    n, G, d = K.shape
    w = Qw.shape[0]
    s = np.zeros(max(n - w, 0), np.float64)
    lib().vro_salience(n, G, H, d, w, _c(K, np.float32), _c(Qw, np.float32), s)
    return s


def pool(s: np.ndarray) -> np.ndarray:
    """Sec. 3.2 length-5 moving average, rounded to fp32."""
    s = _c(s, np.float64)
    out = np.zeros(s.shape[0], np.float32)
    lib().vro_pool(s, s.shape[0], out)
    return out


def weights(sbar: np.ndarray) -> np.ndarray:
    """Sec. 3.2 min-max normalisation as exact integer weights u_t in [1, 2^24 + 1]."""
    sbar = _c(sbar, np.float32)
    u = np.zeros(sbar.shape[0], np.uint32)
    lib().vro_weights(sbar, sbar.shape[0], u)
    return u


@dataclass
class Allocation:
    rank: np.ndarray   # int32 [N]
    k: int             # number of tokens capped at R
    M: int             # B - R k - r_min (N - k)
    Q: int             # sum of u over uncapped tokens


class BudgetError(ValueError):
    pass


def allocate(u: np.ndarray, B: int, r_min: int, R: int) -> Allocation:
    """Eq. (5) / Algorithm 1 water-filling + largest-remainder integer ranks."""
    u = _c(u, np.uint32)
    N = u.shape[0]
    rank = np.zeros(N, np.int32)
    k, M, Q = _i64(), _i64(), _i64()
    rc = lib().vro_allocate(u, N, B, r_min, R, rank, ctypes.byref(k), ctypes.byref(M),
                            ctypes.byref(Q))
    if rc != 0:
        raise BudgetError(f"infeasible budget B={B} for N={N}, r_min={r_min}, R={R}")
    return Allocation(rank, int(k.value), int(M.value), int(Q.value))


def project(X: np.ndarray, P: np.ndarray, rank: np.ndarray, storage: str) -> np.ndarray:
    """Eq. (6) projection + nested truncation, rounded to the storage type ('bf16'|'f32')."""
    n, G, d = X.shape
    out = np.zeros((n, G, d), np.float32)
    lib().vro_project(n, G, d, _c(X, np.float32), _c(P, np.float32), _c(rank, np.int32),
                      1 if storage == "bf16" else 0, out)
    return out


def decode(coefK, coefV, rank, Kx, Vx, PK, PV, q, H: int) -> np.ndarray:
    """Sec. 4.4 reconstruct-in-place decode for one query set q [H][d] -> [H][d] fp64."""
    N, G, d = coefK.shape
    n_exact = Kx.shape[0]
    out = np.zeros((H, d), np.float64)
    lib().vro_decode(N, n_exact, G, H, d, _c(coefK, np.float32), _c(coefV, np.float32),
                     _c(rank, np.int32), _c(Kx, np.float32), _c(Vx, np.float32),
                     _c(PK, np.float32), _c(PV, np.float32), _c(q, np.float32), out)
    return out


def half_round(x: float) -> float:
    """Nearest IEEE binary16 value of an fp32 value (ties to even), as a float."""
    return float(lib().vro_half_round(float(x)))


@dataclass
class Quantized:
    codes: np.ndarray    # int8 [N][G][d], zero past each rank
    scales: np.ndarray   # float32 [N][G][d/32] (binary16 values)
    deq: np.ndarray      # float32 [N][G][d] = codes * scale of their group


def quantize(coef: np.ndarray, rank: np.ndarray, bits: int) -> Quantized:
    """Sec. 3.3 "Composability": group-wise symmetric b-bit codes of stored coefficients
    (groups: one token, one head, 32 consecutive coordinates below its rank)."""
    n, G, d = coef.shape
    codes = np.zeros((n, G, d), np.int8)
    scales = np.zeros((n, G, (d + 31) // 32), np.float32)
    deq = np.zeros((n, G, d), np.float32)
    lib().vro_quantize(n, G, d, _c(coef, np.float32), _c(rank, np.int32), int(bits), codes, scales, deq)
    return Quantized(codes, scales, deq)


@dataclass
class Compressed:
    s: np.ndarray        # fp64 salience [N]
    sbar: np.ndarray     # fp32 pooled salience [N] (allocation input)
    u: np.ndarray        # uint32 weights [N]
    alloc: Allocation
    B: int
    coefK: np.ndarray    # [N][G][d] float32 holding storage-rounded values
    coefV: np.ndarray
    Kx: np.ndarray       # exact tail [w][G][d]
    Vx: np.ndarray


def compress(K, V, Qw, PK, PV, H: int, kappa_pct: int, r_min: int, storage: str,
             sbar: np.ndarray | None = None) -> Compressed:
    """Algorithm 1 for one layer (anchor-free, RoPE-free, per-head bases).

    ``sbar`` optionally replaces the salience stage (used to run the allocation on a
    supplied fp32 signal, e.g. a constant one for the uniform-rank codec)."""
    n, G, d = K.shape
    w = Qw.shape[0]
    N = n - w
    B = budget(n, d, w, kappa_pct)
    if sbar is None:
        s = salience(K, Qw, H)
        sb = pool(s)
    else:
        s = np.full(N, np.nan)
        sb = _c(sbar, np.float32)
    u = weights(sb)
    al = allocate(u, B, r_min, d)
    cK = project(K[:N], PK, al.rank, storage)
    cV = project(V[:N], PV, al.rank, storage)
    return Compressed(s, sb, u, al, B, cK, cV, np.ascontiguousarray(K[N:]),
                      np.ascontiguousarray(V[N:]))


# ---------------------------------------------------------------------------------------
# Sec. 3.1 "Residual codec" (Eq. 2), Algorithm 1: strided anchors kept exact, every other
# prefix token coded as its residual to the mean of its c nearest anchors.

def anchor_nearest(K: np.ndarray, V: np.ndarray, N: int, delta: int, c: int):
    """c nearest anchors (strided prefix tokens 0, delta, ... < N) of every prefix token by
    the exact Euclidean distance over the joint vector [k (all heads); v (all heads)];
    rows of anchors are -1.  Returns (nn [N][c] int32 anchor numbers, dist [N][c] fp64)."""
    n, G, d = K.shape
    nn = np.zeros((N, c), np.int32)
    dist = np.zeros((N, c), np.float64)
    lib().vro_anchor_nearest(N, G, d, delta, c, _c(K[:N], np.float32), _c(V[:N], np.float32), nn, dist)
    return nn, dist


def round_storage(x: np.ndarray, storage: str) -> np.ndarray:
    """Nearest bf16 (ties to even) for bf16 storage, fp32 otherwise."""
    x = np.ascontiguousarray(x, np.float32)
    if storage != "bf16":
        return x
    b = x.view(np.uint32)
    r = (b + (np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1)))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


@dataclass
class AnchorCompressed:
    coded: np.ndarray     # int64 [Nc] token index of each coded token (ascending)
    anchors: np.ndarray   # int64 [na] token index of each anchor
    nn: np.ndarray        # int32 [Nc][c] anchor numbers of each coded token's nearest anchors
    dist: np.ndarray      # fp64 [Nc][c] their distances
    sbar: np.ndarray      # fp32 [N] pooled salience over the whole prefix
    u: np.ndarray         # uint32 [Nc] weights of the coded tokens
    alloc: Allocation
    B: int
    resK: np.ndarray      # [Nc][G][d] residuals (rounded to the storage type)
    resV: np.ndarray
    coefK: np.ndarray     # [Nc][G][d] storage-rounded coefficients of the residuals
    coefV: np.ndarray
    Ka: np.ndarray        # anchor rows [na][G][d]
    Va: np.ndarray
    Kx: np.ndarray        # window rows [w][G][d]
    Vx: np.ndarray


def anchor_budget(n: int, d: int, w: int, kappa_pct: int, na: int) -> int:
    """Eq. (3) with n_ref = |E| = na + w: floor(kappa n d / 100) - (na + w) d."""
    return budget(n, d, w, kappa_pct) - na * d


def compress_anchor(K, V, Qw, PK, PV, H: int, kappa_pct: int, r_min: int, storage: str,
                    delta: int = 16, c: int = 4, sbar: np.ndarray | None = None) -> AnchorCompressed:
    """Algorithm 1 with the residual codec (per-head bases, no RoPE): anchors every delta
    prefix tokens and the window kept exact; salience and its pooling over the whole prefix,
    min-max and water-filling over the coded tokens only (budget net of the anchors); each
    coded token projected as its residual to the mean of its c nearest anchors."""
    n, G, d = K.shape
    w = Qw.shape[0]
    N = n - w
    anchors = np.arange(0, N, delta, dtype=np.int64)
    coded = np.setdiff1d(np.arange(N, dtype=np.int64), anchors)
    na, Nc = len(anchors), len(coded)
    B = anchor_budget(n, d, w, kappa_pct, na)
    sb = pool(salience(K, Qw, H)) if sbar is None else _c(sbar, np.float32)
    u = weights(sb[coded])
    al = allocate(u, B, r_min, d)
    nn_all, dist_all = anchor_nearest(K, V, N, delta, c)
    nn, dist = nn_all[coded], dist_all[coded]
    Ka, Va = np.ascontiguousarray(K[anchors]), np.ascontiguousarray(V[anchors])
    meanK = Ka[nn].astype(np.float64).mean(axis=1)       # [Nc][G][d]
    meanV = Va[nn].astype(np.float64).mean(axis=1)
    resK = round_storage(K[coded].astype(np.float64) - meanK, storage)
    resV = round_storage(V[coded].astype(np.float64) - meanV, storage)
    cK = project(resK, PK, al.rank, storage)
    cV = project(resV, PV, al.rank, storage)
    return AnchorCompressed(coded, anchors, nn, dist, sb, u, al, B, resK, resV, cK, cV, Ka, Va,
                            np.ascontiguousarray(K[N:]), np.ascontiguousarray(V[N:]))


def decode_anchor(ac: AnchorCompressed, PK, PV, q, H: int, Kx=None, Vx=None) -> np.ndarray:
    """Reconstruct-in-place decode with anchors: coded tokens rebuilt as their anchor mean
    plus the truncated projection, anchors and exact rows as stored (fp64)."""
    Nc, G, d = ac.coefK.shape
    Kx = ac.Kx if Kx is None else Kx
    Vx = ac.Vx if Vx is None else Vx
    out = np.zeros((H, d), np.float64)
    c = ac.nn.shape[1]
    lib().vro_decode_anchor(Nc, ac.Ka.shape[0], Kx.shape[0], G, H, d, c, _c(ac.coefK, np.float32),
                            _c(ac.coefV, np.float32), _c(ac.alloc.rank, np.int32), _c(ac.nn, np.int32),
                            _c(ac.Ka, np.float32), _c(ac.Va, np.float32), _c(Kx, np.float32), _c(Vx, np.float32),
                            _c(PK, np.float32), _c(PV, np.float32), _c(q, np.float32), out)
    return out


# ---------------------------------------------------------------------------------------
# Sec. 3.1 "Joint per-token vector", Algorithm 1 first and last steps: keys arrive with
# rotary position embedding (post-RoPE); the codec works on the un-rotated keys and the
# reconstruction is rotated back at each token's position.

def rope(X: np.ndarray, pos, theta: np.ndarray, sign: int = 1) -> np.ndarray:
    """Rotary embedding in the rotate-half layout (pair i = coordinates i and i + d/2) at
    positions pos [n_tok], angle sign * pos * theta[i]; sign -1 removes it.  fp64 out."""
    n, G, d = X.shape
    out = np.zeros((n, G, d), np.float64)
    lib().vro_rope(n, G, d, _c(X, np.float32), _c(np.broadcast_to(pos, (n,)), np.int64),
                   _c(theta, np.float32), int(sign), out)
    return out


def compress_rope(K, V, Qw, PK, PV, H: int, kappa_pct: int, r_min: int, storage: str,
                  theta: np.ndarray, sbar: np.ndarray | None = None) -> Compressed:
    """Algorithm 1 with rotary keys (anchor-free, per-head bases): salience on the
    post-RoPE keys and window queries as the model attends; each coded key is un-rotated at
    its position t (rounded to the storage type) before the projection; the window rows stay
    exact and post-RoPE."""
    n, G, d = K.shape
    w = Qw.shape[0]
    N = n - w
    B = budget(n, d, w, kappa_pct)
    if sbar is None:
        s = salience(K, Qw, H)
        sb = pool(s)
    else:
        s = np.full(N, np.nan)
        sb = _c(sbar, np.float32)
    u = weights(sb)
    al = allocate(u, B, r_min, d)
    Ku = round_storage(rope(K[:N], np.arange(N, dtype=np.int64), theta, -1), storage)
    cK = project(Ku, PK, al.rank, storage)
    cV = project(V[:N], PV, al.rank, storage)
    return Compressed(s, sb, u, al, B, cK, cV, np.ascontiguousarray(K[N:]),
                      np.ascontiguousarray(V[N:]))


def decode_rope(comp: Compressed, PK, PV, q, H: int, theta: np.ndarray, Kx=None, Vx=None) -> np.ndarray:
    """Reconstruct-in-place decode with rotary keys: coded keys rebuilt from their
    coefficients and re-rotated at their positions 0..N-1; exact rows and the query q [H][d]
    post-RoPE as given.  fp64 [H][d]."""
    N, G, d = comp.coefK.shape
    Kx = comp.Kx if Kx is None else Kx
    Vx = comp.Vx if Vx is None else Vx
    out = np.zeros((H, d), np.float64)
    lib().vro_decode_rope(N, Kx.shape[0], G, H, d, _c(comp.coefK, np.float32), _c(comp.coefV, np.float32),
                          _c(comp.alloc.rank, np.int32), _c(Kx, np.float32), _c(Vx, np.float32),
                          _c(PK, np.float32), _c(PV, np.float32), _c(q, np.float32),
                          np.arange(N, dtype=np.int64), _c(theta, np.float32), out)
    return out


# ---------------------------------------------------------------------------------------
# Sec. 3.1 Eq. (1) "Joint per-token vector" and "Shared basis": one basis W in R^{R x Dz},
# Dz = 2 G d, codes z_t = [k_t (all heads); v_t (all heads)]; a token at rank r costs r
# scalars, so Eq. (3) is B = floor(kappa n Dz / 100) - w Dz and ranks run r_min..R.

def project_joint(K: np.ndarray, V: np.ndarray, W: np.ndarray, rank: np.ndarray, storage: str) -> np.ndarray:
    """Eq. (6) with the shared basis: c_t = W z_t truncated to rank[t], storage-rounded.
    K, V [n][G][d]; W [R][2 G d] -> coef [n][R]."""
    n, G, d = K.shape
    R = W.shape[0]
    out = np.zeros((n, R), np.float32)
    lib().vro_project_joint(n, G, d, R, _c(K, np.float32), _c(V, np.float32), _c(W, np.float32),
                            _c(rank, np.int32), 1 if storage == "bf16" else 0, out)
    return out


def decode_joint(coef, rank, Kx, Vx, W, q, H: int) -> np.ndarray:
    """Reconstruct-in-place decode with the shared basis for one query set q [H][d] (fp64)."""
    N, R = coef.shape
    n_exact, G, d = Kx.shape
    out = np.zeros((H, d), np.float64)
    lib().vro_decode_joint(N, n_exact, G, H, d, R, _c(coef, np.float32), _c(rank, np.int32),
                           _c(Kx, np.float32), _c(Vx, np.float32), _c(W, np.float32), _c(q, np.float32), out)
    return out


@dataclass
class JointCompressed:
    sbar: np.ndarray     # fp32 pooled salience [N]
    u: np.ndarray        # uint32 weights [N]
    alloc: Allocation    # ranks in 0..R (joint units)
    B: int               # coded budget in joint units
    coef: np.ndarray     # [N][R] storage-rounded coefficients
    Kx: np.ndarray       # exact window rows [w][G][d]
    Vx: np.ndarray


def joint_budget(n: int, G: int, d: int, w: int, kappa_pct: int) -> int:
    """Eq. (3) in joint units: floor(kappa n Dz / 100) - w Dz, Dz = 2 G d."""
    return budget(n, 2 * G * d, w, kappa_pct)


def compress_joint(K, V, Qw, W, H: int, kappa_pct: int, r_min: int, storage: str,
                   sbar: np.ndarray | None = None) -> JointCompressed:
    """Algorithm 1 with the shared cross-head basis (no anchors, no RoPE): the salience,
    pooling and weights of the per-head codec, water-filling of the joint budget with cap
    R = W.shape[0], one coefficient row per token for every head and both K and V."""
    n, G, d = K.shape
    w = Qw.shape[0]
    N = n - w
    R = W.shape[0]
    B = joint_budget(n, G, d, w, kappa_pct)
    sb = pool(salience(K, Qw, H)) if sbar is None else _c(sbar, np.float32)
    u = weights(sb)
    al = allocate(u, B, r_min, R)
    coef = project_joint(K[:N], V[:N], W, al.rank, storage)
    return JointCompressed(sb, u, al, B, coef, np.ascontiguousarray(K[N:]), np.ascontiguousarray(V[N:]))
