"""VarRate variable-rank KV codec on MI355X: Python binding of libvarrate (HIP, gfx950).

Torch supplies device memory and the current stream; every step of the codec runs in the
HIP kernels behind the C ABI of ``include/varrate.h``.  There is no CPU fallback: the
functions raise when the library is missing or a call fails.

    shape = Shape(n=32768, G=8, H=32, w=32, r_min=16, kappa_pct=20, dtype="bf16")
    cache = compress(shape, K, V, Qw, PK, PV)          # Algorithm 1, one layer
    out = decode(shape, [cache], q, PK, PV)           # rank-space decode attention
"""
from __future__ import annotations

import ctypes
import dataclasses
from typing import List, Optional, Sequence

import torch

from . import _lib
from ._lib import CHUNK, COEF_PAD, HEAD_DIM  # noqa: F401

__all__ = ["VarRateError", "Shape", "Cache", "new_cache", "coded_budget", "salience", "allocate",
           "project", "compress", "append_exact", "decode", "decode_noalloc", "QCache", "new_qcache",
           "quantize", "decode_q", "anchor_search", "anchor_encode", "library"]


class VarRateError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"varrate error {code}: {msg}")
        self.code = code


def library():
    return _lib.load()


def _check(rc: int):
    if rc != 0:
        L = library()
        raise VarRateError(rc, f"{L.varrate_status_string(rc).decode()}: {L.varrate_last_error().decode()}")


@dataclasses.dataclass(frozen=True)
class Shape:
    n: int
    G: int
    H: int
    w: int
    r_min: int
    kappa_pct: int
    dtype: str = "bf16"
    d: int = HEAD_DIM
    anchor_stride: int = 0     # > 0: the residual codec with exact anchors every anchor_stride tokens
    rope_theta: tuple | None = None   # rotary keys: 64 per-pair frequencies (post-RoPE inputs)

    def c(self) -> _lib.Shape:
        th = (ctypes.c_float * 64)(*(self.rope_theta if self.rope_theta is not None else [0.0] * 64))
        return _lib.Shape(self.n, self.G, self.H, self.d, self.w, self.r_min, self.kappa_pct,
                          _lib.VARRATE_BF16 if self.dtype == "bf16" else _lib.VARRATE_F32,
                          self.anchor_stride, 1 if self.rope_theta is not None else 0, th)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    @property
    def na(self) -> int:
        """Anchors of the residual codec (0 without it)."""
        a = self.anchor_stride
        return (self.n - self.w + a - 1) // a if a else 0

    @property
    def N(self) -> int:
        """Coded tokens (the prefix minus its anchors)."""
        return self.n - self.w - self.na


@dataclasses.dataclass
class Cache:
    coef_k: torch.Tensor
    coef_v: torch.Tensor
    rank: torch.Tensor
    srank: torch.Tensor
    sidx: torch.Tensor
    chunk_off: torch.Tensor
    k_exact: torch.Tensor
    v_exact: torch.Tensor
    coef_stride: int
    cap: int
    n_exact: int = 0
    N: int = 0
    B: int = 0
    k_anchor: Optional[torch.Tensor] = None     # residual codec: [na][G][d]
    v_anchor: Optional[torch.Tensor] = None
    snn: Optional[torch.Tensor] = None          # [N][4] int16 anchor numbers (stored order)
    inv_off: Optional[torch.Tensor] = None      # [na + 1] int32
    inv_pos: Optional[torch.Tensor] = None      # [4 N] int32
    piece_off: Optional[torch.Tensor] = None    # [na + 1] int32
    piece_anchor: Optional[torch.Tensor] = None  # [4 N / 64 + na] int16
    na: int = 0

    def c(self) -> _lib.CacheC:
        ptr = lambda t: t.data_ptr() if t is not None else None
        return _lib.CacheC(self.coef_k.data_ptr(), self.coef_v.data_ptr(), self.rank.data_ptr(),
                           self.srank.data_ptr(), self.sidx.data_ptr(), self.chunk_off.data_ptr(),
                           self.k_exact.data_ptr(), self.v_exact.data_ptr(), self.coef_stride,
                           self.cap, self.n_exact, self.N, self.B, ptr(self.k_anchor), ptr(self.v_anchor),
                           ptr(self.snn), ptr(self.inv_off), ptr(self.inv_pos), ptr(self.piece_off),
                           ptr(self.piece_anchor), self.na)

    def _update(self, cc: _lib.CacheC):
        self.n_exact, self.N, self.B, self.na = int(cc.n_exact), int(cc.N), int(cc.B), int(cc.na)


def coded_budget(n: int, w: int, kappa_pct: int, d: int = HEAD_DIM) -> int:
    return int(library().varrate_coded_budget(n, d, w, kappa_pct))


def cache_bytes(shape: Shape, cap: int) -> _lib.CacheBytes:
    out = _lib.CacheBytes()
    _check(library().varrate_cache_bytes(ctypes.byref(shape.c()), cap, ctypes.byref(out)))
    return out


def new_cache(shape: Shape, cap: Optional[int] = None, device="cuda") -> Cache:
    """Allocate (torch) the device buffers of one compressed layer; `cap` exact slots."""
    cap = shape.w if cap is None else cap
    b = cache_bytes(shape, cap)
    dt = shape.torch_dtype
    G = shape.G
    return Cache(
        coef_k=torch.zeros((G, b.coef_stride), dtype=dt, device=device),
        coef_v=torch.zeros((G, b.coef_stride), dtype=dt, device=device),
        rank=torch.zeros(b.rank, dtype=torch.uint8, device=device)[: b.N],
        srank=torch.zeros(b.srank, dtype=torch.uint8, device=device)[: b.N],
        sidx=torch.zeros(b.N, dtype=torch.int32, device=device),
        chunk_off=torch.zeros(b.n_chunks + 1, dtype=torch.int32, device=device),
        k_exact=torch.zeros((G, cap, HEAD_DIM), dtype=dt, device=device),
        v_exact=torch.zeros((G, cap, HEAD_DIM), dtype=dt, device=device),
        coef_stride=int(b.coef_stride), cap=cap, n_exact=0, N=int(b.N), B=int(b.B),
        k_anchor=torch.zeros((b.na, G, HEAD_DIM), dtype=dt, device=device) if b.na else None,
        v_anchor=torch.zeros((b.na, G, HEAD_DIM), dtype=dt, device=device) if b.na else None,
        snn=torch.zeros((b.N, 4), dtype=torch.int16, device=device) if b.na else None,
        inv_off=torch.zeros(b.na + 1, dtype=torch.int32, device=device) if b.na else None,
        inv_pos=torch.zeros(4 * b.N, dtype=torch.int32, device=device) if b.na else None,
        piece_off=torch.zeros(b.na + 1, dtype=torch.int32, device=device) if b.na else None,
        piece_anchor=torch.zeros(4 * b.N // 64 + b.na, dtype=torch.int16, device=device) if b.na else None,
        na=int(b.na))


class _Workspaces:
    """Zero-initialised workspaces, one per (device, kind); kernels leave them zeroed."""

    def __init__(self):
        self._bufs = {}

    def get(self, kind: str, nbytes: int, device) -> torch.Tensor:
        dev = torch.device(device)
        key = (dev, kind)
        buf = self._bufs.get(key)
        if buf is None or buf.numel() < nbytes:
            buf = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=dev)
            self._bufs[key] = buf
        return buf


_WS = _Workspaces()


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev_ptr(t: Optional[torch.Tensor], dtype=None, name="tensor") -> int:
    if t is None:
        return 0
    if not t.is_cuda:
        raise VarRateError(_lib.VARRATE_EINVAL, f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise VarRateError(_lib.VARRATE_EINVAL, f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise VarRateError(_lib.VARRATE_EINVAL, f"{name} has dtype {t.dtype}, expected {dtype}")
    return t.data_ptr()


def _compress_ws(shape: Shape, device, workspace):
    need = int(library().varrate_compress_workspace_bytes(ctypes.byref(shape.c())))
    if need == 0:
        _check(library().varrate_cache_bytes(ctypes.byref(shape.c()), shape.w, ctypes.byref(_lib.CacheBytes())))
    ws = workspace if workspace is not None else _WS.get("compress", need, device)
    return ws, need


def salience(shape: Shape, K: torch.Tensor, Qw: torch.Tensor, sbar: Optional[torch.Tensor] = None,
             workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Sec. 3.2 Eq. (4) + 5-tap pooling: returns sbar [N] fp32 on the device."""
    if sbar is None:
        sbar = torch.empty(shape.n - shape.w, dtype=torch.float32, device=K.device)
    ws, _ = _compress_ws(shape, K.device, workspace)
    _check(library().varrate_salience(ctypes.byref(shape.c()), _dev_ptr(K, shape.torch_dtype, "K"),
                                      _dev_ptr(Qw, shape.torch_dtype, "Qw"),
                                      _dev_ptr(sbar, torch.float32, "sbar"), ws.data_ptr(), ws.numel(),
                                      _stream()))
    return sbar


def allocate(shape: Shape, sbar: torch.Tensor, cache: Cache, workspace: Optional[torch.Tensor] = None) -> Cache:
    """Sec. 3.2 Eq. (5): integer ranks (cache.rank) and chunk offsets from sbar [N] fp32."""
    ws, _ = _compress_ws(shape, sbar.device, workspace)
    cc = cache.c()
    _check(library().varrate_allocate(ctypes.byref(shape.c()), _dev_ptr(sbar, torch.float32, "sbar"),
                                      ctypes.byref(cc), ws.data_ptr(), ws.numel(), _stream()))
    cache._update(cc)
    return cache


def project(shape: Shape, K, V, PK, PV, cache: Cache, workspace: Optional[torch.Tensor] = None) -> Cache:
    """Sec. 3.3 Eq. (6): stored-order layout, truncated coefficients and exact window rows."""
    ws, _ = _compress_ws(shape, K.device, workspace)
    cc = cache.c()
    _check(library().varrate_project(ctypes.byref(shape.c()), _dev_ptr(K, shape.torch_dtype, "K"),
                                     _dev_ptr(V, shape.torch_dtype, "V"), _dev_ptr(PK, torch.float32, "PK"),
                                     _dev_ptr(PV, torch.float32, "PV"), ctypes.byref(cc), ws.data_ptr(),
                                     ws.numel(), _stream()))
    cache._update(cc)
    return cache


def compress(shape: Shape, K, V, Qw, PK, PV, cache: Optional[Cache] = None, cap: Optional[int] = None,
             sbar_out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None) -> Cache:
    """Algorithm 1 for one layer of one sequence (salience -> allocation -> projection)."""
    if cache is None:
        cache = new_cache(shape, cap, K.device)
    ws, _ = _compress_ws(shape, K.device, workspace)
    cc = cache.c()
    _check(library().varrate_compress(ctypes.byref(shape.c()), _dev_ptr(K, shape.torch_dtype, "K"),
                                      _dev_ptr(V, shape.torch_dtype, "V"), _dev_ptr(Qw, shape.torch_dtype, "Qw"),
                                      _dev_ptr(PK, torch.float32, "PK"), _dev_ptr(PV, torch.float32, "PV"),
                                      ctypes.byref(cc), _dev_ptr(sbar_out, torch.float32, "sbar_out"),
                                      ws.data_ptr(), ws.numel(), _stream()))
    cache._update(cc)
    return cache


def append_exact(shape: Shape, cache: Cache, k_new: torch.Tensor, v_new: torch.Tensor) -> Cache:
    """Append one decode-time token ([G][d]) to the exact slots."""
    cc = cache.c()
    _check(library().varrate_append_exact(ctypes.byref(shape.c()), ctypes.byref(cc),
                                          _dev_ptr(k_new, shape.torch_dtype, "k_new"),
                                          _dev_ptr(v_new, shape.torch_dtype, "v_new"), _stream()))
    cache._update(cc)
    return cache


PROBE_WGS = 4096


def read_probe(src: torch.Tensor, nbytes: int, sink: torch.Tensor) -> None:
    """Measurement aid: a plain streaming read of the first `nbytes` bytes of `src` (device
    memory) on the current stream; `sink` is a device int32 tensor of PROBE_WGS elements."""
    if sink.numel() < PROBE_WGS or not sink.is_cuda or sink.element_size() != 4:
        raise VarRateError(_lib.VARRATE_EINVAL, "sink: a device tensor of 4096 32-bit words")
    if nbytes > src.numel() * src.element_size():
        raise VarRateError(_lib.VARRATE_EINVAL, "nbytes past the end of src")
    _check(library().varrate_read_probe(_dev_ptr(src), int(nbytes), _dev_ptr(sink), _stream()))


def decode_workspace(shape: Shape, S: int, Q: int, device="cuda") -> torch.Tensor:
    need = int(library().varrate_decode_workspace_bytes(ctypes.byref(shape.c()), S, Q))
    return _WS.get(f"decode", need, device)


def decode(shape: Shape, caches: Sequence[Cache], q: torch.Tensor, PK, PV, out: Optional[torch.Tensor] = None,
           workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Rank-space decode attention.  q: [S][Q][H][d] (or [Q][H][d] for one cache)."""
    single = q.dim() == 3
    if single:
        q = q.unsqueeze(0)
    S, Q = int(q.shape[0]), int(q.shape[1])
    if len(caches) != S:
        raise VarRateError(_lib.VARRATE_EINVAL, f"{len(caches)} caches for {S} query sets")
    if out is None:
        out = torch.empty_like(q)
    arr = (_lib.CacheC * S)(*[c.c() for c in caches])
    ws = workspace if workspace is not None else decode_workspace(shape, S, Q, q.device)
    _check(library().varrate_decode_attn(ctypes.byref(shape.c()), arr, S, _dev_ptr(q, shape.torch_dtype, "q"), Q,
                                         _dev_ptr(PK, torch.float32, "PK"), _dev_ptr(PV, torch.float32, "PV"),
                                         _dev_ptr(out, shape.torch_dtype, "out"), ws.data_ptr(), ws.numel(),
                                         _stream()))
    return out[0] if single else out


def decode_noalloc(shape: Shape, caches: Sequence[Cache], q: torch.Tensor, PK, PV,
                   out: torch.Tensor) -> torch.Tensor:
    """Rank-space decode through varrate_decode_attn_noalloc: no workspace, the partial
    records go to the library's fixed per-device scratch (calls on one device must not
    overlap).  `out` must be preallocated ([S][Q][H][d] or [Q][H][d])."""
    single = q.dim() == 3
    if single:
        q, out = q.unsqueeze(0), out.unsqueeze(0)
    S, Q = int(q.shape[0]), int(q.shape[1])
    if len(caches) != S:
        raise VarRateError(_lib.VARRATE_EINVAL, f"{len(caches)} caches for {S} query sets")
    arr = (_lib.CacheC * S)(*[c.c() for c in caches])
    _check(library().varrate_decode_attn_noalloc(ctypes.byref(shape.c()), arr, S,
                                                 _dev_ptr(q, shape.torch_dtype, "q"), Q,
                                                 _dev_ptr(PK, torch.float32, "PK"),
                                                 _dev_ptr(PV, torch.float32, "PV"),
                                                 _dev_ptr(out, shape.torch_dtype, "out"), _stream()))
    return out[0] if single else out


@dataclasses.dataclass
class QCache:
    """b-bit codes of one compressed bf16 layer (Sec. 3.3 "Composability")."""
    code_k: torch.Tensor      # [G][q_stride] uint8
    code_v: torch.Tensor
    qchunk_off: torch.Tensor  # [n_chunks + 1] int32 (byte offsets)
    q_stride: int
    bits: int

    def c(self) -> _lib.QCacheC:
        return _lib.QCacheC(self.code_k.data_ptr(), self.code_v.data_ptr(), self.qchunk_off.data_ptr(),
                            self.q_stride, self.bits, 0)


def new_qcache(shape: Shape, bits: int, device="cuda") -> QCache:
    qs, qo = ctypes.c_int64(), ctypes.c_size_t()
    _check(library().varrate_qcache_bytes(ctypes.byref(shape.c()), int(bits), ctypes.byref(qs), ctypes.byref(qo)))
    return QCache(code_k=torch.zeros((shape.G, qs.value), dtype=torch.uint8, device=device),
                  code_v=torch.zeros((shape.G, qs.value), dtype=torch.uint8, device=device),
                  qchunk_off=torch.zeros(qo.value // 4, dtype=torch.int32, device=device),
                  q_stride=int(qs.value), bits=int(bits))


def quantize(shape: Shape, cache: Cache, bits: int, qcache: Optional[QCache] = None) -> QCache:
    """Group-wise b-bit codes of a compressed bf16 layer's coefficients."""
    if qcache is None:
        qcache = new_qcache(shape, bits, cache.coef_k.device)
    cc, qc = cache.c(), qcache.c()
    _check(library().varrate_quantize(ctypes.byref(shape.c()), ctypes.byref(cc), ctypes.byref(qc), _stream()))
    return qcache


def decode_q(shape: Shape, caches: Sequence[Cache], qcaches: Sequence[QCache], q: torch.Tensor, PK, PV,
             out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Rank-space decode over quantised coefficients (q: [S][Q][H][d] or [Q][H][d])."""
    single = q.dim() == 3
    if single:
        q = q.unsqueeze(0)
    S, Q = int(q.shape[0]), int(q.shape[1])
    if len(caches) != S or len(qcaches) != S:
        raise VarRateError(_lib.VARRATE_EINVAL, f"{len(caches)} caches / {len(qcaches)} qcaches for {S} query sets")
    if out is None:
        out = torch.empty_like(q)
    arr = (_lib.CacheC * S)(*[c.c() for c in caches])
    qarr = (_lib.QCacheC * S)(*[c.c() for c in qcaches])
    ws = workspace if workspace is not None else decode_workspace(shape, S, Q, q.device)
    _check(library().varrate_decode_attn_q(ctypes.byref(shape.c()), arr, qarr, S, _dev_ptr(q, shape.torch_dtype, "q"),
                                           Q, _dev_ptr(PK, torch.float32, "PK"), _dev_ptr(PV, torch.float32, "PV"),
                                           _dev_ptr(out, shape.torch_dtype, "out"), ws.data_ptr(), ws.numel(),
                                           _stream()))
    return out[0] if single else out


def anchor_search(shape: Shape, K: torch.Tensor, V: torch.Tensor, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Residual codec (Sec. 3.1 Eq. (2)): the 4 nearest anchors of every coded token,
    [N][4] int16 anchor numbers (nearest first)."""
    nn = torch.empty((shape.N, 4), dtype=torch.int16, device=K.device)
    ws, _ = _compress_ws(shape, K.device, workspace)
    _check(library().varrate_anchor_search(ctypes.byref(shape.c()), _dev_ptr(K, shape.torch_dtype, "K"),
                                           _dev_ptr(V, shape.torch_dtype, "V"), nn.data_ptr(), ws.data_ptr(),
                                           ws.numel(), _stream()))
    return nn


def anchor_encode(shape: Shape, K, V, sbar: torch.Tensor, nn: torch.Tensor, PK, PV, cache: Optional[Cache] = None,
                  cap: Optional[int] = None, workspace: Optional[torch.Tensor] = None) -> Cache:
    """Residual codec, given the prefix's pooled salience sbar [n - w] and the nearest
    anchors nn [N][4]: allocation over the coded tokens, residual projection, exact rows."""
    if cache is None:
        cache = new_cache(shape, cap, K.device)
    ws, _ = _compress_ws(shape, K.device, workspace)
    cc = cache.c()
    _check(library().varrate_anchor_encode(ctypes.byref(shape.c()), _dev_ptr(K, shape.torch_dtype, "K"),
                                           _dev_ptr(V, shape.torch_dtype, "V"), _dev_ptr(sbar, torch.float32, "sbar"),
                                           _dev_ptr(nn, torch.int16, "nn"), _dev_ptr(PK, torch.float32, "PK"),
                                           _dev_ptr(PV, torch.float32, "PV"), ctypes.byref(cc), ws.data_ptr(),
                                           ws.numel(), _stream()))
    cache._update(cc)
    return cache


# ---------------------------------------------------------------------------------------
# Shared cross-head basis (Sec. 3.1 Eq. (1) "Joint per-token vector" and "Shared basis"): one
# basis W [R][2 G d] codes z_t = [k_t (all heads); v_t (all heads)], one coefficient row per
# token for every head and both K and V, in original token order.

@dataclasses.dataclass
class JCache:
    coef: torch.Tensor
    rank: torch.Tensor          # [N] int16 (values 0..R)
    offset: torch.Tensor        # [N + 1] int32
    chunk_off: torch.Tensor
    k_exact: torch.Tensor
    v_exact: torch.Tensor
    coef_stride: int
    cap: int
    R: int
    n_exact: int = 0
    N: int = 0
    B: int = 0

    def c(self) -> _lib.JCacheC:
        return _lib.JCacheC(self.coef.data_ptr(), self.rank.data_ptr(), self.offset.data_ptr(),
                            self.chunk_off.data_ptr(), self.k_exact.data_ptr(), self.v_exact.data_ptr(),
                            self.coef_stride, self.cap, self.n_exact, self.N, self.B, self.R, 0)

    def _update(self, cc: _lib.JCacheC):
        self.n_exact, self.N, self.B = int(cc.n_exact), int(cc.N), int(cc.B)


def jcache_bytes(shape: Shape, R: int, cap: int) -> _lib.JCacheBytes:
    out = _lib.JCacheBytes()
    _check(library().varrate_jcache_bytes(ctypes.byref(shape.c()), R, cap, ctypes.byref(out)))
    return out


def new_jcache(shape: Shape, R: int, cap: Optional[int] = None, device="cuda") -> JCache:
    cap = shape.w if cap is None else cap
    b = jcache_bytes(shape, R, cap)
    dt = shape.torch_dtype
    return JCache(coef=torch.zeros(b.coef_stride, dtype=dt, device=device),
                  rank=torch.zeros(b.rank // 2, dtype=torch.int16, device=device)[: b.N],
                  offset=torch.zeros(b.N + 1, dtype=torch.int32, device=device),
                  chunk_off=torch.zeros(b.n_chunks + 1, dtype=torch.int32, device=device),
                  k_exact=torch.zeros((shape.G, cap, HEAD_DIM), dtype=dt, device=device),
                  v_exact=torch.zeros((shape.G, cap, HEAD_DIM), dtype=dt, device=device),
                  coef_stride=int(b.coef_stride), cap=cap, R=R, N=int(b.N), B=int(b.B))


def joint_compress(shape: Shape, K, V, Qw, W, R: Optional[int] = None, cache: Optional[JCache] = None,
                   cap: Optional[int] = None, sbar_out: Optional[torch.Tensor] = None,
                   workspace: Optional[torch.Tensor] = None) -> JCache:
    """Algorithm 1 with the shared basis W [R][2 G d] (fp32)."""
    R = int(W.shape[0]) if R is None else R
    if cache is None:
        cache = new_jcache(shape, R, cap, K.device)
    need = int(library().varrate_joint_compress_workspace_bytes(ctypes.byref(shape.c()), R))
    if need == 0:
        _check(library().varrate_jcache_bytes(ctypes.byref(shape.c()), R, cache.cap, None))
    ws = workspace if workspace is not None else _WS.get("jcompress", need, K.device)
    cc = cache.c()
    _check(library().varrate_joint_compress(ctypes.byref(shape.c()), _dev_ptr(K, shape.torch_dtype, "K"),
                                            _dev_ptr(V, shape.torch_dtype, "V"), _dev_ptr(Qw, shape.torch_dtype, "Qw"),
                                            _dev_ptr(W, torch.float32, "W"), ctypes.byref(cc),
                                            _dev_ptr(sbar_out, torch.float32, "sbar_out"), ws.data_ptr(), ws.numel(),
                                            _stream()))
    cache._update(cc)
    return cache


def joint_decode_workspace(shape: Shape, R: int, S: int, Q: int, device="cuda") -> torch.Tensor:
    need = int(library().varrate_joint_decode_workspace_bytes(ctypes.byref(shape.c()), R, S, Q))
    return _WS.get("jdecode", need, device)


def joint_decode(shape: Shape, caches: Sequence[JCache], q: torch.Tensor, W, out: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Decode attention over shared-basis caches.  q: [S][Q][H][d] (or [Q][H][d] for one cache)."""
    single = q.dim() == 3
    if single:
        q = q.unsqueeze(0)
    S, Q = int(q.shape[0]), int(q.shape[1])
    if len(caches) != S:
        raise VarRateError(_lib.VARRATE_EINVAL, f"{len(caches)} caches for {S} query sets")
    if out is None:
        out = torch.empty_like(q)
    arr = (_lib.JCacheC * S)(*[c.c() for c in caches])
    ws = workspace if workspace is not None else joint_decode_workspace(shape, caches[0].R, S, Q, q.device)
    _check(library().varrate_joint_decode_attn(ctypes.byref(shape.c()), arr, S, _dev_ptr(q, shape.torch_dtype, "q"),
                                               Q, _dev_ptr(W, torch.float32, "W"),
                                               _dev_ptr(out, shape.torch_dtype, "out"), ws.data_ptr(), ws.numel(),
                                               _stream()))
    return out[0] if single else out


def joint_append_exact(shape: Shape, cache: JCache, k_new: torch.Tensor, v_new: torch.Tensor) -> JCache:
    cc = cache.c()
    _check(library().varrate_joint_append_exact(ctypes.byref(shape.c()), ctypes.byref(cc),
                                                _dev_ptr(k_new, shape.torch_dtype, "k_new"),
                                                _dev_ptr(v_new, shape.torch_dtype, "v_new"), _stream()))
    cache._update(cc)
    return cache
