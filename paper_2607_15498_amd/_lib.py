"""ctypes view of libvarrate's C ABI (include/varrate.h).  Argument marshalling only."""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libvarrate.so")

VARRATE_OK, VARRATE_EINVAL, VARRATE_EBUDGET, VARRATE_EUNSUPPORTED, VARRATE_EHIP = 0, -1, -2, -3, -4
VARRATE_F32, VARRATE_BF16 = 0, 1
HEAD_DIM = 128
CHUNK = 256
COEF_PAD = 64
MAX_SEQS = 64
MAX_QROWS = 256

# every entry point include/varrate.h declares
EXPORTS = (
    "varrate_status_string", "varrate_last_error", "varrate_version", "varrate_coded_budget",
    "varrate_cache_bytes", "varrate_compress_workspace_bytes", "varrate_decode_workspace_bytes",
    "varrate_salience", "varrate_allocate", "varrate_project", "varrate_compress",
    "varrate_append_exact", "varrate_decode_attn", "varrate_decode_scratch_need",
    "varrate_decode_attn_noalloc", "varrate_qcache_bytes", "varrate_quantize", "varrate_decode_attn_q",
    "varrate_anchor_search", "varrate_anchor_encode",
    "varrate_jcache_bytes", "varrate_joint_compress_workspace_bytes", "varrate_joint_decode_workspace_bytes",
    "varrate_joint_compress", "varrate_joint_decode_attn", "varrate_joint_append_exact",
    "varrate_read_probe",
)
DECODE_SCRATCH_BYTES = 8 << 20


class Shape(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("G", ctypes.c_int32), ("H", ctypes.c_int32),
                ("d", ctypes.c_int32), ("w", ctypes.c_int32), ("r_min", ctypes.c_int32),
                ("kappa_pct", ctypes.c_int32), ("dtype", ctypes.c_int32), ("anchor_stride", ctypes.c_int32),
                ("rope", ctypes.c_int32), ("rope_theta", ctypes.c_float * 64)]


class CacheC(ctypes.Structure):
    _fields_ = [("coef_k", ctypes.c_void_p), ("coef_v", ctypes.c_void_p), ("rank", ctypes.c_void_p),
                ("srank", ctypes.c_void_p), ("sidx", ctypes.c_void_p), ("chunk_off", ctypes.c_void_p),
                ("k_exact", ctypes.c_void_p), ("v_exact", ctypes.c_void_p),
                ("coef_stride", ctypes.c_int64), ("cap", ctypes.c_int64), ("n_exact", ctypes.c_int64),
                ("N", ctypes.c_int64), ("B", ctypes.c_int64),
                ("k_anchor", ctypes.c_void_p), ("v_anchor", ctypes.c_void_p), ("snn", ctypes.c_void_p),
                ("inv_off", ctypes.c_void_p), ("inv_pos", ctypes.c_void_p), ("piece_off", ctypes.c_void_p),
                ("piece_anchor", ctypes.c_void_p), ("na", ctypes.c_int64)]


class QCacheC(ctypes.Structure):
    _fields_ = [("code_k", ctypes.c_void_p), ("code_v", ctypes.c_void_p), ("qchunk_off", ctypes.c_void_p),
                ("q_stride", ctypes.c_int64), ("bits", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class CacheBytes(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("B", ctypes.c_int64), ("n_chunks", ctypes.c_int64),
                ("coef_stride", ctypes.c_int64)] + \
               [(k, ctypes.c_size_t) for k in ("coef_k", "coef_v", "rank", "srank", "sidx",
                                               "chunk_off", "k_exact", "v_exact")] + \
               [("na", ctypes.c_int64)] + \
               [(k, ctypes.c_size_t) for k in ("k_anchor", "v_anchor", "snn", "inv_off", "inv_pos", "piece_off",
                                               "piece_anchor")]


class JCacheC(ctypes.Structure):
    _fields_ = [("coef", ctypes.c_void_p), ("rank", ctypes.c_void_p), ("offset", ctypes.c_void_p),
                ("chunk_off", ctypes.c_void_p), ("k_exact", ctypes.c_void_p), ("v_exact", ctypes.c_void_p),
                ("coef_stride", ctypes.c_int64), ("cap", ctypes.c_int64), ("n_exact", ctypes.c_int64),
                ("N", ctypes.c_int64), ("B", ctypes.c_int64), ("R", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class JCacheBytes(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("B", ctypes.c_int64), ("n_chunks", ctypes.c_int64),
                ("coef_stride", ctypes.c_int64)] + \
               [(k, ctypes.c_size_t) for k in ("coef", "rank", "offset", "chunk_off", "k_exact", "v_exact")]


_lib = None


def load() -> ctypes.CDLL:
    """Load the in-tree HIP library; fails loudly when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_15498_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    P = ctypes.POINTER
    sig = {
        "varrate_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "varrate_last_error": (ctypes.c_char_p, []),
        "varrate_version": (ctypes.c_int, []),
        "varrate_coded_budget": (i64, [i64, i32, i32, i32]),
        "varrate_cache_bytes": (ctypes.c_int, [P(Shape), i64, P(CacheBytes)]),
        "varrate_compress_workspace_bytes": (sz, [P(Shape)]),
        "varrate_decode_workspace_bytes": (sz, [P(Shape), i32, i32]),
        "varrate_salience": (ctypes.c_int, [P(Shape), vp, vp, vp, vp, sz, vp]),
        "varrate_allocate": (ctypes.c_int, [P(Shape), vp, P(CacheC), vp, sz, vp]),
        "varrate_project": (ctypes.c_int, [P(Shape), vp, vp, vp, vp, P(CacheC), vp, sz, vp]),
        "varrate_compress": (ctypes.c_int, [P(Shape), vp, vp, vp, vp, vp, P(CacheC), vp, vp, sz, vp]),
        "varrate_append_exact": (ctypes.c_int, [P(Shape), P(CacheC), vp, vp, vp]),
        "varrate_decode_attn": (ctypes.c_int, [P(Shape), P(CacheC), i32, vp, i32, vp, vp, vp, vp, sz, vp]),
        "varrate_decode_scratch_need": (sz, [P(Shape), i32, i32]),
        "varrate_decode_attn_noalloc": (ctypes.c_int, [P(Shape), P(CacheC), i32, vp, i32, vp, vp, vp, vp]),
        "varrate_qcache_bytes": (ctypes.c_int, [P(Shape), i32, P(i64), P(sz)]),
        "varrate_anchor_search": (ctypes.c_int, [P(Shape), vp, vp, vp, vp, sz, vp]),
        "varrate_anchor_encode": (ctypes.c_int, [P(Shape), vp, vp, vp, vp, vp, vp, P(CacheC), vp, sz, vp]),
        "varrate_quantize": (ctypes.c_int, [P(Shape), P(CacheC), P(QCacheC), vp]),
        "varrate_decode_attn_q": (ctypes.c_int, [P(Shape), P(CacheC), P(QCacheC), i32, vp, i32, vp, vp, vp, vp,
                                                 sz, vp]),
        "varrate_jcache_bytes": (ctypes.c_int, [P(Shape), i32, i64, P(JCacheBytes)]),
        "varrate_joint_compress_workspace_bytes": (sz, [P(Shape), i32]),
        "varrate_joint_decode_workspace_bytes": (sz, [P(Shape), i32, i32, i32]),
        "varrate_joint_compress": (ctypes.c_int, [P(Shape), vp, vp, vp, vp, P(JCacheC), vp, vp, sz, vp]),
        "varrate_joint_decode_attn": (ctypes.c_int, [P(Shape), P(JCacheC), i32, vp, i32, vp, vp, vp, sz, vp]),
        "varrate_joint_append_exact": (ctypes.c_int, [P(Shape), P(JCacheC), vp, vp, vp]),
        "varrate_read_probe": (ctypes.c_int, [vp, ctypes.c_size_t, vp, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L
