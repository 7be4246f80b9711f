"""fp64 oracle for causal GQA attention through the paged KV pool.

TEST INFRASTRUCTURE (see the package docstring). A ctypes wrapper over
``pcr_oracle.c``; the definition it computes is stated there (Sec. 2.2: the
reused-prefix output of a suffix row equals full prefill's output for that row).
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import build as _build

_lib = None


def open_library(path):
    """ctypes handle on an oracle library at ``path`` with argument types set."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32 = ctypes.c_int32
    i64 = ctypes.c_int64
    lib.pcr_oracle_attention.argtypes = [P, i32, i32, i32, i32, P, P, i64, P, i32, P, P, i32,
                                         ctypes.c_double, P]
    lib.pcr_oracle_attention.restype = ctypes.c_int
    lib.pcr_oracle_attention_rows.argtypes = [P, i32, i32, i32, i32, P, P, i64, P, i32, P, P,
                                              i32, ctypes.c_double, P, i64, P]
    lib.pcr_oracle_attention_rows.restype = ctypes.c_int
    lib.pcr_oracle_num_threads.argtypes = []
    lib.pcr_oracle_num_threads.restype = ctypes.c_int
    lib.pcr_oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.pcr_oracle_set_num_threads.restype = None
    return lib


def _load():
    global _lib
    if _lib is None:
        _lib = open_library(_build.require_built())
    return _lib


def num_threads() -> int:
    return int(_load().pcr_oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads for the following oracle calls (timing runs only; results do not depend
    on it: every output row is computed by one thread in a fixed order)."""
    _load().pcr_oracle_set_num_threads(int(n))


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def attention(q, pool_k, pool_v, block_tables, prefix_lens, cu_suffix, num_kv_heads,
              block_size=16, sm_scale=None, rows=None, lib=None):
    """Oracle output in float64.

    q            uint16 [T][Hq][d]  (bf16 bits)
    pool_k/v     uint16 [num_blocks][Hkv][block_size*d]  (bf16 bits, layout in pcr_oracle.c)
    block_tables int32 [B][max_blocks]
    prefix_lens  int32 [B]; cu_suffix int32 [B+1]
    rows         None for every (t, h); else int32 [n][2] of (token, q head)
    lib          None for the built oracle; a handle from open_library otherwise
    Returns float64 [T][Hq][d], or [n][d] for a row list.
    """
    lib = _load() if lib is None else lib
    q, qp = _c(q, np.uint16)
    T, Hq, d = q.shape
    pool_k, kp = _c(pool_k, np.uint16)
    pool_v, vp = _c(pool_v, np.uint16)
    nb = pool_k.shape[0]
    bt, btp = _c(block_tables, np.int32)
    if bt.ndim != 2:
        raise ValueError("block_tables must be 2-D")
    pl, plp = _c(prefix_lens, np.int32)
    cu, cup = _c(cu_suffix, np.int32)
    B = pl.shape[0]
    if sm_scale is None:
        sm_scale = 1.0 / np.sqrt(d)
    if rows is None:
        out = np.empty((T, Hq, d), np.float64)
        rc = lib.pcr_oracle_attention(qp, Hq, num_kv_heads, d, block_size, kp, vp, nb, btp,
                                      bt.shape[1], plp, cup, B, float(sm_scale),
                                      out.ctypes.data_as(ctypes.c_void_p))
    else:
        rw, rwp = _c(rows, np.int32)
        rw = rw.reshape(-1, 2)
        out = np.empty((rw.shape[0], d), np.float64)
        rc = lib.pcr_oracle_attention_rows(qp, Hq, num_kv_heads, d, block_size, kp, vp, nb, btp,
                                           bt.shape[1], plp, cup, B, float(sm_scale), rwp,
                                           rw.shape[0], out.ctypes.data_as(ctypes.c_void_p))
    if rc != 0:
        raise ValueError(f"oracle attention failed with code {rc}")
    return out
