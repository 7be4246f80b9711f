"""Thin ctypes binding over libpcr.so with the C ABI's names (include/pcr.h).

Argument marshalling only: tensors become pointers and sizes, streams become
hipStream_t handles; every step runs inside the library. If libpcr.so is not
built, or the library reports an error, these functions raise.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpcr.so")

PCR_OK = 0
PCR_ERR_INVALID_ARG = -1
PCR_ERR_UNSUPPORTED = -2
PCR_ERR_NOT_PINNED = -3
PCR_ERR_HIP = -4

DECODE_NOALLOC_SCRATCH_BYTES = 16 << 20   # PCR_DECODE_NOALLOC_SCRATCH_BYTES

LOAD_AUTO = 0
LOAD_DMA_BATCH = 1
LOAD_DMA_PER_BLOCK = 2
LOAD_KERNEL_PULL = 3
LOAD_DMA_STAGED = 4
LOAD_METHODS = {"auto": LOAD_AUTO, "dma_batch": LOAD_DMA_BATCH, "dma_per_block": LOAD_DMA_PER_BLOCK,
                "kernel_pull": LOAD_KERNEL_PULL, "dma_staged": LOAD_DMA_STAGED}

EXPORTS = ["pcr_plan", "pcr_plan_offload", "pcr_load_kv_layer", "pcr_load_kv_layer_method",
           "pcr_offload_kv_layer", "pcr_offload_kv_layer_method", "pcr_offload_kv_layer_staged",
           "pcr_load_kv_layer_staged", "pcr_append_kv",
           "pcr_prefix_prefill_attn", "pcr_prefill_attn_set_schedule", "pcr_decode_attn", "pcr_decode_attn_noalloc", "pcr_decode_attn_workspace_size", "pcr_gather_kv", "pcr_pipeline_run", "pcr_pipeline_run_staged",
           "pcr_pipeline_run_offload", "pcr_pipeline_run_offload_staged",
           "pcr_store_open", "pcr_store_write_async", "pcr_store_read_async", "pcr_store_wait",
           "pcr_store_poll", "pcr_store_stats", "pcr_store_close", "pcr_last_error", "pcr_version"]


class PcrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libpcr status {status}: {message}")
        self.status = status


class _Pool(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("num_blocks", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32)]


class _Host(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("num_blocks", ctypes.c_int64),
                ("block_size", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32)]


class _LayerIO(ctypes.Structure):
    _fields_ = [("host", _Host), ("pool", _Pool), ("q", ctypes.c_void_p), ("k_new", ctypes.c_void_p),
                ("v_new", ctypes.c_void_p), ("out", ctypes.c_void_p)]


class _Batch(ctypes.Structure):
    _fields_ = [("src_blocks", ctypes.c_void_p), ("dst_blocks", ctypes.c_void_p), ("n_pairs", ctypes.c_int32),
                ("slot_mapping", ctypes.c_void_p), ("T", ctypes.c_int32), ("block_tables", ctypes.c_void_p),
                ("max_blocks", ctypes.c_int32), ("prefix_lens", ctypes.c_void_p), ("cu_suffix", ctypes.c_void_p),
                ("host_prefix_lens", ctypes.c_void_p), ("host_cu_suffix", ctypes.c_void_p),
                ("B", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("sm_scale", ctypes.c_float)]


_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2603_23049_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.pcr_plan.argtypes = [i32, P, P, P, i32, P, i32, i32, P, P, i32, P, P, P]
        L.pcr_load_kv_layer.argtypes = [ctypes.POINTER(_Host), P, ctypes.POINTER(_Pool), P, i32, P]
        L.pcr_load_kv_layer_method.argtypes = [ctypes.POINTER(_Host), P, ctypes.POINTER(_Pool), P, i32,
                                               ctypes.c_int, P]
        L.pcr_append_kv.argtypes = [ctypes.POINTER(_Pool), P, P, P, i32, P]
        L.pcr_prefix_prefill_attn.argtypes = [P, ctypes.POINTER(_Pool), P, i32, P, P, P, P, i32, i32,
                                              ctypes.c_float, P, P]
        L.pcr_prefill_attn_set_schedule.argtypes = [i32]
        L.pcr_decode_attn.argtypes = [P, ctypes.POINTER(_Pool), P, i32, P, P, i32, i32, ctypes.c_float, P, P,
                                      i64, P]
        L.pcr_decode_attn_noalloc.argtypes = [P, ctypes.POINTER(_Pool), P, i32, P, P, i32, i32, ctypes.c_float, P,
                                              P]
        L.pcr_decode_attn_workspace_size.argtypes = [i32, i32, i32, i32, i32, ctypes.POINTER(ctypes.c_int64)]
        L.pcr_gather_kv.argtypes = [ctypes.POINTER(_Pool), P, i32, P, P, i32, i32, P, P, P]
        L.pcr_pipeline_run.argtypes = [ctypes.POINTER(_LayerIO), i32, ctypes.POINTER(_Batch), ctypes.c_int, P, P,
                                       P]
        L.pcr_pipeline_run_staged.argtypes = [ctypes.POINTER(_LayerIO), i32, ctypes.POINTER(_Batch), P, i64, P, P,
                                              P, P]
        L.pcr_pipeline_run_offload_staged.argtypes = [ctypes.POINTER(_LayerIO), ctypes.POINTER(_Host), i32,
                                                      ctypes.POINTER(_Batch), P, P, i32, ctypes.c_int, P, i64, P,
                                                      i64, P, P, P, P, P]
        L.pcr_plan_offload.argtypes = [i32, P, P, P, i32, i32, i32, i32, P, P, i32, P]
        L.pcr_offload_kv_layer.argtypes = [ctypes.POINTER(_Pool), P, ctypes.POINTER(_Host), P, i32, P]
        L.pcr_offload_kv_layer_method.argtypes = [ctypes.POINTER(_Pool), P, ctypes.POINTER(_Host), P, i32,
                                                  ctypes.c_int, P]
        L.pcr_offload_kv_layer_staged.argtypes = [ctypes.POINTER(_Pool), P, ctypes.POINTER(_Host), P, i32, P, i64,
                                                  P]
        L.pcr_load_kv_layer_staged.argtypes = [ctypes.POINTER(_Host), P, ctypes.POINTER(_Pool), P, i32, P, i64, P]
        L.pcr_pipeline_run_offload.argtypes = [ctypes.POINTER(_LayerIO), ctypes.POINTER(_Host), i32,
                                               ctypes.POINTER(_Batch), P, P, i32, ctypes.c_int, ctypes.c_int, P,
                                               i64, P, P, P, P]
        L.pcr_store_open.argtypes = [ctypes.c_char_p, i64, i32, ctypes.POINTER(ctypes.c_void_p)]
        L.pcr_store_write_async.argtypes = [P, i64, P]
        L.pcr_store_read_async.argtypes = [P, i64, P]
        L.pcr_store_wait.argtypes = [P, i64]
        L.pcr_store_poll.argtypes = [P, i64, P]
        L.pcr_store_stats.argtypes = [P, P, P, P, P]
        L.pcr_store_close.argtypes = [P]
        for name in EXPORTS:
            if name not in ("pcr_last_error", "pcr_version"):
                getattr(L, name).restype = ctypes.c_int
        L.pcr_last_error.restype = ctypes.c_char_p
        L.pcr_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(status: int):
    if status != PCR_OK:
        raise PcrError(status, lib().pcr_last_error().decode())


def last_error() -> str:
    return lib().pcr_last_error().decode()


def version() -> str:
    return lib().pcr_version().decode()


# ---------------------------------------------------------------------------
# marshalling helpers
# ---------------------------------------------------------------------------

def _ptr(x) -> Optional[int]:
    """Address of a torch tensor or numpy array (None stays None)."""
    if x is None:
        return None
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _i32_host(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _numel(x) -> int:
    return int(x.size) if isinstance(x, np.ndarray) else int(x.numel())


def _need(x, n: int, what: str):
    """The library reads device arrays by the lengths it is given, which it cannot check
    against the allocations: refuse, before the call, a tensor shorter than that."""
    if x is not None and _numel(x) < n:
        raise ValueError(f"{what} holds {_numel(x)} elements, the call reads {n}")


@dataclass
class KVPool:
    """One layer's pool: k and v are device tensors of 2-byte elements,
    shape [num_blocks][num_kv_heads][block_size*head_dim]."""
    k: "object"
    v: "object"
    num_kv_heads: int
    head_dim: int
    block_size: int = 16

    @property
    def num_blocks(self) -> int:
        return int(self.k.shape[0])

    def c(self) -> _Pool:
        return _Pool(_ptr(self.k), _ptr(self.v), self.num_blocks, self.block_size, self.num_kv_heads, self.head_dim)


@dataclass
class HostKV:
    """One layer's pinned host store (same per-block layout as the pool)."""
    k: "object"
    v: "object"
    num_kv_heads: int
    head_dim: int
    block_size: int = 16

    @property
    def num_blocks(self) -> int:
        return int(self.k.shape[0])

    def c(self) -> _Host:
        return _Host(_ptr(self.k), _ptr(self.v), self.num_blocks, self.block_size, self.num_kv_heads, self.head_dim)


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------

def plan(prefix_lens: Sequence[int], suffix_lens: Sequence[int], block_tables, host_blocks, block_size: int = 16):
    """pcr_plan: returns (src_blocks, dst_blocks, slot_mapping, cu_suffix) as int32 numpy arrays."""
    pl, sl = _i32_host(prefix_lens), _i32_host(suffix_lens)
    bt, hb = _i32_host(block_tables), _i32_host(host_blocks)
    B = int(pl.shape[0])
    if bt.ndim != 2 or hb.ndim != 2 or bt.shape[0] != B or hb.shape[0] != B:
        raise ValueError("block_tables and host_blocks must be [B][*]")
    cap = int(sum(-(-int(p) // block_size) for p in pl))
    src = np.zeros(max(cap, 1), np.int32)
    dst = np.zeros(max(cap, 1), np.int32)
    T = int(sl.sum())
    slots = np.zeros(max(T, 1), np.int32)
    cu = np.zeros(B + 1, np.int32)
    n = ctypes.c_int32(0)
    _check(lib().pcr_plan(B, _ptr(pl), _ptr(sl), _ptr(bt), bt.shape[1], _ptr(hb), hb.shape[1], block_size,
                          _ptr(src), _ptr(dst), cap, ctypes.addressof(n), _ptr(slots), _ptr(cu)))
    return src[:n.value].copy(), dst[:n.value].copy(), slots[:T].copy(), cu


def load_kv_layer(src: HostKV, src_blocks, dst: KVPool, dst_blocks, method: str = "auto", stream=None,
                  workspace=None):
    """pcr_load_kv_layer_method (or _staged with method="dma_staged" and a device workspace
    tensor): enqueue the host-to-pool block copies on `stream`."""
    sb, db = _i32_host(src_blocks), _i32_host(dst_blocks)
    if sb.shape != db.shape:
        raise ValueError("src_blocks and dst_blocks differ in length")
    h, p = src.c(), dst.c()
    if method == "dma_staged":
        ws_bytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
        _check(lib().pcr_load_kv_layer_staged(ctypes.byref(h), _ptr(sb), ctypes.byref(p), _ptr(db),
                                              int(sb.shape[0]), _ptr(workspace), ws_bytes, _stream(stream)))
        return
    _check(lib().pcr_load_kv_layer_method(ctypes.byref(h), _ptr(sb), ctypes.byref(p), _ptr(db), int(sb.shape[0]),
                                          LOAD_METHODS[method], _stream(stream)))


def plan_offload(prefix_lens: Sequence[int], suffix_lens: Sequence[int], block_tables, block_size: int = 16,
                 chunk_tokens: int = 256, first_dst_block: int = 0):
    """pcr_plan_offload: returns (src pool blocks, dst host blocks) of the whole computed
    chunks of every sequence, as int32 numpy arrays."""
    pl, sl = _i32_host(prefix_lens), _i32_host(suffix_lens)
    bt = _i32_host(block_tables)
    B = int(pl.shape[0])
    if bt.ndim != 2 or bt.shape[0] != B:
        raise ValueError("block_tables must be [B][*]")
    cap = int(sum((int(p) + int(s)) // block_size for p, s in zip(pl, sl)))
    src = np.zeros(max(cap, 1), np.int32)
    dst = np.zeros(max(cap, 1), np.int32)
    n = ctypes.c_int32(0)
    _check(lib().pcr_plan_offload(B, _ptr(pl), _ptr(sl), _ptr(bt), bt.shape[1], block_size, chunk_tokens,
                                  first_dst_block, _ptr(src), _ptr(dst), cap, ctypes.addressof(n)))
    return src[:n.value].copy(), dst[:n.value].copy()


def offload_kv_layer(src: KVPool, src_blocks, dst: HostKV, dst_blocks, method: str = "auto", stream=None,
                     workspace=None):
    """pcr_offload_kv_layer_method (or _staged with method="dma_staged" and a device
    workspace tensor of at least 2 * n block bytes): pool-to-host block copies."""
    sb, db = _i32_host(src_blocks), _i32_host(dst_blocks)
    if sb.shape != db.shape:
        raise ValueError("src_blocks and dst_blocks differ in length")
    p, h = src.c(), dst.c()
    if method == "dma_staged":
        ws_bytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
        _check(lib().pcr_offload_kv_layer_staged(ctypes.byref(p), _ptr(sb), ctypes.byref(h), _ptr(db),
                                                 int(sb.shape[0]), _ptr(workspace), ws_bytes, _stream(stream)))
        return
    _check(lib().pcr_offload_kv_layer_method(ctypes.byref(p), _ptr(sb), ctypes.byref(h), _ptr(db),
                                             int(sb.shape[0]), LOAD_METHODS[method], _stream(stream)))


def staged_workspace_bytes(n_blocks: int, num_kv_heads: int, head_dim: int, block_size: int = 16) -> int:
    """Workspace the staged copies need for n_blocks blocks (K and V)."""
    return 2 * n_blocks * block_size * num_kv_heads * head_dim * 2


def append_kv(pool: KVPool, k_new, v_new, slot_mapping, stream=None):
    """pcr_append_kv: k_new/v_new [T][Hkv][d] and slot_mapping [T] are device tensors."""
    T = int(k_new.shape[0])
    row = pool.num_kv_heads * pool.head_dim
    _need(k_new, T * row, "k_new")
    _need(v_new, T * row, "v_new")
    _need(slot_mapping, T, "slot_mapping")
    p = pool.c()
    _check(lib().pcr_append_kv(ctypes.byref(p), _ptr(k_new), _ptr(v_new), _ptr(slot_mapping), T, _stream(stream)))


def prefix_prefill_attn(q, pool: KVPool, block_tables, prefix_lens, cu_suffix, host_prefix_lens, host_cu_suffix,
                        num_q_heads: int, out, sm_scale: Optional[float] = None, stream=None):
    """pcr_prefix_prefill_attn. q/out [T][Hq][d], block_tables [B][max_blocks], prefix_lens [B],
    cu_suffix [B+1] on the device; host_* are the host copies of the lengths."""
    hpl, hcu = _i32_host(host_prefix_lens), _i32_host(host_cu_suffix)
    B = int(hpl.shape[0])
    if hcu.shape[0] != B + 1:
        raise ValueError("host_cu_suffix must have B+1 entries")
    if sm_scale is None:
        sm_scale = 1.0 / float(np.sqrt(pool.head_dim))
    T = int(hcu[-1]) if B > 0 else 0
    _need(q, T * int(num_q_heads) * pool.head_dim, "q")
    _need(out, T * int(num_q_heads) * pool.head_dim, "out")
    _need(block_tables, B * int(block_tables.shape[1]), "block_tables")
    _need(prefix_lens, B, "prefix_lens")
    _need(cu_suffix, B + 1, "cu_suffix")
    p = pool.c()
    _check(lib().pcr_prefix_prefill_attn(_ptr(q), ctypes.byref(p), _ptr(block_tables), int(block_tables.shape[1]),
                                         _ptr(prefix_lens), _ptr(cu_suffix), _ptr(hpl), _ptr(hcu), B,
                                         int(num_q_heads), float(sm_scale), _ptr(out), _stream(stream)))


def decode_attn_workspace_bytes(B: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
                                max_context: int) -> int:
    """pcr_decode_attn_workspace_size on the current device."""
    n = ctypes.c_int64(0)
    _check(lib().pcr_decode_attn_workspace_size(int(B), int(num_q_heads), int(num_kv_heads), int(head_dim),
                                                int(max_context), ctypes.byref(n)))
    return int(n.value)


ATTN_SCHEDULES = {"auto": 0, "key_halves": 1, "row_halves": 2}


def prefill_attn_set_schedule(schedule: str = "auto"):
    """pcr_prefill_attn_set_schedule: process-wide attention schedule ("auto",
    "key_halves" or "row_halves")."""
    _check(lib().pcr_prefill_attn_set_schedule(ATTN_SCHEDULES[schedule]))


def _decode_need(q, out, block_tables, context_lens, B: int, num_q_heads: int, pool: "KVPool"):
    _need(q, B * int(num_q_heads) * pool.head_dim, "q")
    _need(out, B * int(num_q_heads) * pool.head_dim, "out")
    _need(block_tables, B * int(block_tables.shape[1]), "block_tables")
    _need(context_lens, B, "context_lens")


def decode_attn(q, pool: KVPool, block_tables, context_lens, host_context_lens, num_q_heads: int, out,
                workspace=None, sm_scale: Optional[float] = None, stream=None):
    """pcr_decode_attn. q/out [B][Hq][d], block_tables [B][max_blocks], context_lens [B] on the
    device; host_context_lens is the host copy. Without a workspace one of the needed size
    is allocated on q's device, from the pool of the stream the kernels run on, so that
    the caching allocator reuses it only after that stream has passed them."""
    hcl = _i32_host(host_context_lens)
    B = int(hcl.shape[0])
    if sm_scale is None:
        sm_scale = 1.0 / float(np.sqrt(pool.head_dim))
    _decode_need(q, out, block_tables, context_lens, B, num_q_heads, pool)
    if workspace is None and B > 0:
        import torch
        n = decode_attn_workspace_bytes(B, num_q_heads, pool.num_kv_heads, pool.head_dim, int(hcl.max()))
        if n > 0:
            if stream is None:
                s = torch.cuda.current_stream(q.device)
            elif isinstance(stream, int):
                s = torch.cuda.ExternalStream(stream, device=q.device)
            else:
                s = stream
            with torch.cuda.stream(s):
                workspace = torch.empty(n, dtype=torch.uint8, device=q.device)
    ws_bytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
    p = pool.c()
    _check(lib().pcr_decode_attn(_ptr(q), ctypes.byref(p), _ptr(block_tables), int(block_tables.shape[1]),
                                 _ptr(context_lens), _ptr(hcl), B, int(num_q_heads), float(sm_scale), _ptr(out),
                                 _ptr(workspace), ws_bytes, _stream(stream)))


def decode_attn_noalloc(q, pool: KVPool, block_tables, context_lens, host_context_lens, num_q_heads: int, out,
                        sm_scale: Optional[float] = None, stream=None):
    """pcr_decode_attn_noalloc: as decode_attn, with the library's per-device scratch in
    place of a workspace (nothing is allocated)."""
    hcl = _i32_host(host_context_lens)
    B = int(hcl.shape[0])
    if sm_scale is None:
        sm_scale = 1.0 / float(np.sqrt(pool.head_dim))
    _decode_need(q, out, block_tables, context_lens, B, num_q_heads, pool)
    p = pool.c()
    _check(lib().pcr_decode_attn_noalloc(_ptr(q), ctypes.byref(p), _ptr(block_tables), int(block_tables.shape[1]),
                                         _ptr(context_lens), _ptr(hcl), B, int(num_q_heads), float(sm_scale),
                                         _ptr(out), _stream(stream)))


def gather_kv(pool: KVPool, block_tables, starts, cu_out, total: int, k_out, v_out, stream=None):
    """pcr_gather_kv: rows of k_out/v_out [total][Hkv][d] from the pool in logical order."""
    B = int(starts.shape[0])
    row = pool.num_kv_heads * pool.head_dim
    _need(cu_out, B + 1, "cu_out")
    _need(block_tables, B * int(block_tables.shape[1]), "block_tables")
    _need(k_out, int(total) * row, "k_out")
    _need(v_out, int(total) * row, "v_out")
    p = pool.c()
    _check(lib().pcr_gather_kv(ctypes.byref(p), _ptr(block_tables), int(block_tables.shape[1]), _ptr(starts),
                               _ptr(cu_out), B, int(total), _ptr(k_out), _ptr(v_out), _stream(stream)))


@dataclass
class Layer:
    host: HostKV
    pool: KVPool
    q: "object"
    k_new: "object"
    v_new: "object"
    out: "object"


@dataclass
class BatchPlan:
    """Batch structure for the pipeline: host pair lists, device tables and host length copies."""
    src_blocks: np.ndarray
    dst_blocks: np.ndarray
    slot_mapping: "object"       # device int32 [T]
    block_tables: "object"       # device int32 [B][max_blocks]
    prefix_lens: "object"        # device int32 [B]
    cu_suffix: "object"          # device int32 [B+1]
    host_prefix_lens: np.ndarray
    host_cu_suffix: np.ndarray
    num_q_heads: int
    sm_scale: float

    def c(self) -> _Batch:
        self._keep = (_i32_host(self.src_blocks), _i32_host(self.dst_blocks), _i32_host(self.host_prefix_lens),
                      _i32_host(self.host_cu_suffix))
        sb, db, hpl, hcu = self._keep
        B = int(hpl.shape[0])
        if hcu.shape[0] != B + 1:
            raise ValueError("host_cu_suffix must have B+1 entries")
        _need(self.slot_mapping, int(hcu[-1]) if B > 0 else 0, "slot_mapping")
        _need(self.block_tables, B * int(self.block_tables.shape[1]), "block_tables")
        _need(self.prefix_lens, B, "prefix_lens")
        _need(self.cu_suffix, B + 1, "cu_suffix")
        return _Batch(_ptr(sb), _ptr(db), int(sb.shape[0]), _ptr(self.slot_mapping), int(self.slot_mapping.shape[0]),
                      _ptr(self.block_tables), int(self.block_tables.shape[1]), _ptr(self.prefix_lens),
                      _ptr(self.cu_suffix), _ptr(hpl), _ptr(hcu), int(hpl.shape[0]), int(self.num_q_heads),
                      float(self.sm_scale))


def _layers_io(layers: Sequence[Layer], batch: BatchPlan):
    """The layer array of the pipeline calls, each layer's device tensors checked against
    the lengths the batch makes the library read."""
    T = int(_i32_host(batch.host_cu_suffix)[-1])
    arr = (_LayerIO * max(len(layers), 1))()
    for i, L in enumerate(layers):
        d, hkv = L.pool.head_dim, L.pool.num_kv_heads
        _need(L.q, T * int(batch.num_q_heads) * d, f"layer {i} q")
        _need(L.out, T * int(batch.num_q_heads) * d, f"layer {i} out")
        _need(L.k_new, T * hkv * d, f"layer {i} k_new")
        _need(L.v_new, T * hkv * d, f"layer {i} v_new")
        arr[i] = _LayerIO(L.host.c(), L.pool.c(), _ptr(L.q), _ptr(L.k_new), _ptr(L.v_new), _ptr(L.out))
    return arr


def pipeline_run(layers: Sequence[Layer], batch: BatchPlan, copy_stream, compute_stream, method: str = "auto",
                 timing: bool = False):
    """pcr_pipeline_run. With timing=True, waits for the last layer and returns a dict of
    per-layer load/compute/wait ms and totals; otherwise only enqueues and returns None."""
    n = len(layers)
    arr = _layers_io(layers, batch)
    b = batch.c()
    t = np.zeros(4 * n + 2, np.float32) if timing else None
    _check(lib().pcr_pipeline_run(arr, n, ctypes.byref(b), LOAD_METHODS[method], _stream(copy_stream),
                                  _stream(compute_stream), _ptr(t)))
    if not timing:
        return None
    per = t[:4 * n].reshape(n, 4)
    return {"load_ms": per[:, 0].copy(), "compute_ms": per[:, 1].copy(), "wait_ms": per[:, 2].copy(),
            "end_ms": per[:, 3].copy(), "total_ms": float(t[4 * n]), "sum_compute_ms": float(t[4 * n + 1])}


def pipeline_run_staged(layers: Sequence[Layer], batch: BatchPlan, workspace, copy_stream, scatter_stream,
                        compute_stream, timing: bool = False):
    """pcr_pipeline_run_staged: loads as copy-engine transfers into `workspace` slots
    (copy stream) and a scatter into the pool (scatter stream). `workspace`: a device
    tensor of at least one slot, pipeline_staged_slot_bytes(...) bytes; whole slots
    beyond the first let the next transfer run during a scatter. Timing as
    pipeline_run."""
    n = len(layers)
    arr = _layers_io(layers, batch)
    b = batch.c()
    t = np.zeros(4 * n + 2, np.float32) if timing else None
    ws_bytes = 0 if workspace is None else int(workspace.numel() * workspace.element_size())
    _check(lib().pcr_pipeline_run_staged(arr, n, ctypes.byref(b), _ptr(workspace), ws_bytes, _stream(copy_stream),
                                         _stream(scatter_stream), _stream(compute_stream), _ptr(t)))
    if not timing:
        return None
    per = t[:4 * n].reshape(n, 4)
    return {"load_ms": per[:, 0].copy(), "compute_ms": per[:, 1].copy(), "wait_ms": per[:, 2].copy(),
            "end_ms": per[:, 3].copy(), "total_ms": float(t[4 * n]), "sum_compute_ms": float(t[4 * n + 1])}


def pipeline_staged_slot_bytes(n_pairs: int, num_kv_heads: int, head_dim: int, block_size: int = 16) -> int:
    """One slot of pcr_pipeline_run_staged's workspace: one layer's loaded K and V blocks."""
    return staged_workspace_bytes(n_pairs, num_kv_heads, head_dim, block_size)


def _offload_args(layers, batch, offload_dst, off_src, off_dst):
    n = len(layers)
    if len(offload_dst) != n:
        raise ValueError("one offload destination per layer")
    arr = _layers_io(layers, batch)
    dst = (_Host * max(n, 1))()
    for i, h in enumerate(offload_dst):
        dst[i] = h.c()
    sb, db = _i32_host(off_src), _i32_host(off_dst)
    if sb.shape != db.shape:
        raise ValueError("off_src and off_dst differ in length")
    return n, arr, dst, sb, db


def _offload_timing(t, n):
    per = t[:6 * n].reshape(n, 6)
    return {"load_ms": per[:, 0].copy(), "compute_ms": per[:, 1].copy(), "wait_ms": per[:, 2].copy(),
            "end_ms": per[:, 3].copy(), "offload_ms": per[:, 4].copy(), "offload_end_ms": per[:, 5].copy(),
            "total_ms": float(t[6 * n]), "sum_compute_ms": float(t[6 * n + 1]), "compute_end_ms": float(t[6 * n + 2])}


def _nbytes(t) -> int:
    return 0 if t is None else int(t.numel() * t.element_size())


def pipeline_run_offload(layers: Sequence[Layer], offload_dst: Sequence[HostKV], batch: BatchPlan, off_src, off_dst,
                         copy_stream, compute_stream, offload_stream, method: str = "auto",
                         offload_method: str = "auto", workspace=None, timing: bool = False):
    """pcr_pipeline_run_offload: the three-stream pipeline. With timing=True, waits for the
    last offload and returns per-layer load/compute/wait/offload ms and totals."""
    n, arr, dst, sb, db = _offload_args(layers, batch, offload_dst, off_src, off_dst)
    b = batch.c()
    t = np.zeros(6 * n + 3, np.float32) if timing else None
    _check(lib().pcr_pipeline_run_offload(arr, dst, n, ctypes.byref(b), _ptr(sb), _ptr(db), int(sb.shape[0]),
                                          LOAD_METHODS[method], LOAD_METHODS[offload_method], _ptr(workspace),
                                          _nbytes(workspace), _stream(copy_stream), _stream(compute_stream),
                                          _stream(offload_stream), _ptr(t)))
    return _offload_timing(t, n) if timing else None


def pipeline_run_offload_staged(layers: Sequence[Layer], offload_dst: Sequence[HostKV], batch: BatchPlan, off_src,
                                off_dst, load_workspace, copy_stream, scatter_stream, compute_stream, offload_stream,
                                offload_method: str = "auto", offload_workspace=None, timing: bool = False):
    """pcr_pipeline_run_offload_staged: the offload pipeline with staged loads (four
    streams). load_workspace as pipeline_run_staged's workspace; offload_workspace as
    pipeline_run_offload's. Timing as pipeline_run_offload."""
    n, arr, dst, sb, db = _offload_args(layers, batch, offload_dst, off_src, off_dst)
    b = batch.c()
    t = np.zeros(6 * n + 3, np.float32) if timing else None
    _check(lib().pcr_pipeline_run_offload_staged(arr, dst, n, ctypes.byref(b), _ptr(sb), _ptr(db), int(sb.shape[0]),
                                                 LOAD_METHODS[offload_method], _ptr(offload_workspace),
                                                 _nbytes(offload_workspace), _ptr(load_workspace),
                                                 _nbytes(load_workspace), _stream(copy_stream),
                                                 _stream(scatter_stream), _stream(compute_stream),
                                                 _stream(offload_stream), _ptr(t)))
    return _offload_timing(t, n) if timing else None


class ChunkStore:
    """The SSD tier: a file of fixed-size chunk slots with asynchronous reads and writes
    served by native I/O threads (pcr_store_*). Buffers are numpy arrays or host
    tensors of exactly chunk_bytes, kept alive until their chunk's task completes."""

    def __init__(self, path: str, chunk_bytes: int, io_threads: int = 4):
        self.chunk_bytes = int(chunk_bytes)
        h = ctypes.c_void_p()
        _check(lib().pcr_store_open(os.fsencode(path), self.chunk_bytes, int(io_threads), ctypes.byref(h)))
        self._h = h
        self._keep = {}

    def _buf(self, buf):
        n = buf.nbytes if isinstance(buf, np.ndarray) else buf.numel() * buf.element_size()
        if n != self.chunk_bytes:
            raise ValueError(f"buffer of {n} bytes, chunk is {self.chunk_bytes}")
        return _ptr(buf)

    def write_async(self, chunk_id: int, src):
        self._keep.setdefault(int(chunk_id), []).append(src)
        _check(lib().pcr_store_write_async(self._h, int(chunk_id), self._buf(src)))

    def read_async(self, chunk_id: int, dst):
        self._keep.setdefault(int(chunk_id), []).append(dst)
        _check(lib().pcr_store_read_async(self._h, int(chunk_id), self._buf(dst)))

    def wait(self, chunk_id: int = -1):
        _check(lib().pcr_store_wait(self._h, int(chunk_id)))
        if chunk_id < 0:
            self._keep.clear()
        else:
            self._keep.pop(int(chunk_id), None)

    def done(self, chunk_id: int = -1) -> bool:
        d = ctypes.c_int32(0)
        _check(lib().pcr_store_poll(self._h, int(chunk_id), ctypes.addressof(d)))
        return bool(d.value)

    def stats(self):
        r, w, d, fb = ctypes.c_int64(0), ctypes.c_int64(0), ctypes.c_int32(0), ctypes.c_int64(0)
        _check(lib().pcr_store_stats(self._h, ctypes.addressof(r), ctypes.addressof(w), ctypes.addressof(d),
                                     ctypes.addressof(fb)))
        return {"bytes_read": r.value, "bytes_written": w.value, "direct_io": bool(d.value),
                "direct_fallbacks": fb.value}

    def close(self):
        if self._h:
            h, self._h = self._h, None
            _check(lib().pcr_store_close(h))
            self._keep.clear()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
