"""GPU-side test plumbing: numpy bf16 bit arrays <-> torch tensors, and one
layer of a batch set up for the HIP path through the C ABI binding."""
import contextlib
import sys

import numpy as np
import torch

from paper_2603_23049_amd import pcr, synth


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@contextlib.contextmanager
def attn_schedule(name: str):
    """Runs the block under one attention schedule, then restores the default ("auto").
    The pipelines with pull-kernel loads take key halves under "auto", so their serial
    references are computed with key halves."""
    pcr.prefill_attn_set_schedule(name)
    try:
        yield
    finally:
        pcr.prefill_attn_set_schedule("auto")


def dev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


def pinned(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    t = torch.empty(a.shape, dtype=torch.from_numpy(a[:0]).dtype, pin_memory=True)
    t.copy_(torch.from_numpy(a))
    return t


def u16(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


class GpuLayer:
    """One layer of a batch on the GPU: pool (initialised from pool_k0/pool_v0),
    pinned host store, Q and new K/V, output buffer, and the planned batch."""

    def __init__(self, batch: synth.Batch, data: synth.LayerData, pool_k0: np.ndarray, pool_v0: np.ndarray,
                 host_blocks=None, block_tables=None):
        self.batch = batch
        Hkv, d = batch.num_kv_heads, batch.head_dim
        self.bt_np = batch.block_tables if block_tables is None else block_tables
        self.hb_np = batch.host_blocks if host_blocks is None else host_blocks
        self.pool = pcr.KVPool(dev(pool_k0), dev(pool_v0), Hkv, d)
        if data.host_k.shape[0] > 0:
            self.host = pcr.HostKV(pinned(data.host_k), pinned(data.host_v), Hkv, d)
        else:
            self.host = pcr.HostKV(pinned(np.zeros((1, Hkv, 16 * d), np.uint16)),
                                   pinned(np.zeros((1, Hkv, 16 * d), np.uint16)), Hkv, d)
        self.q = dev(data.q)
        self.k_new = dev(data.k_new)
        self.v_new = dev(data.v_new)
        self.out = torch.zeros(data.q.shape, dtype=torch.int16, device="cuda")
        self.src, self.dst, self.slots_np, self.cu_np = pcr.plan(batch.prefix_lens, batch.suffix_lens, self.bt_np,
                                                                 self.hb_np, batch.block_size)
        self.slots = dev(self.slots_np)
        self.bt = dev(self.bt_np)
        self.pl_np = np.asarray(batch.prefix_lens, np.int32)
        self.pl = dev(self.pl_np)
        self.cu = dev(self.cu_np)
        self.sm_scale = 1.0 / float(np.sqrt(d))

    def load(self, method="auto", stream=None):
        pcr.load_kv_layer(self.host, self.src, self.pool, self.dst, method=method, stream=stream)

    def append(self, stream=None):
        pcr.append_kv(self.pool, self.k_new, self.v_new, self.slots, stream=stream)

    def attn(self, stream=None):
        pcr.prefix_prefill_attn(self.q, self.pool, self.bt, self.pl, self.cu, self.pl_np, self.cu_np,
                                self.batch.num_q_heads, self.out, sm_scale=self.sm_scale, stream=stream)

    def run_serial(self, method="auto"):
        self.load(method)
        torch.cuda.synchronize()
        self.append()
        self.attn()
        torch.cuda.synchronize()

    def batch_plan(self) -> pcr.BatchPlan:
        return pcr.BatchPlan(self.src, self.dst, self.slots, self.bt, self.pl, self.cu, self.pl_np, self.cu_np,
                             self.batch.num_q_heads, self.sm_scale)

    def layer_io(self) -> pcr.Layer:
        return pcr.Layer(self.host, self.pool, self.q, self.k_new, self.v_new, self.out)

    def out_f64(self) -> np.ndarray:
        return synth.bf16_bits_to_f32(u16(self.out)).astype(np.float64)


def error_stats(got: np.ndarray, want: np.ndarray):
    err = np.abs(got - want)
    return float(err.max()), float(err.mean())


MAX_ABS = 2e-2
MEAN_ABS = 2e-3
