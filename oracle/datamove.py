"""Oracle for the integer and bit-copy steps of the hot path.

TEST INFRASTRUCTURE (see the package docstring). Plain numpy with explicit
loops over blocks and tokens, so that each step reads as its definition.

Steps (the layer step of Sec. 4.3 / Alg. 1, on a paged pool as in Sec. 5):
  plan    -- for each sequence: which host-store blocks go to which pool blocks
             (the "cpu_to_gpu" list of Alg. 1's planning loop, one entry per
             cached 16-token block) and where each new token's K/V is written
             (its pool slot); the new-token count per sequence is the suffix
             ("AdjustTokens": only the unmatched tokens are computed).
  load    -- pool[dst] <- host[src] for every planned pair, bit for bit; every
             other pool block keeps its bits.
  append  -- the new tokens' K/V rows go to their slots, bit for bit.
  gather  -- read a sequence's K/V back in logical token order, bit for bit.
  plan_offload -- the "gpu_to_cpu" list of Alg. 1: every whole chunk of a
             sequence's computed tokens (chunks aligned to the sequence start)
             goes to the host store after compute, block by block.
  offload -- host[dst] <- pool[src] for every listed pair, bit for bit.

Pool / host-store block layout (bf16 bit patterns, one layer; per block and
kv head a payload of block_size*head_dim elements):
  K payload index of (slot o, dim x) = o*head_dim + x
  V payload index of (slot o, dim x) = x*block_size + o
Logical token t of sequence b is slot t % bs of pool block block_tables[b][t // bs].
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


class PlanError(ValueError):
    pass


def _ceil_div(a, b):
    return -(-a // b)


def plan(prefix_lens: Sequence[int], suffix_lens: Sequence[int], block_tables: np.ndarray,
         host_blocks: np.ndarray, block_size: int = 16):
    """Returns (src_blocks, dst_blocks, slot_mapping, cu_suffix) as int32 arrays.

    Pairs are listed sequence by sequence, logical block ascending; a pair equal to
    an earlier one (a prefix block shared by two sequences) is listed once. A pool
    block named as the destination of two different host blocks is an error, and
    so is a new token whose slot is taken by another token or lies in a pool
    block that another sequence loads.
    """
    bs = block_size
    B = len(prefix_lens)
    src: List[int] = []
    dst: List[int] = []
    seen = {}
    owner = {}   # dst block -> set of sequences loading it
    for b in range(B):
        p = int(prefix_lens[b])
        for j in range(_ceil_div(p, bs)):
            s_blk = int(host_blocks[b][j])
            d_blk = int(block_tables[b][j])
            if s_blk < 0 or d_blk < 0:
                raise PlanError(f"sequence {b}: prefix block {j} has no host or pool block")
            owner.setdefault(d_blk, set()).add(b)
            if d_blk in seen:
                if seen[d_blk] != s_blk:
                    raise PlanError(f"pool block {d_blk} is loaded from two host blocks")
                continue
            seen[d_blk] = s_blk
            src.append(s_blk)
            dst.append(d_blk)
    slots: List[int] = []
    for b in range(B):
        p, s = int(prefix_lens[b]), int(suffix_lens[b])
        for i in range(s):
            t = p + i
            blk = int(block_tables[b][t // bs])
            if blk < 0:
                raise PlanError(f"sequence {b}: token {t} has no pool block")
            if owner.get(blk, {b}) != {b}:
                raise PlanError(f"sequence {b}: new token {t} lands in a block another sequence loads")
            slots.append(blk * bs + t % bs)
    if len(set(slots)) != len(slots):
        raise PlanError("two new tokens share a pool slot")
    cu = [0]
    for s in suffix_lens:
        cu.append(cu[-1] + int(s))
    return (np.asarray(src, np.int32), np.asarray(dst, np.int32),
            np.asarray(slots, np.int32), np.asarray(cu, np.int32))


def load(pool_k: np.ndarray, pool_v: np.ndarray, host_k: np.ndarray, host_v: np.ndarray,
         src_blocks: Sequence[int], dst_blocks: Sequence[int]) -> None:
    """In place: pool[dst_i] <- host[src_i] for every pair (whole block, all kv heads)."""
    for s_blk, d_blk in zip(src_blocks, dst_blocks):
        pool_k[int(d_blk)] = host_k[int(s_blk)]
        pool_v[int(d_blk)] = host_v[int(s_blk)]


def append(pool_k: np.ndarray, pool_v: np.ndarray, k_new: np.ndarray, v_new: np.ndarray,
           slot_mapping: Sequence[int], block_size: int = 16) -> None:
    """In place: the new token t's K/V row (every kv head) goes to slot slot_mapping[t]."""
    bs = block_size
    T, Hkv, d = k_new.shape
    x = np.arange(d)
    for t in range(T):
        slot = int(slot_mapping[t])
        blk, o = slot // bs, slot % bs
        for g in range(Hkv):
            pool_k[blk, g, o * d + x] = k_new[t, g, x]
            pool_v[blk, g, x * bs + o] = v_new[t, g, x]


def gather(pool_k: np.ndarray, pool_v: np.ndarray, block_tables: np.ndarray,
           starts: Sequence[int], lens: Sequence[int], head_dim: int, block_size: int = 16):
    """Contiguous K and V [sum(lens)][Hkv][d] of tokens starts[b] .. starts[b]+lens[b]-1
    of every sequence b, in logical order."""
    bs, d = block_size, head_dim
    Hkv = pool_k.shape[1]
    n = int(sum(int(x) for x in lens))
    k_out = np.empty((n, Hkv, d), np.uint16)
    v_out = np.empty((n, Hkv, d), np.uint16)
    x = np.arange(d)
    r = 0
    for b in range(len(lens)):
        for t in range(int(starts[b]), int(starts[b]) + int(lens[b])):
            blk, o = int(block_tables[b][t // bs]), t % bs
            for g in range(Hkv):
                k_out[r, g, x] = pool_k[blk, g, o * d + x]
                v_out[r, g, x] = pool_v[blk, g, x * bs + o]
            r += 1
    return k_out, v_out


def pool_after_layer(pool_k, pool_v, host_k, host_v, batch_plan, k_new, v_new, block_size=16):
    """Copies of the pools after one layer's load then append (the order the layer
    step requires: a partially cached block is loaded whole, then its free slots
    take the new tokens)."""
    src, dst, slots, _ = batch_plan
    pk, pv = pool_k.copy(), pool_v.copy()
    load(pk, pv, host_k, host_v, src, dst)
    append(pk, pv, k_new, v_new, slots, block_size)
    return pk, pv


def plan_offload(prefix_lens: Sequence[int], suffix_lens: Sequence[int], block_tables: np.ndarray,
                 block_size: int = 16, chunk_tokens: int = 256, first_dst_block: int = 0):
    """(src pool blocks, dst host blocks): for every sequence, the blocks of each whole
    chunk [c*chunk, (c+1)*chunk) that lies inside its computed range [p, p+s), chunks
    and blocks in order; host blocks numbered from first_dst_block."""
    if chunk_tokens % block_size:
        raise PlanError("chunk size must be a multiple of the block size")
    src, dst = [], []
    for b, (p, s) in enumerate(zip(prefix_lens, suffix_lens)):
        p, s = int(p), int(s)
        c = 0
        while (c + 1) * chunk_tokens <= p + s:
            if c * chunk_tokens >= p:                          # the chunk is all computed tokens
                for t in range(c * chunk_tokens, (c + 1) * chunk_tokens, block_size):
                    blk = int(block_tables[b][t // block_size])
                    if blk < 0:
                        raise PlanError(f"sequence {b} token {t} has no pool block")
                    src.append(blk)
                    dst.append(first_dst_block + len(dst))
            c += 1
    return np.asarray(src, np.int32), np.asarray(dst, np.int32)


def offload(pool_k: np.ndarray, pool_v: np.ndarray, host_k: np.ndarray, host_v: np.ndarray,
            src_blocks: Sequence[int], dst_blocks: Sequence[int]) -> None:
    """In place: host[dst_i] <- pool[src_i] for every pair (whole block, all kv heads)."""
    for s_blk, d_blk in zip(src_blocks, dst_blocks):
        host_k[int(d_blk)] = pool_k[int(s_blk)]
        host_v[int(d_blk)] = pool_v[int(s_blk)]
