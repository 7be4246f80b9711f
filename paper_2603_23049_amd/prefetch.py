"""Queue-window prefetch of KV chunks from the SSD tier into DRAM, and asynchronous
write-back (Sec. 4.4; Sec. 5: a prefetch thread fed with the waiting requests inside
a window; Alg. 1's prefetch loop with its window).

Three tiers hold a chunk's KV: GPU (the pool, per batch), DRAM (a bounded set of
host slots, least recently used evicted first) and SSD (a ChunkStore file holding
every chunk ever computed). Serving a request needs all its matched chunks in DRAM
before its prefill can load them layer by layer. Without prefetch the chunks found
only on SSD are read on demand and the request stalls for them; with a window of W,
while request i computes, the chunks of requests i+1 .. i+W that are on SSD but
not in DRAM are already being read by the store's I/O threads, so their reads
overlap compute. New chunks of a request go to DRAM and are written back to SSD
asynchronously (the request does not wait for the disk).

This is the host harness around the data path: bookkeeping in Python, the bytes
moved by the native store (pcr_store_*). Compute is modelled by a sleep of a given
length per computed token (the data path's own timing is measured elsewhere).
"""
from __future__ import annotations

import mmap
import time
from collections import OrderedDict
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import pcr
from .prefix_tree import PrefixTree


def page_aligned_buffer(nbytes: int) -> np.ndarray:
    """A page-aligned byte array (anonymous mapping), so that the store can bypass the
    page cache when reading into it or writing from it."""
    m = mmap.mmap(-1, nbytes)
    return np.frombuffer(m, dtype=np.uint8)


def chunk_pattern(node_id: int, nbytes: int) -> np.ndarray:
    """Deterministic payload of a chunk (stands for its KV bytes)."""
    return np.random.Generator(np.random.PCG64(1_000_003 + node_id)).integers(0, 256, size=nbytes, dtype=np.uint8)


class KVTier:
    """The DRAM tier of KV chunks as pinned host memory on the data path, over the SSD
    tier (Sec. 4.4: chunks are read from SSD into DRAM ahead of use and written back
    after compute; Sec. 5: the load copies DRAM chunks to the GPU layer by layer).

    For each of n_layers layers the DRAM tier is one pinned host store in the pool's
    per-block layout (a pcr.HostKV, [n_slots * blocks_per_chunk][Hkv][bs*d] for K and
    for V). Slot i of every layer holds one chunk: host blocks
    [i * blocks_per_chunk, (i + 1) * blocks_per_chunk). So pcr_load_kv_layer copies a
    resident chunk straight from its slot into the pool, and pcr_offload_kv_layer (or the
    offload pipeline) writes a computed chunk straight into a slot. The SSD store keeps
    one record per (chunk, layer, K or V) of blocks_per_chunk blocks, id
    (node_id * n_layers + layer) * 2 + part. Slots are page-aligned, so the store's reads
    and writes bypass the page cache. Slots are evicted least recently used first, never
    one that is protected, being read, or whose write-back is still in flight (the
    eviction waits for it)."""

    def __init__(self, store_path: str, n_slots: int, n_layers: int, num_kv_heads: int, head_dim: int,
                 block_size: int = 16, chunk_tokens: int = 256, io_threads: int = 4):
        import torch
        self.bpc = chunk_tokens // block_size
        self.n_slots, self.n_layers = n_slots, n_layers
        shape = (n_slots * self.bpc, num_kv_heads, block_size * head_dim)
        self.layers = [pcr.HostKV(torch.zeros(shape, dtype=torch.int16, pin_memory=True),
                                  torch.zeros(shape, dtype=torch.int16, pin_memory=True), num_kv_heads, head_dim,
                                  block_size) for _ in range(n_layers)]
        self.part_bytes = self.bpc * num_kv_heads * block_size * head_dim * 2
        for h in self.layers:
            for t in (h.k, h.v):
                if t.data_ptr() % mmap.PAGESIZE:
                    raise RuntimeError("pinned DRAM tier is not page-aligned")
        self.store = pcr.ChunkStore(store_path, self.part_bytes, io_threads)
        self.free = list(range(n_slots))[::-1]
        self.where: "OrderedDict[int, int]" = OrderedDict()   # node id -> slot, least recent first
        self.reading: Dict[int, int] = {}
        self.on_ssd: set = set()
        self.evictions = 0

    def _rid(self, nid: int, layer: int, part: int) -> int:
        return (nid * self.n_layers + layer) * 2 + part

    def part(self, layer: int, slot: int, part: int):
        """The pinned view of one slot's K (part 0) or V (part 1) blocks of a layer."""
        h = self.layers[layer]
        return (h.k if part == 0 else h.v)[slot * self.bpc:(slot + 1) * self.bpc]

    def slot_blocks(self, slot: int) -> np.ndarray:
        return np.arange(slot * self.bpc, (slot + 1) * self.bpc, dtype=np.int32)

    def slot_of(self, nid: int) -> int:
        return self.where[nid]

    def resident(self, nid: int) -> bool:
        return nid in self.where

    def touch(self, nid: int):
        if nid in self.where:
            self.where.move_to_end(nid)

    def alloc(self, nid: int, protect: set) -> Optional[int]:
        """A slot for chunk nid (evicting the least recently used unprotected chunk), or None."""
        if self.free:
            slot = self.free.pop()
        else:
            slot = None
            for old in self.where:
                if old in protect or old in self.reading:
                    continue
                slot = self.where.pop(old)
                for l in range(self.n_layers):          # its write-back must finish before reuse
                    self.store.wait(self._rid(old, l, 0))
                    self.store.wait(self._rid(old, l, 1))
                self.evictions += 1
                break
            if slot is None:
                return None
        self.where[nid] = slot
        return slot

    def start_read(self, nid: int, protect: set) -> bool:
        """Issue the SSD reads of every layer of chunk nid into a DRAM slot."""
        slot = self.alloc(nid, protect)
        if slot is None:
            return False
        for l in range(self.n_layers):
            for part in (0, 1):
                self.store.read_async(self._rid(nid, l, part), self.part(l, slot, part))
        self.reading[nid] = slot
        return True

    def finish_read(self, nid: int):
        if nid in self.reading:
            for l in range(self.n_layers):
                self.store.wait(self._rid(nid, l, 0))
                self.store.wait(self._rid(nid, l, 1))
            del self.reading[nid]

    def write_back(self, nid: int):
        """Queue the SSD writes of every layer of a resident chunk (asynchronous)."""
        slot = self.where[nid]
        for l in range(self.n_layers):
            for part in (0, 1):
                self.store.write_async(self._rid(nid, l, part), self.part(l, slot, part))
        self.on_ssd.add(nid)

    def drop(self, nid: int):
        """Forget the DRAM copy of a chunk (after its write-back has finished)."""
        slot = self.where.pop(nid)
        for l in range(self.n_layers):
            self.store.wait(self._rid(nid, l, 0))
            self.store.wait(self._rid(nid, l, 1))
        self.free.append(slot)

    def close(self):
        self.store.close()


@dataclass
class ServeStats:
    requests: int = 0
    hit_tokens: int = 0
    total_tokens: int = 0
    stall_ms: float = 0.0
    on_demand_reads: int = 0
    prefetch_reads: int = 0
    prefetch_hits: int = 0          # needed chunks whose read was already issued by the prefetcher
    dram_hits: int = 0              # needed chunks already resident in DRAM
    writes: int = 0
    prefetch_evicted: int = 0       # chunks read ahead but evicted from DRAM before their request
    wall_ms: float = 0.0


class TieredCache:
    """DRAM slots over an SSD ChunkStore, keyed by prefix-tree node id."""

    def __init__(self, store: pcr.ChunkStore, dram_chunks: int, chunk_bytes: int):
        self.store = store
        self.chunk_bytes = chunk_bytes
        self.slots = page_aligned_buffer(dram_chunks * chunk_bytes).reshape(dram_chunks, chunk_bytes)
        self.free = list(range(dram_chunks))[::-1]
        self.where: "OrderedDict[int, int]" = OrderedDict()   # node id -> slot, least recent first
        self.reading: Dict[int, int] = {}                       # node id -> slot with a read in flight
        self.on_ssd: set = set()
        self.prefetched: set = set()       # read ahead and not used yet
        self.prefetch_evicted = 0          # chunks read ahead and evicted before their request came

    def _slot(self, protect: set) -> Optional[int]:
        if self.free:
            return self.free.pop()
        for nid in self.where:
            if nid in protect or nid in self.reading:
                continue
            slot = self.where.pop(nid)
            self.store.wait(nid)           # a write-back of this slot must finish before reuse
            if nid in self.prefetched:
                self.prefetched.discard(nid)
                self.prefetch_evicted += 1
            return slot
        return None

    def resident(self, nid: int) -> bool:
        return nid in self.where

    def touch(self, nid: int):
        if nid in self.where:
            self.where.move_to_end(nid)

    def start_read(self, nid: int, protect: set) -> bool:
        """Issue the SSD read of a chunk into a DRAM slot (False if no slot is free)."""
        slot = self._slot(protect)
        if slot is None:
            return False
        self.store.read_async(nid, self.slots[slot])
        self.where[nid] = slot
        self.reading[nid] = slot
        return True

    def finish_read(self, nid: int):
        if nid in self.reading:
            self.store.wait(nid)
            del self.reading[nid]

    def put_new(self, nid: int, payload: np.ndarray, protect: set):
        """A freshly computed chunk: into DRAM, then written back to SSD asynchronously."""
        slot = self._slot(protect)
        if slot is None:
            raise RuntimeError("DRAM tier too small for one request's chunks")
        self.slots[slot][:] = payload
        self.where[nid] = slot
        self.store.write_async(nid, self.slots[slot])
        self.on_ssd.add(nid)

    def payload(self, nid: int) -> np.ndarray:
        return self.slots[self.where[nid]]


def serve(requests: Sequence[Sequence[int]], *, store_path: str, chunk_bytes: int, dram_chunks: int,
          window: int, compute_ms_per_token: float, warm: int = 64, io_threads: int = 4,
          verify: bool = False, chunk_tokens: int = 256) -> ServeStats:
    """Serve a request stream one request at a time through the three tiers.

    The first `warm` requests fill the tree and the SSD (their chunks are written
    back and then dropped from DRAM except the most recent). For each later request
    i: the prefetcher issues SSD reads for the matched chunks of requests
    i+1 .. i+window that are neither in DRAM nor being read; request i waits for its
    own matched chunks (reading on demand what is still only on SSD; that wait is
    the stall), computes (sleep), and its new chunks go to DRAM with write-back."""
    store = pcr.ChunkStore(store_path, chunk_bytes, io_threads)
    cache = TieredCache(store, dram_chunks, chunk_bytes)
    tree = PrefixTree(chunk_tokens=chunk_tokens)
    st = ServeStats()
    try:
        for i, req in enumerate(requests[:warm]):
            chain = tree.insert(req)
            for node in chain:
                if node.node_id not in cache.on_ssd:
                    cache.put_new(node.node_id, chunk_pattern(node.node_id, chunk_bytes), protect=set())
        store.wait()
        t_start = time.perf_counter()
        for i in range(warm, len(requests)):
            req = requests[i]
            chain = tree.match(req)
            need = [n.node_id for n in chain]
            protect = set(need)
            # prefetch for the waiting requests inside the window (never evicting what
            # the current request needs)
            for nxt in requests[i + 1:i + 1 + window]:
                for node in tree.match(nxt):
                    nid = node.node_id
                    if nid in cache.on_ssd and not cache.resident(nid):
                        if cache.start_read(nid, protect=protect):
                            st.prefetch_reads += 1
                            cache.prefetched.add(nid)
            t0 = time.perf_counter()
            for nid in need:
                if nid in cache.reading:
                    st.prefetch_hits += 1
                elif cache.resident(nid):
                    st.dram_hits += 1
                else:
                    if not cache.start_read(nid, protect):
                        raise RuntimeError("DRAM tier too small for one request's chunks")
                    st.on_demand_reads += 1
                cache.finish_read(nid)
                cache.touch(nid)
                cache.prefetched.discard(nid)
            st.stall_ms += (time.perf_counter() - t0) * 1e3
            if verify:
                for nid in need:
                    if not np.array_equal(cache.payload(nid), chunk_pattern(nid, chunk_bytes)):
                        raise AssertionError(f"chunk {nid} read back wrong")
            hit = len(chain) * chunk_tokens
            st.hit_tokens += hit
            st.total_tokens += len(req)
            time.sleep(max(0, len(req) - hit) * compute_ms_per_token * 1e-3)
            new_chain = tree.insert(req)
            for node in new_chain[len(chain):]:
                cache.put_new(node.node_id, chunk_pattern(node.node_id, chunk_bytes) if verify else
                              np.full(1, node.node_id & 0xFF, np.uint8), protect=protect | {node.node_id})
                st.writes += 1
            st.requests += 1
        store.wait()
        st.wall_ms = (time.perf_counter() - t_start) * 1e3
        st.prefetch_evicted = cache.prefetch_evicted
    finally:
        store.close()
    return st
