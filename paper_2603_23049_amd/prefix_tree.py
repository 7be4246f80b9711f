"""Host-side prefix tree of cached KV chunks, with leaf-only LRU eviction and the
look-ahead priority update (Sec. 4.2, Fig. "Prefix-tree KV cache"; Alg. 1's
cache-engine lookups and inserts).

Documents (and whole requests) are cut into fixed-size chunks of token ids. A
chunk is cached as a tree node under the node of the chunk before it, so a node
stands for one exact prefix: identical chunks after different prefixes are
different nodes, because the KV of a token depends on everything before it.
A request is matched chunk by chunk from the root until the first miss; the
matched chain is the cached prefix whose KV can be loaded instead of computed.

Only leaves can be evicted (a node is reusable only while its parent is cached).
The leaves are kept in recency order. Before choosing victims, the look-ahead
touches the chunks that the next waiting requests will match, so they move to
the recent end and are not evicted just before use. When a leaf is evicted and
its parent has no other child, the parent becomes a leaf (at the recent end);
when a child is inserted under a leaf, the parent leaves the leaf set.

This is bookkeeping only (no KV bytes): each node owns a run of
`blocks_per_chunk` host-store blocks, numbered in insertion order, which the
data path loads through `pcr_load_kv_layer`.
"""
from __future__ import annotations

from collections import OrderedDict
from dataclasses import dataclass, field
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np


@dataclass(eq=False)
class Node:
    node_id: int
    parent: Optional["Node"]
    key: Tuple[int, ...]                 # the chunk's token ids
    depth: int                           # chunks from the root (root: 0)
    host_block0: int = -1                # first host-store block of this chunk
    children: Dict[Tuple[int, ...], "Node"] = field(default_factory=dict)
    name: str = ""

    def path(self) -> List["Node"]:
        out, n = [], self
        while n is not None and n.parent is not None:
            out.append(n)
            n = n.parent
        return out[::-1]


class PrefixTree:
    """Chunked prefix tree with a capacity in chunks (None: unbounded)."""

    def __init__(self, chunk_tokens: int = 256, block_size: int = 16,
                 capacity_chunks: Optional[int] = None, lookahead: bool = True):
        if chunk_tokens % block_size:
            raise ValueError("chunk_tokens must be a multiple of block_size")
        self.chunk_tokens = chunk_tokens
        self.block_size = block_size
        self.blocks_per_chunk = chunk_tokens // block_size
        self.capacity = capacity_chunks
        self.lookahead_enabled = lookahead
        self.root = Node(node_id=0, parent=None, key=(), depth=0, name="root")
        self._next_id = 1
        self._next_block = 0
        self._free_block_runs: List[int] = []
        self.leaves: "OrderedDict[Node, None]" = OrderedDict()   # least recent first
        self.n_chunks = 0
        self.evicted: List[Node] = []

    # ---- queries -------------------------------------------------------------
    def chunks(self, tokens: Sequence[int]) -> List[Tuple[int, ...]]:
        """The full chunks of a token sequence (a trailing partial chunk is not cached)."""
        c = self.chunk_tokens
        t = np.asarray(tokens)
        return [tuple(int(x) for x in t[i:i + c]) for i in range(0, len(t) - c + 1, c)]

    def match(self, tokens: Sequence[int]) -> List[Node]:
        """Longest chain of cached chunks from the root (stops at the first miss)."""
        out, node = [], self.root
        for key in self.chunks(tokens):
            nxt = node.children.get(key)
            if nxt is None:
                break
            out.append(nxt)
            node = nxt
        return out

    def hit_length(self, tokens: Sequence[int]) -> int:
        """Cached prefix length in tokens, on a block boundary, leaving at least one
        token to compute (the last token's output is what prefill must produce)."""
        hit = len(self.match(tokens)) * self.chunk_tokens
        if hit >= len(tokens):
            hit = (len(tokens) - 1) // self.block_size * self.block_size
        return hit - hit % self.block_size

    # ---- recency -------------------------------------------------------------
    def touch(self, nodes: Iterable[Node]) -> None:
        """Mark nodes as just used: cached leaves move to the recent end."""
        for n in nodes:
            if n in self.leaves:
                self.leaves.move_to_end(n)

    def lookahead(self, pending: Sequence[Sequence[int]]) -> None:
        """Raise the priority of the chunks the waiting requests will reuse."""
        if not self.lookahead_enabled:
            return
        for req in pending:
            self.touch(self.match(req))

    # ---- insertion and eviction ---------------------------------------------
    def _alloc_blocks(self) -> int:
        if self._free_block_runs:
            return self._free_block_runs.pop()
        b = self._next_block
        self._next_block += self.blocks_per_chunk
        return b

    def _evict_one(self, protect: set) -> bool:
        for leaf in self.leaves:
            if leaf in protect:
                continue
            parent = leaf.parent
            del self.leaves[leaf]
            del parent.children[leaf.key]
            self._free_block_runs.append(leaf.host_block0)
            self.n_chunks -= 1
            self.evicted.append(leaf)
            if parent is not self.root and not parent.children:
                self.leaves[parent] = None          # the parent is now a leaf (recent end)
            return True
        return False

    def insert(self, tokens: Sequence[int], pending: Sequence[Sequence[int]] = (),
               names: Optional[Sequence[str]] = None) -> List[Node]:
        """Cache every full chunk of `tokens` (after its matched prefix); returns the
        request's whole chain. Evicts leaves when over capacity, after the look-ahead
        over `pending`; the request's own chain is never evicted while inserting."""
        chain = self.match(tokens)
        self.touch(chain)
        node = chain[-1] if chain else self.root
        keys = self.chunks(tokens)[len(chain):]
        looked = False
        for i, key in enumerate(keys):
            if self.capacity is not None and self.n_chunks >= self.capacity:
                if not looked:                        # once per request: the queue is fixed meanwhile
                    self.lookahead(pending)
                    looked = True
                if not self._evict_one(protect=set(chain) | {node}):
                    break                             # everything left is in use
            child = Node(node_id=self._next_id, parent=node, key=key, depth=node.depth + 1,
                         host_block0=self._alloc_blocks(),
                         name=(names[i] if names is not None and i < len(names) else ""))
            self._next_id += 1
            if node is not self.root:
                self.leaves.pop(node, None)           # the parent stops being a leaf
            node.children[key] = child
            self.leaves[child] = None
            self.n_chunks += 1
            chain.append(child)
            node = child
        return chain

    def leaf_names(self) -> List[str]:
        return [n.name for n in self.leaves]

    @property
    def host_store_blocks(self) -> int:
        return self._next_block


# ----------------------------------------------------------------------------
# The RAG-mix batch: 16 requests after a warm-up stream, hits from the tree
# ----------------------------------------------------------------------------

def rag_mix_layout(stream, *, warm: int = 64, batch: int = 16, chunk_tokens: int = 256,
                   block_size: int = 16, capacity_chunks: Optional[int] = None):
    """Warm a tree with the first `warm` requests of the stream, then match the next
    `batch` requests against it. Returns (tree, prefix_lens, suffix_lens, chains),
    where chains[b] are the matched nodes whose KV makes up sequence b's prefix."""
    tree = PrefixTree(chunk_tokens=chunk_tokens, block_size=block_size, capacity_chunks=capacity_chunks)
    reqs = stream.requests
    for i in range(warm):
        tree.insert(reqs[i], pending=reqs[i + 1:i + 1 + 4])
    prefix_lens, suffix_lens, chains = [], [], []
    for req in reqs[warm:warm + batch]:
        hit = tree.hit_length(req)
        chain = tree.match(req)[: hit // chunk_tokens]
        prefix_lens.append(hit)
        suffix_lens.append(len(req) - hit)
        chains.append(chain)
    return tree, prefix_lens, suffix_lens, chains


def rag_mix_batch(seed: int = 4, *, Hq: int = 32, Hkv: int = 8, d: int = 128, warm: int = 64,
                  batch: int = 16, name: str = "rag_mix"):
    """The RAG-mix batch as a ragged Batch: 16 requests of 4-8 Zipf-drawn documents
    plus a 32-512-token query, prefixes hit in a tree warmed by the 64 requests
    before them. Sequences whose hits share tree nodes share the same host-store
    and pool blocks (one load serves them all); suffix blocks are private. Only
    the host-store blocks of matched nodes exist in this batch's host store."""
    from . import synth
    bs = synth.BLOCK_SIZE
    stream = synth.rag_stream(seed, n_requests=warm + batch)
    tree, prefix_lens, suffix_lens, chains = rag_mix_layout(stream, warm=warm, batch=batch, block_size=bs)
    # host-store blocks of the matched nodes only, renumbered densely
    node_slot: Dict[Node, int] = {}
    for chain in chains:
        for n in chain:
            node_slot.setdefault(n, len(node_slot))
    per = tree.blocks_per_chunk
    B = len(prefix_lens)
    max_pb = max([p // bs for p in prefix_lens] + [1])
    host_blocks = np.full((B, max_pb), -1, np.int32)
    for b, (p, chain) in enumerate(zip(prefix_lens, chains)):
        run = [node_slot[n] * per + k for n in chain for k in range(per)][: p // bs]
        host_blocks[b, :len(run)] = run
    # pool: one block per distinct host block, then private suffix blocks; random ids
    need_suffix = [-(-(p + s) // bs) - p // bs for p, s in zip(prefix_lens, suffix_lens)]
    n_pool = len(node_slot) * per + sum(need_suffix)
    rng = np.random.Generator(np.random.PCG64(seed))
    perm = rng.permutation(n_pool).astype(np.int32)
    shared = perm[: len(node_slot) * per]
    private = perm[len(node_slot) * per:]
    max_blocks = max(-(-(p + s) // bs) for p, s in zip(prefix_lens, suffix_lens))
    bt = np.full((B, max_blocks), -1, np.int32)
    off = 0
    for b, (p, s) in enumerate(zip(prefix_lens, suffix_lens)):
        npb = p // bs
        bt[b, :npb] = shared[host_blocks[b, :npb]]
        bt[b, npb:npb + need_suffix[b]] = private[off:off + need_suffix[b]]
        off += need_suffix[b]
    hit_tokens = sum(prefix_lens)
    total_tokens = hit_tokens + sum(suffix_lens)
    return synth.Batch(name=name, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, block_size=bs,
                       pool_blocks=int(n_pool), host_store_blocks=len(node_slot) * per,
                       prefix_lens=[int(x) for x in prefix_lens], suffix_lens=[int(x) for x in suffix_lens],
                       block_tables=bt, host_blocks=host_blocks, seed=seed,
                       note=f"hit ratio {hit_tokens / total_tokens:.3f}; {len(node_slot)} shared tree chunks",
                       extra={"hit_ratio": hit_tokens / total_tokens, "tree_chunks": tree.n_chunks,
                              "matched_nodes": len(node_slot)})


def hit_ratio_under_capacity(seed: int = 4, *, capacity_chunks: Optional[int], lookahead: bool,
                             warm: int = 64, n_requests: int = 400, window: int = 4) -> float:
    """Token hit ratio of a request stream served one request at a time through a
    tree of the given capacity (chunks), with or without the look-ahead over the
    next `window` waiting requests. The first `warm` requests only fill the tree."""
    from . import synth
    stream = synth.rag_stream(seed, n_requests=n_requests)
    tree = PrefixTree(capacity_chunks=capacity_chunks, lookahead=lookahead)
    hit = total = 0
    reqs = stream.requests
    for i, req in enumerate(reqs):
        pending = reqs[i + 1:i + 1 + window]
        if i >= warm:
            hit += tree.hit_length(req)
            total += len(req)
        tree.insert(req, pending=pending)
    return hit / total if total else 0.0
