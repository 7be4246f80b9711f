"""Seeded synthetic inputs for the prefix-reuse prefill path.

This module holds none of the method's arithmetic. It draws random numbers,
rounds them to bf16, draws random physical block tables and token streams, and
names the workload shapes. The HIP path's tests and benchmark and the CPU
oracle's tests both take their inputs from here; neither side's arithmetic
lives here.

Every value is a pure function of a seed: numpy's PCG64 bit generator, fp32
standard normals, rounded to bf16 by round-to-nearest-even on the integer bits.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

BLOCK_SIZE = 16          # tokens per paged KV block (the serving engine's block, Sec. 5)
CHUNK_SIZE = 256         # tokens per cached chunk in the host tiers (Sec. 5)


# ----------------------------------------------------------------------------
# bf16 bit patterns
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit pattern (uint16) by round-to-nearest-even.

    Only finite inputs are accepted (the generator never draws anything else).
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x)):
        raise ValueError("f32_to_bf16_bits: non-finite input")
    u = x.view(np.uint32)
    r = u >> np.uint32(16)          # in place from here: (u + 0x7FFF + lsb) >> 16
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit pattern (uint16) -> fp32, exact."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(rng: np.random.Generator, shape) -> np.ndarray:
    """N(0,1) draws in fp32, returned as bf16 bit patterns of the given shape."""
    return f32_to_bf16_bits(rng.standard_normal(size=shape, dtype=np.float32))


# ----------------------------------------------------------------------------
# Batch structure (integers) and per-layer tensors (bf16 bits)
# ----------------------------------------------------------------------------

@dataclass
class Batch:
    """The integer structure of one ragged batch.

    prefix_lens[b]   cached prefix tokens of sequence b (loaded, not computed)
    suffix_lens[b]   new tokens of sequence b (computed)
    block_tables     [B][max_blocks] physical pool block of each logical block,
                     -1 past ceil((p+s)/block_size)
    host_blocks      [B][max_prefix_blocks] host-store block holding each
                     logical prefix block, -1 past ceil(p/block_size)
    """
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    pool_blocks: int
    host_store_blocks: int
    prefix_lens: List[int]
    suffix_lens: List[int]
    block_tables: np.ndarray
    host_blocks: np.ndarray
    num_layers: int = 1
    seed: int = 0
    layer_seed_base: Optional[int] = None
    note: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def B(self) -> int:
        return len(self.prefix_lens)

    @property
    def T(self) -> int:
        return int(sum(self.suffix_lens))

    @property
    def cu_suffix(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.suffix_lens)]).astype(np.int32)

    @property
    def max_blocks(self) -> int:
        return int(self.block_tables.shape[1])

    def layer_seed(self, layer: int) -> int:
        base = self.layer_seed_base if self.layer_seed_base is not None else self.seed * 1000
        return base + layer


@dataclass
class LayerData:
    """bf16 bit patterns for one layer of a batch.

    q        [T][Hq][d]
    k_new    [T][Hkv][d]
    v_new    [T][Hkv][d]
    host_k   [host_store_blocks][Hkv][block_size*d]   raw per-block payload
    host_v   [host_store_blocks][Hkv][block_size*d]   raw per-block payload
    The host payload is just random bits per block: which element of a block is
    which (token, dim) is the pool layout's business, not the generator's.
    """
    q: np.ndarray
    k_new: np.ndarray
    v_new: np.ndarray
    host_k: np.ndarray
    host_v: np.ndarray


def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def _random_tables(rng, prefix_lens, suffix_lens, bs, pool_blocks):
    """Distinct random physical blocks for every logical block of every sequence."""
    need = [_ceil_div(p + s, bs) for p, s in zip(prefix_lens, suffix_lens)]
    total = sum(need)
    if total > pool_blocks:
        raise ValueError(f"pool of {pool_blocks} blocks cannot hold {total}")
    perm = rng.permutation(pool_blocks).astype(np.int32)
    max_blocks = max(need) if need else 0
    bt = np.full((len(need), max(max_blocks, 1)), -1, dtype=np.int32)
    off = 0
    for b, n in enumerate(need):
        bt[b, :n] = perm[off:off + n]
        off += n
    return bt


def _contiguous_host_blocks(prefix_lens, bs):
    """Sequence b's prefix occupies a contiguous run of host-store blocks."""
    need = [_ceil_div(p, bs) for p in prefix_lens]
    hb = np.full((len(need), max(max(need) if need else 0, 1)), -1, dtype=np.int32)
    off = 0
    for b, n in enumerate(need):
        hb[b, :n] = np.arange(off, off + n, dtype=np.int32)
        off += n
    return hb, off


def uniform_batch(name, *, B, Hq, Hkv, d, p, s, pool_blocks, seed, num_layers=1,
                  layer_seed_base=None, bs=BLOCK_SIZE, note="") -> Batch:
    """Every sequence with the same prefix and suffix length; random block tables."""
    prefix_lens = [int(p)] * B
    suffix_lens = [int(s)] * B
    rng = np.random.Generator(np.random.PCG64(seed))
    bt = _random_tables(rng, prefix_lens, suffix_lens, bs, pool_blocks)
    hb, nhost = _contiguous_host_blocks(prefix_lens, bs)
    return Batch(name=name, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, block_size=bs,
                 pool_blocks=pool_blocks, host_store_blocks=nhost,
                 prefix_lens=prefix_lens, suffix_lens=suffix_lens,
                 block_tables=bt, host_blocks=hb, num_layers=num_layers, seed=seed,
                 layer_seed_base=layer_seed_base, note=note)


def ragged_batch(name, *, Hq, Hkv, d, prefix_lens: Sequence[int], suffix_lens: Sequence[int],
                 pool_blocks, seed, bs=BLOCK_SIZE, note="") -> Batch:
    """Per-sequence lengths given; random distinct block tables; contiguous host blocks."""
    rng = np.random.Generator(np.random.PCG64(seed))
    prefix_lens = [int(x) for x in prefix_lens]
    suffix_lens = [int(x) for x in suffix_lens]
    bt = _random_tables(rng, prefix_lens, suffix_lens, bs, pool_blocks)
    hb, nhost = _contiguous_host_blocks(prefix_lens, bs)
    return Batch(name=name, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, block_size=bs,
                 pool_blocks=pool_blocks, host_store_blocks=nhost,
                 prefix_lens=prefix_lens, suffix_lens=suffix_lens,
                 block_tables=bt, host_blocks=hb, seed=seed, note=note)


def make_layer(batch: Batch, layer: int = 0, host_store: bool = True) -> LayerData:
    """Draw one layer's Q, new K/V and host-store payload from the layer's seed."""
    rng = np.random.Generator(np.random.PCG64(batch.layer_seed(layer)))
    T, Hq, Hkv, d, bs = batch.T, batch.num_q_heads, batch.num_kv_heads, batch.head_dim, batch.block_size
    q = normal_bf16(rng, (T, Hq, d))
    k_new = normal_bf16(rng, (T, Hkv, d))
    v_new = normal_bf16(rng, (T, Hkv, d))
    if host_store:
        nh = batch.host_store_blocks
        host_k = normal_bf16(rng, (nh, Hkv, bs * d))
        host_v = normal_bf16(rng, (nh, Hkv, bs * d))
    else:
        host_k = host_v = np.zeros((0, Hkv, bs * d), np.uint16)
    return LayerData(q=q, k_new=k_new, v_new=v_new, host_k=host_k, host_v=host_v)


def make_layers(batch: Batch, layers: Sequence[int], host_store: bool = True, workers: int = 8) -> List[LayerData]:
    """make_layer for several layers, drawn concurrently (each from its own layer seed, so
    the result is the same as drawing them one by one)."""
    from concurrent.futures import ThreadPoolExecutor
    layers = list(layers)
    with ThreadPoolExecutor(max(1, min(workers, len(layers)))) as ex:
        return list(ex.map(lambda l: make_layer(batch, l, host_store), layers))


def chunk_kv(node_id: int, layer: int, num_kv_heads: int, head_dim: int, blocks_per_chunk: int = 16,
             bs: int = BLOCK_SIZE):
    """K and V payload of one cached chunk of one layer, [blocks_per_chunk][Hkv][bs*d] bf16
    bits each, drawn from a seed derived from the tree node id and the layer (stands for
    the KV a model would have computed for that chunk)."""
    rng = np.random.Generator(np.random.PCG64(7_000_003 * (node_id + 1) + layer))
    shape = (blocks_per_chunk, num_kv_heads, bs * head_dim)
    return normal_bf16(rng, shape), normal_bf16(rng, shape)


def pipeline_data_sets(num_layers: int, distinct: int) -> List[int]:
    """Which of `distinct` generated data sets each layer of a pipeline uses: layer l takes
    set l % distinct. With distinct = num_layers every layer has its own data; with 6 sets
    the first, middle and last layers of the 32- and 80-layer stacks all differ."""
    return [l % max(1, min(distinct, num_layers)) for l in range(num_layers)]


# ----------------------------------------------------------------------------
# Token streams for the RAG-shaped mix (document ids only; no KV arithmetic)
# ----------------------------------------------------------------------------

@dataclass
class RagStream:
    doc_tokens: List[np.ndarray]     # per document: int32 token ids
    requests: List[np.ndarray]       # per request: int32 token ids (docs ++ query suffix)
    request_docs: List[List[int]]    # per request: document ids in order
    query_lens: List[int]


def finite_zipf_without_replacement(rng, n_items: int, k: int, s: float) -> List[int]:
    """k distinct items from {0..n_items-1}, P(item j) proportional to (j+1)^-s,
    drawn one at a time without replacement, kept in draw order."""
    w = np.arange(1, n_items + 1, dtype=np.float64) ** (-s)
    avail = np.ones(n_items, dtype=bool)
    out = []
    for _ in range(k):
        pw = np.where(avail, w, 0.0)
        pw = pw / pw.sum()
        j = int(rng.choice(n_items, p=pw))
        out.append(j)
        avail[j] = False
    return out


def rag_stream(seed: int, *, n_docs=64, doc_len=512, n_requests=80, docs_min=4, docs_max=8,
               zipf_s=1.1, query_min=32, query_max=512, vocab=32000) -> RagStream:
    """Synthetic retrieval-augmented request stream: each request concatenates
    4-8 documents drawn Zipf(1.1) without replacement, then a fresh query of
    32-512 tokens. Token ids are random; only their equality matters."""
    rng = np.random.Generator(np.random.PCG64(seed))
    docs = [rng.integers(0, vocab, size=doc_len, dtype=np.int32) for _ in range(n_docs)]
    reqs, rdocs, qlens = [], [], []
    for _ in range(n_requests):
        k = int(rng.integers(docs_min, docs_max + 1))
        ids = finite_zipf_without_replacement(rng, n_docs, k, zipf_s)
        qlen = int(rng.integers(query_min, query_max + 1))
        query = rng.integers(0, vocab, size=qlen, dtype=np.int32)
        reqs.append(np.concatenate([docs[j] for j in ids] + [query]).astype(np.int32))
        rdocs.append(ids)
        qlens.append(qlen)
    return RagStream(doc_tokens=docs, requests=reqs, request_docs=rdocs, query_lens=qlens)


# ----------------------------------------------------------------------------
# Workload registry (shapes of the measured configurations)
# ----------------------------------------------------------------------------

def tiny() -> Batch:
    """1 sequence, 8 q / 8 kv heads, d=64, 256 cached + 64 new tokens, 64-block pool;
    the block table is the first 20 entries of a random permutation of the pool."""
    return uniform_batch("tiny", B=1, Hq=8, Hkv=8, d=64, p=256, s=64, pool_blocks=64, seed=1)


def l8b_layer() -> Batch:
    """Llama-3-8B-shaped layer: batch 4, 32 q / 8 kv heads, d=128, 4096 cached +
    256 new tokens per sequence, 2048-block pool."""
    return uniform_batch("l8b_layer", B=4, Hq=32, Hkv=8, d=128, p=4096, s=256,
                         pool_blocks=2048, seed=2)


def l8b_pipe32(suffix: int = 256) -> Batch:
    """The Llama-3-8B layer shape repeated over 32 layers (distinct data per layer).
    suffix=6144 gives the compute-bound variant."""
    pool = 2048 if suffix <= 256 else 4096
    name = "l8b_pipe32" if suffix == 256 else f"l8b_pipe32_s{suffix}"
    return uniform_batch(name, B=4, Hq=32, Hkv=8, d=128, p=4096, s=suffix, pool_blocks=pool,
                         seed=3, num_layers=32, layer_seed_base=3000)


def l70b_pipe80() -> Batch:
    """70B-shaped long-context stack: batch 2, 64 q / 8 kv heads, d=128, 80 layers;
    16384-token context with the hit ending at 15360 (1024 new tokens), 4096-block pool."""
    return uniform_batch("l70b_pipe80", B=2, Hq=64, Hkv=8, d=128, p=15360, s=1024,
                         pool_blocks=4096, seed=5, num_layers=80, layer_seed_base=5000)


REGISTRY = {
    "tiny": tiny,
    "l8b_layer": l8b_layer,
    "l8b_pipe32": l8b_pipe32,
    "l70b_pipe80": l70b_pipe80,
}
