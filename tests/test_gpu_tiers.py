"""GPU: the SSD and DRAM tiers on the data path (Sec. 4.4 prefetch and write-back; Alg. 1
upload from DRAM, download after compute).

Chunks of a warm-up request are written to the SSD tier and dropped from DRAM. A later
request sharing its prefix is matched in the prefix tree; its cached chunks are read
from SSD into pinned DRAM slots (KVTier), and the DRAM slots are the host store the
layer loads read. The three-stream pipeline then loads, computes and offloads each
layer, the offload writing the request's newly computed whole chunks straight into
fresh DRAM slots, which are written back to SSD, dropped, and read back into other
slots. Checked bit for bit: every layer's pool against the oracle's load and append
from the chunks' original payloads, and the computed chunks read back from SSD
against the oracle's offload of the oracle pool."""
import os
import shutil
import tempfile

import numpy as np
import pytest
import torch

from oracle import datamove as odm
from paper_2603_23049_amd import pcr, prefetch, synth
from paper_2603_23049_amd.prefix_tree import PrefixTree
from gpuio import dev, say, u16

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BS, CHUNK = 16, 256
NAN_BITS = np.uint16(0x7FC1)


@pytest.fixture
def scratch():
    base = os.path.join(ROOT, ".pytest_store")
    os.makedirs(base, exist_ok=True)
    d = tempfile.mkdtemp(dir=base)
    yield d
    shutil.rmtree(d, ignore_errors=True)


def test_ssd_dram_pool_offload_round_trip(scratch):
    Hq, Hkv, d, n_layers = 16, 2, 128, 3
    bpc = CHUNK // BS
    stream = synth.rag_stream(21, n_docs=6, doc_len=512, n_requests=2, docs_min=3, docs_max=3, query_min=300,
                              query_max=300)
    warm, req = stream.requests
    tree = PrefixTree(chunk_tokens=CHUNK)
    tier = prefetch.KVTier(os.path.join(scratch, "ssd.bin"), n_slots=24, n_layers=n_layers, num_kv_heads=Hkv,
                           head_dim=d)
    try:
        # warm-up request: its chunks' KV (seeded per node and layer) go to DRAM, then SSD, then leave DRAM
        for node in tree.insert(warm):
            slot = tier.alloc(node.node_id, protect=set())
            for l in range(n_layers):
                k, v = synth.chunk_kv(node.node_id, l, Hkv, d, bpc)
                tier.part(l, slot, 0).copy_(torch.from_numpy(k.view(np.int16)))
                tier.part(l, slot, 1).copy_(torch.from_numpy(v.view(np.int16)))
            tier.write_back(node.node_id)
        warm_ids = list(tier.where)
        for nid in warm_ids:
            tier.drop(nid)
        for h in tier.layers:                       # no stale DRAM copy can pass for a read
            h.k.fill_(int(NAN_BITS))
            h.v.fill_(int(NAN_BITS))
        # the request: cached chain read from SSD into DRAM slots
        chain = tree.match(req)
        assert len(chain) >= 2, "the request should share the warm-up request's prefix"
        need = {n.node_id for n in chain}
        for n in chain:
            assert tier.start_read(n.node_id, protect=need)
        for n in chain:
            tier.finish_read(n.node_id)
        p = len(chain) * CHUNK
        s = len(req) - p
        say(f"[gpu] tiers: {len(chain)} cached chunks read from SSD, p={p} s={s}, {n_layers} layers")
        host_blocks = np.concatenate([tier.slot_blocks(tier.slot_of(n.node_id)) for n in chain])[None, :]
        b = synth.ragged_batch("tiers", Hq=Hq, Hkv=Hkv, d=d, prefix_lens=[p], suffix_lens=[s], pool_blocks=160,
                               seed=22)
        b.host_blocks = host_blocks.astype(np.int32)
        b.num_layers = n_layers
        # new whole chunks of the request: tree nodes, DRAM slots, offload list into those slots
        new_nodes = tree.insert(req)[len(chain):]
        off_src, off_dst0 = pcr.plan_offload(b.prefix_lens, b.suffix_lens, b.block_tables, BS, CHUNK)
        assert len(off_src) == len(new_nodes) * bpc and len(new_nodes) > 0
        protect = need | {n.node_id for n in new_nodes}
        new_slots = [tier.alloc(n.node_id, protect) for n in new_nodes]
        off_dst = np.concatenate([tier.slot_blocks(sl) for sl in new_slots]).astype(np.int32)
        # per-layer GPU data and the pipeline (load from DRAM slots, compute, offload into DRAM slots)
        shape = (b.pool_blocks, Hkv, BS * d)
        poison = np.full(shape, NAN_BITS, np.uint16)
        src, dst, slots, cu = pcr.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
        datas = [synth.make_layer(b, l, host_store=False) for l in range(n_layers)]
        layers = []
        for l, data in enumerate(datas):
            pool = pcr.KVPool(dev(poison), dev(poison), Hkv, d)
            layers.append(pcr.Layer(tier.layers[l], pool, dev(data.q), dev(data.k_new), dev(data.v_new),
                                    torch.zeros(data.q.shape, dtype=torch.int16, device="cuda")))
        pl = np.asarray(b.prefix_lens, np.int32)
        bp = pcr.BatchPlan(src, dst, dev(slots), dev(b.block_tables), dev(pl), dev(cu), pl, cu, Hq,
                           1.0 / np.sqrt(d))
        cs, ks, os_ = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
        pcr.pipeline_run_offload(layers, tier.layers, bp, off_src, off_dst, cs, ks, os_, method="auto",
                                 offload_method="kernel_pull")
        torch.cuda.synchronize()
        # oracle: the host store as the chunks' original payloads in the batch's host-block order
        plan = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
        want_chunks = {}
        for l, data in enumerate(datas):
            ref_k = np.zeros((tier.n_slots * bpc, Hkv, BS * d), np.uint16)
            ref_v = np.zeros_like(ref_k)
            for n in chain:
                k, v = synth.chunk_kv(n.node_id, l, Hkv, d, bpc)
                blocks = tier.slot_blocks(tier.slot_of(n.node_id))
                ref_k[blocks], ref_v[blocks] = k, v
            pk, pv = odm.pool_after_layer(poison, poison, ref_k, ref_v, plan, data.k_new, data.v_new, BS)
            assert np.array_equal(u16(layers[l].pool.k), pk) and np.array_equal(u16(layers[l].pool.v), pv), \
                f"layer {l}: pool after SSD -> DRAM -> pool load and append differs from the oracle"
            odm.offload(pk, pv, ref_k, ref_v, off_src, off_dst)
            for i, n in enumerate(new_nodes):
                blocks = tier.slot_blocks(new_slots[i])
                want_chunks[(n.node_id, l)] = (ref_k[blocks].copy(), ref_v[blocks].copy())
        # write the computed chunks back to SSD, drop them from DRAM, read them into other slots
        for n in new_nodes:
            tier.write_back(n.node_id)
        for n in new_nodes:
            tier.drop(n.node_id)
        for h in tier.layers:
            h.k.fill_(int(NAN_BITS))
            h.v.fill_(int(NAN_BITS))
        tier.free.reverse()                         # the read-back lands in different slots
        for n in new_nodes:
            assert tier.start_read(n.node_id, protect={m.node_id for m in new_nodes})
        moved = 0
        for i, n in enumerate(new_nodes):
            tier.finish_read(n.node_id)
            moved += new_slots[i] != tier.slot_of(n.node_id)
            for l in range(n_layers):
                wk, wv = want_chunks[(n.node_id, l)]
                sl = tier.slot_of(n.node_id)
                assert np.array_equal(u16(tier.part(l, sl, 0)), wk) and np.array_equal(u16(tier.part(l, sl, 1)), wv), \
                    f"chunk {n.node_id} layer {l}: SSD round trip differs from the oracle's offload"
        assert moved > 0
        st = tier.store.stats()
        say(f"    {len(new_nodes)} computed chunks offloaded, written back and read back; "
            f"SSD read {st['bytes_read'] >> 20} MiB, written {st['bytes_written'] >> 20} MiB, O_DIRECT={st['direct_io']}, "
            f"{st['direct_fallbacks']} transfers through the page cache")
    finally:
        tier.close()
