"""Host prefix tree (Sec. 4.2): the paper's look-ahead example, hit lengths against a
brute-force oracle, eviction invariants, and the RAG-mix batch built from it."""
import json
import os

import numpy as np
import pytest

from oracle import datamove as odm
from oracle import tree as otree
from paper_2603_23049_amd import prefix_tree as pt
from paper_2603_23049_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "lookahead_lru_leafset.json")


def _example_tree(spec, lookahead):
    """Chunks of one token each; each chunk's token is its number (C7 -> 7)."""
    tok = {name: int(name[1:]) for name, _ in spec["tree"]}
    tok[spec["insert"]["name"]] = int(spec["insert"]["name"][1:])
    parent = {name: par for name, par in spec["tree"]}

    def path(name):
        out = []
        while name != "root":
            out.append(name)
            name = parent[name]
        return out[::-1]

    tree = pt.PrefixTree(chunk_tokens=1, block_size=1, capacity_chunks=spec["capacity_chunks"],
                         lookahead=lookahead)
    # insert root-to-leaf paths in the given recency order (oldest leaf first)
    for leaf in spec["leaf_order_before"]:
        names = path(leaf)
        have = len(tree.match([tok[n] for n in names]))
        tree.insert([tok[n] for n in names], names=names[have:])
    return tree, tok


def test_paper_lookahead_example():
    spec = json.load(open(GOLDEN))
    for lookahead, expect in ((True, spec["leaf_set_after_lookahead"]), (False, spec["leaf_set_after_plain_lru"])):
        tree, tok = _example_tree(spec, lookahead)
        assert tree.leaf_names() == spec["leaf_order_before"]
        assert tree.n_chunks == spec["capacity_chunks"]
        current = [tok[n] for n in spec["current_request_path"]] + [tok[spec["insert"]["name"]]]
        assert [n.name for n in tree.match(current)] == spec["current_request_path"]
        nxt = [tok[n] for n in spec["next_request_path"]]
        tree.insert(current, pending=[nxt], names=[spec["insert"]["name"]])
        assert tree.leaf_names() == expect, (lookahead, tree.leaf_names())
        assert tree.n_chunks == spec["capacity_chunks"]


@pytest.mark.parametrize("seed", [4, 5, 6])
def test_hit_lengths_match_brute_force(seed):
    stream = synth.rag_stream(seed, n_requests=96)
    tree = pt.PrefixTree()
    reqs = stream.requests
    for i in range(64):
        tree.insert(reqs[i])
    for req in reqs[64:]:
        assert tree.hit_length(req) == otree.cached_prefix_tokens(req, reqs[:64], 256, 16)


def test_whole_request_cached_keeps_one_block_to_compute():
    tree = pt.PrefixTree(chunk_tokens=32, block_size=16)
    req = list(range(64))
    tree.insert(req)
    assert tree.hit_length(req) == 48
    assert otree.cached_prefix_tokens(req, [req], 32, 16) == 48


def test_eviction_keeps_tree_consistent_under_capacity():
    stream = synth.rag_stream(7, n_requests=120)
    for lookahead in (True, False):
        tree = pt.PrefixTree(capacity_chunks=60, lookahead=lookahead)
        reqs = stream.requests
        for i, req in enumerate(reqs):
            tree.insert(req, pending=reqs[i + 1:i + 5])
            # walk the tree: leaf set == nodes without children; chunk count; capacity
            seen, stack = 0, [tree.root]
            childless = set()
            while stack:
                n = stack.pop()
                for c in n.children.values():
                    assert c.parent is n
                    seen += 1
                    stack.append(c)
                    if not c.children:
                        childless.add(c)
            assert seen == tree.n_chunks
            assert set(tree.leaves) == childless
            assert tree.n_chunks <= 60 + len(tree.chunks(req))
        assert tree.evicted
        for n in tree.evicted:          # evicted nodes left the tree from a leaf position
            assert n.key not in n.parent.children or n.parent.children[n.key] is not n


def test_lookahead_raises_hit_ratio_under_capacity():
    la = pt.hit_ratio_under_capacity(4, capacity_chunks=200, lookahead=True, n_requests=200)
    lru = pt.hit_ratio_under_capacity(4, capacity_chunks=200, lookahead=False, n_requests=200)
    full = pt.hit_ratio_under_capacity(4, capacity_chunks=None, lookahead=True, n_requests=200)
    assert lru <= la <= full


def test_rag_mix_batch_structure():
    b = pt.rag_mix_batch()
    assert b.B == 16 and b.num_q_heads == 32 and b.num_kv_heads == 8 and b.head_dim == 128
    assert all(p % 16 == 0 for p in b.prefix_lens)
    assert all(s >= 1 for s in b.suffix_lens)
    assert 0.05 < b.extra["hit_ratio"] < 0.5
    # shared tree chunks load once: the plan dedupes them and accepts the tables
    src, dst, slots, cu = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, 16)
    assert len(src) == len(set(dst.tolist())) == b.host_store_blocks
    used = b.block_tables[b.block_tables >= 0]
    assert used.max() < b.pool_blocks
    # hits agree with the brute-force oracle over the warm-up stream
    stream = synth.rag_stream(4, n_requests=80)
    for req, p in zip(stream.requests[64:], b.prefix_lens):
        assert p == otree.cached_prefix_tokens(req, stream.requests[:64], 256, 16)
