"""Test helpers: place contiguous per-sequence K/V into a paged pool.

The pool layout (bf16 bits, per block and kv head a payload of bs*d elements):
K element (slot o, dim x) at payload index o*d + x; V element at x*bs + o.
These helpers restate that layout with numpy reshapes, independently of both
the oracle's element-wise loops and the HIP kernels.
"""
import numpy as np

from paper_2603_23049_amd import synth


def ceil_div(a, b):
    return -(-a // b)


def random_tables(rng, lens, bs, pool_blocks):
    need = [ceil_div(n, bs) for n in lens]
    perm = rng.permutation(pool_blocks).astype(np.int32)
    bt = np.full((len(lens), max(max(need), 1)), -1, np.int32)
    off = 0
    for b, n in enumerate(need):
        bt[b, :n] = perm[off:off + n]
        off += n
    assert off <= pool_blocks
    return bt


def scatter_sequence(pool_k, pool_v, bt_row, k_seq, v_seq, bs):
    """Write contiguous K/V [n][Hkv][d] of one sequence into its blocks."""
    n, Hkv, d = k_seq.shape
    nb = ceil_div(n, bs)
    pad = nb * bs - n
    kp = np.concatenate([k_seq, np.zeros((pad, Hkv, d), k_seq.dtype)]) if pad else k_seq
    vp = np.concatenate([v_seq, np.zeros((pad, Hkv, d), v_seq.dtype)]) if pad else v_seq
    kb = kp.reshape(nb, bs, Hkv, d).transpose(0, 2, 1, 3).reshape(nb, Hkv, bs * d)
    vb = vp.reshape(nb, bs, Hkv, d).transpose(0, 2, 3, 1).reshape(nb, Hkv, d * bs)
    for j in range(nb):
        blk = bt_row[j]
        if pad and j == nb - 1:
            # only the valid slots of a partial last block are written
            full_k = pool_k[blk].reshape(Hkv, bs, d)
            full_v = pool_v[blk].reshape(Hkv, d, bs)
            r = bs - pad
            full_k[:, :r, :] = kb[j].reshape(Hkv, bs, d)[:, :r, :]
            full_v[:, :, :r] = vb[j].reshape(Hkv, d, bs)[:, :, :r]
        else:
            pool_k[blk] = kb[j]
            pool_v[blk] = vb[j]


def bf16_to_f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)
