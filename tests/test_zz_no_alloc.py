"""GPU: the allocation-free decode entry point (pcr_decode_attn_noalloc) against the
workspace entry point (pcr_decode_attn) through the C ABI: bit for bit on the same
inputs, and both within the tolerance of the fp64 oracle, on two calls in a row
whose second batch is smaller (the scratch keeps the first call's contents)."""
import numpy as np
import pytest
import torch

from oracle import attention as oattn
from paper_2603_23049_amd import pcr, synth
from gpuio import MAX_ABS, MEAN_ABS, dev, error_stats, say, u16

pytestmark = pytest.mark.gpu

BS = 16


def _inputs(ctx, Hq, Hkv, d, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    nbs = [-(-n // BS) for n in ctx]
    pool_blocks = sum(nbs) + 5
    perm = rng.permutation(pool_blocks).astype(np.int32)
    bt = np.full((len(ctx), max(nbs) + 1), -1, np.int32)
    off = 0
    for i, nb in enumerate(nbs):
        bt[i, :nb] = perm[off:off + nb]
        off += nb
    shape = (pool_blocks, Hkv, BS * d)
    pk, pv = synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)
    q = synth.normal_bf16(rng, (len(ctx), Hq, d))
    return q, pk, pv, bt


def _both(ctx, Hq, Hkv, d, seed):
    q, pk, pv, bt = _inputs(ctx, Hq, Hkv, d, seed)
    pool = pcr.KVPool(dev(pk), dev(pv), Hkv, d)
    qd, btd = dev(q), dev(bt)
    cl = np.asarray(ctx, np.int32)
    cld = dev(cl)
    out_na = torch.zeros((len(ctx), Hq, d), dtype=torch.int16, device="cuda")
    out_ws = torch.zeros_like(out_na)
    n = pcr.decode_attn_workspace_bytes(len(ctx), Hq, Hkv, d, max(ctx))
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device="cuda")
    pcr.decode_attn_noalloc(qd, pool, btd, cld, cl, Hq, out_na)
    pcr.decode_attn(qd, pool, btd, cld, cl, Hq, out_ws, workspace=ws)
    torch.cuda.synchronize()
    want = oattn.attention(q, pk, pv, bt, cl - 1, np.arange(len(ctx) + 1, dtype=np.int32), Hkv, BS)
    return u16(out_na), u16(out_ws), want, n


def test_noalloc_decode_equals_workspace_decode_twice():
    Hq, Hkv, d = 32, 8, 128
    # first call: chunks merged through the scratch (long contexts, few sequences)
    big = [40000, 17, 12345, 65537]
    # second call, smaller: fewer sequences and keys, still merged through the scratch
    small = [3001, 777]
    for label, ctx, seed in (("first (larger)", big, 5), ("second (smaller)", small, 6)):
        na, ws, want, n = _both(ctx, Hq, Hkv, d, seed)
        say(f"[gpu] noalloc decode {label}: B={len(ctx)} max_ctx={max(ctx)} scratch used={n} bytes")
        assert 0 < n <= pcr.DECODE_NOALLOC_SCRATCH_BYTES
        assert np.array_equal(na, ws), f"{label}: allocation-free result differs from the workspace entry point"
        got = synth.bf16_bits_to_f32(na).astype(np.float64)
        mx, mean = error_stats(got, want)
        say(f"    max_abs={mx:.3e} mean_abs={mean:.3e}")
        assert np.all(np.isfinite(got)) and mx <= MAX_ABS and mean <= MEAN_ABS


def test_noalloc_decode_without_scratch_and_shapes():
    """Batches that need no scratch (one chunk per sequence, or chunks merged in the
    workgroup) and other head shapes give the same bits as the workspace entry point."""
    for ctx, Hq, Hkv, d, seed in (([5, 300, 129] * 60, 32, 8, 128, 7), ([4000] * 40, 32, 8, 128, 8),
                                  ([9000, 31], 16, 1, 64, 9), ([20000, 4097, 1], 64, 8, 128, 10)):
        na, ws, want, n = _both(ctx, Hq, Hkv, d, seed)
        say(f"[gpu] noalloc decode B={len(ctx)} Hq={Hq} Hkv={Hkv} d={d} scratch={n}")
        assert np.array_equal(na, ws)
        got = synth.bf16_bits_to_f32(na).astype(np.float64)
        mx, mean = error_stats(got, want)
        assert np.all(np.isfinite(got)) and mx <= MAX_ABS and mean <= MEAN_ABS, (mx, mean)
