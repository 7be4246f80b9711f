"""GPU: decode rows (one new token per sequence) in the same attention launch as
prefill rows, and a 16-step decode loop (append one token, attend over everything
so far) against the fp64 oracle at every step."""
import numpy as np
import pytest
import torch

from oracle import attention as oattn
from oracle import datamove as odm
from paper_2603_23049_amd import pcr, synth
from gpuio import GpuLayer, MAX_ABS, MEAN_ABS, dev, error_stats, say, u16

pytestmark = pytest.mark.gpu

BS = 16


def _check(got, want, label):
    mx, mean = error_stats(got, want)
    say(f"    {label}: max_abs={mx:.3e} mean_abs={mean:.3e}")
    assert np.all(np.isfinite(got)) and mx <= MAX_ABS and mean <= MEAN_ABS, (label, mx, mean)


def test_mixed_prefill_and_decode_rows():
    """One long prefill beside many single-token sequences (cached contexts of many
    lengths, including none and a partial last block)."""
    prefix = [3072, 4095, 1, 0, 17, 512, 1000, 2047, 2048, 15]
    suffix = [300, 1, 1, 1, 1, 1, 1, 1, 1, 1]
    b = synth.ragged_batch("mixed", Hq=32, Hkv=8, d=128, prefix_lens=prefix, suffix_lens=suffix, pool_blocks=1024,
                           seed=41)
    data = synth.make_layer(b)
    rng = np.random.Generator(np.random.PCG64(42))
    shape = (b.pool_blocks, b.num_kv_heads, BS * b.head_dim)
    pk0, pv0 = synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)
    say("[gpu] mixed prefill + decode rows")
    L = GpuLayer(b, data, pk0, pv0)
    L.run_serial("kernel_pull")
    plan = odm.plan(b.prefix_lens, b.suffix_lens, b.block_tables, b.host_blocks, BS)
    pk, pv = odm.pool_after_layer(pk0, pv0, data.host_k, data.host_v, plan, data.k_new, data.v_new, BS)
    want = oattn.attention(data.q, pk, pv, b.block_tables, np.asarray(prefix, np.int32), plan[3], 8, BS)
    _check(L.out_f64(), want, "mixed")


def test_decode_loop_16_steps():
    """Prefill 2 sequences (cached prefix + prompt), then 16 decode steps: each step
    appends one token per sequence at the next position and attends over all keys."""
    B, Hq, Hkv, d = 2, 32, 8, 128
    prefix, prompt, steps = [1024, 200], [64, 100], 16
    total = [p + s + steps for p, s in zip(prefix, prompt)]
    b = synth.ragged_batch("dec", Hq=Hq, Hkv=Hkv, d=d, prefix_lens=prefix,
                           suffix_lens=[s + steps for s in prompt], pool_blocks=256, seed=43)
    data = synth.make_layer(b)
    # the prefill step over the prompt only (same block tables, shorter suffixes)
    pre = synth.Batch(name="dec_prefill", num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, block_size=BS,
                      pool_blocks=b.pool_blocks, host_store_blocks=b.host_store_blocks, prefix_lens=prefix,
                      suffix_lens=list(prompt), block_tables=b.block_tables, host_blocks=b.host_blocks, seed=43)
    cu_full = b.cu_suffix
    rows_prompt = np.concatenate([np.arange(cu_full[i], cu_full[i] + prompt[i]) for i in range(B)])
    pdata = synth.LayerData(q=data.q[rows_prompt], k_new=data.k_new[rows_prompt], v_new=data.v_new[rows_prompt],
                            host_k=data.host_k, host_v=data.host_v)
    zero = np.zeros((b.pool_blocks, Hkv, BS * d), np.uint16)
    say("[gpu] decode loop: prefill")
    L = GpuLayer(pre, pdata, zero, zero)
    L.run_serial("kernel_pull")
    # oracle pool state, updated step by step the same way
    plan = odm.plan(prefix, prompt, b.block_tables, b.host_blocks, BS)
    pk, pv = odm.pool_after_layer(zero, zero, data.host_k, data.host_v, plan, pdata.k_new, pdata.v_new, BS)
    bt_dev = dev(b.block_tables)
    for step in range(steps):
        ctx = [p + s + step for p, s in zip(prefix, prompt)]            # tokens already in the pool
        rows = np.array([cu_full[i] + prompt[i] + step for i in range(B)])
        q, kn, vn = data.q[rows], data.k_new[rows], data.v_new[rows]
        slots = np.array([int(b.block_tables[i][ctx[i] // BS]) * BS + ctx[i] % BS for i in range(B)], np.int32)
        pcr.append_kv(L.pool, dev(kn), dev(vn), dev(slots))
        out = torch.zeros((B, Hq, d), dtype=torch.int16, device="cuda")
        pl = np.asarray(ctx, np.int32)
        cu = np.arange(B + 1, dtype=np.int32)
        pcr.prefix_prefill_attn(dev(q), L.pool, bt_dev, dev(pl), dev(cu), pl, cu, Hq, out)
        torch.cuda.synchronize()
        odm.append(pk, pv, kn, vn, slots, BS)
        want = oattn.attention(q, pk, pv, b.block_tables, pl, cu, Hkv, BS)
        got = synth.bf16_bits_to_f32(u16(out)).astype(np.float64)
        _check(got, want, f"decode step {step}")
    assert np.array_equal(u16(L.pool.k), pk) and np.array_equal(u16(L.pool.v), pv)
    assert all(t <= b.block_tables.shape[1] * BS for t in total)
