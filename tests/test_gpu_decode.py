"""GPU: decode rows (one new token per sequence) in the same attention launch as
prefill rows; the split-key decode entry point on ragged contexts, many short
sequences, every supported head shape and the decode-step benchmark's full size;
and a 16-step decode loop (append one token, attend over everything so far)
through both attention entry points, against the fp64 oracle at every step.

A decode row of a sequence with n visible keys is the oracle's suffix row of a
sequence with prefix n - 1 and a one-token suffix."""
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


def _decode_oracle(q, pk, pv, bt, ctx, Hkv, rows=None):
    pl = np.asarray(ctx, np.int32) - 1
    cu = np.arange(len(ctx) + 1, dtype=np.int32)
    return oattn.attention(q, pk, pv, bt, pl, cu, Hkv, BS, rows=rows)


def _decode_inputs(ctx, Hq, Hkv, d, seed, pool_blocks=None):
    """Random block tables (distinct blocks per sequence unless pool_blocks is given,
    then drawn with repeats from that many blocks), padded with -1; bf16 N(0,1) pool
    and queries."""
    rng = np.random.Generator(np.random.PCG64(seed))
    nbs = [-(-n // BS) for n in ctx]
    bt = np.full((len(ctx), max(nbs) + 1), -1, np.int32)
    if pool_blocks is None:
        pool_blocks = sum(nbs) + 3
        perm = rng.permutation(pool_blocks).astype(np.int32)
        cum = np.concatenate([[0], np.cumsum(nbs)])
        for i, nb in enumerate(nbs):
            bt[i, :nb] = perm[cum[i]:cum[i] + nb]
    else:
        for i, nb in enumerate(nbs):
            bt[i, :nb] = rng.integers(0, pool_blocks, nb, dtype=np.int32)
    shape = (pool_blocks, Hkv, BS * d)
    pk, pv = synth.normal_bf16(rng, shape), synth.normal_bf16(rng, shape)
    q = synth.normal_bf16(rng, (len(ctx), Hq, d))
    return q, pk, pv, bt


def _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d, workspace=None):
    pool = pcr.KVPool(dev(pk), dev(pv), Hkv, d)
    out = torch.zeros((len(ctx), Hq, d), dtype=torch.int16, device="cuda")
    cl = np.asarray(ctx, np.int32)
    pcr.decode_attn(dev(q), pool, dev(bt), dev(cl), cl, Hq, out, workspace=workspace)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("Hq,Hkv,d", [(32, 8, 128), (64, 8, 128), (64, 4, 128), (8, 8, 128), (32, 8, 64),
                                      (16, 1, 64)])
def test_decode_ragged_contexts(Hq, Hkv, d):
    """Contexts of one key, within one block, at block, step and chunk boundaries, and
    long: single-chunk sequences write the output directly, the others (cut into more
    than four chunks at this batch size) go through the workspace and the merge kernel."""
    ctx = [1, 2, 15, 16, 17, 31, 32, 33, 63, 255, 256, 257, 288, 289, 1000, 1088, 1089, 2176, 3001, 4352]
    q, pk, pv, bt = _decode_inputs(ctx, Hq, Hkv, d, seed=7 + Hq + d)
    say(f"[gpu] decode ragged Hq={Hq} Hkv={Hkv} d={d} B={len(ctx)} "
        f"workspace={pcr.decode_attn_workspace_bytes(len(ctx), Hq, Hkv, d, max(ctx))}")
    out = _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d)
    got = synth.bf16_bits_to_f32(u16(out)).astype(np.float64)
    _check(got, _decode_oracle(q, pk, pv, bt, ctx, Hkv), f"decode Hq={Hq} Hkv={Hkv} d={d}")


@pytest.mark.parametrize("B,d", [(32, 128), (48, 128), (100, 128), (32, 64)])
def test_decode_ragged_merged_in_workgroup(B, d):
    """Batches whose sequences are cut into 2-4 chunks merged inside one workgroup: the
    plan by the largest context, which needs no workspace (a one-byte workspace is
    given, too small for the plan by total keys); ragged contexts, so some chunks lie
    past a short sequence's end. Then the same batch with the workspace the size query
    asks for, which takes the plan by total keys (chunks merged through the workspace)."""
    Hq, Hkv = 32, 8
    rng = np.random.Generator(np.random.PCG64(B + d))
    ctx = [int(x) for x in rng.integers(1, 4353, B)]
    ctx[:6] = [1, 16, 33, 1100, 2200, 4352]
    q, pk, pv, bt = _decode_inputs(ctx, Hq, Hkv, d, seed=B * 3 + d)
    want = _decode_oracle(q, pk, pv, bt, ctx, Hkv)
    say(f"[gpu] decode merged in workgroup B={B} d={d}")
    tiny = torch.empty(1, dtype=torch.uint8, device="cuda")
    out = _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d, workspace=tiny)
    _check(synth.bf16_bits_to_f32(u16(out)).astype(np.float64), want, f"decode merged B={B} d={d}")
    out = _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d)
    _check(synth.bf16_bits_to_f32(u16(out)).astype(np.float64), want, f"decode by total keys B={B} d={d}")


@pytest.mark.parametrize("name", ["b64_1k_8k", "b16_rag_like", "b8_skewed"])
def test_decode_plan_by_total_keys(name):
    """Ragged batches that take the plan by total keys (long sequences get more chunks
    than short ones, merged through the workspace): every row against the oracle, the
    result bit-identical on a second call and to the allocation-free entry point (which
    makes the same plan)."""
    Hq, Hkv, d = 32, 8, 128
    rng = np.random.Generator(np.random.PCG64(41))
    if name == "b64_1k_8k":
        ctx = [int(x) for x in rng.integers(1024, 8193, 64)]
    elif name == "b16_rag_like":
        ctx = [int(x) for x in rng.integers(1200, 4600, 16)]
    else:   # one long sequence among short ones
        ctx = [16000, 40, 300, 17, 1000, 2, 513, 64]
    q, pk, pv, bt = _decode_inputs(ctx, Hq, Hkv, d, seed=43)
    say(f"[gpu] decode plan by total keys {name}: B={len(ctx)} keys={sum(ctx)} max={max(ctx)} "
        f"workspace={pcr.decode_attn_workspace_bytes(len(ctx), Hq, Hkv, d, max(ctx))}")
    out = _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d)
    got = synth.bf16_bits_to_f32(u16(out)).astype(np.float64)
    _check(got, _decode_oracle(q, pk, pv, bt, ctx, Hkv), f"decode total-keys plan {name}")
    again = _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d)
    assert torch.equal(out, again), "second call differs"
    pool = pcr.KVPool(dev(pk), dev(pv), Hkv, d)
    na = torch.zeros_like(out)
    cl = np.asarray(ctx, np.int32)
    pcr.decode_attn_noalloc(dev(q), pool, dev(bt), dev(cl), cl, Hq, na)
    torch.cuda.synchronize()
    assert torch.equal(out, na), "allocation-free entry point differs"


NAN_BITS = np.uint16(0x7FC1)


def _poison_past_end(pk, pv, bt, ctx):
    """NaN bit patterns in every slot of each sequence's last block past its context end
    (K and V): the slots a ragged step reads but must not use."""
    pk, pv = pk.copy(), pv.copy()
    for i, n in enumerate(ctx):
        if n % BS:
            blk = int(bt[i, (n - 1) // BS])
            pk[blk, :, (n % BS) * pk.shape[2] // BS:] = NAN_BITS   # K: slot-major rows of d
            vb = pv[blk].reshape(pv.shape[1], -1, BS)               # V: d-major rows of 16 slots
            vb[:, :, n % BS:] = NAN_BITS
    return pk, pv


@pytest.mark.parametrize("regime,B", [("one_chunk", 160), ("lds_merge", 40), ("workspace", 3)])
def test_decode_nan_past_context_end(regime, B):
    """Pool slots past each context end hold NaN bit patterns (never-written slots, or
    another request's garbage): the output stays finite and equal to the oracle, which
    never reads them. Contexts are not multiples of 16 and end in either block of the
    last 32-key step, for single-chunk sequences, chunks merged in the workgroup and
    chunks merged through the workspace."""
    Hq, Hkv, d = 32, 8, 128
    rng = np.random.Generator(np.random.PCG64(1000 + B))
    hi = {"one_chunk": 250, "lds_merge": 4000, "workspace": 40000}[regime]
    ctx = [int(x) for x in rng.integers(1, hi, B)]
    ctx = [n + 1 if n % BS == 0 else n for n in ctx]
    ctx[0] = 17 if regime == "one_chunk" else hi - 7
    ctx[1] = 9
    q, pk, pv, bt = _decode_inputs(ctx, Hq, Hkv, d, seed=2000 + B)
    pk, pv = _poison_past_end(pk, pv, bt, ctx)
    ws = pcr.decode_attn_workspace_bytes(B, Hq, Hkv, d, max(ctx))
    assert (ws > 0) == (regime != "one_chunk")
    say(f"[gpu] decode NaN past context end: {regime} B={B} max_ctx={max(ctx)} workspace={ws}")
    want = _decode_oracle(q, pk, pv, bt, ctx, Hkv)
    # lds_merge: a one-byte workspace keeps the plan by the largest context (chunks merged
    # in the workgroup); the full workspace then takes the plan by total keys
    runs = [torch.empty(1, dtype=torch.uint8, device="cuda"), None] if regime == "lds_merge" else [None]
    for w in runs:
        out = _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d, workspace=w)
        got = synth.bf16_bits_to_f32(u16(out)).astype(np.float64)
        _check(got, want, f"decode NaN tail {regime} ({'one-byte' if w is not None else 'queried'} workspace)")


def test_decode_long_contexts():
    """Contexts of 131072 and 65537 keys (two sequences): 64 and 33 chunks of 2048 keys
    merged through the workspace (the last one holding a single key), fp32 sums over
    131k keys."""
    ctx = [131072, 65537]
    Hq, Hkv, d = 32, 8, 128
    q, pk, pv, bt = _decode_inputs(ctx, Hq, Hkv, d, seed=13)
    say(f"[gpu] decode long contexts {ctx} workspace={pcr.decode_attn_workspace_bytes(2, Hq, Hkv, d, max(ctx))}")
    out = _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d)
    got = synth.bf16_bits_to_f32(u16(out)).astype(np.float64)
    _check(got, _decode_oracle(q, pk, pv, bt, ctx, Hkv), "decode long contexts")


@pytest.mark.parametrize("scale", [0.0, 8.0, 32.0])
def test_decode_softmax_flat_and_sharp(scale):
    """Queries scaled by 0 (the mean of the values), 8 and 32 (near one-hot, the
    running max rising step after step), across the in-workgroup and workspace merges."""
    ctx = [1, 40, 700, 3000, 4352, 9000]
    Hq, Hkv, d = 32, 8, 128
    q, pk, pv, bt = _decode_inputs(ctx, Hq, Hkv, d, seed=21)
    q = synth.f32_to_bf16_bits(synth.bf16_bits_to_f32(q) * np.float32(scale))
    say(f"[gpu] decode softmax scale x{scale}")
    out = _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d)
    got = synth.bf16_bits_to_f32(u16(out)).astype(np.float64)
    _check(got, _decode_oracle(q, pk, pv, bt, ctx, Hkv), f"decode q x{scale}")


def test_decode_many_short_sequences_without_workspace():
    """300 sequences of 1-300 keys: one chunk each, so no workspace is needed or passed."""
    rng = np.random.Generator(np.random.PCG64(5))
    ctx = [int(x) for x in rng.integers(1, 301, 300)]
    ctx[0], ctx[1] = 1, 300
    Hq, Hkv, d = 32, 8, 128
    assert pcr.decode_attn_workspace_bytes(len(ctx), Hq, Hkv, d, max(ctx)) == 0
    q, pk, pv, bt = _decode_inputs(ctx, Hq, Hkv, d, seed=6)
    say("[gpu] decode 300 short sequences")
    out = _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d, workspace=None)
    got = synth.bf16_bits_to_f32(u16(out)).astype(np.float64)
    _check(got, _decode_oracle(q, pk, pv, bt, ctx, Hkv), "decode short")


def test_decode_workspace_size_is_monotone():
    """A workspace sized for max_context serves every batch of the same size whose
    contexts are shorter: the size never decreases as max_context grows (host only,
    the query reads the device's compute-unit count)."""
    lens = [1, 2, 16, 31, 255, 256, 257, 300, 511, 1000, 1088, 2176, 4352, 4353, 16384, 131072]
    for B, Hq, Hkv, d in [(1, 32, 8, 128), (2, 32, 8, 128), (8, 64, 8, 128), (16, 16, 1, 64), (64, 32, 8, 128),
                          (512, 32, 8, 128)]:
        sizes = [pcr.decode_attn_workspace_bytes(B, Hq, Hkv, d, n) for n in lens]
        assert all(a <= b for a, b in zip(sizes, sizes[1:])), (B, Hq, Hkv, d, sizes)
        assert sizes[0] == 0


def test_decode_workspace_checked():
    """A workspace smaller than the batch needs is refused before anything is enqueued."""
    ctx = [4000, 3000]
    Hq, Hkv, d = 32, 8, 128
    need = pcr.decode_attn_workspace_bytes(len(ctx), Hq, Hkv, d, max(ctx))
    assert need > 0
    q, pk, pv, bt = _decode_inputs(ctx, Hq, Hkv, d, seed=8)
    small = torch.empty(need // 2, dtype=torch.uint8, device="cuda")
    with pytest.raises(pcr.PcrError) as e:
        _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d, workspace=small)
    assert e.value.status == pcr.PCR_ERR_INVALID_ARG and "workspace" in str(e.value)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    out = _decode_gpu(q, pk, pv, bt, ctx, Hq, Hkv, d, workspace=ws)
    got = synth.bf16_bits_to_f32(u16(out)).astype(np.float64)
    _check(got, _decode_oracle(q, pk, pv, bt, ctx, Hkv), "decode exact workspace")


def test_decode_step_full_size_sampled_and_deterministic():
    """The decode-step benchmark's shape (64 sequences x 4352 keys, 32 q / 8 kv heads,
    d = 128) in its launch configuration, over a 4096-block pool that the sequences
    share: every head of six sequences against the oracle, the whole output against
    the prefill kernel's one-token-suffix rows, and a second call bit for bit."""
    B, ctx_len, Hq, Hkv, d = 64, 4352, 32, 8, 128
    ctx = [ctx_len] * B
    q, pk, pv, bt = _decode_inputs(ctx, Hq, Hkv, d, seed=71, pool_blocks=4096)
    say("[gpu] decode full size B=64 x 4352")
    pool = pcr.KVPool(dev(pk), dev(pv), Hkv, d)
    qd, btd = dev(q), dev(bt)
    cl = np.asarray(ctx, np.int32)
    cld = dev(cl)
    out1 = torch.zeros((B, Hq, d), dtype=torch.int16, device="cuda")
    out2 = torch.zeros_like(out1)
    pcr.decode_attn(qd, pool, btd, cld, cl, Hq, out1)
    pcr.decode_attn(qd, pool, btd, cld, cl, Hq, out2)
    ref = torch.zeros_like(out1)
    pl = cl - 1
    cu = np.arange(B + 1, dtype=np.int32)
    pcr.prefix_prefill_attn(qd, pool, btd, dev(pl), dev(cu), pl, cu, Hq, ref)
    torch.cuda.synchronize()
    assert torch.equal(out1, out2)
    seqs = [0, 1, 17, 40, 62, 63]
    rows = np.array([[t, h] for t in seqs for h in range(Hq)], np.int32)
    got = synth.bf16_bits_to_f32(u16(out1)).astype(np.float64)
    _check(got[rows[:, 0], rows[:, 1]], _decode_oracle(q, pk, pv, bt, ctx, Hkv, rows=rows), "decode full sampled")
    # both kernels are within the tolerance of the oracle; against each other the
    # bound is twice that
    diff = np.abs(got - synth.bf16_bits_to_f32(u16(ref)).astype(np.float64))
    say(f"    decode vs prefill kernel: max_abs={diff.max():.3e} mean_abs={diff.mean():.3e}")
    assert diff.max() <= 2 * MAX_ABS and diff.mean() <= MEAN_ABS


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
        out_dec = torch.zeros_like(out)
        n_keys = pl + 1
        pcr.decode_attn(dev(q), L.pool, bt_dev, dev(n_keys), n_keys, Hq, out_dec)
        torch.cuda.synchronize()
        odm.append(pk, pv, kn, vn, slots, BS)
        want = oattn.attention(q, pk, pv, b.block_tables, pl, cu, Hkv, BS)
        got = synth.bf16_bits_to_f32(u16(out)).astype(np.float64)
        _check(got, want, f"decode step {step}")
        got = synth.bf16_bits_to_f32(u16(out_dec)).astype(np.float64)
        _check(got, want, f"decode step {step} (decode entry point)")
    assert np.array_equal(u16(L.pool.k), pk) and np.array_equal(u16(L.pool.v), pv)
    assert all(t <= b.block_tables.shape[1] * BS for t in total)
