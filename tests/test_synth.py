"""Pins for the seeded input generators (CPU only)."""
import numpy as np
import torch

from paper_2603_23049_amd import synth


def test_bf16_rounding_matches_torch():
    rng = np.random.Generator(np.random.PCG64(0))
    x = np.concatenate([rng.standard_normal(200000, dtype=np.float32) * 10.0 ** rng.integers(-30, 30, 200000),
                        np.array([0.0, -0.0, 1.0, -1.0, 3.3895314e38, 1.0000001, 1.00390625,
                                  1.01171875, 65504.0], np.float32)]).astype(np.float32)
    x = x[np.isfinite(x)]
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = synth.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_generators_are_deterministic():
    a = synth.make_layer(synth.tiny())
    b = synth.make_layer(synth.tiny())
    for f in ("q", "k_new", "v_new", "host_k", "host_v"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    c = synth.make_layer(synth.l8b_pipe32(), layer=1, host_store=False)
    d = synth.make_layer(synth.l8b_pipe32(), layer=2, host_store=False)
    assert not np.array_equal(c.q, d.q)


def test_tiny_block_table_is_permutation_prefix():
    b = synth.tiny()
    rng = np.random.Generator(np.random.PCG64(1))
    perm = rng.permutation(64)
    assert list(b.block_tables[0]) == list(perm[:20])
    assert b.host_store_blocks == 16 and b.T == 64


def test_config_shapes():
    b = synth.l8b_layer()
    assert (b.B, b.num_q_heads, b.num_kv_heads, b.head_dim) == (4, 32, 8, 128)
    used = b.block_tables[b.block_tables >= 0]
    assert used.size == 4 * 272 and len(set(used.tolist())) == used.size and used.max() < 2048
    c = synth.l70b_pipe80()
    assert c.prefix_lens == [15360, 15360] and c.suffix_lens == [1024, 1024] and c.num_layers == 80


def test_zipf_without_replacement_distinct_and_skewed():
    rng = np.random.Generator(np.random.PCG64(3))
    counts = np.zeros(64)
    for _ in range(2000):
        ids = synth.finite_zipf_without_replacement(rng, 64, 6, 1.1)
        assert len(set(ids)) == 6
        counts[ids[0]] += 1
    # the first draw follows P(j) ~ (j+1)^-1.1
    w = np.arange(1, 65) ** -1.1
    w /= w.sum()
    assert abs(counts[0] / 2000 - w[0]) < 0.03
    assert counts[0] > counts[10] > counts[60] or counts[60] == 0


def test_kv_bytes_per_token_pins_paper_capacity_example():
    # Sec. 3: an 80 GB GPU holds the KV of about 163,000 Llama2-7B tokens
    # (32 layers, 32 kv heads, head dim 128, 16-bit K and V).
    per_token = 2 * 32 * 32 * 128 * 2
    assert 80 * 2 ** 30 // per_token == 163840
