"""Pins for the fp64 attention oracle (CPU only).

Each test checks the oracle against something other than itself:
  * a library routine on the plain definition: torch's scaled_dot_product_attention
    in float64 over the contiguous full sequence (full prefill), of which the
    suffix rows must equal the reuse-prefill rows (Sec. 2.2: exact prefix reuse);
  * scipy's softmax through a value matrix that is the identity basis;
  * closed forms (constant values, equal keys, the first causal row, one
    dominant logit) and invariants (physical block permutation, reuse = full
    prefill inside the oracle itself).
"""
import numpy as np
import pytest
import torch
from scipy.special import softmax

from oracle import attention as oattn
from paper_2603_23049_amd import synth
from pagedkv import bf16_to_f64, random_tables, scatter_sequence, ceil_div

BS = 16


def _build_case(rng, seqs, Hkv, G, d, pool_extra=3):
    """seqs: list of (p, s). Returns dict with contiguous fp64 tensors and the paged pool."""
    Hq = Hkv * G
    lens = [p + s for p, s in seqs]
    pool_blocks = sum(ceil_div(n, BS) for n in lens) + pool_extra
    bt = random_tables(rng, lens, BS, pool_blocks)
    pool_k = synth.normal_bf16(rng, (pool_blocks, Hkv, BS * d))   # garbage in unused slots
    pool_v = synth.normal_bf16(rng, (pool_blocks, Hkv, BS * d))
    full_q, full_k, full_v = [], [], []
    for b, n in enumerate(lens):
        qf = synth.normal_bf16(rng, (n, Hq, d))
        kf = synth.normal_bf16(rng, (n, Hkv, d))
        vf = synth.normal_bf16(rng, (n, Hkv, d))
        scatter_sequence(pool_k, pool_v, bt[b], kf, vf, BS)
        full_q.append(qf)
        full_k.append(kf)
        full_v.append(vf)
    q_suffix = np.concatenate([full_q[b][p:] for b, (p, s) in enumerate(seqs)])
    prefix_lens = np.array([p for p, _ in seqs], np.int32)
    cu = np.concatenate([[0], np.cumsum([s for _, s in seqs])]).astype(np.int32)
    return dict(Hq=Hq, bt=bt, pool_k=pool_k, pool_v=pool_v, q=q_suffix, prefix_lens=prefix_lens,
                cu=cu, full_q=full_q, full_k=full_k, full_v=full_v)


def _sdpa_full_prefill_rows(case, seqs, G, d):
    """Full causal prefill of each whole sequence (torch, float64), suffix rows kept."""
    outs = []
    for b, (p, s) in enumerate(seqs):
        q = torch.from_numpy(bf16_to_f64(case["full_q"][b])).permute(1, 0, 2)   # [Hq][n][d]
        k = torch.from_numpy(bf16_to_f64(case["full_k"][b])).permute(1, 0, 2)   # [Hkv][n][d]
        v = torch.from_numpy(bf16_to_f64(case["full_v"][b])).permute(1, 0, 2)
        o = torch.nn.functional.scaled_dot_product_attention(
            q.unsqueeze(0), k.unsqueeze(0), v.unsqueeze(0), is_causal=True,
            scale=1.0 / np.sqrt(d), enable_gqa=True)[0]                       # [Hq][n][d]
        outs.append(o.permute(1, 0, 2)[p:].numpy())
    return np.concatenate(outs)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("G", [1, 4, 8])
def test_matches_full_prefill_library(d, G):
    rng = np.random.Generator(np.random.PCG64(100 + d + G))
    Hkv = 2
    for p in [0, 1, 15, 16, 17, 256]:
        for s in [1, 2, 63, 64]:
            seqs = [(p, s)]
            case = _build_case(rng, seqs, Hkv, G, d)
            got = oattn.attention(case["q"], case["pool_k"], case["pool_v"], case["bt"],
                                  case["prefix_lens"], case["cu"], Hkv, BS)
            want = _sdpa_full_prefill_rows(case, seqs, G, d)
            np.testing.assert_allclose(got, want, rtol=0, atol=1e-12, err_msg=f"p={p} s={s}")


def test_ragged_batch_matches_library():
    rng = np.random.Generator(np.random.PCG64(7))
    seqs = [(0, 5), (33, 40), (256, 1), (17, 64), (48, 16)]
    d, G, Hkv = 64, 4, 2
    case = _build_case(rng, seqs, Hkv, G, d)
    got = oattn.attention(case["q"], case["pool_k"], case["pool_v"], case["bt"],
                          case["prefix_lens"], case["cu"], Hkv, BS)
    want = _sdpa_full_prefill_rows(case, seqs, G, d)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_value_identity_basis_gives_softmax_weights():
    """With V[j] = e_j the output row is the softmax weight vector itself."""
    rng = np.random.Generator(np.random.PCG64(8))
    d, Hkv, G, p, s = 64, 1, 2, 40, 20          # p + s = 60 <= d keys
    Hq = Hkv * G
    n = p + s
    q = synth.normal_bf16(rng, (n, Hq, d))
    k = synth.normal_bf16(rng, (n, Hkv, d))
    one = synth.f32_to_bf16_bits(np.ones(1, np.float32))[0]
    v = np.zeros((n, Hkv, d), np.uint16)
    for j in range(n):
        v[j, :, j] = one
    bt = random_tables(rng, [n], BS, 8)
    pool_k = np.zeros((8, Hkv, BS * d), np.uint16)
    pool_v = np.zeros((8, Hkv, BS * d), np.uint16)
    scatter_sequence(pool_k, pool_v, bt[0], k, v, BS)
    got = oattn.attention(q[p:], pool_k, pool_v, bt, np.array([p], np.int32),
                          np.array([0, s], np.int32), Hkv, BS)
    qf, kf = bf16_to_f64(q), bf16_to_f64(k)
    for i in range(s):
        for h in range(Hq):
            nk = p + i + 1
            scores = (kf[:nk, h // G, :] @ qf[p + i, h, :]) / np.sqrt(d)
            w = softmax(scores)
            np.testing.assert_allclose(got[i, h, :nk], w, rtol=0, atol=1e-14)
            assert np.all(got[i, h, nk:] == 0.0)
            assert abs(got[i, h].sum() - 1.0) <= 1e-12


def _single(rng, p, s, d, Hkv, G, k=None, v=None):
    n = p + s
    Hq = Hkv * G
    q = synth.normal_bf16(rng, (n, Hq, d))
    k = synth.normal_bf16(rng, (n, Hkv, d)) if k is None else k
    v = synth.normal_bf16(rng, (n, Hkv, d)) if v is None else v
    nb = ceil_div(n, BS) + 2
    bt = random_tables(rng, [n], BS, nb)
    pool_k = synth.normal_bf16(rng, (nb, Hkv, BS * d))
    pool_v = synth.normal_bf16(rng, (nb, Hkv, BS * d))
    scatter_sequence(pool_k, pool_v, bt[0], k, v, BS)
    out = oattn.attention(q[p:], pool_k, pool_v, bt, np.array([p], np.int32),
                          np.array([0, s], np.int32), Hkv, BS)
    return q, k, v, out


def test_constant_values_give_that_constant():
    rng = np.random.Generator(np.random.PCG64(9))
    p, s, d, Hkv, G = 37, 29, 128, 2, 4
    c = synth.f32_to_bf16_bits(rng.standard_normal((1, Hkv, d), dtype=np.float32))
    v = np.repeat(c, p + s, axis=0)
    _, _, _, out = _single(rng, p, s, d, Hkv, G, v=v)
    want = bf16_to_f64(c)[0]
    for h in range(Hkv * G):
        np.testing.assert_allclose(out[:, h, :], np.broadcast_to(want[h // G], (s, d)),
                                   rtol=0, atol=1e-14)


def test_equal_keys_give_prefix_mean_of_values():
    rng = np.random.Generator(np.random.PCG64(10))
    p, s, d, Hkv, G = 50, 14, 64, 2, 2
    k1 = synth.normal_bf16(rng, (1, Hkv, d))
    k = np.repeat(k1, p + s, axis=0)
    _, _, v, out = _single(rng, p, s, d, Hkv, G, k=k)
    vf = bf16_to_f64(v)
    for i in range(s):
        for h in range(Hkv * G):
            want = vf[:p + i + 1, h // G, :].mean(axis=0)
            np.testing.assert_allclose(out[i, h], want, rtol=0, atol=1e-12)


def test_first_causal_row_is_first_value():
    rng = np.random.Generator(np.random.PCG64(11))
    d, Hkv, G = 64, 2, 4
    _, _, v, out = _single(rng, 0, 9, d, Hkv, G)
    vf = bf16_to_f64(v)
    for h in range(Hkv * G):
        assert np.array_equal(out[0, h], vf[0, h // G])


def test_dominant_logit_selects_its_value():
    rng = np.random.Generator(np.random.PCG64(12))
    p, s, d, Hkv, G = 64, 8, 64, 1, 1
    n = p + s
    k = np.zeros((n, Hkv, d), np.uint16)
    big = synth.f32_to_bf16_bits(np.array([16.0], np.float32))[0]
    jstar = 23
    k[jstar, 0, 5] = big
    q = np.zeros((n, Hkv * G, d), np.uint16)
    q[:, 0, 5] = big
    v = synth.normal_bf16(rng, (n, Hkv, d))
    nb = ceil_div(n, BS)
    bt = random_tables(rng, [n], BS, nb)
    pool_k = np.zeros((nb, Hkv, BS * d), np.uint16)
    pool_v = np.zeros((nb, Hkv, BS * d), np.uint16)
    scatter_sequence(pool_k, pool_v, bt[0], k, v, BS)
    out = oattn.attention(q[p:], pool_k, pool_v, bt, np.array([p], np.int32),
                          np.array([0, s], np.int32), Hkv, BS)
    # score of jstar is 256/8 = 32 above every other score: weights ~ e^-32
    np.testing.assert_allclose(out[:, 0, :], np.broadcast_to(bf16_to_f64(v[jstar, 0]), (s, d)),
                               rtol=0, atol=1e-11)


def test_block_permutation_invariance_exact():
    rng = np.random.Generator(np.random.PCG64(13))
    p, s, d, Hkv, G = 70, 30, 64, 2, 4
    n = p + s
    q = synth.normal_bf16(rng, (n, Hkv * G, d))
    k = synth.normal_bf16(rng, (n, Hkv, d))
    v = synth.normal_bf16(rng, (n, Hkv, d))
    outs = []
    for _ in range(3):
        nb = 16
        bt = random_tables(rng, [n], BS, nb)
        pool_k = synth.normal_bf16(rng, (nb, Hkv, BS * d))
        pool_v = synth.normal_bf16(rng, (nb, Hkv, BS * d))
        scatter_sequence(pool_k, pool_v, bt[0], k, v, BS)
        outs.append(oattn.attention(q[p:], pool_k, pool_v, bt, np.array([p], np.int32),
                                    np.array([0, s], np.int32), Hkv, BS))
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_reuse_rows_equal_full_prefill_rows_exact():
    """Suffix rows of a reused-prefix call equal the same rows of a call that
    computes every token (p = 0), bit for bit in the oracle."""
    rng = np.random.Generator(np.random.PCG64(14))
    p, s, d, Hkv, G = 48, 16, 64, 2, 2
    n = p + s
    q = synth.normal_bf16(rng, (n, Hkv * G, d))
    k = synth.normal_bf16(rng, (n, Hkv, d))
    v = synth.normal_bf16(rng, (n, Hkv, d))
    bt = random_tables(rng, [n], BS, 8)
    pool_k = np.zeros((8, Hkv, BS * d), np.uint16)
    pool_v = np.zeros((8, Hkv, BS * d), np.uint16)
    scatter_sequence(pool_k, pool_v, bt[0], k, v, BS)
    reuse = oattn.attention(q[p:], pool_k, pool_v, bt, np.array([p], np.int32),
                            np.array([0, s], np.int32), Hkv, BS)
    full = oattn.attention(q, pool_k, pool_v, bt, np.array([0], np.int32),
                           np.array([0, n], np.int32), Hkv, BS)
    assert np.array_equal(reuse, full[p:])


def test_row_list_matches_full_output():
    rng = np.random.Generator(np.random.PCG64(15))
    seqs = [(16, 20), (0, 7), (33, 12)]
    d, G, Hkv = 64, 2, 2
    case = _build_case(rng, seqs, Hkv, G, d)
    full = oattn.attention(case["q"], case["pool_k"], case["pool_v"], case["bt"],
                           case["prefix_lens"], case["cu"], Hkv, BS)
    rows = np.array([[0, 0], [19, 3], [20, 1], [26, 2], [38, 0]], np.int32)
    part = oattn.attention(case["q"], case["pool_k"], case["pool_v"], case["bt"],
                           case["prefix_lens"], case["cu"], Hkv, BS, rows=rows)
    for k_, (t, h) in enumerate(rows):
        assert np.array_equal(part[k_], full[t, h])


def test_rejects_out_of_range_block():
    rng = np.random.Generator(np.random.PCG64(16))
    p, s, d, Hkv = 16, 4, 64, 1
    q = synth.normal_bf16(rng, (s, Hkv, d))
    pool = synth.normal_bf16(rng, (2, Hkv, BS * d))
    bt = np.array([[0, 5]], np.int32)
    with pytest.raises(ValueError):
        oattn.attention(q, pool, pool, bt, np.array([p], np.int32), np.array([0, s], np.int32),
                        Hkv, BS)
