"""The attention pins must catch plausible mistakes in the oracle.

Each case copies the oracle's C source, plants one mistake by text
substitution, builds the copy in a temporary directory and runs the pin
battery (full-prefill library comparison on a ragged GQA batch, the
identity-basis softmax check, and the closed forms) against it. Every planted
mistake must fail at least one pin; the unmodified source must pass them all.
Only the CPU is involved.
"""
import os
import subprocess
import tempfile

import numpy as np
import pytest
import torch
from scipy.special import softmax

from oracle import attention as oattn
from oracle import build as obuild
from paper_2603_23049_amd import synth
from pagedkv import bf16_to_f64, random_tables, scatter_sequence, ceil_div

BS = 16

MUTANTS = {
    "gqa_modulo_mapping": ("const int g = h / G;", "const int g = h % Hkv;"),
    "causal_excludes_diagonal": ("const int64_t nkeys = pos + 1;", "const int64_t nkeys = pos;"),
    "causal_one_too_many": ("const int64_t nkeys = pos + 1;", "const int64_t nkeys = pos + 2;"),
    "position_ignores_prefix": ("const int64_t pos = (int64_t)prefix_lens[b] + i;",
                                "const int64_t pos = i;"),
    "missing_scale": ("score[j] = sm_scale * dot;", "score[j] = dot;"),
    "missing_normaliser": ("out_row[x] = acc[x] / sum;", "out_row[x] = acc[x];"),
    "v_read_in_k_layout": ("acc[x] += w * bf16_to_f64(vbase[(int64_t)x * bs]);",
                           "acc[x] += w * bf16_to_f64(pool_v[((blk * Hkv + g) * bs + o) * d + x]);"),
    "slot_from_wrong_index": ("const int64_t blk = bt[j / bs];\n        const int64_t o = j % bs;\n        if",
                              "const int64_t blk = bt[j / bs];\n        const int64_t o = (j + 1) % bs;\n        if"),
    "token_row_of_wrong_sequence": ("const int32_t i = t - cu_suffix[b];",
                                    "const int32_t i = t - cu_suffix[b] + (b > 0);"),
}


def _build_variant(src_text, tmpdir, name):
    c = os.path.join(tmpdir, f"{name}.c")
    so = os.path.join(tmpdir, f"{name}.so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11", c, "-o", so, "-lm"],
                   check=True, capture_output=True)
    return oattn.open_library(so)


def _pin_battery(lib):
    """Returns a list of failed pin names (empty if every pin holds)."""
    failed = []
    rng = np.random.Generator(np.random.PCG64(77))
    # 1. ragged GQA batch vs torch SDPA on the full sequences
    seqs = [(0, 9), (17, 23), (40, 8)]
    d, G, Hkv = 64, 4, 2
    Hq = G * Hkv
    lens = [p + s for p, s in seqs]
    nb = sum(ceil_div(n, BS) for n in lens) + 2
    bt = random_tables(rng, lens, BS, nb)
    pool_k = synth.normal_bf16(rng, (nb, Hkv, BS * d))
    pool_v = synth.normal_bf16(rng, (nb, Hkv, BS * d))
    qs, want = [], []
    for b, (p, s) in enumerate(seqs):
        n = p + s
        q = synth.normal_bf16(rng, (n, Hq, d))
        k = synth.normal_bf16(rng, (n, Hkv, d))
        v = synth.normal_bf16(rng, (n, Hkv, d))
        scatter_sequence(pool_k, pool_v, bt[b], k, v, BS)
        qs.append(q[p:])
        o = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(bf16_to_f64(q)).permute(1, 0, 2)[None],
            torch.from_numpy(bf16_to_f64(k)).permute(1, 0, 2)[None],
            torch.from_numpy(bf16_to_f64(v)).permute(1, 0, 2)[None],
            is_causal=True, scale=1.0 / np.sqrt(d), enable_gqa=True)[0]
        want.append(o.permute(1, 0, 2)[p:].numpy())
    try:
        got = oattn.attention(np.concatenate(qs), pool_k, pool_v, bt,
                              np.array([p for p, _ in seqs], np.int32),
                              np.concatenate([[0], np.cumsum([s for _, s in seqs])]).astype(np.int32),
                              Hkv, BS, lib=lib)
        if not np.allclose(got, np.concatenate(want), rtol=0, atol=1e-12):
            failed.append("sdpa")
    except ValueError:
        failed.append("sdpa(error)")
    # 2. identity-basis values give the softmax weights
    d, Hkv, G, p, s = 64, 1, 1, 30, 20
    n = p + s
    q = synth.normal_bf16(rng, (n, 1, d))
    k = synth.normal_bf16(rng, (n, 1, d))
    one = synth.f32_to_bf16_bits(np.ones(1, np.float32))[0]
    v = np.zeros((n, 1, d), np.uint16)
    for j in range(n):
        v[j, 0, j] = one
    bt = random_tables(rng, [n], BS, 6)
    pk = np.zeros((6, 1, BS * d), np.uint16)
    pv = np.zeros((6, 1, BS * d), np.uint16)
    scatter_sequence(pk, pv, bt[0], k, v, BS)
    try:
        got = oattn.attention(q[p:], pk, pv, bt, np.array([p], np.int32),
                              np.array([0, s], np.int32), 1, BS, lib=lib)
        qf, kf = bf16_to_f64(q), bf16_to_f64(k)
        ok = True
        for i in range(s):
            nk = p + i + 1
            w = softmax(kf[:nk, 0] @ qf[p + i, 0] / np.sqrt(d))
            ok &= np.allclose(got[i, 0, :nk], w, rtol=0, atol=1e-14) and np.all(got[i, 0, nk:] == 0)
        if not ok:
            failed.append("softmax_basis")
    except ValueError:
        failed.append("softmax_basis(error)")
    return failed


def test_unmodified_oracle_passes_battery():
    assert _pin_battery(oattn.open_library(obuild.ensure_built())) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    src = open(obuild.SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    with tempfile.TemporaryDirectory() as td:
        lib = _build_variant(src.replace(old, new), td, name)
        assert _pin_battery(lib), f"planted mistake {name} passed every pin"
