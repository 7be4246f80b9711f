"""Host logic of the build's register-budget check: an attention workgroup (two
waves per SIMD) must leave one copy-kernel wave's registers free on every SIMD, so
the next layer's KV keeps streaming while a long attention occupies every CU."""
import pytest

from paper_2603_23049_amd import build


REMARKS = """x.hip:1:1: remark: Function Name: _ZN3pcr12_GLOBAL__N_119prefill_attn_kernelILi128EEEv [-Rpass-analysis=kernel-resource-usage]
x.hip:1:1: remark:     VGPRs: 230 [-Rpass-analysis=kernel-resource-usage]
x.hip:1:1: remark:     AGPRs: 0 [-Rpass-analysis=kernel-resource-usage]
y.hip:2:1: remark: Function Name: _ZN3pcr12_GLOBAL__N_118copy_blocks_kernelILi0EEEv [-Rpass-analysis=kernel-resource-usage]
y.hip:2:1: remark:     VGPRs: 40 [-Rpass-analysis=kernel-resource-usage]
y.hip:2:1: remark:     AGPRs: 2 [-Rpass-analysis=kernel-resource-usage]
"""


def test_remarks_parse_vgprs_plus_agprs():
    u = build._vgprs(REMARKS)
    assert u == {"_ZN3pcr12_GLOBAL__N_119prefill_attn_kernelILi128EEEv": 230,
                 "_ZN3pcr12_GLOBAL__N_118copy_blocks_kernelILi0EEEv": 42}


def test_budget_accepts_a_copy_wave_beside_two_attention_waves():
    build.check_register_budget({"prefill_attn_kernel<128>": 232, "copy_blocks_kernel<0>": 42})  # 464 + 48 = 512


@pytest.mark.parametrize("attn,copy", [(254, 42), (233, 42), (232, 49)])
def test_budget_rejects_when_the_copy_wave_cannot_fit(attn, copy):
    with pytest.raises(RuntimeError, match="register budget"):
        build.check_register_budget({"prefill_attn_kernel<128>": attn, "copy_blocks_kernel<0>": copy})


def test_budget_requires_both_kernels():
    with pytest.raises(RuntimeError, match="not found"):
        build.check_register_budget({"prefill_attn_kernel<128>": 200})
