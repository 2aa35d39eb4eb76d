"""The build's kernel resource guard (host only): the compiler's
kernel-resource-usage remarks are parsed per kernel, and any spill, any
scratch, or an attention/copy kernel above its VGPR budget fails the build."""
from paper_2607_01817_amd import build

R = "[-Rpass-analysis=kernel-resource-usage]"


def _remarks(name, vgprs, sgpr_spill=0, vgpr_spill=0, scratch=0):
    pre = "x.hip:1:1: remark: "
    return "\n".join([
        f"{pre}Function Name: {name} {R}",
        "    1 | int x;",
        "      | ^",
        f"{pre}    TotalSGPRs: 90 {R}",
        f"{pre}    VGPRs: {vgprs} {R}",
        f"{pre}    AGPRs: 0 {R}",
        f"{pre}    ScratchSize [bytes/lane]: {scratch} {R}",
        f"{pre}    Dynamic Stack: False {R}",
        f"{pre}    SGPRs Spill: {sgpr_spill} {R}",
        f"{pre}    VGPRs Spill: {vgpr_spill} {R}",
        f"{pre}    LDS Size [bytes/block]: 163840 {R}",
    ])


def test_parse_resource_remarks():
    text = _remarks("_Z20attention_dma_kernelv", 248) + "\nunrelated line\n" + \
        _remarks("_Z11pack_kernelv", 13)
    res = build.parse_resource_remarks(text)
    assert res["_Z20attention_dma_kernelv"]["VGPRs"] == 248
    assert res["_Z20attention_dma_kernelv"]["ScratchSize"] == 0
    assert res["_Z20attention_dma_kernelv"]["LDS Size"] == 163840
    assert res["_Z11pack_kernelv"]["VGPRs"] == 13
    assert build.resource_problems(res) == []


def test_resource_problems_flag_spills_scratch_and_budgets():
    cases = [
        (_remarks("_Z20attention_dma_kernelv", 255, sgpr_spill=28), ["SGPRs Spill 28", "255 VGPRs > 248"]),
        (_remarks("_Z11linear_kernelv", 200, vgpr_spill=4), ["VGPRs Spill 4"]),
        (_remarks("_Z11dq_kernelv", 256, scratch=16), ["ScratchSize 16"]),
        (_remarks("_Z13unpack_kernelv", 24), ["24 VGPRs > 16"]),
        (_remarks("_Z11dq_kernelv", 256), []),   # no budget for other kernels
    ]
    for text, want in cases:
        bad = build.resource_problems(build.parse_resource_remarks(text))
        assert len(bad) == len(want), bad
        for w, b in zip(want, bad):
            assert w in b, (w, b)
