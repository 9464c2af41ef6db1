"""The build's guard against kernels that the compiler moved to scratch memory."""
from paper_2608_21157_amd import build

REMARKS = """\
k.hip:10:1: remark: Function Name: _Z4fastPf [-Rpass-analysis=kernel-resource-usage]
k.hip:10:1: remark:     VGPRs: 127 [-Rpass-analysis=kernel-resource-usage]
k.hip:10:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
k.hip:20:1: remark: Function Name: _Z4slowPf [-Rpass-analysis=kernel-resource-usage]
k.hip:20:1: remark:     VGPRs: 168 [-Rpass-analysis=kernel-resource-usage]
k.hip:20:1: remark:     ScratchSize [bytes/lane]: 880 [-Rpass-analysis=kernel-resource-usage]
"""


def test_scratch_kernels_names_only_the_kernels_with_scratch():
    assert build.scratch_kernels(REMARKS) == [("_Z4slowPf", 880)]
    assert build.scratch_kernels(REMARKS.replace("880", "0")) == []
    assert build.scratch_kernels("") == []
