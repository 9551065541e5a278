"""The build's guard against kernels that use scratch memory (host logic only)."""
import pytest

from paper_2608_09160_amd import build as B

REMARKS = """\
a.hip:1:1: remark: Function Name: k_spills [-Rpass-analysis=kernel-resource-usage]
a.hip:1:1: remark:     VGPRs: 256 [-Rpass-analysis=kernel-resource-usage]
a.hip:1:1: remark:     ScratchSize [bytes/lane]: 192 [-Rpass-analysis=kernel-resource-usage]
a.hip:1:1: remark:     VGPRs Spill: 40 [-Rpass-analysis=kernel-resource-usage]
a.hip:1:1: remark:     SGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]
   12 | source excerpt
      | ^
a.hip:9:1: remark: Function Name: k_clean [-Rpass-analysis=kernel-resource-usage]
a.hip:9:1: remark:     VGPRs: 96 [-Rpass-analysis=kernel-resource-usage]
a.hip:9:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
a.hip:9:1: remark:     VGPRs Spill: 0 [-Rpass-analysis=kernel-resource-usage]
a.hip:9:1: remark:     SGPRs Spill: 10 [-Rpass-analysis=kernel-resource-usage]
a.hip:9:1: remark:     Occupancy [waves/SIMD]: 5 [-Rpass-analysis=kernel-resource-usage]
"""


def test_resource_remarks_are_parsed_per_kernel():
    res = B.kernel_resources(REMARKS)
    assert set(res) == {"k_spills", "k_clean"}
    assert res["k_spills"]["ScratchSize [bytes/lane]"] == "192"
    assert res["k_clean"]["Occupancy [waves/SIMD]"] == "5"
    assert res["k_clean"]["VGPRs"] == "96"


def test_scratch_or_vector_spills_fail_the_build():
    res = B.kernel_resources(REMARKS)
    with pytest.raises(RuntimeError, match="k_spills: scratch 192"):
        B.check_resources(res)
    # scalar spills go to vector-register lanes, not memory: allowed
    B.check_resources({"k_clean": res["k_clean"]})
