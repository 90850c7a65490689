"""The build's guard against kernels that use scratch memory (no GPU)."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2402_15106_amd import build  # noqa: E402

REMARKS = """\
a.hip:1:1: remark: Function Name: k_one [-Rpass-analysis=kernel-resource-usage]
a.hip:1:1: remark:     VGPRs: 64 [-Rpass-analysis=kernel-resource-usage]
a.hip:1:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
a.hip:9:1: remark: Function Name: k_two [-Rpass-analysis=kernel-resource-usage]
a.hip:9:1: remark:     ScratchSize [bytes/lane]: 240 [-Rpass-analysis=kernel-resource-usage]
"""


def test_scratch_kernels_names_only_the_spilling_kernel():
    assert build.scratch_kernels(REMARKS) == ["k_two (240 bytes/lane)"]
    assert build.scratch_kernels("") == []
