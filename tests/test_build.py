"""CPU checks of the build's guard on kernel resources (no GPU, no compile)."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from paper_2404_08573_amd import build as B  # noqa: E402

REPORT = """\
ff_kernels.hip:557:1: remark: Function Name: _ZN3ffk5k_fwdILb1EEEvv [-Rpass-analysis=kernel-resource-usage]
ff_kernels.hip:557:1: remark:     VGPRs: 74 [-Rpass-analysis=kernel-resource-usage]
ff_kernels.hip:557:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
ff_kernels.hip:601:1: remark: Function Name: _ZN3ffk6k_fwd4ILi256EEEvv [-Rpass-analysis=kernel-resource-usage]
ff_kernels.hip:601:1: remark:     ScratchSize [bytes/lane]: 80 [-Rpass-analysis=kernel-resource-usage]
ff_kernels.hip:601:1: remark:     Occupancy [waves/SIMD]: 1 [-Rpass-analysis=kernel-resource-usage]
"""


def test_scratch_users_lists_only_kernels_with_scratch():
    assert B.scratch_users(REPORT) == [("_ZN3ffk6k_fwd4ILi256EEEvv", 80)]
    assert B.scratch_users(REPORT.replace("80 [", "0 [")) == []


def test_build_keeps_arrays_out_of_lds_and_reports_kernel_resources():
    assert "-disable-promote-alloca-to-lds" in B.FLAGS
    assert B.KERNELS in B.SOURCES
