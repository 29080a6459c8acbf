"""The build's guard against kernels that use private (scratch) memory: it reads the
compiler's per-kernel resource report and names every kernel with a non-zero scratch size."""
import pytest

from paper_2405_00263_amd.build import _check_no_scratch

REPORT = """\
gemm.hip:97:1: remark: Function Name: _ZN6clover11gemm_kernelA [-Rpass-analysis=kernel-resource-usage]
gemm.hip:97:1: remark:     VGPRs: 114 [-Rpass-analysis=kernel-resource-usage]
gemm.hip:97:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
gemm.hip:97:1: remark: Function Name: _ZN6clover11gemm_kernelB [-Rpass-analysis=kernel-resource-usage]
gemm.hip:97:1: remark:     ScratchSize [bytes/lane]: 272 [-Rpass-analysis=kernel-resource-usage]
"""


def test_scratch_guard_names_the_offending_kernel():
    with pytest.raises(RuntimeError) as e:
        _check_no_scratch(REPORT, "gemm.hip")
    assert "gemm_kernelB: 272 bytes/lane" in str(e.value)
    assert "gemm_kernelA" not in str(e.value)


def test_scratch_guard_passes_a_clean_report():
    _check_no_scratch(REPORT.replace("272", "0"), "gemm.hip")
    _check_no_scratch("", "api.cpp")
