"""The build's guard against scratch memory in the hot kernels (parses the
compiler's resource-usage remarks)."""
from paper_2608_07974_amd import build

REMARKS = """x.hip:1:1: remark: Function Name: _ZN2zl15gemm_dma_kernelILi256E [-Rpass-analysis=kernel-resource-usage]
x.hip:1:1: remark:     VGPRs: 214 [-Rpass-analysis=kernel-resource-usage]
x.hip:1:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
x.hip:2:1: remark: Function Name: _ZN2zl15gemm_dma_kernelILi128E [-Rpass-analysis=kernel-resource-usage]
x.hip:2:1: remark:     ScratchSize [bytes/lane]: 768 [-Rpass-analysis=kernel-resource-usage]
x.hip:3:1: remark: Function Name: _ZN2zl16gemm_simt_kernelILb1E [-Rpass-analysis=kernel-resource-usage]
x.hip:3:1: remark:     ScratchSize [bytes/lane]: 52 [-Rpass-analysis=kernel-resource-usage]
"""


def test_scratch_users_reports_only_matching_kernels_with_scratch():
    assert build._scratch_users(REMARKS, "gemm_dma_kernel") == [("_ZN2zl15gemm_dma_kernelILi128E", 768)]
    assert build._scratch_users(REMARKS, "attn_") == []
