"""The build's guard against spilling forward kernels reads the compiler's
resource remarks (CPU only: parses text, compiles nothing)."""
from paper_2512_13921_amd import build

REMARKS = """\
swr_kernels.hip:80:1: remark: Function Name: _ZN3swr12_GLOBAL__N_114swr_fwd_kernelINS0_6IoBf16ELi8ELi4ELi1ELb0ELi4EEEvNS_6ParamsE [-Rpass-analysis=kernel-resource-usage]
swr_kernels.hip:80:1: remark:     VGPRs: 168 [-Rpass-analysis=kernel-resource-usage]
swr_kernels.hip:80:1: remark:     ScratchSize [bytes/lane]: 20 [-Rpass-analysis=kernel-resource-usage]
swr_kernels.hip:80:1: remark: Function Name: _ZN3swr12_GLOBAL__N_114swr_fwd_kernelINS0_6IoBf16ELi8ELi2ELi2ELb0ELi0EEEvNS_6ParamsE [-Rpass-analysis=kernel-resource-usage]
swr_kernels.hip:80:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
swr_kernels.hip:380:1: remark: Function Name: _ZN3swr12_GLOBAL__N_114swr_bwd_kernelINS0_5IoF32ELi8ELi8ELi1ELb1ELi0EEEvNS_6ParamsE [-Rpass-analysis=kernel-resource-usage]
swr_kernels.hip:380:1: remark:     ScratchSize [bytes/lane]: 16 [-Rpass-analysis=kernel-resource-usage]
swr_chain.hip:80:1: remark: Function Name: _ZN3swr12_GLOBAL__N_120swr_fwd_chain_kernelINS0_6IoBf16ELi8ELb0EEEvNS_6ParamsE [-Rpass-analysis=kernel-resource-usage]
swr_chain.hip:80:1: remark:     ScratchSize [bytes/lane]: 56 [-Rpass-analysis=kernel-resource-usage]
"""


def test_spilling_forward_kernels_are_reported():
    bad = build.spilled_kernels(REMARKS)
    assert len(bad) == 2
    assert "swr_fwd_kernel" in bad[0] and "20 bytes/lane" in bad[0]
    assert "swr_fwd_chain_kernel" in bad[1] and "56 bytes/lane" in bad[1]


def test_other_kernels_may_spill():
    # the float32 128-channel backward spills by design; only NO_SPILL kernels are checked
    without_bwd = "".join(ln for ln in REMARKS.splitlines(keepends=True) if not ln.startswith("swr_kernels.hip:380"))
    assert build.spilled_kernels(without_bwd) == build.spilled_kernels(REMARKS)


def test_remark_lines_are_not_shown_as_messages():
    import subprocess
    res = subprocess.CompletedProcess([], 0, REMARKS + "  80 | __global__ void k()\n      | ^\nreal warning: x\n", "")
    assert build._messages(res) == ["real warning: x"]


def test_only_the_guarded_sources_are_compiled_with_remarks():
    for src in build.SOURCES:
        guarded = src.endswith(("swr_kernels.hip", "swr_chain.hip"))
        assert (build.RESOURCE_REMARKS in build.compile_command(src, "k.o")) == guarded, src
