"""Host checks of the build driver (no GPU): the scratch report parser that
keeps spills out of the kernels."""
import os

from paper_2609_34380_amd.csrc import build


REPORT = """\
a.hip:10:0: remark: Function Name: _Zk1 [-Rpass-analysis=kernel-resource-usage]
a.hip:10:0: remark:     VGPRs: 90 [-Rpass-analysis=kernel-resource-usage]
a.hip:10:0: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
a.hip:20:0: remark: Function Name: _Zk2 [-Rpass-analysis=kernel-resource-usage]
a.hip:20:0: remark:     ScratchSize [bytes/lane]: 44 [-Rpass-analysis=kernel-resource-usage]
"""


def test_scratch_users_names_only_spilling_kernels():
    assert build._scratch_users(REPORT) == [("_Zk2", 44)]
    assert build._scratch_users("") == []


def test_every_kernel_source_is_checked():
    every = build.SOURCES + build.PROBE_SOURCES
    here = os.path.dirname(build.__file__)
    kernels = {s for s in every if s.endswith(".hip") and
               "__global__" in open(os.path.join(here, s)).read()}
    assert {"dps_gemm.hip", "dps_probe.hip"} <= kernels
    assert kernels <= build.NO_SCRATCH <= set(every)
