"""The build refuses kernels that use scratch memory (register spills, private
arrays): the compiler's resource remarks are read for every kernel."""
import os
import subprocess

import pytest

from paper_1907_03739_amd import build

REMARKS = """\
a.hip:10:1: remark: Function Name: _Z4goodPf [-Rpass-analysis=kernel-resource-usage]
a.hip:10:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass-analysis=kernel-resource-usage]
a.hip:20:1: remark: Function Name: _Z5spillPf [-Rpass-analysis=kernel-resource-usage]
a.hip:20:1: remark:     ScratchSize [bytes/lane]: 28 [-Rpass-analysis=kernel-resource-usage]
"""


def test_scratch_remarks_are_parsed():
    assert build.scratch_kernels(REMARKS) == [("_Z5spillPf", 28)]
    assert build.scratch_kernels(REMARKS.replace(": 28 ", ": 0 ")) == []


# a private array indexed by a run-time value lives in scratch
SPILLING_KERNEL = """
#include <hip/hip_runtime.h>
__global__ void private_array(float* out, int k) {
    float a[64];
    for (int i = 0; i < 64; i++) a[i] = out[i * blockDim.x + threadIdx.x];
    out[threadIdx.x] = a[(k + threadIdx.x) & 63];
}
"""


@pytest.mark.skipif(not os.path.exists(build.HIPCC), reason="hipcc not installed")
def test_compile_rejects_a_kernel_with_scratch(tmp_path, monkeypatch):
    src = tmp_path / "private_array.hip"
    src.write_text(SPILLING_KERNEL)
    monkeypatch.setattr(build, "BUILD", str(tmp_path))
    with pytest.raises(RuntimeError, match="scratch"):
        build._compile(str(src), verbose=False)


@pytest.mark.skipif(not os.path.exists(build.HIPCC), reason="hipcc not installed")
def test_library_kernels_use_no_scratch():
    # the committed kernels compile with the check on (one file, the largest)
    src = os.path.join(build.CSRC, "conv3d.hip")
    r = subprocess.run([build.HIPCC, *build.FLAGS, build.RESOURCE_REMARKS, "-c", src, "-o",
                        os.devnull], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    remarks = r.stdout + r.stderr
    assert "ScratchSize" in remarks
    assert build.scratch_kernels(remarks) == []
