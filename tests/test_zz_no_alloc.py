"""pvconv_conv3d_noalloc, whose repacked weights live in the library's static
device array, gives exactly what pvconv_conv3d gives with a caller's workspace
(the same kernels run on the same inputs), call after call on one GPU.
"""
import numpy as np
import pytest
import torch

import synth
from paper_1907_03739_amd import binding as pv
from _helpers import bf16_round, dev, dev_bn

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu_case(request):
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    print(f"\n[gpu case] {request.node.nodeid}", flush=True)
    yield
    torch.cuda.synchronize()


def _inputs(seed, B, R, Cin, Cout):
    rng = np.random.default_rng(seed)
    x = rng.normal(size=(B, R ** 3, Cin))
    x *= rng.random(size=(B, R ** 3, 1)) < 0.3
    w = synth.kaiming_normal(rng, (Cout, 3, 3, 3, Cin), 27 * Cin, bf16=True)
    bn = synth.draw_bn(rng, Cout)
    return (dev(bf16_round(x), torch.bfloat16), dev(w, torch.bfloat16), dev_bn(bn))


def _both(seed, B, R, Cin, Cout, odt):
    x, w, bn = _inputs(seed, B, R, Cin, Cout)
    ref = pv.pvconv_conv3d(x, w, R, bn=bn, out_dtype=odt)
    # a dirty output buffer: every element must be written
    out = torch.full((B, R ** 3, Cout), float("nan"), dtype=odt, device="cuda")
    pv.pvconv_conv3d_noalloc(x, w, R, out, bn=bn)
    torch.cuda.synchronize()
    return ref, out


# consecutive calls on one GPU, each smaller than the one before, so stale
# packed weights of a larger call lie beyond what the next call packs
SEQUENCE = [
    # seed, B, R, Cin, Cout, out dtype
    (1, 1, 8, 256, 256, torch.bfloat16),   # 3.4 MiB of packed weights, near the limit
    (2, 2, 32, 64, 128, torch.bfloat16),   # part-segmentation conv 1 (batch reduced)
    (3, 1, 16, 32, 64, torch.float32),     # smaller still, fp32 output
    (4, 1, 13, 3, 32, torch.bfloat16),     # ragged R, 3 input channels
]


def test_noalloc_matches_workspace_entry_point_over_consecutive_calls():
    for case in SEQUENCE:
        ref, out = _both(*case)
        assert torch.equal(ref, out), f"noalloc differs from pvconv_conv3d for {case}"


def test_noalloc_on_a_side_stream_twice():
    side = torch.cuda.Stream()
    big, small = (5, 2, 32, 128, 128), (6, 1, 16, 64, 64)
    with torch.cuda.stream(side):
        for seed, B, R, Cin, Cout in (big, small):
            x, w, bn = _inputs(seed, B, R, Cin, Cout)
            ref = pv.pvconv_conv3d(x, w, R, bn=bn, out_dtype=torch.bfloat16)
            out = torch.empty((B, R ** 3, Cout), dtype=torch.bfloat16, device="cuda")
            pv.pvconv_conv3d_noalloc(x, w, R, out, bn=bn)
            side.synchronize()
            assert torch.equal(ref, out), (seed, B, R, Cin, Cout)


def test_noalloc_rejects_weights_beyond_its_array():
    x = torch.zeros((1, 8, 512), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((512, 3, 3, 3, 512), dtype=torch.bfloat16, device="cuda")
    out = torch.empty((1, 8, 512), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(pv.PVConvError):
        pv.pvconv_conv3d_noalloc(x, w, 2, out)
