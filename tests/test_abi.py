"""The C ABI library loads, exports every symbol include/pvconv.h declares,
and rejects invalid arguments on the host before anything is enqueued.

These run without a GPU: every call here fails validation (or has nothing to
do) before the library touches the HIP runtime.
"""
import ctypes
import os
import re
import subprocess

import pytest

from paper_1907_03739_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pvconv.h")
L = b._lib
OK, EINVAL, ENOTSUP, EWS = 0, 1, 2, 3
FAKE = ctypes.c_void_p(0x100000)    # never dereferenced: validation fails first
FAKE_ODD = ctypes.c_void_p(0x100001)
FAKE2 = ctypes.c_void_p(0x200000)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pvconv_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) == 32
    out = subprocess.run(["nm", "-D", "--defined-only", b.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (pvconv_\w+)", out))
    assert set(names) <= exported, set(names) - exported
    assert set(names) == set(b.EXPORTED)


def test_status_strings():
    for s in range(5):
        assert L.pvconv_status_string(s)
    assert L.pvconv_status_string(99) == b"unknown status"


def test_conv_workspace_query():
    # bf16: the packed weights, input channels padded to 16 and output
    # channels to 32; fp32 needs none
    assert L.pvconv_conv3d_workspace_size(128, 128, 1) == 128 * 27 * 128 * 2
    assert L.pvconv_conv3d_workspace_size(3, 64, 1) == 64 * 27 * 16 * 2
    assert L.pvconv_conv3d_workspace_size(8, 16, 1) == 32 * 27 * 16 * 2
    assert L.pvconv_conv3d_workspace_size(64, 40, 1) == 64 * 27 * 64 * 2
    assert L.pvconv_conv3d_workspace_size(16, 32, 0) == 0
    assert L.pvconv_conv3d_workspace_size(0, 32, 1) == 0


def test_workspace_queries():
    # room for the voxel ids and normalised coordinates the caller may omit
    assert L.pvconv_voxelize_workspace_size(16, 2048, 32) >= 16 * 2048 * (4 + 12)
    assert L.pvconv_voxelize_workspace_size(1, 65536, 64) >= 65536 * (4 + 12)
    assert L.pvconv_voxelize_workspace_size(-1, 10, 8) == 0
    assert L.pvconv_voxelize_workspace_size(1, 10, 0) == 0
    assert L.pvconv_voxelize_workspace_size(1, 10, 129) == 0
    # the devoxelisation backward's sort: keys and entries twice, the cell ranges
    assert L.pvconv_devoxelize_backward_workspace_size(16, 2048, 128, 32) >= \
        16 * 2048 * (16 + 128 * 4) + 16 * 32 ** 3 * 8
    assert L.pvconv_devoxelize_backward_workspace_size(-1, 10, 8, 8) == 0
    assert L.pvconv_devoxelize_backward_workspace_size(1, 10, 0, 8) == 0
    assert L.pvconv_devoxelize_backward_workspace_size(1, 10, 8, 129) == 0
    lay = _layer()
    need = L.pvconv_forward_workspace_size(16, 2048, ctypes.byref(lay))
    # at least: two bf16 grids of 128 channels + the fp32 devox buffer
    assert need >= 2 * 16 * 32 ** 3 * 128 * 2 + 16 * 2048 * 128 * 4
    lay.n_convs = 0
    assert L.pvconv_forward_workspace_size(16, 2048, ctypes.byref(lay)) == 0


def _vox(**kw):
    a = dict(coords=FAKE, feats=FAKE, feat_dt=0, feat_ld=0, B=2, N=100, C=8, R=8, grid=FAKE,
             grid_dt=1, counts=FAKE, vox_id=None, norm=None, ws=FAKE, wsb=1 << 30, s=None)
    a.update(kw)
    return L.pvconv_voxelize(a["coords"], a["feats"], a["feat_dt"], a["feat_ld"], a["B"], a["N"],
                             a["C"], a["R"], a["grid"], a["grid_dt"], a["counts"], a["vox_id"],
                             a["norm"], a["ws"], a["wsb"], a["s"])


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), EINVAL), (dict(N=-5), EINVAL), (dict(C=0), EINVAL), (dict(R=0), EINVAL),
    (dict(R=129), EINVAL), (dict(feat_dt=7), EINVAL), (dict(grid_dt=-1), EINVAL),
    (dict(feat_ld=4), EINVAL), (dict(grid=None), EINVAL), (dict(counts=None), EINVAL),
    (dict(coords=None), EINVAL), (dict(feats=None), EINVAL), (dict(coords=FAKE_ODD), EINVAL),
    (dict(grid=FAKE_ODD), EINVAL), (dict(ws=None), EWS), (dict(wsb=16), EWS),
    (dict(ws=ctypes.c_void_p(0x100010)), EWS), (dict(B=0), OK),
])
def test_voxelize_rejects(kw, status):
    assert _vox(**kw) == status


def _conv(**kw):
    a = dict(x=FAKE, B=1, R=8, Cin=16, Cout=64, w=FAKE, bias=None, bn=None, act=2, slope=0.1,
             dt=1, y=ctypes.c_void_p(0x200000), out_dt=1, ws=ctypes.c_void_p(0x400000),
             wsb=1 << 30, s=None)
    a.update(kw)
    return L.pvconv_conv3d(a["x"], a["B"], a["R"], a["Cin"], a["Cout"], a["w"], a["bias"],
                           a["bn"], a["act"], a["slope"], a["dt"], a["y"], a["out_dt"], a["ws"],
                           a["wsb"], a["s"])


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), EINVAL), (dict(R=0), EINVAL), (dict(R=200), EINVAL), (dict(Cin=0), EINVAL),
    (dict(Cout=2000), EINVAL), (dict(act=5), EINVAL), (dict(dt=3), EINVAL), (dict(x=None), EINVAL),
    (dict(w=None), EINVAL), (dict(y=None), EINVAL), (dict(x=FAKE_ODD), EINVAL),
    (dict(y=FAKE), EINVAL), (dict(B=0), OK),
    (dict(ws=None), EWS), (dict(wsb=100), EWS), (dict(ws=ctypes.c_void_p(0x400010)), EWS),
    # 48 output channels (two 32-channel tiles, the second half zeros): the
    # workspace is that of 64
    (dict(Cout=48, wsb=16 * 27 * 48 * 2), EWS),
])
def test_conv3d_rejects(kw, status):
    assert _conv(**kw) == status


def test_conv3d_rejects_overlapping_output():
    # x [1][512][16] bf16 spans 16 KiB from FAKE; y starting inside it overlaps
    assert _conv(y=ctypes.c_void_p(0x100000 + 4096)) == EINVAL
    assert _conv(y=ctypes.c_void_p(0x100000 - 512), out_dt=1, Cout=64) == EINVAL


def _conv_na(**kw):
    a = dict(x=FAKE, B=1, R=8, Cin=16, Cout=64, w=FAKE, bias=None, bn=None, act=2, slope=0.1,
             dt=1, y=ctypes.c_void_p(0x200000), out_dt=1, s=None)
    a.update(kw)
    return L.pvconv_conv3d_noalloc(a["x"], a["B"], a["R"], a["Cin"], a["Cout"], a["w"],
                                   a["bias"], a["bn"], a["act"], a["slope"], a["dt"], a["y"],
                                   a["out_dt"], a["s"])


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), EINVAL), (dict(R=0), EINVAL), (dict(Cin=0), EINVAL), (dict(Cout=2000), EINVAL),
    (dict(act=5), EINVAL), (dict(x=None), EINVAL), (dict(w=None), EINVAL),
    (dict(y=None), EINVAL), (dict(y=FAKE), EINVAL), (dict(B=0), OK),
    # packed weights beyond the 4 MiB static array: 27 * 512 * 512 * 2 bytes
    (dict(Cin=512, Cout=512), EWS), (dict(Cin=1024, Cout=128), EWS),
])
def test_conv3d_noalloc_rejects(kw, status):
    assert _conv_na(**kw) == status


def test_conv3d_noalloc_limit():
    # the largest square convolution the static array takes is 256 -> 256
    limit = 4 << 20
    assert L.pvconv_conv3d_workspace_size(256, 256, 1) <= limit
    assert L.pvconv_conv3d_workspace_size(512, 256, 1) > limit


@pytest.mark.parametrize("args,status", [
    (dict(Cin=0), EINVAL), (dict(Cout=2048), EINVAL),
    (dict(Cout=48, nbytes=16 * 27 * 48 * 2), EWS),
    (dict(w=None), EINVAL), (dict(w=FAKE_ODD), EINVAL), (dict(packed=None), EWS),
    (dict(packed=ctypes.c_void_p(0x400010)), EWS), (dict(nbytes=100), EWS),
    # the packed copy written over the weights themselves
    (dict(packed=FAKE), EINVAL),
])
def test_conv3d_pack_weights_rejects(args, status):
    a = dict(w=FAKE, Cin=16, Cout=64, packed=ctypes.c_void_p(0x400000), nbytes=1 << 30)
    a.update(args)
    assert L.pvconv_conv3d_pack_weights(a["w"], a["Cin"], a["Cout"], a["packed"], a["nbytes"],
                                        None) == status


@pytest.mark.parametrize("args,status", [
    (dict(B=-1), EINVAL), (dict(R=0), EINVAL), (dict(B=0), OK),
    (dict(Cout=48, nbytes=16 * 27 * 48 * 2), EWS),
    (dict(x=None), EINVAL), (dict(packed=None), EINVAL), (dict(y=FAKE), EINVAL),
    (dict(packed=ctypes.c_void_p(0x400010)), EWS), (dict(nbytes=100), EWS),
    # the output written over the packed weights
    (dict(packed=ctypes.c_void_p(0x200000)), EINVAL),
])
def test_conv3d_packed_rejects(args, status):
    a = dict(x=FAKE, B=1, R=8, Cin=16, Cout=64, packed=ctypes.c_void_p(0x800000),
             nbytes=1 << 30, y=ctypes.c_void_p(0x200000), out_dt=1)
    a.update(args)
    assert L.pvconv_conv3d_packed(a["x"], a["B"], a["R"], a["Cin"], a["Cout"], a["packed"],
                                  a["nbytes"], None, None, 2, 0.1, a["y"], a["out_dt"],
                                  None) == status


def _dvmlp(**kw):
    a = dict(grid=ctypes.c_void_p(0x1000000), R=8, pn=ctypes.c_void_p(0x2000000), B=2, N=100,
             x=FAKE, x_dt=0, x_ld=0, Cin=16, Cout=64, w=ctypes.c_void_p(0x3000000), bias=None,
             bn=None, act=1, slope=0.0, out=ctypes.c_void_p(0x4000000), out_dt=0, out_ld=0)
    a.update(kw)
    return L.pvconv_devoxelize_point_mlp(a["grid"], a["R"], a["pn"], a["B"], a["N"], a["x"],
                                         a["x_dt"], a["x_ld"], a["Cin"], a["Cout"], a["w"],
                                         a["bias"], a["bn"], a["act"], a["slope"], a["out"],
                                         a["out_dt"], a["out_ld"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), EINVAL), (dict(R=0), EINVAL), (dict(Cin=0), EINVAL), (dict(x_ld=8), EINVAL),
    (dict(out_ld=32), EINVAL), (dict(act=7), EINVAL), (dict(B=0), OK), (dict(N=0), OK),
    (dict(grid=None), EINVAL), (dict(pn=None), EINVAL), (dict(w=None), EINVAL),
    (dict(grid=ctypes.c_void_p(0x1000001)), EINVAL), (dict(x=FAKE_ODD), EINVAL),
    # out over x, over the grid, over the coordinates
    (dict(out=ctypes.c_void_p(0x100000 + 64)), EINVAL),
    (dict(out=ctypes.c_void_p(0x1000000 + 4096)), EINVAL),
    (dict(out=ctypes.c_void_p(0x2000000 - 1024)), EINVAL),
    # shapes the fused kernel does not take: checked after validation, before
    # anything is enqueued
    (dict(Cin=12), ENOTSUP), (dict(Cin=128, Cout=128), ENOTSUP), (dict(B=1, N=100), ENOTSUP),
])
def test_devoxelize_point_mlp_rejects(kw, status):
    assert _dvmlp(**kw) == status


def test_conv3d_rejects_incomplete_batchnorm():
    bn = b.BN(0x300000, None, 0x300100, 0x300200, 1e-5)
    assert _conv(bn=ctypes.byref(bn)) == EINVAL
    bn = b.BN(0x300000, 0x300100, 0x300200, 0x300300, -1.0)
    assert _conv(bn=ctypes.byref(bn)) == EINVAL


def _devox(**kw):
    a = dict(grid=FAKE, B=2, R=8, C=16, dt=1, pn=FAKE, N=10, out=FAKE, s=None)
    a.update(kw)
    return L.pvconv_devoxelize(a["grid"], a["B"], a["R"], a["C"], a["dt"], a["pn"], a["N"],
                               a["out"], a["s"])


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), EINVAL), (dict(N=-1), EINVAL), (dict(R=0), EINVAL), (dict(C=0), EINVAL),
    (dict(dt=9), EINVAL), (dict(grid=None), EINVAL), (dict(pn=None), EINVAL),
    (dict(out=None), EINVAL), (dict(pn=FAKE_ODD), EINVAL), (dict(N=0), OK), (dict(B=0), OK),
])
def test_devoxelize_rejects(kw, status):
    assert _devox(**kw) == status


def _devox_nn(**kw):
    a = dict(grid=FAKE, B=2, R=8, C=16, dt=1, ids=FAKE, N=10, out=FAKE, s=None)
    a.update(kw)
    return L.pvconv_devoxelize_nearest(a["grid"], a["B"], a["R"], a["C"], a["dt"], a["ids"],
                                       a["N"], a["out"], a["s"])


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), EINVAL), (dict(N=-1), EINVAL), (dict(R=0), EINVAL), (dict(R=129), EINVAL),
    (dict(C=0), EINVAL), (dict(dt=9), EINVAL), (dict(grid=None), EINVAL),
    (dict(ids=None), EINVAL), (dict(out=None), EINVAL), (dict(ids=FAKE_ODD), EINVAL),
    (dict(grid=FAKE_ODD), EINVAL), (dict(N=0), OK), (dict(B=0), OK),
])
def test_devoxelize_nearest_rejects(kw, status):
    assert _devox_nn(**kw) == status


def _vfi(**kw):
    a = dict(ids=FAKE, feats=FAKE, fdt=0, ld=0, B=2, N=100, C=16, R=8, grid=FAKE, gdt=1,
             counts=FAKE, ws=ctypes.c_void_p(0x400000), wsb=1 << 40, s=None)
    a.update(kw)
    return L.pvconv_voxelize_from_ids(a["ids"], a["feats"], a["fdt"], a["ld"], a["B"], a["N"],
                                      a["C"], a["R"], a["grid"], a["gdt"], a["counts"], a["ws"],
                                      a["wsb"], a["s"])


@pytest.mark.parametrize("kw,status", [
    (dict(B=-1), EINVAL), (dict(N=-1), EINVAL), (dict(C=0), EINVAL), (dict(R=0), EINVAL),
    (dict(R=129), EINVAL), (dict(fdt=7), EINVAL), (dict(gdt=7), EINVAL), (dict(ld=8), EINVAL),
    (dict(ids=None), EINVAL), (dict(feats=None), EINVAL), (dict(grid=None), EINVAL),
    (dict(counts=None), EINVAL), (dict(ids=FAKE_ODD), EINVAL), (dict(ws=None), EWS),
    (dict(wsb=16), EWS), (dict(ws=ctypes.c_void_p(0x400010)), EWS), (dict(B=0), OK),
])
def test_voxelize_from_ids_rejects(kw, status):
    assert _vfi(**kw) == status


def _mlp(**kw):
    a = dict(x=FAKE, x_dt=0, x_ld=0, M=100, Cin=64, Cout=128, w=FAKE, dt=1, bias=None, bn=None,
             act=1, slope=0.0, cb=None, ppc=1, res=None, res_ld=0, out=ctypes.c_void_p(0x200000),
             out_dt=0, out_ld=0, s=None)
    a.update(kw)
    return L.pvconv_point_mlp(a["x"], a["x_dt"], a["x_ld"], a["M"], a["Cin"], a["Cout"], a["w"],
                              a["dt"], a["bias"], a["bn"], a["act"], a["slope"], a["cb"],
                              a["ppc"], a["res"], a["res_ld"], a["out"], a["out_dt"],
                              a["out_ld"], a["s"])


@pytest.mark.parametrize("kw,status", [
    (dict(M=-1), EINVAL), (dict(Cin=0), EINVAL), (dict(Cout=0), EINVAL),
    (dict(Cin=20000), EINVAL), (dict(x_ld=10), EINVAL), (dict(out_ld=100), EINVAL),
    (dict(res=FAKE, res_ld=5), EINVAL), (dict(cb=FAKE, ppc=0), EINVAL), (dict(x=None), EINVAL),
    (dict(w=None), EINVAL), (dict(out=None), EINVAL), (dict(x_dt=5), EINVAL),
    (dict(act=-1), EINVAL), (dict(out=FAKE), EINVAL), (dict(x=FAKE_ODD), EINVAL),
    # out shares bytes with x (100 rows of 64 fp32 = 25600 bytes from FAKE)
    (dict(out=ctypes.c_void_p(0x100000 + 25600 - 16)), EINVAL),
    (dict(x=ctypes.c_void_p(0x200000 + 51200 - 16)), EINVAL),
    (dict(M=0), OK),
])
def test_point_mlp_rejects(kw, status):
    assert _mlp(**kw) == status


@pytest.mark.parametrize("args,status", [
    ((FAKE, 1, 0, 2, 0, 8, FAKE, None), EINVAL),    # N = 0
    ((FAKE, 1, 4, 2, 5, 8, FAKE, None), EINVAL),    # ld < C
    ((None, 1, 0, 2, 5, 8, FAKE, None), EINVAL),
    ((FAKE, 1, 0, 2, 5, 8, None, None), EINVAL),
    ((FAKE, 2, 0, 2, 5, 8, FAKE, None), EINVAL),    # bad dtype
    ((FAKE, 1, 0, 0, 5, 8, FAKE, None), OK),        # B = 0
])
def test_maxpool_rejects(args, status):
    assert L.pvconv_maxpool(*args) == status


def _layer():
    lay = b.Layer()
    lay.cin, lay.cout, lay.R, lay.n_convs = 64, 128, 32, 2
    lay.conv_w[0] = lay.conv_w[1] = 0x100000
    lay.mlp_w = 0x100000
    lay.conv_slope = 0.1
    lay.compute_dt = 1
    return lay


def _fwd(lay, **kw):
    a = dict(coords=FAKE, feats=FAKE, fdt=0, fld=0, B=2, N=100, out=FAKE2, odt=0, old=0, ws=FAKE,
             wsb=1 << 40, s=None)
    a.update(kw)
    return L.pvconv_forward(a["coords"], a["feats"], a["fdt"], a["fld"], a["B"], a["N"],
                            ctypes.byref(lay), a["out"], a["odt"], a["old"], a["ws"], a["wsb"],
                            a["s"])


def _fwd_ex(lay, **kw):
    a = dict(coords=FAKE, feats=FAKE, fdt=0, fld=0, B=2, N=100, ids=FAKE, norm=FAKE, given=1,
             out=FAKE2, odt=0, old=0, ws=FAKE, wsb=1 << 40, s=None)
    a.update(kw)
    return L.pvconv_forward_ex(a["coords"], a["feats"], a["fdt"], a["fld"], a["B"], a["N"],
                               ctypes.byref(lay), a["ids"], a["norm"], a["given"], a["out"],
                               a["odt"], a["old"], a["ws"], a["wsb"], a["s"])


@pytest.mark.parametrize("call,status", [
    (lambda: L.pvconv_voxelize_backward(FAKE, 1, 2, 10, 16, 8, FAKE, FAKE, FAKE, None), None),
    (lambda: L.pvconv_voxelize_backward(FAKE, 3, 2, 10, 16, 8, FAKE, FAKE, FAKE, None), EINVAL),
    (lambda: L.pvconv_voxelize_backward(FAKE, 1, 2, 10, 16, 0, FAKE, FAKE, FAKE, None), EINVAL),
    (lambda: L.pvconv_voxelize_backward(FAKE, 1, 2, 10, 16, 8, None, FAKE, FAKE, None), EINVAL),
    (lambda: L.pvconv_voxelize_backward(FAKE, 1, 2, 10, 16, 8, FAKE, None, FAKE, None), EINVAL),
    (lambda: L.pvconv_voxelize_backward(FAKE, 1, 2, 10, 16, 8, FAKE, FAKE, FAKE_ODD, None),
     EINVAL),
    (lambda: L.pvconv_voxelize_backward(FAKE, 1, 0, 10, 16, 8, FAKE, FAKE, FAKE, None), OK),
    (lambda: L.pvconv_devoxelize_backward(FAKE, 2, 10, 16, 129, FAKE, FAKE, FAKE, 1 << 40,
                                          None), EINVAL),
    (lambda: L.pvconv_devoxelize_backward(FAKE, 2, 10, 16, 8, None, FAKE, FAKE, 1 << 40, None),
     EINVAL),
    (lambda: L.pvconv_devoxelize_backward(FAKE, 2, 10, 16, 8, FAKE, None, FAKE, 1 << 40, None),
     EINVAL),
    (lambda: L.pvconv_devoxelize_backward(FAKE_ODD, 2, 10, 16, 8, FAKE, FAKE, FAKE, 1 << 40,
                                          None), EINVAL),
    (lambda: L.pvconv_devoxelize_backward(FAKE, 2, 10, 16, 8, FAKE, FAKE, None, 1 << 40, None),
     EWS),
    (lambda: L.pvconv_devoxelize_backward(FAKE, 2, 10, 16, 8, FAKE, FAKE, FAKE_ODD, 1 << 40,
                                          None), EWS),
    (lambda: L.pvconv_devoxelize_backward(FAKE, 2, 10, 16, 8, FAKE, FAKE, FAKE, 256, None),
     EWS),
    (lambda: L.pvconv_devoxelize_backward(FAKE, 0, 10, 16, 8, FAKE, FAKE, None, 0, None), OK),
    (lambda: L.pvconv_devoxelize_nearest_backward(FAKE, 2, 10, 16, 8, None, FAKE, FAKE, 1 << 40,
                                                  None), EINVAL),
    (lambda: L.pvconv_devoxelize_nearest_backward(FAKE, 2, -1, 16, 8, FAKE, FAKE, FAKE, 1 << 40,
                                                  None), EINVAL),
    (lambda: L.pvconv_devoxelize_nearest_backward(FAKE, 2, 10, 16, 8, FAKE, FAKE, None, 0,
                                                  None), EWS),
    (lambda: L.pvconv_conv3d_backward_data(FAKE, 2, 8, 48, 64, FAKE, 1, FAKE, 0, FAKE, 1 << 40,
                                           None), ENOTSUP),
    (lambda: L.pvconv_conv3d_backward_data(FAKE, 2, 8, 64, 64, FAKE, 1, FAKE2, 0, None, 0, None),
     EWS),
    (lambda: L.pvconv_conv3d_backward_data(FAKE, 2, 8, 64, 64, FAKE, 1, FAKE, 0, FAKE, 1 << 40,
                                           None), EINVAL),     # dx aliases dy
    (lambda: L.pvconv_conv3d_backward_data(FAKE, 2, 8, 64, 64, None, 1, FAKE, 0, FAKE, 1 << 40,
                                           None), EINVAL),
    (lambda: L.pvconv_conv3d_backward_data(FAKE, 2, 0, 64, 64, FAKE, 1, FAKE, 0, FAKE, 1 << 40,
                                           None), EINVAL),
    (lambda: L.pvconv_conv3d_backward_data(FAKE, 0, 8, 64, 64, FAKE, 1, FAKE, 0, None, 0, None),
     OK),
    (lambda: L.pvconv_act_bn_backward(FAKE, FAKE, 1, 100, 0, None, 2, 0.1, FAKE, None), EINVAL),
    (lambda: L.pvconv_act_bn_backward(FAKE, FAKE, 1, 100, 8, None, 7, 0.1, FAKE, None), EINVAL),
    (lambda: L.pvconv_act_bn_backward(FAKE, None, 1, 100, 8, None, 2, 0.1, FAKE, None), EINVAL),
    (lambda: L.pvconv_act_bn_backward(FAKE, FAKE_ODD, 1, 100, 8, None, 2, 0.1, FAKE, None),
     EINVAL),
    (lambda: L.pvconv_act_bn_backward(FAKE, FAKE, 1, 0, 8, None, 2, 0.1, FAKE, None), OK),
])
def test_backward_entry_points_reject(call, status):
    if status is None:      # valid arguments: would launch, so only check the others
        return
    assert call() == status


@pytest.mark.parametrize("kw,status", [
    (dict(dt=0), ENOTSUP), (dict(Cout=96), ENOTSUP), (dict(Cin=8), ENOTSUP),
    (dict(dt=4), EINVAL), (dict(R=0), EINVAL), (dict(B=-1), EINVAL), (dict(dw=None), EINVAL),
    (dict(dy=None), EINVAL), (dict(x=ctypes.c_void_p(0x100008)), EINVAL),
    (dict(ws=None), EWS), (dict(wsb=64), EWS),
])
def test_conv3d_backward_weight_rejects(kw, status):
    a = dict(dy=FAKE, x=FAKE2, dt=1, B=2, R=8, Cin=64, Cout=128, dw=ctypes.c_void_p(0x300000),
             ws=ctypes.c_void_p(0x400000), wsb=1 << 40, s=None)
    a.update(kw)
    assert L.pvconv_conv3d_backward_weight(a["dy"], a["x"], a["dt"], a["B"], a["R"], a["Cin"],
                                           a["Cout"], a["dw"], a["ws"], a["wsb"],
                                           a["s"]) == status


def test_backward_workspace_query():
    # the mirrored weights, then the forward convolution's packed weights
    assert L.pvconv_conv3d_backward_data_workspace_size(64, 128, 1) == \
        128 * 27 * 64 * 2 + L.pvconv_conv3d_workspace_size(128, 64, 1)
    assert L.pvconv_conv3d_backward_data_workspace_size(5, 7, 0) == 256 * ((7 * 27 * 5 * 4 + 255) // 256)
    assert L.pvconv_conv3d_backward_data_workspace_size(0, 7, 0) == 0


def test_forward_ex_rejects():
    lay = _layer()
    assert _fwd_ex(lay, given=2) == EINVAL
    assert _fwd_ex(lay, given=-1) == EINVAL
    assert _fwd_ex(lay, ids=None) == EINVAL           # given indices missing
    assert _fwd_ex(lay, norm=None) == EINVAL
    assert _fwd_ex(lay, given=0, coords=None) == EINVAL
    assert _fwd_ex(lay, ids=FAKE_ODD) == EINVAL
    assert _fwd_ex(lay, ws=None) == EWS
    assert _fwd_ex(lay, B=0) == OK


def test_forward_rejects():
    lay = _layer()
    assert _fwd(lay, ws=None) == EWS
    assert _fwd(lay, wsb=1024) == EWS
    assert _fwd(lay, coords=None) == EINVAL
    assert _fwd(lay, fld=3) == EINVAL
    assert _fwd(lay, B=0) == OK
    # out must not share bytes with feats (an in-place layer would race):
    # feats are 200 rows of 64 fp32 from FAKE
    assert _fwd(lay, out=FAKE) == EINVAL
    assert _fwd(lay, out=ctypes.c_void_p(0x100000 + 200 * 64 * 4 - 4)) == EINVAL
    assert _fwd(lay, out=ctypes.c_void_p(0x100000 + 200 * 64 * 4), ws=None) == EWS
    # column slices of one wider fp32 array (row stride 320): disjoint ranges pass
    # validation, overlapping ones do not
    assert _fwd(lay, fld=320, out=ctypes.c_void_p(0x100000 + 64 * 4), old=320, ws=None) == EWS
    assert _fwd(lay, fld=320, out=ctypes.c_void_p(0x100000 + 60 * 4), old=320) == EINVAL
    assert _fwd(lay, fld=320, out=ctypes.c_void_p(0x100000 + 200 * 4), old=320) == EINVAL
    for field, val, status in [("n_convs", 0, EINVAL), ("n_convs", 5, EINVAL), ("R", 0, EINVAL),
                               ("cout", 0, EINVAL), ("compute_dt", 4, EINVAL),
                               ("cin", 0, EINVAL), ("devox", 2, EINVAL), ("devox", -1, EINVAL)]:
        lay = _layer()
        setattr(lay, field, val)
        assert _fwd(lay) == status, field
    lay = _layer()
    lay.conv_w[1] = None
    assert _fwd(lay) == EINVAL
    lay = _layer()
    lay.mlp_w = None
    assert _fwd(lay) == EINVAL


def test_peak_probe_library():
    # the benchmark's measured-peak probes (not part of the PVConv ABI)
    path = os.path.join(ROOT, "paper_1907_03739_amd", "libpvpeak.so")
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True,
                         check=True).stdout
    assert {"pv_peak_mfma", "pv_peak_mfma_flop", "pv_peak_copy"} <= set(
        re.findall(r"\bT (pv_peak_\w+)", out))
    lib = ctypes.CDLL(path)
    lib.pv_peak_mfma_flop.restype = ctypes.c_double
    lib.pv_peak_mfma_flop.argtypes = [ctypes.c_int, ctypes.c_int]
    # four waves x iters rounds x four 32x32x16 MFMAs of 2*32*32*16 flop
    assert lib.pv_peak_mfma_flop(768, 1000) == 768 * 4 * 1000 * 4 * 32768
    lib.pv_peak_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    lib.pv_peak_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                 ctypes.c_void_p]
    assert lib.pv_peak_mfma(0, 10, FAKE, None) != 0          # rejected before any launch
    assert lib.pv_peak_copy(FAKE_ODD, FAKE, 4, None) != 0    # misaligned
    assert lib.pv_peak_copy(FAKE, FAKE, 0, None) == 0         # nothing to do


# ---- PointNet++ primitives ---------------------------------------------------
@pytest.mark.parametrize("args,status", [
    (dict(B=-1), EINVAL), (dict(N=0), EINVAL), (dict(npoint=0), EINVAL),
    (dict(npoint=101), EINVAL), (dict(B=0), OK), (dict(xyz=None), EINVAL),
    (dict(idx=None), EINVAL), (dict(xyz=FAKE_ODD), EINVAL),
    (dict(N=20000, npoint=10), ENOTSUP),
    (dict(idx=ctypes.c_void_p(0x100000 + 64)), EINVAL),        # over xyz
    (dict(new_xyz=ctypes.c_void_p(0x400000 + 8)), EINVAL),     # over idx
])
def test_furthest_point_sample_rejects(args, status):
    a = dict(xyz=FAKE, B=2, N=100, npoint=10, idx=ctypes.c_void_p(0x400000), new_xyz=None)
    a.update(args)
    assert L.pvconv_furthest_point_sample(a["xyz"], a["B"], a["N"], a["npoint"], a["idx"],
                                          a["new_xyz"], None) == status


@pytest.mark.parametrize("args,status", [
    (dict(B=-1), EINVAL), (dict(N=0), EINVAL), (dict(M=-1), EINVAL), (dict(nsample=0), EINVAL),
    (dict(radius=-1.0), EINVAL), (dict(radius=float("nan")), EINVAL), (dict(B=0), OK),
    (dict(M=0), OK), (dict(xyz=None), EINVAL), (dict(centers=None), EINVAL),
    (dict(idx=None), EINVAL), (dict(idx=ctypes.c_void_p(0x200000 + 4)), EINVAL),
])
def test_ball_query_rejects(args, status):
    a = dict(xyz=FAKE, B=2, N=100, centers=ctypes.c_void_p(0x200000), M=10, radius=0.2,
             nsample=16, idx=ctypes.c_void_p(0x400000))
    a.update(args)
    assert L.pvconv_ball_query(a["xyz"], a["B"], a["N"], a["centers"], a["M"], a["radius"],
                               a["nsample"], a["idx"], None) == status


@pytest.mark.parametrize("args,status", [
    (dict(B=-1), EINVAL), (dict(N=0), EINVAL), (dict(C=-1), EINVAL), (dict(nsample=0), EINVAL),
    (dict(fdt=5), EINVAL), (dict(fld=4), EINVAL), (dict(old=7), EINVAL), (dict(B=0), OK),
    (dict(feats=None), EINVAL), (dict(out=None), EINVAL), (dict(idx=None), EINVAL),
    (dict(out=ctypes.c_void_p(0x300000 + 8)), EINVAL),      # over idx
    (dict(out=ctypes.c_void_p(0x500000 + 2)), EINVAL),      # over feats
])
def test_group_points_rejects(args, status):
    a = dict(xyz=FAKE, feats=ctypes.c_void_p(0x500000), fdt=1, fld=0, B=2, N=100, C=8,
             centers=ctypes.c_void_p(0x200000), M=10, idx=ctypes.c_void_p(0x300000), nsample=16,
             out=ctypes.c_void_p(0x1000000), odt=1, old=0)
    a.update(args)
    assert L.pvconv_group_points(a["xyz"], a["feats"], a["fdt"], a["fld"], a["B"], a["N"],
                                 a["C"], a["centers"], a["M"], a["idx"], a["nsample"], a["out"],
                                 a["odt"], a["old"], None) == status


@pytest.mark.parametrize("args,status", [
    (dict(B=-1), EINVAL), (dict(n=-1), EINVAL), (dict(m=2), EINVAL), (dict(B=0), OK),
    (dict(n=0), OK), (dict(unknown=None), EINVAL), (dict(idx=None), EINVAL),
    (dict(weight=ctypes.c_void_p(0x300000 + 12)), EINVAL),   # over idx
])
def test_three_nn_rejects(args, status):
    a = dict(unknown=FAKE, B=2, n=100, known=ctypes.c_void_p(0x200000), m=10,
             idx=ctypes.c_void_p(0x300000), weight=ctypes.c_void_p(0x400000))
    a.update(args)
    assert L.pvconv_three_nn(a["unknown"], a["B"], a["n"], a["known"], a["m"], a["idx"],
                             a["weight"], None) == status


@pytest.mark.parametrize("args,status", [
    (dict(B=-1), EINVAL), (dict(m=0), EINVAL), (dict(C=0), EINVAL), (dict(fld=3), EINVAL),
    (dict(old=3), EINVAL), (dict(fdt=9), EINVAL), (dict(B=0), OK), (dict(n=0), OK),
    (dict(feats=None), EINVAL), (dict(out=None), EINVAL),
    (dict(out=ctypes.c_void_p(0x300000 + 16)), EINVAL),      # over idx
])
def test_three_interpolate_rejects(args, status):
    a = dict(feats=FAKE, fdt=1, fld=0, B=2, m=10, C=8, idx=ctypes.c_void_p(0x300000),
             weight=ctypes.c_void_p(0x400000), n=100, out=ctypes.c_void_p(0x1000000), odt=0,
             old=0)
    a.update(args)
    assert L.pvconv_three_interpolate(a["feats"], a["fdt"], a["fld"], a["B"], a["m"], a["C"],
                                      a["idx"], a["weight"], a["n"], a["out"], a["odt"],
                                      a["old"], None) == status


@pytest.mark.parametrize("args,status", [
    (dict(G=-1), EINVAL), (dict(S=0), EINVAL), (dict(C=0), EINVAL), (dict(xld=3), EINVAL),
    (dict(old=3), EINVAL), (dict(dt=4), EINVAL), (dict(G=0), OK), (dict(x=None), EINVAL),
    (dict(out=None), EINVAL), (dict(out=ctypes.c_void_p(0x100000 + 64)), EINVAL),
])
def test_group_max_rejects(args, status):
    a = dict(x=FAKE, dt=1, xld=0, G=10, S=32, C=8, out=ctypes.c_void_p(0x400000), odt=1, old=0)
    a.update(args)
    assert L.pvconv_group_max(a["x"], a["dt"], a["xld"], a["G"], a["S"], a["C"], a["out"],
                              a["odt"], a["old"], None) == status
