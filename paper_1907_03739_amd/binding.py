"""Thin Python binding of libpvconv (include/pvconv.h).

Argument marshalling only: every function allocates its outputs (and any
workspace) as torch tensors on the input's device, passes raw device pointers,
sizes and the current torch stream to the C ABI, and raises on a non-OK
status. All computation happens in the library's HIP kernels. There is no
fallback: if libpvconv.so is missing the import fails.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpvconv.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build the HIP library first "
        "(python -m paper_1907_03739_amd.build, or __graft_entry__.build())")

_lib = ctypes.CDLL(LIB_PATH)

F32, BF16 = 0, 1
ACT = {"none": 0, "relu": 1, "leaky": 2}
MAX_CONVS = 4

_VP = ctypes.c_void_p
_I = ctypes.c_int
_SZ = ctypes.c_size_t
_F = ctypes.c_float


class BN(ctypes.Structure):
    _fields_ = [("gamma", _VP), ("beta", _VP), ("mean", _VP), ("var", _VP), ("eps", _F)]


class Layer(ctypes.Structure):
    _fields_ = [("cin", _I), ("cout", _I), ("R", _I), ("n_convs", _I),
                ("conv_w", _VP * MAX_CONVS), ("conv_bn", BN * MAX_CONVS),
                ("conv_slope", _F), ("mlp_w", _VP), ("mlp_b", _VP), ("mlp_bn", BN),
                ("compute_dt", _I), ("devox", _I)]

DEVOX = {"trilinear": 0, "nearest": 1}


_SIGS = {
    "pvconv_voxelize_workspace_size": ([_I, _I, _I], _SZ),
    "pvconv_voxelize": ([_VP, _VP, _I, _I, _I, _I, _I, _I, _VP, _I, _VP, _VP, _VP, _VP, _SZ, _VP],
                        _I),
    "pvconv_voxelize_from_ids": ([_VP, _VP, _I, _I, _I, _I, _I, _I, _VP, _I, _VP, _VP, _SZ,
                                  _VP], _I),
    "pvconv_conv3d_workspace_size": ([_I, _I, _I], _SZ),
    "pvconv_conv3d": ([_VP, _I, _I, _I, _I, _VP, _VP, _VP, _I, _F, _I, _VP, _I, _VP, _SZ, _VP],
                      _I),
    "pvconv_conv3d_pack_weights": ([_VP, _I, _I, _VP, _SZ, _VP], _I),
    "pvconv_conv3d_packed": ([_VP, _I, _I, _I, _I, _VP, _SZ, _VP, _VP, _I, _F, _VP, _I, _VP],
                             _I),
    "pvconv_devoxelize_point_mlp": ([_VP, _I, _VP, _I, _I, _VP, _I, _I, _I, _I, _VP, _VP, _VP,
                                     _I, _F, _VP, _I, _I, _VP], _I),
    "pvconv_furthest_point_sample": ([_VP, _I, _I, _I, _VP, _VP, _VP], _I),
    "pvconv_ball_query": ([_VP, _I, _I, _VP, _I, _F, _I, _VP, _VP], _I),
    "pvconv_group_points": ([_VP, _VP, _I, _I, _I, _I, _I, _VP, _I, _VP, _I, _VP, _I, _I, _VP],
                            _I),
    "pvconv_group_max": ([_VP, _I, _I, _I, _I, _I, _VP, _I, _I, _VP], _I),
    "pvconv_three_nn": ([_VP, _I, _I, _VP, _I, _VP, _VP, _VP], _I),
    "pvconv_three_interpolate": ([_VP, _I, _I, _I, _I, _I, _VP, _VP, _I, _VP, _I, _I, _VP], _I),
    "pvconv_conv3d_noalloc": ([_VP, _I, _I, _I, _I, _VP, _VP, _VP, _I, _F, _I, _VP, _I, _VP],
                              _I),
    "pvconv_devoxelize": ([_VP, _I, _I, _I, _I, _VP, _I, _VP, _VP], _I),
    "pvconv_devoxelize_nearest": ([_VP, _I, _I, _I, _I, _VP, _I, _VP, _VP], _I),
    "pvconv_point_mlp": ([_VP, _I, _I, _I, _I, _I, _VP, _I, _VP, _VP, _I, _F, _VP, _I, _VP, _I,
                          _VP, _I, _I, _VP], _I),
    "pvconv_maxpool": ([_VP, _I, _I, _I, _I, _I, _VP, _VP], _I),
    "pvconv_forward_workspace_size": ([_I, _I, ctypes.POINTER(Layer)], _SZ),
    "pvconv_forward": ([_VP, _VP, _I, _I, _I, _I, ctypes.POINTER(Layer), _VP, _I, _I, _VP, _SZ,
                        _VP], _I),
    "pvconv_forward_ex": ([_VP, _VP, _I, _I, _I, _I, ctypes.POINTER(Layer), _VP, _VP, _I, _VP,
                           _I, _I, _VP, _SZ, _VP], _I),
    "pvconv_status_string": ([_I], ctypes.c_char_p),
    "pvconv_voxelize_backward": ([_VP, _I, _I, _I, _I, _I, _VP, _VP, _VP, _VP], _I),
    "pvconv_devoxelize_backward_workspace_size": ([_I, _I, _I, _I], _SZ),
    "pvconv_devoxelize_backward": ([_VP, _I, _I, _I, _I, _VP, _VP, _VP, _SZ, _VP], _I),
    "pvconv_devoxelize_nearest_backward": ([_VP, _I, _I, _I, _I, _VP, _VP, _VP, _SZ, _VP], _I),
    "pvconv_conv3d_backward_data_workspace_size": ([_I, _I, _I], _SZ),
    "pvconv_conv3d_backward_data": ([_VP, _I, _I, _I, _I, _VP, _I, _VP, _I, _VP, _SZ, _VP],
                                    _I),
    "pvconv_act_bn_backward": ([_VP, _VP, _I, _I, _I, _VP, _I, _F, _VP, _VP], _I),
    "pvconv_conv3d_backward_weight_workspace_size": ([_I, _I, _I, _I], _SZ),
    "pvconv_conv3d_backward_weight": ([_VP, _VP, _I, _I, _I, _I, _I, _VP, _VP, _SZ, _VP], _I),
}
for _name, (_args, _res) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = _res

EXPORTED = tuple(_SIGS)


class PVConvError(RuntimeError):
    def __init__(self, fn, status):
        msg = _lib.pvconv_status_string(status).decode()
        super().__init__(f"{fn}: status {status} ({msg})")
        self.status = status


def _check(fn, status):
    if status != 0:
        raise PVConvError(fn, status)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _torch_dt(d) -> torch.dtype:
    if d in (F32, torch.float32, "f32"):
        return torch.float32
    if d in (BF16, torch.bfloat16, "bf16"):
        return torch.bfloat16
    raise TypeError(f"unsupported dtype {d}")


def _p(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _rows(t: torch.Tensor, nrows: int, ncols: int) -> int:
    """Row stride (elements) of a [.., rows, cols] view whose rows are evenly
    spaced and whose channels are contiguous."""
    if t.shape[-1] != ncols:
        raise ValueError("channel count mismatch")
    if t.numel() == 0:
        return ncols
    if t.stride(-1) != 1:
        raise ValueError("channels must be the innermost, contiguous dimension")
    ld = t.stride(-2) if t.dim() >= 2 else ncols
    if t.dim() == 3 and t.shape[0] > 1 and t.stride(0) != t.shape[1] * ld:
        raise ValueError("rows must be evenly spaced across clouds")
    return ld


def _bn_struct(bn) -> BN:
    if bn is None:
        return BN()
    g, b, m, v, eps = bn
    return BN(g.data_ptr(), b.data_ptr(), m.data_ptr(), v.data_ptr(), float(eps))


# ----------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ----------------------------------------------------------------------------
def _out(t: Optional[torch.Tensor], shape, dtype, device, what):
    """A caller-given output (checked) or a new one."""
    if t is None:
        return torch.empty(shape, dtype=dtype, device=device)
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype or not t.is_contiguous():
        raise ValueError(f"{what} must be a contiguous {tuple(shape)} {dtype} tensor")
    return t


def pvconv_voxelize(coords: torch.Tensor, feats: torch.Tensor, R: int,
                    grid_dtype=torch.float32, want_ids=True, want_norm=True, grid=None,
                    counts=None, ids=None, norm=None, workspace=None):
    """coords [B][N][3] f32, feats [B][N][C] -> (grid [B][R^3][C], counts [B][R^3],
    vox_id [B][N] or None, norm_coords [B][N][3] or None). Outputs and the
    workspace may be passed in (then nothing is allocated)."""
    B, N, _ = coords.shape
    C = feats.shape[-1]
    dev = coords.device
    ld = _rows(feats, N, C)
    grid = _out(grid, (B, R ** 3, C), _torch_dt(grid_dtype), dev, "grid")
    counts = _out(counts, (B, R ** 3), torch.int32, dev, "counts")
    ids = _out(ids, (B, N), torch.int32, dev, "ids") if want_ids else None
    pn = _out(norm, (B, N, 3), torch.float32, dev, "norm") if want_norm else None
    wsb = _lib.pvconv_voxelize_workspace_size(B, N, R)
    ws = workspace if workspace is not None and workspace.numel() >= wsb else \
        torch.empty(max(wsb, 256), dtype=torch.uint8, device=dev)
    _check("pvconv_voxelize", _lib.pvconv_voxelize(
        _p(coords), _p(feats), _dt(feats), ld, B, N, C, R, _p(grid), _dt(grid), _p(counts),
        _p(ids), _p(pn), _p(ws), wsb, _stream(coords)))
    return grid, counts, ids, pn


def pvconv_voxelize_from_ids(vox_id: torch.Tensor, feats: torch.Tensor, R: int,
                             grid_dtype=torch.float32, grid=None, counts=None, workspace=None):
    """vox_id [B][N] int32 (from pvconv_voxelize at the same R), feats [B][N][C]
    -> (grid [B][R^3][C], counts [B][R^3])."""
    B, N = vox_id.shape
    C = feats.shape[-1]
    dev = feats.device
    if vox_id.dtype != torch.int32 or not vox_id.is_contiguous():
        raise TypeError("vox_id must be a contiguous int32 tensor")
    ld = _rows(feats, N, C)
    grid = _out(grid, (B, R ** 3, C), _torch_dt(grid_dtype), dev, "grid")
    counts = _out(counts, (B, R ** 3), torch.int32, dev, "counts")
    wsb = _lib.pvconv_voxelize_workspace_size(B, N, R)
    ws = workspace if workspace is not None and workspace.numel() >= wsb else \
        torch.empty(max(wsb, 256), dtype=torch.uint8, device=dev)
    _check("pvconv_voxelize_from_ids", _lib.pvconv_voxelize_from_ids(
        _p(vox_id), _p(feats), _dt(feats), ld, B, N, C, R, _p(grid), _dt(grid), _p(counts),
        _p(ws), wsb, _stream(feats)))
    return grid, counts


def pvconv_conv3d(x: torch.Tensor, weight: torch.Tensor, R: int, bn=None,
                  bias: Optional[torch.Tensor] = None, act="leaky", slope=0.1,
                  out_dtype=None, out: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None):
    """x [B][R^3][Cin], weight [Cout][3][3][3][Cin] (same dtype) -> y [B][R^3][Cout]."""
    B, V, Cin = x.shape
    Cout = weight.shape[0]
    if V != R ** 3 or tuple(weight.shape[1:]) != (3, 3, 3, Cin):
        raise ValueError("shape mismatch")
    y = out if out is not None else torch.empty(
        (B, V, Cout), dtype=_torch_dt(out_dtype or x.dtype), device=x.device)
    need = _lib.pvconv_conv3d_workspace_size(Cin, Cout, _dt(x))
    if need and (workspace is None or workspace.numel() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    bns = _bn_struct(bn)
    _check("pvconv_conv3d", _lib.pvconv_conv3d(
        _p(x.contiguous()), B, R, Cin, Cout, _p(weight.contiguous()), _p(bias),
        ctypes.byref(bns) if bn is not None else None, ACT[act], slope, _dt(x), _p(y), _dt(y),
        _p(workspace) if need else None, workspace.numel() if need else 0, _stream(x)))
    return y


def pvconv_conv3d_pack_weights(weight: torch.Tensor, out: Optional[torch.Tensor] = None):
    """bf16 weight [Cout][3][3][3][Cin] -> its MFMA-order copy (uint8 bytes) for
    pvconv_conv3d_packed."""
    Cout, Cin = weight.shape[0], weight.shape[-1]
    if tuple(weight.shape[1:]) != (3, 3, 3, Cin) or weight.dtype != torch.bfloat16:
        raise ValueError("weight must be [Cout][3][3][3][Cin] bf16")
    need = _lib.pvconv_conv3d_workspace_size(Cin, Cout, BF16)
    if out is None:
        out = torch.empty(max(need, 256), dtype=torch.uint8, device=weight.device)
    _check("pvconv_conv3d_pack_weights", _lib.pvconv_conv3d_pack_weights(
        _p(weight.contiguous()), Cin, Cout, _p(out), out.numel(), _stream(weight)))
    return out


def pvconv_conv3d_packed(x: torch.Tensor, packed: torch.Tensor, Cout: int, R: int, bn=None,
                         bias: Optional[torch.Tensor] = None, act="leaky", slope=0.1,
                         out_dtype=None, out: Optional[torch.Tensor] = None):
    """x [B][R^3][Cin] bf16 with pre-packed weights -> y [B][R^3][Cout]."""
    B, V, Cin = x.shape
    if V != R ** 3:
        raise ValueError("shape mismatch")
    y = out if out is not None else torch.empty(
        (B, V, Cout), dtype=_torch_dt(out_dtype or x.dtype), device=x.device)
    bns = _bn_struct(bn)
    _check("pvconv_conv3d_packed", _lib.pvconv_conv3d_packed(
        _p(x.contiguous()), B, R, Cin, Cout, _p(packed), packed.numel(), _p(bias),
        ctypes.byref(bns) if bn is not None else None, ACT[act], slope, _p(y), _dt(y),
        _stream(x)))
    return y


def pvconv_devoxelize_point_mlp(grid: torch.Tensor, R: int, norm_coords: torch.Tensor,
                                x: torch.Tensor, weight: torch.Tensor, bias=None, bn=None,
                                act="relu", slope=0.0, out: Optional[torch.Tensor] = None,
                                out_dtype=torch.float32):
    """grid [B][R^3][Cout] bf16, norm_coords [B][N][3], x [B][N][Cin] (rows evenly
    strided), weight [Cout][Cin] bf16 -> act(BN(W x + b)) + devoxelised grid."""
    B, N, Cin = x.shape
    Cout = weight.shape[0]
    if tuple(grid.shape) != (B, R ** 3, Cout) or tuple(norm_coords.shape) != (B, N, 3):
        raise ValueError("shape mismatch")
    x_ld = _rows(x, N, Cin)
    if out is None:
        out = torch.empty((B, N, Cout), dtype=_torch_dt(out_dtype), device=x.device)
    out_ld = _rows(out, N, Cout)
    bns = _bn_struct(bn)
    _check("pvconv_devoxelize_point_mlp", _lib.pvconv_devoxelize_point_mlp(
        _p(grid.contiguous()), R, _p(norm_coords.contiguous()), B, N, _p(x), _dt(x), x_ld,
        Cin, Cout, _p(weight.contiguous()), _p(bias),
        ctypes.byref(bns) if bn is not None else None, ACT[act], slope, _p(out), _dt(out),
        out_ld, _stream(x)))
    return out


def _xyz(t: torch.Tensor, what: str):
    if t.dim() != 3 or t.shape[2] != 3 or t.dtype != torch.float32 or not t.is_contiguous():
        raise ValueError(f"{what} must be a contiguous [B][N][3] float32 tensor")
    return t


def pvconv_furthest_point_sample(xyz: torch.Tensor, npoint: int, idx=None, new_xyz=None,
                                 want_xyz=True):
    """xyz [B][N][3] f32 -> idx [B][npoint] int32 (and the sampled points
    [B][npoint][3] f32 unless want_xyz is False)."""
    B, N, _ = _xyz(xyz, "xyz").shape
    idx = _out(idx, (B, npoint), torch.int32, xyz.device, "idx")
    if want_xyz:
        new_xyz = _out(new_xyz, (B, npoint, 3), torch.float32, xyz.device, "new_xyz")
    _check("pvconv_furthest_point_sample", _lib.pvconv_furthest_point_sample(
        _p(xyz), B, N, npoint, _p(idx), _p(new_xyz) if want_xyz else None, _stream(xyz)))
    return (idx, new_xyz) if want_xyz else idx


def pvconv_ball_query(xyz: torch.Tensor, centers: torch.Tensor, radius: float, nsample: int,
                      idx=None):
    """-> idx [B][M][nsample] int32: the first nsample points within radius."""
    B, N, _ = _xyz(xyz, "xyz").shape
    M = _xyz(centers, "centers").shape[1]
    idx = _out(idx, (B, M, nsample), torch.int32, xyz.device, "idx")
    _check("pvconv_ball_query", _lib.pvconv_ball_query(
        _p(xyz), B, N, _p(centers), M, float(radius), nsample, _p(idx), _stream(xyz)))
    return idx


def pvconv_group_points(xyz: torch.Tensor, feats: Optional[torch.Tensor], centers: torch.Tensor,
                        idx: torch.Tensor, out: Optional[torch.Tensor] = None,
                        out_dtype=torch.bfloat16):
    """-> [B][M][nsample][3 + C]: neighbour coordinates relative to the centre,
    then the neighbour's features (feats [B][N][C], rows evenly strided, or None)."""
    B, N, _ = _xyz(xyz, "xyz").shape
    M, S = idx.shape[1], idx.shape[2]
    C = 0 if feats is None else feats.shape[2]
    fld = 0 if feats is None else _rows(feats, N, C)
    if out is None:
        out = torch.empty((B, M, S, 3 + C), dtype=_torch_dt(out_dtype), device=xyz.device)
    # a contiguous [B][M][nsample][3 + C] tensor, or [B*M*nsample][3 + C] rows
    # (possibly a column slice of a wider array)
    flat = out.view(B * M * S, out.shape[-1]) if out.dim() == 4 else out
    old = _rows(flat, B * M * S, 3 + C)
    _check("pvconv_group_points", _lib.pvconv_group_points(
        _p(xyz), _p(feats), _dt(feats) if feats is not None else F32, fld, B, N, C,
        _p(centers.contiguous()), M, _p(idx.contiguous()), S, _p(out), _dt(out), old,
        _stream(xyz)))
    return out


def pvconv_group_max(x: torch.Tensor, nsample: int, out: Optional[torch.Tensor] = None,
                     out_dtype=torch.float32):
    """x [G*nsample][C] (rows evenly strided) -> [G][C]: the maximum over each
    group of nsample rows; out may be a column slice of a wider [G][*] tensor."""
    rows, C = x.shape
    if rows % nsample:
        raise ValueError("rows must be a multiple of nsample")
    G = rows // nsample
    xld = _rows(x, rows, C)
    if out is None:
        out = torch.empty((G, C), dtype=_torch_dt(out_dtype), device=x.device)
    old = _rows(out, G, C)
    _check("pvconv_group_max", _lib.pvconv_group_max(_p(x), _dt(x), xld, G, nsample, C, _p(out),
                                                     _dt(out), old, _stream(x)))
    return out


def pvconv_three_nn(unknown: torch.Tensor, known: torch.Tensor, idx=None, weight=None):
    """-> idx [B][n][3] int32, weight [B][n][3] f32."""
    B, n, _ = _xyz(unknown, "unknown").shape
    m = _xyz(known, "known").shape[1]
    idx = _out(idx, (B, n, 3), torch.int32, unknown.device, "idx")
    weight = _out(weight, (B, n, 3), torch.float32, unknown.device, "weight")
    _check("pvconv_three_nn", _lib.pvconv_three_nn(_p(unknown), B, n, _p(known), m, _p(idx),
                                                   _p(weight), _stream(unknown)))
    return idx, weight


def pvconv_three_interpolate(feats: torch.Tensor, idx: torch.Tensor, weight: torch.Tensor,
                             out: Optional[torch.Tensor] = None, out_dtype=torch.float32):
    """feats [B][m][C] (rows evenly strided) -> [B][n][C]; out may be a column
    slice of a wider [B][n][*] tensor."""
    B, m, C = feats.shape
    n = idx.shape[1]
    fld = _rows(feats, m, C)
    if out is None:
        out = torch.empty((B, n, C), dtype=_torch_dt(out_dtype), device=feats.device)
    old = _rows(out, n, C)
    _check("pvconv_three_interpolate", _lib.pvconv_three_interpolate(
        _p(feats), _dt(feats), fld, B, m, C, _p(idx.contiguous()), _p(weight.contiguous()), n,
        _p(out), _dt(out), old, _stream(feats)))
    return out


def pvconv_conv3d_noalloc(x: torch.Tensor, weight: torch.Tensor, R: int, out: torch.Tensor,
                          bn=None, bias: Optional[torch.Tensor] = None, act="leaky", slope=0.1):
    """pvconv_conv3d into the caller's `out` [B][R^3][Cout] (its dtype is the output
    dtype), with the library's static workspace: the C call allocates nothing."""
    B, V, Cin = x.shape
    Cout = weight.shape[0]
    if V != R ** 3 or tuple(weight.shape[1:]) != (3, 3, 3, Cin):
        raise ValueError("shape mismatch")
    if tuple(out.shape) != (B, V, Cout) or not out.is_contiguous():
        raise ValueError("out must be a contiguous [B][R^3][Cout] tensor")
    if not (x.is_contiguous() and weight.is_contiguous()):
        raise ValueError("x and weight must be contiguous")
    bns = _bn_struct(bn)
    _check("pvconv_conv3d_noalloc", _lib.pvconv_conv3d_noalloc(
        _p(x), B, R, Cin, Cout, _p(weight), _p(bias),
        ctypes.byref(bns) if bn is not None else None, ACT[act], slope, _dt(x), _p(out),
        _dt(out), _stream(x)))
    return out


def pvconv_devoxelize(grid: torch.Tensor, R: int, norm_coords: torch.Tensor, out=None):
    """grid [B][R^3][C], norm_coords [B][N][3] f32 -> [B][N][C] f32."""
    B, V, C = grid.shape
    N = norm_coords.shape[1]
    out = _out(out, (B, N, C), torch.float32, grid.device, "out")
    _check("pvconv_devoxelize", _lib.pvconv_devoxelize(
        _p(grid.contiguous()), B, R, C, _dt(grid), _p(norm_coords.contiguous()), N, _p(out),
        _stream(grid)))
    return out


def pvconv_devoxelize_nearest(grid: torch.Tensor, R: int, vox_id: torch.Tensor, out=None):
    """grid [B][R^3][C], vox_id [B][N] int32 -> [B][N][C] f32 (each point takes
    the row of its voxel)."""
    B, V, C = grid.shape
    N = vox_id.shape[1]
    if vox_id.dtype != torch.int32:
        raise TypeError("vox_id must be int32")
    out = _out(out, (B, N, C), torch.float32, grid.device, "out")
    _check("pvconv_devoxelize_nearest", _lib.pvconv_devoxelize_nearest(
        _p(grid.contiguous()), B, R, C, _dt(grid), _p(vox_id.contiguous()), N, _p(out),
        _stream(grid)))
    return out


def pvconv_point_mlp(x: torch.Tensor, weight: torch.Tensor, bias=None, bn=None, act="relu",
                     slope=0.0, cloud_bias=None, points_per_cloud=1, residual=None,
                     out: Optional[torch.Tensor] = None, out_dtype=torch.float32):
    """x [..][Cin] (rows evenly strided), weight [Cout][Cin] -> [..][Cout]."""
    Cin = x.shape[-1]
    Cout = weight.shape[0]
    M = 1
    for d in x.shape[:-1]:
        M *= int(d)
    x_ld = _rows(x, M, Cin)
    if out is None:
        out = torch.empty(tuple(x.shape[:-1]) + (Cout,), dtype=_torch_dt(out_dtype),
                          device=x.device)
    out_ld = _rows(out, M, Cout)
    res_ld = _rows(residual, M, Cout) if residual is not None else 0
    bns = _bn_struct(bn)
    _check("pvconv_point_mlp", _lib.pvconv_point_mlp(
        _p(x), _dt(x), x_ld, M, Cin, Cout, _p(weight.contiguous()), _dt(weight), _p(bias),
        ctypes.byref(bns) if bn is not None else None, ACT[act], slope, _p(cloud_bias),
        points_per_cloud, _p(residual), res_ld, _p(out), _dt(out), out_ld, _stream(x)))
    return out


def pvconv_maxpool(x: torch.Tensor, out: Optional[torch.Tensor] = None):
    """x [B][N][C] (rows evenly strided) -> [B][C] f32."""
    B, N, C = x.shape
    ld = _rows(x, N, C)
    if out is None:
        out = torch.empty((B, C), dtype=torch.float32, device=x.device)
    elif tuple(out.shape) != (B, C) or out.dtype != torch.float32 or not out.is_contiguous():
        raise ValueError("out must be a contiguous [B][C] float32 tensor")
    _check("pvconv_maxpool", _lib.pvconv_maxpool(_p(x), _dt(x), ld, B, N, C, _p(out),
                                                 _stream(x)))
    return out


# ----------------------------------------------------------------------------
# backward (gradients with respect to the steps' inputs; fp32 gradients)
# ----------------------------------------------------------------------------
def pvconv_voxelize_backward(dgrid: torch.Tensor, R: int, vox_id: torch.Tensor,
                             counts: torch.Tensor, out=None):
    """dgrid [B][R^3][C] -> dfeats [B][N][C] f32 (dV of each point's voxel / count)."""
    B, V, C = dgrid.shape
    N = vox_id.shape[1]
    out = _out(out, (B, N, C), torch.float32, dgrid.device, "out")
    _check("pvconv_voxelize_backward", _lib.pvconv_voxelize_backward(
        _p(dgrid.contiguous()), _dt(dgrid), B, N, C, R, _p(vox_id.contiguous()),
        _p(counts.contiguous()), _p(out), _stream(dgrid)))
    return out


def _devox_bwd_ws(B: int, N: int, C: int, R: int, device, workspace):
    wsb = _lib.pvconv_devoxelize_backward_workspace_size(B, N, C, R)
    if workspace is not None and workspace.numel() >= wsb:
        return workspace, wsb
    return torch.empty(max(wsb, 256), dtype=torch.uint8, device=device), wsb


def pvconv_devoxelize_backward(dout: torch.Tensor, R: int, norm_coords: torch.Tensor, out=None,
                               workspace=None):
    """dout [B][N][C] f32 -> dgrid [B][R^3][C] f32 (trilinear weights, transposed)."""
    B, N, C = dout.shape
    out = _out(out, (B, R ** 3, C), torch.float32, dout.device, "out")
    ws, wsb = _devox_bwd_ws(B, N, C, R, dout.device, workspace)
    _check("pvconv_devoxelize_backward", _lib.pvconv_devoxelize_backward(
        _p(dout.contiguous()), B, N, C, R, _p(norm_coords.contiguous()), _p(out), _p(ws), wsb,
        _stream(dout)))
    return out


def pvconv_devoxelize_nearest_backward(dout: torch.Tensor, R: int, vox_id: torch.Tensor,
                                       out=None, workspace=None):
    """dout [B][N][C] f32 -> dgrid [B][R^3][C] f32 (each point's gradient to its cell)."""
    B, N, C = dout.shape
    out = _out(out, (B, R ** 3, C), torch.float32, dout.device, "out")
    ws, wsb = _devox_bwd_ws(B, N, C, R, dout.device, workspace)
    _check("pvconv_devoxelize_nearest_backward", _lib.pvconv_devoxelize_nearest_backward(
        _p(dout.contiguous()), B, N, C, R, _p(vox_id.contiguous()), _p(out), _p(ws), wsb,
        _stream(dout)))
    return out


def pvconv_conv3d_backward_data(dy: torch.Tensor, weight: torch.Tensor, R: int,
                                out_dtype=torch.float32, out=None, workspace=None):
    """dy [B][R^3][Cout], weight [Cout][3][3][3][Cin] (same dtype) -> dx [B][R^3][Cin]."""
    B, V, Cout = dy.shape
    Cin = weight.shape[-1]
    if V != R ** 3 or tuple(weight.shape[:4]) != (Cout, 3, 3, 3):
        raise ValueError("shape mismatch")
    dx = _out(out, (B, V, Cin), _torch_dt(out_dtype), dy.device, "out")
    need = _lib.pvconv_conv3d_backward_data_workspace_size(Cin, Cout, _dt(dy))
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dy.device)
    _check("pvconv_conv3d_backward_data", _lib.pvconv_conv3d_backward_data(
        _p(dy.contiguous()), B, R, Cin, Cout, _p(weight.contiguous()), _dt(dy), _p(dx),
        _dt(dx), _p(workspace), workspace.numel(), _stream(dy)))
    return dx


def pvconv_conv3d_backward_weight(dy: torch.Tensor, x: torch.Tensor, R: int, out=None,
                                  workspace=None):
    """dy [B][R^3][Cout], x [B][R^3][Cin] (bf16) -> dW [Cout][3][3][3][Cin] f32."""
    B, V, Cout = dy.shape
    Cin = x.shape[-1]
    if V != R ** 3 or tuple(x.shape[:2]) != (B, V):
        raise ValueError("shape mismatch")
    dw = _out(out, (Cout, 3, 3, 3, Cin), torch.float32, dy.device, "out")
    need = _lib.pvconv_conv3d_backward_weight_workspace_size(B, R, Cin, Cout)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dy.device)
    _check("pvconv_conv3d_backward_weight", _lib.pvconv_conv3d_backward_weight(
        _p(dy.contiguous()), _p(x.contiguous()), _dt(dy), B, R, Cin, Cout, _p(dw),
        _p(workspace), workspace.numel(), _stream(dy)))
    return dw


def pvconv_act_bn_backward(dy: torch.Tensor, y: torch.Tensor, bn=None, act="leaky", slope=0.1,
                           out=None):
    """y = act(BN(z)) [..][C]; dy [..][C] f32 -> dz [..][C] f32."""
    C = y.shape[-1]
    M = y.numel() // C
    if dy.shape != y.shape:
        raise ValueError("dy and y must have the same shape")
    out = _out(out, tuple(y.shape), torch.float32, y.device, "out")
    bns = _bn_struct(bn)
    _check("pvconv_act_bn_backward", _lib.pvconv_act_bn_backward(
        _p(dy.contiguous()), _p(y.contiguous()), _dt(y), M, C,
        ctypes.byref(bns) if bn is not None else None, ACT[act], slope, _p(out), _stream(y)))
    return out


class DeviceLayer:
    """Device copies of one PVConv layer's parameters plus the C struct that
    points at them. Weights are stored in the compute dtype."""

    def __init__(self, params, device, compute_dtype=torch.bfloat16):
        self.params = params
        dt = _torch_dt(compute_dtype)
        f = lambda a: torch.as_tensor(a, dtype=torch.float32).to(device)
        self.conv_w = [f(w).to(dt).contiguous() for w in params.conv_w]
        self.conv_bn = [(f(b.gamma), f(b.beta), f(b.mean), f(b.var), b.eps)
                        for b in params.conv_bn]
        self.mlp_w = f(params.mlp_w).to(dt).contiguous()
        self.mlp_b = f(params.mlp_b) if params.mlp_b is not None else None
        mb = params.mlp_bn
        self.mlp_bn = (f(mb.gamma), f(mb.beta), f(mb.mean), f(mb.var), mb.eps)
        L = Layer()
        L.cin, L.cout, L.R, L.n_convs = params.cin, params.cout, params.R, params.n_convs
        for i, (w, bn) in enumerate(zip(self.conv_w, self.conv_bn)):
            L.conv_w[i] = w.data_ptr()
            L.conv_bn[i] = _bn_struct(bn)
        L.conv_slope = params.slope
        L.mlp_w = self.mlp_w.data_ptr()
        L.mlp_b = self.mlp_b.data_ptr() if self.mlp_b is not None else None
        L.mlp_bn = _bn_struct(self.mlp_bn)
        L.compute_dt = _dt(self.mlp_w)
        L.devox = DEVOX[getattr(params, "devox", "trilinear")]
        self.struct = L
        self.dtype = dt


def pvconv_forward_workspace_size(B: int, N: int, layer: DeviceLayer) -> int:
    return _lib.pvconv_forward_workspace_size(B, N, ctypes.byref(layer.struct))


def pvconv_forward(coords: torch.Tensor, feats: torch.Tensor, layer: DeviceLayer,
                   out: Optional[torch.Tensor] = None, out_dtype=torch.float32,
                   workspace: Optional[torch.Tensor] = None,
                   vox_id: Optional[torch.Tensor] = None, norm: Optional[torch.Tensor] = None,
                   ids_given: bool = False):
    """One PVConv layer: coords [B][N][3] f32, feats [B][N][cin] -> [B][N][cout].

    vox_id [B][N] int32 and norm [B][N][3] f32: written by the call (outputs),
    or with ids_given=True read instead of normalising again (from an earlier
    call on the same coordinates at the same R; coords is then not read)."""
    B, N = feats.shape[0], feats.shape[1]
    cin, cout = layer.params.cin, layer.params.cout
    f_ld = _rows(feats, N, cin)
    if out is None:
        out = torch.empty((B, N, cout), dtype=_torch_dt(out_dtype), device=feats.device)
    o_ld = _rows(out, N, cout)
    need = pvconv_forward_workspace_size(B, N, layer)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=feats.device)
    for t, shape, dt in ((vox_id, (B, N), torch.int32), (norm, (B, N, 3), torch.float32)):
        if t is not None and (tuple(t.shape) != shape or t.dtype != dt or not t.is_contiguous()):
            raise ValueError(f"expected a contiguous {shape} {dt} tensor")
    if ids_given and (vox_id is None or norm is None):
        raise ValueError("ids_given needs vox_id and norm")
    _check("pvconv_forward_ex", _lib.pvconv_forward_ex(
        _p(coords), _p(feats), _dt(feats), f_ld, B, N, ctypes.byref(layer.struct), _p(vox_id),
        _p(norm), int(ids_given), _p(out), _dt(out), o_ld, _p(workspace), workspace.numel(),
        _stream(feats)))
    return out
