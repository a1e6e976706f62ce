"""PVConv CPU oracle -- TEST INFRASTRUCTURE ONLY.

Plain fp64 reference of one Point-Voxel Convolution layer and of the PVCNN
network glue, written from the paper (Liu et al., "Point-Voxel CNN for
Efficient 3D Deep Learning", Section 4 and Section 5.1 "Models"). The per-step
arithmetic is in pvconv_oracle.c; this module loads it with ctypes and composes
the steps in the paper's order. Only tests, the package smoke check and the
benchmark's CPU-baseline leg may import it; the GPU library never does, and
nothing here imports the GPU library.

Every function takes and returns numpy arrays. Floating-point inputs are
upcast to float64 exactly (fp32 and bf16-representable values are exact in
fp64).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pvconv_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libpvconv_oracle.so")
_lib = None

_P = ctypes.c_void_p
_I64 = ctypes.c_int64


# A build of the same source with AddressSanitizer and UndefinedBehaviorSanitizer
# (host code only), for the test that runs the oracle under them.
SANITIZED_LIB_PATH = os.path.join(_HERE, "libpvconv_oracle_san.so")


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compile the oracle with gcc (fp64, no FMA contraction, OpenMP);
    sanitize: the ASan + UBSan build at SANITIZED_LIB_PATH instead."""
    out = SANITIZED_LIB_PATH if sanitize else _LIB_PATH
    extra = ["-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined"] if sanitize else []
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-Wall", "-Wextra", *extra, "-o", out + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = os.environ.get("PV_ORACLE_LIB", _LIB_PATH)
    if path == _LIB_PATH and (not os.path.exists(_LIB_PATH) or
                              os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
        build()
    lib = ctypes.CDLL(path)
    sig = {
        "ref_normalize": [_P, _I64, _I64, _P, _P, _P],
        "ref_voxel_ids": [_P, _I64, _I64, ctypes.c_int, _P],
        "ref_voxelize": [_P, _P, _I64, _I64, _I64, ctypes.c_int, _P, _P],
        "ref_conv3d": [_P, _I64, ctypes.c_int, _I64, _I64, _P, _P],
        "ref_conv3d_at": [_P, _I64, ctypes.c_int, _I64, _I64, _P, _I64, _P, _P],
        "ref_batchnorm": [_P, _I64, _I64, _P, _P, _P, _P, ctypes.c_double],
        "ref_devoxelize": [_P, _I64, ctypes.c_int, _I64, _P, _I64, _P],
        "ref_devoxelize_weights": [_P, _I64, ctypes.c_int, _P, _P],
        "ref_devoxelize_nearest": [_P, _I64, ctypes.c_int, _I64, _P, _I64, _P],
        "ref_voxelize_backward": [_P, _P, _P, _I64, _I64, _I64, ctypes.c_int, _P],
        "ref_devoxelize_backward": [_P, _P, _I64, _I64, _I64, ctypes.c_int, _P],
        "ref_devoxelize_nearest_backward": [_P, _P, _I64, _I64, _I64, ctypes.c_int, _P],
        "ref_conv3d_backward_data": [_P, _I64, ctypes.c_int, _I64, _I64, _P, _P],
        "ref_conv3d_backward_weight": [_P, _P, _I64, ctypes.c_int, _I64, _I64, _P],
        "ref_linear": [_P, _I64, _I64, _I64, _P, _P, _P],
        "ref_maxpool": [_P, _I64, _I64, _I64, _P],
        "ref_fps": [_P, _I64, _I64, _I64, _P],
        "ref_ball_query": [_P, _I64, _I64, _P, _I64, ctypes.c_float, _I64, _P],
        "ref_group": [_P, _P, _I64, _I64, _I64, _P, _I64, _P, _I64, _P],
        "ref_three_nn": [_P, _I64, _I64, _P, _I64, _P, _P],
        "ref_three_interpolate": [_P, _I64, _I64, _I64, _P, _P, _I64, _P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.ref_leaky_relu.argtypes = [_P, _I64, ctypes.c_double]
    lib.ref_leaky_relu.restype = None
    lib.ref_relu.argtypes = [_P, _I64]
    lib.ref_relu.restype = None
    # the OpenMP runtime the library links (thread count of its loops)
    lib.omp_set_num_threads.argtypes = [ctypes.c_int]
    lib.omp_set_num_threads.restype = None
    lib.omp_get_max_threads.argtypes = []
    lib.omp_get_max_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def set_threads(n: int) -> None:
    """Number of threads the oracle's parallel loops use from now on."""
    _load().omp_set_num_threads(int(n))


def threads() -> int:
    """Number of threads the oracle's parallel loops use."""
    return int(_load().omp_get_max_threads())


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what}: invalid input (rc={rc})")


# ----------------------------------------------------------------------------
# single steps (Section 4)
# ----------------------------------------------------------------------------
def normalize(coords: np.ndarray):
    """coords [B][N][3] fp32 -> (centroid [B][3], radius [B], pnorm [B][N][3])."""
    lib = _load()
    coords = np.ascontiguousarray(coords, dtype=np.float32)
    B, N, _ = coords.shape
    c = np.empty((B, 3))
    m = np.empty(B)
    pn = np.empty((B, N, 3))
    _check(lib.ref_normalize(_ptr(coords), B, N, _ptr(c), _ptr(m), _ptr(pn)), "normalize")
    return c, m, pn


def voxel_ids(pnorm: np.ndarray, R: int) -> np.ndarray:
    """pnorm [B][N][3] -> ids [B][N] int32 (Eq. 2 indicator, clamped)."""
    lib = _load()
    pnorm = _f64(pnorm)
    B, N, _ = pnorm.shape
    ids = np.empty((B, N), np.int32)
    _check(lib.ref_voxel_ids(_ptr(pnorm), B, N, R, _ptr(ids)), "voxel_ids")
    return ids


def voxelize(ids: np.ndarray, feats: np.ndarray, R: int):
    """ids [B][N], feats [B][N][C] -> (grid [B][R^3][C] fp64, counts [B][R^3] int32)."""
    lib = _load()
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    feats = _f64(feats)
    B, N, C = feats.shape
    V = R ** 3
    grid = np.empty((B, V, C))
    counts = np.empty((B, V), np.int32)
    _check(lib.ref_voxelize(_ptr(ids), _ptr(feats), B, N, C, R, _ptr(grid), _ptr(counts)),
           "voxelize")
    return grid, counts


def conv3d(x: np.ndarray, w: np.ndarray, R: int) -> np.ndarray:
    """x [B][R^3][Cin], w [Cout][3][3][3][Cin] -> y [B][R^3][Cout] (no BN)."""
    lib = _load()
    x = _f64(x)
    w = _f64(w)
    B, V, Cin = x.shape
    assert V == R ** 3 and w.shape[1:] == (3, 3, 3, Cin)
    Cout = w.shape[0]
    y = np.empty((B, V, Cout))
    _check(lib.ref_conv3d(_ptr(x), B, R, Cin, Cout, _ptr(w), _ptr(y)), "conv3d")
    return y


def conv3d_at(x: np.ndarray, w: np.ndarray, R: int, sel: np.ndarray) -> np.ndarray:
    """The convolution at the selected outputs sel[j] = b*R^3 + voxel -> [n_sel][Cout]."""
    lib = _load()
    x = _f64(x)
    w = _f64(w)
    B, V, Cin = x.shape
    Cout = w.shape[0]
    sel = np.ascontiguousarray(sel, dtype=np.int64)
    y = np.empty((len(sel), Cout))
    _check(lib.ref_conv3d_at(_ptr(x), B, R, Cin, Cout, _ptr(w), len(sel), _ptr(sel), _ptr(y)),
           "conv3d_at")
    return y


def batchnorm(y: np.ndarray, bn) -> np.ndarray:
    """Running-statistics batch normalisation over the last axis (copy)."""
    lib = _load()
    out = _f64(y).copy()
    C = out.shape[-1]
    M = out.size // C
    g, b, mu, var = (_f64(bn.gamma), _f64(bn.beta), _f64(bn.mean), _f64(bn.var))
    _check(lib.ref_batchnorm(_ptr(out), M, C, _ptr(g), _ptr(b), _ptr(mu), _ptr(var),
                             float(bn.eps)), "batchnorm")
    return out


def leaky_relu(y: np.ndarray, slope: float) -> np.ndarray:
    lib = _load()
    out = _f64(y).copy()
    lib.ref_leaky_relu(_ptr(out), out.size, slope)
    return out


def relu(y: np.ndarray) -> np.ndarray:
    lib = _load()
    out = _f64(y).copy()
    lib.ref_relu(_ptr(out), out.size)
    return out


def devoxelize(grid: np.ndarray, R: int, pnorm: np.ndarray) -> np.ndarray:
    """grid [B][R^3][C], pnorm [B][N][3] -> [B][N][C] (trilinear)."""
    lib = _load()
    grid = _f64(grid)
    pnorm = _f64(pnorm)
    B, V, C = grid.shape
    N = pnorm.shape[1]
    out = np.empty((B, N, C))
    _check(lib.ref_devoxelize(_ptr(grid), B, R, C, _ptr(pnorm), N, _ptr(out)), "devoxelize")
    return out


def devoxelize_nearest(grid: np.ndarray, R: int, ids: np.ndarray) -> np.ndarray:
    """grid [B][R^3][C], ids [B][N] -> [B][N][C]: each point takes the row of
    the voxel it falls into (Section 4.1 "Devoxelization", nearest neighbour)."""
    lib = _load()
    grid = _f64(grid)
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    B, V, C = grid.shape
    N = ids.shape[1]
    out = np.empty((B, N, C))
    _check(lib.ref_devoxelize_nearest(_ptr(grid), B, R, C, _ptr(ids), N, _ptr(out)),
           "devoxelize_nearest")
    return out


def devoxelize_weights(pnorm: np.ndarray, R: int):
    """The 8 cells (linear id within the cloud) and trilinear weights per point."""
    lib = _load()
    pn = _f64(pnorm).reshape(-1, 3)
    cells = np.empty((pn.shape[0], 8), np.int64)
    wts = np.empty((pn.shape[0], 8))
    _check(lib.ref_devoxelize_weights(_ptr(pn), pn.shape[0], R, _ptr(cells), _ptr(wts)),
           "devoxelize_weights")
    shape = pnorm.shape[:-1] + (8,)
    return cells.reshape(shape), wts.reshape(shape)


# ----------------------------------------------------------------------------
# backward: gradients of the steps with respect to their inputs (and of the
# convolution with respect to its weights), the adjoints of the forward maps
# ----------------------------------------------------------------------------
def voxelize_backward(dgrid: np.ndarray, ids: np.ndarray, counts: np.ndarray,
                      R: int) -> np.ndarray:
    """dL/dV [B][R^3][C] -> dL/df [B][N][C] (Eq. 2's average, transposed)."""
    lib = _load()
    dgrid = _f64(dgrid)
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    B, V, C = dgrid.shape
    N = ids.shape[1]
    out = np.empty((B, N, C))
    _check(lib.ref_voxelize_backward(_ptr(dgrid), _ptr(ids), _ptr(counts), B, N, C, R,
                                     _ptr(out)), "voxelize_backward")
    return out


def devoxelize_backward(dout: np.ndarray, R: int, pnorm: np.ndarray) -> np.ndarray:
    """dL/dout [B][N][C] -> dL/dV [B][R^3][C] (trilinear weights, transposed)."""
    lib = _load()
    dout = _f64(dout)
    pnorm = _f64(pnorm)
    B, N, C = dout.shape
    out = np.empty((B, R ** 3, C))
    _check(lib.ref_devoxelize_backward(_ptr(dout), _ptr(pnorm), B, N, C, R, _ptr(out)),
           "devoxelize_backward")
    return out


def devoxelize_nearest_backward(dout: np.ndarray, R: int, ids: np.ndarray) -> np.ndarray:
    """dL/dout [B][N][C] -> dL/dV [B][R^3][C] (each point's gradient to its cell)."""
    lib = _load()
    dout = _f64(dout)
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    B, N, C = dout.shape
    out = np.empty((B, R ** 3, C))
    _check(lib.ref_devoxelize_nearest_backward(_ptr(dout), _ptr(ids), B, N, C, R, _ptr(out)),
           "devoxelize_nearest_backward")
    return out


def conv3d_backward_data(dy: np.ndarray, w: np.ndarray, R: int) -> np.ndarray:
    """dL/dy [B][R^3][Cout], w [Cout][3][3][3][Cin] -> dL/dx [B][R^3][Cin]."""
    lib = _load()
    dy = _f64(dy)
    w = _f64(w)
    B, V, Cout = dy.shape
    Cin = w.shape[-1]
    out = np.empty((B, V, Cin))
    _check(lib.ref_conv3d_backward_data(_ptr(dy), B, R, Cin, Cout, _ptr(w), _ptr(out)),
           "conv3d_backward_data")
    return out


def conv3d_backward_weight(dy: np.ndarray, x: np.ndarray, R: int) -> np.ndarray:
    """dL/dy [B][R^3][Cout], x [B][R^3][Cin] -> dL/dW [Cout][3][3][3][Cin]."""
    lib = _load()
    dy = _f64(dy)
    x = _f64(x)
    B, V, Cout = dy.shape
    Cin = x.shape[-1]
    out = np.empty((Cout, 3, 3, 3, Cin))
    _check(lib.ref_conv3d_backward_weight(_ptr(dy), _ptr(x), B, R, Cin, Cout, _ptr(out)),
           "conv3d_backward_weight")
    return out


def act_bn_backward(dy: np.ndarray, y: np.ndarray, bn, act: str, slope: float = 0.1):
    """y = act(BN(z)) per channel: dL/dz = dL/dy * act'(y) * gamma / sqrt(var + eps).
    The rectifiers' derivative is read from the sign of y (equal to that of
    BN(z) for a positive slope): 1 where y > 0, slope (leaky) or 0 (relu)
    elsewhere. bn None: identity."""
    dy = _f64(dy)
    y = _f64(y)
    if act == "leaky":
        d = np.where(y > 0, 1.0, slope)
    elif act == "relu":
        d = np.where(y > 0, 1.0, 0.0)
    else:
        d = np.ones_like(y)
    scale = 1.0 if bn is None else (_f64(bn.gamma) / np.sqrt(_f64(bn.var) + bn.eps))
    return dy * d * scale


def linear(x: np.ndarray, w: np.ndarray, bias: Optional[np.ndarray] = None) -> np.ndarray:
    """x [..][Cin], w [Cout][Cin] -> x w^T + bias."""
    lib = _load()
    x = _f64(x)
    w = _f64(w)
    Cin = x.shape[-1]
    M = x.size // Cin
    Cout = w.shape[0]
    y = np.empty(x.shape[:-1] + (Cout,))
    bias_arr = _f64(bias) if bias is not None else None
    bp = _ptr(bias_arr) if bias_arr is not None else None
    _check(lib.ref_linear(_ptr(x), M, Cin, Cout, _ptr(w), bp, _ptr(y)), "linear")
    return y


def maxpool(x: np.ndarray) -> np.ndarray:
    """x [B][N][C] -> [B][C]."""
    lib = _load()
    x = _f64(x)
    B, N, C = x.shape
    out = np.empty((B, C))
    _check(lib.ref_maxpool(_ptr(x), B, N, C, _ptr(out)), "maxpool")
    return out


# ----------------------------------------------------------------------------
# PointNet++ primitives of PVCNN++ (Section 5.2 "Models": PointNet++ extended
# with PVConv), as PointNet++ defines them. The choices of an index (farthest
# point, ball membership, nearest neighbours) compare fp32 squared distances
# formed as the kernels form them: fma(dz, dz, fma(dy, dy, dx * dx)).
# ----------------------------------------------------------------------------
def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def fps(xyz: np.ndarray, npoint: int) -> np.ndarray:
    """Iterative farthest point sampling: xyz [B][N][3] -> indices [B][npoint]
    (the first is point 0; each next maximises the distance to the samples
    taken so far, the lowest index among equals)."""
    lib = _load()
    xyz = _f32(xyz)
    B, N, _ = xyz.shape
    idx = np.empty((B, npoint), np.int32)
    _check(lib.ref_fps(_ptr(xyz), B, N, npoint, _ptr(idx)), "fps")
    return idx


def gather_points(xyz: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """xyz [B][N][D], idx [B][M] -> [B][M][D] (the sampled points)."""
    return np.stack([xyz[b][idx[b]] for b in range(xyz.shape[0])])


def ball_query(xyz: np.ndarray, centers: np.ndarray, radius: float, nsample: int) -> np.ndarray:
    """For each centre, the first nsample points in index order within the
    radius (squared distance below radius^2), short lists completed with
    their first entry: xyz [B][N][3], centers [B][M][3] -> [B][M][nsample]."""
    lib = _load()
    xyz, centers = _f32(xyz), _f32(centers)
    B, N, _ = xyz.shape
    M = centers.shape[1]
    idx = np.empty((B, M, nsample), np.int32)
    _check(lib.ref_ball_query(_ptr(xyz), B, N, _ptr(centers), M, float(radius), nsample,
                              _ptr(idx)), "ball_query")
    return idx


def group(xyz: np.ndarray, feats: np.ndarray, centers: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """Rows (x_j - c_i, f_j) for each centre i and each of its neighbours j:
    -> [B][M][nsample][3 + C]."""
    lib = _load()
    xyz, centers = _f32(xyz), _f32(centers)
    feats = _f64(feats)
    idx = np.ascontiguousarray(idx, np.int32)
    B, N, _ = xyz.shape
    C = feats.shape[2]
    M, S = idx.shape[1], idx.shape[2]
    out = np.empty((B, M, S, 3 + C))
    _check(lib.ref_group(_ptr(xyz), _ptr(feats), B, N, C, _ptr(centers), M, _ptr(idx), S,
                         _ptr(out)), "group")
    return out


def three_nn(unknown: np.ndarray, known: np.ndarray):
    """The three nearest known points of each unknown point and their
    normalised inverse-distance weights: -> idx [B][n][3], weight [B][n][3]."""
    lib = _load()
    unknown, known = _f32(unknown), _f32(known)
    B, n, _ = unknown.shape
    m = known.shape[1]
    idx = np.empty((B, n, 3), np.int32)
    w = np.empty((B, n, 3))
    _check(lib.ref_three_nn(_ptr(unknown), B, n, _ptr(known), m, _ptr(idx), _ptr(w)),
           "three_nn")
    return idx, w


def three_interpolate(feats: np.ndarray, idx: np.ndarray, weight: np.ndarray) -> np.ndarray:
    """out[b][i] = sum_k weight[b][i][k] * feats[b][idx[b][i][k]]: feats
    [B][m][C] -> [B][n][C]."""
    lib = _load()
    feats = _f64(feats)
    idx = np.ascontiguousarray(idx, np.int32)
    weight = _f64(weight)
    B, m, C = feats.shape
    n = idx.shape[1]
    out = np.empty((B, n, C))
    _check(lib.ref_three_interpolate(_ptr(feats), B, m, C, _ptr(idx), _ptr(weight), n,
                                     _ptr(out)), "three_interpolate")
    return out


# ----------------------------------------------------------------------------
# composition: one PVConv layer (Figure "overview", Sections 4.1-4.3)
# ----------------------------------------------------------------------------
def _storage(stage_dtype):
    if stage_dtype not in ("f64", "bf16"):
        raise ValueError("stage_dtype must be 'f64' or 'bf16'")
    return round_bf16 if stage_dtype == "bf16" else (lambda v: v)


def voxel_branch(coords, feats, layer, stage_dtype="f64"):
    """Normalise, voxelise, n_convs x (conv + BN + leaky ReLU), devoxelise
    (trilinear, or nearest neighbour when layer.devox == "nearest").

    stage_dtype "bf16" stores the voxel grid and each convolution's output in
    bf16 (round_bf16) before the next step reads it, as a layer with bf16
    grids does; "f64" keeps every value in fp64.

    Returns a dict with every intermediate: centroid, radius, pnorm, ids, grid,
    counts, conv outputs (list, post-activation) and devox [B][N][Cout]."""
    store = _storage(stage_dtype)
    c, m, pn = normalize(coords)
    ids = voxel_ids(pn, layer.R)
    grid, counts = voxelize(ids, feats, layer.R)
    grid = store(grid)
    h = grid
    convs = []
    for w, bn in zip(layer.conv_w, layer.conv_bn):
        h = store(leaky_relu(batchnorm(conv3d(h, w, layer.R), bn), layer.slope))
        convs.append(h)
    if getattr(layer, "devox", "trilinear") == "nearest":
        dv = devoxelize_nearest(h, layer.R, ids)
    else:
        dv = devoxelize(h, layer.R, pn)
    return dict(centroid=c, radius=m, pnorm=pn, ids=ids, grid=grid, counts=counts,
                convs=convs, devox=dv)


def point_branch(feats, layer, stage_dtype="f64"):
    """Section 4.2: h = ReLU(BN(W f (+ b))). stage_dtype "bf16" rounds the
    features to bf16 before the product (the operand precision of a bf16
    layer)."""
    f = _storage(stage_dtype)(feats)
    return relu(batchnorm(linear(f, layer.mlp_w, layer.mlp_b), layer.mlp_bn))


def pvconv_forward(coords, feats, layer, return_parts=False, stage_dtype="f64"):
    """Section 4.3: the two branches fused by addition (no activation after
    it). stage_dtype as in voxel_branch and point_branch; the output itself
    is never rounded."""
    vb = voxel_branch(coords, feats, layer, stage_dtype)
    pb = point_branch(feats, layer, stage_dtype)
    out = vb["devox"] + pb
    if return_parts:
        vb["point"] = pb
        vb["out"] = out
        return vb
    return out


def layer_backward_features(coords, feats, layer, dout):
    """Gradient of one layer's output with respect to its input features
    (Sections 4.1-4.3 differentiated): the voxel branch back through the
    devoxelisation, each conv's BN + leaky and input gradient, and the
    voxelisation; the point branch back through ReLU + BN and the linear map;
    the fusion adds the two."""
    parts = pvconv_forward(coords, feats, layer, return_parts=True)
    R = layer.R
    if getattr(layer, "devox", "trilinear") == "nearest":
        g = devoxelize_nearest_backward(dout, R, parts["ids"])
    else:
        g = devoxelize_backward(dout, R, parts["pnorm"])
    for i in range(len(layer.conv_w) - 1, -1, -1):
        g = act_bn_backward(g, parts["convs"][i], layer.conv_bn[i], "leaky", layer.slope)
        g = conv3d_backward_data(g, layer.conv_w[i], R)
    dvox = voxelize_backward(g, parts["ids"], parts["counts"], R)
    dz = act_bn_backward(dout, parts["point"], layer.mlp_bn, "relu")
    dpoint = linear(dz, _f64(layer.mlp_w).T.copy())
    return dvox + dpoint


def shared_mlp(x, lp):
    """One point-only layer: Linear (+ bias), then BN and ReLU unless final."""
    y = linear(x, lp.w, lp.b)
    if lp.bn is not None:
        y = batchnorm(y, lp.bn)
    if lp.relu:
        y = relu(y)
    return y


def round_bf16(a) -> np.ndarray:
    """Each value rounded to the nearest bfloat16 (8 significant bits, fp32's
    exponent range; round to nearest, ties to even), returned as float64.

    This is the storage precision of the networks' activations ("bf16 weights
    and activations", the configuration of Section 5.1's networks used here).
    For x = m 2^e with m in [0.5, 1) the bf16 grid spacing near x is
    2^(e-8), and 2^-133 below the normal range."""
    x = _f64(a)
    _, e = np.frexp(x)
    q = np.ldexp(1.0, np.maximum(e - 8, -133))
    r = np.rint(x / q) * q          # x / q is exact: q is a power of two
    return np.where(np.isfinite(x), r, x)


def network_forward(wl, return_stages=False, stage_dtype="f64"):
    """PVCNN segmentation forward (Section 5.1 "Models": PointNet with its
    per-point MLP layers replaced by PVConv).

    Stages: the PVConv blocks, then the point-only MLPs, each feeding the next;
    a per-cloud max over the points of the last stage gives the global feature;
    the head's input is the concatenation of every stage's per-point output and
    the global feature broadcast to every point; the head is a stack of shared
    per-point layers ending in logits.

    stage_dtype "f64" keeps every value in fp64; "bf16" stores each stage's
    output and each hidden head layer's output in bf16 (round_bf16) before the
    next step reads it, as a network with bf16 activations does. The logits
    are never rounded."""
    if stage_dtype not in ("f64", "bf16"):
        raise ValueError("stage_dtype must be 'f64' or 'bf16'")
    store = round_bf16 if stage_dtype == "bf16" else (lambda v: v)
    x = wl.feats
    stages = []
    for L in wl.layers:
        x = store(pvconv_forward(wl.coords, x, L))
        stages.append(x)
    for lp in wl.mlps:
        x = store(shared_mlp(x, lp))
        stages.append(x)
    g = maxpool(x)
    B, N = wl.B, wl.N
    cat = np.concatenate(stages + [np.broadcast_to(g[:, None, :], (B, N, g.shape[1]))], axis=2)
    h = cat
    for k, lp in enumerate(wl.head):
        h = shared_mlp(h, lp)
        if k + 1 < len(wl.head):
            h = store(h)
    if return_stages:
        return h, stages, g
    return h


def pvcnn2_forward(wl, stage_dtype="f64", return_levels=False):
    """PVCNN++ segmentation forward (Section 5.2 "Models": PointNet++ extended
    with PVConv).

    Set abstraction, per level: the level's PVConv layers on its points
    (features of the same points), then npoint centres by farthest point
    sampling, the first nsample points within the radius of each centre, the
    grouped rows (relative coordinates, then features) through the shared
    MLP, and the maximum over each centre's neighbours: the next level's
    points and features. Feature propagation, from the coarsest level down:
    the coarser features interpolated onto the level's points from the three
    nearest coarser points, concatenated with the features that level's set
    abstraction consumed (its skip link), through a shared MLP. Then the
    head on the original points.

    stage_dtype "bf16" stores every step's output in bf16 (round_bf16) before
    the next step reads it, the storage of the bf16 network; the logits are
    never rounded. Returns logits [B][N][classes] (and with return_levels the
    level coordinates, the skip features and the propagated features)."""
    store = _storage(stage_dtype)
    xyz = [_f32(wl.coords)]
    x = _f64(wl.feats)
    skips = []
    for lev in wl.sa:
        for L in lev.pvconvs:
            x = store(pvconv_forward(xyz[-1], x, L, stage_dtype=stage_dtype))
        skips.append(x)
        centers = gather_points(xyz[-1], fps(xyz[-1], lev.npoint))
        nb = ball_query(xyz[-1], centers, lev.radius, lev.nsample)
        h = store(group(xyz[-1], x, centers, nb))
        for lp in lev.mlps:
            h = store(shared_mlp(h, lp))
        x = h.max(axis=2)
        xyz.append(centers)
    props = []
    for k, lev in enumerate(wl.fp):
        lvl = len(wl.sa) - 1 - k
        idx, w = three_nn(xyz[lvl], xyz[lvl + 1])
        h = np.concatenate([store(three_interpolate(x, idx, w)), skips[lvl]], axis=2)
        for lp in lev.mlps:
            h = store(shared_mlp(h, lp))
        x = h
        props.append(x)
    for k, lp in enumerate(wl.head):
        x = shared_mlp(x, lp)
        if k + 1 < len(wl.head):
            x = store(x)
    if return_levels:
        return x, dict(xyz=xyz, skips=skips, props=props)
    return x
