"""GPU parity of the backward entry points against the fp64 oracle's
gradients (pinned in tests/test_oracle_pins.py by adjoint identities, finite
differences and torch autograd). Tolerances as in tests/_helpers.py: fp32
sums within 1e-5 of (|ref| + the same sum over magnitudes); bf16 convolution
inputs as the forward convolution.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_1907_03739_amd import binding as pv
from _helpers import (assert_bf16_chain, assert_bf16_step, assert_dot_f32, assert_rel,
                      bf16_round, dev, dev_bn, host)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu_case(request):
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    print(f"\n[gpu case] {request.node.nodeid}", flush=True)
    yield
    torch.cuda.synchronize()


def _ids_counts(wl_idx, B, N, R):
    wl = synth.make_workload(wl_idx, B=B, N=N)
    _, _, pn = oracle.normalize(wl.coords)
    ids = oracle.voxel_ids(pn, R)
    counts = np.stack([np.bincount(ids[b], minlength=R ** 3) for b in range(B)]).astype(np.int32)
    return pn, ids, counts


def _i32(a):
    return torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32).cuda()


@pytest.mark.parametrize("wl_idx,B,N,R,C,gdt", [
    (2, 4, 2048, 32, 64, "bf16"), (2, 2, 2048, 32, 64, "f32"), (2, 2, 999, 24, 20, "f32"),
    (5, 1, 65536, 64, 64, "bf16"), (1, 1, 1024, 8, 3, "bf16"),
])
def test_voxelize_backward_matches_oracle(wl_idx, B, N, R, C, gdt):
    _, ids, counts = _ids_counts(wl_idx, B, N, R)
    rng = np.random.default_rng(R + C)
    dV = rng.normal(size=(B, R ** 3, C)).astype(np.float32).astype(np.float64)
    if gdt == "bf16":
        dV = bf16_round(dV)
    ref = oracle.voxelize_backward(dV, ids, counts, R)
    got = pv.pvconv_voxelize_backward(dev(dV, torch.bfloat16 if gdt == "bf16" else
                                          torch.float32), R, _i32(ids), _i32(counts))
    assert_rel(host(got), ref, 1e-6, "voxelize backward")


@pytest.mark.parametrize("wl_idx,B,N,R,C", [
    (2, 2, 2048, 32, 64), (2, 16, 2048, 32, 128), (5, 1, 65536, 64, 64), (1, 1, 1024, 8, 3),
    (4, 2, 4096, 16, 20),
])
def test_devoxelize_backward_matches_oracle(wl_idx, B, N, R, C):
    pn, ids, _ = _ids_counts(wl_idx, B, N, R)
    pn32 = pn.astype(np.float32)
    rng = np.random.default_rng(3 * R + C)
    dout = rng.normal(size=(B, N, C)).astype(np.float32).astype(np.float64)
    # trilinear: fp32 sums in the kernel's fixed order
    ref = oracle.devoxelize_backward(dout, R, pn32)
    mag = oracle.devoxelize_backward(np.abs(dout), R, pn32)
    dirty = torch.full((B, R ** 3, C), float("nan"), device="cuda")
    got = pv.pvconv_devoxelize_backward(dev(dout), R, dev(pn32), out=dirty)
    assert_dot_f32(host(got), ref, mag, "devoxelize backward")
    # nearest
    ref = oracle.devoxelize_nearest_backward(dout, R, ids)
    mag = oracle.devoxelize_nearest_backward(np.abs(dout), R, ids)
    got = pv.pvconv_devoxelize_nearest_backward(dev(dout), R, _i32(ids), out=dirty)
    assert_dot_f32(host(got), ref, mag, "nearest devoxelize backward")


DEVOX_BWD_EDGES = [
    # B, N, R, C, cloud: a one-cell grid (every corner clamped onto it), points
    # on the grid's faces and corners (both corners of an axis clamped to one
    # cell), clouds spanning several sort chunks with ragged ends, three radix
    # passes (R = 64), channel rows of 1 and 3 floats
    (2, 300, 1, 4, "uniform"),
    (3, 700, 5, 3, "faces"),
    (2, 2500, 16, 8, "uniform"),
    (1, 3000, 64, 1, "faces"),
    (4, 1025, 7, 12, "uniform"),
]


def _cloud(kind, B, N, seed):
    rng = np.random.default_rng(seed)
    pn = rng.uniform(0.0, 1.0, size=(B, N, 3))
    if kind == "faces":  # a third of the coordinates exactly on 0 or 1
        m = rng.uniform(size=pn.shape) < 0.33
        pn[m] = rng.integers(0, 2, size=int(m.sum()))
    return pn.astype(np.float32)


@pytest.mark.parametrize("B,N,R,C,kind", DEVOX_BWD_EDGES)
def test_devoxelize_backward_edges_and_repeatability(B, N, R, C, kind):
    pn = _cloud(kind, B, N, N + R)
    ids = np.clip(np.floor(pn.astype(np.float64) * R), 0, R - 1).astype(np.int64)
    ids = ((ids[..., 0] * R + ids[..., 1]) * R + ids[..., 2]).astype(np.int32)
    dout = np.random.default_rng(C).normal(size=(B, N, C)).astype(np.float32)
    ws = torch.empty(pv._lib.pvconv_devoxelize_backward_workspace_size(B, N, C, R),
                     dtype=torch.uint8, device="cuda")
    for nearest in (False, True):
        call = (lambda w: pv.pvconv_devoxelize_nearest_backward(dev(dout), R, _i32(ids),
                                                                workspace=w)) if nearest else \
               (lambda w: pv.pvconv_devoxelize_backward(dev(dout), R, dev(pn), workspace=w))
        ws.fill_(0x5A)
        first = call(ws)
        ws.fill_(0xA7)  # the result does not depend on what the workspace held
        again = call(ws)
        assert torch.equal(first, again), "devoxelize backward is not repeatable"
        d64 = dout.astype(np.float64)
        ref = (oracle.devoxelize_nearest_backward(d64, R, ids) if nearest
               else oracle.devoxelize_backward(d64, R, pn))
        mag = (oracle.devoxelize_nearest_backward(np.abs(d64), R, ids) if nearest
               else oracle.devoxelize_backward(np.abs(d64), R, pn))
        assert_dot_f32(host(first), ref, mag, f"devoxelize backward (nearest={nearest})")


def test_devoxelize_backward_unaligned_rows_and_no_points():
    B, N, R, C = 2, 400, 6, 8
    pn = _cloud("uniform", B, N, 5)
    dout = np.random.default_rng(6).normal(size=(B, N, C)).astype(np.float32)
    # rows that start 4 bytes past a 16-byte boundary take the channel-by-channel items
    buf = torch.zeros(B * N * C + 1, dtype=torch.float32, device="cuda")
    shifted = buf[1:].view(B, N, C)
    shifted.copy_(dev(dout))
    got = pv.pvconv_devoxelize_backward(shifted, R, dev(pn))
    d64 = dout.astype(np.float64)
    assert_dot_f32(host(got), oracle.devoxelize_backward(d64, R, pn),
                   oracle.devoxelize_backward(np.abs(d64), R, pn), "unaligned rows")
    assert torch.equal(got, pv.pvconv_devoxelize_backward(dev(dout), R, dev(pn)))
    # no points: the whole gradient grid is zero
    dirty = torch.full((B, R ** 3, C), float("nan"), device="cuda")
    empty = pv.pvconv_devoxelize_backward(torch.zeros((B, 0, C), device="cuda"), R,
                                          torch.zeros((B, 0, 3), device="cuda"), out=dirty)
    assert torch.count_nonzero(empty).item() == 0 and not torch.isnan(empty).any()


@pytest.mark.parametrize("B,R,Cin,Cout,dt", [
    (2, 32, 64, 128, "bf16"),      # the part-seg layer's first conv, input gradient
    (1, 16, 128, 128, "bf16"),
    (1, 13, 32, 64, "bf16"),       # ragged bricks
    (2, 8, 16, 32, "f32"),
    (1, 9, 5, 7, "f32"),           # fp32 path, odd channel counts
])
def test_conv3d_backward_data_matches_oracle(B, R, Cin, Cout, dt):
    rng = np.random.default_rng(R * 5 + Cin)
    dy = rng.normal(size=(B, R ** 3, Cout)) * (rng.random((B, R ** 3, 1)) < 0.4)
    w = synth.kaiming_normal(rng, (Cout, 3, 3, 3, Cin), 27 * Cin, bf16=dt == "bf16")
    if dt == "bf16":
        dy = bf16_round(dy)
    else:
        dy = dy.astype(np.float32).astype(np.float64)
        w = w.astype(np.float32).astype(np.float64)
    ref = oracle.conv3d_backward_data(dy, w, R)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    got = host(pv.pvconv_conv3d_backward_data(dev(dy, tdt), dev(w, tdt), R))
    if dt == "bf16":
        # fp32 accumulation of exact bf16 products: the forward conv's bound
        assert_bf16_step(got, ref, "conv input gradient bf16")
    else:
        mag = oracle.conv3d_backward_data(np.abs(dy), np.abs(w), R)
        assert_dot_f32(got, ref, mag, "conv input gradient fp32")


def test_conv3d_backward_data_is_the_adjoint_of_the_forward_on_gpu():
    # <dy, conv(x)> = <conv_bwd(dy), x> with both sides from the GPU kernels
    rng = np.random.default_rng(11)
    R, Cin, Cout = 16, 64, 64
    x = bf16_round(rng.normal(size=(1, R ** 3, Cin)))
    dy = bf16_round(rng.normal(size=(1, R ** 3, Cout)))
    w = synth.kaiming_normal(rng, (Cout, 3, 3, 3, Cin), 27 * Cin, bf16=True)
    y = host(pv.pvconv_conv3d(dev(x, torch.bfloat16), dev(w, torch.bfloat16), R, act="none",
                              out_dtype=torch.float32))
    dx = host(pv.pvconv_conv3d_backward_data(dev(dy, torch.bfloat16), dev(w, torch.bfloat16),
                                             R))
    lhs, rhs = float(np.sum(dy * y)), float(np.sum(dx * x))
    scale = max(float(np.sum(np.abs(dy * y))), float(np.sum(np.abs(dx * x))))
    assert abs(lhs - rhs) <= 1e-5 * scale, (lhs, rhs, scale)


@pytest.mark.parametrize("B,R,Cin,Cout", [
    (2, 32, 64, 128),    # the part-seg layer's first conv (batch reduced)
    (1, 16, 128, 128),
    (1, 13, 32, 64),     # ragged bricks
    (3, 8, 16, 64),      # one brick per cloud
    (1, 9, 48, 64),      # 16-channel chunks (48 is no multiple of 32), ragged bricks
    (1, 1, 16, 64),      # a single voxel: only the centre tap sees data
])
def test_conv3d_backward_weight_matches_oracle(B, R, Cin, Cout):
    rng = np.random.default_rng(R * 3 + Cin + Cout)
    dy = bf16_round(rng.normal(size=(B, R ** 3, Cout)) * (rng.random((B, R ** 3, 1)) < 0.5))
    x = bf16_round(rng.normal(size=(B, R ** 3, Cin)) * (rng.random((B, R ** 3, 1)) < 0.3))
    ref = oracle.conv3d_backward_weight(dy, x, R)
    mag = oracle.conv3d_backward_weight(np.abs(dy), np.abs(x), R)
    got = host(pv.pvconv_conv3d_backward_weight(dev(dy, torch.bfloat16), dev(x, torch.bfloat16),
                                                R))
    assert_dot_f32(got, ref, mag, "conv weight gradient")


def test_conv3d_backward_weight_is_deterministic_and_the_adjoint_on_gpu():
    # <dW, W> = <dy, conv(x, W)> with both sides from the GPU kernels
    rng = np.random.default_rng(12)
    R, Cin, Cout = 16, 32, 64
    x = bf16_round(rng.normal(size=(2, R ** 3, Cin)))
    dy = bf16_round(rng.normal(size=(2, R ** 3, Cout)))
    w = synth.kaiming_normal(rng, (Cout, 3, 3, 3, Cin), 27 * Cin, bf16=True)
    dyd, xd = dev(dy, torch.bfloat16), dev(x, torch.bfloat16)
    dw1 = host(pv.pvconv_conv3d_backward_weight(dyd, xd, R))
    dw2 = host(pv.pvconv_conv3d_backward_weight(dyd, xd, R))
    assert np.array_equal(dw1, dw2)
    y = host(pv.pvconv_conv3d(xd, dev(w, torch.bfloat16), R, act="none",
                              out_dtype=torch.float32))
    lhs, rhs = float(np.sum(dy * y)), float(np.sum(dw1 * w))
    scale = max(float(np.sum(np.abs(dy * y))), float(np.sum(np.abs(dw1 * w))))
    assert abs(lhs - rhs) <= 1e-5 * scale, (lhs, rhs, scale)


@pytest.mark.parametrize("ydt,act,with_bn,M,C", [
    ("f32", "leaky", True, 20000, 96), ("bf16", "leaky", True, 20000, 96),
    ("f32", "relu", True, 20000, 96), ("bf16", "none", False, 20000, 96),
    ("f32", "leaky", False, 20000, 96),
    # a channel count that is no multiple of 4 (element by element); more
    # channels than the per-channel scale table holds (scales per element)
    ("bf16", "leaky", True, 3001, 13), ("f32", "leaky", True, 40, 16500),
    ("bf16", "relu", True, 7, 16387),
])
def test_act_bn_backward_matches_oracle(ydt, act, with_bn, M, C):
    rng = np.random.default_rng(5)
    bn = synth.draw_bn(rng, C) if with_bn else None
    y = rng.normal(size=(M, C)).astype(np.float32).astype(np.float64)
    if ydt == "bf16":
        y = bf16_round(y)
    dy = rng.normal(size=(M, C)).astype(np.float32).astype(np.float64)
    ref = oracle.act_bn_backward(dy, y, bn, act, 0.1)
    got = pv.pvconv_act_bn_backward(dev(dy), dev(y, torch.bfloat16 if ydt == "bf16" else
                                                 torch.float32),
                                    bn=dev_bn(bn) if bn is not None else None, act=act,
                                    slope=0.1)
    assert_rel(host(got), ref, 1e-5, "act + BN backward")


@pytest.mark.parametrize("wl_idx,B,devox", [(1, 1, "trilinear"), (2, 2, "trilinear"),
                                            (2, 2, "nearest")])
def test_layer_feature_gradient_composed_from_the_entry_points(wl_idx, B, devox):
    # The whole layer's input-feature gradient from the backward entry points
    # (and the point MLP with the transposed weight). The reference chains the
    # oracle's backward steps (pinned one by one, and their composition by
    # finite differences) through the same forward state: the rectifiers'
    # derivatives are read from the GPU's own activations, since an
    # activation within rounding of zero may take either side, and the
    # gradients are rounded to bf16 where the GPU chain stores them in bf16.
    import dataclasses
    wl = synth.make_workload(wl_idx, B=B)
    L = dataclasses.replace(wl.layers[0], devox=devox)
    bf = wl.dtype == "bf16"
    cdt = torch.bfloat16 if bf else torch.float32
    rnd = bf16_round if bf else (lambda a: a.astype(np.float32).astype(np.float64))
    R = L.R
    rng = np.random.default_rng(9)
    dout = rng.normal(size=(B, wl.N, L.cout)).astype(np.float32).astype(np.float64)

    layer = pv.DeviceLayer(L, "cuda", cdt)
    feats = dev(wl.feats)
    grid, counts, ids, pn = pv.pvconv_voxelize(dev(wl.coords), feats, R, grid_dtype=cdt)
    ys, h = [], grid
    for i in range(L.n_convs):
        h = pv.pvconv_conv3d(h, layer.conv_w[i], R, bn=layer.conv_bn[i], act="leaky",
                             slope=L.slope)
        ys.append(h)
    hp = pv.pvconv_point_mlp(feats, layer.mlp_w, bias=layer.mlp_b, bn=layer.mlp_bn, act="relu")
    d = dev(dout)
    g = (pv.pvconv_devoxelize_nearest_backward(d, R, ids) if devox == "nearest"
         else pv.pvconv_devoxelize_backward(d, R, pn))
    for i in range(L.n_convs - 1, -1, -1):
        g = pv.pvconv_act_bn_backward(g, ys[i], bn=layer.conv_bn[i], act="leaky", slope=L.slope)
        g = pv.pvconv_conv3d_backward_data(g.to(cdt), layer.conv_w[i], R)
    dvox = pv.pvconv_voxelize_backward(g.to(cdt), R, ids, counts)
    dz = pv.pvconv_act_bn_backward(d, hp, bn=layer.mlp_bn, act="relu")
    wT = torch.as_tensor(L.mlp_w, dtype=torch.float32).t().contiguous().cuda()
    dpoint = pv.pvconv_point_mlp(dz, wT, act="none")
    got = host(dvox) + host(dpoint)

    ids_h, counts_h = ids.cpu().numpy(), counts.cpu().numpy()
    r = (oracle.devoxelize_nearest_backward(dout, R, ids_h) if devox == "nearest"
         else oracle.devoxelize_backward(dout, R, host(pn)))
    for i in range(L.n_convs - 1, -1, -1):
        r = oracle.act_bn_backward(r, host(ys[i]), L.conv_bn[i], "leaky", L.slope)
        r = oracle.conv3d_backward_data(rnd(r), L.conv_w[i], R)
    ref = oracle.voxelize_backward(rnd(r), ids_h, counts_h, R)
    ref = ref + oracle.linear(oracle.act_bn_backward(dout, host(hp), L.mlp_bn, "relu"),
                              np.ascontiguousarray(np.asarray(L.mlp_w, np.float64).T))
    # a sum over chains of bf16-stored gradients: the chain bound of the
    # forward layer tests (relative to |ref| + its rms)
    assert_bf16_chain(got, ref, f"layer feature gradient ({devox})")
