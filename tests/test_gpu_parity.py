"""GPU parity: every C-ABI entry point against the fp64 CPU oracle on the same
seeded inputs. Tolerances are explained in tests/_helpers.py.

Sizes: the workloads' own shapes with the batch reduced so that the oracle
finishes in seconds (they still span many tiles and a ragged tail), the full
part-segmentation and stress sizes where the oracle is cheap (voxelisation,
the whole stress layer), and sampled outputs at full size where it is not
(the part-segmentation convolutions and layer).
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import synth
from paper_1907_03739_amd import binding as pv
from _helpers import (assert_bf16_chain, assert_bf16_step, assert_dot_f32, assert_rel,
                      bf16_round, bn_scale, dev, dev_bn, host)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu_case(request):
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    print(f"\n[gpu case] {request.node.nodeid}", flush=True)
    yield
    torch.cuda.synchronize()


def test_device_is_gfx950():
    assert "gfx950" in torch.cuda.get_device_properties(0).gcnArchName


# ----------------------------------------------------------------------------
# voxelisation
# ----------------------------------------------------------------------------
def _cloud(wl_idx, B, N, C, seed=0, feat_scale=1.0):
    wl = synth.make_workload(wl_idx, B=B, N=N)
    f = np.random.default_rng(seed).normal(size=(B, N, C)).astype(np.float32) * feat_scale
    return wl.coords, f


def _oracle_vox(coords, feats, R):
    _, _, pn = oracle.normalize(coords)
    ids = oracle.voxel_ids(pn, R)
    grid, counts = oracle.voxelize(ids, feats, R)
    return pn, ids, grid, counts


VOX_CASES = [
    # workload, B, N, R, C, feat dtype, grid dtype
    (1, 1, 1024, 8, 16, "f32", "f32"),        # single-layer fp32 shape
    (2, 2, 2048, 32, 64, "f32", "f32"),       # part-seg shape, fused path
    (2, 2, 2048, 32, 64, "f32", "bf16"),
    (2, 16, 2048, 32, 64, "f32", "bf16"),     # part-seg full size
    (3, 2, 2048, 32, 3, "f32", "bf16"),       # 3 channels: element-wise path
    (4, 2, 4096, 16, 9, "f32", "bf16"),       # scene-seg shape, 9 channels
    (5, 1, 65536, 64, 64, "f32", "bf16"),     # stress size: split path, 8 partitions
    (2, 1, 20000, 32, 64, "f32", "f32"),      # split path with a single partition
    (2, 2, 2048, 24, 32, "bf16", "f32"),      # R not a power of two, bf16 features
    (1, 3, 1000, 1, 8, "f32", "f32"),         # R = 1: one voxel holds every point
]


@pytest.mark.parametrize("case", VOX_CASES, ids=lambda c: "wl{}_B{}_N{}_R{}_C{}_{}_{}".format(*c))
def test_voxelize_matches_oracle(case):
    wl_idx, B, N, R, C, fdt, gdt = case
    coords, feats = _cloud(wl_idx, B, N, C)
    if fdt == "bf16":
        feats = synth.round_to_bf16(feats)
    pn, ids, grid, counts = _oracle_vox(coords, feats, R)
    g, c, i, p = pv.pvconv_voxelize(dev(coords), dev(feats, getattr(torch, "bfloat16" if fdt ==
                                    "bf16" else "float32")), R,
                                    grid_dtype=torch.bfloat16 if gdt == "bf16" else torch.float32)
    assert np.array_equal(i.cpu().numpy(), ids)
    assert np.array_equal(c.cpu().numpy(), counts)
    assert np.array_equal(p.cpu().numpy(), pn.astype(np.float32))
    if gdt == "f32":
        assert_rel(host(g), grid, 1e-5, "voxel grid fp32")
    else:
        assert_bf16_step(host(g), grid, "voxel grid bf16")


@pytest.mark.parametrize("wl_idx,B,N,R,C,gdt", [
    (2, 4, 2048, 32, 64, "bf16"),    # small clouds, 16-byte rows
    (2, 2, 2048, 16, 20, "f32"),     # small clouds, grid zeroed first
    (5, 1, 65536, 64, 64, "bf16"),   # large cloud: tile counts and buckets from the indices
    (5, 1, 65536, 32, 20, "f32"),    # large cloud, grid zeroed first
])
def test_voxelize_from_given_ids(wl_idx, B, N, R, C, gdt):
    # Eq. 2 with the indices of an earlier call (the cross-layer reuse of the
    # normalisation): the same grid and counts, over a grid left dirty
    coords, feats = _cloud(wl_idx, B, N, C, seed=7)
    gt = torch.bfloat16 if gdt == "bf16" else torch.float32
    pn, ids, grid, counts = _oracle_vox(coords, feats, R)
    ids_d = torch.as_tensor(ids, dtype=torch.int32).cuda()
    g0 = torch.full((B, R ** 3, C), float("nan"), dtype=gt, device="cuda")
    c0 = torch.full((B, R ** 3), -7, dtype=torch.int32, device="cuda")
    g, c = pv.pvconv_voxelize_from_ids(ids_d, dev(feats), R, grid_dtype=gt, grid=g0, counts=c0)
    assert np.array_equal(c.cpu().numpy(), counts)
    if gdt == "f32":
        assert_rel(host(g), grid, 1e-5, "voxel grid fp32, given ids")
    else:
        assert_bf16_step(host(g), grid, "voxel grid bf16, given ids")
    # indices outside the grid drop their points (invalid input, memory-safe)
    bad = ids.copy()
    bad[:, ::97] = -1
    bad[:, 1::89] = R ** 3 + 5
    keep = (bad >= 0) & (bad < R ** 3)
    gk, ck = pv.pvconv_voxelize_from_ids(torch.as_tensor(bad, dtype=torch.int32).cuda(),
                                         dev(feats), R, grid_dtype=gt)
    for b in range(B):
        gb, cb = oracle.voxelize(ids[b:b + 1, keep[b]], feats[b:b + 1, keep[b]], R)
        assert np.array_equal(ck.cpu().numpy()[b], cb[0])
        if gdt == "f32":
            assert_rel(host(gk)[b], gb[0], 1e-5, "dropped indices")
        else:
            assert_bf16_step(host(gk)[b], gb[0], "dropped indices")


def test_forward_reusing_the_indices_of_an_earlier_layer():
    wl = synth.make_workload(2, B=2)
    L = wl.layers[0]
    layer = pv.DeviceLayer(L, "cuda", torch.bfloat16)
    coords, feats = dev(wl.coords), dev(wl.feats)
    ids = torch.empty((2, wl.N), dtype=torch.int32, device="cuda")
    norm = torch.empty((2, wl.N, 3), dtype=torch.float32, device="cuda")
    first = host(pv.pvconv_forward(coords, feats, layer, vox_id=ids, norm=norm))
    _, _, pn = oracle.normalize(wl.coords)
    assert np.array_equal(ids.cpu().numpy(), oracle.voxel_ids(pn, L.R))
    assert np.array_equal(norm.cpu().numpy(), pn.astype(np.float32))
    again = host(pv.pvconv_forward(None, feats, layer, vox_id=ids, norm=norm, ids_given=True))
    np.testing.assert_allclose(again, first, rtol=1e-6, atol=1e-6)
    ref = oracle.pvconv_forward(wl.coords, wl.feats, L)
    assert_bf16_chain(again, ref, "layer from given indices")


def test_voxelize_strided_features_and_optional_outputs():
    coords, wide = _cloud(2, 2, 2048, 96)
    feats = wide[:, :, 16:80]
    pn, ids, grid, counts = _oracle_vox(coords, feats, 32)
    wide_d = dev(wide)
    g, c, i, p = pv.pvconv_voxelize(dev(coords), wide_d[:, :, 16:80], 32, want_ids=False,
                                    want_norm=False)
    assert i is None and p is None
    assert np.array_equal(c.cpu().numpy(), counts)
    assert_rel(host(g), grid, 1e-5)


def test_voxelize_single_point_and_coincident_clouds():
    rng = np.random.default_rng(3)
    for N in (1, 37):
        coords = np.repeat(rng.normal(size=(4, 1, 3)).astype(np.float32), N, axis=1)
        feats = rng.normal(size=(4, N, 8)).astype(np.float32)
        pn, ids, grid, counts = _oracle_vox(coords, feats, 8)
        g, c, i, p = pv.pvconv_voxelize(dev(coords), dev(feats), 8)
        assert np.all(i.cpu().numpy() == (4 * 8 + 4) * 8 + 4)
        assert np.array_equal(c.cpu().numpy(), counts)
        assert np.all(p.cpu().numpy() == 0.5)
        assert_rel(host(g), grid, 1e-5)


@pytest.mark.parametrize("N,spread", [(60000, 1.0), (9000, 0.0), (40000, 0.02)],
                         ids=["tile_overflow", "one_voxel_beyond_capacity", "dense_cluster"])
def test_voxelize_crowded_tiles(N, spread):
    # More points in one tile than the LDS keeps (segmented path), every point
    # in one voxel (whole-workgroup path), and one tight cluster (heavy voxels).
    rng = np.random.default_rng(N)
    R = 8
    coords = (rng.uniform(-1, 1, size=(1, N, 3)) * spread).astype(np.float32)
    coords[0, 0] = [1.0, 1.0, 1.0]   # fixes the radius so the cluster stays central
    coords[0, 1] = [-1.0, -1.0, -1.0]
    feats = rng.normal(size=(1, N, 16)).astype(np.float32)
    pn, ids, grid, counts = _oracle_vox(coords, feats, R)
    g, c, i, p = pv.pvconv_voxelize(dev(coords), dev(feats), R)
    assert np.array_equal(i.cpu().numpy(), ids)
    assert np.array_equal(c.cpu().numpy(), counts)
    assert_rel(host(g), grid, 1e-5, "crowded voxel grid")


@pytest.mark.parametrize("C,fdt,gdt", [(128, "bf16", torch.bfloat16), (24, "f32", torch.float32),
                                       (136, "f32", torch.bfloat16)],
                         ids=["C128_bf16", "C24_f32", "C136_wider_than_the_queue_sums"])
def test_voxelize_clustered_large_clouds(C, fdt, gdt):
    # Large clouds whose dense voxels (more than 32 points) are handed to the
    # heavy-voxel kernels in chunks of 256 points (up to 128 channels), or
    # summed in their tile (wider rows); two clouds, a voxel of ~3000 points.
    rng = np.random.default_rng(C)
    B, N, R = 2, 12000, 16
    centers = rng.uniform(-0.6, 0.6, size=(B, 6, 1, 3))
    pts = centers + rng.normal(size=(B, 6, N // 6, 3)) * rng.uniform(0.005, 0.05, size=(B, 6, 1, 1))
    coords = pts.reshape(B, N, 3).astype(np.float32)
    coords[:, :3000] = coords[:, :1]          # one voxel of 3000 points per cloud
    coords[:, -1] = [1.5, 1.5, 1.5]           # spread the grid
    feats = rng.normal(size=(B, N, C)).astype(np.float32)
    if fdt == "bf16":
        feats = synth.round_to_bf16(feats)
    pn, ids, grid, counts = _oracle_vox(coords, feats, R)
    assert counts.max() >= 3000
    g = torch.full((B, R ** 3, C), float("nan"), dtype=gdt, device="cuda")
    g, c, i, p = pv.pvconv_voxelize(dev(coords), dev(feats, torch.bfloat16 if fdt == "bf16" else
                                                      torch.float32), R, grid_dtype=gdt, grid=g)
    assert np.array_equal(i.cpu().numpy(), ids)
    assert np.array_equal(c.cpu().numpy(), counts)
    got = host(g)
    if gdt == torch.float32:
        assert_rel(got, grid, 1e-5, "clustered grid fp32")
    else:
        assert_bf16_step(got, grid, "clustered grid bf16")


@pytest.mark.parametrize("N,R,C,gdt", [(2048, 32, 64, torch.bfloat16), (3000, 7, 16, torch.float32),
                                        (20000, 31, 32, torch.bfloat16), (1, 5, 8, torch.float32)],
                         ids=["vec_rows", "odd_R", "split_path", "one_point"])
def test_voxelize_writes_every_row_of_a_dirty_grid(N, R, C, gdt):
    # Every grid row is written by the kernels (empty rows as zeros by the
    # tile kernel, or by the normalisation launch for rows that are not
    # 16-byte vectors): with the grid filled with NaN beforehand every row
    # must come out right. Half the points lie on a sphere, so after
    # normalisation they sit on the ball's surface (the cells on the grid's
    # edge), the other half inside it.
    rng = np.random.default_rng(N + R)
    B = 2
    d = rng.normal(size=(B, N, 3))
    d /= np.linalg.norm(d, axis=2, keepdims=True)
    d[:, N // 2:] *= rng.uniform(0, 1, size=(B, N - N // 2, 1))
    coords = (d * 3.0 + rng.normal(size=(B, 1, 3))).astype(np.float32)
    feats = rng.normal(size=(B, N, C)).astype(np.float32)
    if gdt == torch.bfloat16:
        feats = synth.round_to_bf16(feats)
    pn, ids, grid, counts = _oracle_vox(coords, feats, R)
    g = torch.full((B, R ** 3, C), float("nan"), dtype=gdt, device="cuda")
    cnt = torch.full((B, R ** 3), -7, dtype=torch.int32, device="cuda")
    g, c, i, p = pv.pvconv_voxelize(dev(coords), dev(feats), R, grid_dtype=gdt, grid=g, counts=cnt)
    assert np.array_equal(i.cpu().numpy(), ids)
    assert np.array_equal(c.cpu().numpy(), counts)
    got = host(g)
    assert not np.isnan(got).any()
    assert np.all(got[counts == 0] == 0)
    if gdt == torch.float32:
        assert_rel(got, grid, 1e-5, "voxel grid fp32")
    else:
        assert_bf16_step(got, grid, "voxel grid bf16")


def test_voxelize_empty_clouds_give_zero_grids():
    coords = torch.empty((2, 0, 3), device="cuda")
    feats = torch.empty((2, 0, 16), device="cuda")
    g, c, i, p = pv.pvconv_voxelize(coords, feats, 8)
    assert g.shape == (2, 512, 16) and torch.all(g == 0) and torch.all(c == 0)
    g, c, _, _ = pv.pvconv_voxelize(torch.empty((0, 5, 3), device="cuda"),
                                    torch.empty((0, 5, 16), device="cuda"), 8)
    assert g.numel() == 0


@pytest.mark.parametrize("wl_idx,B,N,R,C", [(2, 4, 2048, 32, 64), (4, 2, 4096, 16, 64),
                                         (1, 1, 1024, 8, 16), (3, 2, 2048, 16, 24)],
                         ids=["partseg", "scene_R16", "fp32_layer", "C24"])
def test_voxelize_small_clouds_sum_in_point_order(wl_idx, B, N, R, C):
    # Clouds of up to 4096 points: within a voxel of up to 16 points the
    # features are summed in point order from zero in fp64, as the oracle
    # sums them, so those rows equal the oracle's, rounded to fp32, bit for
    # bit; heavier voxels (subset sums added in a fixed order) are within
    # the fp32 bound. Two runs give the same bits.
    coords, feats = _cloud(wl_idx, B, N, C, seed=11)
    pn, ids, grid, counts = _oracle_vox(coords, feats, R)
    g1, c1, i1, p1 = pv.pvconv_voxelize(dev(coords), dev(feats), R, grid_dtype=torch.float32)
    g2, c2, i2, p2 = pv.pvconv_voxelize(dev(coords), dev(feats), R, grid_dtype=torch.float32)
    assert torch.equal(g1, g2) and torch.equal(c1, c2) and torch.equal(i1, i2)
    assert np.array_equal(c1.cpu().numpy(), counts)
    got = g1.cpu().numpy()
    light = (counts >= 1) & (counts <= 16)
    assert light.sum() > 0
    assert np.array_equal(got[light], grid[light].astype(np.float32))
    assert_rel(got, grid, 1e-5, "small-cloud grid fp32")
    # bf16 grids: the same fp32 means, rounded once more
    gb, _, _, _ = pv.pvconv_voxelize(dev(coords), dev(feats), R, grid_dtype=torch.bfloat16)
    want = torch.as_tensor(grid[light].astype(np.float32)).to(torch.bfloat16)
    assert torch.equal(gb.cpu()[torch.as_tensor(light)], want)


def test_voxelize_dense_slabs_past_the_stage():
    # Sixteen clouds of 2048 points at R = 32 give slabs of 2048 voxels. A
    # slab's LDS stage holds 384 rows of 64 fp32 channels; cloud 0 packs
    # ~460 points into one slab (the rest of its rows are staged after the
    # sort in the sort's tables, up to 492), cloud 1 ~720 (beyond that:
    # segments). Both must give the oracle's grid, light voxels bit for bit.
    rng = np.random.default_rng(21)
    B, N, R, C = 16, 2048, 32, 64
    coords = rng.uniform(-1, 1, (B, N, 3)).astype(np.float32)
    for b, k in ((0, 280), (1, 560)):  # a thin layer across x: one or two u-slices
        coords[b, :k, 0] = rng.uniform(0.30, 0.32, k).astype(np.float32)
    feats = rng.normal(size=(B, N, C)).astype(np.float32)
    pn, ids, grid, counts = _oracle_vox(coords, feats, R)
    dense = [int(np.bincount(ids[b] // 2048, minlength=16).max()) for b in range(3)]
    assert 384 < dense[0] <= 492 < dense[1] and dense[2] <= 384, dense
    g1, c1, _, _ = pv.pvconv_voxelize(dev(coords), dev(feats), R, grid_dtype=torch.float32)
    g2, c2, _, _ = pv.pvconv_voxelize(dev(coords), dev(feats), R, grid_dtype=torch.float32)
    assert torch.equal(g1, g2) and torch.equal(c1, c2)
    assert np.array_equal(c1.cpu().numpy(), counts)
    got = g1.cpu().numpy()
    light = (counts >= 1) & (counts <= 16)
    assert np.array_equal(got[light], grid[light].astype(np.float32))
    assert_rel(got, grid, 1e-5, "dense-slab grid fp32")


def test_voxelize_is_deterministic_and_permutation_equivariant():
    coords, feats = _cloud(5, 1, 65536, 64)
    g1, c1, i1, p1 = pv.pvconv_voxelize(dev(coords), dev(feats), 64)
    g2, c2, i2, p2 = pv.pvconv_voxelize(dev(coords), dev(feats), 64)
    assert torch.equal(i1, i2) and torch.equal(c1, c2) and torch.equal(g1, g2)
    perm = np.random.default_rng(4).permutation(65536)
    g3, c3, i3, p3 = pv.pvconv_voxelize(dev(coords[:, perm]), dev(feats[:, perm]), 64)
    assert np.array_equal(i3.cpu().numpy(), i1.cpu().numpy()[:, perm])
    assert torch.equal(c3, c1)
    assert_rel(host(g3), host(g1), 1e-6, "permuted grid")


# ----------------------------------------------------------------------------
# convolution
# ----------------------------------------------------------------------------
def _sparse_grid(rng, B, R, C, occupied=0.3):
    x = rng.normal(size=(B, R ** 3, C))
    x *= rng.random(size=(B, R ** 3, 1)) < occupied
    return bf16_round(x)


def _oracle_conv(x, w, bn, R, act="leaky", slope=0.1):
    y = oracle.batchnorm(oracle.conv3d(x, w, R), bn)
    return oracle.leaky_relu(y, slope) if act == "leaky" else oracle.relu(y)


CONV_CASES = [
    # B, R, Cin, Cout, out dtype
    (2, 32, 64, 128, "bf16"),      # part-seg conv 1 (batch reduced)
    (1, 32, 128, 128, "bf16"),     # part-seg conv 2
    (1, 64, 64, 64, "bf16"),       # stress conv
    (2, 16, 128, 128, "bf16"),     # R=16 blocks
    (2, 32, 3, 64, "bf16"),        # 3 input channels (element-wise loads)
    (2, 32, 9, 64, "f32"),         # 9 input channels, fp32 out
    (1, 13, 32, 32, "bf16"),       # ragged R, 32-channel tiles
    (1, 7, 40, 96, "f32"),         # Cin not a multiple of 32, Cout = 3 x 32
    (3, 1, 16, 64, "bf16"),        # R = 1
    (2, 32, 8, 16, "bf16"),        # 0.125 x C: 16 output channels, half a tile
    (2, 16, 8, 8, "bf16"),         # 8 output channels
    (1, 8, 16, 12, "bf16"),        # 12 channels: rows of 24 bytes, element stores
    (1, 13, 24, 40, "f32"),        # a second tile of 8 channels
]


@pytest.mark.parametrize("case", CONV_CASES, ids=lambda c: "B{}_R{}_{}to{}_{}".format(*c))
def test_conv3d_bf16_matches_oracle(case):
    B, R, Cin, Cout, odt = case
    rng = np.random.default_rng(R * 1000 + Cin)
    x = _sparse_grid(rng, B, R, Cin)
    w = synth.kaiming_normal(rng, (Cout, 3, 3, 3, Cin), 27 * Cin, bf16=True)
    bn = synth.draw_bn(rng, Cout)
    ref = _oracle_conv(x, w, bn, R)
    y = pv.pvconv_conv3d(dev(x, torch.bfloat16), dev(w, torch.bfloat16), R, bn=dev_bn(bn),
                         out_dtype=torch.bfloat16 if odt == "bf16" else torch.float32)
    assert_bf16_step(host(y), ref, f"conv {case}")


@pytest.mark.parametrize("case", CONV_CASES[:5], ids=lambda c: "B{}_R{}_{}to{}_{}".format(*c))
def test_conv3d_packed_weights_give_the_same_bits(case):
    # packing once and convolving on the packed copy is the same computation
    # as the one-call convolution, which packs internally
    B, R, Cin, Cout, odt = case
    rng = np.random.default_rng(R * 1000 + Cin + 1)
    x = dev(_sparse_grid(rng, B, R, Cin), torch.bfloat16)
    w = dev(synth.kaiming_normal(rng, (Cout, 3, 3, 3, Cin), 27 * Cin, bf16=True), torch.bfloat16)
    bn = dev_bn(synth.draw_bn(rng, Cout))
    odt = torch.bfloat16 if odt == "bf16" else torch.float32
    ref = pv.pvconv_conv3d(x, w, R, bn=bn, out_dtype=odt)
    packed = pv.pvconv_conv3d_pack_weights(w)
    got = pv.pvconv_conv3d_packed(x, packed, Cout, R, bn=bn, out_dtype=odt)
    assert torch.equal(ref, got)
    # a second convolution on the same packed copy
    assert torch.equal(ref, pv.pvconv_conv3d_packed(x, packed, Cout, R, bn=bn, out_dtype=odt))


def test_conv3d_bias_and_activations():
    rng = np.random.default_rng(7)
    B, R, Cin, Cout = 1, 16, 32, 64
    x = _sparse_grid(rng, B, R, Cin)
    w = synth.kaiming_normal(rng, (Cout, 3, 3, 3, Cin), 27 * Cin, bf16=True)
    bias = rng.normal(size=Cout).astype(np.float32)
    raw = oracle.conv3d(x, w, R) + bias
    y = pv.pvconv_conv3d(dev(x, torch.bfloat16), dev(w, torch.bfloat16), R, bias=dev(bias),
                         act="none", out_dtype=torch.float32)
    assert_bf16_step(host(y), raw, "conv + bias, no BN, no activation")
    y = pv.pvconv_conv3d(dev(x, torch.bfloat16), dev(w, torch.bfloat16), R, bias=dev(bias),
                         act="relu", out_dtype=torch.float32)
    assert_bf16_step(host(y), oracle.relu(raw), "conv + bias + ReLU")


@pytest.mark.parametrize("B,R,Cin,Cout", [(1, 8, 16, 32), (2, 9, 5, 7), (1, 1, 3, 4)])
def test_conv3d_f32_matches_oracle(B, R, Cin, Cout):
    rng = np.random.default_rng(R + Cin)
    x = rng.normal(size=(B, R ** 3, Cin)).astype(np.float32).astype(np.float64)
    w = synth.kaiming_normal(rng, (Cout, 3, 3, 3, Cin), 27 * Cin, bf16=False)
    bn = synth.draw_bn(rng, Cout)
    ref = _oracle_conv(x, w, bn, R)
    mag = oracle.conv3d(np.abs(x), np.abs(w), R) * bn_scale(bn) + np.abs(
        bn.mean * bn_scale(bn)) + np.abs(bn.beta)
    y = pv.pvconv_conv3d(dev(x), dev(w), R, bn=dev_bn(bn), out_dtype=torch.float32)
    assert_dot_f32(host(y), ref, mag, "conv fp32")


@pytest.mark.parametrize("B,R,Cin,Cout,odt", [
    (16, 32, 64, 128, "bf16"),    # part-seg conv 1: 64-channel tiles, two workgroups per CU
    (16, 32, 128, 128, "bf16"),   # part-seg conv 2: 64-channel tiles, two workgroups per CU
    (4, 32, 192, 128, "bf16"),    # wide input: 128-channel tiles, four waves, double-buffered
    (4, 32, 128, 64, "bf16"),     # 64-channel tiles, four waves
    (8, 32, 9, 64, "bf16"),       # scene-seg first conv: two workgroups per CU, value loads
    (1, 64, 64, 64, "bf16"),      # stress conv: two workgroups per CU
    (8, 32, 16, 64, "f32"),       # two workgroups per CU, fp32 output (two staging passes)
    (2, 60, 64, 64, "bf16"),      # two workgroups per CU, ragged bricks on the far faces
])
def test_conv3d_full_size_sampled(B, R, Cin, Cout, odt):
    # full batch in the launch configuration the benchmark uses (the channel
    # tile and wave count depend on the grid size); the oracle evaluates 600
    # sampled outputs, a third of them on the grid's faces.
    rng = np.random.default_rng(11 + Cin + Cout)
    x = _sparse_grid(rng, B, R, Cin, occupied=0.06 if Cin <= 64 else 0.5)
    w = synth.kaiming_normal(rng, (Cout, 3, 3, 3, Cin), 27 * Cin, bf16=True)
    bn = synth.draw_bn(rng, Cout)
    y = host(pv.pvconv_conv3d(dev(x, torch.bfloat16), dev(w, torch.bfloat16), R, bn=dev_bn(bn),
                              out_dtype=torch.float32 if odt == "f32" else None))
    sel = rng.choice(B * R ** 3, size=400, replace=False)
    face = rng.integers(0, R, size=(200, 3))
    face[np.arange(200), rng.integers(0, 3, 200)] = rng.choice([0, R - 1], 200)
    sel = np.concatenate([sel, rng.integers(0, B, 200) * R ** 3 +
                          (face[:, 0] * R + face[:, 1]) * R + face[:, 2]])
    ref = oracle.leaky_relu(oracle.batchnorm(oracle.conv3d_at(x, w, R, sel), bn), 0.1)
    assert_bf16_step(y.reshape(-1, Cout)[sel], ref, "full-size conv samples")


# ----------------------------------------------------------------------------
# devoxelisation
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("wl_idx,B,N,R,C,gdt", [
    (2, 2, 2048, 32, 128, "bf16"), (5, 1, 65536, 64, 64, "bf16"), (1, 1, 1024, 8, 32, "f32"),
    (4, 2, 4096, 16, 64, "bf16"), (2, 2, 999, 24, 3, "f32"), (2, 16, 2048, 32, 128, "bf16"),
])
def test_devoxelize_matches_oracle(wl_idx, B, N, R, C, gdt):
    rng = np.random.default_rng(R * 7 + C)
    wl = synth.make_workload(wl_idx, B=B, N=N)
    _, _, pn = oracle.normalize(wl.coords)
    pn32 = pn.astype(np.float32)
    G = rng.normal(size=(B, R ** 3, C))
    if gdt == "bf16":
        G = bf16_round(G)
    ref = oracle.devoxelize(G, R, pn32)
    mag = oracle.devoxelize(np.abs(G), R, pn32)
    out = pv.pvconv_devoxelize(dev(G, torch.bfloat16 if gdt == "bf16" else torch.float32), R,
                               dev(pn32))
    assert_dot_f32(host(out), ref, mag, "devoxelize")


@pytest.mark.parametrize("wl_idx,B,N,R,C,gdt", [
    (2, 16, 2048, 32, 128, "bf16"), (5, 1, 65536, 64, 64, "bf16"), (1, 1, 1024, 8, 32, "f32"),
    (2, 3, 999, 24, 20, "bf16"), (2, 2, 777, 7, 3, "f32"), (4, 2, 4096, 16, 9, "bf16"),
])
def test_devoxelize_nearest_matches_oracle(wl_idx, B, N, R, C, gdt):
    # a copy of the voxel's row: bit-exact against the oracle
    rng = np.random.default_rng(R * 11 + C)
    wl = synth.make_workload(wl_idx, B=B, N=N)
    _, _, pn = oracle.normalize(wl.coords)
    ids = oracle.voxel_ids(pn, R)
    ids[:, :5] = [0, R ** 3 - 1, R - 1, R * R, R ** 3 // 2]   # grid corners and middle
    G = rng.normal(size=(B, R ** 3, C)).astype(np.float32).astype(np.float64)
    if gdt == "bf16":
        G = bf16_round(G)
    ref = oracle.devoxelize_nearest(G, R, ids)
    out = pv.pvconv_devoxelize_nearest(
        dev(G, torch.bfloat16 if gdt == "bf16" else torch.float32), R,
        torch.as_tensor(ids, dtype=torch.int32).cuda())
    assert np.array_equal(host(out), ref)


# ----------------------------------------------------------------------------
# point MLP with fused epilogue
# ----------------------------------------------------------------------------
MLP_CASES = [
    # M, Cin, Cout, x dtype, bias, bn, act, residual, cloud bias (points per cloud)
    (4096, 64, 128, "bf16", False, True, "relu", True, 0),
    (32768, 64, 128, "bf16", False, True, "relu", True, 0),   # part-seg point branch, full
    (1000, 3, 64, "bf16", False, True, "relu", False, 0),
    (1000, 9, 64, "bf16", True, True, "leaky", True, 0),
    (777, 128, 50, "bf16", True, False, "none", False, 0),    # logits layer
    (4100, 256, 13, "bf16", True, False, "none", False, 0),
    (2048, 512, 256, "bf16", False, True, "relu", False, 512),
    (65536, 64, 64, "bf16", False, True, "relu", True, 0),    # stress point branch, full
    (777, 96, 100, "bf16", True, True, "leaky", True, 0),     # ragged K chunk, N and M tails
    (1500, 40, 36, "bf16", False, True, "relu", True, 500),   # ragged K step, 3 clouds
    (2500, 128, 260, "f32", True, True, "relu", True, 0),     # fp32 rows, 3 channel blocks
    (3000, 200, 136, "bf16", True, True, "leaky", True, 0),   # wide: ragged K chunk and tiles
    (16384, 512, 2048, "bf16", False, True, "relu", False, 0),  # wide: part-seg MLP 512->2048
    (4100, 2880, 256, "bf16", False, True, "relu", False, 2050),  # wide: head with cloud rows
    (65600, 160, 264, "bf16", True, True, "leaky", True, 0),  # 256x256 tiles: ragged M, N, K
    (65536, 128, 256, "f32", False, True, "relu", True, 2048),  # 256x256 tiles: cloud rows
    (8, 2048, 256, "f32", False, False, "none", False, 0),    # one row per cloud (global)
    (100, 72, 36, "bf16", True, True, "leaky", True, 50),     # few rows, 2 clouds
    (37, 9, 5, "bf16", True, True, "relu", True, 0),          # few rows, odd widths
]


@pytest.mark.parametrize("case", MLP_CASES, ids=lambda c: "M{}_{}to{}_{}_{}".format(*c[:4], c[6]))
def test_point_mlp_bf16_matches_oracle(case):
    M, Cin, Cout, xdt, use_b, use_bn, act, use_res, ppc = case
    rng = np.random.default_rng(M + Cin)
    x = rng.normal(size=(M, Cin)).astype(np.float32)
    x_in = dev(x) if xdt == "f32" else dev(bf16_round(x), torch.bfloat16)
    x = bf16_round(x)  # fp32 rows are rounded to bf16 by the kernel
    w = synth.kaiming_normal(rng, (Cout, Cin), Cin, bf16=True)
    bias = rng.normal(size=Cout).astype(np.float32) if use_b else None
    bn = synth.draw_bn(rng, Cout) if use_bn else None
    res = rng.normal(size=(M, Cout)).astype(np.float32) if use_res else None
    cb = rng.normal(size=(M // ppc, Cout)).astype(np.float32) if ppc else None
    y = oracle.linear(x, w, bias)
    if cb is not None:
        y = y + np.repeat(cb, ppc, axis=0)
    if bn is not None:
        y = oracle.batchnorm(y, bn)
    y = {"relu": oracle.relu, "leaky": lambda a: oracle.leaky_relu(a, 0.2),
         "none": lambda a: a}[act](y)
    if res is not None:
        y = y + res
    out = pv.pvconv_point_mlp(x_in, dev(w, torch.bfloat16),
                              bias=dev(bias) if use_b else None,
                              bn=dev_bn(bn) if use_bn else None, act=act, slope=0.2,
                              cloud_bias=dev(cb) if ppc else None, points_per_cloud=max(ppc, 1),
                              residual=dev(res) if use_res else None)
    assert_bf16_step(host(out), y, f"point mlp {case}")


def test_point_mlp_fp32_inputs_strided_rows_and_bf16_out():
    rng = np.random.default_rng(21)
    M, Cin, Cout = 3000, 64, 128
    wide = rng.normal(size=(M, 200)).astype(np.float32)
    w = synth.kaiming_normal(rng, (Cout, Cin), Cin, bf16=True)
    bn = synth.draw_bn(rng, Cout)
    # fp32 inputs are rounded to bf16 by the kernel: the oracle takes the same rounded values
    ref = oracle.relu(oracle.batchnorm(oracle.linear(bf16_round(wide[:, 40:104]), w), bn))
    dst = torch.zeros((M, 300), dtype=torch.bfloat16, device="cuda")
    xd = dev(wide)
    pv.pvconv_point_mlp(xd[:, 40:104], dev(w, torch.bfloat16), bn=dev_bn(bn),
                        out=dst[:, 100:228])
    got = host(dst)
    assert_bf16_step(got[:, 100:228], ref, "strided mlp")
    assert np.all(got[:, :100] == 0) and np.all(got[:, 228:] == 0)


@pytest.mark.parametrize("M,Cin,Cout", [(1024, 16, 32), (333, 7, 5)])
def test_point_mlp_f32_matches_oracle(M, Cin, Cout):
    rng = np.random.default_rng(M)
    x = rng.normal(size=(M, Cin)).astype(np.float32).astype(np.float64)
    w = synth.kaiming_normal(rng, (Cout, Cin), Cin, bf16=False)
    bn = synth.draw_bn(rng, Cout)
    res = rng.normal(size=(M, Cout)).astype(np.float32)
    ref = oracle.relu(oracle.batchnorm(oracle.linear(x, w), bn)) + res
    mag = np.abs(x) @ np.abs(w.T) * bn_scale(bn) + np.abs(bn.mean * bn_scale(bn)) + \
        np.abs(bn.beta) + np.abs(res)
    out = pv.pvconv_point_mlp(dev(x), dev(w), bn=dev_bn(bn), residual=dev(res))
    assert_dot_f32(host(out), ref, mag, "mlp fp32")


@pytest.mark.parametrize("B,N,R,cin,cout,xdt,odt", [
    (2, 2048, 32, 64, 128, "f32", "f32"),    # part-seg layer's end, two clouds
    (3, 777, 16, 64, 96, "bf16", "f32"),     # ragged last tile, 96 = 1.5 channel blocks
    (2, 1000, 24, 16, 32, "f32", "bf16"),    # narrow layer, bf16 output
])
def test_devoxelize_point_mlp_matches_oracle_and_the_two_steps(B, N, R, cin, cout, xdt, odt):
    rng = np.random.default_rng(N + cout)
    wl = synth.make_workload(2, B=B, N=N)
    pn = oracle.normalize(wl.coords)[2]
    grid = bf16_round(rng.normal(size=(B, R ** 3, cout)))
    x = wl.feats[..., :cin]
    if xdt == "bf16":
        x = bf16_round(x)
    w = synth.kaiming_normal(rng, (cout, cin), cin, bf16=True)
    bias = rng.uniform(-0.1, 0.1, size=cout).astype(np.float32)
    bn = synth.draw_bn(rng, cout)
    ref = oracle.devoxelize(grid, R, pn) + oracle.relu(
        oracle.batchnorm(oracle.linear(bf16_round(x), w, bias), bn))
    tdt = torch.bfloat16 if odt == "bf16" else torch.float32
    g_grid, g_pn = dev(grid, torch.bfloat16), dev(pn)
    g_x = dev(x, torch.bfloat16 if xdt == "bf16" else torch.float32)
    g_w, g_b, g_bn = dev(w, torch.bfloat16), dev(bias), dev_bn(bn)
    got = pv.pvconv_devoxelize_point_mlp(g_grid, R, g_pn, g_x, g_w, bias=g_b, bn=g_bn,
                                         out_dtype=tdt)
    what = f"fused devox + MLP B{B} N{N} R{R} {cin}->{cout}"
    if odt == "bf16":
        assert_bf16_step(host(got), ref, what)
    else:
        # fp32 sums of bf16 products and of eight weighted corners
        mag = oracle.devoxelize(np.abs(grid), R, pn) + oracle.linear(
            np.abs(bf16_round(x)), np.abs(w), np.abs(bias)) * bn_scale(bn)
        assert_dot_f32(host(got), ref, mag, what)
    # the same arithmetic as the devoxelisation into a buffer followed by the
    # point MLP with that buffer as its residual
    dv = pv.pvconv_devoxelize(g_grid, R, g_pn)
    two = pv.pvconv_point_mlp(g_x, g_w, bias=g_b, bn=g_bn, act="relu", residual=dv,
                              out_dtype=tdt)
    assert torch.equal(got, two), what


@pytest.mark.parametrize("dt,off,C,N,shift", [
    ("f32", 300, 2048, 2048, 0.0),    # 16-byte rows: vector path
    ("bf16", 304, 2048, 2048, 0.0),
    ("bf16", 300, 2048, 2048, 0.0),   # unaligned rows: scalar path
    ("bf16", 8, 520, 333, 0.0),       # partial channel group, ragged point slice
    ("f32", 0, 13, 1000, 0.0),
    ("f32", 16, 1024, 700, -50.0),    # all negative
    ("bf16", 0, 64, 1, 0.0),          # one point
])
def test_maxpool_matches_oracle(dt, off, C, N, shift):
    rng = np.random.default_rng(5 + C + N)
    x = (rng.normal(size=(8, N, off + C + 7)) + shift).astype(np.float32).astype(np.float64)
    if dt == "bf16":
        x = bf16_round(x)
    ref = oracle.maxpool(x[:, :, off:off + C])
    xd = dev(x, torch.bfloat16 if dt == "bf16" else torch.float32)
    out = pv.pvconv_maxpool(xd[:, :, off:off + C])
    assert np.array_equal(host(out), ref)
    again = pv.pvconv_maxpool(xd[:, :, off:off + C], out=out)   # reused output starts over
    assert np.array_equal(host(again), ref)


# ----------------------------------------------------------------------------
# whole layer
# ----------------------------------------------------------------------------
def _run_layer(wl, L, dtype):
    layer = pv.DeviceLayer(L, "cuda", dtype)
    return host(pv.pvconv_forward(dev(wl.coords), dev(wl.feats), layer))


def test_forward_fp32_single_layer_full_size():
    wl = synth.make_workload(1)
    ref = oracle.pvconv_forward(wl.coords, wl.feats, wl.layers[0])
    got = _run_layer(wl, wl.layers[0], torch.float32)
    rms = np.sqrt(np.mean(ref ** 2))
    assert_dot_f32(got, ref, np.full_like(ref, rms), "fp32 layer")


@pytest.mark.parametrize("wl_idx,B", [(2, 2), (5, 1)])
def test_forward_bf16_layer(wl_idx, B):
    wl = synth.make_workload(wl_idx, B=B)
    ref = oracle.pvconv_forward(wl.coords, wl.feats, wl.layers[0])
    got = _run_layer(wl, wl.layers[0], torch.bfloat16)
    assert_bf16_chain(got, ref, f"layer wl{wl_idx}")


@pytest.mark.parametrize("wl_idx,B", [(2, 2), (1, 1)])
def test_forward_nearest_devox_layer(wl_idx, B):
    # the layer with the nearest-neighbour mapping (Section 4.1 "Devoxelization")
    wl = synth.make_workload(wl_idx, B=B)
    L = dataclasses.replace(wl.layers[0], devox="nearest")
    ref = oracle.pvconv_forward(wl.coords, wl.feats, L)
    if wl_idx == 1:
        got = _run_layer(wl, L, torch.float32)
        rms = np.sqrt(np.mean(ref ** 2))
        assert_dot_f32(got, ref, np.full_like(ref, rms), "fp32 layer, nearest devox")
    else:
        got = _run_layer(wl, L, torch.bfloat16)
        assert_bf16_chain(got, ref, "bf16 layer, nearest devox")


@pytest.mark.parametrize("R,n_convs,width,devox", [
    (24, 2, 1.0, "trilinear"), (32, 1, 1.0, "trilinear"), (32, 3, 1.0, "trilinear"),
    (32, 2, 0.25, "trilinear"), (16, 3, 0.5, "nearest"), (24, 2, 0.5, "nearest"),
    (32, 2, 0.125, "trilinear"), (16, 2, 0.125, "nearest"),
    (8, 2, 1.0, "trilinear"),   # a grid of 2 x 1 bricks: the convs split their input channels
])
def test_forward_layer_variants(R, n_convs, width, devox):
    # the variants the paper's resolution and ablation tables vary: R (24 is
    # not a power of two), one to three convolutions, narrower channels, and
    # the devoxelisation mapping; two part-seg clouds each
    wl = synth.make_workload(2, B=2)
    cin, cout = int(64 * width), int(128 * width)
    L = synth.draw_pvconv(np.random.default_rng(R + 10 * n_convs), cin, cout, R, n_convs,
                          bf16=True)
    L.devox = devox
    feats = np.ascontiguousarray(wl.feats[..., :cin])
    ref = oracle.pvconv_forward(wl.coords, feats, L)
    layer = pv.DeviceLayer(L, "cuda", torch.bfloat16)
    got = host(pv.pvconv_forward(dev(wl.coords), dev(feats), layer))
    assert_bf16_chain(got, ref, f"layer R{R} x{n_convs} {cin}->{cout} {devox}")


@pytest.mark.parametrize("N,cin,cout", [(1000, 16, 32), (777, 64, 96), (300, 12, 64)])
def test_forward_ragged_points_and_channels(N, cin, cout):
    # point counts that leave the last 128-point tile of the point MLP (which
    # gathers the trilinear voxel branch itself) partly empty, an output width
    # (96) that fills its 128-channel block only partly, and an input width
    # (12) that the fused kernel does not take (separate devoxelisation)
    wl = synth.make_workload(2, B=3, N=N)
    L = synth.draw_pvconv(np.random.default_rng(N), cin, cout, 16, 1, bf16=True)
    feats = np.ascontiguousarray(wl.feats[..., :cin])
    ref = oracle.pvconv_forward(wl.coords, feats, L)
    layer = pv.DeviceLayer(L, "cuda", torch.bfloat16)
    got = host(pv.pvconv_forward(dev(wl.coords), dev(feats), layer))
    assert_bf16_chain(got, ref, f"layer N{N} {cin}->{cout}")


def test_forward_scene_first_block_nine_channels():
    wl = synth.make_workload(4, B=2)
    L = wl.layers[0]
    ref = oracle.pvconv_forward(wl.coords, wl.feats, L)
    assert_bf16_chain(_run_layer(wl, L, torch.bfloat16), ref, "scene block 1")


def _oracle_layer_at(coords, feats, L, pts):
    """The layer's output at selected points (b, k), computing each
    convolution only at the voxels those points depend on."""
    clouds = sorted({b for b, _ in pts})
    loc = {b: i for i, b in enumerate(clouds)}
    R, V = L.R, L.R ** 3
    _, _, pn = oracle.normalize(coords[clouds])
    grid, _ = oracle.voxelize(oracle.voxel_ids(pn, R), feats[clouds], R)
    sel_pn = np.stack([pn[loc[b], k] for b, k in pts])
    cells, _ = oracle.devoxelize_weights(sel_pn, R)
    need = [set() for _ in range(L.n_convs)]
    for (b, _), cs in zip(pts, cells):
        need[-1].update(loc[b] * V + int(c) for c in cs)
    for i in range(L.n_convs - 1, 0, -1):   # conv i reads conv i-1 at the 27 neighbours
        for s in need[i]:
            lb, r = divmod(s, V)
            u, v, w = r // (R * R), (r // R) % R, r % R
            for du in (-1, 0, 1):
                for dv in (-1, 0, 1):
                    for dw in (-1, 0, 1):
                        a, bb, c = u + du, v + dv, w + dw
                        if 0 <= a < R and 0 <= bb < R and 0 <= c < R:
                            need[i - 1].add(lb * V + (a * R + bb) * R + c)
    h = grid
    for i, (wt, bn) in enumerate(zip(L.conv_w, L.conv_bn)):
        sel = np.array(sorted(need[i]), np.int64)
        y = oracle.leaky_relu(oracle.batchnorm(oracle.conv3d_at(h, wt, R, sel), bn), L.slope)
        h = np.zeros((len(clouds), V, L.cout))
        h.reshape(-1, L.cout)[sel] = y
    out = []
    for j, (b, k) in enumerate(pts):
        dvx = oracle.devoxelize(h[loc[b]][None], R, sel_pn[j][None, None])[0, 0]
        pt = oracle.point_branch(feats[b, k][None], L)[0]
        out.append(dvx + pt)
    return np.array(out)


def test_forward_part_seg_full_size_sampled():
    wl = synth.make_workload(2)
    L = wl.layers[0]
    got = _run_layer(wl, L, torch.bfloat16)
    rng = np.random.default_rng(9)
    pts = [(int(b), int(k)) for b in (3, 11) for k in rng.choice(wl.N, 24, replace=False)]
    ref = _oracle_layer_at(wl.coords, wl.feats, L, pts)
    sub = np.stack([got[b, k] for b, k in pts])
    # the chain tolerance's RMS floor uses the whole sampled block
    assert_bf16_chain(sub, ref, "part-seg layer, sampled points")


def test_forward_part_seg_full_size_every_element():
    # all 16 clouds x 2048 points x 128 channels of the part-segmentation
    # layer, in the launch configuration the benchmark times
    wl = synth.make_workload(2)
    L = wl.layers[0]
    got = _run_layer(wl, L, torch.bfloat16)
    # against the fp64 layer: the chain bound
    assert_bf16_chain(got, oracle.pvconv_forward(wl.coords, wl.feats, L),
                      "part-seg layer, every element")
    # against the layer that stores its grid and convolution outputs in bf16
    # as the GPU does: the single-step bound. What is left is the fp32
    # accumulation and the values whose fp32 and fp64 sums round to
    # neighbouring bf16 numbers (each at most 2^-7 |h|, few, and spread over
    # the trilinear weights)
    ref16 = oracle.pvconv_forward(wl.coords, wl.feats, L, stage_dtype="bf16")
    d = np.abs(got - ref16)
    print(f"[bf16-stage layer] max |d| = {d.max():.3g}, "
          f"max |d| / (1e-3 + 2e-2 |ref|) = {np.max(d / (1e-3 + 2e-2 * np.abs(ref16))):.3g}",
          flush=True)
    assert_bf16_step(got, ref16, "part-seg layer vs bf16-stage oracle")


@pytest.mark.parametrize("cloud", ["workload", "uniform", "clustered"])
def test_composed_entry_points_give_the_forward_bits(cloud):
    # the layer as separate C-ABI calls (voxelise, two convolutions on packed
    # weights, the fused devoxelisation + point MLP) is the forward's own
    # sequence of kernels: the same bits at full size. Inside the forward the
    # first convolution runs on the sparse grid and skips the MFMAs of empty
    # fragments; clouds of different occupancy (points spread through the
    # cube, or packed into a few blobs) exercise that.
    wl = synth.make_workload(2)
    L = wl.layers[0]
    layer = pv.DeviceLayer(L, "cuda", torch.bfloat16)
    xyz = wl.coords
    rng = np.random.default_rng(31)
    if cloud == "uniform":
        xyz = rng.uniform(-1, 1, xyz.shape).astype(np.float32)
    elif cloud == "clustered":
        centres = rng.uniform(-1, 1, (xyz.shape[0], 4, 1, 3))
        blobs = centres + 0.03 * rng.normal(size=(xyz.shape[0], 4, xyz.shape[1] // 4, 3))
        xyz = blobs.reshape(xyz.shape).astype(np.float32)
    coords, feats = dev(xyz), dev(wl.feats)
    want = pv.pvconv_forward(coords, feats, layer)
    grid, _, _, pn = pv.pvconv_voxelize(coords, feats, L.R, grid_dtype=torch.bfloat16)
    h = grid
    for i in range(L.n_convs):
        packed = pv.pvconv_conv3d_pack_weights(layer.conv_w[i])
        h = pv.pvconv_conv3d_packed(h, packed, L.cout, L.R, bn=layer.conv_bn[i], act="leaky",
                                    slope=L.slope, out_dtype=torch.bfloat16)
    got = pv.pvconv_devoxelize_point_mlp(h, L.R, pn, feats, layer.mlp_w, bias=layer.mlp_b,
                                         bn=layer.mlp_bn, act="relu")
    assert torch.equal(got, want)
    # and with the one-call convolutions, which pack internally
    h = grid
    for i in range(L.n_convs):
        h = pv.pvconv_conv3d(h, layer.conv_w[i], L.R, bn=layer.conv_bn[i], act="leaky",
                             slope=L.slope, out_dtype=torch.bfloat16)
    dv = pv.pvconv_devoxelize(h, L.R, pn)
    got2 = pv.pvconv_point_mlp(feats, layer.mlp_w, bias=layer.mlp_b, bn=layer.mlp_bn,
                               act="relu", residual=dv)
    assert torch.equal(got2, want)


@pytest.mark.parametrize("n_convs,devox,R", [
    (2, "trilinear", 32), (2, "nearest", 32), (1, "trilinear", 32), (1, "nearest", 32),
    (3, "trilinear", 32),
    (2, "trilinear", 20),   # bricks cut by the grid's faces
])
def test_forward_computes_every_voxel_the_devoxelisation_reads(n_convs, devox, R):
    # Inside the forward the last convolution computes only the outputs
    # within one voxel of an occupied voxel (the devoxelisation reads nothing
    # else) and leaves the rest of its grid as the workspace held it. With
    # the workspace full of NaN bytes, the output must still be the bits of
    # the separate calls, whose grids are complete: no unneeded voxel is read.
    wl = synth.make_workload(2)
    L = synth.draw_pvconv(np.random.default_rng(50 + n_convs), 64, 128, R, n_convs, bf16=True)
    L.devox = devox
    layer = pv.DeviceLayer(L, "cuda", torch.bfloat16)
    coords, feats = dev(wl.coords), dev(wl.feats)
    size = pv.pvconv_forward_workspace_size(wl.B, wl.N, layer)
    ws = torch.full((size,), 0xFF, dtype=torch.uint8, device="cuda")
    want = pv.pvconv_forward(coords, feats, layer, workspace=ws)
    grid, _, ids, pn = pv.pvconv_voxelize(coords, feats, L.R, grid_dtype=torch.bfloat16)
    h = grid
    for i in range(L.n_convs):
        h = pv.pvconv_conv3d(h, layer.conv_w[i], L.R, bn=layer.conv_bn[i], act="leaky",
                             slope=L.slope, out_dtype=torch.bfloat16)
    dv = (pv.pvconv_devoxelize_nearest(h, L.R, ids) if devox == "nearest"
          else pv.pvconv_devoxelize(h, L.R, pn))
    got = pv.pvconv_point_mlp(feats, layer.mlp_w, bias=layer.mlp_b, bn=layer.mlp_bn,
                              act="relu", residual=dv)
    assert torch.isfinite(want).all()
    assert torch.equal(got, want)


def test_forward_on_a_side_stream_and_repeatable():
    wl = synth.make_workload(2, B=2)
    layer = pv.DeviceLayer(wl.layers[0], "cuda", torch.bfloat16)
    c, f = dev(wl.coords), dev(wl.feats)
    a = pv.pvconv_forward(c, f, layer)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        b = pv.pvconv_forward(c, f, layer)
    s.synchronize()
    assert torch.equal(a, b)
