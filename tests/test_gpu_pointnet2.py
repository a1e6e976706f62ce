"""The PointNet++ primitives of PVCNN++ (Section 5.2 "Models") on the GPU
against the oracle: farthest point sampling, ball query, grouping, three
nearest neighbours and inverse-distance interpolation. Index results are
compared exactly (both sides choose on the same fp32 squared distances, ties
to the lower index); values within the bound of their arithmetic.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_1907_03739_amd import binding as pv
from _helpers import assert_bf16_step, bf16_round, dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu_case(request):
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    print(f"\n[gpu case] {request.node.nodeid}", flush=True)
    yield
    torch.cuda.synchronize()


def _rooms(B, N, seed):
    coords, feats = synth.rooms(np.random.default_rng(seed), B, N)
    return coords, feats


def _duplicates(B, N, seed):
    """Points on a coarse lattice: many coincide, so farthest distances tie
    and, once every distinct point is taken, fall to zero."""
    rng = np.random.default_rng(seed)
    return (rng.integers(0, 5, size=(B, N, 3)) * 0.25).astype(np.float32)


def _cloud(kind, B, N, seed):
    if kind == "rooms":
        return _rooms(B, N, seed)[0]
    if kind == "duplicates":
        return _duplicates(B, N, seed)
    if kind == "flat":  # a floor: no extent along z
        xyz = _rooms(B, N, seed)[0]
        xyz[..., 2] = 0.5
        return xyz
    assert kind == "identical"  # one place: no extent at all
    return np.full((B, N, 3), -0.25, np.float32)


FPS_CASES = [
    # B, N, npoint, cloud (every launch configuration of the kernel, ragged
    # sizes, and clouds whose distances tie: duplicates, a flat floor, one
    # point repeated)
    (3, 64, 16, "rooms"),
    (2, 200, 50, "rooms"),
    (2, 1000, 250, "rooms"),
    (2, 1025, 1025, "rooms"),        # every point
    (2, 3000, 700, "rooms"),
    (4, 8192, 1024, "rooms"),
    (1, 8191, 2048, "rooms"),
    (1, 12000, 300, "rooms"),
    (2, 300, 300, "duplicates"),     # every point, past the distinct ones
    (1, 5000, 1500, "duplicates"),
    (2, 4096, 512, "flat"),
    (1, 2000, 40, "identical"),
    (1, 16384, 64, "duplicates"),
]


@pytest.mark.parametrize("B,N,npoint,cloud", FPS_CASES)
def test_fps_matches_oracle(B, N, npoint, cloud):
    xyz = _cloud(cloud, B, N, N)
    want = oracle.fps(xyz, npoint)
    idx, new_xyz = pv.pvconv_furthest_point_sample(dev(xyz), npoint)
    got = idx.cpu().numpy()
    assert np.array_equal(got, want), np.argwhere(got != want)[:5]
    np.testing.assert_array_equal(new_xyz.cpu().numpy(), oracle.gather_points(xyz, want))


def test_fps_is_repeatable_and_takes_one_point():
    xyz = dev(_rooms(2, 5000, 1)[0])
    a = pv.pvconv_furthest_point_sample(xyz, 400, want_xyz=False)
    b = pv.pvconv_furthest_point_sample(xyz, 400, want_xyz=False)
    assert torch.equal(a, b)
    one = pv.pvconv_furthest_point_sample(xyz, 1, want_xyz=False)
    assert one.cpu().numpy().tolist() == [[0], [0]]


BALL_CASES = [
    # B, N, M, radius, nsample
    (4, 8192, 1024, 0.2, 32),     # the first set-abstraction level of the rooms
    (4, 1024, 256, 0.4, 32),
    (2, 1000, 77, 0.8, 16),       # N not a multiple of 64
    (2, 256, 64, 0.0, 8),         # radius 0: nothing strictly inside
    (1, 300, 40, 50.0, 64),       # everything inside: the first 64 in index order
]


@pytest.mark.parametrize("B,N,M,radius,nsample", BALL_CASES)
def test_ball_query_matches_oracle(B, N, M, radius, nsample):
    xyz = _rooms(B, N, N + M)[0]
    centers = oracle.gather_points(xyz, oracle.fps(xyz, M))
    want = oracle.ball_query(xyz, centers, radius, nsample)
    got = pv.pvconv_ball_query(dev(xyz), dev(centers), radius, nsample).cpu().numpy()
    assert np.array_equal(got, want), np.argwhere(got != want)[:5]


def test_ball_query_far_centres_and_duplicates():
    xyz = _duplicates(2, 500, 3)
    centers = np.concatenate([oracle.gather_points(xyz, oracle.fps(xyz, 20)),
                              np.full((2, 4, 3), 9.0, np.float32)], axis=1)
    want = oracle.ball_query(xyz, centers, 0.3, 24)
    got = pv.pvconv_ball_query(dev(xyz), dev(centers), 0.3, 24).cpu().numpy()
    assert np.array_equal(got, want)
    assert np.all(got[:, 20:] == 0)


@pytest.mark.parametrize("C,fdt,odt", [(32, "f32", "bf16"), (64, "bf16", "bf16"),
                                       (9, "f32", "f32"), (0, None, "bf16")])
def test_group_points_matches_oracle(C, fdt, odt):
    B, N, M, S = 2, 2048, 256, 32
    xyz, _ = _rooms(B, N, 5)
    rng = np.random.default_rng(C)
    feats = rng.normal(size=(B, N, C)).astype(np.float32)
    if fdt == "bf16":
        feats = bf16_round(feats).astype(np.float32)
    centers = oracle.gather_points(xyz, oracle.fps(xyz, M))
    idx = oracle.ball_query(xyz, centers, 0.4, S)
    want = oracle.group(xyz, feats, centers, idx)
    tdt = torch.bfloat16 if odt == "bf16" else torch.float32
    gf = None if C == 0 else dev(feats, torch.bfloat16 if fdt == "bf16" else torch.float32)
    got = host(pv.pvconv_group_points(dev(xyz), gf, dev(centers),
                                      torch.as_tensor(idx).cuda(), out_dtype=tdt))
    # features are copied (rounded to bf16 once for a bf16 output)
    fw = bf16_round(want[..., 3:]) if odt == "bf16" else want[..., 3:]
    np.testing.assert_array_equal(got[..., 3:], fw)
    # relative coordinates: one fp32 subtraction, then (bf16 output) one
    # rounding: within one bf16 spacing (2^-7 |x|) or fp32's half ulp
    rel = want[..., :3]
    tol = 2.0 ** -7 * np.abs(rel) if odt == "bf16" else 2.0 ** -24 * np.abs(rel)
    assert np.all(np.abs(got[..., :3] - rel) <= tol + 1e-30)


def test_group_points_into_a_column_slice():
    B, N, M, S, C = 1, 512, 64, 16, 8
    xyz, _ = _rooms(B, N, 9)
    feats = np.random.default_rng(9).normal(size=(B, N, C)).astype(np.float32)
    centers = oracle.gather_points(xyz, oracle.fps(xyz, M))
    idx = oracle.ball_query(xyz, centers, 0.5, S)
    wide = torch.full((B * M * S, 20), 7.0, dtype=torch.float32, device="cuda")
    pv.pvconv_group_points(dev(xyz), dev(feats), dev(centers), torch.as_tensor(idx).cuda(),
                           out=wide[:, 4:15])
    full = pv.pvconv_group_points(dev(xyz), dev(feats), dev(centers),
                                  torch.as_tensor(idx).cuda(), out_dtype=torch.float32)
    assert torch.equal(wide[:, 4:15], full.view(-1, 11))
    assert torch.all(wide[:, :4] == 7.0) and torch.all(wide[:, 15:] == 7.0)


@pytest.mark.parametrize("B,n,m", [(4, 8192, 1024), (4, 1024, 256), (2, 256, 64),
                                   (2, 64, 16), (1, 3000, 2500), (2, 100, 3)])
def test_three_nn_matches_oracle(B, n, m):
    xyz, _ = _rooms(B, n, n + m)
    known = oracle.gather_points(xyz, oracle.fps(xyz, m))
    want_i, want_w = oracle.three_nn(xyz, known)
    gi, gw = pv.pvconv_three_nn(dev(xyz), dev(known))
    got_i = gi.cpu().numpy()
    assert np.array_equal(got_i, want_i), np.argwhere(got_i != want_i)[:5]
    # fp32 square roots, reciprocals and a three-term sum
    np.testing.assert_allclose(host(gw), want_w, rtol=2e-6, atol=1e-7)


@pytest.mark.parametrize("C,fdt,odt", [(64, "bf16", "f32"), (256, "f32", "bf16"),
                                       (13, "f32", "f32")])
def test_three_interpolate_matches_oracle(C, fdt, odt):
    B, n, m = 2, 2048, 512
    xyz, _ = _rooms(B, n, 17)
    known = oracle.gather_points(xyz, oracle.fps(xyz, m))
    feats = np.random.default_rng(C).normal(size=(B, m, C)).astype(np.float32)
    if fdt == "bf16":
        feats = bf16_round(feats).astype(np.float32)
    gi, gw = pv.pvconv_three_nn(dev(xyz), dev(known))
    # the oracle interpolates with the GPU's indices and fp32 weights: this
    # test is about the interpolation
    idx, w = gi.cpu().numpy(), host(gw)
    want = oracle.three_interpolate(feats, idx, w)
    tdt = torch.bfloat16 if odt == "bf16" else torch.float32
    got = host(pv.pvconv_three_interpolate(
        dev(feats, torch.bfloat16 if fdt == "bf16" else torch.float32), gi, gw, out_dtype=tdt))
    if odt == "bf16":
        assert_bf16_step(got, want, "three_interpolate bf16")
    else:
        mag = oracle.three_interpolate(np.abs(feats), idx, w)
        assert np.all(np.abs(got - want) <= 1e-6 * mag + 1e-30)


def test_three_interpolate_into_a_column_slice():
    B, n, m, C = 2, 500, 100, 16
    xyz, _ = _rooms(B, n, 21)
    known = oracle.gather_points(xyz, oracle.fps(xyz, m))
    feats = dev(np.random.default_rng(3).normal(size=(B, m, C)))
    gi, gw = pv.pvconv_three_nn(dev(xyz), dev(known))
    wide = torch.zeros((B, n, 40), dtype=torch.float32, device="cuda")
    pv.pvconv_three_interpolate(feats, gi, gw, out=wide[:, :, 10:26])
    assert torch.equal(wide[:, :, 10:26], pv.pvconv_three_interpolate(feats, gi, gw))
    assert torch.all(wide[:, :, :10] == 0) and torch.all(wide[:, :, 26:] == 0)
