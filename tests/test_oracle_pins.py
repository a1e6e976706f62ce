"""Pins for the CPU oracle: each checks it against something other than itself.

The paper prints no worked example, intermediate values or test vectors, so the
pins are hand-worked examples of the definitions (tests/golden/), invariants
that the definitions imply, special cases that reduce to a library routine
(numpy, torch CPU fp64), and brute force on tiny inputs. Each is chosen so that
a plausible slip (a dropped term, a wrong sign or index, an axis swap, a
transposed operand, convolution instead of correlation, a shifted cell centre)
fails at least one of them.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _rng(seed=0):
    return np.random.default_rng(seed)


# ----------------------------------------------------------------------------
# Normalization (Section 4.1) and voxel indices (Eq. 2)
# ----------------------------------------------------------------------------
def test_normalize_worked_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "normalize_two_points.json")))
    coords = np.array([g["coords"]], np.float32)
    c, m, pn = oracle.normalize(coords)
    assert np.array_equal(c[0], g["centroid"])
    assert m[0] == g["radius"]
    assert np.array_equal(pn[0], np.array(g["pnorm"]))
    assert oracle.voxel_ids(pn, g["R"])[0].tolist() == g["ids"]


@pytest.mark.parametrize("R", [1, 2, 8, 32, 64])
def test_single_point_and_coincident_points_map_to_centre(R):
    # A one-point cloud has zero radius; the reading maps it to (1/2,1/2,1/2).
    for coords in (np.array([[[0.3, -7.0, 2.5]]], np.float32),
                   np.full((1, 17, 3), 4.25, np.float32)):
        c, m, pn = oracle.normalize(coords)
        assert m[0] == 0.0
        assert np.all(pn == 0.5)
        ids = oracle.voxel_ids(pn, R)
        h = R // 2
        assert np.all(ids == (h * R + h) * R + h)


def test_centroid_is_the_mean_and_radius_the_largest_norm():
    rng = _rng(1)
    coords = rng.uniform(-3, 5, size=(3, 1000, 3)).astype(np.float32)
    c, m, pn = oracle.normalize(coords)
    mean = coords.astype(np.float64).mean(axis=1)
    np.testing.assert_allclose(c, mean, rtol=0, atol=1e-13)
    d = coords.astype(np.float64) - c[:, None, :]
    np.testing.assert_allclose(m, np.linalg.norm(d, axis=2).max(axis=1), rtol=1e-15)


def test_normalized_cloud_is_centred_in_the_half_unit_sphere():
    rng = _rng(2)
    coords = (rng.normal(size=(4, 777, 3)) * [3.0, 0.2, 1.0] + [10, -4, 2]).astype(np.float32)
    _, _, pn = oracle.normalize(coords)
    # the gravity centre maps to the cube centre ...
    np.testing.assert_allclose(pn.mean(axis=1), 0.5, atol=1e-12)
    # ... the furthest point lands on the sphere of radius 1/2, nothing outside it
    r = np.linalg.norm(pn - 0.5, axis=2)
    np.testing.assert_allclose(r.max(axis=1), 0.5, rtol=1e-15)
    assert np.all(pn >= -1e-15) and np.all(pn <= 1 + 1e-15)


def test_normalization_is_uniform_not_per_axis():
    # Rotating the cloud rotates the normalised coordinates about the centre:
    # this fails for any per-axis (min-max or max-abs) scaling.
    rng = _rng(3)
    p = rng.normal(size=(1, 500, 3)) * [2.0, 0.5, 1.0]
    q = np.linalg.qr(rng.normal(size=(3, 3)))[0]
    a = p.astype(np.float32)
    b = (p @ q.T).astype(np.float32)
    _, _, pa = oracle.normalize(a)
    _, _, pb = oracle.normalize(b)
    np.testing.assert_allclose((pa - 0.5) @ q.T, pb - 0.5, atol=2e-7)


def test_scaling_by_power_of_two_leaves_ids_bit_identical():
    wl = synth.make_workload(2, B=2, N=2048)
    _, _, pn = oracle.normalize(wl.coords)
    for k in (-3, 1, 5):
        _, _, pk = oracle.normalize(wl.coords * np.float32(2.0 ** k))
        assert np.array_equal(pk, pn)
        assert np.array_equal(oracle.voxel_ids(pk, 32), oracle.voxel_ids(pn, 32))


def test_translation_and_scale_invariance_approximately():
    rng = _rng(4)
    p = rng.uniform(-1, 1, size=(1, 300, 3))
    _, _, p0 = oracle.normalize(p.astype(np.float32))
    _, _, p1 = oracle.normalize((p * 3.7 + [0.5, -2.0, 1.25]).astype(np.float32))
    np.testing.assert_allclose(p0, p1, atol=1e-6)


def test_permuting_points_permutes_ids_exactly():
    wl = synth.make_workload(5, B=1, N=20000)
    perm = _rng(5).permutation(wl.N)
    _, _, pn = oracle.normalize(wl.coords)
    _, _, pp = oracle.normalize(wl.coords[:, perm])
    assert np.array_equal(pp, pn[:, perm])
    assert np.array_equal(oracle.voxel_ids(pp, 64), oracle.voxel_ids(pn, 64)[:, perm])


@pytest.mark.parametrize("R", [1, 3, 8, 24, 32])
def test_each_point_lies_in_its_voxel(R):
    # Eq. 2: point k belongs to voxel (u,v,w) iff floor(x*r)=u etc.; so x lies
    # in [u/r, (u+1)/r), except that the top face x = 1 is clamped into u = r-1.
    rng = _rng(6)
    coords = rng.uniform(-1, 1, size=(2, 3000, 3)).astype(np.float32)
    _, _, pn = oracle.normalize(coords)
    ids = oracle.voxel_ids(pn, R).astype(np.int64)
    uvw = np.stack([ids // (R * R), (ids // R) % R, ids % R], axis=-1)
    lo = uvw / R
    hi = (uvw + 1) / R
    inside = (pn >= lo) & ((pn < hi) | ((uvw == R - 1) & (pn <= 1 + 1e-15)))
    inside |= (uvw == 0) & (pn < 0)
    assert inside.all()


def test_boundary_tie_uses_floor_not_round():
    # x exactly on a cell face belongs to the upper cell; x just below does not.
    pn = np.array([[[0.25, 0.5, 0.75], [np.nextafter(0.25, 0), 0.5, 0.75]]])
    ids = oracle.voxel_ids(pn, 4)[0]
    assert ids.tolist() == [(1 * 4 + 2) * 4 + 3, (0 * 4 + 2) * 4 + 3]


def test_non_finite_coordinates_are_rejected():
    bad = np.zeros((1, 4, 3), np.float32)
    bad[0, 2, 1] = np.nan
    with pytest.raises(ValueError):
        oracle.normalize(bad)


# ----------------------------------------------------------------------------
# Voxelization (Eq. 2)
# ----------------------------------------------------------------------------
def _brute_voxelize(ids, feats, R):
    B, N, C = feats.shape
    V = R ** 3
    s = np.zeros((B, V, C))
    n = np.zeros((B, V), np.int64)
    for b in range(B):
        np.add.at(s[b], ids[b], feats[b])
        n[b] = np.bincount(ids[b], minlength=V)
    with np.errstate(invalid="ignore", divide="ignore"):
        g = np.where(n[..., None] > 0, s / np.maximum(n, 1)[..., None], 0.0)
    return g, n


@pytest.mark.parametrize("wl_idx,R", [(1, 8), (2, 32), (5, 64)])
def test_voxelize_matches_bincount_brute_force(wl_idx, R):
    wl = synth.make_workload(wl_idx, B=2 if wl_idx != 5 else 1, N=4096)
    _, _, pn = oracle.normalize(wl.coords)
    ids = oracle.voxel_ids(pn, R)
    grid, counts = oracle.voxelize(ids, wl.feats, R)
    g, n = _brute_voxelize(ids, wl.feats.astype(np.float64), R)
    assert np.array_equal(counts, n)
    assert np.all(counts.sum(axis=1) == wl.N)  # counts sum to N per cloud
    np.testing.assert_allclose(grid, g, rtol=1e-13, atol=1e-14)


def test_voxelize_constant_field_is_preserved():
    wl = synth.make_workload(2, B=2, N=2048)
    _, _, pn = oracle.normalize(wl.coords)
    ids = oracle.voxel_ids(pn, 32)
    kappa = 0.7071
    grid, counts = oracle.voxelize(ids, np.full((2, 2048, 5), kappa), 32)
    occ = counts > 0
    assert np.all(grid[occ] == kappa)  # exact: n*kappa/n in fp64 for these n
    assert np.all(grid[~occ] == 0.0)


def test_all_points_in_one_voxel():
    rng = _rng(7)
    feats = rng.normal(size=(1, 50, 3))
    ids = np.full((1, 50), 123, np.int32)
    grid, counts = oracle.voxelize(ids, feats, 8)
    assert counts[0, 123] == 50 and counts.sum() == 50
    np.testing.assert_allclose(grid[0, 123], feats[0].mean(axis=0), rtol=1e-14)
    assert np.count_nonzero(grid[0, np.arange(512) != 123]) == 0


# ----------------------------------------------------------------------------
# 3x3x3 convolution (Section 4.1 "Feature Aggregation", Section 3)
# ----------------------------------------------------------------------------
def _torch_conv(x, w, R):
    B, V, Cin = x.shape
    Cout = w.shape[0]
    xt = torch.from_numpy(x.reshape(B, R, R, R, Cin)).permute(0, 4, 1, 2, 3).contiguous()
    wt = torch.from_numpy(np.ascontiguousarray(w.transpose(0, 4, 1, 2, 3)))
    y = torch.nn.functional.conv3d(xt.double(), wt.double(), padding=1)
    return y.permute(0, 2, 3, 4, 1).reshape(B, V, Cout).numpy()


def test_conv_orientation_worked_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "conv_orientation_r3.json")))
    x = np.zeros((1, 27, 1))
    x[0, 13, 0] = 1.0  # centre voxel (1,1,1)
    w = np.arange(27, dtype=np.float64).reshape(1, 3, 3, 3, 1)
    y = oracle.conv3d(x, w, 3)
    assert y[0, :, 0].tolist() == g["output_uvw_row_major"]


@pytest.mark.parametrize("R,Cin,Cout,B", [(1, 2, 3, 1), (2, 3, 2, 2), (4, 4, 3, 1), (5, 2, 4, 2),
                                          (6, 3, 2, 1)])
def test_conv_matches_torch_conv3d_fp64(R, Cin, Cout, B):
    rng = _rng(R * 100 + Cin)
    x = rng.normal(size=(B, R ** 3, Cin))
    w = rng.normal(size=(Cout, 3, 3, 3, Cin))
    np.testing.assert_allclose(oracle.conv3d(x, w, R), _torch_conv(x, w, R), rtol=1e-12,
                               atol=1e-12)


def test_conv_matches_shifted_sum_brute_force():
    # independent brute force: pad with zeros and add the 27 shifted copies
    rng = _rng(11)
    R, Cin, Cout = 5, 3, 2
    x = rng.normal(size=(1, R ** 3, Cin))
    w = rng.normal(size=(Cout, 3, 3, 3, Cin))
    xg = np.pad(x.reshape(R, R, R, Cin), ((1, 1), (1, 1), (1, 1), (0, 0)))
    y = np.zeros((R, R, R, Cout))
    for a in range(3):
        for b in range(3):
            for c in range(3):
                y += xg[a:a + R, b:b + R, c:c + R] @ w[:, a, b, c, :].T
    np.testing.assert_allclose(oracle.conv3d(x, w, R)[0], y.reshape(-1, Cout), rtol=1e-12,
                               atol=1e-12)


def test_conv_delta_kernels_identity_shift_and_box():
    rng = _rng(12)
    R = 4
    x = rng.normal(size=(1, R ** 3, 1))
    xg = x.reshape(R, R, R)
    w = np.zeros((1, 3, 3, 3, 1))
    w[0, 1, 1, 1, 0] = 1.0
    np.testing.assert_array_equal(oracle.conv3d(x, w, R), x)  # centre delta: identity
    w = np.zeros((1, 3, 3, 3, 1))
    w[0, 2, 1, 1, 0] = 1.0  # offset (+1, 0, 0): y[u] = x[u+1], zero past the edge
    y = oracle.conv3d(x, w, R)[0, :, 0].reshape(R, R, R)
    np.testing.assert_array_equal(y[:-1], xg[1:])
    np.testing.assert_array_equal(y[-1], 0.0)
    w = np.zeros((1, 3, 3, 3, 1))
    w[0, 1, 1, 0, 0] = 1.0  # offset (0, 0, -1): y[..., w] = x[..., w-1]
    y = oracle.conv3d(x, w, R)[0, :, 0].reshape(R, R, R)
    np.testing.assert_array_equal(y[:, :, 1:], xg[:, :, :-1])
    np.testing.assert_array_equal(y[:, :, 0], 0.0)
    ones = np.ones((1, 3, 3, 3, 1))
    y = oracle.conv3d(np.ones((1, R ** 3, 1)), ones, R)[0, :, 0].reshape(R, R, R)
    interior = np.array([2, 3, 3, 2])  # neighbours per axis incl. self at R=4
    np.testing.assert_array_equal(y, np.einsum("i,j,k->ijk", interior, interior, interior))


def test_conv_is_linear_and_sampled_matches_dense():
    rng = _rng(13)
    R, Cin, Cout = 6, 4, 5
    x1, x2 = rng.normal(size=(2, 2, R ** 3, Cin))
    w = rng.normal(size=(Cout, 3, 3, 3, Cin))
    y = oracle.conv3d(2.5 * x1 + x2, w, R)
    np.testing.assert_allclose(y, 2.5 * oracle.conv3d(x1, w, R) + oracle.conv3d(x2, w, R),
                               rtol=1e-12, atol=1e-12)
    sel = rng.choice(2 * R ** 3, size=40, replace=False)
    np.testing.assert_array_equal(oracle.conv3d_at(2.5 * x1 + x2, w, R, sel),
                                  y.reshape(-1, Cout)[sel])


def test_batchnorm_and_activations_closed_form():
    bn = synth.BNParams(gamma=np.array([2.0, 0.5]), beta=np.array([1.0, -1.0]),
                        mean=np.array([3.0, -2.0]), var=np.array([4.0, 0.25]), eps=0.0)
    y = np.array([[3.0, -2.0], [5.0, 0.0], [1.0, -3.0]])
    z = oracle.batchnorm(y, bn)
    np.testing.assert_array_equal(z, [[1.0, -1.0], [3.0, 1.0], [-1.0, -2.0]])
    np.testing.assert_array_equal(oracle.leaky_relu(z, 0.1), [[1.0, -0.1], [3.0, 1.0],
                                                              [-0.1, -0.2]])
    np.testing.assert_array_equal(oracle.relu(z), [[1.0, 0.0], [3.0, 1.0], [0.0, 0.0]])
    # folding into scale and shift agrees with the unfolded form
    bn = synth.draw_bn(_rng(14), 7)
    y = _rng(15).normal(size=(11, 7))
    s = bn.gamma.astype(np.float64) / np.sqrt(bn.var.astype(np.float64) + bn.eps)
    t = bn.beta - bn.mean.astype(np.float64) * s
    np.testing.assert_allclose(oracle.batchnorm(y, bn), y * s + t, rtol=1e-12, atol=1e-12)


# ----------------------------------------------------------------------------
# Devoxelization (Section 4.1)
# ----------------------------------------------------------------------------
def test_devox_worked_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "devox_r2.json")))
    R = g["R"]
    u, v, w = np.meshgrid(range(R), range(R), range(R), indexing="ij")
    grid = (100 * u + 10 * v + w).reshape(1, R ** 3, 1).astype(np.float64)
    out = oracle.devoxelize(grid, R, np.array([g["points"]]))
    np.testing.assert_allclose(out[0, :, 0], g["values"], rtol=1e-15)


def test_devox_weights_sum_to_one_and_constant_is_preserved():
    rng = _rng(16)
    pn = rng.uniform(-0.01, 1.01, size=(2, 500, 3))
    for R in (1, 2, 7, 32):
        _, wts = oracle.devoxelize_weights(pn, R)
        np.testing.assert_allclose(wts.sum(axis=-1), 1.0, atol=1e-15)
        assert np.all(wts >= 0)
        out = oracle.devoxelize(np.full((2, R ** 3, 3), -1.25), R, pn)
        np.testing.assert_allclose(out, -1.25, rtol=1e-15)


def test_devox_reproduces_affine_field_and_cell_centres():
    # V at cell (u,v,w) = a . centre + b with centre = ((u,v,w) + 1/2) / R.
    # Trilinear interpolation reproduces it exactly for points whose cell
    # coordinate is not clamped, i.e. inside [1/(2R), 1 - 1/(2R)]^3.
    R = 8
    a = np.array([1.5, -2.0, 0.25])
    u, v, w = np.meshgrid(range(R), range(R), range(R), indexing="ij")
    cen = (np.stack([u, v, w], -1) + 0.5) / R
    grid = (cen @ a + 0.3).reshape(1, R ** 3, 1)
    rng = _rng(17)
    pn = rng.uniform(0.5 / R, 1 - 0.5 / R, size=(1, 400, 3))
    out = oracle.devoxelize(grid, R, pn)
    np.testing.assert_allclose(out[0, :, 0], pn[0] @ a + 0.3, rtol=1e-13, atol=1e-13)
    # a point at a cell centre returns that cell's value
    pc = cen.reshape(1, -1, 3)
    np.testing.assert_allclose(oracle.devoxelize(grid, R, pc)[0, :, 0], grid[0, :, 0],
                               rtol=1e-14, atol=1e-14)


def test_voxelize_then_devoxelize_preserves_constant_where_corners_occupied():
    wl = synth.make_workload(2, B=2, N=2048)
    R = 16
    _, _, pn = oracle.normalize(wl.coords)
    ids = oracle.voxel_ids(pn, R)
    kappa = 2.5
    grid, counts = oracle.voxelize(ids, np.full((2, 2048, 1), kappa), R)
    out = oracle.devoxelize(grid, R, pn)[..., 0]
    cells, wts = oracle.devoxelize_weights(pn, R)
    occupied = np.take_along_axis(counts[:, None, :].repeat(2048, 1), cells, axis=2) > 0
    full = (occupied | (wts == 0)).all(axis=2)
    assert full.sum() > 100
    np.testing.assert_allclose(out[full], kappa, rtol=1e-14)
    # elsewhere empty corners contribute zero: the value is kappa times the
    # occupied corners' weight
    occ_w = (wts * occupied).sum(axis=2)
    np.testing.assert_allclose(out, kappa * occ_w, rtol=1e-13, atol=1e-15)


def test_lone_point_gets_an_eighth_at_even_R():
    # one point -> centre (1/2,1/2,1/2) -> cell coordinate R/2 - 1/2: all 8
    # corners weigh 1/8 and only one of them is occupied
    for R in (2, 8, 32):
        _, _, pn = oracle.normalize(np.array([[[1.0, 2.0, 3.0]]], np.float32))
        grid, _ = oracle.voxelize(oracle.voxel_ids(pn, R), np.array([[[4.0]]]), R)
        assert oracle.devoxelize(grid, R, pn)[0, 0, 0] == 0.5


def test_nearest_devox_of_voxelize_is_the_voxel_mean_by_brute_force():
    # Section 4.1 "Devoxelization", nearest neighbour: each point gets the
    # features of the grid cell it falls into, so after voxelisation (no
    # convolution) every point reads the mean over the points sharing its cell.
    # The expectation groups points by their cell with a Python dict.
    wl = synth.make_workload(2, B=2, N=600)
    rng = _rng(30)
    feats = rng.normal(size=(2, 600, 5))
    for R in (4, 13, 32):
        _, _, pn = oracle.normalize(wl.coords)
        ids = oracle.voxel_ids(pn, R)
        grid, _ = oracle.voxelize(ids, feats, R)
        out = oracle.devoxelize_nearest(grid, R, ids)
        for b in range(2):
            groups = {}
            for k in range(600):
                groups.setdefault(int(ids[b, k]), []).append(k)
            for cell, members in groups.items():
                mean = feats[b, members].mean(axis=0)
                np.testing.assert_allclose(out[b, members], np.broadcast_to(mean, (len(members), 5)),
                                           rtol=1e-13, atol=1e-13)
                # the paper's stated property: one cell, one shared feature
                assert (out[b, members] == out[b, members[0]]).all()


def test_nearest_devox_reads_the_cell_of_each_index_and_matches_trilinear_at_centres():
    # a grid whose row is its own (u, v, w) digits: the output names the cell
    R = 6
    u, v, w = np.meshgrid(range(R), range(R), range(R), indexing="ij")
    grid = (100 * u + 10 * v + w).reshape(1, R ** 3, 1).astype(np.float64)
    ids = np.array([[0, 1, R, R * R, R ** 3 - 1, (2 * R + 3) * R + 5]], np.int32)
    out = oracle.devoxelize_nearest(grid, R, ids)[0, :, 0]
    np.testing.assert_array_equal(out, [0, 1, 10, 100, 555, 235])
    # at a cell centre trilinear weights collapse onto that cell, and the
    # centre's Eq. 2 index is that cell: the two mappings agree there
    rng = _rng(31)
    g = rng.normal(size=(1, R ** 3, 3))
    cen = ((np.stack([u, v, w], -1) + 0.5) / R).reshape(1, -1, 3)
    cid = oracle.voxel_ids(cen, R)
    np.testing.assert_array_equal(cid[0], np.arange(R ** 3))
    np.testing.assert_allclose(oracle.devoxelize_nearest(g, R, cid), oracle.devoxelize(g, R, cen),
                               rtol=1e-14, atol=1e-14)


def test_nearest_devox_rejects_indices_outside_the_grid():
    grid = np.zeros((1, 8, 2))
    for bad in (-1, 8):
        with pytest.raises(ValueError):
            oracle.devoxelize_nearest(grid, 2, np.array([[0, bad]], np.int32))


def test_layer_with_nearest_devox_differs_only_in_the_voxel_branch_mapping():
    wl = synth.make_workload(1, N=300)
    L = wl.layers[0]
    Ln = synth.PVConvParams(L.cin, L.cout, L.R, L.conv_w, L.conv_bn, L.mlp_w, L.mlp_bn,
                            devox="nearest")
    pt = oracle.pvconv_forward(wl.coords, wl.feats, L, return_parts=True)
    pn_ = oracle.pvconv_forward(wl.coords, wl.feats, Ln, return_parts=True)
    np.testing.assert_array_equal(pt["point"], pn_["point"])
    np.testing.assert_array_equal(pt["convs"][-1], pn_["convs"][-1])
    h = pt["convs"][-1]
    ref = np.stack([h[b, pt["ids"][b]] for b in range(h.shape[0])])
    np.testing.assert_array_equal(pn_["devox"], ref)
    assert np.array_equal(pn_["out"], pn_["devox"] + pn_["point"])


# ----------------------------------------------------------------------------
# Backward: each gradient is pinned by the adjoint identity <dy, f(x)> =
# <f*(dy), x> of its (linear) forward step, by finite differences, or by torch
# autograd on the CPU in fp64
# ----------------------------------------------------------------------------
def _dot(a, b):
    return float(np.sum(np.asarray(a, np.float64) * np.asarray(b, np.float64)))


def test_voxelize_backward_is_the_adjoint_of_the_average():
    wl = synth.make_workload(2, B=2, N=500)
    rng = _rng(40)
    R, C = 8, 3
    _, _, pn = oracle.normalize(wl.coords)
    ids = oracle.voxel_ids(pn, R)
    f = rng.normal(size=(2, 500, C))
    grid, counts = oracle.voxelize(ids, f, R)
    dV = rng.normal(size=grid.shape)
    df = oracle.voxelize_backward(dV, ids, counts, R)
    assert abs(_dot(dV, grid) - _dot(df, f)) <= 1e-11 * (abs(_dot(dV, grid)) + 1)
    # finite difference in one feature (the map is linear: exact up to rounding)
    for (b, k, c) in [(0, 0, 0), (1, 37, 2), (0, 499, 1)]:
        e = np.zeros_like(f)
        e[b, k, c] = 1.0
        g1, _ = oracle.voxelize(ids, f + e, R)
        np.testing.assert_allclose(_dot(dV, g1) - _dot(dV, grid), df[b, k, c], rtol=1e-9,
                                   atol=1e-12)


def test_devoxelize_backward_is_the_adjoint_trilinear_and_nearest():
    rng = _rng(41)
    B, N, C = 2, 300, 4
    for R in (1, 5, 8):
        pn = rng.uniform(-0.02, 1.02, size=(B, N, 3))
        G = rng.normal(size=(B, R ** 3, C))
        dout = rng.normal(size=(B, N, C))
        dG = oracle.devoxelize_backward(dout, R, pn)
        lhs = _dot(dout, oracle.devoxelize(G, R, pn))
        assert abs(lhs - _dot(dG, G)) <= 1e-11 * (abs(lhs) + 1)
        ids = rng.integers(0, R ** 3, size=(B, N)).astype(np.int32)
        dGn = oracle.devoxelize_nearest_backward(dout, R, ids)
        lhs = _dot(dout, oracle.devoxelize_nearest(G, R, ids))
        assert abs(lhs - _dot(dGn, G)) <= 1e-11 * (abs(lhs) + 1)
        # every point hands each of its cells its trilinear weight: the
        # gradient of an all-ones output sums to N per cloud
        np.testing.assert_allclose(oracle.devoxelize_backward(np.ones((B, N, 1)), R, pn)
                                   .sum(axis=(1, 2)), N, rtol=1e-12)


@pytest.mark.parametrize("R,Cin,Cout,B", [(1, 2, 3, 1), (3, 3, 2, 2), (5, 4, 3, 1)])
def test_conv_backward_matches_torch_autograd_fp64(R, Cin, Cout, B):
    rng = _rng(42 + R)
    x = rng.normal(size=(B, R ** 3, Cin))
    w = rng.normal(size=(Cout, 3, 3, 3, Cin))
    dy = rng.normal(size=(B, R ** 3, Cout))
    xt = torch.tensor(x.reshape(B, R, R, R, Cin)).permute(0, 4, 1, 2, 3).requires_grad_(True)
    wt = torch.tensor(w).permute(0, 4, 1, 2, 3).contiguous().requires_grad_(True)
    yt = torch.nn.functional.conv3d(xt, wt, padding=1)
    dyt = torch.tensor(dy.reshape(B, R, R, R, Cout)).permute(0, 4, 1, 2, 3)
    yt.backward(dyt)
    dx_ref = xt.grad.permute(0, 2, 3, 4, 1).reshape(B, R ** 3, Cin).numpy()
    dw_ref = wt.grad.permute(0, 2, 3, 4, 1).numpy()
    np.testing.assert_allclose(oracle.conv3d_backward_data(dy, w, R), dx_ref, rtol=1e-12,
                               atol=1e-12)
    np.testing.assert_allclose(oracle.conv3d_backward_weight(dy, x, R), dw_ref, rtol=1e-12,
                               atol=1e-12)


def test_conv_backward_is_the_adjoint_at_a_realistic_shape():
    rng = _rng(43)
    R, Cin, Cout = 6, 5, 7
    x = rng.normal(size=(2, R ** 3, Cin)) * (rng.random((2, R ** 3, 1)) < 0.3)
    w = rng.normal(size=(Cout, 3, 3, 3, Cin))
    dy = rng.normal(size=(2, R ** 3, Cout))
    y = oracle.conv3d(x, w, R)
    lhs = _dot(dy, y)
    assert abs(lhs - _dot(oracle.conv3d_backward_data(dy, w, R), x)) <= 1e-10 * (abs(lhs) + 1)
    assert abs(lhs - _dot(oracle.conv3d_backward_weight(dy, x, R), w)) <= 1e-10 * (abs(lhs) + 1)


def test_layer_feature_gradient_matches_finite_differences():
    # the layer is piecewise linear in its features: central differences of
    # the pinned forward give the directional derivative exactly away from the
    # rectifiers' kinks
    wl = synth.make_workload(1, N=200)
    L = wl.layers[0]
    rng = _rng(45)
    feats = wl.feats.astype(np.float64)
    dout = rng.normal(size=(1, 200, L.cout))
    for devox in ("trilinear", "nearest"):
        Ld = synth.PVConvParams(L.cin, L.cout, L.R, L.conv_w, L.conv_bn, L.mlp_w, L.mlp_bn,
                                devox=devox)
        df = oracle.layer_backward_features(wl.coords, feats, Ld, dout)
        h = 1e-6
        for _ in range(4):
            e = rng.normal(size=feats.shape)
            fp = oracle.pvconv_forward(wl.coords, feats + h * e, Ld)
            fm = oracle.pvconv_forward(wl.coords, feats - h * e, Ld)
            fd = _dot(dout, fp - fm) / (2 * h)
            np.testing.assert_allclose(_dot(df, e), fd, rtol=1e-6)


def test_act_bn_backward_matches_finite_differences():
    rng = _rng(44)
    bn = synth.draw_bn(rng, 6)
    z = rng.normal(size=(50, 6)) * 2
    dy = rng.normal(size=(50, 6))
    h = 1e-6
    for act, fwd in [("leaky", lambda t: oracle.leaky_relu(oracle.batchnorm(t, bn), 0.1)),
                     ("relu", lambda t: oracle.relu(oracle.batchnorm(t, bn))),
                     ("none", lambda t: oracle.batchnorm(t, bn))]:
        y = fwd(z)
        dz = oracle.act_bn_backward(dy, y, bn, act, 0.1)
        fd = (fwd(z + h) - fwd(z - h)) / (2 * h) * dy   # elementwise: one step per entry
        np.testing.assert_allclose(dz, fd, rtol=1e-6, atol=1e-8)


# ----------------------------------------------------------------------------
# Point branch, fusion, max-pool (Sections 4.2, 4.3, 5.1)
# ----------------------------------------------------------------------------
def test_linear_matches_numpy_matmul():
    rng = _rng(18)
    x = rng.normal(size=(3, 50, 7))
    w = rng.normal(size=(5, 7))
    b = rng.normal(size=5)
    np.testing.assert_allclose(oracle.linear(x, w, b), np.matmul(x, w.T) + b, rtol=1e-13,
                               atol=1e-13)
    np.testing.assert_allclose(oracle.linear(x, w), np.matmul(x, w.T), rtol=1e-13, atol=1e-13)


def test_maxpool_matches_numpy():
    x = _rng(19).normal(size=(3, 40, 6))
    np.testing.assert_array_equal(oracle.maxpool(x), x.max(axis=1))


def test_layer_is_the_sum_of_its_branches():
    wl = synth.make_workload(1, N=256)
    L = wl.layers[0]
    parts = oracle.pvconv_forward(wl.coords, wl.feats, L, return_parts=True)
    assert np.array_equal(parts["out"], parts["devox"] + parts["point"])
    # point branch against numpy: ReLU(BN(W f))
    bn = L.mlp_bn
    s = bn.gamma.astype(np.float64) / np.sqrt(bn.var.astype(np.float64) + bn.eps)
    ref = np.maximum((wl.feats.astype(np.float64) @ L.mlp_w.T.astype(np.float64) - bn.mean) * s
                     + bn.beta, 0)
    np.testing.assert_allclose(parts["point"], ref, rtol=1e-12, atol=1e-12)
    # with zero conv weights the voxel branch is constant: LReLU(BN(0)) per channel
    L0 = synth.PVConvParams(L.cin, L.cout, L.R, [np.zeros_like(L.conv_w[0])], L.conv_bn,
                            L.mlp_w, L.mlp_bn)
    p0 = oracle.pvconv_forward(wl.coords, wl.feats, L0, return_parts=True)
    cb = L.conv_bn[0]
    z = cb.beta - cb.mean.astype(np.float64) * cb.gamma / np.sqrt(cb.var.astype(np.float64) +
                                                                  cb.eps)
    z = np.where(z < 0, 0.1 * z, z)
    np.testing.assert_allclose(p0["devox"], np.broadcast_to(z, p0["devox"].shape), rtol=1e-12)


# ----------------------------------------------------------------------------
# Network glue (Section 5.1 "Models") and bf16 storage of activations
# ----------------------------------------------------------------------------
def test_round_bf16_matches_torch_and_breaks_ties_to_even():
    rng = _rng(20)
    x = np.concatenate([rng.normal(size=4000) * 10.0 ** rng.integers(-30, 30, size=4000),
                        rng.normal(size=200) * 2.0 ** -128]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.round_bf16(x), ref)
    one = 1.0
    cases = {one + 2 ** -8: one,                       # tie, even neighbour below
             one + 3 * 2 ** -8: one + 2 ** -6,          # tie, even neighbour above
             -(one + 2 ** -8): -one,
             one + 2 ** -8 + 2 ** -30: one + 2 ** -7,   # just past the tie
             0.0: 0.0, 3.0: 3.0}
    for v, want in cases.items():
        assert oracle.round_bf16(np.array([v]))[0] == want, v
    assert np.isnan(oracle.round_bf16(np.array([np.nan]))[0])


@pytest.mark.parametrize("idx", [3, 4])
def test_network_clouds_are_independent(idx):
    wl = synth.make_workload(idx, B=2, N=96)
    full = oracle.network_forward(wl)
    for b in range(2):
        one = synth.make_workload(idx, B=2, N=96)
        one.B, one.coords, one.feats = 1, wl.coords[b:b + 1], wl.feats[b:b + 1]
        np.testing.assert_array_equal(oracle.network_forward(one)[0], full[b])


def test_network_global_feature_is_broadcast_last():
    """With the head's stage columns zeroed, the first head layer sees only
    the pooled global feature: every point of a cloud gets the same logits,
    equal to the head applied to g alone."""
    wl = synth.make_workload(3, B=2, N=80)
    h0 = wl.head[0]
    cg = wl.mlps[-1].w.shape[0]
    w = h0.w.copy()
    w[:, :-cg] = 0.0
    wl.head = [synth.LinearParams(w=w, b=h0.b, bn=h0.bn, relu=h0.relu)] + wl.head[1:]
    out, stages, g = oracle.network_forward(wl, return_stages=True)
    np.testing.assert_allclose(out, np.broadcast_to(out[:, :1], out.shape), rtol=0, atol=1e-12)
    np.testing.assert_array_equal(g, stages[-1].max(axis=1))
    h = g
    for lp in [synth.LinearParams(w=w[:, -cg:], b=h0.b, bn=h0.bn, relu=h0.relu)] + wl.head[1:]:
        h = oracle.shared_mlp(h, lp)
    np.testing.assert_allclose(out[:, 0], h, rtol=1e-12, atol=1e-12)


def test_network_concat_order_follows_the_stages():
    """A head whose first layer is the identity on one stage-column range
    (then no BN/activation) returns exactly that stage's output."""
    wl = synth.make_workload(4, B=1, N=64)
    widths = [L.cout for L in wl.layers] + [m.w.shape[0] for m in wl.mlps]
    total = sum(widths) + widths[-1]
    k = 1                                   # the second PVConv block
    off = sum(widths[:k])
    w = np.zeros((widths[k], total))
    w[np.arange(widths[k]), off + np.arange(widths[k])] = 1.0
    wl.head = [synth.LinearParams(w=w, b=None, bn=None, relu=False)]
    out, stages, _ = oracle.network_forward(wl, return_stages=True)
    np.testing.assert_array_equal(out, stages[k])


def test_network_bf16_storage_rounds_every_stage():
    wl = synth.make_workload(4, B=1, N=64)
    out16, st16, g16 = oracle.network_forward(wl, return_stages=True, stage_dtype="bf16")
    out64 = oracle.network_forward(wl)
    for s in st16:
        np.testing.assert_array_equal(oracle.round_bf16(s), s)
    np.testing.assert_array_equal(oracle.round_bf16(g16), g16)
    rms = np.sqrt(np.mean(out64 ** 2))
    assert np.max(np.abs(out16 - out64)) < 0.05 * rms   # bf16 storage, not a different net
    assert np.max(np.abs(out16 - out64)) > 0.0
    with pytest.raises(ValueError):
        oracle.network_forward(wl, stage_dtype="f16")


def _identity_layer(C, R):
    """A layer whose convolutions copy the grid (centre tap = identity, all
    other taps zero), with identity batch norms and no point branch weight."""
    one = synth.BNParams(gamma=np.ones(C, np.float32), beta=np.zeros(C, np.float32),
                         mean=np.zeros(C, np.float32), var=np.ones(C, np.float32), eps=0.0)
    w = np.zeros((C, 3, 3, 3, C), np.float32)
    w[:, 1, 1, 1, :] = np.eye(C, dtype=np.float32)
    return synth.PVConvParams(cin=C, cout=C, R=R, conv_w=[w, w.copy()], conv_bn=[one, one],
                              mlp_w=np.zeros((C, C), np.float32), mlp_bn=one)


def test_layer_bf16_storage_is_lossless_on_bf16_values_and_rounds_others():
    # a 4 x 4 x 4 lattice, one point per voxel of an R = 16 grid: the grid is
    # the features themselves and the identity convolutions copy it exactly
    R, C = 16, 8
    cells = np.array([(u, v, w) for u in range(4) for v in range(4) for w in range(4)])
    coords = ((cells + 0.5) / 4.0)[None] * 2.0 - 1.0
    rng = np.random.default_rng(3)
    feats = rng.integers(1, 200, size=(1, len(cells), C)).astype(np.float64)
    L = _identity_layer(C, R)
    parts = oracle.pvconv_forward(coords, feats, L, return_parts=True)
    assert parts["counts"].max() == 1
    # small positive integers are bf16 values: storage changes nothing
    np.testing.assert_array_equal(
        oracle.pvconv_forward(coords, feats, L, stage_dtype="bf16"), parts["out"])
    # features of thirds are not: every stored stage is rounded, and as every
    # step before the devoxelisation is exact, storing in bf16 is the same as
    # rounding the features once and computing in fp64
    thirds = feats / 3.0
    p16 = oracle.pvconv_forward(coords, thirds, L, return_parts=True, stage_dtype="bf16")
    for stage in [p16["grid"]] + p16["convs"]:
        np.testing.assert_array_equal(oracle.round_bf16(stage), stage)
    np.testing.assert_array_equal(
        p16["out"], oracle.pvconv_forward(coords, oracle.round_bf16(thirds), L))
    assert np.max(np.abs(p16["out"] - oracle.pvconv_forward(coords, thirds, L))) > 0.0


def test_layer_bf16_storage_stays_within_a_bf16_ulp_chain():
    wl = synth.make_workload(2, B=1, N=256)
    L = wl.layers[0]
    p16 = oracle.pvconv_forward(wl.coords, wl.feats, L, return_parts=True, stage_dtype="bf16")
    p64 = oracle.pvconv_forward(wl.coords, wl.feats, L, return_parts=True)
    for stage in [p16["grid"]] + p16["convs"]:
        np.testing.assert_array_equal(oracle.round_bf16(stage), stage)
    # the grid is rounded once: within half a bf16 spacing, at most 2^-8 |x|
    g64 = p64["grid"]
    assert np.all(np.abs(p16["grid"] - g64) <= np.abs(g64) * 2.0 ** -8)
    rms = np.sqrt(np.mean(p64["out"] ** 2))
    d = np.abs(p16["out"] - p64["out"])
    assert 0.0 < np.max(d) < 0.05 * rms
    with pytest.raises(ValueError):
        oracle.pvconv_forward(wl.coords, wl.feats, L, stage_dtype="f16")


# ----------------------------------------------------------------------------
# PointNet++ primitives of PVCNN++ (Section 5.2 "Models")
# ----------------------------------------------------------------------------
def test_fps_on_a_line_follows_the_halving_order():
    # nine points at x = 0..8: after 0 the farthest is 8, then 4, then 2 and
    # 6 (equal: the lower index first), then 1, 3, 5, 7
    xyz = np.zeros((1, 9, 3), np.float32)
    xyz[0, :, 0] = np.arange(9)
    assert oracle.fps(xyz, 9)[0].tolist() == [0, 8, 4, 2, 6, 1, 3, 5, 7]
    assert oracle.fps(xyz, 3)[0].tolist() == [0, 8, 4]


def test_fps_each_pick_is_the_farthest_from_the_picks_before_it():
    from scipy.spatial.distance import cdist
    rng = np.random.default_rng(11)
    xyz = rng.random((2, 300, 3)).astype(np.float32)
    idx = oracle.fps(xyz, 40)
    for b in range(2):
        pts = xyz[b].astype(np.float64)
        picks = idx[b].tolist()
        assert picks[0] == 0 and len(set(picks)) == len(picks)
        for s in range(1, len(picks)):
            dmin = cdist(pts, pts[picks[:s]]).min(axis=1)
            assert picks[s] == int(np.argmax(dmin)), (b, s)


def _lattice(rng, B, N, step=1.0 / 8):
    """Points on a lattice of spacing 1/8 in [0, 2): every coordinate
    difference and squared distance is exact in fp32 and fp64."""
    return (rng.integers(0, 16, size=(B, N, 3)) * step).astype(np.float32)


def test_ball_query_matches_a_kd_tree():
    from scipy.spatial import cKDTree
    rng = np.random.default_rng(12)
    xyz = _lattice(rng, 2, 400)
    centers = _lattice(rng, 2, 30)
    # radius^2 = 0.1 is no multiple of 1/64: no point lies on a sphere
    radius, nsample = np.float32(np.sqrt(0.1)), 16
    idx = oracle.ball_query(xyz, centers, radius, nsample)
    for b in range(2):
        tree = cKDTree(xyz[b].astype(np.float64))
        for i in range(30):
            near = sorted(tree.query_ball_point(centers[b, i].astype(np.float64),
                                                float(radius)))[:nsample]
            want = near + [near[0] if near else 0] * (nsample - len(near))
            assert idx[b, i].tolist() == want, (b, i)


def test_ball_query_with_no_neighbour_fills_point_zero():
    xyz = np.zeros((1, 5, 3), np.float32)
    centers = np.full((1, 1, 3), 5.0, np.float32)
    assert oracle.ball_query(xyz, centers, 1.0, 4)[0, 0].tolist() == [0, 0, 0, 0]


def test_group_rows_are_relative_coordinates_then_features():
    rng = np.random.default_rng(13)
    xyz = _lattice(rng, 2, 64)
    feats = rng.normal(size=(2, 64, 5))
    cidx = oracle.fps(xyz, 8)
    centers = oracle.gather_points(xyz, cidx)
    idx = oracle.ball_query(xyz, centers, 0.5, 6)
    g = oracle.group(xyz, feats, centers, idx)
    assert g.shape == (2, 8, 6, 8)
    for b in range(2):
        nb = xyz[b][idx[b]]
        np.testing.assert_array_equal(g[b, ..., :3] + centers[b][:, None, :], nb)
        np.testing.assert_array_equal(g[b, ..., 3:], feats[b][idx[b]])
    # wherever a centre appears among its own neighbours, its row is (0, 0, 0, f_c)
    own = idx == cidx[:, :, None]
    assert own.any()
    assert np.all(g[own][:, :3] == 0.0)


def test_three_nn_matches_a_kd_tree_and_weights_sum_to_one():
    from scipy.spatial import cKDTree
    rng = np.random.default_rng(14)
    known = rng.random((2, 50, 3)).astype(np.float32)
    unknown = rng.random((2, 200, 3)).astype(np.float32)
    idx, w = oracle.three_nn(unknown, known)
    for b in range(2):
        d, j = cKDTree(known[b].astype(np.float64)).query(unknown[b].astype(np.float64), k=3)
        np.testing.assert_array_equal(idx[b], j)
        inv = 1.0 / (d + 1e-8)
        np.testing.assert_allclose(w[b], inv / inv.sum(axis=1, keepdims=True), rtol=1e-6)
    np.testing.assert_allclose(w.sum(axis=2), 1.0, rtol=1e-12)
    # an unknown point on a known one takes (nearly) all its weight from it
    idx2, w2 = oracle.three_nn(known[:, :5], known)
    assert np.array_equal(idx2[:, :, 0], np.tile(np.arange(5), (2, 1)))
    assert np.all(w2[:, :, 0] > 1.0 - 1e-6)


def test_three_interpolate_is_linear_and_keeps_constants():
    rng = np.random.default_rng(15)
    known = rng.random((1, 20, 3)).astype(np.float32)
    unknown = rng.random((1, 70, 3)).astype(np.float32)
    idx, w = oracle.three_nn(unknown, known)
    F, G = rng.normal(size=(1, 20, 4)), rng.normal(size=(1, 20, 4))
    np.testing.assert_allclose(oracle.three_interpolate(2.5 * F + G, idx, w),
                               2.5 * oracle.three_interpolate(F, idx, w) +
                               oracle.three_interpolate(G, idx, w), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.three_interpolate(np.full((1, 20, 3), 7.0), idx, w), 7.0,
                               rtol=1e-12)
    # one-hot features give back each neighbour's weight
    onehot = np.eye(20)[None]
    out = oracle.three_interpolate(onehot, idx, w)
    for i in range(70):
        for k in range(3):
            assert out[0, i, idx[0, i, k]] == pytest.approx(w[0, i, k], rel=1e-12)


def test_pvcnn2_concat_puts_the_interpolation_first_and_stores_bf16():
    import copy
    wl = synth.make_workload(6, B=1, N=2048)
    out16, lv = oracle.pvcnn2_forward(wl, "bf16", return_levels=True)
    for s in lv["skips"] + lv["props"]:
        np.testing.assert_array_equal(oracle.round_bf16(s), s)
    out64 = oracle.pvcnn2_forward(wl)
    rms = np.sqrt(np.mean(out64 ** 2))
    assert 0.0 < np.max(np.abs(out16 - out64)) < 0.1 * rms
    # the last propagation level's first layer sees [interpolated | skip]:
    # with zero weights on the interpolated columns, the coarse levels (here
    # perturbed through the deepest MLP's weights) no longer matter
    wl2 = copy.deepcopy(wl)
    lp = wl2.fp[-1].mlps[0]
    c_interp = lp.w.shape[1] - lv["skips"][0].shape[2]
    lp.w[:, :c_interp] = 0.0
    a = oracle.pvcnn2_forward(wl2)
    wl2.sa[-1].mlps[-1].w *= 3.0
    np.testing.assert_array_equal(oracle.pvcnn2_forward(wl2), a)
    # ... while with the skip columns zeroed instead, they do
    wl3 = copy.deepcopy(wl)
    wl3.fp[-1].mlps[0].w[:, c_interp:] = 0.0
    b3 = oracle.pvcnn2_forward(wl3)
    wl3.sa[-1].mlps[-1].w *= 3.0
    assert np.max(np.abs(oracle.pvcnn2_forward(wl3) - b3)) > 0.0
