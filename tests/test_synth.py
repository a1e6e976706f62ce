"""The seeded generators produce what their recipes state."""
import numpy as np

import oracle
import synth


def test_generators_are_deterministic_and_shaped():
    for i, (B, N, C) in {1: (1, 1024, 16), 2: (16, 2048, 64), 3: (8, 2048, 3), 4: (8, 4096, 9),
                         5: (1, 65536, 64)}.items():
        a = synth.make_workload(i)
        assert a.coords.shape == (B, N, 3) and a.coords.dtype == np.float32
        assert a.feats.shape == (B, N, C) and a.feats.dtype == np.float32
        assert np.isfinite(a.coords).all() and np.isfinite(a.feats).all()
        if i in (2, 5):
            b = synth.make_workload(i)
            assert a.sha256() == b.sha256()


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 0.0], np.float32)
    r = synth.round_to_bf16(x)
    # 1+2^-8 is a tie between 1 and 1+2^-7: rounds to the even mantissa (1.0)
    assert r.tolist() == [1.0, 1.0, 1.0 + 2 ** -6, 1.0, -2.5, 0.0]
    w = synth.make_workload(2, B=1, N=64).layers[0].conv_w[0]
    assert np.all((w.view(np.uint32) & 0xFFFF) == 0)


def test_clustered_cloud_has_heavy_voxel_collisions():
    # the stress recipe: 80 % of the points fall within 5 % of the R=64 voxels
    wl = synth.make_workload(5)
    _, _, pn = oracle.normalize(wl.coords)
    ids = oracle.voxel_ids(pn, 64)[0]
    counts = np.sort(np.bincount(ids, minlength=64 ** 3))[::-1]
    need = np.searchsorted(np.cumsum(counts), 0.8 * wl.N) + 1
    assert need <= 0.05 * 64 ** 3
    assert counts[0] >= 20


def test_scene_features_are_xyz_rgb_and_room_normalised_xyz():
    wl = synth.make_workload(4, B=2, N=4096)
    f = wl.feats
    assert np.array_equal(f[..., :3], wl.coords)
    assert f[..., 3:6].min() >= 0 and f[..., 3:6].max() <= 1
    assert f[..., 6:9].min() >= -1e-6 and f[..., 6:9].max() <= 1 + 1e-6
