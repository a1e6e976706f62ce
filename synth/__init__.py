"""Seeded synthetic inputs shaped like the paper's workloads.

This module is shared by the CPU oracle tests, the GPU parity tests and the
benchmark. It holds no step of PVConv itself: only point sampling on synthetic
surfaces, feature and parameter draws, and the bf16 rounding that turns drawn
weights into the values both sides then use.

The paper evaluates on ShapeNet Part (2048 points per shape, batch 8; Section 5.1
"Setups") and S3DIS (4096-point blocks, 32768 points per batch; Section 5.2
"Setups"). Neither dataset is used here: seeded surface samples of random
primitives stand in for part-segmentation shapes, and seeded synthetic rooms
stand in for indoor scene blocks.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Dict, List, Optional

import numpy as np

BN_EPS = 1e-5
LEAKY_SLOPE = 0.1


# ----------------------------------------------------------------------------
# bf16 rounding of drawn parameters (round to nearest even on the fp32 bits)
# ----------------------------------------------------------------------------
def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Return float32 values that are exactly representable in bfloat16 (RNE)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    u = (u + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)
    return u.astype(np.uint32).view(np.float32).reshape(a.shape)


# ----------------------------------------------------------------------------
# geometry helpers
# ----------------------------------------------------------------------------
def _random_rotation(rng: np.random.Generator) -> np.ndarray:
    q = rng.normal(size=4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array([
        [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
        [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
        [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)],
    ])


def _sample_box_faces(rng, n, lo, hi, faces=(0, 1, 2, 3, 4, 5)):
    """n points uniform over the chosen faces of the axis-aligned box [lo, hi].

    Face f: axis f // 2, at lo (f even) or hi (f odd).
    """
    lo = np.asarray(lo, float)
    hi = np.asarray(hi, float)
    ext = hi - lo
    areas = []
    for f in faces:
        ax = f // 2
        o = [a for a in range(3) if a != ax]
        areas.append(ext[o[0]] * ext[o[1]])
    areas = np.asarray(areas)
    which = rng.choice(len(faces), size=n, p=areas / areas.sum())
    pts = lo + rng.random((n, 3)) * ext
    for i, f in enumerate(faces):
        sel = which == i
        ax = f // 2
        pts[sel, ax] = lo[ax] if f % 2 == 0 else hi[ax]
    return pts


def _sample_primitive(rng, kind, n):
    """Points on the surface of one primitive centred at the origin; also its area."""
    if kind == 0:  # sphere
        r = rng.uniform(0.2, 0.6)
        v = rng.normal(size=(n, 3))
        v /= np.linalg.norm(v, axis=1, keepdims=True)
        return v * r
    if kind == 1:  # box
        h = rng.uniform(0.1, 0.5, size=3)
        return _sample_box_faces(rng, n, -h, h)
    # cylinder along z
    r = rng.uniform(0.1, 0.4)
    hh = rng.uniform(0.3, 1.0) / 2
    a_side = 2 * np.pi * r * (2 * hh)
    a_cap = np.pi * r * r
    part = rng.choice(3, size=n, p=np.array([a_side, a_cap, a_cap]) / (a_side + 2 * a_cap))
    th = rng.uniform(0, 2 * np.pi, size=n)
    pts = np.empty((n, 3))
    side = part == 0
    pts[side, 0] = r * np.cos(th[side])
    pts[side, 1] = r * np.sin(th[side])
    pts[side, 2] = rng.uniform(-hh, hh, size=side.sum())
    cap = ~side
    rr = r * np.sqrt(rng.random(cap.sum()))
    pts[cap, 0] = rr * np.cos(th[cap])
    pts[cap, 1] = rr * np.sin(th[cap])
    pts[cap, 2] = np.where(part[cap] == 1, -hh, hh)
    return pts


# ----------------------------------------------------------------------------
# cloud generators: each returns coords [B][N][3] float32 (and extras)
# ----------------------------------------------------------------------------
def uniform_cube(rng, B, N):
    """xyz uniform in [-1, 1]^3."""
    return rng.uniform(-1.0, 1.0, size=(B, N, 3)).astype(np.float32)


def part_shapes(rng, B, N):
    """Part-segmentation-like shapes: 1-4 random primitives (sphere, box,
    cylinder) per cloud, randomly rotated, centres in [-0.5, 0.5]^3, surface
    samples allotted evenly per primitive, plus N(0, 0.01^2) jitter."""
    out = np.empty((B, N, 3), np.float32)
    for b in range(B):
        n_prim = int(rng.integers(1, 5))
        alloc = rng.multinomial(N, np.full(n_prim, 1.0 / n_prim))
        pts = []
        for i in range(n_prim):
            kind = int(rng.integers(0, 3))
            p = _sample_primitive(rng, kind, int(alloc[i]))
            p = p @ _random_rotation(rng).T + rng.uniform(-0.5, 0.5, size=3)
            pts.append(p)
        p = np.concatenate(pts, axis=0)
        p += rng.normal(scale=0.01, size=p.shape)
        out[b] = p[rng.permutation(N)]
    return out


def rooms(rng, B, N):
    """Indoor-scene-like blocks: a room of L_x, L_y ~ U(3, 8) m and height 3 m
    (floor, ceiling and four walls) plus 5-15 clutter boxes with sides
    U(0.3, 1.5) m standing on the floor, sampled uniformly by area.

    Returns coords [B][N][3] and features [B][N][9] = (xyz, rgb ~ U[0,1],
    xyz / (L_x, L_y, 3))."""
    coords = np.empty((B, N, 3), np.float32)
    feats = np.empty((B, N, 9), np.float32)
    H = 3.0
    for b in range(B):
        Lx, Ly = rng.uniform(3.0, 8.0, size=2)
        surfaces = []  # (area, sampler)
        room_lo, room_hi = np.zeros(3), np.array([Lx, Ly, H])
        for f in range(6):
            ax = f // 2
            o = [a for a in range(3) if a != ax]
            area = (room_hi[o[0]]) * (room_hi[o[1]])
            surfaces.append((area, ("room", f)))
        n_box = int(rng.integers(5, 16))
        boxes = []
        for _ in range(n_box):
            s = rng.uniform(0.3, 1.5, size=3)
            x0 = rng.uniform(0, Lx - s[0])
            y0 = rng.uniform(0, Ly - s[1])
            lo = np.array([x0, y0, 0.0])
            hi = lo + s
            boxes.append((lo, hi))
            for f in (0, 1, 2, 3, 5):  # all faces except the one on the floor
                ax = f // 2
                o = [a for a in range(3) if a != ax]
                surfaces.append((s[o[0]] * s[o[1]], ("box", len(boxes) - 1, f)))
        areas = np.array([a for a, _ in surfaces])
        counts = rng.multinomial(N, areas / areas.sum())
        pts = []
        for (area, tag), c in zip(surfaces, counts):
            if c == 0:
                continue
            if tag[0] == "room":
                pts.append(_sample_box_faces(rng, int(c), room_lo, room_hi, faces=(tag[1],)))
            else:
                lo, hi = boxes[tag[1]]
                pts.append(_sample_box_faces(rng, int(c), lo, hi, faces=(tag[2],)))
        p = np.concatenate(pts, axis=0)[rng.permutation(N)]
        coords[b] = p
        feats[b, :, 0:3] = p
        feats[b, :, 3:6] = rng.random((N, 3))
        feats[b, :, 6:9] = p / np.array([Lx, Ly, H])
    return coords, feats


def clustered(rng, B, N):
    """Heavy-collision stress cloud: 80 % of the points from a mixture of 16
    anisotropic Gaussians (means U(-0.8, 0.8)^3, per-axis sigma log-uniform in
    [0.01, 0.06], random rotations), 20 % uniform in [-1, 1]^3."""
    out = np.empty((B, N, 3), np.float32)
    for b in range(B):
        n_cl = int(round(0.8 * N))
        comp = rng.integers(0, 16, size=n_cl)
        means = rng.uniform(-0.8, 0.8, size=(16, 3))
        sig = np.exp(rng.uniform(np.log(0.01), np.log(0.06), size=(16, 3)))
        rots = [_random_rotation(rng) for _ in range(16)]
        p = rng.normal(size=(n_cl, 3)) * sig[comp]
        for g in range(16):
            sel = comp == g
            p[sel] = p[sel] @ rots[g].T
        p += means[comp]
        u = rng.uniform(-1.0, 1.0, size=(N - n_cl, 3))
        out[b] = np.concatenate([p, u], axis=0)[rng.permutation(N)]
    return out


# ----------------------------------------------------------------------------
# parameters
# ----------------------------------------------------------------------------
@dataclasses.dataclass
class BNParams:
    gamma: np.ndarray
    beta: np.ndarray
    mean: np.ndarray
    var: np.ndarray
    eps: float = BN_EPS


def draw_bn(rng, C) -> BNParams:
    return BNParams(
        gamma=rng.uniform(0.5, 1.5, size=C).astype(np.float32),
        beta=rng.uniform(-0.5, 0.5, size=C).astype(np.float32),
        mean=rng.normal(0.0, 0.5, size=C).astype(np.float32),
        var=rng.uniform(0.5, 2.0, size=C).astype(np.float32),
    )


def kaiming_normal(rng, shape, fan_in, bf16):
    w = (rng.normal(size=shape) * np.sqrt(2.0 / fan_in)).astype(np.float32)
    return round_to_bf16(w) if bf16 else w


@dataclasses.dataclass
class PVConvParams:
    """One PVConv layer. Conv weights are [C_out][3][3][3][C_in] (offset-indexed,
    du, dv, dw in {-1, 0, 1} mapped to 0..2); the point-branch weight is
    [C_out][C_in]."""
    cin: int
    cout: int
    R: int
    conv_w: List[np.ndarray]
    conv_bn: List[BNParams]
    mlp_w: np.ndarray
    mlp_bn: BNParams
    mlp_b: Optional[np.ndarray] = None
    slope: float = LEAKY_SLOPE
    devox: str = "trilinear"   # or "nearest"

    @property
    def n_convs(self):
        return len(self.conv_w)


def draw_pvconv(rng, cin, cout, R, n_convs, bf16) -> PVConvParams:
    conv_w, conv_bn = [], []
    c = cin
    for _ in range(n_convs):
        conv_w.append(kaiming_normal(rng, (cout, 3, 3, 3, c), 27 * c, bf16))
        conv_bn.append(draw_bn(rng, cout))
        c = cout
    return PVConvParams(cin=cin, cout=cout, R=R, conv_w=conv_w, conv_bn=conv_bn,
                        mlp_w=kaiming_normal(rng, (cout, cin), cin, bf16),
                        mlp_bn=draw_bn(rng, cout))


@dataclasses.dataclass
class LinearParams:
    """Shared per-point Linear [C_out][C_in] (+ optional bias), then BN and ReLU
    unless it is the final logits layer (bn is None, relu False)."""
    w: np.ndarray
    b: Optional[np.ndarray]
    bn: Optional[BNParams]
    relu: bool


def draw_linear(rng, cin, cout, bf16, final=False) -> LinearParams:
    w = kaiming_normal(rng, (cout, cin), cin, bf16)
    if final:
        return LinearParams(w=w, b=rng.uniform(-0.1, 0.1, size=cout).astype(np.float32),
                            bn=None, relu=False)
    return LinearParams(w=w, b=None, bn=draw_bn(rng, cout), relu=True)


@dataclasses.dataclass
class SAParams:
    """One set-abstraction level of PVCNN++: PVConv layers on the level's
    points (possibly none), then npoint centres by farthest point sampling,
    nsample neighbours within radius, a shared MLP on the grouped rows
    (relative coordinates, then features) and the maximum over the
    neighbours."""
    pvconvs: List[PVConvParams]
    npoint: int
    radius: float
    nsample: int
    mlps: List[LinearParams]


@dataclasses.dataclass
class FPParams:
    """One feature-propagation level: the coarser level's features
    interpolated onto this level's points (three nearest neighbours),
    concatenated with this level's features, then a shared MLP."""
    mlps: List[LinearParams]


def draw_pvcnn2(rng, cin, width=1.0):
    """PVCNN++ for scene segmentation: PointNet++'s four set-abstraction and
    four feature-propagation levels, with a PVConv layer (two convolutions)
    on the points of each of the first three levels, then the head. Channel
    counts scale by `width` (the compact models' channel multiplier).

    Returns (sa levels, fp levels, head)."""
    w = lambda c: max(1, int(round(c * width)))
    sa_cfg = [  # npoint, radius (m), PVConv (cout, R) or None, MLP widths
        (1024, 0.2, (32, 32), [32, 32, 64]),
        (256, 0.4, (64, 16), [64, 64, 128]),
        (64, 0.8, (128, 8), [128, 128, 256]),
        (16, 1.6, None, [256, 256, 512]),
    ]
    sa, feat_widths, c = [], [], cin
    for npoint, radius, pvc, mlp in sa_cfg:
        pvconvs = []
        if pvc:
            pvconvs.append(draw_pvconv(rng, c, w(pvc[0]), pvc[1], 2, bf16=True))
            c = w(pvc[0])
        feat_widths.append(c)  # the level's features: the skip link of its FP level
        layers, ci = [], 3 + c
        for co in mlp:
            layers.append(draw_linear(rng, ci, w(co), True))
            ci = w(co)
        sa.append(SAParams(pvconvs, npoint, radius, 32, layers))
        c = ci
    fp = []
    for widths, skip in zip([[256, 256], [256, 256], [256, 128], [128, 128, 128]],
                            reversed(feat_widths)):
        layers, ci = [], c + skip
        for co in widths:
            layers.append(draw_linear(rng, ci, w(co), True))
            ci = w(co)
        fp.append(FPParams(layers))
        c = ci
    head = [draw_linear(rng, c, w(128), True), draw_linear(rng, w(128), 13, True, final=True)]
    return sa, fp, head


# ----------------------------------------------------------------------------
# the workloads
# ----------------------------------------------------------------------------
@dataclasses.dataclass
class Workload:
    index: int
    name: str
    B: int
    N: int
    dtype: str                        # "f32" or "bf16": the arithmetic the GPU path computes in
    coords: np.ndarray                # [B][N][3] float32
    feats: np.ndarray                 # [B][N][C_in] float32
    layers: List[PVConvParams]        # PVConv blocks in order
    mlps: List[LinearParams] = dataclasses.field(default_factory=list)   # point-only MLPs
    head: List[LinearParams] = dataclasses.field(default_factory=list)   # seg head
    n_classes: int = 0
    sa: List[SAParams] = dataclasses.field(default_factory=list)         # PVCNN++ levels
    fp: List[FPParams] = dataclasses.field(default_factory=list)

    @property
    def is_pvcnn2(self):
        return bool(self.sa)

    @property
    def is_network(self):
        return bool(self.head)

    def sha256(self) -> str:
        h = hashlib.sha256()
        h.update(self.coords.tobytes())
        h.update(self.feats.tobytes())
        for L in self.layers:
            for w in L.conv_w:
                h.update(w.tobytes())
            h.update(L.mlp_w.tobytes())
        for L in self.mlps + self.head:
            h.update(L.w.tobytes())
        for lev in self.sa:
            for L in lev.pvconvs:
                for w in L.conv_w:
                    h.update(w.tobytes())
                h.update(L.mlp_w.tobytes())
            for L in lev.mlps:
                h.update(L.w.tobytes())
        for lev in self.fp:
            for L in lev.mlps:
                h.update(L.w.tobytes())
        return h.hexdigest()


WORKLOAD_NAMES = {
    1: "pvconv_layer_fp32_B1_N1024_C16to32_R8",
    2: "pvconv_layer_bf16_B16_N2048_C64to128_R32",
    3: "pvcnn_partseg_bf16_B8_N2048",
    4: "pvcnn_sceneseg_bf16_B8_N4096",
    5: "pvconv_layer_bf16_B1_N65536_C64to64_R64_clustered",
    6: "pvcnn2_sceneseg_bf16_B4_N8192",
}


def make_workload(index: int, seed: Optional[int] = None, B: Optional[int] = None,
                  N: Optional[int] = None) -> Workload:
    """Build workload `index` (1..6) from seed 1000 + index unless given.

    B and N may be overridden to make reduced-size variants of the same shape
    family (the parity tests use that to keep the oracle within seconds)."""
    if seed is None:
        seed = 1000 + index
    rng = np.random.default_rng(seed)
    if index == 1:
        B_, N_ = B or 1, N or 1024
        coords = uniform_cube(rng, B_, N_)
        feats = rng.normal(size=(B_, N_, 16)).astype(np.float32)
        layers = [draw_pvconv(rng, 16, 32, 8, 1, bf16=False)]
        return Workload(1, WORKLOAD_NAMES[1], B_, N_, "f32", coords, feats, layers)
    if index == 2:
        B_, N_ = B or 16, N or 2048
        coords = part_shapes(rng, B_, N_)
        feats = rng.normal(size=(B_, N_, 64)).astype(np.float32)
        layers = [draw_pvconv(rng, 64, 128, 32, 2, bf16=True)]
        return Workload(2, WORKLOAD_NAMES[2], B_, N_, "bf16", coords, feats, layers)
    if index == 3:
        B_, N_ = B or 8, N or 2048
        coords = part_shapes(rng, B_, N_)
        feats = coords.copy()
        blocks = [(3, 64, 32), (64, 128, 16), (128, 128, 16)]
        layers = [draw_pvconv(rng, ci, co, r, 2, bf16=True) for ci, co, r in blocks]
        mlps = [draw_linear(rng, 128, 512, True), draw_linear(rng, 512, 2048, True)]
        cat = 64 + 128 + 128 + 512 + 2048 + 2048
        head = [draw_linear(rng, cat, 256, True), draw_linear(rng, 256, 128, True),
                draw_linear(rng, 128, 50, True, final=True)]
        return Workload(3, WORKLOAD_NAMES[3], B_, N_, "bf16", coords, feats, layers, mlps,
                        head, 50)
    if index == 4:
        B_, N_ = B or 8, N or 4096
        coords, feats = rooms(rng, B_, N_)
        blocks = [(9, 64, 32), (64, 64, 16), (64, 128, 16)]
        layers = [draw_pvconv(rng, ci, co, r, 2, bf16=True) for ci, co, r in blocks]
        mlps = [draw_linear(rng, 128, 1024, True)]
        cat = 64 + 64 + 128 + 1024 + 1024
        head = [draw_linear(rng, cat, 512, True), draw_linear(rng, 512, 256, True),
                draw_linear(rng, 256, 13, True, final=True)]
        return Workload(4, WORKLOAD_NAMES[4], B_, N_, "bf16", coords, feats, layers, mlps,
                        head, 13)
    if index == 5:
        B_, N_ = B or 1, N or 65536
        coords = clustered(rng, B_, N_)
        feats = rng.normal(size=(B_, N_, 64)).astype(np.float32)
        layers = [draw_pvconv(rng, 64, 64, 64, 2, bf16=True)]
        return Workload(5, WORKLOAD_NAMES[5], B_, N_, "bf16", coords, feats, layers)
    if index == 6:
        # PVCNN++ on indoor scenes: 4 x 8192 points (the batch the paper times
        # its scene-segmentation models on), 9 input channels, 13 classes
        B_, N_ = B or 4, N or 8192
        coords, feats = rooms(rng, B_, N_)
        sa, fp, head = draw_pvcnn2(rng, 9)
        return Workload(6, WORKLOAD_NAMES[6], B_, N_, "bf16", coords, feats, [], [], head, 13,
                        sa, fp)
    raise ValueError(f"unknown workload {index}")
