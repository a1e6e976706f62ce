"""PVCNN segmentation network on the library's kernels (Section 5.1 "Models":
PointNet with its per-point MLP layers replaced by PVConv; the part- and
scene-segmentation networks of Sections 5.1 and 5.2).

Every arithmetic step runs in libpvconv through the C-ABI calls of the
binding; this module only lays out device buffers and orders the calls.

Forward, for B clouds of N points:
  * the PVConv blocks, each feeding the next (Sections 4.1-4.3), then the
    point-only shared MLPs (Linear + BN + ReLU). Every block normalises the
    same coordinates, so the voxel indices are computed once per resolution:
    a block whose R an earlier block of the same forward used takes that
    block's indices and normalised coordinates (pvconv_forward_ex);
  * every stage writes its per-point output straight into its column range of
    one [B][N][C_stages] bf16 buffer, so the concatenation the head reads costs
    no copy;
  * a per-cloud max over the points of the last stage gives the global
    feature g [B][C_g];
  * the head's first layer acts on concat(stages, g broadcast to every point).
    Its weight splits column-wise into W_s (stage channels) and W_g (global
    channels): W [s; g] = W_s s + W_g g, and W_g g is one row per cloud, so it
    is computed once per cloud ([B] x [C_g] GEMM) and added to every point of
    that cloud in the epilogue of the W_s GEMM instead of broadcasting g into
    [B][N][C_g];
  * the remaining head layers, the last one giving fp32 logits.
Activations between stages are stored in bf16 and every GEMM accumulates in
fp32 (bf16 weights and activations).
"""
from __future__ import annotations

from typing import Callable, Optional

import torch

from . import binding as pv


class _Linear:
    """Device copy of one shared per-point layer: W [C_out][C_in] in bf16,
    optional bias and BN, ReLU or no activation."""

    def __init__(self, w, b, bn, relu: bool, device):
        f = lambda a: torch.as_tensor(a, dtype=torch.float32).to(device)
        self.w = f(w).to(torch.bfloat16).contiguous()
        self.b = f(b) if b is not None else None
        self.bn = (f(bn.gamma), f(bn.beta), f(bn.mean), f(bn.var), bn.eps) if bn is not None \
            else None
        self.act = "relu" if relu else "none"
        self.cout, self.cin = self.w.shape

    @classmethod
    def of(cls, lp, device):
        return cls(lp.w, lp.b, lp.bn, lp.relu, device)


class DeviceNetwork:
    """Device copy of a segmentation network's parameters and the buffers of
    one forward at fixed (B, N).

    layers: PVConv blocks (PVConvParams); mlps, head: LinearParams lists. The
    head's first layer takes C_stages + C_g inputs, C_g being the last stage's
    width."""

    def __init__(self, layers, mlps, head, B: int, N: int, device="cuda"):
        if not head:
            raise ValueError("a segmentation network needs a head")
        self.B, self.N = B, N
        self.blocks = [pv.DeviceLayer(L, device, torch.bfloat16) for L in layers]
        self.mlps = [_Linear.of(lp, device) for lp in mlps]
        widths = [L.cout for L in layers] + [m.cout for m in self.mlps]
        self.offsets = [sum(widths[:i]) for i in range(len(widths))]
        self.widths = widths
        self.c_stages = sum(widths)
        self.c_global = widths[-1]
        h0 = head[0]
        if h0.w.shape[1] != self.c_stages + self.c_global:
            raise ValueError("head input width must be C_stages + C_global")
        self.head0_s = _Linear(h0.w[:, :self.c_stages], h0.b, h0.bn, h0.relu, device)
        self.head0_g = _Linear(h0.w[:, self.c_stages:], None, None, False, device)
        self.head = [_Linear.of(lp, device) for lp in head[1:]]
        self.n_classes = (self.head[-1] if self.head else self.head0_s).cout

        bf = dict(dtype=torch.bfloat16, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        self.cat = torch.empty((B, N, self.c_stages), **bf)
        self.g = torch.empty((B, self.c_global), **f32)
        self.cloud_bias = torch.empty((B, self.head0_s.cout), **f32)
        hid = [self.head0_s] + self.head[:-1]
        self.hidden = [torch.empty((B, N, h.cout), **bf) for h in hid] if self.head else []
        self.logits = torch.empty((B, N, self.n_classes), **f32)
        ws = max(pv.pvconv_forward_workspace_size(B, N, L) for L in self.blocks)
        self.workspace = torch.empty(max(ws, 256), dtype=torch.uint8, device=device)
        # voxel indices per resolution, and the normalised coordinates
        self.ids = {R: torch.empty((B, N), dtype=torch.int32, device=device)
                    for R in {L.R for L in layers}}
        self.norm = torch.empty((B, N, 3), **f32)

    def stage_view(self, i: int) -> torch.Tensor:
        o, w = self.offsets[i], self.widths[i]
        return self.cat[:, :, o:o + w]

    # -- the steps, callable one by one (the tests feed each from the oracle) --
    def run_block(self, i: int, coords: torch.Tensor, feats: torch.Tensor,
                  reuse_ids: bool = False) -> torch.Tensor:
        """Block i. reuse_ids: take the voxel indices and normalised
        coordinates an earlier block at the same R wrote for these coords."""
        out = self.stage_view(i)
        pv.pvconv_forward(coords, feats, self.blocks[i], out=out, workspace=self.workspace,
                          vox_id=self.ids[self.blocks[i].params.R], norm=self.norm,
                          ids_given=reuse_ids)
        return out

    def _run_blocks(self, coords, x, marks=None):
        seen = set()
        for i, blk in enumerate(self.blocks):
            if marks:
                marks(f"pvconv{i + 1}")
            R = blk.params.R
            x = self.run_block(i, coords, x, reuse_ids=R in seen)
            seen.add(R)
        return x

    def run_mlp(self, j: int, x: torch.Tensor) -> torch.Tensor:
        m = self.mlps[j]
        out = self.stage_view(len(self.blocks) + j)
        pv.pvconv_point_mlp(x, m.w, bias=m.b, bn=m.bn, act=m.act, out=out)
        return out

    def run_global(self, last: torch.Tensor) -> torch.Tensor:
        """Per-cloud max-pool of the last stage, then W_g g per cloud."""
        pv.pvconv_maxpool(last, out=self.g)
        pv.pvconv_point_mlp(self.g, self.head0_g.w, act="none", out=self.cloud_bias)
        return self.g

    def run_head(self, stages: torch.Tensor) -> torch.Tensor:
        """stages: [B][N][C_stages] (the concatenated stage outputs)."""
        h0 = self.head0_s
        last = not self.head
        x = pv.pvconv_point_mlp(stages, h0.w, bias=h0.b, bn=h0.bn, act=h0.act,
                                cloud_bias=self.cloud_bias, points_per_cloud=self.N,
                                out=self.logits if last else self.hidden[0])
        for k, lin in enumerate(self.head):
            out = self.logits if k == len(self.head) - 1 else self.hidden[k + 1]
            x = pv.pvconv_point_mlp(x, lin.w, bias=lin.b, bn=lin.bn, act=lin.act, out=out)
        return x

    def forward(self, coords: torch.Tensor, feats: torch.Tensor) -> torch.Tensor:
        """coords [B][N][3] f32, feats [B][N][C_in] (f32 or bf16) -> logits
        [B][N][n_classes] f32 (a view of a buffer reused by the next call)."""
        x = self._run_blocks(coords, feats)
        for j in range(len(self.mlps)):
            x = self.run_mlp(j, x)
        self.run_global(x)
        return self.run_head(self.cat)

    def steps(self):
        """Names of the forward's steps in order (for per-step timing)."""
        return ([f"pvconv{i + 1}" for i in range(len(self.blocks))] +
                [f"mlp{j + 1}" for j in range(len(self.mlps))] + ["global", "head"])

    def forward_timed(self, coords, feats, marks: Callable[[Optional[str]], None]):
        """forward() with marks(name) called before each step and marks(None)
        after the last; used to place timing events between the steps."""
        x = self._run_blocks(coords, feats, marks)
        for j in range(len(self.mlps)):
            marks(f"mlp{j + 1}")
            x = self.run_mlp(j, x)
        marks("global")
        self.run_global(x)
        marks("head")
        out = self.run_head(self.cat)
        marks(None)
        return out


def _ceil8(c: int) -> int:
    return (c + 7) // 8 * 8


class DevicePVCNN2:
    """PVCNN++ (Section 5.2 "Models": PointNet++ extended with PVConv) on the
    library's kernels: device parameters and the buffers of one forward at
    fixed (B, N).

    Set abstraction level l (points xyz_l, N_l of them): its PVConv layers on
    the level's features; farthest point sampling of N_{l+1} centres (their
    coordinates are xyz_{l+1}); ball query; grouping into rows of relative
    coordinates and features, padded with zero columns to a multiple of 8
    channels (the first MLP layer's weight has zero columns there); the
    shared MLP; the maximum over each centre's neighbours. Feature
    propagation to level l: the three nearest level-(l+1) points of each
    level-l point, the interpolated features written into the first columns
    of the level's concat buffer, whose last columns already hold the
    level's skip features (its PVConv, or at the level without one the
    group maximum, writes them there), then the shared MLP. The head takes
    the level-0 features. Activations are bf16, accumulation fp32, logits
    fp32.

    sa, fp, head: synth.SAParams / FPParams / LinearParams lists; cin: the
    input feature width."""

    def __init__(self, sa, fp, head, B: int, N: int, cin: int, device="cuda"):
        if len(fp) != len(sa):
            raise ValueError("one feature-propagation level per set-abstraction level")
        self.B, self.N = B, N
        bf = dict(dtype=torch.bfloat16, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        i32 = dict(dtype=torch.int32, device=device)
        L = len(sa)
        self.L = L
        self.npts = [N] + [lev.npoint for lev in sa]
        self.sa = sa
        self.pvconvs = [[pv.DeviceLayer(p, device, torch.bfloat16) for p in lev.pvconvs]
                        for lev in sa]
        # widths: the features level l's set abstraction consumes (its skip
        # link), and the features each level hands down
        c_feat, c_in, c = [], [], cin
        for lev in sa:
            c_in.append(c)
            if lev.pvconvs:
                c = lev.pvconvs[-1].cout
            c_feat.append(c)
            c = lev.mlps[-1].w.shape[0]
        self.c_in, self.c_feat = c_in, c_feat
        c_deep = c
        # set-abstraction MLPs; the first takes the padded grouped rows
        self.sa_mlps = []
        self.group_w = []
        for l, lev in enumerate(sa):
            w0 = lev.mlps[0]
            wp = _ceil8(3 + c_feat[l])
            pad = torch.zeros((w0.w.shape[0], wp), dtype=torch.float32)
            pad[:, :3 + c_feat[l]] = torch.as_tensor(w0.w, dtype=torch.float32)
            first = _Linear(pad.numpy(), w0.b, w0.bn, w0.relu, device)
            self.sa_mlps.append([first] + [_Linear.of(lp, device) for lp in lev.mlps[1:]])
            self.group_w.append(wp)
        # feature propagation: level l = L-1 .. 0 takes c_interp[l] channels
        # interpolated from level l+1 plus c_feat[l] skip channels
        self.fp_mlps = [[_Linear.of(lp, device) for lp in lev.mlps] for lev in fp]
        self.c_interp = [0] * L
        c = c_deep
        for k in range(L):
            l = L - 1 - k
            self.c_interp[l] = c
            if self.fp_mlps[k][0].cin != c + c_feat[l]:
                raise ValueError(f"feature-propagation level {k}: input width mismatch")
            c = self.fp_mlps[k][-1].cout
        self.head = [_Linear.of(lp, device) for lp in head]
        self.n_classes = self.head[-1].cout

        # buffers
        # level coordinates: level 0 is the caller's (set by each forward)
        self.xyz = [None] + [torch.empty((B, n, 3), **f32) for n in self.npts[1:]]
        self.fps_idx = [torch.empty((B, n), **i32) for n in self.npts[1:]]
        self.ball = [torch.empty((B, lev.npoint, lev.nsample), **i32) for lev in sa]
        self.cat = [torch.empty((B, self.npts[l], self.c_interp[l] + c_feat[l]), **bf)
                    for l in range(L)]
        # the inputs of the PVConv layers of levels 1.. (the previous level's
        # group maximum); level 0 takes the caller's features
        self.pv_in = [None] + [torch.empty((B, self.npts[l], c_in[l]), **bf)
                               if sa[l].pvconvs else None for l in range(1, L)]
        self.deep = torch.empty((B, self.npts[L], c_deep), **bf)
        rows = max(B * lev.npoint * lev.nsample for lev in sa)
        self.grouped = [torch.zeros((B * lev.npoint * lev.nsample, self.group_w[l]), **bf)
                        for l, lev in enumerate(sa)]
        hid = max(m.cout for ms in self.sa_mlps for m in ms)
        self.sa_hidden = [torch.empty(rows * hid, **bf), torch.empty(rows * hid, **bf)]
        self.nn_idx = [torch.empty((B, self.npts[l], 3), **i32) for l in range(L)]
        self.nn_w = [torch.empty((B, self.npts[l], 3), **f32) for l in range(L)]
        fph = max(m.cout for ms in self.fp_mlps for m in ms)
        self.fp_hidden = [torch.empty(B * N * fph, **bf), torch.empty(B * N * fph, **bf)]
        self.props = [torch.empty((B, self.npts[l], self.fp_mlps[L - 1 - l][-1].cout), **bf)
                      for l in range(L)]
        self.head_hidden = [torch.empty((B, N, h.cout), **bf) for h in self.head[:-1]]
        self.logits = torch.empty((B, N, self.n_classes), **f32)
        ws = 256
        for l, lev in enumerate(self.pvconvs):
            for layer in lev:
                ws = max(ws, pv.pvconv_forward_workspace_size(B, self.npts[l], layer))
        self.workspace = torch.empty(ws, dtype=torch.uint8, device=device)
        # forward(): the coordinate-only steps (sampling, ball queries, three
        # nearest neighbours) on a second stream, at the default priority
        self.side = torch.cuda.Stream(device=device)
        self.sampled = [torch.cuda.Event() for _ in range(L)]
        self.nn_ready = torch.cuda.Event()

    def _hidden(self, bufs, k, rows, c):
        return bufs[k % 2][:rows * c].view(rows, c)

    def skip_view(self, l: int) -> torch.Tensor:
        return self.cat[l][:, :, self.c_interp[l]:]

    # -- the steps, callable one by one ----------------------------------------
    def run_pvconv(self, l: int, xyz: torch.Tensor, feats: torch.Tensor) -> torch.Tensor:
        """Level l's PVConv layers; the last writes the level's skip features."""
        layers = self.pvconvs[l]
        x = feats
        for k, layer in enumerate(layers):
            out = self.skip_view(l) if k == len(layers) - 1 else torch.empty(
                (self.B, self.npts[l], layer.params.cout), dtype=torch.bfloat16,
                device=feats.device)
            pv.pvconv_forward(xyz, x, layer, out=out, workspace=self.workspace)
            x = out
        return x

    def run_sample(self, l: int, xyz: torch.Tensor):
        """Centres of level l (farthest point sampling) and their neighbours."""
        lev = self.sa[l]
        pv.pvconv_furthest_point_sample(xyz, lev.npoint, idx=self.fps_idx[l],
                                        new_xyz=self.xyz[l + 1])
        pv.pvconv_ball_query(xyz, self.xyz[l + 1], lev.radius, lev.nsample, idx=self.ball[l])
        return self.xyz[l + 1], self.ball[l]

    def sa_target(self, l: int) -> torch.Tensor:
        """Where level l's set abstraction writes: the next level's PVConv
        input, its skip slice, or the deepest features."""
        if l + 1 == self.L:
            return self.deep
        if self.sa[l + 1].pvconvs:
            return self.pv_in[l + 1]
        return self.skip_view(l + 1)

    def run_group_mlp(self, l: int, xyz: torch.Tensor, feats: torch.Tensor,
                      centers: torch.Tensor, ball: torch.Tensor) -> torch.Tensor:
        """Grouping, the shared MLP and the maximum over the neighbours."""
        lev = self.sa[l]
        rows = self.B * lev.npoint * lev.nsample
        g = self.grouped[l]
        pv.pvconv_group_points(xyz, feats, centers, ball, out=g[:, :3 + feats.shape[2]])
        x = g
        for k, m in enumerate(self.sa_mlps[l]):
            out = self._hidden(self.sa_hidden, k, rows, m.cout)
            pv.pvconv_point_mlp(x, m.w, bias=m.b, bn=m.bn, act=m.act, out=out)
            x = out
        target = self.sa_target(l)
        # [B][M][C] rows (a column slice of a concat buffer is still a view)
        pv.pvconv_group_max(x, lev.nsample, out=target.view(-1, target.shape[2]))
        return target

    def run_three_nn(self, k: int):
        """The three nearest level-(l+1) points of each level-l point, l = L-1-k."""
        l = self.L - 1 - k
        pv.pvconv_three_nn(self.xyz[l], self.xyz[l + 1], idx=self.nn_idx[l], weight=self.nn_w[l])

    def run_fp(self, k: int, coarse: torch.Tensor, nn_done: bool = False) -> torch.Tensor:
        """Feature propagation k (to level L-1-k) from the coarser features
        (the three nearest neighbours found here unless nn_done)."""
        l = self.L - 1 - k
        if not nn_done:
            self.run_three_nn(k)
        pv.pvconv_three_interpolate(coarse, self.nn_idx[l], self.nn_w[l],
                                    out=self.cat[l][:, :, :self.c_interp[l]])
        x = self.cat[l]
        ms = self.fp_mlps[k]
        rows = self.B * self.npts[l]
        for j, m in enumerate(ms):
            out = self.props[l] if j == len(ms) - 1 else \
                self._hidden(self.fp_hidden, j, rows, m.cout).view(self.B, self.npts[l], m.cout)
            pv.pvconv_point_mlp(x, m.w, bias=m.b, bn=m.bn, act=m.act, out=out)
            x = out
        return x

    def run_head(self, x: torch.Tensor) -> torch.Tensor:
        for k, m in enumerate(self.head):
            out = self.logits if k == len(self.head) - 1 else self.head_hidden[k]
            x = pv.pvconv_point_mlp(x, m.w, bias=m.b, bn=m.bn, act=m.act, out=out)
        return x

    def steps(self):
        names = []
        for l, lev in enumerate(self.sa):
            if lev.pvconvs:
                names.append(f"pvconv{l + 1}")
            names += [f"sample{l + 1}", f"group_mlp{l + 1}"]
        return names + [f"fp{k + 1}" for k in range(self.L)] + ["head"]

    def forward_timed(self, coords: torch.Tensor, feats: torch.Tensor,
                      marks: Callable[[Optional[str]], None]) -> torch.Tensor:
        """forward() with marks(name) called before each step and marks(None)
        after the last."""
        self.xyz[0] = coords  # level 0 is the caller's points
        xyz, x = coords, feats
        for l, lev in enumerate(self.sa):
            if lev.pvconvs:
                marks(f"pvconv{l + 1}")
                x = self.run_pvconv(l, xyz, x)
            marks(f"sample{l + 1}")
            centers, ball = self.run_sample(l, xyz)
            marks(f"group_mlp{l + 1}")
            x = self.run_group_mlp(l, xyz, x, centers, ball)
            xyz = centers
        for k in range(self.L):
            marks(f"fp{k + 1}")
            x = self.run_fp(k, x)
        marks("head")
        out = self.run_head(x)
        marks(None)
        return out

    def forward(self, coords: torch.Tensor, feats: torch.Tensor) -> torch.Tensor:
        """coords [B][N][3] f32, feats [B][N][C_in] (f32 or bf16) -> logits
        [B][N][13] f32 (a view of a buffer reused by the next call).

        The same steps as forward_timed, on two streams: the sampling of
        every level and the nearest neighbours of the propagation, which
        depend on the coordinates alone, run on the side stream while the
        main stream runs the PVConv layers (farthest point sampling of a
        large cloud keeps one CU per cloud busy for a long sequential
        chain); the main stream waits for level l's sampling before level
        l's grouping, and for the neighbours before the propagation. The
        side stream first waits for the main stream's earlier work, so
        the buffers the previous forward still reads are not overwritten."""
        main = torch.cuda.current_stream(coords.device)
        self.xyz[0] = coords  # level 0 is the caller's points
        self.side.wait_stream(main)
        with torch.cuda.stream(self.side):
            xyz = coords
            for l in range(self.L):
                xyz, _ = self.run_sample(l, xyz)
                self.sampled[l].record(self.side)
            for k in range(self.L):
                self.run_three_nn(k)
            self.nn_ready.record(self.side)
        xyz, x = coords, feats
        for l, lev in enumerate(self.sa):
            if lev.pvconvs:
                x = self.run_pvconv(l, xyz, x)
            main.wait_event(self.sampled[l])
            x = self.run_group_mlp(l, xyz, x, self.xyz[l + 1], self.ball[l])
            xyz = self.xyz[l + 1]
        main.wait_event(self.nn_ready)
        for k in range(self.L):
            x = self.run_fp(k, x, nn_done=True)
        return self.run_head(x)
