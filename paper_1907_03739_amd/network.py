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
