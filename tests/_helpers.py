"""Shared helpers for the GPU parity tests: device transfers and the
tolerance checks, each derived from the arithmetic it covers.

Tolerances
----------
* Integers (voxel ids, counts): bit-exact.
* fp32 results whose GPU arithmetic accumulates in fp64 before one final
  rounding (voxel means, normalised coordinates): rtol 1e-5.
* fp32 dot products (fp32 conv, fp32 MLP): |d| <= 1e-5 * (|ref| + mag), where
  mag is the same expression evaluated on absolute values (sum |w||x|, scaled
  by |BN scale|). Accumulating K products in fp32 has error <= K u mag in the
  worst case and about sqrt(K) u mag typically (u = 2^-24); for K <= 3456 the
  floor sits several standard deviations above the typical error.
* One bf16 step on identical inputs (bf16 conv, bf16 MLP, voxel grid stored
  as bf16): rtol 2e-2 with absolute floor 1e-3 (bf16 rounding of the output is
  2^-9 relative).
* A chain of bf16 steps compared against the all-fp64 oracle (a whole layer):
  each bf16 rounding of an intermediate perturbs its successors by up to 2^-9
  of their magnitude, and batch norm may move a value near zero after that,
  so the floor scales with the output's RMS: |d| <= 2e-2 * (|ref| + rms(ref)).
  An emulation of the bf16 roundings on the CPU gives max |d|/(|ref|+rms) of
  about 1e-2 on the part-segmentation layer.
"""
from __future__ import annotations

import numpy as np
import torch

import synth


def dev(a, dtype=torch.float32):
    return torch.as_tensor(np.ascontiguousarray(a), dtype=torch.float32).to("cuda").to(dtype)


def bf16_round(a):
    """fp64/fp32 numpy values rounded to the nearest bf16 (RNE), as float64."""
    return synth.round_to_bf16(np.asarray(a, np.float32)).astype(np.float64)


def host(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def dev_bn(bn):
    return (dev(bn.gamma), dev(bn.beta), dev(bn.mean), dev(bn.var), bn.eps)


def bn_scale(bn):
    return np.abs(bn.gamma.astype(np.float64)) / np.sqrt(bn.var.astype(np.float64) + bn.eps)


def _report(d, tol, what):
    bad = d > tol
    if bad.any():
        i = np.unravel_index(np.argmax(d - tol), d.shape)
        raise AssertionError(f"{what}: {bad.sum()} of {d.size} outside tolerance; worst at {i}: "
                             f"|d|={d[i]:.3g} tol={tol[i]:.3g}")


def assert_rel(gpu, ref, rtol=1e-5, what="fp32"):
    d = np.abs(gpu - ref)
    _report(d, rtol * np.abs(ref), what)


def assert_dot_f32(gpu, ref, mag, what="fp32 dot"):
    d = np.abs(gpu - ref)
    _report(d, 1e-5 * (np.abs(ref) + mag), what)


def assert_bf16_step(gpu, ref, what="bf16"):
    d = np.abs(gpu - ref)
    _report(d, 2e-2 * np.abs(ref) + 1e-3, what)


def assert_bf16_chain(gpu, ref, what="bf16 chain"):
    d = np.abs(gpu - ref)
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    if d.size:
        print(f"[{what}] max |d|/(|ref|+rms) = {float(np.max(d / (np.abs(ref) + rms))):.3g}",
              flush=True)
    _report(d, 2e-2 * (np.abs(ref) + rms), what)
