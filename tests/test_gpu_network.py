"""GPU parity of the PVCNN segmentation networks (part- and scene-shaped
workloads) against the fp64 oracle.

The networks store every stage's per-point output in bf16 ("bf16 weights and
activations"), so the oracle side rounds each stage output to bf16 at the same
stage boundaries before feeding the next stage; inside a stage it stays fp64.

* Stage by stage (teacher forcing): each GPU step gets the oracle's rounded
  input and is compared with the oracle's output of that step, with the
  tolerance of what the step is: a whole PVConv layer (a chain of bf16 steps),
  a single bf16 GEMM step, or an exact max.
* End to end: the GPU forward from the raw inputs against the oracle's
  rounded chain. Each of the S stages that store bf16 (PVConv blocks, point
  MLPs, hidden head layers) differs from the oracle by at most the chain
  bound 2e-2 (|ref| + rms) when fed identical inputs (the stage-by-stage
  test); batch norm keeps each layer's gain near one, and the stages' rounding
  and summation-order deviations are independent, so they add in quadrature:
  the end-to-end bound is sqrt(S) times the chain bound.
* Full size: the networks are per cloud (normalisation, voxel grids and the
  max-pool never mix clouds, batch norm is in inference mode), so the full
  B=8 forward is checked on two of its clouds, each run alone in the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_1907_03739_amd.network import DeviceNetwork
from _helpers import assert_bf16_chain, assert_bf16_step, dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu_case(request):
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    print(f"\n[gpu case] {request.node.nodeid}", flush=True)
    yield
    torch.cuda.synchronize()


def _oracle_chain(wl):
    """Oracle stage outputs (fp64) and their bf16-rounded copies, the global
    feature and the head outputs (hidden layers rounded to bf16, logits not)."""
    raw, rnd = [], []
    x = wl.feats
    for L in wl.layers:
        y = oracle.pvconv_forward(wl.coords, x, L)
        raw.append(y)
        x = oracle.round_bf16(y)
        rnd.append(x)
    for lp in wl.mlps:
        y = oracle.shared_mlp(x, lp)
        raw.append(y)
        x = oracle.round_bf16(y)
        rnd.append(x)
    g = oracle.maxpool(x)
    B, N = wl.B, wl.N
    h = np.concatenate(rnd + [np.broadcast_to(g[:, None, :], (B, N, g.shape[1]))], axis=2)
    heads = []
    for k, lp in enumerate(wl.head):
        y = oracle.shared_mlp(h, lp)
        heads.append(y)
        h = oracle.round_bf16(y) if k + 1 < len(wl.head) else y
    return raw, rnd, g, heads


def assert_network(got, ref, wl, what):
    stages = len(wl.layers) + len(wl.mlps) + len(wl.head) - 1
    d = np.abs(got - ref)
    rms = float(np.sqrt(np.mean(ref ** 2)))
    ratio = float(np.max(d / (np.abs(ref) + rms)))
    print(f"[{what}] max |d|/(|ref|+rms) = {ratio:.3g} (S = {stages})", flush=True)
    assert ratio <= 2e-2 * np.sqrt(stages), f"{what}: {ratio:.3g}"


def _net(wl):
    return DeviceNetwork(wl.layers, wl.mlps, wl.head, wl.B, wl.N)


@pytest.mark.parametrize("idx,N", [(3, 500), (4, 700)])
def test_network_stage_by_stage(idx, N):
    wl = synth.make_workload(idx, B=2, N=N)
    raw, rnd, g, heads = _oracle_chain(wl)
    net = _net(wl)
    coords = dev(wl.coords)
    nb = len(wl.layers)
    for i in range(nb):
        xin = dev(wl.feats) if i == 0 else dev(rnd[i - 1], torch.bfloat16)
        got = host(net.run_block(i, coords, xin))
        assert_bf16_chain(got, raw[i], f"wl{idx} pvconv block {i + 1}")
    for j in range(len(wl.mlps)):
        got = host(net.run_mlp(j, dev(rnd[nb + j - 1], torch.bfloat16)))
        assert_bf16_step(got, raw[nb + j], f"wl{idx} mlp {j + 1}")
    net.run_global(dev(rnd[-1], torch.bfloat16))
    assert np.array_equal(host(net.g), g), "global max-pool must be exact"
    stages = dev(np.concatenate(rnd, axis=2), torch.bfloat16)
    got = host(net.run_head(stages))
    assert got.shape == (wl.B, wl.N, wl.n_classes)
    # the head's hidden layers round to bf16 on both sides: a chain
    assert_bf16_chain(got, heads[-1], f"wl{idx} head")
    # first head layer alone: the split W_s s + W_g g equals W [s; g]
    assert_bf16_step(host(net.hidden[0]), heads[0], f"wl{idx} head layer 1")


@pytest.mark.parametrize("idx,N", [(3, 500), (4, 700)])
def test_network_end_to_end(idx, N):
    wl = synth.make_workload(idx, B=2, N=N)
    _, _, _, heads = _oracle_chain(wl)
    ref = oracle.network_forward(wl, stage_dtype="bf16")
    assert np.array_equal(ref, heads[-1])   # the test's chain is the oracle's network
    net = _net(wl)
    got = host(net.forward(dev(wl.coords), dev(wl.feats)))
    assert_network(got, ref, wl, f"wl{idx} logits")
    # repeatable: the same call again gives the same bits
    again = host(net.forward(dev(wl.coords), dev(wl.feats)))
    assert np.array_equal(got, again)


@pytest.mark.parametrize("idx", [3, 4])
def test_network_full_size_two_clouds(idx):
    wl = synth.make_workload(idx)
    net = _net(wl)
    got = host(net.forward(dev(wl.coords), dev(wl.feats)))
    for b in (0, 5):
        one = synth.make_workload(idx)
        one.B = 1
        one.coords = wl.coords[b:b + 1]
        one.feats = wl.feats[b:b + 1]
        ref = oracle.network_forward(one, stage_dtype="bf16")
        assert_network(got[b:b + 1], ref, wl, f"wl{idx} cloud {b} logits")


def test_network_rejects_a_head_of_the_wrong_width():
    wl = synth.make_workload(3, B=1, N=64)
    bad = list(wl.head)
    bad[0] = synth.LinearParams(w=wl.head[0].w[:, :100], b=None, bn=wl.head[0].bn, relu=True)
    with pytest.raises(ValueError):
        DeviceNetwork(wl.layers, wl.mlps, bad, wl.B, wl.N)


# ----------------------------------------------------------------------------
# PVCNN++ (Section 5.2 "Models": PointNet++ extended with PVConv)
# ----------------------------------------------------------------------------
def _pvcnn2_stages(wl):
    """bf16-stored stages on the longest path: PVConv layers, grouped rows
    and MLP layers of the set abstraction, interpolations and MLP layers of
    the feature propagation, the hidden head layer."""
    s = sum(len(lev.pvconvs) + 1 + len(lev.mlps) for lev in wl.sa)
    s += sum(1 + len(lev.mlps) for lev in wl.fp)
    return s + len(wl.head) - 1


def test_pvcnn2_full_size_two_clouds():
    from paper_1907_03739_amd.network import DevicePVCNN2
    wl = synth.make_workload(6)
    net = DevicePVCNN2(wl.sa, wl.fp, wl.head, wl.B, wl.N, wl.feats.shape[2])
    logits = host(net.forward(dev(wl.coords), dev(wl.feats)))
    S = _pvcnn2_stages(wl)
    for b in (0, wl.B - 1):
        one = synth.make_workload(6)
        one.B, one.coords, one.feats = 1, wl.coords[b:b + 1], wl.feats[b:b + 1]
        ref, lv = oracle.pvcnn2_forward(one, "bf16", return_levels=True)
        # the sampled points of every level: the same choices, bit for bit
        for l in range(1, len(lv["xyz"])):
            np.testing.assert_array_equal(net.xyz[l][b].cpu().numpy(), lv["xyz"][l][0])
        # level-0 features after the last propagation, then the logits
        got0 = host(net.props[0][b:b + 1])
        ref0 = lv["props"][-1]
        for got, want, what in ((got0, ref0, "features"), (logits[b:b + 1], ref, "logits")):
            d = np.abs(got - want)
            rms = float(np.sqrt(np.mean(want ** 2)))
            ratio = float(np.max(d / (np.abs(want) + rms)))
            print(f"[pvcnn2 cloud {b} {what}] max |d|/(|ref|+rms) = {ratio:.3g} (S = {S})",
                  flush=True)
            assert ratio <= 2e-2 * np.sqrt(S), f"cloud {b} {what}: {ratio:.3g}"


def test_pvcnn2_indices_of_every_level():
    from paper_1907_03739_amd.network import DevicePVCNN2
    wl = synth.make_workload(6, B=2, N=4096)
    net = DevicePVCNN2(wl.sa, wl.fp, wl.head, wl.B, wl.N, wl.feats.shape[2])
    net.forward(dev(wl.coords), dev(wl.feats))
    torch.cuda.synchronize()
    xyz = wl.coords
    for l, lev in enumerate(wl.sa):
        idx = oracle.fps(xyz, lev.npoint)
        np.testing.assert_array_equal(net.fps_idx[l].cpu().numpy(), idx)
        centers = oracle.gather_points(xyz, idx)
        np.testing.assert_array_equal(net.ball[l].cpu().numpy(),
                                      oracle.ball_query(xyz, centers, lev.radius, lev.nsample))
        nn_i, _ = oracle.three_nn(xyz, centers)
        np.testing.assert_array_equal(net.nn_idx[l].cpu().numpy(), nn_i)
        xyz = centers


def test_pvcnn2_forward_is_repeatable():
    from paper_1907_03739_amd.network import DevicePVCNN2
    wl = synth.make_workload(6, B=2, N=2048)
    net = DevicePVCNN2(wl.sa, wl.fp, wl.head, wl.B, wl.N, wl.feats.shape[2])
    c, f = dev(wl.coords), dev(wl.feats)
    a = net.forward(c, f).clone()
    b = net.forward(c, f)
    assert torch.equal(a, b)
