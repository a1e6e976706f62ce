"""The oracle's C code run under AddressSanitizer and UndefinedBehaviorSanitizer
(host build, gcc): every function on small inputs, in a child process that
preloads the ASan runtime. A memory error or undefined behaviour makes the
child fail."""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import dataclasses
import numpy as np
import oracle, synth
rng = np.random.default_rng(0)
# every C function of the oracle on small inputs (the compositions in
# oracle/__init__.py only chain these)
wl = synth.make_workload(2, B=2, N=200)
L = dataclasses.replace(synth.draw_pvconv(rng, 16, 32, 8, 2, bf16=True))
f = np.ascontiguousarray(wl.feats[..., :16])
parts = oracle.pvconv_forward(wl.coords, f, L, return_parts=True, stage_dtype="bf16")
oracle.pvconv_forward(wl.coords, f, dataclasses.replace(L, devox="nearest"))
oracle.layer_backward_features(wl.coords, f, L, rng.normal(size=parts["out"].shape))
oracle.conv3d_backward_weight(rng.normal(size=(2, 8 ** 3, 32)), parts["grid"], 8)
oracle.conv3d_at(parts["grid"], L.conv_w[0], 8, np.array([0, 5, 8 ** 3 - 1]))
oracle.devoxelize_weights(parts["pnorm"][0], 8)
oracle.maxpool(f)
x = rng.random((2, 300, 3)).astype(np.float32)
i = oracle.fps(x, 300)
c = oracle.gather_points(x, i[:, :40])
nb = oracle.ball_query(x, c, 0.2, 16)
oracle.ball_query(x, c, 0.0, 3)
oracle.group(x, rng.normal(size=(2, 300, 5)), c, nb)
ni, nw = oracle.three_nn(x, c)
oracle.three_interpolate(rng.normal(size=(2, 40, 6)), ni, nw)
print("sanitized oracle ok")
"""


@pytest.mark.skipif(sys.platform != "linux", reason="gcc sanitizers on Linux")
def test_oracle_runs_clean_under_asan_and_ubsan(tmp_path):
    lib = oracle.build(sanitize=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True, check=True).stdout.strip()
    if not os.path.isabs(asan):
        pytest.skip("libasan not found")
    env = dict(os.environ, PV_ORACLE_LIB=lib, LD_PRELOAD=asan, OMP_NUM_THREADS="2",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1",
               PYTHONPATH=ROOT + os.pathsep + os.environ.get("PYTHONPATH", ""))
    r = subprocess.run([sys.executable, "-c", CHILD], capture_output=True, text=True, env=env,
                       timeout=600, cwd=str(tmp_path))
    assert r.returncode == 0, r.stderr[-4000:]
    assert "sanitized oracle ok" in r.stdout
