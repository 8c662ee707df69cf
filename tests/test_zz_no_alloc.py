"""GPU test of gradlev_scan_fwd_static, the forward scan that allocates
nothing: its scratch is the library's static per-device array.

Two calls in a row, the second with a smaller input (the array keeps the
first call's contents), each compared with gradlev_scan_fwd on the same
inputs (the same kernels and plan: bitwise equal) and with the float64
oracle (the parity tolerance), for the chunked 64 x 64 and 128 x 128 scans
with forced multi-segment carries and for a wide map (parallel form).
"""

import numpy as np
import pytest

from oracle import gradlev_oracle as orc
from paper_2609_34174_amd import workloads as W
from parity_util import check, log, to_dev, to_host

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2609_34174_amd as gl  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no ROCm GPU visible")
    gl.lib()
    yield
    torch.cuda.synchronize()


def inputs(B, H, T, d, m, dtype, seed):
    rng = np.random.default_rng(seed)
    W0 = (rng.standard_normal((H, m, d)) * d ** -0.5).astype(np.float32)
    X = W.quantise(rng.standard_normal((B, H, T, d)) * d ** -0.5, dtype)
    G = W.quantise(rng.standard_normal((B, H, T, m)) * 0.1, dtype)
    eta = rng.uniform(0.0, 0.2, (B, H, T)).astype(np.float32)
    return W0, X, G, eta


# (B, H, T, d, m, dtype, segment): first call, then a smaller second call.
CASES = [
    ((4, 8, 1000, 64, 64, "bf16", 128), (2, 4, 300, 64, 64, "bf16", 64)),
    ((2, 4, 777, 128, 128, "f32", 128), (1, 3, 130, 128, 128, "f32", 64)),
    ((2, 1, 300, 256, 128, "bf16", 0), (1, 1, 129, 128, 256, "bf16", 0)),
]


@pytest.mark.parametrize("first,second", CASES)
def test_static_forward_matches_workspace_forward(first, second):
    for k, (B, H, T, d, m, dt, seg) in enumerate((first, second)):
        log(f"static forward call {k + 1}: B={B} H={H} T={T} d={d} m={m} {dt} segment={seg}")
        W0, X, G, eta = inputs(B, H, T, d, m, dt, seed=100 * k + d + m + T)
        dW0, dX, dG, de = to_dev(W0, "f32", torch), to_dev(X, dt, torch), to_dev(G, dt, torch), to_dev(eta, "f32", torch)
        s = gl.make_shape(B, H, T, d, m, gl.BF16 if dt == "bf16" else gl.F32, segment=seg)
        assert gl.workspace_bytes(s) <= gl.STATIC_SCRATCH_BYTES
        y_static = gl.scan_fwd_static(dW0, dX, dG, de, segment=seg)
        y_ws = gl.scan_fwd(dW0, dX, dG, de, segment=seg)
        torch.cuda.synchronize()
        ys, yw = to_host(y_static), to_host(y_ws)
        np.testing.assert_array_equal(ys, yw)
        check("y", ys, orc.scan_fwd(W0, X, G, eta), dt)
