"""GPU parity of the two-map online MLP (Appendix A) against the oracle.

Forward: z_hat (first gated scan), h_hat = sigma(z_hat) stored in the input
dtype, y_hat (second gated scan).  Reverse: g_z = sigma'(z_hat) times the
transpose read of the second scan, g_x through the first, and the training
gradients of the shared gates and the slow weights (writes detached).  A further case
feeds the serial learner's exact costates (fp32) and checks that the GPU
scans reproduce serial test-time training, as the paper's FP64 experiment
does on the CPU.
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


def q(a, dtype):
    return W.quantise(np.asarray(a, np.float64), dtype)


CASES = [("f32", "tanh", 64, 128, 64, 0), ("bf16", "tanh", 64, 128, 64, 64), ("bf16", "gelu", 128, 64, 128, 0),
         ("f32", "gelu", 64, 64, 128, 128), ("bf16", "tanh", 128, 128, 64, 0),
         ("f32", "gelu_tanh", 64, 128, 64, 0), ("bf16", "gelu_tanh", 64, 128, 128, 0),
         # wide maps (parallel form): both scans above 128 wide
         ("bf16", "gelu_tanh", 128, 256, 128, 0), ("f32", "tanh", 256, 384, 128, 0)]


@pytest.mark.parametrize("dtype,act,d,hid,o,seg", CASES)
def test_mlp_parity(dtype, act, d, hid, o, seg):
    log(f"mlp dtype={dtype} act={act} {d}->{hid}->{o} seg={seg}")
    rng = np.random.default_rng(d + hid + o)
    B, H, T = 2, 2, 230
    W10 = (rng.standard_normal((H, hid, d)) * d ** -0.5).astype(np.float32)
    W20 = (rng.standard_normal((H, o, hid)) * hid ** -0.5).astype(np.float32)
    X = q(rng.standard_normal((B, H, T, d)), dtype)
    Gz = q(rng.standard_normal((B, H, T, hid)) * 0.3, dtype)
    Gy = q(rng.standard_normal((B, H, T, o)) * 0.3, dtype)
    gY = q(rng.standard_normal((B, H, T, o)), dtype)
    al, mu = W.gate_tokens(B, H, T, d, d + 5)
    mu = mu * d            # the MLP divides by each map's input width itself
    rs = W.reset_flags(B, T, 9, mean_len=80)
    dev = lambda a, dt=dtype: to_dev(a, dt, torch)  # noqa: E731
    args = (dev(W10, "f32"), dev(W20, "f32"), dev(X), dev(Gz), dev(Gy))
    mud, ald, rsd = dev(mu, "f32"), dev(al, "f32"), torch.from_numpy(rs).to("cuda")
    Z, Hid, Y = gl.mlp_fwd(*args, mud, ald, rsd, act=act, segment=seg)
    gZ, gX, gr = gl.mlp_reverse(*args, Z, Hid, dev(gY), mud, ald, rsd, act=act, segment=seg, grads=gl.MLP_GRADS)
    torch.cuda.synchronize()
    kw = dict(kind=act, hidden_bf16=dtype == "bf16", reset=rs)
    f = orc.mlp_fwd(W10, W20, X, Gz, Gy, al, mu, **kw)
    # The hidden target meets the first scan in bf16 when the pipeline is bf16
    # (as the library stores it); the oracle rounds its own fp64 target alike.
    r = orc.mlp_reverse(W10, W20, X, Gz, Gy, al, mu, gY, target_bf16=dtype == "bf16", **kw)
    check("z", to_host(Z), f["z"], dtype)
    check("h", to_host(Hid), f["h"], dtype)
    check("y", to_host(Y), f["y"], dtype)
    check("gz", to_host(gZ), r["gz"], dtype)
    check("gx", to_host(gX), r["gx"], dtype)
    for k in gl.MLP_GRADS:
        check(k, to_host(gr[k]), r[k], dtype)


def test_mlp_gradient_subsets_are_bitwise_identical():
    """Each MLP training gradient requested alone equals the full call's."""
    rng = np.random.default_rng(12)
    B, H, T, d, hid, o = 2, 1, 150, 64, 128, 64
    W10 = (rng.standard_normal((H, hid, d)) * d ** -0.5).astype(np.float32)
    W20 = (rng.standard_normal((H, o, hid)) * hid ** -0.5).astype(np.float32)
    X, Gz, Gy, gY = (q(rng.standard_normal((B, H, T, w)) * sc, "bf16")
                     for w, sc in ((d, 1.0), (hid, 0.3), (o, 0.3), (o, 1.0)))
    al, mu = W.gate_tokens(B, H, T, d, 13)
    dev = lambda a, dt="bf16": to_dev(a, dt, torch)  # noqa: E731
    args = (dev(W10, "f32"), dev(W20, "f32"), dev(X), dev(Gz), dev(Gy))
    mud, ald = dev(mu * d, "f32"), dev(al, "f32")
    Z, Hid, _ = gl.mlp_fwd(*args, mud, ald, act="gelu_tanh")
    gz0, gx0, full = gl.mlp_reverse(*args, Z, Hid, dev(gY), mud, ald, act="gelu_tanh", grads=gl.MLP_GRADS)
    gz1, _ = gl.mlp_reverse(*args, Z, Hid, dev(gY), mud, ald, act="gelu_tanh", with_gx=False)
    np.testing.assert_array_equal(to_host(gz1), to_host(gz0))
    for k in gl.MLP_GRADS:
        _, _, part = gl.mlp_reverse(*args, Z, Hid, dev(gY), mud, ald, act="gelu_tanh", with_gx=False, grads=(k,))
        np.testing.assert_array_equal(to_host(part[k]), to_host(full[k]), err_msg=k)


def test_mlp_scans_reproduce_serial_ttt():
    """Exact costates from serial TTT (fp64 oracle, 64 -> 128 -> 64, tanh, the
    paper's gate family) fed to the GPU scans in fp32: outputs, hidden and
    input costates match the serial learner to fp32 rounding."""
    log("mlp serial recovery on the GPU")
    rng = np.random.default_rng(7)
    T, d, hid, o = 256, 64, 128, 64
    W10 = rng.normal(0, 0.5 / np.sqrt(d), (hid, d))
    W20 = rng.normal(0, 0.5 / np.sqrt(hid), (o, hid))
    va, vm = rng.normal(0, 0.25, d), rng.normal(0, 0.25, d)
    X, C = rng.standard_normal((T, d)), rng.standard_normal((T, o))
    al = 1 / (1 + np.exp(-(X @ va / np.sqrt(d) + 1.5)))
    mu = 1 / (1 + np.exp(-(X @ vm / np.sqrt(d) - 0.2)))
    # fp32-representable inputs so that both sides see the same values
    W10, W20, X, C, al, mu = (np.asarray(a, np.float32).astype(np.float64) for a in (W10, W20, X, C, al, mu))
    ser = orc.mlp_serial(W10, W20, X, C, al, mu)
    Gz, Gy = (np.asarray(ser[k], np.float32).astype(np.float64) for k in ("gz", "gy"))
    b = lambda a: a[None, None]  # noqa: E731
    args = (to_dev(W10[None], "f32", torch), to_dev(W20[None], "f32", torch), to_dev(b(X), "f32", torch),
            to_dev(b(Gz), "f32", torch), to_dev(b(Gy), "f32", torch))
    mud, ald = to_dev(b(mu), "f32", torch), to_dev(b(al), "f32", torch)
    Z, Hid, Y = gl.mlp_fwd(*args, mud, ald, act="tanh")
    # The output costate is the serial learner's (exact, as in the paper's
    # experiment), not one derived from the GPU's own outputs.
    gy = np.asarray(ser["gy"], np.float32).astype(np.float64)
    gZ, gX = gl.mlp_reverse(*args, Z, Hid, to_dev(b(gy), "f32", torch), mud, ald, act="tanh")
    torch.cuda.synchronize()
    check("y", to_host(Y)[0, 0], ser["y"], "f32")
    check("gz", to_host(gZ)[0, 0], ser["gz"], "f32")
    check("gx", to_host(gX)[0, 0], ser["gx"], "f32")
