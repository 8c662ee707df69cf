"""GPU parity of the two-map online MLP (Appendix A) against the oracle.

Forward: z_hat (first gated scan), h_hat = sigma(z_hat) stored in the input
dtype, y_hat (second gated scan).  Reverse: g_z = sigma'(z_hat) times the
transpose read of the second scan, and g_x through the first.  A further case
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
    gZ, gX = gl.mlp_reverse(*args, Z, Hid, dev(gY), mud, ald, rsd, act=act, segment=seg)
    torch.cuda.synchronize()
    kw = dict(kind=act, hidden_bf16=dtype == "bf16", reset=rs)
    f = orc.mlp_fwd(W10, W20, X, Gz, Gy, al, mu, **kw)
    r = orc.mlp_reverse(W10, W20, X, Gz, Gy, al, mu, gY, **kw)
    check("z", to_host(Z), f["z"], dtype)
    check("h", to_host(Hid), f["h"], dtype)
    check("y", to_host(Y), f["y"], dtype)
    check("gz", to_host(gZ), r["gz"], dtype)
    if dtype == "f32":
        check("gx", to_host(gX), r["gx"], dtype)
    else:
        # The hidden target meets the first scan in bf16 (as the library
        # stores it); the oracle rounds its own fp64 target the same way.
        gzq = orc.round_bf16(r["gz"])
        gx_ref = orc.scan_bwd(W10, X, Gz, mu / d, gzq, alpha=al, reset=rs)["gtilde"]
        check("gx", to_host(gX), gx_ref, dtype)


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
