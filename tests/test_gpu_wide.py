"""GPU parity of the wide-map scans (the parallel form, widths above 128).

The HIP path runs through the C ABI (gated and unit-retention entry points,
the two-map MLP); the float64 oracle (the sequential learner of Section 3,
Eq. 2 general form) checks the forward outputs and every backward output
(gtilde, dX, dG, deta, dalpha, dW0).  Small cases compare every element, with ragged tails (T not a
multiple of the 128-token tile), T = 1, and the three retention modes the
kernels distinguish (none, resets only, general retention with exact zeros
and negative values).  The paper's adapted MLP at its LM width
(1024 -> 4096 -> 1024, 1024-token context, two sequences, unit retention with
document resets) is checked on sampled tokens against closed-form sums over
each token's document.
"""

import dataclasses

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


def inputs(B, H, T, d, m, dtype, seed, alpha_kind, eta_kind, with_reset):
    base = W.SCAN_WORKLOADS["lm-bf16"]
    wl = dataclasses.replace(base, B=B, H=H, T=T, d=d, m=m, dtype=dtype, x_dist="normal",
                             x_std=d ** -0.5, g_std=0.1, seed=seed)
    inp = W.scan_inputs(wl)
    a, e = W.gate_tokens(B, H, T, d, seed + 1)
    rng = np.random.default_rng(seed + 2)
    if alpha_kind == "family":
        inp["alpha"] = a
    elif alpha_kind == "uniform":
        al = rng.uniform(0, 1, (B, H, T)).astype(np.float32)
        al[..., ::11] = 0.0
        inp["alpha"] = al
    elif alpha_kind == "signed":
        al = rng.uniform(0.6, 1.0, (B, H, T)).astype(np.float32)
        al *= np.where(rng.uniform(size=(B, H, T)) < 0.1, -1, 1).astype(np.float32)
        inp["alpha"] = al
    else:
        inp["alpha"] = float(alpha_kind)
    inp["eta"] = e * 8 if eta_kind == "token" else 0.1
    inp["reset"] = W.reset_flags(B, T, seed + 3, mean_len=60) if with_reset else None
    return inp


def dev_inputs(inp, dtype):
    W0 = to_dev(inp["W0"], "f32", torch)
    X, G, dY = (to_dev(inp[k], dtype, torch) for k in ("X", "G", "dY"))
    eta, al = inp["eta"], inp["alpha"]
    e = to_dev(eta, "f32", torch) if isinstance(eta, np.ndarray) else eta
    a = to_dev(al, "f32", torch) if isinstance(al, np.ndarray) else al
    r = None if inp["reset"] is None else torch.from_numpy(inp["reset"]).to("cuda")
    return W0, X, G, dY, e, a, r


CASES = [
    ("f32", 256, 128, 300, "1", "scalar", False),
    ("bf16", 256, 128, 300, "1", "scalar", False),
    ("f32", 128, 384, 200, "1", "token", True),
    ("bf16", 384, 256, 333, "family", "token", True),
    ("f32", 256, 256, 129, "uniform", "token", False),
    ("bf16", 128, 256, 1, "family", "scalar", False),
    ("bf16", 512, 128, 128, "0.9", "token", True),
    ("f32", 128, 256, 250, "signed", "token", True),
    ("bf16", 256, 512, 700, "family", "token", True),
    # contractions of 1024 and 768 split four and two ways (fp32 partials)
    ("f32", 1024, 128, 200, "family", "token", True),
    ("bf16", 128, 768, 260, "uniform", "scalar", True),
]


# Every backward output of the wide path (unit-retention entry points have
# no dalpha).
WIDE_BWD = ("gtilde", "dx", "dg", "deta", "dalpha", "dw0")
UNIT_BWD = ("gtilde", "dx", "dg", "deta", "dw0")


@pytest.mark.parametrize("dtype,d,m,T,ak,ek,rs", CASES)
def test_wide_gated_parity(dtype, d, m, T, ak, ek, rs):
    log(f"wide gated dtype={dtype} d={d} m={m} T={T} alpha={ak} eta={ek} reset={rs}")
    inp = inputs(2, 2, T, d, m, dtype, seed=T + d + 3 * m, alpha_kind=ak, eta_kind=ek, with_reset=rs)
    W0, X, G, dY, e, a, r = dev_inputs(inp, dtype)
    y = gl.scan_fwd_gated(W0, X, G, e, a, r)
    out = gl.scan_bwd_gated(W0, X, G, dY, e, a, r, outputs=WIDE_BWD)
    torch.cuda.synchronize()
    kw = dict(alpha=inp["alpha"], reset=inp["reset"])
    args = (inp["W0"], inp["X"], inp["G"], inp["eta"])
    check("y", to_host(y), orc.scan_fwd(*args, **kw), dtype)
    ref = orc.scan_bwd(*args, inp["dY"], **kw)
    for k in WIDE_BWD:
        check(k, to_host(out[k]), ref[k], dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_wide_unit_entry_points(dtype):
    """The unit-retention entry points route wide shapes to the same kernels."""
    log(f"wide unit dtype={dtype}")
    inp = inputs(3, 1, 270, 128, 256, dtype, seed=11, alpha_kind="1", eta_kind="token", with_reset=False)
    W0, X, G, dY, e, _, _ = dev_inputs(inp, dtype)
    y = gl.scan_fwd(W0, X, G, e)
    out = gl.scan_bwd(W0, X, G, dY, e, outputs=UNIT_BWD)
    torch.cuda.synchronize()
    args = (inp["W0"], inp["X"], inp["G"], inp["eta"])
    check("y", to_host(y), orc.scan_fwd(*args), dtype)
    ref = orc.scan_bwd(*args, inp["dY"])
    for k in UNIT_BWD:
        check(k, to_host(out[k]), ref[k], dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_wide_output_subsets_are_bitwise_identical(dtype):
    """Each backward output requested alone (or in a subset) equals the same
    output of the full call bitwise: dX alone lands the read in dX itself,
    dalpha alone runs the gate pass without deta's reduction."""
    inp = inputs(2, 1, 333, 256, 128, dtype, seed=5, alpha_kind="family", eta_kind="token", with_reset=True)
    W0, X, G, dY, e, a, r = dev_inputs(inp, dtype)
    full = {k: to_host(v) for k, v in gl.scan_bwd_gated(W0, X, G, dY, e, a, r, outputs=WIDE_BWD).items()}
    for subset in (("dx",), ("dg",), ("dalpha",), ("deta", "dalpha"), ("gtilde", "dg"), ("dw0",)):
        log(f"  subset {subset}")
        part = gl.scan_bwd_gated(W0, X, G, dY, e, a, r, outputs=subset)
        for k in subset:
            np.testing.assert_array_equal(to_host(part[k]), full[k], err_msg=str(subset))


@pytest.mark.timeout(600)
def test_mlp_at_lm_width():
    """The paper's adapted final MLP at its LM shape: d = 1024, hidden = 4096,
    1024-token context, two sequences per GPU, bf16 activations, tanh-GELU,
    unit retention with document resets and the write gate of the gate family.
    Every output of both sequences (z, h, y, g_z, g_x) is checked against
    references built by the oracle alone: the explicit causal sums of the
    scan reads, with the oracle's own hidden activations (rounded to bf16 as
    the pipeline stores them) feeding the second map, and its own hidden
    target (rounded to bf16 before it queries the first map) feeding g_x."""
    B, H, T, d, hid, o = 2, 1, 1024, 1024, 4096, 1024
    log(f"mlp lm width B={B} T={T} {d}->{hid}->{o} bf16 gelu_tanh resets")
    rng = np.random.default_rng(2024)
    W10 = (rng.standard_normal((H, hid, d)) * d ** -0.5).astype(np.float32)
    W20 = (rng.standard_normal((H, o, hid)) * hid ** -0.5).astype(np.float32)
    X = W.quantise(rng.standard_normal((B, H, T, d)), "bf16")
    Gz = W.quantise(rng.standard_normal((B, H, T, hid)) * 0.3, "bf16")
    Gy = W.quantise(rng.standard_normal((B, H, T, o)) * 0.3, "bf16")
    gY = W.quantise(rng.standard_normal((B, H, T, o)), "bf16")
    _, mu = W.gate_tokens(B, H, T, 1, 77)        # mu = 4 sigmoid(b), the write strength
    rs = W.reset_flags(B, T, 78, mean_len=400)
    dv = lambda a, dt="bf16": to_dev(a, dt, torch)  # noqa: E731
    args = (dv(W10, "f32"), dv(W20, "f32"), dv(X), dv(Gz), dv(Gy))
    mud, rsd = dv(mu, "f32"), torch.from_numpy(rs).to("cuda")
    Z, Hid, Y = gl.mlp_fwd(*args, mud, 1.0, rsd, act="gelu_tanh")
    gZ, gX = gl.mlp_reverse(*args, Z, Hid, dv(gY), mud, 1.0, rsd, act="gelu_tanh")
    torch.cuda.synchronize()
    log("  oracle: explicit scan reads of both maps (float64)")
    e1, e2 = mu / d, mu / hid
    z = orc.scan_reads(W10, X, Gz, e1, reset=rs)["y"]
    h = orc.round_bf16(orc.act(z, "gelu_tanh"))
    r2 = orc.scan_reads(W20, h, Gy, e2, Bq=gY, reset=rs)
    gz = orc.act_grad(z, "gelu_tanh") * r2["gtilde"]
    gx = orc.scan_reads(W10, X, Gz, e1, Bq=orc.round_bf16(gz), reset=rs)["gtilde"]
    for k, out, ref in (("z", Z, z), ("h", Hid, h), ("y", Y, r2["y"]), ("gz", gZ, gz), ("gx", gX, gx)):
        check(k, to_host(out), ref, "bf16")


@pytest.mark.timeout(300)
def test_decode_at_lm_width():
    """Deployment steps of the paper's LM-width MLP maps (1024 -> 4096 and
    4096 -> 1024, fp32 states of 16 MiB per sequence), plain and gated with a
    document reset, against the float64 decode step of the oracle."""
    rng = np.random.default_rng(31)
    S, H, steps = 2, 1, 3
    for d, m in ((1024, 4096), (4096, 1024)):
        log(f"decode lm width {d}->{m}, S={S}, {steps} steps, plain then gated")
        W0 = (rng.standard_normal((H, m, d)) * d ** -0.5).astype(np.float32)
        for gated in (False, True):
            Wh = (W0[None] + 0.02 * rng.standard_normal((S, H, m, d))).astype(np.float32)
            Wd, W0d = to_dev(Wh, "f32", torch), to_dev(W0, "f32", torch)
            Wr = Wh.astype(np.float64)
            for step in range(steps):
                x = rng.standard_normal((S, H, d)).astype(np.float32)
                g = (rng.standard_normal((S, H, m)) * 0.1).astype(np.float32)
                eta = (rng.uniform(0.5, 1.5, (S, H)) / d).astype(np.float32)
                if gated:
                    al = rng.uniform(0.8, 1.0, (S, H)).astype(np.float32)
                    rs = np.array([0, 1 if step == 1 else 0], np.uint8)
                    y = gl.decode_step_gated(Wd, W0d, to_dev(x, "f32", torch), to_dev(g, "f32", torch),
                                             to_dev(eta, "f32", torch), to_dev(al, "f32", torch),
                                             torch.from_numpy(rs).to("cuda"))
                    yr, Wr = orc.decode_step(Wr, x, g, eta, alpha=al, W0=W0, reset=rs)
                else:
                    y = gl.decode_step(Wd, to_dev(x, "f32", torch), to_dev(g, "f32", torch), to_dev(eta, "f32", torch))
                    yr, Wr = orc.decode_step(Wr, x, g, eta)
                check("y", to_host(y), yr, "f32")
            check("W", to_host(Wd), Wr, "f32")


@pytest.mark.timeout(600)
def test_lm_width_training_gradients_sampled():
    """The first map of the paper's adapted MLP (1024 -> 4096) at its training
    shape: two 1024-token sequences, bf16, per-token step sizes from the gate
    family, unit retention, document resets.  The forward, the transpose read
    and the write-strength gradient of sampled tokens are checked against the
    closed forms of the sequential learner restricted to the token's
    document (W_read = W_0 minus the writes before it, R = the dY x^T sum
    after it), and dW0 = sum dY^T X in full."""
    B, H, T, d, m = 2, 1, 1024, 1024, 4096
    log(f"lm width training gradients B={B} T={T} {d}->{m} bf16 resets")
    rng = np.random.default_rng(99)
    W0 = (rng.standard_normal((H, m, d)) * d ** -0.5).astype(np.float32)
    X = W.quantise(rng.standard_normal((B, H, T, d)), "bf16")
    G = W.quantise(rng.standard_normal((B, H, T, m)) * 0.3, "bf16")
    dY = W.quantise(rng.standard_normal((B, H, T, m)), "bf16")
    _, eta = W.gate_tokens(B, H, T, d, 101)
    rs = W.reset_flags(B, T, 102, mean_len=400)
    dv = lambda a, dt="bf16": to_dev(a, dt, torch)  # noqa: E731
    args = (dv(W0, "f32"), dv(X), dv(G))
    y = gl.scan_fwd_gated(*args, dv(eta, "f32"), 1.0, torch.from_numpy(rs).to("cuda"))
    out = gl.scan_bwd_gated(*args, dv(dY), dv(eta, "f32"), 1.0, torch.from_numpy(rs).to("cuda"), outputs=UNIT_BWD)
    torch.cuda.synchronize()
    yh, gth, deh, dwh = to_host(y), to_host(out["gtilde"]), to_host(out["deta"]), to_host(out["dw0"])
    dxh, dgh = to_host(out["dx"]), to_host(out["dg"])
    picks = sorted({0, 1, 127, 128, 500, 1022, 1023, *rng.integers(0, T, 5).tolist()})
    got = {k: [] for k in ("y", "gtilde", "dx", "dg", "deta")}
    ref = {k: [] for k in got}
    for b in range(B):
        starts = np.nonzero(rs[b])[0].tolist() + [T]
        for t in picks:
            lo = max(s for s in starts if s <= t)
            hi = min(s for s in starts if s > t)
            W_read = W0[0].astype(np.float64) - orc.outer_sum(G[b, 0], X[b, 0], eta[b, 0], lo, t)
            R = orc.outer_sum(dY[b, 0], X[b, 0], 1.0, t + 1, hi)
            r = orc.token_outputs(W_read, R, X[b, 0, t], G[b, 0, t], eta[b, 0, t], dY[b, 0, t])
            # a token whose write the next document's reset drops has deta = 0
            de = 0.0 if hi == t + 1 and t + 1 < T else r["deta"]
            for k, g_, r_ in (("y", yh[b, 0, t], r["y"]), ("gtilde", gth[b, 0, t], r["gtilde"]),
                              ("dx", dxh[b, 0, t], r["dx"]), ("dg", dgh[b, 0, t], r["dg"]),
                              ("deta", deh[b, 0, t], de)):
                got[k].append(g_)
                ref[k].append(r_)
    for k in got:
        check(k, np.array(got[k]), np.array(ref[k]), "bf16")
    dw_ref = np.einsum("bhtm,bhtd->hmd", dY.astype(np.float64), X.astype(np.float64))
    check("dw0", dwh, dw_ref, "bf16")
