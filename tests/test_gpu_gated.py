"""GPU parity of the gated scans and decode step (retention and resets).

The HIP path runs through the C ABI; the float64 oracle (sequential
definition of Eq. 2's general form) checks every output, dalpha included.
Tolerances are those of tests/parity_util.py (normwise per tensor).  Cases
span several chunks, forced segments and ragged tails; retentions cover the
paper's gate family, the full range [0, 1) with exact zeros, constant values,
and resets of packed documents.
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


KEYS = ("y", "gtilde", "dx", "dg", "deta", "dalpha", "dw0")


def inputs(B, H, T, d, m, dtype, seed, alpha_kind, eta_kind, with_reset):
    base = W.SCAN_WORKLOADS["lm-bf16"]
    wl = dataclasses.replace(base, B=B, H=H, T=T, d=d, m=m, dtype=dtype, x_dist="normal",
                             x_std=d ** -0.5, g_std=0.1, seed=seed)
    inp = W.scan_inputs(wl)
    a, e = W.gate_tokens(B, H, T, d, seed + 1)
    if alpha_kind == "family":
        inp["alpha"] = a
    elif alpha_kind == "uniform":
        al = np.random.default_rng(seed + 2).uniform(0, 1, (B, H, T)).astype(np.float32)
        al[..., ::11] = 0.0
        inp["alpha"] = al
    else:
        inp["alpha"] = float(alpha_kind)
    inp["eta"] = e * 8 if eta_kind == "token" else 0.1
    inp["reset"] = W.reset_flags(B, T, seed + 3, mean_len=60) if with_reset else None
    return inp


def run_gpu(inp, dtype, segment=0):
    W0 = to_dev(inp["W0"], "f32", torch)
    X, G, dY = (to_dev(inp[k], dtype, torch) for k in ("X", "G", "dY"))
    eta = inp["eta"]
    e = to_dev(eta, "f32", torch) if isinstance(eta, np.ndarray) else eta
    al = inp["alpha"]
    a = to_dev(al, "f32", torch) if isinstance(al, np.ndarray) else al
    r = None if inp["reset"] is None else torch.from_numpy(inp["reset"]).to("cuda")
    res = {"y": gl.scan_fwd_gated(W0, X, G, e, a, r, segment=segment)}
    res.update(gl.scan_bwd_gated(W0, X, G, dY, e, a, r, segment=segment))
    torch.cuda.synchronize()
    return {k: to_host(v) for k, v in res.items()}


def oracle_all(inp):
    args = (inp["W0"], inp["X"], inp["G"], inp["eta"])
    kw = dict(alpha=inp["alpha"], reset=inp["reset"])
    ref = {"y": orc.scan_fwd(*args, **kw)}
    ref.update(orc.scan_bwd(*args, inp["dY"], **kw))
    return ref


CASES = []
for dtype in ("f32", "bf16"):
    for (d, m) in ((64, 64), (128, 128), (64, 128), (128, 64)):
        for T, seg, ak, ek, rs in ((1, 0, "family", "scalar", False), (45, 0, "uniform", "token", False),
                                   (200, 64, "family", "token", True), (333, 128, "uniform", "scalar", False),
                                   (300, 64, "0.9", "token", True)):
            CASES.append((dtype, d, m, T, seg, ak, ek, rs))


@pytest.mark.parametrize("dtype,d,m,T,seg,ak,ek,rs", CASES)
def test_gated_parity(dtype, d, m, T, seg, ak, ek, rs):
    log(f"gated dtype={dtype} d={d} m={m} T={T} seg={seg} alpha={ak} eta={ek} reset={rs}")
    inp = inputs(2, 3, T, d, m, dtype, seed=T + d + 2 * m, alpha_kind=ak, eta_kind=ek, with_reset=rs)
    out = run_gpu(inp, dtype, segment=seg)
    ref = oracle_all(inp)
    for k in KEYS:
        check(k, out[k], ref[k], dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gated_unit_retention_matches_plain_scan(dtype):
    """alpha = 1 through the gated kernels agrees with the unit-retention kernels."""
    log(f"gated alpha=1 vs plain dtype={dtype}")
    inp = inputs(2, 2, 250, 64, 64, dtype, seed=71, alpha_kind="1.0", eta_kind="scalar", with_reset=False)
    g = run_gpu(inp, dtype, segment=64)
    W0 = to_dev(inp["W0"], "f32", torch)
    X, G, dY = (to_dev(inp[k], dtype, torch) for k in ("X", "G", "dY"))
    y = to_host(gl.scan_fwd(W0, X, G, 0.1, segment=64))
    p = {k: to_host(v) for k, v in gl.scan_bwd(W0, X, G, dY, 0.1, segment=64).items()}
    check("y", g["y"], y, dtype)
    for k in ("gtilde", "dx", "dg", "deta", "dw0"):
        check(k, g[k], p[k], dtype)


def test_gated_sixteen_segments_and_determinism():
    log("gated 16 segments, repeated")
    inp = inputs(1, 2, 1000, 64, 64, "bf16", seed=72, alpha_kind="family", eta_kind="token", with_reset=True)
    a = run_gpu(inp, "bf16", segment=64)
    b = run_gpu(inp, "bf16", segment=64)
    ref = oracle_all(inp)
    for k in KEYS:
        check(k, a[k], ref[k], "bf16")
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def test_gated_optional_outputs():
    log("gated optional outputs")
    inp = inputs(2, 2, 200, 64, 64, "bf16", seed=73, alpha_kind="uniform", eta_kind="token", with_reset=False)
    W0 = to_dev(inp["W0"], "f32", torch)
    X, G, dY = (to_dev(inp[k], "bf16", torch) for k in ("X", "G", "dY"))
    e, al = to_dev(inp["eta"], "f32", torch), to_dev(inp["alpha"], "f32", torch)
    full = {k: to_host(v) for k, v in gl.scan_bwd_gated(W0, X, G, dY, e, al).items()}
    for subset in (("dalpha",), ("gtilde", "deta"), ("dw0",), ("dx", "dg")):
        part = gl.scan_bwd_gated(W0, X, G, dY, e, al, outputs=subset)
        for k in subset:
            np.testing.assert_array_equal(to_host(part[k]), full[k], err_msg=str(subset))


@pytest.mark.parametrize("d,m,alpha_kind,with_reset", [(64, 64, "state", True), (16, 7, "scalar", False),
                                                        (128, 128, "state", False), (256, 64, "scalar", True),
                                                        (1024, 200, "state", True), (4096, 17, "scalar", False)])
def test_gated_decode(d, m, alpha_kind, with_reset):
    log(f"gated decode d={d} m={m} alpha={alpha_kind} reset={with_reset}")
    rng = np.random.default_rng(d + m)
    S, H, steps = 5, 3, 8
    W0 = (rng.standard_normal((H, m, d)) * d ** -0.5).astype(np.float32)
    Wh = (W0[None] + 0.1 * rng.standard_normal((S, H, m, d))).astype(np.float32)
    Wd, W0d = to_dev(Wh, "f32", torch), to_dev(W0, "f32", torch)
    Wr = Wh.astype(np.float64)
    for step in range(steps):
        x = (rng.standard_normal((S, H, d)) * d ** -0.5).astype(np.float32)
        g = (rng.standard_normal((S, H, m)) * 0.1).astype(np.float32)
        eta = rng.uniform(0, 0.2, (S, H)).astype(np.float32)
        al = rng.uniform(0, 1, (S, H)).astype(np.float32) if alpha_kind == "state" else np.float32(0.8)
        rs = (rng.uniform(0, 1, S) < 0.3).astype(np.uint8) if with_reset else None
        y = gl.decode_step_gated(Wd, W0d, to_dev(x, "f32", torch), to_dev(g, "f32", torch),
                                 to_dev(eta, "f32", torch),
                                 to_dev(al, "f32", torch) if alpha_kind == "state" else float(al),
                                 None if rs is None else torch.from_numpy(rs).to("cuda"))
        yr, Wr = orc.decode_step(Wr, x, g, eta, alpha=al, W0=W0, reset=rs)
        check("y", to_host(y), yr, "f32")
    check("W", to_host(Wd), Wr, "f32")


@pytest.mark.timeout(300)
def test_gated_lm_bf16_config():
    """The lm-bf16 shape with the paper's gate family and packed-document
    resets at full size; the oracle checks every output of sampled heads."""
    wl = W.SCAN_WORKLOADS["lm-bf16"]
    B, H, T, d, m = wl.B, wl.H, wl.T, wl.d, wl.m
    log("gated lm-bf16 config: drawing inputs on the device")
    inp = W.device_scan_inputs(wl, 0, "cuda", torch=torch)
    a, e = W.gate_tokens(B, H, T, d, wl.seed + 11)
    rs = W.reset_flags(B, T, wl.seed + 12, mean_len=512)
    ad, ed, rd = (torch.from_numpy(v).to("cuda") for v in (a, e, rs))
    out = {"y": gl.scan_fwd_gated(inp["W0"], inp["X"], inp["G"], ed, ad, rd)}
    out.update(gl.scan_bwd_gated(inp["W0"], inp["X"], inp["G"], inp["dY"], ed, ad, rd))
    torch.cuda.synchronize()
    for h in (2, 13):
        log(f"  oracle on head h={h} (all {B} batch rows, T={T})")
        sl = {"W0": to_host(inp["W0"][h:h + 1]), "X": to_host(inp["X"][:, h:h + 1]),
              "G": to_host(inp["G"][:, h:h + 1]), "dY": to_host(inp["dY"][:, h:h + 1]),
              "eta": e[:, h:h + 1].astype(np.float64), "alpha": a[:, h:h + 1].astype(np.float64),
              "reset": rs}
        ref = oracle_all(sl)
        for k in ("y", "gtilde", "dx", "dg", "deta", "dalpha"):
            check(k, to_host(out[k][:, h:h + 1]), ref[k], "bf16")
        check("dw0", to_host(out["dw0"][h:h + 1]), ref["dw0"], "bf16")
