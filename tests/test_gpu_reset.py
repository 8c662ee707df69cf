"""GPU parity of the reset pair: unit retention with document resets
(gradlev_scan_fwd_reset_save + gradlev_scan_bwd_reset_saved) against the
float64 oracle's sequential learner with the same reset flags.

Resets are placed where the kernels' masks and carries have edges: at chunk
starts (multiples of 64) and segment starts, at t = 1, at the last token,
several in one chunk, one-token documents (consecutive flags), and a flag at
t = 0 (which changes nothing).  Shapes span several chunks and segments with
ragged tails; both eta forms and both storage types.  The full lm-bf16 shape
with packed documents of mean length 512 is checked on sampled heads.
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

OUTS = ("gtilde", "dx", "dg", "deta", "dw0")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no ROCm GPU visible")
    gl.lib()
    yield
    torch.cuda.synchronize()


def flags(B, T, seed, mean_len, extra=()):
    r = W.reset_flags(B, T, seed, mean_len=mean_len) if mean_len else np.zeros((B, T), np.uint8)
    for b, t in extra:
        if b < B and t < T:
            r[b, t] = 1
    return r


def run_case(dtype, B, H, T, seg, eta_kind, r, seed):
    wl = dataclasses.replace(W.SCAN_WORKLOADS["lm-bf16"], B=B, H=H, T=T, dtype=dtype, x_dist="normal",
                             x_std=64 ** -0.5, g_std=0.3, seed=seed)
    inp = W.scan_inputs(wl)
    eta = W.eta_tokens(B, H, T, seed + 1, 0.0, 0.4) if eta_kind == "token" else 0.2
    W0, X, G, dY = to_dev(inp["W0"], "f32", torch), *(to_dev(inp[k], dtype, torch) for k in ("X", "G", "dY"))
    e = to_dev(eta, "f32", torch) if isinstance(eta, np.ndarray) else eta
    rd = torch.from_numpy(r).to("cuda")
    Y, saved = gl.scan_fwd_reset_save(W0, X, G, e, rd, segment=seg)
    out = gl.scan_bwd_reset_saved(W0, X, G, dY, saved, e, rd, segment=seg)
    torch.cuda.synchronize()
    ref_y = orc.scan_fwd(inp["W0"], inp["X"], inp["G"], eta, reset=r)
    ref = orc.scan_bwd(inp["W0"], inp["X"], inp["G"], eta, inp["dY"], reset=r)
    check("y", to_host(Y), ref_y, dtype)
    for k in OUTS:
        check(k, to_host(out[k]), ref[k], dtype)
    return (W0, X, G, dY, e, rd, seg), out


EDGE = ((0, 0), (0, 1), (0, 64), (0, 65), (0, 128), (1, 100), (1, 101), (1, 102), (0, 190), (1, 191),
        (1, 192), (0, 255), (1, 256), (0, 320), (1, 383), (0, 448))

CASES = [
    # dtype, B, H, T, segment hint, eta, mean document length, extra flags
    ("bf16", 2, 3, 300, 64, "scalar", 40, EDGE),
    ("bf16", 2, 2, 1000, 128, "token", 60, EDGE),
    ("f32", 2, 2, 200, 64, "scalar", 12, EDGE),
    ("f32", 1, 3, 333, 0, "token", 90, EDGE),
    ("bf16", 2, 2, 37, 0, "token", 8, ((0, 5), (1, 36))),
    ("bf16", 1, 2, 1, 0, "scalar", 0, ((0, 0),)),
    ("bf16", 2, 2, 2048, 0, "scalar", 512, ()),
    ("bf16", 3, 2, 700, 64, "scalar", 0, ()),  # no resets at all
    ("bf16", 2, 2, 512, 64, "token", 1, ()),   # a document at every token
]


@pytest.mark.parametrize("dtype,B,H,T,seg,ek,mean,extra", CASES)
def test_reset_pair_parity(dtype, B, H, T, seg, ek, mean, extra):
    log(f"reset pair dtype={dtype} B={B} H={H} T={T} seg={seg} eta={ek} mean={mean}")
    r = flags(B, T, T + 7, mean, extra)
    run_case(dtype, B, H, T, seg, ek, r, seed=T + B)


def test_reset_pair_null_flags_match_the_plain_pair():
    """reset = NULL means no document starts: the oracle's plain scan."""
    log("reset pair without flags")
    wl = dataclasses.replace(W.SCAN_WORKLOADS["lm-bf16"], B=2, H=2, T=400)
    inp = W.scan_inputs(wl)
    W0, X, G, dY = to_dev(inp["W0"], "f32", torch), *(to_dev(inp[k], "bf16", torch) for k in ("X", "G", "dY"))
    Y, saved = gl.scan_fwd_reset_save(W0, X, G, 0.1, None, segment=128)
    out = gl.scan_bwd_reset_saved(W0, X, G, dY, saved, 0.1, None, segment=128)
    torch.cuda.synchronize()
    check("y", to_host(Y), orc.scan_fwd(inp["W0"], inp["X"], inp["G"], 0.1), "bf16")
    ref = orc.scan_bwd(inp["W0"], inp["X"], inp["G"], 0.1, inp["dY"])
    for k in OUTS:
        check(k, to_host(out[k]), ref[k], "bf16")


def test_reset_pair_subsets_and_repeats_are_bitwise_identical():
    log("reset pair subsets and repeats")
    r = flags(2, 700, 3, 50, EDGE)
    (W0, X, G, dY, e, rd, seg), full = run_case("bf16", 2, 2, 700, 64, "token", r, seed=9)
    full = {k: to_host(v) for k, v in full.items()}
    _, saved = gl.scan_fwd_reset_save(W0, X, G, e, rd, segment=seg)
    for subset in (("gtilde",), ("dx", "dg"), ("deta",), ("dw0",), OUTS):
        part = gl.scan_bwd_reset_saved(W0, X, G, dY, saved, e, rd, segment=seg, outputs=subset)
        for k in subset:
            np.testing.assert_array_equal(to_host(part[k]), full[k], err_msg=str(subset))


@pytest.mark.timeout(300)
def test_reset_pair_lm_bf16_config():
    """The lm-bf16 shape (B=8, H=16, T=2048) at unit retention with packed
    documents of mean length 512; the oracle checks every output of sampled
    heads over all batch rows."""
    wl = W.SCAN_WORKLOADS["lm-bf16"]
    B, H, T = wl.B, wl.H, wl.T
    log("reset pair lm-bf16: drawing inputs on the device")
    inp = W.device_scan_inputs(wl, 0, "cuda", torch=torch)
    rs = W.reset_flags(B, T, wl.seed + 12, mean_len=512)
    rd = torch.from_numpy(rs).to("cuda")
    Y, saved = gl.scan_fwd_reset_save(inp["W0"], inp["X"], inp["G"], inp["eta"], rd)
    out = gl.scan_bwd_reset_saved(inp["W0"], inp["X"], inp["G"], inp["dY"], saved, inp["eta"], rd)
    torch.cuda.synchronize()
    for h in (5, 11):
        log(f"  oracle on head h={h} (all {B} batch rows, T={T})")
        sl = {k: to_host(inp[k][:, h:h + 1]) for k in ("X", "G", "dY")}
        W0h = to_host(inp["W0"][h:h + 1])
        check("y", to_host(Y[:, h:h + 1]), orc.scan_fwd(W0h, sl["X"], sl["G"], inp["eta"], reset=rs), "bf16")
        ref = orc.scan_bwd(W0h, sl["X"], sl["G"], inp["eta"], sl["dY"], reset=rs)
        for k in ("gtilde", "dx", "dg", "deta"):
            check(k, to_host(out[k][:, h:h + 1]), ref[k], "bf16")
        check("dw0", to_host(out["dw0"][h:h + 1]), ref["dw0"], "bf16")
