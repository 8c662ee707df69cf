"""GPU parity of the gated save-for-backward pair (gradlev_scan_fwd_gated_save
and gradlev_scan_bwd_gated_saved) against the float64 oracle.

The forward runs on the backward's tile and stores Delta at every tile start
(Section 3, Eq. 2 with retention, carried forward); the backward reads those
states instead of recomputing them.  Checked here: every output, dalpha
included, against the oracle (tolerances of tests/parity_util.py) over the
same shapes, gate kinds, resets and ragged tails as the plain gated tests;
the saved states against the oracle's token-by-token gated update; the pair
against the plain gated calls; optional outputs and determinism; and the
lm-bf16 shape with the gate family and packed documents on sampled heads.
"""

import numpy as np
import pytest

from oracle import gradlev_oracle as orc
from paper_2609_34174_amd import workloads as W
from parity_util import check, log, to_dev, to_host
from test_gpu_gated import CASES, KEYS, inputs, oracle_all

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


def dev(inp, dtype):
    e, al = inp["eta"], inp["alpha"]
    return {"W0": to_dev(inp["W0"], "f32", torch), "X": to_dev(inp["X"], dtype, torch),
            "G": to_dev(inp["G"], dtype, torch), "dY": to_dev(inp["dY"], dtype, torch),
            "eta": to_dev(e, "f32", torch) if isinstance(e, np.ndarray) else e,
            "alpha": to_dev(al, "f32", torch) if isinstance(al, np.ndarray) else al,
            "reset": None if inp["reset"] is None else torch.from_numpy(inp["reset"]).to("cuda")}


def run_pair(t, segment=0, outputs=gl.GATED_OUTPUTS):
    Y, saved = gl.scan_fwd_gated_save(t["W0"], t["X"], t["G"], t["eta"], t["alpha"], t["reset"], segment=segment)
    res = gl.scan_bwd_gated_saved(t["W0"], t["X"], t["G"], t["dY"], saved, t["eta"], t["alpha"], t["reset"],
                                  segment=segment, outputs=outputs)
    res["y"] = Y
    torch.cuda.synchronize()
    return {k: to_host(v) for k, v in res.items()}, saved


@pytest.mark.parametrize("dtype,d,m,T,seg,ak,ek,rs", CASES)
def test_gated_saved_pair_parity(dtype, d, m, T, seg, ak, ek, rs):
    log(f"gated saved pair dtype={dtype} d={d} m={m} T={T} seg={seg} alpha={ak} eta={ek} reset={rs}")
    inp = inputs(2, 3, T, d, m, dtype, seed=T + d + 2 * m + 5, alpha_kind=ak, eta_kind=ek, with_reset=rs)
    out, _ = run_pair(dev(inp, dtype), segment=seg)
    ref = oracle_all(inp)
    for k in KEYS:
        check(k, out[k], ref[k], dtype)


def _tile(dtype, d, m):
    return 64 if (dtype == "bf16" and d == 64 and m == 64) else 32


@pytest.mark.parametrize("dtype,d,m", [("bf16", 64, 64), ("f32", 64, 64), ("bf16", 128, 64)])
def test_gated_saved_states_are_tile_starts(dtype, d, m):
    """The saved buffer holds Delta at every tile start.  Its layout is the
    backward's private register order, so the test reads it through that
    order: tile n, column block w, row block ib, lane (c, q), slot r holds
    Delta[16 ib + 4 q + r][16 w + c]."""
    B, H, T = 2, 2, 230
    log(f"gated saved states dtype={dtype} d={d} m={m} T={T}")
    inp = inputs(B, H, T, d, m, dtype, seed=91 + d + m, alpha_kind="family", eta_kind="token", with_reset=True)
    s = gl.make_shape(B=B, H=H, T=T, d_in=d, d_out=m, dtype=gl.BF16 if dtype == "bf16" else gl.F32)
    C = _tile(dtype, d, m)
    nch = -(-T // C)
    sv, _ = gl.gated_saved_bytes(s)
    assert sv == B * H * nch * m * d * 4
    t = dev(inp, dtype)
    _, saved = gl.scan_fwd_gated_save(t["W0"], t["X"], t["G"], t["eta"], t["alpha"], t["reset"])
    torch.cuda.synchronize()
    raw = to_host(saved).reshape(B, H, nch, d // 16, m // 16, 4, 16, 4)  # n, w, ib, q, c, r
    # Delta[16 ib + 4 q + r][16 w + c] = raw[b, h, n, w, ib, q, c, r]
    got = np.transpose(raw, (0, 1, 2, 4, 5, 7, 3, 6)).reshape(B, H, nch, m, d)
    # Oracle: token-by-token centered decay from Delta_0 = 0 (W0 = 0 isolates Delta).
    e = inp["eta"]
    al = inp["alpha"]
    rs = inp["reset"]
    Dl = np.zeros((B, H, m, d))
    ref = np.zeros((B, H, nch, m, d))
    for tt in range(T):
        if tt % C == 0:
            ref[:, :, tt // C] = Dl
        a_t = al[:, :, tt].astype(np.float64) if isinstance(al, np.ndarray) else np.full((B, H), al)
        e_t = e[:, :, tt].astype(np.float64) if isinstance(e, np.ndarray) else np.full((B, H), e)
        if rs is not None and tt + 1 < T:
            cut = rs[:, tt + 1].astype(bool)  # a document starts at tt+1: alpha_tt = eta_tt = 0
            a_t = np.where(cut[:, None], 0.0, a_t)
            e_t = np.where(cut[:, None], 0.0, e_t)
        _, Dl = orc.decode_step(Dl, inp["X"][:, :, tt], inp["G"][:, :, tt], e_t, alpha=a_t,
                                W0=np.zeros((H, m, d)))
    check("states", got, ref, dtype)


def test_gated_saved_matches_plain_gated():
    """The pair and the plain gated calls agree up to rounding order."""
    log("gated saved pair vs plain gated")
    inp = inputs(2, 2, 700, 64, 64, "bf16", seed=97, alpha_kind="family", eta_kind="token", with_reset=True)
    t = dev(inp, "bf16")
    out, _ = run_pair(t, segment=128)
    y = to_host(gl.scan_fwd_gated(t["W0"], t["X"], t["G"], t["eta"], t["alpha"], t["reset"], segment=128))
    p = {k: to_host(v) for k, v in gl.scan_bwd_gated(t["W0"], t["X"], t["G"], t["dY"], t["eta"], t["alpha"],
                                                      t["reset"], segment=128).items()}
    check("y", out["y"], y, "bf16")
    for k in ("gtilde", "dx", "dg", "deta", "dalpha", "dw0"):
        check(k, out[k], p[k], "bf16")


def test_gated_saved_optional_outputs_and_determinism():
    log("gated saved pair optional outputs / determinism")
    inp = inputs(2, 2, 400, 64, 64, "bf16", seed=98, alpha_kind="uniform", eta_kind="token", with_reset=False)
    t = dev(inp, "bf16")
    full, _ = run_pair(t)
    again, _ = run_pair(t)
    for k in KEYS:
        np.testing.assert_array_equal(again[k], full[k], err_msg=k)
    for subset in (("dalpha",), ("gtilde", "deta"), ("dw0",), ("dx", "dg")):
        part, _ = run_pair(t, outputs=subset)
        for k in subset:
            np.testing.assert_array_equal(part[k], full[k], err_msg=str(subset))


@pytest.mark.timeout(300)
def test_gated_saved_lm_shape_sampled():
    """The lm-bf16 shape with the gate family, per-token step sizes and packed
    documents (the gated benchmark's inputs), through the pair at full size;
    the oracle checks sampled heads over all batch rows."""
    wl = W.SCAN_WORKLOADS["lm-bf16"]
    B, H, T, d, m = wl.B, wl.H, wl.T, wl.d, wl.m
    log("gated saved pair at the lm-bf16 shape: drawing inputs")
    inp = W.device_scan_inputs(wl, 0, "cuda", torch=torch)
    a, e = W.gate_tokens(B, H, T, d, wl.seed + 11)
    rs = W.reset_flags(B, T, wl.seed + 12, mean_len=512)
    al, et, r = torch.from_numpy(a).cuda(), torch.from_numpy(e).cuda(), torch.from_numpy(rs).cuda()
    Y, saved = gl.scan_fwd_gated_save(inp["W0"], inp["X"], inp["G"], et, al, r)
    out = gl.scan_bwd_gated_saved(inp["W0"], inp["X"], inp["G"], inp["dY"], saved, et, al, r)
    out["y"] = Y
    torch.cuda.synchronize()
    for h in (4,):
        log(f"  oracle on head h={h} (all {B} batch rows, T={T})")
        sl = {"W0": to_host(inp["W0"][h:h + 1]), "X": to_host(inp["X"][:, h:h + 1]),
              "G": to_host(inp["G"][:, h:h + 1]), "dY": to_host(inp["dY"][:, h:h + 1]),
              "eta": e[:, h:h + 1], "alpha": a[:, h:h + 1], "reset": rs}
        ref = oracle_all(sl)
        for k in ("y", "gtilde", "dx", "dg", "deta", "dalpha"):
            check(k, to_host(out[k][:, h:h + 1]), ref[k], "bf16")
        check("dw0", to_host(out["dw0"][h:h + 1]), ref["dw0"], "bf16")
