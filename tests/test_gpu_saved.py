"""GPU parity of the save-for-backward pair (gradlev_scan_fwd_save and
gradlev_scan_bwd_saved) against the float64 oracle.

The forward keeps the fast weights at the end of each token segment (the
prefix sums of Section 3 step 2, Eq. 3, at the boundaries); the backward
starts its segments from them.  Checked here: every output of the pair
against the oracle (tolerances of tests/parity_util.py), the saved states
against the oracle's token-by-token update (Eq. 1 applied once per token),
bitwise agreement of the pair's forward output with the plain forward on the
same segmentation, independence of optional outputs, determinism, and the
lm-bf16 workload at full size on sampled heads.
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

KEYS = ("y", "gtilde", "dx", "dg", "deta", "dw0")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("no ROCm GPU visible")
    gl.lib()  # raises if the HIP library is missing: there is no fallback
    yield
    torch.cuda.synchronize()


def small_inputs(B, H, T, d, m, dtype, seed, eta_kind):
    base = W.SCAN_WORKLOADS["lm-bf16"]
    wl = dataclasses.replace(base, B=B, H=H, T=T, d=d, m=m, dtype=dtype, x_dist="normal",
                             x_std=d ** -0.5, g_std=0.1, seed=seed)
    inp = W.scan_inputs(wl)
    if eta_kind == "token":
        inp["eta"] = W.eta_tokens(B, H, T, seed + 100)
    return inp


def dev(inp, dtype):
    eta = inp["eta"]
    return {"W0": to_dev(inp["W0"], "f32", torch), "X": to_dev(inp["X"], dtype, torch),
            "G": to_dev(inp["G"], dtype, torch), "dY": to_dev(inp["dY"], dtype, torch),
            "eta": to_dev(eta, "f32", torch) if isinstance(eta, np.ndarray) else eta}


def run_pair(t, prefix, chunk=0, segment=0, outputs=gl.BWD_OUTPUTS):
    Y, saved = gl.scan_fwd_save(t["W0"], t["X"], t["G"], t["eta"], prefix=prefix, chunk=chunk, segment=segment)
    res = gl.scan_bwd_saved(t["W0"], t["X"], t["G"], t["dY"], saved, t["eta"], prefix=prefix, chunk=chunk,
                            segment=segment, outputs=outputs)
    res["y"] = Y
    torch.cuda.synchronize()
    return {k: to_host(v) for k, v in res.items()}, saved


def oracle_all(inp, prefix):
    ref = {"y": orc.scan_fwd(inp["W0"], inp["X"], inp["G"], inp["eta"], prefix)}
    ref.update(orc.scan_bwd(inp["W0"], inp["X"], inp["G"], inp["eta"], inp["dY"], prefix))
    return ref


def oracle_segment_ends(inp, seg):
    """W after the last write of each segment, by the token-by-token update."""
    X, G, W0 = inp["X"], inp["G"], inp["W0"]
    B, H, T, _ = X.shape
    eta = inp["eta"]
    Wt = np.broadcast_to(np.asarray(W0, np.float64), (B, H) + W0.shape[1:]).copy()
    ends = []
    for t in range(T):
        e = eta[:, :, t] if isinstance(eta, np.ndarray) else eta
        _, Wt = orc.decode_step(Wt, X[:, :, t], G[:, :, t], e)
        if (t + 1) % seg == 0 or t + 1 == T:
            ends.append(Wt.copy())
    return np.stack(ends, axis=2)  # [B, H, nseg, m, d]


CASES = []
for dtype in ("f32", "bf16"):
    for prefix in ("exclusive", "inclusive"):
        for (d, m) in ((64, 64), (128, 128), (64, 128), (128, 64)):
            for T, seg in ((1, 0), (200, 64), (333, 128)):
                CASES.append((dtype, prefix, d, m, T, seg))


@pytest.mark.parametrize("dtype,prefix,d,m,T,seg", CASES)
def test_saved_pair_parity(dtype, prefix, d, m, T, seg):
    eta_kind = "token" if (T + d + m) % 2 else "scalar"
    log(f"saved pair dtype={dtype} prefix={prefix} d={d} m={m} T={T} seg={seg} eta={eta_kind}")
    inp = small_inputs(2, 3, T, d, m, dtype, seed=T * 5 + d + 2 * m, eta_kind=eta_kind)
    out, _ = run_pair(dev(inp, dtype), prefix, segment=seg)
    ref = oracle_all(inp, prefix)
    for k in KEYS:
        check(k, out[k], ref[k], dtype)


@pytest.mark.parametrize("dtype,d,m,B,H,T,hint", [("f32", 64, 64, 2, 2, 700, 256), ("bf16", 64, 64, 2, 2, 700, 256),
                                                  ("bf16", 128, 64, 2, 2, 700, 256), ("f32", 64, 128, 2, 2, 700, 256),
                                                  ("bf16", 64, 64, 8, 16, 517, 0)])
def test_saved_states_are_segment_ends(dtype, d, m, B, H, T, hint):
    """The saved buffer holds W_0 + Delta after each of the backward's
    segments, [B*H][nseg][m][d].  The last case has the automatic plan, where
    the forward's segments span two of the backward's (B*H = 128)."""
    log(f"saved states dtype={dtype} d={d} m={m} B={B} H={H} T={T} segment={hint}")
    inp = small_inputs(B, H, T, d, m, dtype, seed=77 + d + m + T, eta_kind="token")
    s = gl.make_shape(B=B, H=H, T=T, d_in=d, d_out=m, dtype=gl.BF16 if dtype == "bf16" else gl.F32,
                      segment=hint)
    p = gl.plan(s)
    seg = -(-p.bwd_segment // p.fwd_chunk) * p.fwd_chunk
    nseg = -(-T // seg)
    if hint == 0:
        assert p.fwd_segment > seg, (p.fwd_segment, seg)  # the case this test is for
    sv, _ = gl.saved_bytes(s)
    assert sv == B * H * nseg * m * d * 4
    t = dev(inp, dtype)
    _, saved = gl.scan_fwd_save(t["W0"], t["X"], t["G"], t["eta"], segment=hint)
    torch.cuda.synchronize()
    got = to_host(saved).reshape(B, H, nseg, m, d)
    check("w_end", got, oracle_segment_ends(inp, seg), dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sixteen_saved_segments(dtype):
    """The most segments a plan has: 16 of 64 tokens, the last one ragged."""
    log(f"16 saved segments dtype={dtype}")
    inp = small_inputs(1, 2, 1000, 64, 64, dtype, seed=23, eta_kind="token")
    s = gl.make_shape(B=1, H=2, T=1000, d_in=64, d_out=64, dtype=gl.BF16 if dtype == "bf16" else gl.F32,
                      segment=64)
    assert gl.saved_bytes(s)[0] == 2 * 16 * 64 * 64 * 4
    out, _ = run_pair(dev(inp, dtype), "inclusive", segment=64)
    ref = oracle_all(inp, "inclusive")
    for k in KEYS:
        check(k, out[k], ref[k], dtype)


@pytest.mark.parametrize("dtype,d,m", [("bf16", 64, 64), ("f32", 128, 128), ("bf16", 128, 64)])
def test_automatic_segments(dtype, d, m):
    """No hints: the pair's own segmentation (B*H = 15, several segments)."""
    log(f"saved pair automatic segments dtype={dtype} d={d} m={m}")
    inp = small_inputs(3, 5, 3000, d, m, dtype, seed=91 + d, eta_kind="scalar")
    s = gl.make_shape(B=3, H=5, T=3000, d_in=d, d_out=m, dtype=gl.BF16 if dtype == "bf16" else gl.F32)
    assert gl.saved_bytes(s)[0] > 15 * m * d * 4  # more than one segment
    out, _ = run_pair(dev(inp, dtype), "exclusive")
    ref = oracle_all(inp, "exclusive")
    for k in KEYS:
        check(k, out[k], ref[k], dtype)


def test_forward_output_matches_plain_forward():
    """Saving the states changes nothing in Y (same segmentation: bitwise)."""
    log("fwd_save Y == fwd Y")
    inp = small_inputs(2, 2, 900, 64, 64, "bf16", seed=31, eta_kind="token")
    t = dev(inp, "bf16")
    for seg in (128, 256):
        Y0 = gl.scan_fwd(t["W0"], t["X"], t["G"], t["eta"], segment=seg)
        Y1, _ = gl.scan_fwd_save(t["W0"], t["X"], t["G"], t["eta"], segment=seg)
        torch.cuda.synchronize()
        assert torch.equal(Y0, Y1)


def test_saved_optional_outputs_and_determinism():
    """A NULL output skips work without changing the others; repeated calls
    are bitwise identical."""
    log("saved pair optional outputs / determinism")
    inp = small_inputs(2, 2, 500, 64, 64, "bf16", seed=13, eta_kind="token")
    t = dev(inp, "bf16")
    full, _ = run_pair(t, "exclusive", segment=128)
    again, _ = run_pair(t, "exclusive", segment=128)
    for k in KEYS:
        np.testing.assert_array_equal(again[k], full[k], err_msg=k)
    for subset in (("gtilde",), ("dx",), ("dg", "deta"), ("dw0",)):
        part, _ = run_pair(t, "exclusive", segment=128, outputs=subset)
        for k in subset:
            np.testing.assert_array_equal(part[k], full[k], err_msg=str(subset))


@pytest.mark.timeout(300)
@pytest.mark.parametrize("prefix,token_eta", [("exclusive", False), ("inclusive", True)])
def test_lm_bf16_config_saved(prefix, token_eta):
    """The lm-bf16 workload at full size through the pair; the oracle checks
    every output of sampled heads over all batch rows."""
    wl = W.SCAN_WORKLOADS["lm-bf16"]
    log(f"config {wl.name} saved pair prefix={prefix} token_eta={token_eta}: drawing inputs on the device")
    inp = W.device_scan_inputs(wl, 0, "cuda", torch=torch)
    eta = inp["eta"]
    if token_eta:
        gen = torch.Generator(device="cuda")
        gen.manual_seed(wl.layer_seed(0) + 9)
        eta = (torch.rand(wl.B, wl.H, wl.T, device="cuda", generator=gen) * 0.2).contiguous()
    Y, saved = gl.scan_fwd_save(inp["W0"], inp["X"], inp["G"], eta, prefix=prefix, chunk=wl.chunk)
    out = gl.scan_bwd_saved(inp["W0"], inp["X"], inp["G"], inp["dY"], saved, eta, prefix=prefix, chunk=wl.chunk)
    out["y"] = Y
    torch.cuda.synchronize()
    for h in (2, 11):
        log(f"  oracle on head h={h} (all {wl.B} batch rows, T={wl.T})")
        sl = {"W0": to_host(inp["W0"][h:h + 1]), "X": to_host(inp["X"][:, h:h + 1]),
              "G": to_host(inp["G"][:, h:h + 1]), "dY": to_host(inp["dY"][:, h:h + 1]),
              "eta": to_host(eta[:, h:h + 1]) if token_eta else eta}
        ref = oracle_all(sl, prefix)
        for k in ("y", "gtilde", "dx", "dg", "deta"):
            check(k, to_host(out[k][:, h:h + 1]), ref[k], wl.dtype)
        check("dw0", to_host(out["dw0"][h:h + 1]), ref["dw0"], wl.dtype)
