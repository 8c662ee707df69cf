"""GPU parity: the HIP scans and decode step against the float64 oracle.

Every call goes through the C ABI (via the thin ctypes binding).  Inputs are
seeded and synthetic with the workloads' distributions; the oracle consumes
the same already-quantised values.  Tolerances (normwise, per output tensor)
are those of tests/parity_util.py: fp32 max_rel <= 1e-5; bf16 max_rel <= 2e-2
and mean_rel <= 1e-3.

Small cases span several chunks, several segments (forced with the segment
hint) and a ragged last chunk; the five workload configurations run at full
size, with the oracle on sampled sequences where the full oracle would take
minutes (every (b, h) sequence is an independent problem, so a sampled
sequence is checked completely).
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


def run_gpu(inp, dtype, prefix, chunk=0, segment=0, outputs=gl.BWD_OUTPUTS, with_bwd=True):
    W0 = to_dev(inp["W0"], "f32", torch)
    X = to_dev(inp["X"], dtype, torch)
    G = to_dev(inp["G"], dtype, torch)
    eta = inp["eta"]
    eta_d = to_dev(eta, "f32", torch) if isinstance(eta, np.ndarray) else eta
    Y = gl.scan_fwd(W0, X, G, eta_d, prefix=prefix, chunk=chunk, segment=segment)
    res = {"y": Y}
    if with_bwd:
        dY = to_dev(inp["dY"], dtype, torch)
        res.update(gl.scan_bwd(W0, X, G, dY, eta_d, prefix=prefix, chunk=chunk, segment=segment,
                               outputs=outputs))
    torch.cuda.synchronize()
    return {k: to_host(v) for k, v in res.items()}


def oracle_all(inp, prefix):
    ref = {"y": orc.scan_fwd(inp["W0"], inp["X"], inp["G"], inp["eta"], prefix)}
    ref.update(orc.scan_bwd(inp["W0"], inp["X"], inp["G"], inp["eta"], inp["dY"], prefix))
    return ref


KEYS = ("y", "gtilde", "dx", "dg", "deta", "dw0")


# ---------------------------------------------------------------------------
# Small cases: every dtype / convention / width / eta form, ragged T, forced
# multi-segment carries.
# ---------------------------------------------------------------------------

SMALL = []
for dtype in ("f32", "bf16"):
    for prefix in ("exclusive", "inclusive"):
        for (d, m) in ((64, 64), (128, 128), (64, 128), (128, 64)):
            for T, seg in ((1, 0), (37, 0), (200, 64), (333, 128)):
                SMALL.append((dtype, prefix, d, m, T, seg))


@pytest.mark.parametrize("dtype,prefix,d,m,T,seg", SMALL)
def test_small_parity(dtype, prefix, d, m, T, seg):
    eta_kind = "token" if (T + d) % 2 else "scalar"
    log(f"small dtype={dtype} prefix={prefix} d={d} m={m} T={T} seg={seg} eta={eta_kind}")
    inp = small_inputs(2, 3, T, d, m, dtype, seed=T * 7 + d + m, eta_kind=eta_kind)
    out = run_gpu(inp, dtype, prefix, segment=seg)
    ref = oracle_all(inp, prefix)
    for k in KEYS:
        check(k, out[k], ref[k], dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_chunk_hint_and_segments_change_rounding_only(dtype):
    log(f"chunk/segment hints dtype={dtype}")
    inp = small_inputs(1, 2, 700, 64, 64, dtype, seed=5, eta_kind="token")
    ref = oracle_all(inp, "exclusive")
    for chunk, seg in ((0, 0), (128, 0), (64, 64), (128, 256), (0, 640)):
        out = run_gpu(inp, dtype, "exclusive", chunk=chunk, segment=seg)
        for k in KEYS:
            check(f"{k}", out[k], ref[k], dtype)


@pytest.mark.parametrize("prefix,T,seg", [("exclusive", 200, 0), ("inclusive", 333, 128), ("exclusive", 1000, 256),
                                          ("inclusive", 1000, 0), ("exclusive", 130, 128)])
def test_128_wide_tiles(prefix, T, seg):
    """128 x 128 maps with 128-token forward tiles (shared score tiles in
    LDS), several segments and ragged tails, both read conventions."""
    log(f"128x128 chunk 128 prefix={prefix} T={T} seg={seg}")
    inp = small_inputs(2, 3, T, 128, 128, "bf16", seed=T + seg + 5, eta_kind="scalar")
    assert gl.plan(gl.make_shape(B=2, H=3, T=T, d_in=128, d_out=128, dtype=gl.BF16, chunk=128)).fwd_chunk == 128
    out = run_gpu(inp, "bf16", prefix, chunk=128, segment=seg)
    ref = oracle_all(inp, prefix)
    for k in KEYS:
        check(k, out[k], ref[k], "bf16")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sixteen_segments(dtype):
    """The largest carry: 16 segments of 64 tokens, the last one ragged."""
    log(f"16 segments dtype={dtype}")
    inp = small_inputs(1, 2, 1000, 64, 64, dtype, seed=21, eta_kind="token")
    assert gl.plan(gl.make_shape(B=1, H=2, T=1000, d_in=64, d_out=64, dtype=gl.BF16 if dtype == "bf16" else gl.F32,
                                 prefix="inclusive", segment=64)).bwd_nseg == 16
    out = run_gpu(inp, dtype, "inclusive", segment=64)
    ref = oracle_all(inp, "inclusive")
    for k in KEYS:
        check(k, out[k], ref[k], dtype)


@pytest.mark.parametrize("dtype,d,m", [("f32", 64, 64), ("bf16", 64, 64), ("bf16", 128, 64)])
def test_heads_not_multiple_of_eight(dtype, d, m):
    """B*H = 15 with automatic segments: the XCD-ordered grid has idle slots."""
    log(f"B*H=15 auto segments dtype={dtype} d={d} m={m}")
    inp = small_inputs(3, 5, 3000, d, m, dtype, seed=33 + d, eta_kind="token")
    p = gl.plan(gl.make_shape(B=3, H=5, T=3000, d_in=d, d_out=m,
                              dtype=gl.BF16 if dtype == "bf16" else gl.F32))
    assert p.fwd_nseg > 1 and p.bwd_nseg > 1
    out = run_gpu(inp, dtype, "exclusive")
    ref = oracle_all(inp, "exclusive")
    for k in KEYS:
        check(k, out[k], ref[k], dtype)


def test_eta_zero_reads_slow_weights():
    log("eta = 0")
    inp = small_inputs(2, 2, 150, 64, 64, "bf16", seed=9, eta_kind="scalar")
    inp["eta"] = 0.0
    out = run_gpu(inp, "bf16", "exclusive", segment=64)
    ref = oracle_all(inp, "exclusive")
    for k in ("y", "gtilde", "dx", "deta", "dw0"):
        check(k, out[k], ref[k], "bf16")
    assert np.all(out["dg"] == 0.0)


def test_optional_outputs_are_independent():
    """A NULL output skips work without changing the others (bitwise)."""
    log("optional outputs")
    inp = small_inputs(2, 2, 300, 64, 64, "bf16", seed=11, eta_kind="token")
    full = run_gpu(inp, "bf16", "exclusive", segment=128)
    for subset in (("gtilde",), ("dx",), ("dg",), ("deta",), ("dw0",), ("gtilde", "deta")):
        part = run_gpu(inp, "bf16", "exclusive", segment=128, outputs=subset)
        for k in subset:
            np.testing.assert_array_equal(part[k], full[k], err_msg=str(subset))


def test_backward_is_deterministic():
    log("determinism")
    inp = small_inputs(4, 4, 1000, 64, 64, "bf16", seed=12, eta_kind="scalar")
    a = run_gpu(inp, "bf16", "exclusive")
    b = run_gpu(inp, "bf16", "exclusive")
    for k in KEYS:
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)


@pytest.mark.parametrize("d,m,chunk,seg,eta_kind", [(64, 64, 128, 256, "token"), (64, 64, 64, 128, "token"),
                                                    (64, 64, 0, 0, "scalar"), (128, 128, 0, 256, "token"),
                                                    (64, 128, 0, 0, "token"), (128, 64, 128, 0, "scalar")])
def test_repeated_calls_are_bitwise_identical(d, m, chunk, seg, eta_kind):
    """Every tile variant (64- and 128-token forward tiles, register and LDS
    score tiles, paired and wave-specialised backward tiles) reduces in a
    fixed order, so repeated calls agree bitwise; a race between waves would
    show here as run-to-run differences."""
    log(f"repeat d={d} m={m} chunk={chunk} seg={seg} eta={eta_kind}")
    inp = small_inputs(2, 3, 700, d, m, "bf16", seed=d + m + seg, eta_kind=eta_kind)
    runs = [run_gpu(inp, "bf16", "exclusive", chunk=chunk, segment=seg) for _ in range(3)]
    for r in runs[1:]:
        for k in KEYS:
            np.testing.assert_array_equal(r[k], runs[0][k], err_msg=k)


# ---------------------------------------------------------------------------
# Workload configurations at full size
# ---------------------------------------------------------------------------

def test_small_f32_config():
    wl = W.SCAN_WORKLOADS["small-f32"]
    for prefix in ("exclusive", "inclusive"):
        log(f"config small-f32 prefix={prefix}")
        inp = W.scan_inputs(wl)
        out = run_gpu(inp, "f32", prefix, chunk=wl.chunk)
        ref = oracle_all(inp, prefix)
        for k in KEYS:
            check(k, out[k], ref[k], "f32")


def _sampled_config(wl, layer, heads, prefix="exclusive", token_eta=False):
    """Full-size GPU run; the oracle checks every output of the sampled heads.

    Inputs are drawn on the device with the workload's seeded generator (the
    full host draw would take minutes at these sizes); the sampled heads are
    copied back and handed to the oracle as they are.  Each sampled head is
    checked over all batch rows, which also covers dW0[h].
    """
    log(f"config {wl.name} layer={layer}: drawing inputs on the device")
    inp = W.device_scan_inputs(wl, layer, "cuda", torch=torch)
    eta = inp["eta"]
    if token_eta:
        gen = torch.Generator(device="cuda")
        gen.manual_seed(wl.layer_seed(layer) + 7)
        eta = (torch.rand(wl.B, wl.H, wl.T, device="cuda", generator=gen) * 0.2).contiguous()
    log(f"config {wl.name} layer={layer} prefix={prefix} token_eta={token_eta}: GPU fwd+bwd (full size)")
    Y = gl.scan_fwd(inp["W0"], inp["X"], inp["G"], eta, prefix=prefix, chunk=wl.chunk)
    out = gl.scan_bwd(inp["W0"], inp["X"], inp["G"], inp["dY"], eta, prefix=prefix, chunk=wl.chunk)
    out["y"] = Y
    torch.cuda.synchronize()
    for h in heads:
        log(f"  oracle on head h={h} (all {wl.B} batch rows, T={wl.T})")
        sl = {"W0": to_host(inp["W0"][h:h + 1]), "X": to_host(inp["X"][:, h:h + 1]),
              "G": to_host(inp["G"][:, h:h + 1]), "dY": to_host(inp["dY"][:, h:h + 1]),
              "eta": to_host(eta[:, h:h + 1]) if token_eta else eta}
        ref = oracle_all(sl, prefix)
        for k in ("y", "gtilde", "dx", "dg", "deta"):
            check(k, to_host(out[k][:, h:h + 1]), ref[k], wl.dtype)
        check("dw0", to_host(out["dw0"][h:h + 1]), ref["dw0"], wl.dtype)


@pytest.mark.timeout(300)
def test_lm_bf16_config():
    _sampled_config(W.SCAN_WORKLOADS["lm-bf16"], 0, [0, 9])


@pytest.mark.timeout(300)
@pytest.mark.parametrize("prefix,token_eta", [("inclusive", False), ("exclusive", True), ("inclusive", True)])
def test_lm_bf16_config_conventions(prefix, token_eta):
    """The lm-bf16 shape with the inclusive read and per-token step sizes."""
    _sampled_config(W.SCAN_WORKLOADS["lm-bf16"], 0, [5], prefix, token_eta)


@pytest.mark.timeout(300)
def test_long_bf16_config():
    _sampled_config(W.SCAN_WORKLOADS["long-bf16"], 0, [3])


@pytest.mark.timeout(300)
@pytest.mark.parametrize("layer", [0, 23])
def test_stack_bf16_config_layers(layer):
    _sampled_config(W.SCAN_WORKLOADS["stack-bf16"], layer, [31])


# ---------------------------------------------------------------------------
# Longest accepted sequences (per-sequence byte offsets just under 2^31)
# ---------------------------------------------------------------------------

def _longest_T(width):
    """The largest T the library accepts for this map width: T * width * 4 < 2^31."""
    return (1 << 31) // (4 * width) - 1


def _point_check(inp, eta, prefix, out, ts, dtype, block=1 << 20):
    """Check sampled tokens of one sequence against the closed-form oracle.

    The writes before each sampled read and the costate suffix after it are
    summed block by block on the host in float64 (sums over disjoint token
    ranges add up), then every output of the token is evaluated from them.
    """
    X, G, dY = inp["X"][0, 0], inp["G"][0, 0], inp["dY"][0, 0]
    T = X.shape[0]
    inc = prefix == "inclusive"
    tok_eta = not isinstance(eta, float)
    eh = to_host(eta[0, 0]) if tok_eta else eta

    def ew(lo, hi):
        return eh[lo:hi] if tok_eta else eh

    ts = sorted(set(int(t) for t in ts))
    W0h = to_host(inp["W0"][0])
    P = np.zeros_like(W0h)
    pos, Wread = 0, {}
    for t in ts:
        end = t + 1 if inc else t
        while pos < end:
            hi = min(end, pos + block)
            P += orc.outer_sum(to_host(G[pos:hi]), to_host(X[pos:hi]), ew(pos, hi), 0, hi - pos)
            pos = hi
        Wread[t] = W0h - P
    R = np.zeros_like(W0h)
    pos, Rs = T, {}
    for t in reversed(ts):
        start = t if inc else t + 1
        while pos > start:
            lo = max(start, pos - block)
            R += orc.outer_sum(to_host(dY[lo:pos]), to_host(X[lo:pos]), 1.0, 0, pos - lo)
            pos = lo
        Rs[t] = R.copy()
    while pos > 0:
        lo = max(0, pos - block)
        R += orc.outer_sum(to_host(dY[lo:pos]), to_host(X[lo:pos]), 1.0, 0, pos - lo)
        pos = lo
    idx = torch.tensor(ts, device=X.device)
    rows = {k: to_host(out[k][0, 0].index_select(0, idx)) for k in ("y", "gtilde", "dx", "dg", "deta")}
    xs, gs, ds = to_host(X.index_select(0, idx)), to_host(G.index_select(0, idx)), to_host(dY.index_select(0, idx))
    ref = {k: [] for k in rows}
    for i, t in enumerate(ts):
        o = orc.token_outputs(Wread[t], Rs[t], xs[i], gs[i], eh[t] if tok_eta else eh, ds[i])
        for k in rows:
            ref[k].append(o[k])
    for k in rows:
        check(k, rows[k], np.array(ref[k]), dtype)
    check("dw0", to_host(out["dw0"][0]), R, dtype)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("d,prefix,token_eta", [(64, "exclusive", False), (128, "inclusive", True)])
def test_longest_sequence(d, prefix, token_eta):
    """One bf16 sequence of the longest accepted length, sampled at the chunk
    and segment seams, the ragged tail and random tokens."""
    T = _longest_T(d)
    p = gl.plan(gl.make_shape(B=1, H=1, T=T, d_in=d, d_out=d, dtype=gl.BF16, prefix=prefix))
    log(f"longest sequence T={T} d=m={d} prefix={prefix} token_eta={token_eta} "
        f"fwd {p.fwd_nseg}x{p.fwd_segment} bwd {p.bwd_nseg}x{p.bwd_segment}")
    with pytest.raises(gl.GradLevError):
        gl.plan(gl.make_shape(B=1, H=1, T=T + 1, d_in=d, d_out=d, dtype=gl.BF16))
    wl = dataclasses.replace(W.SCAN_WORKLOADS["lm-bf16"], B=1, H=1, T=T, d=d, m=d, seed=40 + d)
    inp = W.device_scan_inputs(wl, 0, "cuda", torch=torch)
    eta = inp["eta"]
    if token_eta:
        gen = torch.Generator(device="cuda")
        gen.manual_seed(41 + d)
        eta = (torch.rand(1, 1, T, device="cuda", generator=gen) * 0.2).contiguous()
    out = {"y": gl.scan_fwd(inp["W0"], inp["X"], inp["G"], eta, prefix=prefix)}
    out.update(gl.scan_bwd(inp["W0"], inp["X"], inp["G"], inp["dY"], eta, prefix=prefix))
    torch.cuda.synchronize()
    log("  GPU done; oracle on sampled tokens")
    seams = [0, 1, p.fwd_chunk - 1, p.fwd_chunk, p.bwd_chunk - 1, p.bwd_chunk]
    for seg in (p.fwd_segment, p.bwd_segment):
        for k in (1, p.fwd_nseg // 2, (T - 1) // seg):
            seams += [k * seg - 1, k * seg, k * seg + 1]
    seams += [T // 2, T - p.bwd_chunk, T - 2, T - 1]
    rng = np.random.default_rng(d)
    seams += list(rng.integers(0, T, 8))
    _point_check(inp, eta, prefix, out, [t for t in seams if 0 <= t < T], "bf16")


# ---------------------------------------------------------------------------
# Decode
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d,m,eta_kind", [(64, 64, "scalar"), (16, 7, "state"), (32, 300, "scalar"),
                                          (128, 128, "state"), (256, 64, "scalar"), (64, 1, "state"),
                                          # wide states: one wave per row, ragged row blocks
                                          (512, 300, "scalar"), (1024, 129, "state"), (2048, 33, "state"),
                                          (4096, 64, "scalar"), (8192, 5, "state")])
def test_decode_small(d, m, eta_kind):
    log(f"decode small d={d} m={m} eta={eta_kind}")
    rng = np.random.default_rng(d * 1000 + m)
    S, H, steps = 5, 3, 6
    Wh = (rng.standard_normal((S, H, m, d)) * d ** -0.5).astype(np.float32)
    Wd = to_dev(Wh, "f32", torch)
    Wr = Wh.astype(np.float64)
    for step in range(steps):
        x = (rng.standard_normal((S, H, d)) * d ** -0.5).astype(np.float32)
        g = (rng.standard_normal((S, H, m)) * 0.1).astype(np.float32)
        eta = rng.uniform(0, 0.2, (S, H)).astype(np.float32) if eta_kind == "state" else 0.1
        ed = to_dev(eta, "f32", torch) if eta_kind == "state" else eta
        y = gl.decode_step(Wd, to_dev(x, "f32", torch), to_dev(g, "f32", torch), ed)
        yr, Wr = orc.decode_step(Wr, x, g, eta if eta_kind == "state" else np.float32(0.1))
        check("y", to_host(y), yr, "f32")
    check("W", to_host(Wd), Wr, "f32")


@pytest.mark.timeout(300)
def test_decode_config():
    wl = W.DECODE_WORKLOADS["decode-f32"]
    log(f"config {wl.name}: {wl.steps} steps of S={wl.S} H={wl.H}")
    W0 = W.decode_initial_state(wl)
    Wd = to_dev(W0, "f32", torch)
    picks = [(0, 0), (17, 5), (255, 15)]
    Wr = np.stack([W0[s, h] for s, h in picks]).astype(np.float64)[:, None]
    worst = 0.0
    for step in range(wl.steps):
        x, g = W.decode_step_inputs(wl, step)
        y = to_host(gl.decode_step(Wd, to_dev(x, "f32", torch), to_dev(g, "f32", torch), wl.eta))
        xs = np.stack([x[s, h] for s, h in picks])[:, None]
        gs = np.stack([g[s, h] for s, h in picks])[:, None]
        yr, Wr = orc.decode_step(Wr, xs, gs, np.float32(wl.eta))
        ys = np.stack([y[s, h] for s, h in picks])[:, None]
        mx = np.max(np.abs(ys - yr)) / np.max(np.abs(yr))
        worst = max(worst, mx)
        if step % 128 == 0:
            log(f"  step {step}: y max_rel {mx:.2e}")
    log(f"  worst y max_rel over {wl.steps} steps: {worst:.2e}")
    assert worst <= 1e-5
    Wf = to_host(Wd)
    check("W", np.stack([Wf[s, h] for s, h in picks])[:, None], Wr, "f32")
