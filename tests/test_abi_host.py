"""Host-side tests of the C ABI (no GPU needed).

The library must load, export every symbol that include/gradlev.h declares,
and reject invalid calls with the documented status codes before touching
the HIP runtime.  Pointers passed here are fake but never dereferenced,
because every call below fails validation.
"""

import ctypes
import os
import re

import pytest

import paper_2609_34174_amd as gl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gradlev.h")

FAKE = ctypes.c_void_p(1 << 20)        # aligned, never dereferenced
MISALIGNED = ctypes.c_void_p((1 << 20) + 8)


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(gl.LIB_PATH):
        pytest.skip("library not built")
    return gl.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gradlev_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("gradlev_scan_fwd", "gradlev_scan_bwd", "gradlev_decode_step",
                     "gradlev_scan_workspace_bytes", "gradlev_scan_plan", "gradlev_error_string"):
        assert required in names


def test_every_declared_symbol_is_exported(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_error_strings(L):
    for code in (0, -1, -2, -3, -4, -5, -6, 7):
        assert isinstance(gl.error_string(code), str) and gl.error_string(code)
    assert gl.error_string(0) == "success"


def shape(**kw):
    base = dict(B=2, H=4, T=300, d_in=64, d_out=64, dtype=gl.BF16, prefix="exclusive")
    base.update(kw)
    return gl.make_shape(**base)


def plan_rc(s):
    p = gl.Plan()
    return gl.lib().gradlev_scan_plan(ctypes.byref(s), ctypes.byref(p)), p


@pytest.mark.parametrize("bad,code", [
    (dict(B=0), gl.ERR_INVALID), (dict(H=-1), gl.ERR_INVALID), (dict(T=0), gl.ERR_INVALID),
    (dict(d_in=0), gl.ERR_INVALID), (dict(dtype=7), gl.ERR_INVALID), (dict(prefix=3), gl.ERR_INVALID),
    (dict(chunk=-64), gl.ERR_INVALID), (dict(d_in=96), gl.ERR_UNSUPPORTED),
    (dict(d_out=256), gl.ERR_UNSUPPORTED), (dict(chunk=32), gl.ERR_UNSUPPORTED),
    (dict(segment=100), gl.ERR_UNSUPPORTED), (dict(T=1025, segment=64), gl.ERR_UNSUPPORTED),
])
def test_plan_rejects(L, bad, code):
    rc, _ = plan_rc(shape(**bad))
    assert rc == code


@pytest.mark.parametrize("kw", [dict(), dict(dtype=gl.F32), dict(d_in=128, d_out=128),
                                dict(d_in=64, d_out=128), dict(d_in=128, d_out=64, dtype=gl.F32),
                                dict(T=1), dict(T=16384, B=2, H=16, d_in=128, d_out=128, chunk=128),
                                dict(segment=64), dict(prefix="inclusive"), dict(T=1024, segment=64),
                                dict(B=1, H=1, T=1 << 20), dict(B=1, H=1, T=1 << 20, segment=1 << 16)])
def test_plan_is_consistent(L, kw):
    s = shape(**kw)
    rc, p = plan_rc(s)
    assert rc == gl.OK
    for C, seg, n in ((p.fwd_chunk, p.fwd_segment, p.fwd_nseg), (p.bwd_chunk, p.bwd_segment, p.bwd_nseg)):
        assert C in (32, 64, 128)
        assert seg % C == 0 and seg >= C
        assert n == -(-s.T // seg) and n >= 1
    assert gl.workspace_bytes(s) == p.workspace_bytes
    if kw.get("segment"):
        assert p.fwd_segment == max(kw["segment"], p.fwd_chunk)
    assert p.fwd_nseg <= 16 and p.bwd_nseg <= 16


def test_workspace_covers_aggregates(L):
    s = shape(B=8, H=16, T=2048)
    p = gl.plan(s)
    md = 64 * 64 * 4
    bwd = (2 * p.bwd_nseg if p.bwd_nseg > 1 else 1) + 1
    assert p.workspace_bytes >= 8 * 16 * max(p.fwd_nseg, bwd) * md


def fwd_call(s, W0=FAKE, X=FAKE, G=FAKE, eta=None, Y=FAKE, ws=FAKE, wsn=1 << 40):
    return gl.lib().gradlev_scan_fwd(ctypes.byref(s), W0, X, G, eta, 0.1, Y, ws, wsn, None)


def bwd_call(s, outs=(FAKE, FAKE, FAKE, FAKE, FAKE), ws=FAKE, wsn=1 << 40, dY=FAKE):
    return gl.lib().gradlev_scan_bwd(ctypes.byref(s), FAKE, FAKE, FAKE, None, 0.1, dY, *outs, ws, wsn, None)


def test_fwd_validation_before_launch(L):
    s = shape()
    assert fwd_call(s, W0=None) == gl.ERR_INVALID
    assert fwd_call(s, Y=None) == gl.ERR_INVALID
    assert fwd_call(s, X=MISALIGNED) == gl.ERR_ALIGN
    assert fwd_call(s, eta=MISALIGNED) == gl.ERR_ALIGN
    assert fwd_call(s, ws=None) == gl.ERR_WORKSPACE
    assert fwd_call(s, wsn=16) == gl.ERR_WORKSPACE
    assert fwd_call(s, ws=MISALIGNED) == gl.ERR_ALIGN
    assert fwd_call(shape(d_in=32)) == gl.ERR_UNSUPPORTED
    assert gl.lib().gradlev_scan_fwd(None, FAKE, FAKE, FAKE, None, 0.1, FAKE, FAKE, 1 << 40, None) == gl.ERR_INVALID


def test_bwd_validation_before_launch(L):
    s = shape()
    assert bwd_call(s, outs=(None,) * 5) == gl.ERR_INVALID
    assert bwd_call(s, dY=None) == gl.ERR_INVALID
    assert bwd_call(s, outs=(None, MISALIGNED, None, None, None)) == gl.ERR_ALIGN
    assert bwd_call(s, ws=None) == gl.ERR_WORKSPACE
    assert bwd_call(s, wsn=1024) == gl.ERR_WORKSPACE


@pytest.mark.parametrize("kw", [dict(), dict(B=8, H=16, T=2048), dict(d_in=128, d_out=128, chunk=128),
                                dict(dtype=gl.F32, d_in=128), dict(T=1), dict(segment=64, T=1000),
                                dict(B=1, H=1, T=1 << 20)])
def test_saved_pair_sizes(L, kw):
    """The saved state is one fp32 [m][d] matrix per sequence and backward
    segment, the backward's segment rounded up to whole forward tiles; the
    workspace covers both calls of the pair."""
    s = shape(**kw)
    p = gl.plan(s)
    sv, ws = gl.saved_bytes(s)
    md = s.d_in * s.d_out * 4
    assert sv % (s.B * s.H * md) == 0
    nseg = sv // (s.B * s.H * md)
    seg = -(-p.bwd_segment // p.fwd_chunk) * p.fwd_chunk
    assert nseg == -(-s.T // seg) and 1 <= nseg <= 16
    agg = s.B * s.H * nseg * md if nseg > 1 else 0
    assert ws >= agg + s.B * s.H * md


def saved_fwd_call(s, saved=FAKE, svn=1 << 40, Y=FAKE):
    return gl.lib().gradlev_scan_fwd_save(ctypes.byref(s), FAKE, FAKE, FAKE, None, 0.1, Y, saved, svn,
                                          FAKE, 1 << 40, None)


def saved_bwd_call(s, saved=FAKE, svn=1 << 40, outs=(FAKE, FAKE, FAKE, FAKE, FAKE), wsn=1 << 40):
    return gl.lib().gradlev_scan_bwd_saved(ctypes.byref(s), FAKE, FAKE, FAKE, None, 0.1, FAKE, saved, svn,
                                           *outs, FAKE, wsn, None)


def test_saved_pair_validation_before_launch(L):
    s = shape()
    sv, _ = gl.saved_bytes(s)
    for call in (saved_fwd_call, saved_bwd_call):
        assert call(s, saved=None) == gl.ERR_INVALID
        assert call(s, saved=MISALIGNED) == gl.ERR_ALIGN
        assert call(s, svn=sv - 4) == gl.ERR_WORKSPACE
        assert call(shape(d_in=32)) == gl.ERR_UNSUPPORTED
        assert call(shape(B=0)) == gl.ERR_INVALID
        # Parallel-form widths keep no segment states.
        assert call(shape(d_in=1024, d_out=128)) == gl.ERR_UNSUPPORTED
    assert saved_fwd_call(s, Y=None) == gl.ERR_INVALID
    assert saved_bwd_call(s, outs=(None,) * 5) == gl.ERR_INVALID
    assert saved_bwd_call(s, wsn=16) == gl.ERR_WORKSPACE
    n = ctypes.c_size_t(0)
    assert L.gradlev_scan_saved_bytes(ctypes.byref(shape(d_in=1024)), ctypes.byref(n), ctypes.byref(n)) \
        == gl.ERR_UNSUPPORTED
    assert L.gradlev_scan_saved_bytes(ctypes.byref(s), None, ctypes.byref(n)) == gl.ERR_INVALID


def test_gated_saved_pair_sizes_and_validation(L):
    """Saved states: one fp32 m x d matrix per sequence and backward tile (64
    tokens for bf16 64 x 64 maps, else 32); the backward's workspace needs no
    state region."""
    for kw, tile in ((dict(), 64), (dict(dtype=gl.F32), 32), (dict(d_in=128), 32), (dict(T=1), 64)):
        s = shape(**kw)
        sv, ws = gl.gated_saved_bytes(s)
        assert sv == s.B * s.H * -(-s.T // tile) * s.d_in * s.d_out * 4
        assert ws <= gl.gated_workspace_bytes(s)
    s = shape()
    sv, _ = gl.gated_saved_bytes(s)
    g = gl.Gates()
    g.alpha, g.alpha_scalar, g.reset = None, 0.9, None

    def fwd(sh=s, saved=FAKE, svn=1 << 40):
        return L.gradlev_scan_fwd_gated_save(ctypes.byref(sh), ctypes.byref(g), FAKE, FAKE, FAKE, None, 0.1, FAKE,
                                             saved, svn, FAKE, 1 << 40, None)

    def bwd(sh=s, saved=FAKE, svn=1 << 40):
        return L.gradlev_scan_bwd_gated_saved(ctypes.byref(sh), ctypes.byref(g), FAKE, FAKE, FAKE, None, 0.1, FAKE,
                                              saved, svn, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 40, None)
    for call in (fwd, bwd):
        assert call(saved=None) == gl.ERR_INVALID
        assert call(saved=MISALIGNED) == gl.ERR_ALIGN
        assert call(svn=sv - 4) == gl.ERR_WORKSPACE
        assert call(sh=shape(prefix="inclusive")) == gl.ERR_UNSUPPORTED
        assert call(sh=shape(d_in=1024, d_out=128)) == gl.ERR_UNSUPPORTED


def test_decode_validation_before_launch(L):
    f = gl.lib().gradlev_decode_step
    assert f(0, 16, 64, 64, FAKE, FAKE, FAKE, None, 0.1, FAKE, None) == gl.ERR_INVALID
    assert f(4, 16, 64, 64, None, FAKE, FAKE, None, 0.1, FAKE, None) == gl.ERR_INVALID
    assert f(4, 16, 48, 64, FAKE, FAKE, FAKE, None, 0.1, FAKE, None) == gl.ERR_UNSUPPORTED
    assert f(4, 16, 64, 2048, FAKE, FAKE, FAKE, None, 0.1, FAKE, None) == gl.ERR_UNSUPPORTED
    assert f(4, 16, 64, 64, MISALIGNED, FAKE, FAKE, None, 0.1, FAKE, None) == gl.ERR_ALIGN


def test_binding_refuses_cpu_tensors(L):
    torch = pytest.importorskip("torch")
    X = torch.zeros(1, 1, 8, 64, dtype=torch.bfloat16)
    G = torch.zeros(1, 1, 8, 64, dtype=torch.bfloat16)
    W0 = torch.zeros(1, 64, 64)
    with pytest.raises(ValueError, match="ROCm GPU"):
        gl.scan_fwd(W0, X, G, 0.1)


# ---------------------------------------------------------------------------
# Gated entry points
# ---------------------------------------------------------------------------

def gates(alpha=None, scalar=0.9, reset=None):
    g = gl.Gates()
    g.alpha, g.alpha_scalar, g.reset = alpha, scalar, reset
    return g


def test_gated_workspace_covers_states(L):
    s = shape(B=2, H=4, T=300)
    n = gl.gated_workspace_bytes(s)
    # the backward keeps one fp32 m x d state per chunk start (chunks of at most 64 tokens)
    assert n >= 2 * 4 * ((300 + 63) // 64) * 64 * 64 * 4
    with pytest.raises(gl.GradLevError) as e:
        gl.gated_workspace_bytes(shape(prefix="inclusive"))
    assert e.value.code == gl.ERR_UNSUPPORTED


def test_gated_validation_before_launch(L):
    s = shape()
    g = gates()
    fwd = gl.lib().gradlev_scan_fwd_gated
    bwd = gl.lib().gradlev_scan_bwd_gated
    assert fwd(ctypes.byref(s), None, FAKE, FAKE, FAKE, None, 0.1, FAKE, FAKE, 1 << 40, None) == gl.ERR_INVALID
    assert fwd(ctypes.byref(s), ctypes.byref(gates(alpha=MISALIGNED)), FAKE, FAKE, FAKE, None, 0.1, FAKE,
               FAKE, 1 << 40, None) == gl.ERR_ALIGN
    assert fwd(ctypes.byref(s), ctypes.byref(g), FAKE, FAKE, FAKE, None, 0.1, FAKE, None, 0, None) == gl.ERR_WORKSPACE
    si = shape(prefix="inclusive")
    assert fwd(ctypes.byref(si), ctypes.byref(g), FAKE, FAKE, FAKE, None, 0.1, FAKE, FAKE, 1 << 40, None) == gl.ERR_UNSUPPORTED
    outs = (None,) * 6
    assert bwd(ctypes.byref(s), ctypes.byref(g), FAKE, FAKE, FAKE, None, 0.1, FAKE, *outs, FAKE, 1 << 40, None) == gl.ERR_INVALID
    outs = (None, None, None, None, MISALIGNED, None)
    assert bwd(ctypes.byref(s), ctypes.byref(g), FAKE, FAKE, FAKE, None, 0.1, FAKE, *outs, FAKE, 1 << 40, None) == gl.ERR_ALIGN
    outs = (None, None, None, None, FAKE, None)
    assert bwd(ctypes.byref(s), ctypes.byref(g), FAKE, FAKE, FAKE, None, 0.1, FAKE, *outs, FAKE, 1024, None) == gl.ERR_WORKSPACE
    dec = gl.lib().gradlev_decode_step_gated
    assert dec(4, 16, 64, 64, FAKE, None, FAKE, FAKE, None, 0.1, None, 0.9, None, FAKE, None) == gl.ERR_INVALID
    assert dec(4, 16, 64, 64, FAKE, FAKE, FAKE, FAKE, None, 0.1, MISALIGNED, 0.9, None, FAKE, None) == gl.ERR_ALIGN
    assert dec(4, 16, 48, 64, FAKE, FAKE, FAKE, FAKE, None, 0.1, None, 0.9, None, FAKE, None) == gl.ERR_UNSUPPORTED


def test_mlp_validation_before_launch(L):
    def ms(**kw):
        base = dict(B=2, H=2, T=100, d_in=64, hidden=128, d_out=64, segment=0, in_dtype=gl.BF16, act=0)
        base.update(kw)
        return gl.MlpShape(**base)
    n = ctypes.c_size_t(0)
    assert L.gradlev_mlp_workspace_bytes(ctypes.byref(ms()), ctypes.byref(n)) == gl.OK and n.value > 0
    assert L.gradlev_mlp_workspace_bytes(ctypes.byref(ms(act=7)), ctypes.byref(n)) == gl.ERR_INVALID
    assert L.gradlev_mlp_workspace_bytes(ctypes.byref(ms(hidden=96)), ctypes.byref(n)) == gl.ERR_UNSUPPORTED
    g = gates(scalar=1.0)
    fwd = L.gradlev_mlp_fwd
    args = [FAKE] * 5 + [None, 0.9, FAKE, FAKE, FAKE, FAKE, 1 << 40, None]
    bad = list(args)
    bad[7] = None                      # Z missing
    assert fwd(ctypes.byref(ms()), ctypes.byref(g), *bad) == gl.ERR_INVALID
    bad = list(args)
    bad[2] = MISALIGNED                # X misaligned
    assert fwd(ctypes.byref(ms()), ctypes.byref(g), *bad) == gl.ERR_ALIGN
    bad = list(args)
    bad[11] = 16                       # workspace too small
    assert fwd(ctypes.byref(ms()), ctypes.byref(g), *bad) == gl.ERR_WORKSPACE
    rev = L.gradlev_mlp_reverse
    # W1_0, W2_0, X, Gz, Gy, mu, mu_scalar, Z, Hid, gY, gZ, gX, dMu, dAlpha, dW1_0, dW2_0, ws, bytes, stream
    rargs = [FAKE] * 5 + [None, 0.9, FAKE, FAKE, FAKE, None, None, None, None, None, None, FAKE, 1 << 40, None]
    assert rev(ctypes.byref(ms()), ctypes.byref(g), *rargs) == gl.ERR_INVALID   # gZ missing
    for k in range(12, 16):                                                   # each gradient output misaligned
        bad = list(rargs)
        bad[10] = FAKE
        bad[k] = MISALIGNED
        assert rev(ctypes.byref(ms()), ctypes.byref(g), *bad) == gl.ERR_ALIGN, k
    ok = list(rargs)
    ok[10] = ok[12] = ok[13] = ok[14] = ok[15] = FAKE
    ok[17] = 16                                                               # workspace too small
    assert rev(ctypes.byref(ms()), ctypes.byref(g), *ok) == gl.ERR_WORKSPACE


# ---------------------------------------------------------------------------
# Wide maps (parallel form): widths that are multiples of 128, one above 128
# ---------------------------------------------------------------------------

def test_wide_plan_is_one_chunk(L):
    s = shape(B=2, H=1, T=1000, d_in=1024, d_out=4096)
    rc, p = plan_rc(s)
    assert rc == gl.OK
    assert p.fwd_chunk == p.bwd_chunk == 1024 and p.fwd_nseg == p.bwd_nseg == 1
    # gate prefixes (16 B per padded token), the causal score matrix (4 B per
    # pair), with 72 triangle tiles for 256 compute units the fp32 partials
    # of a 4-way split of the score contraction, and the bf16 hi + lo planes
    # of W_0, the gate gradients' partial column sums (two row halves per
    # 128-token block) and the retention gradient's fp32 F tiles (4 B per pair)
    BH, Tp = 2, 1024
    gates = (BH * Tp * 16 + 255) // 256 * 256
    planes = 1024 * 4096 * 4
    dpart = BH * 2 * (Tp // 128) * Tp * 4
    assert p.workspace_bytes == gates + BH * Tp * Tp * 4 + 4 * BH * Tp * Tp * 4 + planes + dpart + BH * Tp * Tp * 4
    # many sequences fill the chip without splitting
    _, p2 = plan_rc(shape(B=16, H=4, T=1000, d_in=1024, d_out=4096))
    assert p2.workspace_bytes == ((64 * Tp * 16 + 255) // 256 * 256 + 64 * Tp * Tp * 4 + 4 * planes
                                  + 64 * 2 * (Tp // 128) * Tp * 4 + 64 * Tp * Tp * 4)
    # fp32 operands need no planes
    _, p3 = plan_rc(shape(B=16, H=4, T=1000, d_in=1024, d_out=4096, dtype=gl.F32))
    assert p3.workspace_bytes == p2.workspace_bytes - 4 * planes
    assert gl.workspace_bytes(s) == p.workspace_bytes


@pytest.mark.parametrize("bad,code", [
    (dict(d_in=192, d_out=256), gl.ERR_UNSUPPORTED), (dict(d_in=256, d_out=64), gl.ERR_UNSUPPORTED),
    (dict(d_in=256, prefix="inclusive"), gl.ERR_UNSUPPORTED), (dict(d_in=256, T=16385), gl.ERR_UNSUPPORTED),
    (dict(d_in=8320, d_out=128), gl.ERR_UNSUPPORTED), (dict(d_in=256, B=0), gl.ERR_INVALID),
    (dict(d_in=256, d_out=128, chunk=-1), gl.ERR_INVALID),
])
def test_wide_plan_rejects(L, bad, code):
    base = dict(d_out=128)
    base.update(bad)
    rc, _ = plan_rc(shape(**base))
    assert rc == code


def test_wide_backward_validation_before_launch(L):
    """Every backward output is accepted for wide maps; its alignment and the
    workspace are checked before any launch."""
    s = shape(B=1, H=1, T=100, d_in=256, d_out=128)
    g = gl.Gates()
    g.alpha, g.alpha_scalar, g.reset = None, 1.0, None
    args = [ctypes.byref(s), ctypes.byref(g)] + [FAKE] * 4 + [ctypes.c_float(0.1), FAKE]
    # gtilde, dX, dG, deta, dalpha, dW0, ws, bytes, stream
    for k in range(6):
        outs = [None] * 6
        outs[k] = MISALIGNED
        rc = L.gradlev_scan_bwd_gated(*args, *outs, FAKE, ctypes.c_size_t(1 << 30), None)
        assert rc == gl.ERR_ALIGN, k
        outs[k] = FAKE
        rc = L.gradlev_scan_bwd_gated(*args, *outs, FAKE, ctypes.c_size_t(16), None)
        assert rc == gl.ERR_WORKSPACE, k
    rc = L.gradlev_scan_bwd_gated(*args, *([None] * 6), FAKE, ctypes.c_size_t(1 << 30), None)
    assert rc == gl.ERR_INVALID


@pytest.mark.parametrize("d_in,d_out,ok", [(512, 4096, True), (1024, 4096, True), (4096, 1024, True),
                                           (8192, 65536, False), (8192, 65535, True), (8192, 8192, True), (384, 64, False),
                                           (1024, 65537, False), (256, 1025, False), (3072, 64, False)])
def test_decode_shapes(L, d_in, d_out, ok):
    """Decode validates its state shape before any launch (fake pointers are
    never touched: an accepted shape is checked here only through the
    alignment error that a misaligned y produces)."""
    rc = L.gradlev_decode_step(ctypes.c_int64(2), ctypes.c_int64(1), ctypes.c_int64(d_in), ctypes.c_int64(d_out),
                               FAKE, FAKE, FAKE, None, ctypes.c_float(0.1), MISALIGNED, None)
    assert rc == (gl.ERR_ALIGN if ok else gl.ERR_UNSUPPORTED)


@pytest.mark.parametrize("B,H,T,seg,ok", [
    # 16 segments of 64 tokens: 8 * 16 * ceil(BH / 8) workgroups of up to 1024 work-items
    (1 << 18, 1, 1024, 64, False), ((1 << 18) - 8, 1, 1024, 64, True),
    # default plans at T = 1: one segment, 8 * ceil(BH / 8) workgroups
    ((1 << 22) - 8, 1, 1, 0, True), (1 << 22, 1, 1, 0, False), (1 << 12, (1 << 10) - 1, 1, 0, True),
    (1 << 12, 1 << 10, 1, 0, False)])
def test_plan_rejects_grids_past_the_work_item_limit(L, B, H, T, seg, ok):
    """A plan whose grid would reach 2^32 work-items is refused on the host
    (the widest scan kernels run 1024 work-items per workgroup)."""
    s = shape(B=B, H=H, T=T, segment=seg)
    rc, p = plan_rc(s)
    assert rc == (gl.OK if ok else gl.ERR_UNSUPPORTED)
    if ok:
        for n in (p.fwd_nseg, p.bwd_nseg):
            assert 8 * n * -(-(B * H) // 8) * 1024 < 2 ** 32
    sz, ws = ctypes.c_size_t(0), ctypes.c_size_t(0)
    rc2 = L.gradlev_scan_saved_bytes(ctypes.byref(s), ctypes.byref(sz), ctypes.byref(ws))
    assert (rc2 == gl.OK) == ok
    rc3 = L.gradlev_scan_gated_workspace_bytes(ctypes.byref(s), ctypes.byref(ws))
    assert (rc3 == gl.OK) == ok


@pytest.mark.parametrize("S,H,ok", [((1 << 24) - 1, 1, True), (1 << 24, 1, False), (1 << 12, 1 << 12, False),
                                    (1 << 12, (1 << 12) - 1, True)])
def test_decode_rejects_grids_past_the_work_item_limit(L, S, H, ok):
    """Decode at 64-wide states runs one 256-work-item workgroup per state:
    S * H states must stay below 2^24 (fake pointers; an accepted shape is seen
    through the alignment error of a misaligned y)."""
    for fn in ("plain", "gated"):
        if fn == "plain":
            rc = L.gradlev_decode_step(ctypes.c_int64(S), ctypes.c_int64(H), ctypes.c_int64(64), ctypes.c_int64(64),
                                       FAKE, FAKE, FAKE, None, ctypes.c_float(0.1), MISALIGNED, None)
        else:
            rc = L.gradlev_decode_step_gated(ctypes.c_int64(S), ctypes.c_int64(H), ctypes.c_int64(64),
                                             ctypes.c_int64(64), FAKE, FAKE, FAKE, FAKE, None, ctypes.c_float(0.1),
                                             None, ctypes.c_float(1.0), None, MISALIGNED, None)
        assert rc == (gl.ERR_ALIGN if ok else gl.ERR_UNSUPPORTED), fn


def test_static_forward_validation_before_any_hip_call(L):
    """gradlev_scan_fwd_static checks its arguments, and that the call's
    workspace fits the static scratch, on the host before any HIP call (here
    there is no GPU: an accepted call would fail in the scratch lookup)."""
    f = L.gradlev_scan_fwd_static
    s = shape()
    assert f(ctypes.byref(s), None, FAKE, FAKE, None, 0.1, FAKE, None) == gl.ERR_INVALID
    assert f(ctypes.byref(s), FAKE, FAKE, FAKE, None, 0.1, None, None) == gl.ERR_INVALID
    assert f(ctypes.byref(s), FAKE, MISALIGNED, FAKE, None, 0.1, FAKE, None) == gl.ERR_ALIGN
    assert f(ctypes.byref(s), FAKE, FAKE, FAKE, MISALIGNED, 0.1, FAKE, None) == gl.ERR_ALIGN
    assert f(ctypes.byref(shape(d_in=32)), FAKE, FAKE, FAKE, None, 0.1, FAKE, None) == gl.ERR_UNSUPPORTED
    assert f(None, FAKE, FAKE, FAKE, None, 0.1, FAKE, None) == gl.ERR_INVALID
    # A forward whose segment aggregates exceed the 64 MiB scratch.
    big = shape(B=64, H=64, T=1 << 14, segment=1024, d_in=128, d_out=128)
    assert gl.workspace_bytes(big) > gl.STATIC_SCRATCH_BYTES
    assert f(ctypes.byref(big), FAKE, FAKE, FAKE, None, 0.1, FAKE, None) == gl.ERR_SCRATCH
    # The wide maps' score matrix counts too: 8 sequences of 4096 tokens.
    wide = shape(B=8, H=1, T=4096, d_in=1024, d_out=4096)
    assert gl.workspace_bytes(wide) > gl.STATIC_SCRATCH_BYTES
    assert f(ctypes.byref(wide), FAKE, FAKE, FAKE, None, 0.1, FAKE, None) == gl.ERR_SCRATCH
    assert "GRADLEV_STATIC_SCRATCH_BYTES" in gl.error_string(gl.ERR_SCRATCH)
    m = re.search(r"#define GRADLEV_STATIC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == gl.STATIC_SCRATCH_BYTES


def test_reset_pair_sizes_and_validation(L):
    """The reset pair (unit retention with document resets) takes 64 x 64
    exclusive maps; its saved buffer holds the segment-end weights and room for
    a state at every 64-token chunk start; arguments are checked before any
    launch."""
    s = shape(B=2, H=4, T=1000)
    sv, ws = gl.reset_saved_bytes(s)
    sv_plain, _ = gl.saved_bytes(shape(B=2, H=4, T=1000, chunk=64))
    md = 64 * 64 * 4
    assert sv >= sv_plain + 2 * 4 * -(-1000 // 64) * md
    for bad, code in ((dict(d_in=128), gl.ERR_UNSUPPORTED), (dict(d_out=128), gl.ERR_UNSUPPORTED),
                      (dict(prefix="inclusive"), gl.ERR_UNSUPPORTED), (dict(T=0), gl.ERR_INVALID)):
        a, b = ctypes.c_size_t(0), ctypes.c_size_t(0)
        assert L.gradlev_scan_reset_saved_bytes(ctypes.byref(shape(**bad)), ctypes.byref(a), ctypes.byref(b)) == code
    fwd, bwd = L.gradlev_scan_fwd_reset_save, L.gradlev_scan_bwd_reset_saved
    # W0, X, G, eta, eta_scalar, reset, Y, saved, saved_bytes, ws, ws_bytes, stream
    fa = [FAKE, FAKE, FAKE, None, 0.1, FAKE, FAKE, FAKE, sv, FAKE, ws, None]
    for k, v, code in ((0, None, gl.ERR_INVALID), (6, None, gl.ERR_INVALID), (7, None, gl.ERR_INVALID),
                       (1, MISALIGNED, gl.ERR_ALIGN), (3, MISALIGNED, gl.ERR_ALIGN), (8, sv - 4, gl.ERR_WORKSPACE),
                       (10, 16, gl.ERR_WORKSPACE)):
        bad = list(fa)
        bad[k] = v
        assert fwd(ctypes.byref(s), *bad) == code, k
    # W0, X, G, eta, eta_scalar, dY, reset, saved, saved_bytes, gtilde, dX, dG, deta, dW0, ws, ws_bytes, stream
    ba = [FAKE, FAKE, FAKE, None, 0.1, FAKE, FAKE, FAKE, sv, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ws, None]
    for k, v, code in ((5, None, gl.ERR_INVALID), (7, None, gl.ERR_INVALID), (12, MISALIGNED, gl.ERR_ALIGN),
                       (8, 16, gl.ERR_WORKSPACE), (15, 16, gl.ERR_WORKSPACE)):
        bad = list(ba)
        bad[k] = v
        assert bwd(ctypes.byref(s), *bad) == code, k
    none = list(ba)
    for k in range(9, 14):
        none[k] = None
    assert bwd(ctypes.byref(s), *none) == gl.ERR_INVALID   # no output requested
