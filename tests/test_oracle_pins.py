"""Pins of the float64 oracle against what the paper and the mathematics fix.

None of these compare the oracle with itself.  Each pin restates a fact
independently of the oracle's token-by-token recurrence:

* a hand-derived three-token example (tests/golden/hand_T3_d2.json);
* the closed-form scan reads of Appendix C (Eq. 16) with retention one,
  written as dense masked matrix products;
* textbook special cases: eta = 0, T = 1, identical unit inputs (a plain
  exclusive prefix sum), orthonormal inputs;
* central finite differences of L = sum <dY, y> (exact up to rounding here,
  because L is at most quadratic in every input), including a read-only
  perturbation that isolates the transpose read gtilde;
* a complex-step Jacobian-vector product against the reverse sweep (adjoint
  identity);
* Theorem 1's statement that the scan equals the serial learner: token-by-token
  decode steps reproduce the scan and end at W_0 + Delta_T;
* dW_0 = sum_b dY^T X, a plain matrix product.
"""

import json
import os

import numpy as np
import pytest

from oracle import gradlev_oracle as orc

pytestmark = []

PREFIXES = [orc.EXCLUSIVE, orc.INCLUSIVE]


def rand_problem(B=2, H=3, T=7, d=4, m=5, seed=0, eta="token"):
    rng = np.random.default_rng(seed)
    W0 = rng.standard_normal((H, m, d))
    X = rng.standard_normal((B, H, T, d))
    G = rng.standard_normal((B, H, T, m))
    dY = rng.standard_normal((B, H, T, m))
    e = rng.uniform(0.05, 0.6, size=(B, H, T)) if eta == "token" else float(eta)
    return W0, X, G, e, dY


def closed_form_fwd(W0, X, G, eta, prefix):
    """Appendix C, Eq. 16 with alpha = 1, as dense masked products."""
    B, H, T, d = X.shape
    e = np.broadcast_to(np.asarray(eta, float), (B, H, T))
    k = -1 if prefix == orc.EXCLUSIVE else 0
    mask = np.tril(np.ones((T, T)), k)
    Y = np.empty(G.shape)
    for b in range(B):
        for h in range(H):
            A = (X[b, h] @ X[b, h].T) * mask           # A[t, s] = x_t . x_s
            Y[b, h] = X[b, h] @ W0[h].T - A @ (e[b, h][:, None] * G[b, h])
    return Y


def closed_form_gtilde(W0, X, G, eta, dY, prefix):
    """Second line of Eq. 16 queried by dY_t: W_0^T dY_t + Delta_t^T dY_t."""
    B, H, T, d = X.shape
    e = np.broadcast_to(np.asarray(eta, float), (B, H, T))
    k = -1 if prefix == orc.EXCLUSIVE else 0
    mask = np.tril(np.ones((T, T)), k)
    out = np.empty(X.shape)
    for b in range(B):
        for h in range(H):
            E = (dY[b, h] @ G[b, h].T) * mask * e[b, h][None, :]   # E[t, s]
            out[b, h] = dY[b, h] @ W0[h] - E @ X[b, h]
    return out


def rel_err(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


# --------------------------------------------------------------------------
# Hand-derived example
# --------------------------------------------------------------------------

@pytest.mark.parametrize("prefix", PREFIXES)
def test_hand_example(golden_dir, prefix):
    with open(os.path.join(golden_dir, "hand_T3_d2.json")) as f:
        gd = json.load(f)
    W0 = np.array(gd["W0"], float)[None]
    X = np.array(gd["X"], float)[None, None]
    G = np.array(gd["G"], float)[None, None]
    dY = np.array(gd["dY"], float)[None, None]
    exp = gd[prefix]
    Y = orc.scan_fwd(W0, X, G, gd["eta"], prefix)
    np.testing.assert_array_equal(Y[0, 0], np.array(exp["y"], float))
    out = orc.scan_bwd(W0, X, G, gd["eta"], dY, prefix)
    for key in ("gtilde", "dx", "dg", "deta"):
        np.testing.assert_array_equal(out[key][0, 0], np.array(exp[key], float), err_msg=key)
    np.testing.assert_array_equal(out["dw0"][0], np.array(exp["dw0"], float))


def test_hand_example_decode(golden_dir):
    with open(os.path.join(golden_dir, "hand_T3_d2.json")) as f:
        gd = json.load(f)
    W = np.array(gd["W0"], float)[None, None]
    for t in range(3):
        x = np.array(gd["X"][t], float)[None, None]
        g = np.array(gd["G"][t], float)[None, None]
        y, W = orc.decode_step(W, x, g, gd["eta"])
        np.testing.assert_array_equal(y[0, 0], np.array(gd["exclusive"]["y"][t], float))
    np.testing.assert_array_equal(W[0, 0], np.array(gd["decode_final_W"], float))


# --------------------------------------------------------------------------
# Closed forms (Theorem 1: the scan equals the serial learner)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("prefix", PREFIXES)
@pytest.mark.parametrize("shape", [(2, 3, 7, 4, 5), (1, 2, 33, 6, 3), (1, 1, 1, 3, 3)])
def test_fwd_equals_closed_form(prefix, shape):
    B, H, T, d, m = shape
    W0, X, G, e, _ = rand_problem(B, H, T, d, m, seed=T)
    Y = orc.scan_fwd(W0, X, G, e, prefix)
    assert rel_err(Y, closed_form_fwd(W0, X, G, e, prefix)) < 1e-12


@pytest.mark.parametrize("prefix", PREFIXES)
def test_gtilde_equals_closed_form(prefix):
    W0, X, G, e, dY = rand_problem(2, 2, 19, 5, 3, seed=4)
    out = orc.scan_bwd(W0, X, G, e, dY, prefix)
    assert rel_err(out["gtilde"], closed_form_gtilde(W0, X, G, e, dY, prefix)) < 1e-12


def test_scalar_eta_matches_broadcast():
    W0, X, G, _, dY = rand_problem(1, 2, 9, 4, 4, seed=8)
    e = np.full((1, 2, 9), 0.3)
    Y1 = orc.scan_fwd(W0, X, G, 0.3)
    Y2 = orc.scan_fwd(W0, X, G, e)
    np.testing.assert_array_equal(Y1, Y2)
    b1 = orc.scan_bwd(W0, X, G, 0.3, dY)
    b2 = orc.scan_bwd(W0, X, G, e, dY)
    for k in b1:
        np.testing.assert_array_equal(b1[k], b2[k])


# --------------------------------------------------------------------------
# Special cases
# --------------------------------------------------------------------------

def test_eta_zero_is_static_map():
    W0, X, G, _, dY = rand_problem(2, 2, 11, 4, 6, seed=1)
    Y = orc.scan_fwd(W0, X, G, 0.0)
    for b in range(2):
        for h in range(2):
            np.testing.assert_allclose(Y[b, h], X[b, h] @ W0[h].T, rtol=0, atol=1e-14)
    out = orc.scan_bwd(W0, X, G, 0.0, dY)
    for b in range(2):
        for h in range(2):
            np.testing.assert_allclose(out["gtilde"][b, h], dY[b, h] @ W0[h], rtol=0, atol=1e-14)
    np.testing.assert_array_equal(out["dg"], 0.0)
    np.testing.assert_allclose(out["dx"], out["gtilde"], rtol=0, atol=0)
    # deta does not vanish at eta = 0: d/d eta_t of -eta_t <dY_u, g_t>(x_t.x_u).
    ref = np.zeros((2, 2, 11))
    for t in range(11):
        for u in range(t + 1, 11):
            ref[:, :, t] -= np.einsum("bhm,bhm->bh", dY[:, :, u], G[:, :, t]) * \
                np.einsum("bhd,bhd->bh", X[:, :, t], X[:, :, u])
    assert rel_err(out["deta"], ref) < 1e-12


def test_single_token_reads_slow_weights():
    W0, X, G, e, dY = rand_problem(3, 2, 1, 5, 4, seed=2)
    Y = orc.scan_fwd(W0, X, G, e)
    np.testing.assert_allclose(Y[:, :, 0], np.einsum("hmd,bhd->bhm", W0, X[:, :, 0]), atol=1e-14)
    out = orc.scan_bwd(W0, X, G, e, dY)
    np.testing.assert_array_equal(out["dg"], 0.0)
    np.testing.assert_array_equal(out["deta"], 0.0)


@pytest.mark.parametrize("prefix", PREFIXES)
def test_identical_unit_inputs_give_prefix_sum(prefix):
    """x_t = e_k for all t: y_t = W0 e_k - (exclusive|inclusive) cumsum of eta g."""
    rng = np.random.default_rng(5)
    T, d, m, k = 13, 4, 3, 2
    W0 = rng.standard_normal((1, m, d))
    X = np.zeros((1, 1, T, d))
    X[..., k] = 1.0
    G = rng.standard_normal((1, 1, T, m))
    e = rng.uniform(0.1, 0.5, size=(1, 1, T))
    Y = orc.scan_fwd(W0, X, G, e, prefix)
    writes = e[0, 0, :, None] * G[0, 0]
    incl = np.cumsum(writes, axis=0)
    pre = incl if prefix == orc.INCLUSIVE else np.vstack([np.zeros((1, m)), incl[:-1]])
    np.testing.assert_allclose(Y[0, 0], W0[0][:, k][None, :] - pre, rtol=0, atol=1e-13)


def test_orthonormal_inputs_read_slow_weights():
    """Exclusive reads of mutually orthogonal inputs never see earlier writes."""
    rng = np.random.default_rng(6)
    d, m, T = 8, 5, 8
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    X = Q.T[None, None]                      # rows are orthonormal
    W0 = rng.standard_normal((1, m, d))
    G = rng.standard_normal((1, 1, T, m))
    Y = orc.scan_fwd(W0, X, G, 0.7)
    np.testing.assert_allclose(Y[0, 0], X[0, 0] @ W0[0].T, atol=1e-13)
    # Inclusive reads see exactly their own write: y_t = W0 x_t - eta g_t |x_t|^2.
    Yi = orc.scan_fwd(W0, X, G, 0.7, orc.INCLUSIVE)
    np.testing.assert_allclose(Yi[0, 0], X[0, 0] @ W0[0].T - 0.7 * G[0, 0], atol=1e-13)


def test_input_scaling():
    """Scaling X by c scales the W0 term by c and the Delta term by c^2."""
    W0, X, G, e, _ = rand_problem(1, 2, 10, 4, 3, seed=9)
    c = 1.7
    base = orc.scan_fwd(W0, X, G, 0.0)
    full = orc.scan_fwd(W0, X, G, e)
    scaled = orc.scan_fwd(W0, c * X, G, e)
    np.testing.assert_allclose(scaled, c * base + c * c * (full - base), rtol=1e-12, atol=1e-12)


def test_dw0_is_plain_product():
    W0, X, G, e, dY = rand_problem(3, 2, 9, 4, 5, seed=10)
    out = orc.scan_bwd(W0, X, G, e, dY)
    ref = np.einsum("bhtm,bhtd->hmd", dY, X)
    assert rel_err(out["dw0"], ref) < 1e-13


# --------------------------------------------------------------------------
# Finite differences (exact up to rounding: L is quadratic in X, linear else)
# --------------------------------------------------------------------------

def _loss(W0, X, G, e, dY, prefix):
    return float(np.sum(orc.scan_fwd(W0, X, G, e, prefix) * dY))


def _fd(f, a, h=1e-3):
    g = np.zeros_like(a)
    it = np.nditer(a, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        ap, am = a.copy(), a.copy()
        ap[i] += h
        am[i] -= h
        g[i] = (f(ap) - f(am)) / (2 * h)
    return g


@pytest.mark.parametrize("prefix", PREFIXES)
def test_backward_matches_finite_differences(prefix):
    W0, X, G, e, dY = rand_problem(2, 1, 5, 3, 4, seed=11)
    out = orc.scan_bwd(W0, X, G, e, dY, prefix)
    fd_x = _fd(lambda a: _loss(W0, a, G, e, dY, prefix), X)
    fd_g = _fd(lambda a: _loss(W0, X, a, e, dY, prefix), G)
    fd_e = _fd(lambda a: _loss(W0, X, G, a, dY, prefix), e)
    fd_w = _fd(lambda a: _loss(a, X, G, e, dY, prefix), W0)
    assert rel_err(out["dx"], fd_x) < 1e-9
    assert rel_err(out["dg"], fd_g) < 1e-9
    assert rel_err(out["deta"], fd_e) < 1e-9
    assert rel_err(out["dw0"], fd_w) < 1e-9


def _split_read_write(W0, Xr, Xw, G, e, prefix):
    """y_t = (W0 - sum_{s<t or s<=t} e_s g_s xw_s^T) xr_t, reads and writes separate."""
    B, H, T, d = Xr.shape
    Y = np.zeros(G.shape)
    for t in range(T):
        last = t if prefix == orc.EXCLUSIVE else t + 1
        for s in range(last):
            Y[:, :, t] -= e[:, :, s, None] * G[:, :, s] * np.einsum(
                "bhd,bhd->bh", Xw[:, :, s], Xr[:, :, t])[..., None]
        Y[:, :, t] += np.einsum("hmd,bhd->bhm", W0, Xr[:, :, t])
    return Y


@pytest.mark.parametrize("prefix", PREFIXES)
def test_gtilde_is_read_side_gradient(prefix):
    """gtilde is dL/dx through the read alone (Eq. 4); dx - gtilde is the write side."""
    W0, X, G, e, dY = rand_problem(1, 2, 6, 3, 4, seed=12)
    out = orc.scan_bwd(W0, X, G, e, dY, prefix)
    fd_read = _fd(lambda a: float(np.sum(_split_read_write(W0, a, X, G, e, prefix) * dY)), X)
    fd_write = _fd(lambda a: float(np.sum(_split_read_write(W0, X, a, G, e, prefix) * dY)), X)
    assert rel_err(out["gtilde"], fd_read) < 1e-9
    assert rel_err(out["dx"] - out["gtilde"], fd_write) < 1e-9


@pytest.mark.parametrize("prefix", PREFIXES)
def test_adjoint_identity_complex_step(prefix):
    """<dY, J v> (complex-step JVP, exact to rounding) equals <J^T dY, v>."""
    W0, X, G, e, dY = rand_problem(2, 2, 8, 4, 3, seed=13)
    rng = np.random.default_rng(14)
    vW, vX, vG, ve = (rng.standard_normal(a.shape) for a in (W0, X, G, e))
    h = 1e-30
    Yc = orc.scan_fwd(W0 + 1j * h * vW, X + 1j * h * vX, G + 1j * h * vG, e + 1j * h * ve, prefix)
    jvp = float(np.sum(np.imag(Yc) / h * dY))
    out = orc.scan_bwd(W0, X, G, e, dY, prefix)
    vjp = float(np.sum(out["dw0"] * vW) + np.sum(out["dx"] * vX) +
                np.sum(out["dg"] * vG) + np.sum(out["deta"] * ve))
    assert abs(jvp - vjp) <= 1e-12 * max(1.0, abs(jvp))


# --------------------------------------------------------------------------
# Deployment: decode steps equal the exclusive scan (Theorem 1)
# --------------------------------------------------------------------------

def test_decode_steps_equal_scan():
    rng = np.random.default_rng(15)
    S, H, T, d, m = 3, 2, 12, 5, 4
    W0 = rng.standard_normal((H, m, d))
    X = rng.standard_normal((S, H, T, d))
    G = rng.standard_normal((S, H, T, m))
    e = rng.uniform(0.1, 0.4, size=(S, H, T))
    Y = orc.scan_fwd(W0, X, G, e)
    W = np.broadcast_to(W0, (S, H, m, d)).copy()
    for t in range(T):
        y, W = orc.decode_step(W, X[:, :, t], G[:, :, t], e[:, :, t])
        np.testing.assert_allclose(y, Y[:, :, t], rtol=0, atol=1e-12)
    final = W0[None] - np.einsum("sht,shtm,shtd->shmd", e, G, X)
    np.testing.assert_allclose(W, final, rtol=0, atol=1e-12)


def test_oracle_rejects_unknown_prefix():
    W0, X, G, e, dY = rand_problem(1, 1, 2, 2, 2)
    with pytest.raises(ValueError):
        orc.scan_fwd(W0, X, G, e, "shifted")


# --------------------------------------------------------------------------
# Point evaluation from the closed-form sums (used for sampled checks of
# sequences too long for the sequential sweeps)
# --------------------------------------------------------------------------

def test_outer_sum_of_repeated_token():
    """n copies of (a, b) with step w sum to n w a b^T; ranges add up."""
    rng = np.random.default_rng(31)
    a, b = rng.standard_normal(5), rng.standard_normal(3)
    A, Bm = np.tile(a, (40, 1)), np.tile(b, (40, 1))
    np.testing.assert_allclose(orc.outer_sum(A, Bm, 0.25, 7, 19), 12 * 0.25 * np.outer(a, b), rtol=1e-13)
    w = rng.uniform(0, 1, 40)
    whole = orc.outer_sum(A, Bm, w, 0, 40)
    parts = orc.outer_sum(A, Bm, w, 0, 13) + orc.outer_sum(A, Bm, w, 13, 40)
    np.testing.assert_allclose(parts, whole, rtol=1e-13)
    np.testing.assert_allclose(whole, w.sum() * np.outer(a, b), rtol=1e-13)
    assert np.all(orc.outer_sum(A, Bm, w, 5, 5) == 0.0)


@pytest.mark.parametrize("prefix", PREFIXES)
def test_token_outputs_match_sweeps(prefix):
    """Closed-form point outputs equal the sequential sweeps at every token."""
    W0, X, G, e, dY = rand_problem(1, 1, 23, 6, 4, seed=17)
    Y = orc.scan_fwd(W0, X, G, e, prefix)
    ref = orc.scan_bwd(W0, X, G, e, dY, prefix)
    x, g, dy, et = X[0, 0], G[0, 0], dY[0, 0], e[0, 0]
    T = x.shape[0]
    inc = prefix == orc.INCLUSIVE
    for t in range(T):
        Wr = W0[0] - orc.outer_sum(g, x, et, 0, t + 1 if inc else t)
        R = orc.outer_sum(dy, x, 1.0, t if inc else t + 1, T)
        o = orc.token_outputs(Wr, R, x[t], g[t], et[t], dy[t])
        assert rel_err(o["y"], Y[0, 0, t]) < 1e-12
        for k in ("gtilde", "dx", "dg"):
            assert rel_err(o[k], ref[k][0, 0, t]) < 1e-12, (k, t)
        assert abs(o["deta"] - ref["deta"][0, 0, t]) <= 1e-12 * max(1.0, np.max(np.abs(ref["deta"])))
    np.testing.assert_allclose(orc.outer_sum(dy, x, 1.0, 0, T), ref["dw0"][0], rtol=1e-12)


# --------------------------------------------------------------------------
# Retention (Section 3, Eq. 2 general form) and resets
# --------------------------------------------------------------------------

def rand_alpha(B, H, T, seed, lo=0.0, hi=1.0):
    return np.random.default_rng(seed).uniform(lo, hi, size=(B, H, T))


def closed_form_retention(W0, X, G, eta, alpha, prefix):
    """Eq. 2 expanded: each write discounted by the explicit product of the
    retentions between it and the read (empty products are one)."""
    B, H, T, d = X.shape
    e = np.broadcast_to(np.asarray(eta, float), (B, H, T))
    Y = np.empty(G.shape)
    for b in range(B):
        for h in range(H):
            for t in range(T):
                y = W0[h] @ X[b, h, t]
                last = t if prefix == orc.EXCLUSIVE else t + 1
                for i in range(last):
                    hi = t if prefix == orc.EXCLUSIVE else t + 1
                    f = np.prod(alpha[b, h, i + 1:hi])
                    y = y - e[b, h, i] * f * (X[b, h, i] @ X[b, h, t]) * G[b, h, i]
                Y[b, h, t] = y
    return Y


@pytest.mark.parametrize("prefix", PREFIXES)
def test_retention_equals_expanded_sum(prefix):
    W0, X, G, e, _ = rand_problem(2, 2, 9, 4, 3, seed=40)
    a = rand_alpha(2, 2, 9, 41)
    Y = orc.scan_fwd(W0, X, G, e, prefix, alpha=a)
    assert rel_err(Y, closed_form_retention(W0, X, G, e, a, prefix)) < 1e-12


def test_unit_retention_is_the_plain_scan():
    W0, X, G, e, dY = rand_problem(2, 2, 10, 4, 3, seed=42)
    for prefix in PREFIXES:
        np.testing.assert_allclose(orc.scan_fwd(W0, X, G, e, prefix, alpha=1.0),
                                   orc.scan_fwd(W0, X, G, e, prefix), rtol=1e-13, atol=1e-13)
        r1 = orc.scan_bwd(W0, X, G, e, dY, prefix, alpha=1.0)
        r0 = orc.scan_bwd(W0, X, G, e, dY, prefix)
        for k in r0:
            np.testing.assert_allclose(r1[k], r0[k], rtol=1e-12, atol=1e-12)


def test_zero_retention_keeps_only_the_last_write():
    """alpha = 0: y_t = W0 x_t - eta_{t-1} (x_{t-1} . x_t) g_{t-1} (exclusive)."""
    W0, X, G, e, _ = rand_problem(1, 2, 8, 4, 3, seed=43)
    Y = orc.scan_fwd(W0, X, G, e, alpha=0.0)
    for h in range(2):
        x, g = X[0, h], G[0, h]
        ref = x @ W0[h].T
        ref[1:] -= (e[0, h, :-1] * np.sum(x[:-1] * x[1:], axis=1))[:, None] * g[:-1]
        np.testing.assert_allclose(Y[0, h], ref, rtol=0, atol=1e-13)


def test_constant_retention_on_unit_inputs_is_an_ema():
    """x_t = e_k, constant alpha: y_t = W0 e_k - sum_{s<t} alpha^(t-1-s) eta_s g_s."""
    rng = np.random.default_rng(44)
    T, d, m, k, al = 12, 4, 3, 1, 0.7
    W0 = rng.standard_normal((1, m, d))
    X = np.zeros((1, 1, T, d))
    X[..., k] = 1.0
    G = rng.standard_normal((1, 1, T, m))
    e = rng.uniform(0.1, 0.5, size=(1, 1, T))
    Y = orc.scan_fwd(W0, X, G, e, alpha=al)
    for t in range(T):
        ref = W0[0][:, k] - sum(al ** (t - 1 - s) * e[0, 0, s] * G[0, 0, s] for s in range(t))
        np.testing.assert_allclose(Y[0, 0, t], ref, rtol=0, atol=1e-13)


def test_retention_without_writes_is_static():
    """eta = 0 keeps W = W0 whatever alpha is: no gate gradient, gtilde = W0^T dY."""
    W0, X, G, _, dY = rand_problem(2, 1, 7, 4, 3, seed=45)
    a = rand_alpha(2, 1, 7, 46)
    Y = orc.scan_fwd(W0, X, G, 0.0, alpha=a)
    np.testing.assert_allclose(Y, np.einsum("hmd,bhtd->bhtm", W0, X), atol=1e-14)
    out = orc.scan_bwd(W0, X, G, 0.0, dY, alpha=a)
    np.testing.assert_array_equal(out["dalpha"], 0.0)
    np.testing.assert_allclose(out["gtilde"], np.einsum("hmd,bhtm->bhtd", W0, dY), atol=1e-14)


@pytest.mark.parametrize("prefix", PREFIXES)
def test_retention_gradients_complex_step(prefix):
    """Every gradient, dalpha included, against per-element complex-step
    derivatives of L = sum <dY, y> (exact to rounding)."""
    W0, X, G, e, dY = rand_problem(1, 1, 6, 3, 2, seed=47)
    a = rand_alpha(1, 1, 6, 48, 0.2, 1.0)
    out = orc.scan_bwd(W0, X, G, e, dY, prefix, alpha=a)
    h = 1e-30

    def cs(which, arr):
        g = np.zeros(arr.shape)
        for i in np.ndindex(arr.shape):
            args = {"W0": W0, "X": X, "G": G, "e": e, "a": a}
            p = arr.astype(complex)
            p[i] += 1j * h
            args[which] = p
            Y = orc.scan_fwd(args["W0"], args["X"], args["G"], args["e"], prefix, alpha=args["a"])
            g[i] = np.sum(np.imag(Y) * dY) / h
        return g

    assert rel_err(out["dalpha"], cs("a", a)) < 1e-12
    assert rel_err(out["deta"], cs("e", e)) < 1e-12
    assert rel_err(out["dg"], cs("G", G)) < 1e-12
    assert rel_err(out["dx"], cs("X", X)) < 1e-12
    assert rel_err(out["dw0"], cs("W0", W0)) < 1e-12


@pytest.mark.parametrize("prefix", PREFIXES)
def test_retention_gtilde_is_read_side(prefix):
    """gtilde stays the transpose read (W_0 + Delta_t)^T dY_t of Eq. 4."""
    W0, X, G, e, dY = rand_problem(1, 2, 7, 3, 4, seed=49)
    a = rand_alpha(1, 2, 7, 50)
    out = orc.scan_bwd(W0, X, G, e, dY, prefix, alpha=a)
    # The read weights follow from the expanded sum with x replaced by basis vectors.
    B, H, T, d = X.shape
    for h in range(H):
        for t in range(T):
            W = W0[h].copy()
            last = t if prefix == orc.EXCLUSIVE else t + 1
            for i in range(last):
                f = np.prod(a[0, h, i + 1:last])
                W -= e[0, h, i] * f * np.outer(G[0, h, i], X[0, h, i])
            np.testing.assert_allclose(out["gtilde"][0, h, t], W.T @ dY[0, h, t], rtol=1e-12, atol=1e-12)


def test_decode_with_retention_equals_scan():
    rng = np.random.default_rng(51)
    S, H, T, d, m = 3, 2, 10, 5, 4
    W0 = rng.standard_normal((H, m, d))
    X = rng.standard_normal((S, H, T, d))
    G = rng.standard_normal((S, H, T, m))
    e = rng.uniform(0.1, 0.4, size=(S, H, T))
    a = rng.uniform(0.0, 1.0, size=(S, H, T))
    Y = orc.scan_fwd(W0, X, G, e, alpha=a)
    W = np.broadcast_to(W0, (S, H, m, d)).copy()
    for t in range(T):
        y, W = orc.decode_step(W, X[:, :, t], G[:, :, t], e[:, :, t], alpha=a[:, :, t], W0=W0)
        np.testing.assert_allclose(y, Y[:, :, t], rtol=0, atol=1e-12)
    final = np.broadcast_to(W0, (S, H, m, d)).copy()
    for s in range(S):
        for h in range(H):
            for i in range(T):
                final[s, h] -= e[s, h, i] * np.prod(a[s, h, i + 1:T]) * np.outer(G[s, h, i], X[s, h, i])
    np.testing.assert_allclose(W, final, rtol=0, atol=1e-12)


@pytest.mark.parametrize("with_alpha", [False, True])
def test_reset_equals_separate_segments(with_alpha):
    """A reset splits the sequence: every output and gradient equals running
    the two segments on their own (the cut token's gates have no effect)."""
    W0, X, G, e, dY = rand_problem(2, 2, 11, 4, 3, seed=52)
    a = rand_alpha(2, 2, 11, 53) if with_alpha else None
    r = np.zeros((2, 11), np.int8)
    r[:, 0] = 1                      # a reset at t = 0 is a no-op
    r[0, 4] = r[1, 7] = 1
    Y = orc.scan_fwd(W0, X, G, e, alpha=a, reset=r)
    out = orc.scan_bwd(W0, X, G, e, dY, alpha=a, reset=r)
    for b, cut in ((0, 4), (1, 7)):
        for lo, hi in ((0, cut), (cut, 11)):
            sl = (slice(b, b + 1), slice(None), slice(lo, hi))
            asl = None if a is None else a[sl]
            Yp = orc.scan_fwd(W0, X[sl], G[sl], e[sl], alpha=asl)
            np.testing.assert_allclose(Y[sl], Yp, rtol=1e-13, atol=1e-13)
            op = orc.scan_bwd(W0, X[sl], G[sl], e[sl], dY[sl], alpha=asl)
            for k in ("gtilde", "dx", "dg", "deta") + (("dalpha",) if with_alpha else ()):
                np.testing.assert_allclose(out[k][sl], op[k], rtol=1e-12, atol=1e-12, err_msg=k)
    np.testing.assert_allclose(out["dw0"], np.einsum("bhtm,bhtd->hmd", dY, X), rtol=1e-13)


def test_hand_example_reset(golden_dir):
    """The hand example with a document starting at token 2: the scan, the
    explicit scan reads and decode all read W_0 there."""
    with open(os.path.join(golden_dir, "hand_T3_d2.json")) as f:
        gd = json.load(f)
    W0 = np.array(gd["W0"], float)[None]
    X = np.array(gd["X"], float)[None, None]
    G = np.array(gd["G"], float)[None, None]
    dY = np.array(gd["dY"], float)[None, None]
    r = np.array([[1, 0, 1]], np.uint8)
    exp = gd["reset_at_2"]
    np.testing.assert_array_equal(orc.scan_fwd(W0, X, G, gd["eta"], reset=r)[0, 0], np.array(exp["y"], float))
    np.testing.assert_array_equal(orc.scan_bwd(W0, X, G, gd["eta"], dY, reset=r)["gtilde"][0, 0],
                                  np.array(exp["gtilde"], float))
    reads = orc.scan_reads(W0, X, G, gd["eta"], Bq=dY, reset=r)
    np.testing.assert_array_equal(reads["y"][0, 0], np.array(exp["y"], float))
    np.testing.assert_array_equal(reads["gtilde"][0, 0], np.array(exp["gtilde"], float))
    W = np.array(gd["W0"], float)[None, None]
    for t in range(3):
        y, W = orc.decode_step(W, X[:, :, t], G[:, :, t], gd["eta"], W0=W0, reset=r[:, t])
        np.testing.assert_array_equal(y[0, 0], np.array(exp["y"][t], float))
    np.testing.assert_array_equal(W[0, 0], np.array(exp["decode_final_W"], float))


@pytest.mark.parametrize("with_alpha", [False, True])
def test_decode_with_resets_equals_scan(with_alpha):
    """T decode steps whose reset flags mark document starts reproduce the
    scan with the same flags, and end at the closed-form state: W_0 minus the
    writes of the last document, each discounted by the retentions after it."""
    rng = np.random.default_rng(56)
    S, H, T, d, m = 4, 2, 13, 5, 3
    W0 = rng.standard_normal((H, m, d))
    X = rng.standard_normal((S, H, T, d))
    G = rng.standard_normal((S, H, T, m))
    e = rng.uniform(0.1, 0.4, size=(S, H, T))
    a = rng.uniform(0.0, 1.0, size=(S, H, T)) if with_alpha else None
    r = (rng.uniform(size=(S, T)) < 0.25).astype(np.uint8)
    r[0] = 0
    r[1, 5] = r[2, 0] = r[2, T - 1] = 1
    Y = orc.scan_fwd(W0, X, G, e, alpha=a, reset=r)
    W = np.broadcast_to(W0, (S, H, m, d)).copy()
    for t in range(T):
        y, W = orc.decode_step(W, X[:, :, t], G[:, :, t], e[:, :, t],
                               alpha=None if a is None else a[:, :, t], W0=W0, reset=r[:, t])
        np.testing.assert_allclose(y, Y[:, :, t], rtol=0, atol=1e-12)
    for s in range(S):
        starts = np.nonzero(r[s])[0]
        lo = int(starts[-1]) if len(starts) else 0
        for h in range(H):
            final = W0[h].copy()
            for i in range(lo, T):
                f = 1.0 if a is None else np.prod(a[s, h, i + 1:T])
                final -= e[s, h, i] * f * np.outer(G[s, h, i], X[s, h, i])
            np.testing.assert_allclose(W[s, h], final, rtol=0, atol=1e-12)


def test_decode_reset_forgets_the_history():
    """After a reset the decode trajectory is that of a fresh state W_0: the
    steps before the reset have no effect on any later output."""
    rng = np.random.default_rng(57)
    S, H, T, d, m, cut = 2, 3, 9, 4, 4, 4
    W0 = rng.standard_normal((H, m, d))
    X = rng.standard_normal((S, H, T, d))
    G = rng.standard_normal((S, H, T, m))
    e, a = rng.uniform(0.1, 0.4, size=(S, H, T)), rng.uniform(0.5, 1.0, size=(S, H, T))
    W = rng.standard_normal((S, H, m, d))           # arbitrary history
    Wf = np.broadcast_to(W0, (S, H, m, d)).copy()   # fresh start at the cut
    flag = np.ones(S, np.uint8)
    for t in range(T):
        y, W = orc.decode_step(W, X[:, :, t], G[:, :, t], e[:, :, t], a[:, :, t], W0,
                               reset=flag if t == cut else None)
        if t >= cut:
            yf, Wf = orc.decode_step(Wf, X[:, :, t], G[:, :, t], e[:, :, t], a[:, :, t], W0)
            np.testing.assert_allclose(y, yf, rtol=0, atol=1e-12)
    np.testing.assert_allclose(W, Wf, rtol=0, atol=1e-12)


@pytest.mark.parametrize("alpha_kind", ["none", "uniform", "zeros"])
def test_scan_reads_equal_the_sweeps(alpha_kind):
    """The explicit causal sums of the scan-read equation equal the sequential
    learner's reads, forward and transpose, with retentions and resets."""
    B, H, T, d, m = 3, 2, 23, 4, 6
    W0, X, G, e, dY = rand_problem(B, H, T, d, m, seed=58)
    a = None
    if alpha_kind == "uniform":
        a = rand_alpha(B, H, T, 59)
    elif alpha_kind == "zeros":
        a = rand_alpha(B, H, T, 60)
        a[:, :, ::5] = 0.0
    r = np.zeros((B, T), np.uint8)
    r[0, 7] = r[1, 0] = r[1, 1] = r[2, 22] = r[2, 10] = 1
    reads = orc.scan_reads(W0, X, G, e, Bq=dY, alpha=a, reset=r)
    assert rel_err(reads["y"], orc.scan_fwd(W0, X, G, e, alpha=a, reset=r)) < 1e-12
    assert rel_err(reads["gtilde"], orc.scan_bwd(W0, X, G, e, dY, alpha=a, reset=r)["gtilde"]) < 1e-12


def test_scan_reads_equal_the_expanded_sum():
    """Retention without resets: the explicit sums equal Eq. 2 expanded with
    explicit products (a triple loop written independently above)."""
    W0, X, G, e, _ = rand_problem(2, 2, 9, 4, 3, seed=61)
    a = rand_alpha(2, 2, 9, 62)
    ref = closed_form_retention(W0, X, G, e, a, orc.EXCLUSIVE)
    assert rel_err(orc.scan_reads(W0, X, G, e, alpha=a)["y"], ref) < 1e-12


def test_scan_reads_with_other_queries():
    """Forward queries other than the inputs: (W_0 + Delta_t) a_t is linear in
    a_t, so querying with basis vectors recovers each W_t column by column."""
    B, H, T, d, m = 1, 1, 6, 3, 2
    W0, X, G, e, _ = rand_problem(B, H, T, d, m, seed=63)
    for k in range(d):
        A = np.zeros((B, H, T, d))
        A[..., k] = 1.0
        col = orc.scan_reads(W0, X, G, e, A=A)["y"][0, 0]
        for t in range(T):
            Wt = W0[0] - sum(e[0, 0, i] * np.outer(G[0, 0, i], X[0, 0, i]) for i in range(t))
            np.testing.assert_allclose(col[t], Wt[:, k], rtol=0, atol=1e-13)


def test_retention_dw0_is_plain_product():
    W0, X, G, e, dY = rand_problem(3, 2, 9, 4, 5, seed=54)
    out = orc.scan_bwd(W0, X, G, e, dY, alpha=rand_alpha(3, 2, 9, 55))
    assert rel_err(out["dw0"], np.einsum("bhtm,bhtd->hmd", dY, X)) < 1e-13


# --------------------------------------------------------------------------
# Two-map online MLP (Appendix A) and the FP64 recovery experiment
# (Section 5.1, Appendix B): tests/golden/mlp_toy.json
# --------------------------------------------------------------------------

def _toy(seed):
    rng = np.random.default_rng(seed)
    W10 = rng.normal(0, 0.5 / np.sqrt(4), (7, 4))
    W20 = rng.normal(0, 0.5 / np.sqrt(7), (3, 7))
    va, vm = rng.normal(0, 0.25, 4), rng.normal(0, 0.25, 4)
    X, C = rng.standard_normal((32, 4)), rng.standard_normal((32, 3))
    al = 1 / (1 + np.exp(-(X @ va + 1.5)))
    mu = 1 / (1 + np.exp(-(X @ vm - 0.2)))
    return W10, W20, X, C, al, mu


def test_mlp_toy_recovers_serial_ttt(golden_dir):
    """Serial TTT supplies exact costates; the parallel scans reproduce its
    outputs, hidden costates, input costates and first-matrix gradients at
    rounding level, and the slow-transpose control misses by O(0.1-1)."""
    gd = json.load(open(os.path.join(golden_dir, "mlp_toy.json")))
    paper, ctrl = gd["paper_max_abs_error"], gd["paper_slow_transpose_control"]
    worst = {"y": 0.0, "gz": 0.0, "gx": 0.0, "dW1": 0.0}
    cworst = {"gz": 0.0, "dW1": 0.0, "y": 0.0}
    for seed in gd["protocol"]["seeds"]:
        W10, W20, X, C, al, mu = _toy(seed)
        ser = orc.mlp_serial(W10, W20, X, C, al, mu)
        b = lambda a: a[None, None]  # noqa: E731
        f = orc.mlp_fwd(W10[None], W20[None], b(X), b(ser["gz"]), b(ser["gy"]), b(al), b(mu))
        gy = f["y"][0, 0] - C           # the reverse target from the scanned output
        r = orc.mlp_reverse(W10[None], W20[None], b(X), b(ser["gz"]), b(ser["gy"]), b(al), b(mu), b(gy))
        rc = orc.mlp_reverse(W10[None], W20[None], b(X), b(ser["gz"]), b(ser["gy"]), b(al), b(mu), b(gy),
                             slow_transpose=True)
        worst["y"] = max(worst["y"], np.max(np.abs(f["y"][0, 0] - ser["y"])))
        worst["gz"] = max(worst["gz"], np.max(np.abs(r["gz"][0, 0] - ser["gz"])))
        worst["gx"] = max(worst["gx"], np.max(np.abs(r["gx"][0, 0] - ser["gx"])))
        dW1 = np.einsum("tm,td->tmd", r["gz"][0, 0], X)
        worst["dW1"] = max(worst["dW1"], np.max(np.abs(dW1 - ser["dW1"])))
        cworst["gz"] = max(cworst["gz"], np.max(np.abs(rc["gz"][0, 0] - ser["gz"])))
        cworst["dW1"] = max(cworst["dW1"], np.max(np.abs(np.einsum("tm,td->tmd", rc["gz"][0, 0], X) - ser["dW1"])))
        cworst["y"] = max(cworst["y"], np.max(np.abs(rc["h"][0, 0] - ser["h"])))
    # Rounding level: within a few ulps of the paper's maxima.
    assert worst["y"] <= 4 * paper["outputs"]
    assert worst["gz"] <= 4 * paper["hidden_costates"]
    assert worst["dW1"] <= 4 * paper["first_matrix_gradients"]
    assert worst["gx"] <= 1e-15
    # The control changes only the reverse: same forward, gradients off by the
    # paper's order of magnitude.
    assert cworst["y"] <= 4 * paper["outputs"]
    for k, name in (("gz", "hidden_costates"), ("dW1", "first_matrix_gradients")):
        assert ctrl[name] / 10 <= cworst[k] <= 10 * ctrl[name], (k, cworst[k])


def test_mlp_with_unit_gates_is_two_scans():
    """alpha = 1, constant mu: the MLP forward is the plain scans of the two maps."""
    rng = np.random.default_rng(60)
    B, H, T, d, m, o = 2, 2, 9, 4, 5, 3
    W10, W20 = rng.standard_normal((H, m, d)), rng.standard_normal((H, o, m))
    X = rng.standard_normal((B, H, T, d))
    Gz, Gy = rng.standard_normal((B, H, T, m)), rng.standard_normal((B, H, T, o))
    f = orc.mlp_fwd(W10, W20, X, Gz, Gy, 1.0, 0.6)
    z = closed_form_fwd(W10, X, Gz, 0.6 / d, orc.EXCLUSIVE)
    np.testing.assert_allclose(f["z"], z, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(f["y"], closed_form_fwd(W20, np.tanh(z), Gy, 0.6 / m, orc.EXCLUSIVE),
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("with_alpha", [False, True])
def test_mlp_training_gradients_complex_step(with_alpha):
    """The MLP's gate and slow-weight gradients with the writes detached
    (Appendix E) against complex-step derivatives of
    L = sum_t <g_y, y_t>, y_t = (W2_0 + Delta2_t) h_t, h = sigma(z_hat), where
    Delta2 takes its write inputs from a fixed copy of h (the detached
    writes) and z_hat is the first scan; resets included.  y is evaluated with
    the explicit scan reads (reads of h, writes of the fixed copy)."""
    rng = np.random.default_rng(64)
    B, H, T, d, m, o = 2, 1, 9, 3, 4, 2
    W10 = rng.standard_normal((H, m, d)) * 0.5
    W20 = rng.standard_normal((H, o, m)) * 0.5
    X, Gz, Gy = rng.standard_normal((B, H, T, d)), rng.standard_normal((B, H, T, m)), rng.standard_normal((B, H, T, o))
    gy = rng.standard_normal((B, H, T, o))
    mu = rng.uniform(0.3, 1.5, (B, H, T))
    al = rng.uniform(0.3, 1.0, (B, H, T)) if with_alpha else None
    rs = np.zeros((B, T), np.uint8)
    rs[1, 4] = 1
    hbar = orc.act(orc.scan_fwd(W10, X, Gz, mu / d, alpha=al, reset=rs), "tanh")

    def loss(W10_, W20_, mu_, al_):
        z = orc.scan_fwd(W10_, X, Gz, mu_ / d, alpha=al_, reset=rs)
        y = orc.scan_reads(W20_, hbar, Gy, mu_ / m, A=orc.act(z, "tanh"), alpha=al_, reset=rs)["y"]
        return np.sum(y * gy)

    r = orc.mlp_reverse(W10, W20, X, Gz, Gy, al, mu, gy, kind="tanh", reset=rs)
    h_ = 1e-30
    params = {"W10": W10, "W20": W20, "mu": mu, "al": al}

    def cs(name):
        base = params[name]
        g = np.zeros(base.shape)
        for i in np.ndindex(base.shape):
            p_ = dict(params)
            v = base.astype(complex)
            v[i] += 1j * h_
            p_[name] = v
            g[i] = np.imag(loss(p_["W10"], p_["W20"], p_["mu"], p_["al"])) / h_
        return g

    assert rel_err(r["dw10"], cs("W10")) < 1e-12
    assert rel_err(r["dw20"], cs("W20")) < 1e-12
    assert rel_err(r["dmu"], cs("mu")) < 1e-12
    if with_alpha:
        assert rel_err(r["dalpha"], cs("al")) < 1e-12
    else:
        assert "dalpha" not in r


@pytest.mark.parametrize("kind", orc.ACTS)
def test_activation_derivatives(kind):
    z = np.linspace(-4, 4, 41)
    h = 1e-6
    fd = (orc.act(z + h, kind) - orc.act(z - h, kind)) / (2 * h)
    np.testing.assert_allclose(orc.act_grad(z, kind), fd, rtol=0, atol=1e-8)
    if kind in ("gelu", "gelu_tanh"):
        # GELU(z) - GELU(-z) = z, GELU(0) = 0, GELU -> z for large z (both forms)
        np.testing.assert_allclose(orc.act(z, kind) - orc.act(-z, kind), z, atol=1e-15)
        assert orc.act(np.array(0.0), kind) == 0.0
        np.testing.assert_allclose(orc.act(np.array(10.0), kind), 10.0, rtol=1e-15)
    if kind == "gelu_tanh":
        # The tanh form approximates z Phi(z) to within 5e-4 everywhere
        # (largest gap near |z| = 2.7), slopes to within 1e-3; a dropped cubic
        # term or a wrong sqrt(2/pi) factor breaks both bounds.
        from scipy.special import erf
        zz = np.linspace(-8, 8, 20001)
        exact = 0.5 * zz * (1.0 + erf(zz / np.sqrt(2.0)))
        slope = 0.5 * (1.0 + erf(zz / np.sqrt(2.0))) + zz * np.exp(-0.5 * zz * zz) / np.sqrt(2.0 * np.pi)
        gap = np.abs(orc.act(zz, kind) - exact)
        assert gap.max() < 5e-4 and gap.max() > 1e-4
        assert np.abs(orc.act_grad(zz, kind) - slope).max() < 1e-3


def test_bf16_rounding_of_hidden_activations():
    v = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -7, -2.5, 3.0 + 2 ** -6 + 2 ** -9, 0.0])
    r = orc.round_bf16(v)
    # representable values are kept; ties go to the even mantissa
    np.testing.assert_array_equal(r, [1.0, 1.0, 1.0 + 2 ** -6, 1.0 + 2 ** -7, -2.5, 3.0 + 2 ** -6 + 2 ** -9 - 2 ** -9, 0.0])
