"""Float64 CPU oracle for the GradLev fast-weight scans and decode step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the test suite, the smoke check and the CPU-baseline
leg of the benchmark use it.  It shares no code, tables or constants with the
HIP library; the two meet only through the seeded input generators.

What is computed (GradLev, arXiv 2609.34174):

* Section 3, "Observation": with retention alpha = 1 the adapted map
  y_t = W_t x_t evolves by online gradient descent,
  W_{t+1} = W_t - eta_t g_t x_t^T, so W_t = W_0 + Delta_t with
  Delta_t = -sum_{i<t} eta_i g_i x_i^T and Delta_0 = 0 (Eq. 2, empty sums are
  zero).
* Section 3, step 2 (Eq. 3): the forward scan replaces g by the proposals
  g_hat and reads *before* it writes: y_hat_t = (W_0 + Delta_hat_t) x_t.
  The optional "inclusive" convention reads after the token's own write
  (y_t = (W_0 + Delta_hat_{t+1}) x_t); the paper's method is exclusive.
* Section 3, step 3 (Eq. 4): the grounded target passed to the map input is
  g_tilde^x_t = (W_0 + Delta_hat_t)^T g_tilde_t, a transpose read over the same
  historical writes, queried by the upstream costate (here called dY).
* The reverse-time terms are the vector-Jacobian product of
  L = sum_t <dY_t, y_hat_t> through the prefix sums: the gradients with respect
  to the proposals g_hat, the write-side inputs x, the step sizes eta and W_0.
  They are accumulated by an explicit reverse-time sweep over the suffix
  R_t = sum_{u>t} dY_u x_u^T (u >= t for the inclusive convention).
  The paper keeps read and gate derivatives and detaches writes during its own
  training (Appendix E, "Initialization and gradients"); the full set is
  returned and callers drop what they detach.
* Deployment (Section 3, "Training objective", last sentences): score with
  the current weights, then write the true costate: y = W x, W <- W - eta g x^T.
* Retention (Section 3, Eq. 2, general form): with per-token alpha_t in [0, 1]
  the write is centered weight decay, W_{t+1} = W_0 + alpha_t (W_t - W_0)
  - eta_t g_t x_t^T, so that Delta_t = W_t - W_0 discounts write i by the
  retentions alpha_{i+1} .. alpha_{t-1}.  The reverse sweep then carries
  Lambda_t = dL/dDelta_t = dY_t x_t^T + alpha_t Lambda_{t+1} (the retention
  scales the suffix), and the gate gradient is dalpha_t = <Lambda_{t+1},
  Delta_t>_F (Appendix E keeps gate derivatives).  Without alpha every
  retention is one and the arithmetic is the plain prefix sum above.
* Two-map online MLP (Appendix A): z = W1 x, h = sigma(z), y = W2 h, both
  maps written with the shared retention and eta_1 = mu / d, eta_2 = mu / m.
  Given costate proposals the forward is two exclusive scans in layer order;
  the reverse target of the hidden layer is sigma'(z) times the transpose
  read of the second scan (mlp_fwd, mlp_reverse), and the serial learner it
  must reproduce is mlp_serial.
* Resets (Section 3, Eq. 2 holds within each reset segment): a token flagged
  as a reset reads W_0 again, i.e. Delta_t = 0.  That is the same as a zero
  retention and a zero step size at the token before it, which is how the
  sweeps apply it; the gate gradients of that token are then reported as 0
  (its gates have no effect).

Everything here is the plain sequential definition, token by token, in float64
(complex inputs are also accepted, which the tests use for complex-step
derivatives).  It is deliberately slow and obviously correct; there is no
chunking, blocking or reordering.

Shapes (row-major):
  W0  [H, m, d]      slow weights, one matrix per head
  X   [B, H, T, d]   map inputs x_t
  G   [B, H, T, m]   proposed costates g_hat_t
  eta [B, H, T]      step sizes (a Python scalar is broadcast)
  dY  [B, H, T, m]   upstream costates dL/dy_hat_t
  alpha [B, H, T]    retentions (optional; a Python scalar is broadcast)
  reset [B, T]       optional 0/1 flags, 1 = the token starts a new segment
"""

from __future__ import annotations

import numpy as np

EXCLUSIVE = "exclusive"
INCLUSIVE = "inclusive"


def _as_array(a):
    a = np.asarray(a)
    if a.dtype.kind in "iub":
        a = a.astype(np.float64)
    if a.dtype.kind == "f":
        a = a.astype(np.float64)
    return a


def _eta_array(eta, B, H, T):
    e = _as_array(eta)
    if e.ndim == 0:
        return np.broadcast_to(e, (B, H, T))
    if e.shape != (B, H, T):
        raise ValueError(f"eta must be a scalar or [B,H,T]={B,H,T}, got {e.shape}")
    return e


def _gates(eta, alpha, reset, B, H, T):
    """Per-token (eta, alpha) with resets applied; alpha None means one.

    A reset at token t (t > 0) clears the fast weights before t's read: the
    write of token t - 1 is dropped and the state it would carry is
    forgotten (eta_{t-1} = alpha_{t-1} = 0).  A reset at t = 0 changes
    nothing (Delta_0 = 0).  Returns (eta, alpha_or_None, gate_mask) where
    gate_mask zeroes the gate gradients of the tokens a reset overrides.
    """
    e = _eta_array(eta, B, H, T)
    a = None if alpha is None else _eta_array(alpha, B, H, T)
    keep = np.ones((B, H, T))
    if reset is not None:
        r = np.asarray(reset)
        if r.shape != (B, T):
            raise ValueError(f"reset must be [B,T]={B,T}, got {r.shape}")
        cut = np.zeros((B, T), bool)
        cut[:, :-1] = r[:, 1:] != 0
        cut = np.broadcast_to(cut[:, None, :], (B, H, T))
        e = np.where(cut, 0.0, e)
        a = np.where(cut, 0.0, 1.0 if a is None else a)
        keep = np.where(cut, 0.0, keep)
    return e, a, keep


def _check(prefix):
    if prefix not in (EXCLUSIVE, INCLUSIVE):
        raise ValueError(f"prefix must be '{EXCLUSIVE}' or '{INCLUSIVE}'")


def _write(W, W0, a_t, e_t, g, x):
    """One write of Eq. 2: W_0 + alpha (W - W_0) - eta g x^T (alpha None: W - eta g x^T)."""
    write = e_t[:, :, None, None] * g[:, :, :, None] * x[:, :, None, :]
    if a_t is None:
        return W - write
    return W0 + a_t[:, :, None, None] * (W - W0) - write


def scan_fwd(W0, X, G, eta, prefix=EXCLUSIVE, alpha=None, reset=None):
    """Adapted outputs y_hat_t = W_t x_t of the sequential online learner.

    Follows Section 3, Eq. 3: Delta_0 = 0, read y_t with the current weights,
    then write (exclusive).  The inclusive reading writes first.  The write
    is W <- W - eta_t g_t x_t^T, or the centered decay of Eq. 2 when
    retentions are given.  Returns Y [B, H, T, m].
    """
    _check(prefix)
    W0, X, G = _as_array(W0), _as_array(X), _as_array(G)
    B, H, T, d = X.shape
    m = G.shape[-1]
    e, a, _ = _gates(eta, alpha, reset, B, H, T)
    dt = np.result_type(W0, X, G, e, 0.0 if a is None else a)
    W0b = np.broadcast_to(W0, (B, H, m, d)).astype(dt)
    W = W0b.copy()
    Y = np.zeros((B, H, T, m), dt)
    for t in range(T):
        x, g = X[:, :, t, :], G[:, :, t, :]
        at = None if a is None else a[:, :, t]
        if prefix == INCLUSIVE:
            W = _write(W, W0b, at, e[:, :, t], g, x)
        Y[:, :, t, :] = np.einsum("bhmd,bhd->bhm", W, x)
        if prefix == EXCLUSIVE:
            W = _write(W, W0b, at, e[:, :, t], g, x)
    return Y


def scan_bwd(W0, X, G, eta, dY, prefix=EXCLUSIVE, alpha=None, reset=None):
    """Backward of the forward scan for L = sum_t <dY_t, y_hat_t>.

    Two sweeps, each the plain definition:

    * forward-time sweep (Section 3, Eq. 4 and Appendix C, Eq. 16): the
      transpose read gtilde_t = W_t^T dY_t with the same weights the forward
      read used (W_0 + Delta_hat_t, or Delta_hat_{t+1} when inclusive);
    * reverse-time sweep: Lambda is dL/dDelta of the state that token t's
      write produces: the suffix sum of dY_u x_u^T over the reads that see
      write t (u > t, or u >= t when inclusive), each discounted by the
      retentions between (Lambda_t = dY_t x_t^T + alpha_t Lambda_{t+1}).
      u_t = -Lambda x_t, dG_t = eta_t u_t, deta_t = <g_t, u_t>,
      write-side dx_t = -eta_t Lambda^T g_t and, with retentions,
      dalpha_t = <Lambda, Delta_t>_F (Delta_t = W_t - W_0 before t's write).

    Returns a dict with
      gtilde [B,H,T,d]  read-side gradient (the paper's grounded target),
      dx     [B,H,T,d]  total dL/dx = gtilde + write-side term,
      dg     [B,H,T,m], deta [B,H,T], dw0 [H,m,d] (summed over the batch),
      dalpha [B,H,T]    (only when alpha is given).
    """
    _check(prefix)
    W0, X, G, dY = _as_array(W0), _as_array(X), _as_array(G), _as_array(dY)
    B, H, T, d = X.shape
    m = G.shape[-1]
    e, a, keep = _gates(eta, alpha, reset, B, H, T)
    dt = np.result_type(W0, X, G, e, dY, 0.0 if a is None else a)
    W0b = np.broadcast_to(W0, (B, H, m, d)).astype(dt)

    def write(W, t):
        return _write(W, W0b, None if a is None else a[:, :, t], e[:, :, t], G[:, :, t], X[:, :, t])

    # Forward-time sweep: transpose reads over the historical writes.  With
    # retentions, the weights before every block of K writes are kept so the
    # reverse sweep can replay each block (Delta_t is needed there).
    K = 64
    ckpt = {}
    W = W0b.copy()
    gtilde = np.zeros((B, H, T, d), dt)
    for t in range(T):
        if a is not None and t % K == 0:
            ckpt[t] = W.copy()
        if prefix == INCLUSIVE:
            W = write(W, t)
        gtilde[:, :, t, :] = np.einsum("bhmd,bhm->bhd", W, dY[:, :, t, :])
        if prefix == EXCLUSIVE:
            W = write(W, t)

    # Reverse-time sweep: explicit suffix accumulation.
    Lam = np.zeros((B, H, m, d), dt)
    dg = np.zeros((B, H, T, m), dt)
    deta = np.zeros((B, H, T), dt)
    dalpha = np.zeros((B, H, T), dt)
    dxw = np.zeros((B, H, T, d), dt)
    hist = []
    for t in range(T - 1, -1, -1):
        x, g, dy = X[:, :, t, :], G[:, :, t, :], dY[:, :, t, :]
        if a is not None and not hist:
            # Replay the block holding t: hist[i] = W_{b0 + i} before its write.
            b0 = t - t % K
            Wr = ckpt[b0].copy()
            for s in range(b0, t + 1):
                hist.append(Wr)
                Wr = write(Wr, s)
        read = dy[:, :, :, None] * x[:, :, None, :]
        if prefix == INCLUSIVE:
            # Lambda becomes dL/dDelta_{t+1}; the next token's retention
            # discounts what lies beyond it.
            if a is not None and t + 1 < T:
                Lam = a[:, :, t + 1, None, None] * Lam
            Lam = Lam + read
        u = -np.einsum("bhmd,bhd->bhm", Lam, x)
        dg[:, :, t, :] = e[:, :, t, None] * u
        deta[:, :, t] = np.einsum("bhm,bhm->bh", g, u)
        dxw[:, :, t, :] = -e[:, :, t, None] * np.einsum("bhmd,bhm->bhd", Lam, g)
        if a is not None:
            Delta = hist.pop() - W0b
            dalpha[:, :, t] = np.einsum("bhmd,bhmd->bh", Lam, Delta)
        if prefix == EXCLUSIVE:
            if a is not None:
                Lam = a[:, :, t, None, None] * Lam
            Lam = Lam + read
    # dL/dW_0: every read sees W_0 undiscounted (the decay is centered), so it
    # is sum_t dY_t x_t^T, which the sweep accumulates when alpha is one.
    dw0 = np.einsum("bhtm,bhtd->hmd", dY, X) if a is not None else Lam.sum(axis=0)
    out = {
        "gtilde": gtilde,
        "dx": gtilde + dxw,
        "dg": dg,
        "deta": deta * keep,
        "dw0": dw0,
    }
    if alpha is not None:
        out["dalpha"] = dalpha * keep
    return out


# ---------------------------------------------------------------------------
# Two-map online MLP (Appendix A): z = W1 x, h = sigma(z), y = W2 h
# ---------------------------------------------------------------------------

ACTS = ("tanh", "gelu", "gelu_tanh")

# Constants of the tanh approximation of GELU (Hendrycks and Gimpel, 2016):
# GELU(z) ~ z/2 (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))).
_GELU_K0 = np.sqrt(2.0 / np.pi)
_GELU_K1 = 0.044715


def act(z, kind):
    """sigma(z): tanh; GELU written with the Gaussian CDF (erf form); or the
    tanh-approximate GELU that the paper's backbone uses (Appendix E,
    "Model and prefiller")."""
    if kind == "tanh":
        return np.tanh(z)
    if kind == "gelu":
        from scipy.special import erf
        return 0.5 * z * (1.0 + erf(z / np.sqrt(2.0)))
    if kind == "gelu_tanh":
        return 0.5 * z * (1.0 + np.tanh(_GELU_K0 * (z + _GELU_K1 * z ** 3)))
    raise ValueError(kind)


def act_grad(z, kind):
    """sigma'(z)."""
    if kind == "tanh":
        return 1.0 - np.tanh(z) ** 2
    if kind == "gelu":
        from scipy.special import erf
        return 0.5 * (1.0 + erf(z / np.sqrt(2.0))) + z * np.exp(-0.5 * z * z) / np.sqrt(2.0 * np.pi)
    if kind == "gelu_tanh":
        th = np.tanh(_GELU_K0 * (z + _GELU_K1 * z ** 3))
        return 0.5 * (1.0 + th) + 0.5 * z * (1.0 - th * th) * _GELU_K0 * (1.0 + 3.0 * _GELU_K1 * z * z)
    raise ValueError(kind)


def round_bf16(a):
    """Nearest bfloat16 value (ties to even), as float64; for hidden
    activations stored in bf16 between the two scans."""
    f = np.asarray(a, np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def mlp_serial(W10, W20, X, C, alpha, mu, kind="tanh"):
    """Serial test-time training of the two-map MLP on l_t = |y_t - c_t|^2 / 2.

    Appendix A, Eqs. for the online forward, reverse and simultaneous writes:
    both gradients use the pre-update weights, eta_1 = mu / d, eta_2 = mu / m,
    centered decay with the shared retention.  One sequence: X [T, d],
    C [T, o], alpha and mu [T].  Returns y, h, z, the costates g_y = y - c,
    g_z = sigma'(z) * W2^T g_y and g_x = W1^T g_z, and the first-matrix
    gradients g_z x^T [T, m, d].
    """
    W10, W20, X, C = (_as_array(a) for a in (W10, W20, X, C))
    a, mu = _as_array(alpha), _as_array(mu)
    T, d = X.shape
    m = W10.shape[0]
    W1, W2 = W10.copy(), W20.copy()
    out = {k: [] for k in ("y", "h", "z", "gy", "gz", "gx", "dW1")}
    for t in range(T):
        x = X[t]
        z = W1 @ x
        h = act(z, kind)
        y = W2 @ h
        gy = y - C[t]
        gz = act_grad(z, kind) * (W2.T @ gy)
        gx = W1.T @ gz
        W1 = W10 + a[t] * (W1 - W10) - (mu[t] / d) * np.outer(gz, x)
        W2 = W20 + a[t] * (W2 - W20) - (mu[t] / m) * np.outer(gy, h)
        for k, v in (("y", y), ("h", h), ("z", z), ("gy", gy), ("gz", gz), ("gx", gx),
                     ("dW1", np.outer(gz, x))):
            out[k].append(v)
    return {k: np.array(v) for k, v in out.items()}


def mlp_fwd(W10, W20, X, Gz, Gy, alpha, mu, kind="tanh", hidden_bf16=False, reset=None):
    """Parallel forward of Appendix A with costate proposals: z_hat by the
    first exclusive scan, h_hat = sigma(z_hat), y_hat by the second scan.

    Batched like the scans: W10 [H, m, d], W20 [H, o, m], X [B, H, T, d],
    Gz [B, H, T, m], Gy [B, H, T, o], alpha and mu scalars or [B, H, T].
    hidden_bf16 rounds h_hat to bfloat16 before the second scan (the storage
    of a bf16 pipeline).  Returns dict(z, h, y).
    """
    X = _as_array(X)
    B, H, T, d = X.shape
    m = _as_array(W10).shape[1]
    e1 = _as_array(mu) / d
    e2 = _as_array(mu) / m
    z = scan_fwd(W10, X, Gz, e1, alpha=alpha, reset=reset)
    h = act(z, kind)
    if hidden_bf16:
        h = round_bf16(h)
    y = scan_fwd(W20, h, Gy, e2, alpha=alpha, reset=reset)
    return {"z": z, "h": h, "y": y}


def mlp_reverse(W10, W20, X, Gz, Gy, alpha, mu, gy, kind="tanh", hidden_bf16=False,
                slow_transpose=False, reset=None, target_bf16=False):
    """Reconstructed costates of Appendix A (Eq. for the reverse targets):
    g_z = sigma'(z_hat) * (W2_0 + Delta2_hat_t)^T g_y, a transpose read of the
    second scan queried by the output costate g_y [B, H, T, o], and the input
    costate g_x = (W1_0 + Delta1_hat_t)^T g_z.  slow_transpose keeps only W2_0
    (the control of Section 5.1).  target_bf16 rounds g_z to bfloat16 before
    it queries the first scan (the storage of a bf16 pipeline).

    Also returns the training gradients of L = sum_t <g_y, y_hat_t> with the
    writes detached (Appendix E: costates and write inputs are detached; gate
    and read derivatives remain): the slow weights, dw20 = sum g_y h^T and
    dw10 = sum g_z x^T; the shared write strength, dmu = deta_1 / d + deta_2 / m
    (eta_1 = mu / d, eta_2 = mu / m, per token); and, with retentions, the
    shared retention, dalpha = dalpha_1 + dalpha_2 - each scan's gate gradient
    for its own upstream costate (g_y for the second, g_z for the first).
    Returns dict(z, h, gh, gz, gx, dmu, dw10, dw20[, dalpha]).
    """
    f = mlp_fwd(W10, W20, X, Gz, Gy, alpha, mu, kind, hidden_bf16, reset)
    X = _as_array(X)
    B, H, T, d = X.shape
    m = _as_array(W10).shape[1]
    e1 = _as_array(mu) / d
    e2 = _as_array(mu) / m
    gy = _as_array(gy)
    r2 = scan_bwd(W20, f["h"], Gy, e2, gy, alpha=alpha, reset=reset)
    if slow_transpose:
        gh = np.einsum("hom,bhto->bhtm", _as_array(W20), gy)
    else:
        gh = r2["gtilde"]
    gz = act_grad(f["z"], kind) * gh
    r1 = scan_bwd(W10, X, Gz, e1, round_bf16(gz) if target_bf16 else gz, alpha=alpha, reset=reset)
    out = {"z": f["z"], "h": f["h"], "gh": gh, "gz": gz, "gx": r1["gtilde"],
           "dmu": r1["deta"] / d + r2["deta"] / m, "dw10": r1["dw0"], "dw20": r2["dw0"]}
    if alpha is not None:
        out["dalpha"] = r1["dalpha"] + r2["dalpha"]
    return out


def outer_sum(A, Bm, w, lo, hi):
    """sum_{lo <= i < hi} w_i a_i b_i^T over tokens [lo, hi) of one sequence.

    A [T, m], Bm [T, d], w a scalar or [T].  Returns [m, d].  With A = G and
    w = eta this is minus the accumulated fast weights of Section 3, Eq. 2
    (Delta_t = -outer_sum(G, X, eta, 0, t)); with A = dY and w = 1 it is the
    costate suffix R of the reverse-time sweep.  Sums over disjoint ranges add
    up (linearity), which is how long sequences are handled a block at a time.
    """
    a, b = _as_array(A)[lo:hi], _as_array(Bm)[lo:hi]
    wv = _as_array(w)
    if wv.ndim:
        wv = wv[lo:hi, None]
    return (a * wv).T @ b


def token_outputs(W_read, R, x, g, eta_t, dy):
    """Every scan output at one token from the closed forms of the sums.

    W_read is the weight matrix the token's read sees (W_0 minus the writes
    before it, or up to and including it for the inclusive convention), R the
    suffix sum of dY_u x_u^T over the reads that see the token's write.  The
    formulas are those of the sequential sweeps in :func:`scan_fwd` and
    :func:`scan_bwd`: y = W x, gtilde = W^T dY, u = -R x, dg = eta u,
    deta = <g, u>, dx = gtilde - eta R^T g.
    """
    W_read, R = _as_array(W_read), _as_array(R)
    x, g, dy, e = _as_array(x), _as_array(g), _as_array(dy), _as_array(eta_t)
    gt = W_read.T @ dy
    u = -(R @ x)
    return {"y": W_read @ x, "gtilde": gt, "dx": gt - e * (R.T @ g), "dg": e * u,
            "deta": g @ u}


def decode_step(W, x, g, eta, alpha=None, W0=None, reset=None):
    """One deployment step for every (sequence, head): score, then write.

    W [S,H,m,d], x [S,H,d], g [S,H,m], eta scalar or [S,H].
    Returns (y, W_next) with y = W x computed before the write and
    W_next = W - eta g x^T, or, with retentions alpha (scalar or [S,H]) and
    the slow weights W0 [H,m,d], the centered decay of Eq. 2:
    W_next = W0 + alpha (W - W0) - eta g x^T.

    reset [S] (0/1, optional, needs W0): a flagged sequence starts a new
    document at this step.  Its read excludes every earlier write (the scan
    reads of the appendix on forward and transpose reads; Eq. 2 holds within
    each reset segment), so the state is replaced by W0 before the read.
    """
    W, x, g = _as_array(W), _as_array(x), _as_array(g)
    if reset is not None:
        if W0 is None:
            raise ValueError("a reset needs the slow weights W0")
        r = np.asarray(reset)
        if r.shape != W.shape[:1]:
            raise ValueError(f"reset must be [S]={W.shape[:1]}, got {r.shape}")
        W = np.where((r != 0)[:, None, None, None], np.broadcast_to(_as_array(W0), W.shape), W)
    e = _as_array(eta)
    if e.ndim == 0:
        e = np.broadcast_to(e, W.shape[:2])
    y = np.einsum("shmd,shd->shm", W, x)
    write = e[:, :, None, None] * g[:, :, :, None] * x[:, :, None, :]
    if alpha is None:
        return y, W - write
    if W0 is None:
        raise ValueError("retention needs the slow weights W0")
    a = _as_array(alpha)
    if a.ndim == 0:
        a = np.broadcast_to(a, W.shape[:2])
    W0b = np.broadcast_to(_as_array(W0), W.shape)
    return y, W0b + a[:, :, None, None] * (W - W0b) - write


def scan_reads(W0, X, G, eta, A=None, Bq=None, alpha=None, reset=None):
    """The forward and transpose scan reads as explicit causal sums.

    The appendix on forward and transpose scan reads writes both reads of the
    exclusive scan out from the expanded form of Eq. 2 (Eq. 16):

        Delta_t a_t   = - sum_{i<t} eta_i (prod_{j=i+1}^{t-1} alpha_j) g_i (x_i . a_t)
        Delta_t^T b_t = - sum_{i<t} eta_i (prod_{j=i+1}^{t-1} alpha_j) x_i (g_i . b_t)

    where each read excludes the current write and every write before the
    most recent document or context reset.  This function evaluates those
    sums directly: a coefficient matrix K[t, i] = -eta_i prod(alpha) for the
    writes a read sees (i < t, no reset in i+1..t) and zero otherwise, then
    y_t = W_0 a_t + sum_i K[t, i] (x_i . a_t) g_i and
    gtilde_t = W_0^T b_t + sum_i K[t, i] (g_i . b_t) x_i with matrix
    products.  It is the same quantity the sequential sweeps produce, summed
    in another order, and costs O(T^2) per sequence, which is cheaper than
    the sweeps when the maps are wide.

    A [B,H,T,d] forward queries (default X), Bq [B,H,T,m] transpose queries
    (optional); eta and alpha scalars or [B,H,T] (alpha None means one);
    reset [B,T] 0/1 flags, 1 = the token starts a new document.
    Returns dict(y [B,H,T,m], and gtilde [B,H,T,d] when Bq is given).
    """
    W0, X, G = _as_array(W0), _as_array(X), _as_array(G)
    B, H, T, d = X.shape
    m = G.shape[-1]
    A = X if A is None else _as_array(A)
    e = _eta_array(eta, B, H, T)
    a = np.ones((B, H, T)) if alpha is None else _eta_array(alpha, B, H, T)
    doc = np.zeros((B, T), np.int64)
    if reset is not None:
        r = np.asarray(reset)
        if r.shape != (B, T):
            raise ValueError(f"reset must be [B,T]={B,T}, got {r.shape}")
        doc = np.cumsum(r != 0, axis=1)
    if Bq is not None:
        Bq = _as_array(Bq)
    dt = np.result_type(W0, X, G, A, e, a, 0.0 if Bq is None else Bq)
    y = np.zeros((B, H, T, m), dt)
    gt = None if Bq is None else np.zeros((B, H, T, d), dt)
    for b in range(B):
        sees = (doc[b][:, None] == doc[b][None, :]) & np.tri(T, T, -1, dtype=bool)
        for h in range(H):
            K = np.zeros((T, T), dt)
            for i in range(T - 1):
                # prod_{j=i+1}^{t-1} alpha_j for t = i+1 .. T-1 (empty product first)
                K[i + 1:, i] = -e[b, h, i] * np.cumprod(np.concatenate(([1.0], a[b, h, i + 1:T - 1])))
            K = np.where(sees, K, 0.0)
            x, g = X[b, h], G[b, h]
            y[b, h] = A[b, h] @ W0[h].T + (K * (A[b, h] @ x.T)) @ g
            if Bq is not None:
                gt[b, h] = Bq[b, h] @ W0[h] + (K * (Bq[b, h] @ g.T)) @ x
    out = {"y": y}
    if Bq is not None:
        out["gtilde"] = gt
    return out
