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


def _check(prefix):
    if prefix not in (EXCLUSIVE, INCLUSIVE):
        raise ValueError(f"prefix must be '{EXCLUSIVE}' or '{INCLUSIVE}'")


def scan_fwd(W0, X, G, eta, prefix=EXCLUSIVE):
    """Adapted outputs y_hat_t = W_t x_t of the sequential online learner.

    Follows Section 3, Eq. 3: Delta_0 = 0, read y_t with the current weights,
    then write W <- W - eta_t g_t x_t^T (exclusive).  The inclusive reading
    writes first.  Returns Y [B, H, T, m].
    """
    _check(prefix)
    W0, X, G = _as_array(W0), _as_array(X), _as_array(G)
    B, H, T, d = X.shape
    m = G.shape[-1]
    e = _eta_array(eta, B, H, T)
    dt = np.result_type(W0, X, G, e)
    W = np.broadcast_to(W0, (B, H, m, d)).astype(dt).copy()
    Y = np.zeros((B, H, T, m), dt)
    for t in range(T):
        x, g = X[:, :, t, :], G[:, :, t, :]
        write = e[:, :, t, None, None] * g[:, :, :, None] * x[:, :, None, :]
        if prefix == INCLUSIVE:
            W -= write
        Y[:, :, t, :] = np.einsum("bhmd,bhd->bhm", W, x)
        if prefix == EXCLUSIVE:
            W -= write
    return Y


def scan_bwd(W0, X, G, eta, dY, prefix=EXCLUSIVE):
    """Backward of the forward scan for L = sum_t <dY_t, y_hat_t>.

    Two sweeps, each the plain definition:

    * forward-time sweep (Section 3, Eq. 4 and Appendix C, Eq. 16): the
      transpose read gtilde_t = W_t^T dY_t with the same weights the forward
      read used (W_0 + Delta_hat_t, or Delta_hat_{t+1} when inclusive);
    * reverse-time sweep: with R the suffix sum of dY_u x_u^T over the reads
      that see write t (u > t, or u >= t when inclusive),
      u_t = -R x_t, dG_t = eta_t u_t, deta_t = <g_t, u_t>,
      write-side dx_t = -eta_t R^T g_t.

    Returns a dict with
      gtilde [B,H,T,d]  read-side gradient (the paper's grounded target),
      dx     [B,H,T,d]  total dL/dx = gtilde + write-side term,
      dg     [B,H,T,m], deta [B,H,T], dw0 [H,m,d] (summed over the batch).
    """
    _check(prefix)
    W0, X, G, dY = _as_array(W0), _as_array(X), _as_array(G), _as_array(dY)
    B, H, T, d = X.shape
    m = G.shape[-1]
    e = _eta_array(eta, B, H, T)
    dt = np.result_type(W0, X, G, e, dY)

    # Forward-time sweep: transpose reads over the historical writes.
    W = np.broadcast_to(W0, (B, H, m, d)).astype(dt).copy()
    gtilde = np.zeros((B, H, T, d), dt)
    for t in range(T):
        x, g = X[:, :, t, :], G[:, :, t, :]
        write = e[:, :, t, None, None] * g[:, :, :, None] * x[:, :, None, :]
        if prefix == INCLUSIVE:
            W -= write
        gtilde[:, :, t, :] = np.einsum("bhmd,bhm->bhd", W, dY[:, :, t, :])
        if prefix == EXCLUSIVE:
            W -= write

    # Reverse-time sweep: explicit suffix accumulation.
    R = np.zeros((B, H, m, d), dt)
    dg = np.zeros((B, H, T, m), dt)
    deta = np.zeros((B, H, T), dt)
    dxw = np.zeros((B, H, T, d), dt)
    for t in range(T - 1, -1, -1):
        x, g, dy = X[:, :, t, :], G[:, :, t, :], dY[:, :, t, :]
        if prefix == INCLUSIVE:
            R += dy[:, :, :, None] * x[:, :, None, :]
        u = -np.einsum("bhmd,bhd->bhm", R, x)
        dg[:, :, t, :] = e[:, :, t, None] * u
        deta[:, :, t] = np.einsum("bhm,bhm->bh", g, u)
        dxw[:, :, t, :] = -e[:, :, t, None] * np.einsum("bhmd,bhm->bhd", R, g)
        if prefix == EXCLUSIVE:
            R += dy[:, :, :, None] * x[:, :, None, :]
    # After the sweep R = sum over all t of dY_t x_t^T, which is dL/dW_0.
    return {
        "gtilde": gtilde,
        "dx": gtilde + dxw,
        "dg": dg,
        "deta": deta,
        "dw0": R.sum(axis=0),
    }


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


def decode_step(W, x, g, eta):
    """One deployment step for every (sequence, head): score, then write.

    W [S,H,m,d], x [S,H,d], g [S,H,m], eta scalar or [S,H].
    Returns (y, W_next) with y = W x computed before the write and
    W_next = W - eta g x^T.
    """
    W, x, g = _as_array(W), _as_array(x), _as_array(g)
    e = _as_array(eta)
    if e.ndim == 0:
        e = np.broadcast_to(e, W.shape[:2])
    y = np.einsum("shmd,shd->shm", W, x)
    W_next = W - e[:, :, None, None] * g[:, :, :, None] * x[:, :, None, :]
    return y, W_next
