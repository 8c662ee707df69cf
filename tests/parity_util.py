"""Shared helpers for the GPU parity tests (tolerances, transfers, printing).

Tolerances are normwise per output tensor (elementwise relative error is
ill-posed at zero crossings):
    max_rel  = ||o - r||_inf / ||r||_inf
    mean_rel = ||o - r||_1   / ||r||_1
fp32 inputs: max_rel <= 1e-5.  bf16 inputs: max_rel <= 2e-2 and
mean_rel <= 1e-3.  The oracle always sees the already-rounded bf16 inputs,
so input quantisation never counts as error.
"""

import sys

import numpy as np

TOL = {"f32": dict(max_rel=1e-5, mean_rel=1e-5), "bf16": dict(max_rel=2e-2, mean_rel=1e-3)}


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def errs(out, ref):
    out = np.asarray(out, np.float64)
    ref = np.asarray(ref, np.float64)
    assert out.shape == ref.shape, (out.shape, ref.shape)
    assert np.all(np.isfinite(out)), "non-finite output"
    d = np.abs(out - ref)
    den_inf = max(np.max(np.abs(ref)), 1e-30)
    den_1 = max(np.sum(np.abs(ref)), 1e-30)
    return float(np.max(d) / den_inf), float(np.sum(d) / den_1)


def check(name, out, ref, dtype):
    mx, mn = errs(out, ref)
    tol = TOL[dtype]
    log(f"    {name:7s} max_rel={mx:.3e} mean_rel={mn:.3e}")
    assert mx <= tol["max_rel"], f"{name}: max_rel {mx:.3e} > {tol['max_rel']}"
    assert mn <= tol["mean_rel"], f"{name}: mean_rel {mn:.3e} > {tol['mean_rel']}"


def to_dev(a, dtype, torch):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.contiguous()


def to_host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)
