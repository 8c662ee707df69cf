"""Seeded synthetic inputs for the scan and decode workloads.

This module only draws and quantises inputs; it contains none of the
method's arithmetic.  Both the HIP path (tests, benchmark) and the float64
oracle consume what it produces, so the oracle always sees exactly the values
the GPU sees (bf16 inputs are rounded here, once, with round-to-nearest-even,
and handed to the oracle already rounded).

The five workload shapes mirror the paper's setting of adapted linear maps in
an LM layer (Section 3; Appendix E gives the paper's own widths):

  small-f32   fp32, B=1, H=1, T=256, d=m=64, eta=0.01, chunk 64, seed 0
  lm-bf16     bf16, B=8, H=16, T=2048, d=m=64, eta=0.1, chunk 64, seed 1,
              x L2-normalised per head, g ~ N(0, 0.1^2)
  long-bf16   bf16, B=2, H=16, T=16384, d=m=128, eta=0.05, chunk 128, seed 2,
              x ~ N(0, 1/128), g ~ N(0, 0.05^2)
  stack-bf16  24 independent layers, each bf16 B=4, H=32, T=4096, d=m=64,
              eta=0.1, chunk 64, inputs drawn as lm-bf16, seed 3000 + layer
  decode-f32  256 sequences x 16 heads of 64x64 fp32 state, 512 steps,
              y = W x then W <- W - eta g x^T, x ~ N(0, 1/64),
              g ~ N(0, 0.1^2), eta = 0.1, seed 4

Draw order for a scan workload is W0, X, G, dY with numpy's PCG64 in float64.
W0 ~ N(0, 1/d); dY ~ N(0, 1).
"""

from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass(frozen=True)
class ScanWorkload:
    name: str
    B: int
    H: int
    T: int
    d: int
    m: int
    chunk: int
    dtype: str  # "f32" or "bf16"
    eta: float
    x_dist: str  # "normal" (std x_std) or "l2" (unit-norm rows)
    x_std: float
    g_std: float
    seed: int
    layers: int = 1

    def layer_seed(self, layer: int) -> int:
        return self.seed + layer

    @property
    def tokens(self) -> int:
        """Tokens per pass through one layer (B * T; every token spans H heads)."""
        return self.B * self.T


@dataclasses.dataclass(frozen=True)
class DecodeWorkload:
    name: str
    S: int
    H: int
    d: int
    m: int
    steps: int
    eta: float
    x_std: float
    g_std: float
    w_std: float
    seed: int


SCAN_WORKLOADS = {
    "small-f32": ScanWorkload("small-f32", 1, 1, 256, 64, 64, 64, "f32", 0.01,
                              "normal", 64 ** -0.5, 1.0, 0),
    "lm-bf16": ScanWorkload("lm-bf16", 8, 16, 2048, 64, 64, 64, "bf16", 0.1,
                            "l2", 0.0, 0.1, 1),
    "long-bf16": ScanWorkload("long-bf16", 2, 16, 16384, 128, 128, 128, "bf16",
                              0.05, "normal", 128 ** -0.5, 0.05, 2),
    "stack-bf16": ScanWorkload("stack-bf16", 4, 32, 4096, 64, 64, 64, "bf16", 0.1,
                               "l2", 0.0, 0.1, 3000, layers=24),
}

DECODE_WORKLOADS = {
    "decode-f32": DecodeWorkload("decode-f32", 256, 16, 64, 64, 512, 0.1,
                                 64 ** -0.5, 0.1, 64 ** -0.5, 4),
}


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even); returns float32 values."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # Adding 0x7FFF plus the lowest kept bit and truncating is round-to-nearest-
    # even on the upper 16 bits.  Finite inputs never wrap in uint32.
    r = ((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF)
    r += u
    r &= np.uint32(0xFFFF0000)
    out = r.view(np.float32)
    bad = ~np.isfinite(a)
    if bad.any():
        out = np.where(bad, a, out)
    return out


def quantise(a: np.ndarray, dtype: str) -> np.ndarray:
    """Values exactly representable in the storage dtype, held as float32."""
    if dtype == "bf16":
        return round_bf16(a)
    if dtype == "f32":
        return np.ascontiguousarray(a, dtype=np.float32)
    raise ValueError(dtype)


def _draw_x(rng, shape, wl: ScanWorkload):
    x = rng.standard_normal(shape)
    if wl.x_dist == "l2":
        x /= np.linalg.norm(x, axis=-1, keepdims=True)
    else:
        x *= wl.x_std
    return x


def scan_inputs(wl: ScanWorkload, layer: int = 0, *, B=None, T=None, seed=None):
    """Inputs for one layer of a scan workload as float32 numpy arrays.

    Values are already quantised to the workload dtype.  ``B``/``T``/``seed``
    override the workload for smaller parity cases of the same distribution.
    Returns dict(W0 [H,m,d], X [B,H,T,d], G [B,H,T,m], dY [B,H,T,m], eta float).
    """
    B = wl.B if B is None else B
    T = wl.T if T is None else T
    s = wl.layer_seed(layer) if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(s))
    W0 = rng.standard_normal((wl.H, wl.m, wl.d)) * wl.d ** -0.5
    X = _draw_x(rng, (B, wl.H, T, wl.d), wl)
    G = rng.standard_normal((B, wl.H, T, wl.m)) * wl.g_std
    dY = rng.standard_normal((B, wl.H, T, wl.m))
    return {
        # Slow weights and fast states are fp32 in every configuration.
        "W0": np.ascontiguousarray(W0, dtype=np.float32),
        "X": quantise(X, wl.dtype),
        "G": quantise(G, wl.dtype),
        "dY": quantise(dY, wl.dtype),
        "eta": float(np.float32(wl.eta)),
    }


def eta_tokens(B, H, T, seed, lo=0.0, hi=0.2):
    """Per-token step sizes in [lo, hi) (fp32), for the per-token eta path."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.uniform(lo, hi, size=(B, H, T)).astype(np.float32)


def gate_tokens(B, H, T, d, seed, a_mean=1.5, a_std=0.5, mu_max=4.0, b_std=0.5):
    """Per-token retention and step size from the paper's gate family.

    alpha = sigmoid(a) and eta = (mu_max / d) sigmoid(b) (Section 3, "Practical
    architecture and training"), with the logits drawn around the values the
    paper starts from: a ~ N(1.5, 0.5^2) (the toy of Appendix D uses a bias of
    1.5) and b ~ N(log(0.9 / 3.1), 0.5^2) (write strength starting at 0.9 with
    mu_max = 4, Appendix E).  Returns (alpha, eta) as fp32 [B, H, T].
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    a = rng.normal(a_mean, a_std, size=(B, H, T))
    b = rng.normal(np.log(0.9 / 3.1), b_std, size=(B, H, T))
    alpha = 1.0 / (1.0 + np.exp(-a))
    eta = mu_max / d / (1.0 + np.exp(-b))
    return alpha.astype(np.float32), eta.astype(np.float32)


def reset_flags(B, T, seed, mean_len=300):
    """Document starts for packed rows: uint8 [B, T], 1 where a document begins.

    Document lengths are geometric with the given mean (a packed stream of
    variable-length documents); token 0 always starts one.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    r = np.zeros((B, T), np.uint8)
    for b in range(B):
        t = 0
        while t < T:
            r[b, t] = 1
            t += int(rng.geometric(1.0 / mean_len))
    return r


def decode_initial_state(wl: DecodeWorkload, S=None):
    S = wl.S if S is None else S
    rng = np.random.Generator(np.random.PCG64(wl.seed))
    W = rng.standard_normal((S, wl.H, wl.m, wl.d)) * wl.w_std
    return np.ascontiguousarray(W, dtype=np.float32)


def decode_step_inputs(wl: DecodeWorkload, step: int, S=None):
    """x [S,H,d], g [S,H,m] for one decode step (seeded per step)."""
    S = wl.S if S is None else S
    rng = np.random.Generator(np.random.PCG64([wl.seed, step + 1]))
    x = rng.standard_normal((S, wl.H, wl.d)) * wl.x_std
    g = rng.standard_normal((S, wl.H, wl.m)) * wl.g_std
    return (np.ascontiguousarray(x, dtype=np.float32),
            np.ascontiguousarray(g, dtype=np.float32))


def device_scan_inputs(wl: ScanWorkload, layer: int, device, *, torch):
    """Seeded inputs drawn directly on a device, for timing-only runs.

    Same distributions as :func:`scan_inputs` but drawn with torch's device
    generator (not bit-identical to the numpy draw), so that multi-gigabyte
    workloads do not have to be generated on the host.  Parity checks use
    :func:`scan_inputs`.
    """
    gen = torch.Generator(device=device)
    gen.manual_seed(wl.layer_seed(layer))
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    W0 = torch.randn(wl.H, wl.m, wl.d, device=device, generator=gen) * wl.d ** -0.5
    X = torch.randn(wl.B, wl.H, wl.T, wl.d, device=device, generator=gen)
    if wl.x_dist == "l2":
        X = X / X.norm(dim=-1, keepdim=True)
    else:
        X = X * wl.x_std
    G = torch.randn(wl.B, wl.H, wl.T, wl.m, device=device, generator=gen) * wl.g_std
    dY = torch.randn(wl.B, wl.H, wl.T, wl.m, device=device, generator=gen)
    return {"W0": W0.float().contiguous(), "X": X.to(dt).contiguous(),
            "G": G.to(dt).contiguous(), "dY": dY.to(dt).contiguous(),
            "eta": float(np.float32(wl.eta))}
