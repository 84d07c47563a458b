"""FP8 (OCP E4M3) quantisation for the low-precision MLP mode of the oracle.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py). Plain numpy.

The paper's Ascend system streams W8A8 weights and activations (Sec. 3.4,
system-level optimisations; the quantised rows of Table 6). The quantisation
scheme is not given; the reading used here (both sides):
  * format: E4M3 with no infinities (largest finite 448, smallest normal
    2^-6, subnormal spacing 2^-9), round to nearest, ties to even, values
    beyond +-448 saturate;
  * weights: one scale per output channel; activations: one scale per row
    (token), computed where the row is produced. For a vector v with
    a = max|v| (float32): inv = 448 / a and s = a / 448 (both float32,
    correctly rounded), q_i = E4M3(float32(v_i * inv)); a = 0 gives inv = s = 0
    and q = 0;
  * y[m, n] = s_act[m] * s_w[n] * sum_k q_act[m, k] q_w[n, k] (the products of
    E4M3 values are exact; the oracle sums in float64).
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0


def e4m3_round(x) -> np.ndarray:
    """Nearest E4M3 value (ties to even), saturating at +-448; float64 out.

    Normal range (|x| >= 2^-6): the value spacing is 2^(e-3) for the binade
    [2^e, 2^(e+1)); below it the spacing is the subnormal 2^-9."""
    x = np.asarray(x, dtype=np.float64)
    ax = np.abs(x)
    _, ex = np.frexp(ax)                       # ax = m 2^ex, m in [0.5, 1)
    e = np.where(ax >= 2.0 ** -6, ex - 1, -6)  # binade exponent (subnormals: -6)
    quantum = np.ldexp(1.0, e - 3)
    q = np.rint(ax / quantum) * quantum        # np.rint: half to even
    q = np.minimum(q, E4M3_MAX)
    return np.copysign(q, x)


def quantize_rows(v):
    """Per-row scaling and E4M3 rounding of v [..., K] (the rule in the module
    docstring). Returns (q [..., K] float64, s [...] float64)."""
    v32 = np.asarray(v, dtype=np.float32)
    a = np.max(np.abs(v32), axis=-1)
    nz = a > 0
    with np.errstate(divide="ignore"):
        inv = np.where(nz, np.float32(E4M3_MAX) / np.where(nz, a, np.float32(1)), np.float32(0))
    s = np.where(nz, a / np.float32(E4M3_MAX), np.float32(0))
    inv = inv.astype(np.float32)
    q = e4m3_round((v32 * inv[..., None]).astype(np.float32))
    return q, s.astype(np.float64)


def fp8_matmul(x, qw, sw):
    """y = x W^T with x quantised per row and W given as (qw [N, K], sw [N])."""
    qx, sx = quantize_rows(x)
    return (qx @ qw.T) * sx[..., None] * sw
