"""fp64 reference of the substitute quantizer with an HQQ-style optimised zero-point.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``): nothing in the product path
may import this module.

What is computed, and where it comes from
-----------------------------------------
* SubSpec Sec. 4.1 and Sec. 5.1: the substitute layers are quantized data-free with
  HQQ, 4 bits, groups of 64.  The paper gives no algorithm; it follows the cited
  work (Half-Quadratic Quantization, Badri and Shaji, 2023).  That work keeps the
  group's scale and optimises its zero point z to minimise an l_p norm (p < 1) of
  the weight error w - s (Q(w) - z), with a half-quadratic splitting solved by
  alternating two closed-form steps:
    1. the error variable e: a generalised soft threshold of the current residual,
       shrink(x) = sign(x) max(|x| - |x|^(p-1) / beta, 0);
    2. the zero: the least-squares fit z = mean(q - (w - e) / s) over the group,
  with beta growing by a factor kappa after each round.  Published defaults:
  p = 0.7, beta = 10, kappa = 1.01, 20 rounds.
* Readings (listed in the design doc): the scale is the min/max scale of the baseline
  quantizer (fp16); the iteration starts from the min/max zero; after each round
  the group's sum of |w - s (q - z)| is evaluated for the new zero, the best zero is
  kept and the iteration stops at the first round that does not improve it; the best
  zero is rounded to fp16 and kept only if, in fp16, it still beats the min/max zero;
  codes are then q = clamp(rint(w / s + z), 0, 2^b - 1) as in the min/max quantizer.
  Every step is float64; sums run in index order (the arithmetic is fixed so that a
  GPU implementation takes the same rounding decisions).

``quantize_hqq`` returns ``(q, s16, z16)`` like ``quantize_minmax``.
"""
from __future__ import annotations

import numpy as np

from .qlinear import fp16_round, quantize_minmax

HQQ_P = 0.7
HQQ_BETA = 10.0
HQQ_KAPPA = 1.01
HQQ_ITERS = 20


def shrink_lp(x, beta: float, p: float = HQQ_P) -> np.ndarray:
    """Generalised soft threshold for the l_p norm: sign(x) max(|x| - |x|^(p-1) / beta, 0)
    (zero stays zero)."""
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    with np.errstate(divide="ignore"):
        t = np.power(a, p - 1.0)  # +inf at 0
    return np.sign(x) * np.maximum(a - t / beta, 0.0)


def seq_sum(a) -> np.ndarray:
    """Sum over the last axis in index order (float64)."""
    return np.cumsum(np.asarray(a, dtype=np.float64), axis=-1)[..., -1]


def codes_for(w, s, z, qmax: float) -> np.ndarray:
    """clamp(rint(w / s + z), 0, qmax), float64; s, z broadcast over the last axis."""
    return np.clip(np.rint(w / s[..., None] + z[..., None]), 0.0, qmax)


def group_l1(w, s, z, qmax: float) -> np.ndarray:
    """sum_i |w_i - s (q_i - z)| per group, in index order."""
    q = codes_for(w, s, z, qmax)
    return seq_sum(np.abs(w - (q - z[..., None]) * s[..., None]))


def zero_step(w, q, e, s) -> np.ndarray:
    """The zero that minimises sum_i (q_i - z - (w_i - e_i) / s)^2: their mean."""
    return seq_sum(q - (w - e) / s[..., None]) / w.shape[-1]


def optimise_zero(w, s, z0, qmax: float, p: float = HQQ_P, beta: float = HQQ_BETA,
                  kappa: float = HQQ_KAPPA, iters: int = HQQ_ITERS):
    """Best zero (float64) per group of w [..., G] from the HQQ rounds, with its l1
    error; starts from z0 (its error is the one to beat)."""
    w = np.asarray(w, dtype=np.float64)
    z = np.array(z0, dtype=np.float64, copy=True)
    best_z = z.copy()
    best_err = group_l1(w, s, z, qmax)
    active = np.ones(z.shape, dtype=bool)
    b = beta
    for _ in range(iters):
        q = codes_for(w, s, z, qmax)
        r = (q - z[..., None]) * s[..., None]
        e = shrink_lp(w - r, b, p)
        z_new = zero_step(w, q, e, s)
        err = group_l1(w, s, z_new, qmax)
        better = active & (err < best_err)
        best_z = np.where(better, z_new, best_z)
        best_err = np.where(better, err, best_err)
        active = better  # a group stops at its first round without improvement
        z = np.where(active, z_new, z)
        if not active.any():
            break
        b = b * kappa
    return best_z, best_err


def quantize_hqq(w, bits: int, group: int):
    """Group-wise quantization of float32 w [N][K] along K with the min/max scale and
    an HQQ-optimised zero.  Returns (q uint8 [N][K], s16, z16 float16 [K/group][N])."""
    w32 = np.asarray(w, dtype=np.float32)
    N, K = w32.shape
    qmax = float(2 ** bits - 1)
    _, s16, z16_0 = quantize_minmax(w32, bits, group)
    wg = w32.astype(np.float64).reshape(N, K // group, group)
    s = s16.T.astype(np.float64)            # [N][K/group]
    z0 = z16_0.T.astype(np.float64)
    wmin, wmax = wg.min(axis=2), wg.max(axis=2)
    degenerate = (wmax == wmin) | (fp16_round((wmax - wmin) / qmax) == 0)
    best_z, _ = optimise_zero(wg, s, z0, qmax)
    z16 = fp16_round(best_z)
    keep = group_l1(wg, s, z16.astype(np.float64), qmax) < group_l1(wg, s, z0, qmax)
    z16 = np.where(keep & ~degenerate, z16, z16_0.T)
    q = codes_for(wg, s, z16.astype(np.float64), qmax)
    q = np.where(degenerate[:, :, None], 0.0, q)
    return (q.reshape(N, K).astype(np.uint8), np.ascontiguousarray(s16),
            np.ascontiguousarray(z16.T.astype(np.float16)))
