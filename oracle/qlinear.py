"""fp64 reference of the SubSpec substitute-layer linear.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``): nothing in the product path
may import this module.

What is computed, and where it comes from
-----------------------------------------
* Sec. 4.1 ("Quantized Substitute Weights for Offloaded Layers"): an offloaded
  linear layer of the target model is replaced by a GPU-resident low-bit copy made
  by a fast, data-free, group-wise quantizer; the draft model then evaluates that
  copy as an ordinary linear layer.  Sec. 5.1 (evaluation parameters) fixes 4-bit
  codes with groups of 64.  The paper names HQQ but does not state its algorithm;
  the quantizer here is the plain per-group min/max asymmetric rule (scale and zero
  stored as fp16), the reading listed in the design doc.
* A substitute layer is therefore  y[m, n] = sum_k x[m, k] * W^[n, k]  with
  W^[n, k] = s[g, n] * (q[n, k] - z[g, n]),  g = floor(k / G).
* The packed layout read by :func:`unpack` is the one specified in
  ``include/subspec.h`` (this project's own layout; the paper gives none).

Parity status: every function here is pinned by the ``-m "not gpu"`` tests in
``tests/test_oracle.py`` (closed forms, invariants, brute force with exact rational
arithmetic, hand-derived golden bytes).  How faithful min/max quantization is to
HQQ is "parity unpinned": the paper prints no HQQ numerics.
"""
from __future__ import annotations

import numpy as np

# ----------------------------------------------------------------------------
# Floating-point formats (IEEE-754 binary16 via NumPy; bfloat16 written out).
# ----------------------------------------------------------------------------


def fp16_round(v) -> np.ndarray:
    """Round float64 values to IEEE binary16, nearest-even (NumPy's direct
    float64 -> float16 conversion, a single correctly rounded step)."""
    return np.asarray(v, dtype=np.float64).astype(np.float16)


def bf16_round_bits(f32) -> np.ndarray:
    """Round float32 values to bfloat16 (the top 16 bits of a float32) with
    round-to-nearest-even; returns the uint16 bit patterns.  Finite inputs only."""
    u = np.asarray(f32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact value of bfloat16 bit patterns (uint16) as float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


# ----------------------------------------------------------------------------
# Quantizer: per-group min/max, asymmetric, fp16 scale and zero (Sec. 4.1, 5.1).
# ----------------------------------------------------------------------------


def quantize_minmax(w, bits: int, group: int):
    """Quantize float32 weights ``w`` [N][K] group-wise along K.

    For every column n and group g (the ``group`` consecutive k of that column):
      s   = (wmax - wmin) / (2^bits - 1)            in float64
      s16 = fp16(s)                                  nearest-even
      z16 = fp16(-wmin / s16)                        from the *rounded* scale
      q   = clamp(rint(w / s16 + z16), 0, 2^bits-1)  float64, ties to even
    A degenerate group (wmax == wmin, or s16 == 0) gets s16 = 1, z16 = fp16(-wmin)
    and q = 0.

    Returns ``(q, s16, z16)``: q uint8 [N][K]; s16, z16 float16 [K/group][N].
    """
    w = np.asarray(w, dtype=np.float32)
    N, K = w.shape
    if K % group:
        raise ValueError("K must be a multiple of the group size")
    qmax = float(2 ** bits - 1)
    wg = w.astype(np.float64).reshape(N, K // group, group)
    wmin = wg.min(axis=2)
    wmax = wg.max(axis=2)
    s16 = fp16_round((wmax - wmin) / qmax)
    degenerate = (wmax == wmin) | (s16 == 0)
    s16 = np.where(degenerate, np.float16(1.0), s16)
    s64 = s16.astype(np.float64)
    z16 = np.where(degenerate, fp16_round(-wmin), fp16_round(-wmin / s64))
    z64 = z16.astype(np.float64)
    t = wg / s64[:, :, None] + z64[:, :, None]
    q = np.clip(np.rint(t), 0.0, qmax)
    q = np.where(degenerate[:, :, None], 0.0, q)
    return (q.reshape(N, K).astype(np.uint8),
            np.ascontiguousarray(s16.T),
            np.ascontiguousarray(z16.T))


# ----------------------------------------------------------------------------
# Dequantization (exact in float64) and the two canonical rounded forms.
# ----------------------------------------------------------------------------


def dequant(q, s16, z16, group: int) -> np.ndarray:
    """W^[n, k] = s16[g, n] * (q[n, k] - z16[g, n]) in float64, g = k // group.

    Exact: fp16 values carry bits from 2^15 down to 2^-24, so q - z16 needs at most
    41 significant bits and the product with an 11-bit scale at most 52, below
    float64's 53."""
    q = np.asarray(q)
    N, K = q.shape
    s = np.asarray(s16, dtype=np.float16).astype(np.float64).T  # [N][K/G]
    z = np.asarray(z16, dtype=np.float16).astype(np.float64).T
    s_full = np.repeat(s, group, axis=1)
    z_full = np.repeat(z, group, axis=1)
    return s_full * (q.astype(np.float64) - z_full)


def dequant_f32(q, s16, z16, group: int) -> np.ndarray:
    """Canonical float32 dequantized weight: the exact value rounded once."""
    return dequant(q, s16, z16, group).astype(np.float32)


def dequant_bf16_bits(q, s16, z16, group: int) -> np.ndarray:
    """Canonical bfloat16 dequantized weight: nearest-even bf16 of the canonical
    float32 value (a deliberate double rounding)."""
    return bf16_round_bits(dequant_f32(q, s16, z16, group))


# ----------------------------------------------------------------------------
# Packed layout reader, written from the specification in include/subspec.h.
# ----------------------------------------------------------------------------


def _pair_fields(words: np.ndarray, bits: int, p: int):
    """(even code, odd code) of pair p in every slice; ``words`` is
    [..., bits] uint32 holding the slice's little-endian 32-bit words."""
    if bits == 4:
        w, off, mask = p // 4, 4 * (p % 4), 0xF
    elif bits == 2:
        w, off, mask = p // 8, 2 * (p % 8), 0x3
    elif bits == 3:
        if p == 15:
            even = np.zeros(words.shape[:-1], dtype=np.uint32)
            odd = np.zeros(words.shape[:-1], dtype=np.uint32)
            for c in range(3):
                even |= ((words[..., c] >> np.uint32(15)) & np.uint32(1)) << np.uint32(c)
                odd |= ((words[..., c] >> np.uint32(31)) & np.uint32(1)) << np.uint32(c)
            return even, odd
        w, off, mask = p // 5, 3 * (p % 5), 0x7
    else:
        raise ValueError("bits must be 2, 3 or 4")
    word = words[..., w]
    even = (word >> np.uint32(off)) & np.uint32(mask)
    odd = (word >> np.uint32(16 + off)) & np.uint32(mask)
    return even, odd


def unpack(packed, bits: int, N: int, K: int) -> np.ndarray:
    """Codes q [N][K] (uint8) from a packed buffer laid out as in subspec.h.

    Tile (nt, kb) covers columns 16*nt..16*nt+15 and k = 128*kb..128*kb+127 and
    starts at byte 256*bits*(nt*(K/128) + kb).  Slice L (0..63) of a tile is
    4*bits bytes long and belongs to column 16*nt + L%16; its pair p (0..15) holds
    the codes of k = 128*kb + 32*(p//4) + 8*(L//16) + 2*(p%4) (+1 for the odd one).
    """
    if N % 16 or K % 128:
        raise ValueError("N must be a multiple of 16 and K of 128")
    buf = np.frombuffer(np.asarray(packed, dtype=np.uint8).tobytes(), dtype="<u4")
    NT, KB = N // 16, K // 128
    if buf.size != NT * KB * 64 * bits:
        raise ValueError("packed buffer has the wrong size")
    words = buf.reshape(NT, KB, 64, bits)
    L = np.arange(64)
    nt = np.arange(NT)[:, None, None]
    kb = np.arange(KB)[None, :, None]
    n_idx = 16 * nt + (L % 16)[None, None, :]
    codes = np.full((N, K), 255, dtype=np.uint8)
    for p in range(16):
        even, odd = _pair_fields(words, bits, p)
        k_even = 128 * kb + 32 * (p // 4) + 8 * (L // 16)[None, None, :] + 2 * (p % 4)
        n_b, k_b = np.broadcast_arrays(n_idx, k_even)
        codes[n_b, k_b] = even
        codes[n_b, k_b + 1] = odd
    return codes


# ----------------------------------------------------------------------------
# The substitute layer itself.
# ----------------------------------------------------------------------------


def _weights(q, s16, z16, group, wprec):
    w = dequant(q, s16, z16, group)
    if wprec == "exact":
        return w
    if wprec == "fp32":
        return w.astype(np.float32).astype(np.float64)
    if wprec == "bf16":
        return bf16_bits_to_f64(bf16_round_bits(w.astype(np.float32)))
    raise ValueError("wprec must be 'exact', 'fp32' or 'bf16'")


def qlinear_ref(x_bf16_bits, q, s16, z16, group: int, wprec: str = "exact") -> np.ndarray:
    """y [M][N] in float64: y = x @ W^^T with x the exact values of the bf16
    activations [M][K] and W^ the dequantized weights (``wprec`` selects the exact
    value or its canonical float32 / bfloat16 rounding)."""
    x = bf16_bits_to_f64(x_bf16_bits)
    w = _weights(q, s16, z16, group, wprec)
    return x @ w.T


def qlinear_ref_cols(x_bf16_bits, q_cols, s_cols, z_cols, group: int,
                     wprec: str = "exact") -> np.ndarray:
    """Same as :func:`qlinear_ref` for a subset of output columns: q_cols is
    [n_s][K] and s_cols, z_cols are [K/group][n_s]; returns y [M][n_s]."""
    return qlinear_ref(x_bf16_bits, q_cols, s_cols, z_cols, group, wprec)
