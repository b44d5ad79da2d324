"""fp64 reference of the draft model's tree attention over the shared KV cache.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``): nothing in the product path
may import this module.

What is computed, and where it comes from
-----------------------------------------
* Sec. 4.1 ("Shared KV-Cache", and the figure of the draft model and its cache
  pipeline): the draft model keeps no cache of its own.  It reads the target's
  cache for the committed context and appends keys and values for the tokens it
  speculates; the target later overwrites those slots when it verifies.
* Sec. 2 ("Speculative Decoding", tree decoding) and Sec. 4.2: the tree is kept
  flattened, and attention masks restrict every tree token to the committed context,
  its ancestors in the tree and itself.
* The attention itself is the standard scaled dot-product attention of the
  Qwen2.5 models the paper evaluates, with grouped key/value heads: query head h
  reads key/value head h // (Hq / Hkv).

Readings (listed in the design doc): the M tokens of one draft pass are appended at
cache positions P + T ... P + T + M - 1 (P committed tokens, T tree tokens of
earlier passes) before they attend; a query sees all P committed positions and the
tree positions P + j whose mask bit j is set; the scale is passed in (1/sqrt(D)).

The function follows the definition step by step in float64 on bf16 inputs: write
the new keys and values into copies of the caches, gather each query's visible
keys, take q.k * scale, a numerically stable softmax, and the weighted sum of the
values.
"""
from __future__ import annotations

import numpy as np

from .qlinear import bf16_bits_to_f64


def mask_bit(mask_bits, i: int, j: int) -> bool:
    """Bit j of row i of a uint32 bit-row mask."""
    return bool((int(mask_bits[i, j // 32]) >> (j % 32)) & 1)


def append_kv(k_cache_bits, v_cache_bits, k_new_bits, v_new_bits, pos: int):
    """Copies of the caches [Hkv][S][D] with the new rows [M][Hkv][D] written at
    positions pos ... pos + M - 1 (bit patterns, unchanged)."""
    kc = np.array(k_cache_bits, copy=True)
    vc = np.array(v_cache_bits, copy=True)
    M = k_new_bits.shape[0]
    for i in range(M):
        kc[:, pos + i, :] = k_new_bits[i]
        vc[:, pos + i, :] = v_new_bits[i]
    return kc, vc


def visible_positions(mask_bits, i: int, P: int, T: int, M: int) -> np.ndarray:
    """Cache positions query i may attend to: 0 ... P - 1, then P + j for every tree
    token j < T + M whose bit is set."""
    tree = [P + j for j in range(T + M) if mask_bit(mask_bits, i, j)]
    return np.array(list(range(P)) + tree, dtype=np.int64)


def tree_attention(q_bits, k_cache_bits, v_cache_bits, P: int, T: int, k_new_bits, v_new_bits,
                   mask_bits, scale: float):
    """Output [M][Hq][D] (float64) and the caches after the append (bit patterns).

    A query with no visible position gets zeros."""
    M, Hq, D = q_bits.shape
    Hkv = k_cache_bits.shape[0]
    G = Hq // Hkv
    kc, vc = append_kv(k_cache_bits, v_cache_bits, k_new_bits, v_new_bits, P + T)
    q = bf16_bits_to_f64(q_bits)
    K = bf16_bits_to_f64(kc)
    V = bf16_bits_to_f64(vc)
    out = np.zeros((M, Hq, D), dtype=np.float64)
    for i in range(M):
        pos = visible_positions(mask_bits, i, P, T, M)
        if pos.size == 0:
            continue
        for h in range(Hq):
            g = h // G
            s = (K[g, pos, :] @ q[i, h]) * scale
            p = np.exp(s - s.max())
            p /= p.sum()
            out[i, h] = p @ V[g, pos, :]
    return out, kc, vc


def weighted_abs_v(q_bits, k_cache_bits, v_cache_bits, P: int, T: int, k_new_bits, v_new_bits,
                   mask_bits, scale: float) -> np.ndarray:
    """sum_j p_j |v_j| per output element [M][Hq][D]: the scale of the error that
    rounding the probabilities p_j can cause (used to state tolerances)."""
    M, Hq, D = q_bits.shape
    Hkv = k_cache_bits.shape[0]
    G = Hq // Hkv
    kc, vc = append_kv(k_cache_bits, v_cache_bits, k_new_bits, v_new_bits, P + T)
    q = bf16_bits_to_f64(q_bits)
    K = bf16_bits_to_f64(kc)
    V = np.abs(bf16_bits_to_f64(vc))
    out = np.zeros((M, Hq, D), dtype=np.float64)
    for i in range(M):
        pos = visible_positions(mask_bits, i, P, T, M)
        if pos.size == 0:
            continue
        for h in range(Hq):
            g = h // G
            s = (K[g, pos, :] @ q[i, h]) * scale
            p = np.exp(s - s.max())
            p /= p.sum()
            out[i, h] = p @ V[g, pos, :]
    return out
