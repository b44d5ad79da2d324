"""fp64 reference of SubSpec's draft-tree expansion step with probability sharpening.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``): nothing in the product path
may import this module.

What is computed, and where it comes from
-----------------------------------------
* Sec. 4.2 ("Constructing Deep Context-Aware Dynamic Draft Tree"): in each draft
  pass every leaf of the tree is fed to the draft model, which gives a distribution
  over the next token for each leaf.  A candidate (leaf i, token v) scores the
  product of its conditional probability and the path score of its parent leaf,
  and the k best candidates over all leaves become the next leaves.
* Sec. 4.2 ("Draft Probability Sharpening") and App. D: under greedy decoding the
  draft distribution is taken at a low temperature (0.2) before the products are
  formed: p_i(v) = softmax(l_i / T)(v).
* Readings (listed in the design doc): path scores are carried as natural logarithms
  (the product over a path of depth 48 underflows otherwise; the logarithm is
  monotonic, so the ranking is the same), i.e.  score(i, v) = s_i + log p_i(v);
  ties are broken by the smaller flat index i * V + v; the k winners are returned
  best first.

The functions are NumPy in float64 and follow the definition step by step: divide
the logits by T, take a numerically stable log-softmax per row (subtract the row
maximum, log of the summed exponentials), add the parent score, and sort.
"""
from __future__ import annotations

import numpy as np

from .qlinear import bf16_bits_to_f64


def log_softmax_rows(z) -> np.ndarray:
    """log softmax of every row of z (float64): z - (max + log sum exp(z - max))."""
    z = np.asarray(z, dtype=np.float64)
    m = z.max(axis=1, keepdims=True)
    return z - (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))


def expand_scores(logits_bf16_bits, parent_logp, temperature: float) -> np.ndarray:
    """score[i, v] = parent_logp[i] + log softmax(l_i / T)[v] for bf16 logits [R][V]."""
    z = bf16_bits_to_f64(logits_bf16_bits) / float(temperature)
    return np.asarray(parent_logp, dtype=np.float64)[:, None] + log_softmax_rows(z)


def tree_expand(logits_bf16_bits, parent_logp, temperature: float, k: int):
    """The k best candidates (score descending, ties by smaller flat index).

    Returns (parent_index[k], token[k], score[k]) as int64, int64, float64."""
    s = expand_scores(logits_bf16_bits, parent_logp, temperature)
    V = s.shape[1]
    flat = s.ravel()
    order = np.argsort(-flat, kind="stable")  # stable: equal scores keep index order
    sel = order[:k]
    return sel // V, sel % V, flat[sel]


def kth_gap(logits_bf16_bits, parent_logp, temperature: float, k: int) -> float:
    """Score difference between the k-th and (k+1)-th best candidates (inf if there
    are only k): how far the selection is from a tie."""
    s = np.sort(expand_scores(logits_bf16_bits, parent_logp, temperature).ravel())[::-1]
    return float(s[k - 1] - s[k]) if s.size > k else float("inf")
