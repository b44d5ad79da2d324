"""Pins of the draft-tree expansion oracle (oracle/tree.py) against what the paper and
the mathematics fix: a library log-softmax, closed forms of the sharpened two-token
case, uniform logits, pure-Python brute force on tiny inputs, and invariants (each
chosen so that a dropped parent term, a multiplied instead of divided temperature,
a missing normalisation or a wrong tie rule fails one of them)."""
import math

import numpy as np
import pytest
from scipy.special import log_softmax as scipy_log_softmax

import oracle


def _bf16(a):
    return oracle.bf16_round_bits(np.asarray(a, dtype=np.float32))


def test_log_softmax_matches_library_routine():
    rng = np.random.default_rng(0)
    z = rng.normal(0, 3, (5, 37))
    assert np.allclose(oracle.log_softmax_rows(z), scipy_log_softmax(z, axis=1), atol=1e-13, rtol=0)


def test_sharpened_two_token_closed_form():
    # logits (a, a - 1) at T = 0.2: p0 = 1 / (1 + e^-5), p1 = e^-5 / (1 + e^-5)
    bits = _bf16([[3.0, 2.0]])
    s = oracle.expand_scores(bits, np.array([0.0]), 0.2)
    assert math.isclose(s[0, 0], -math.log1p(math.exp(-5.0)), rel_tol=0, abs_tol=1e-14)
    assert math.isclose(s[0, 1], -5.0 - math.log1p(math.exp(-5.0)), rel_tol=0, abs_tol=1e-14)
    # T = 1 is the plain softmax: p0 = 1 / (1 + e^-1)
    s1 = oracle.expand_scores(bits, np.array([0.0]), 1.0)
    assert math.isclose(s1[0, 0], -math.log1p(math.exp(-1.0)), abs_tol=1e-14)
    # sharpening raises the best token's probability
    assert s[0, 0] > s1[0, 0]


def test_uniform_logits_and_parent_scores():
    R, V, k = 3, 50, 7
    bits = _bf16(np.full((R, V), 1.5))
    parent = np.array([-2.0, -0.5, -1.0])
    s = oracle.expand_scores(bits, parent, 0.2)
    assert np.allclose(s, parent[:, None] - math.log(V), atol=1e-13)
    # every candidate of the best parent ties; ties go to the smaller flat index
    pi, tok, sc = oracle.tree_expand(bits, parent, 0.2, k)
    assert list(pi) == [1] * k and list(tok) == list(range(k))
    assert np.allclose(sc, -0.5 - math.log(V), atol=1e-13)


def test_parent_term_decides_between_identical_rows():
    rng = np.random.default_rng(1)
    row = rng.normal(0, 2, 40)
    bits = _bf16(np.stack([row, row]))
    # a parent 50 nats behind loses every one of the five places
    pi, tok, sc = oracle.tree_expand(bits, np.array([-50.0, 0.0]), 0.2, 5)
    assert set(pi) == {1}
    pi2, tok2, sc2 = oracle.tree_expand(bits, np.array([0.0, -50.0]), 0.2, 5)
    assert set(pi2) == {0} and list(tok2) == list(tok) and np.allclose(sc2, sc)
    # with equal parents the two rows interleave: each candidate appears twice
    pi3, tok3, _ = oracle.tree_expand(bits, np.array([0.0, 0.0]), 0.2, 4)
    assert list(pi3) == [0, 1, 0, 1] and tok3[0] == tok3[1] and tok3[2] == tok3[3]


def _brute(bits, parent, T, k):
    vals = oracle.bf16_bits_to_f64(bits)
    R, V = vals.shape
    cands = []
    for i in range(R):
        z = [vals[i, v] / T for v in range(V)]
        m = max(z)
        lse = m + math.log(sum(math.exp(t - m) for t in z))
        for v in range(V):
            cands.append((-(parent[i] + z[v] - lse), i * V + v))
    cands.sort()
    return [(f // V, f % V, -neg) for neg, f in cands[:k]]


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_tiny(seed):
    rng = np.random.default_rng(100 + seed)
    R, V = rng.integers(1, 5), rng.integers(2, 9)
    k = int(rng.integers(1, R * V + 1))
    bits = _bf16(rng.normal(0, 2, (R, V)))
    if seed == 0:  # exact ties inside a row and across rows
        bits[:, :] = bits[0, 0]
    parent = rng.normal(-1, 1, R)
    if seed == 0:
        parent[:] = -0.25
    T = [0.2, 1.0, 0.5][seed % 3]
    pi, tok, sc = oracle.tree_expand(bits, parent, T, k)
    want = _brute(bits, parent, T, k)
    assert [(int(a), int(b)) for a, b in zip(pi, tok)] == [(a, b) for a, b, _ in want]
    assert np.allclose(sc, [c for _, _, c in want], atol=1e-12, rtol=0)


def test_invariants():
    rng = np.random.default_rng(7)
    R, V, k = 6, 1000, 6
    bits = _bf16(rng.normal(0, 3, (R, V)))
    parent = np.sort(rng.normal(-3, 1, R))
    s = oracle.expand_scores(bits, parent, 0.2)
    # each row's conditional distribution sums to one
    assert np.allclose(np.exp(s - parent[:, None]).sum(axis=1), 1.0, atol=1e-12)
    assert (s <= parent[:, None] + 1e-15).all()
    pi, tok, sc = oracle.tree_expand(bits, parent, 0.2, k)
    assert (np.diff(sc) <= 0).all()
    assert len(set(zip(pi.tolist(), tok.tolist()))) == k
    # nothing outside the selection beats its last member
    mask = np.ones_like(s, dtype=bool)
    mask[pi, tok] = False
    assert s[mask].max() <= sc[-1]
    assert oracle.kth_gap(bits, parent, 0.2, k) >= 0


def _brute_gap(bits, parent, T, k):
    # pure-Python scores and a plain sort, independent of numpy's sorting
    vals = oracle.bf16_bits_to_f64(bits)
    R, V = vals.shape
    scores = []
    for i in range(R):
        z = [float(vals[i, v]) / T for v in range(V)]
        m = max(z)
        lse = m + math.log(sum(math.exp(t - m) for t in z))
        scores += [float(parent[i]) + t - lse for t in z]
    scores.sort(reverse=True)
    return scores[k - 1] - scores[k] if len(scores) > k else math.inf


@pytest.mark.parametrize("seed", range(5))
def test_kth_gap_brute_force_tiny(seed):
    rng = np.random.default_rng(400 + seed)
    R, V = int(rng.integers(1, 4)), int(rng.integers(2, 7))
    k = int(rng.integers(1, R * V))
    bits = _bf16(rng.normal(0, 2, (R, V)))
    parent = rng.normal(-1, 1, R)
    T = [0.2, 1.0, 0.5][seed % 3]
    got = oracle.kth_gap(bits, parent, T, k)
    want = _brute_gap(bits, parent, T, k)
    assert got > 0 and math.isclose(got, want, rel_tol=1e-9, abs_tol=1e-12)


def test_kth_gap_tie_and_full_selection():
    # two equal rows under equal parents: every candidate appears twice, so the
    # gap after an odd k is an exact tie (0) and after an even k it is positive
    rng = np.random.default_rng(9)
    row = rng.normal(0, 2, 6)
    bits = _bf16(np.stack([row, row]))
    parent = np.array([-0.5, -0.5])
    assert oracle.kth_gap(bits, parent, 0.2, 1) == 0.0
    assert oracle.kth_gap(bits, parent, 0.2, 3) == 0.0
    g2 = oracle.kth_gap(bits, parent, 0.2, 2)
    assert g2 > 0 and math.isclose(g2, _brute_gap(bits, parent, 0.2, 2), rel_tol=1e-9)
    # uniform logits: all scores of a row tie; the gap between rows is the parent gap
    ub = _bf16(np.full((2, 5), 0.75))
    assert oracle.kth_gap(ub, np.array([-1.0, -3.0]), 0.2, 2) == 0.0
    assert math.isclose(oracle.kth_gap(ub, np.array([-1.0, -3.0]), 0.2, 5), 2.0, abs_tol=1e-13)
    # k = R * V: nothing is left out of the selection
    assert oracle.kth_gap(bits, parent, 0.2, 12) == math.inf
    assert oracle.kth_gap(ub, np.array([-1.0, -3.0]), 0.2, 10) == math.inf
