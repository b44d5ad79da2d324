"""GPU parity of the tree attention over the shared KV cache against the fp64 oracle,
through the C ABI.

Tolerance, from the arithmetic: the kernel carries every probability p_j as two
bf16 terms (hi = bf16(p), lo = bf16(p - hi), within 2^-16 p_j of p_j) and uses the
same terms for the weighted sum and its normaliser, so the output is an exact
weighted average under weights within 2^-15 (relative) of the true ones:
|o - o_ref| <= 2^-15 sum_j p_j |v_j - o| <= 2^-14 sum_j p_j |v_j|.  Rounding the
output to bf16 (8 significant bits) adds at most 2^-8 |o_ref|; the scores (fp32 sums
of exact bf16 products), the exponentials and the fp32 sums contribute ~1e-6
relative.  The test allows 2^-8 |o_ref| + 2^-14 sum_j p_j |v_j| + 1e-6.  The cache
after the call must equal the oracle's bit for bit (the new rows appended, nothing
else changed)."""
import math

import numpy as np
import pytest

import oracle
import paper_2509_18344_amd as ss
from paper_2509_18344_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"
D = 128


def _tol(ref, wabs):
    return 2.0 ** -8 * np.abs(ref) + 2.0 ** -14 * wabs + 1e-6


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV)


def _run(x, mask, M, Hq, Hkv, S, P, T, scale):
    q, kc, vc, kn, vn = (_dev(x[n]) for n in ("q", "k_cache", "v_cache", "k_new", "v_new"))
    mk = torch.from_numpy(mask.view(np.int32)).to(DEV)
    out = torch.empty((M, Hq, D), dtype=torch.int16, device=DEV)
    ss.subspec_tree_attention(q, kc, vc, kn, vn, mk, M, Hq, Hkv, S, P, T, scale, out)
    torch.cuda.synchronize()
    return (out.cpu().numpy().view(np.uint16), kc.cpu().numpy().view(np.uint16),
            vc.cpu().numpy().view(np.uint16))


def _check(M, Hq, Hkv, P, T, k, seed, q_scale=1.0, mask=None, S=None, what=""):
    S = S or P + T + M + 40
    x = synth.tree_attn_inputs(M, Hq, Hkv, D, S, seed, q_scale=q_scale)
    if mask is None:
        mask = synth.tree_levels_mask(T, k, M, seed)
    scale = 1.0 / math.sqrt(D)
    out, kc, vc = _run(x, mask, M, Hq, Hkv, S, P, T, scale)
    ref, kref, vref = oracle.tree_attention(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"],
                                            mask, scale)
    wabs = oracle.weighted_abs_v(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, scale)
    got = oracle.bf16_bits_to_f64(out)
    tol = _tol(ref, wabs)
    err = np.abs(got - ref)
    assert np.all(err <= tol), (what, float(err.max()), float((err / tol).max()))
    assert np.array_equal(kc, kref) and np.array_equal(vc, vref), what
    return x, mask, out


@pytest.mark.parametrize("M,Hq,Hkv,P,T,k,qs", [
    (6, 28, 4, 2048, 282, 6, 1.0),   # Qwen2.5-7B, last pass of a depth-48 tree
    (6, 28, 4, 2048, 282, 6, 4.0),   # peaked scores
    (6, 40, 8, 1000, 60, 6, 1.0),    # Qwen2.5-32B
    (1, 28, 4, 1, 0, 6, 1.0),        # the first pass after a one-token context
    (6, 28, 4, 100, 0, 6, 2.0),      # first pass of a tree: no earlier tree tokens
    (6, 28, 4, 0, 36, 6, 1.0),       # no committed context
    (8, 16, 2, 33, 7, 4, 1.0),       # 64 query rows per head (4 row tiles), ragged tails
    (3, 4, 4, 77, 13, 3, 1.5),       # no grouping, one row tile
    (5, 10, 2, 5000, 95, 5, 1.0),    # long context: several tiles per range
])
def test_tree_attention_matches_oracle(M, Hq, Hkv, P, T, k, qs):
    _check(M, Hq, Hkv, P, T, k, 7 * P + T + M, q_scale=qs, what=f"M={M} Hq={Hq} Hkv={Hkv} P={P} T={T}")


def test_tree_attention_query_without_visible_keys_gets_zeros():
    M, Hq, Hkv, P, T = 2, 4, 2, 0, 3
    mask = np.zeros((M, 1), np.uint32)
    mask[1, 0] = 1 << (T + 1)  # token 1 sees itself; token 0 sees nothing
    x, _, out = _check(M, Hq, Hkv, P, T, 3, 5, mask=mask, what="empty row")
    assert not out[0].any()


def test_tree_attention_deterministic():
    M, Hq, Hkv, P, T = 6, 28, 4, 700, 42
    S = P + T + M
    x = synth.tree_attn_inputs(M, Hq, Hkv, D, S, 77)
    mask = synth.tree_levels_mask(T, 6, M, 77)
    a = _run(x, mask, M, Hq, Hkv, S, P, T, 0.125)
    for _ in range(2):
        b = _run(x, mask, M, Hq, Hkv, S, P, T, 0.125)
        for u, w in zip(a, b):
            assert np.array_equal(u, w)


def test_tree_attention_chained_passes_read_what_was_appended():
    # three draft passes on one cache: each pass appends its six tokens and the next
    # pass reads them from the cache as tree tokens
    M, Hq, Hkv, P, k = 6, 28, 4, 300, 6
    S = P + 3 * M + 8
    x = synth.tree_attn_inputs(M, Hq, Hkv, D, S, 99)
    kc, vc = _dev(x["k_cache"]), _dev(x["v_cache"])
    kc_ref, vc_ref = x["k_cache"].copy(), x["v_cache"].copy()
    scale = 1.0 / math.sqrt(D)
    for depth in range(3):
        T = depth * M
        y = synth.tree_attn_inputs(M, Hq, Hkv, D, 1, 100 + depth)
        mask = synth.tree_levels_mask(T, k, M, 100 + depth)
        out = torch.empty((M, Hq, D), dtype=torch.int16, device=DEV)
        ss.subspec_tree_attention(_dev(y["q"]), kc, vc, _dev(y["k_new"]), _dev(y["v_new"]),
                                  torch.from_numpy(mask.view(np.int32)).to(DEV), M, Hq, Hkv, S, P, T, scale, out)
        torch.cuda.synchronize()
        ref, kc_ref, vc_ref = oracle.tree_attention(y["q"], kc_ref, vc_ref, P, T, y["k_new"], y["v_new"], mask,
                                                    scale)
        wabs = oracle.weighted_abs_v(y["q"], kc_ref, vc_ref, P, T, y["k_new"], y["v_new"], mask, scale)
        got = oracle.bf16_bits_to_f64(out.cpu().numpy().view(np.uint16))
        assert np.all(np.abs(got - ref) <= _tol(ref, wabs)), depth
        assert np.array_equal(kc.cpu().numpy().view(np.uint16), kc_ref), depth
        assert np.array_equal(vc.cpu().numpy().view(np.uint16), vc_ref), depth
