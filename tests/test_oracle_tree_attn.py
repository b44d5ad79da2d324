"""Pins of the tree-attention oracle (oracle/tree_attn.py) against what the
mathematics and a library fix: PyTorch's scaled_dot_product_attention in float64 on
the CPU with an explicit mask, closed forms (identical keys average the visible
values; one dominant key returns its value; a lone visible key returns its value),
invariances (a masked key's value does not matter, the order of the committed
positions does not matter), the grouping of query heads onto key/value heads, the
append, and pure-Python brute force on tiny inputs.  Each is chosen so that a
dropped scale, a wrong head grouping, a mask read with the wrong bit order or an
append at the wrong position fails one of them."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle.tree_attn import append_kv, mask_bit, tree_attention, visible_positions
from paper_2509_18344_amd import synth


def _bf(a):
    return oracle.bf16_round_bits(np.asarray(a, dtype=np.float32))


def _case(M, Hq, Hkv, D, P, T, k, seed, q_scale=1.0):
    S = P + T + M + 5
    x = synth.tree_attn_inputs(M, Hq, Hkv, D, S, seed, q_scale=q_scale)
    mask = synth.tree_levels_mask(T, k, M, seed)
    return x, mask


@pytest.mark.parametrize("M,Hq,Hkv,D,P,T,k,qs", [(6, 28, 4, 16, 40, 12, 6, 1.0), (1, 4, 4, 8, 9, 0, 6, 3.0),
                                                  (6, 10, 2, 32, 0, 18, 6, 2.0), (3, 6, 3, 16, 33, 7, 4, 1.0)])
def test_matches_library_sdpa(M, Hq, Hkv, D, P, T, k, qs):
    x, mask = _case(M, Hq, Hkv, D, P, T, k, 3 + P + T, q_scale=qs)
    scale = 1.0 / math.sqrt(D)
    out, kc, vc = tree_attention(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, scale)
    L = P + T + M
    # the library's view: full caches with the appended rows, heads expanded, a
    # boolean mask over positions 0 .. L-1 (bits decoded here independently)
    q = torch.from_numpy(oracle.bf16_bits_to_f64(x["q"])).permute(1, 0, 2)[None]  # [1][Hq][M][D]
    K = torch.from_numpy(oracle.bf16_bits_to_f64(kc[:, :L])).repeat_interleave(Hq // Hkv, 0)[None]
    V = torch.from_numpy(oracle.bf16_bits_to_f64(vc[:, :L])).repeat_interleave(Hq // Hkv, 0)[None]
    allow = np.zeros((M, L), dtype=bool)
    allow[:, :P] = True
    for i in range(M):
        for j in range(T + M):
            allow[i, P + j] = (int(mask[i, j >> 5]) >> (j & 31)) & 1 == 1
    ref = torch.nn.functional.scaled_dot_product_attention(q, K, V, attn_mask=torch.from_numpy(allow),
                                                           scale=scale)
    assert np.allclose(out, ref[0].permute(1, 0, 2).numpy(), atol=1e-12, rtol=0)


def test_append_writes_only_the_new_rows():
    x, mask = _case(6, 4, 2, 8, 20, 12, 6, 5)
    kc, vc = append_kv(x["k_cache"], x["v_cache"], x["k_new"], x["v_new"], 32)
    for i in range(6):
        assert np.array_equal(kc[:, 32 + i], x["k_new"][i]) and np.array_equal(vc[:, 32 + i], x["v_new"][i])
    keep = np.ones(kc.shape[1], bool)
    keep[32:38] = False
    assert np.array_equal(kc[:, keep], x["k_cache"][:, keep]) and np.array_equal(vc[:, keep], x["v_cache"][:, keep])


def test_identical_keys_average_the_visible_values():
    M, Hq, Hkv, D, P, T = 2, 2, 1, 8, 5, 6
    x, _ = _case(M, Hq, Hkv, D, P, T, 3, 9)
    x["k_cache"][:] = _bf(0.5)
    x["k_new"][:] = _bf(0.5)
    mask = np.zeros((M, 1), np.uint32)
    mask[0, 0] = (1 << 1) | (1 << 4) | (1 << (T + 0))
    mask[1, 0] = 1 << (T + 1)
    out, kc, vc = tree_attention(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, 0.3)
    V = oracle.bf16_bits_to_f64(vc)
    want0 = V[0, [0, 1, 2, 3, 4, P + 1, P + 4, P + T]].mean(axis=0)
    want1 = V[0, [0, 1, 2, 3, 4, P + T + 1]].mean(axis=0)
    assert np.allclose(out[0, 0], want0, atol=1e-13) and np.allclose(out[0, 1], want0, atol=1e-13)
    assert np.allclose(out[1, 0], want1, atol=1e-13)


def test_dominant_key_and_lone_key():
    M, Hq, Hkv, D, P, T = 1, 1, 1, 16, 30, 0
    x, _ = _case(M, Hq, Hkv, D, P, T, 6, 12)
    # the query equals key 17 scaled up: that key's score dominates by far
    x["q"][0, 0] = _bf(oracle.bf16_bits_to_f64(x["k_cache"][0, 17]) * 8.0)
    mask = np.array([[1]], np.uint32)
    out, kc, vc = tree_attention(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, 1.0)
    assert np.allclose(out[0, 0], oracle.bf16_bits_to_f64(vc[0, 17]), atol=1e-9)
    # no committed tokens and only its own bit: the token sees itself alone
    out2, _, _ = tree_attention(x["q"], x["k_cache"], x["v_cache"], 0, 0, x["k_new"], x["v_new"], mask, 1.0)
    assert np.array_equal(out2[0, 0], oracle.bf16_bits_to_f64(x["v_new"][0, 0]))
    # nothing visible: zeros
    out3, _, _ = tree_attention(x["q"], x["k_cache"], x["v_cache"], 0, 0, x["k_new"], x["v_new"],
                                np.zeros((1, 1), np.uint32), 1.0)
    assert not out3.any()


def test_masked_values_do_not_matter_and_prefix_order_does_not_matter():
    M, Hq, Hkv, D, P, T, k = 6, 6, 2, 16, 25, 18, 6
    x, mask = _case(M, Hq, Hkv, D, P, T, k, 21)
    scale = 0.25
    out, _, _ = tree_attention(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, scale)
    # tree token 2 is hidden from query 0 only if its bit is clear; change the values
    # of every tree token hidden from all queries
    hidden = [j for j in range(T) if not any(mask_bit(mask, i, j) for i in range(M))]
    assert hidden
    v2 = x["v_cache"].copy()
    for j in hidden:
        v2[:, P + j] = _bf(np.full(D, 100.0))
    out2, _, _ = tree_attention(x["q"], x["k_cache"], v2, P, T, x["k_new"], x["v_new"], mask, scale)
    assert np.array_equal(out, out2)
    perm = np.random.default_rng(0).permutation(P)
    k3, v3 = x["k_cache"].copy(), x["v_cache"].copy()
    k3[:, :P], v3[:, :P] = x["k_cache"][:, perm], x["v_cache"][:, perm]
    out3, _, _ = tree_attention(x["q"], k3, v3, P, T, x["k_new"], x["v_new"], mask, scale)
    assert np.allclose(out, out3, atol=1e-13)


def test_query_heads_share_their_group_key_value_head():
    M, Hq, Hkv, D, P, T = 2, 6, 3, 8, 10, 4
    x, mask = _case(M, Hq, Hkv, D, P, T, 4, 33)
    x["q"][:, :, :] = x["q"][:, :1, :]  # every head asks the same question
    out, _, _ = tree_attention(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, 0.4)
    for g in range(Hkv):
        assert np.array_equal(out[:, 2 * g], out[:, 2 * g + 1])
    assert not np.allclose(out[:, 0], out[:, 2])


@pytest.mark.parametrize("seed", range(4))
def test_brute_force_tiny(seed):
    rng = np.random.default_rng(200 + seed)
    M, Hkv, G, D = int(rng.integers(1, 4)), int(rng.integers(1, 3)), int(rng.integers(1, 3)), 4
    P, T = int(rng.integers(0, 4)), int(rng.integers(0, 5))
    Hq = Hkv * G
    x = synth.tree_attn_inputs(M, Hq, Hkv, D, P + T + M, seed + 50)
    mask = rng.integers(0, 2 ** 31, (M, 1)).astype(np.uint32)
    for i in range(M):
        mask[i, 0] |= np.uint32(1 << (T + i))
    scale = 0.7
    out, _, _ = tree_attention(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, scale)
    f = oracle.bf16_bits_to_f64
    for i in range(M):
        for h in range(Hq):
            g = h // G
            keys, vals = [], []
            for t in range(P + T + M):
                if t >= P and not (int(mask[i, 0]) >> (t - P)) & 1:
                    continue
                src_k = f(x["k_new"][t - P - T, g]) if t >= P + T else f(x["k_cache"][g, t])
                src_v = f(x["v_new"][t - P - T, g]) if t >= P + T else f(x["v_cache"][g, t])
                keys.append(sum(float(a) * float(b) for a, b in zip(f(x["q"][i, h]), src_k)) * scale)
                vals.append(src_v)
            mx = max(keys)
            w = [math.exp(s - mx) for s in keys]
            tot = sum(w)
            want = [sum(w[j] * vals[j][d] for j in range(len(w))) / tot for d in range(D)]
            assert np.allclose(out[i, h], want, atol=1e-12), (seed, i, h)
    assert list(visible_positions(mask, 0, P, T, M))[:P] == list(range(P))


@pytest.mark.parametrize("M,Hq,Hkv,D,P,T,k,qs", [(6, 28, 4, 16, 40, 12, 6, 1.0), (3, 6, 3, 16, 33, 7, 4, 2.0)])
def test_weighted_abs_v_matches_library_sdpa_on_abs_values(M, Hq, Hkv, D, P, T, k, qs):
    # sum_j p_j |v_j| is attention with the values replaced by their magnitudes:
    # the library routine on |V| must give the same numbers (pins the weights p_j,
    # the gather of visible keys and the head grouping of weighted_abs_v).
    x, mask = _case(M, Hq, Hkv, D, P, T, k, 11 + P + T, q_scale=qs)
    scale = 1.0 / math.sqrt(D)
    wabs = oracle.weighted_abs_v(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, scale)
    _, kc, vc = tree_attention(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, scale)
    L = P + T + M
    q = torch.from_numpy(oracle.bf16_bits_to_f64(x["q"])).permute(1, 0, 2)[None]
    K = torch.from_numpy(oracle.bf16_bits_to_f64(kc[:, :L])).repeat_interleave(Hq // Hkv, 0)[None]
    V = torch.from_numpy(np.abs(oracle.bf16_bits_to_f64(vc[:, :L]))).repeat_interleave(Hq // Hkv, 0)[None]
    allow = np.zeros((M, L), dtype=bool)
    allow[:, :P] = True
    for i in range(M):
        for j in range(T + M):
            allow[i, P + j] = (int(mask[i, j >> 5]) >> (j & 31)) & 1 == 1
    ref = torch.nn.functional.scaled_dot_product_attention(q, K, V, attn_mask=torch.from_numpy(allow),
                                                           scale=scale)
    assert np.allclose(wabs, ref[0].permute(1, 0, 2).numpy(), atol=1e-12, rtol=0)


def test_weighted_abs_v_bounds_and_sign_cases():
    M, Hq, Hkv, D, P, T, k = 4, 6, 2, 8, 17, 9, 4
    x, mask = _case(M, Hq, Hkv, D, P, T, k, 23)
    scale = 1.0 / math.sqrt(D)
    args = (x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, scale)
    out, _, _ = tree_attention(*args)
    wabs = oracle.weighted_abs_v(*args)
    # triangle inequality: |sum p v| <= sum p |v|, with p_j >= 0 summing to one
    assert (np.abs(out) <= wabs + 1e-15).all()
    assert (wabs >= 0).all()
    # values of one sign: the bound is attained (|v| = v or -v everywhere)
    vc_pos = x["v_cache"] & np.uint16(0x7FFF)  # clear the bf16 sign bits
    vn_pos = x["v_new"] & np.uint16(0x7FFF)
    args_pos = (x["q"], x["k_cache"], vc_pos, P, T, x["k_new"], vn_pos, mask, scale)
    out_pos, _, _ = tree_attention(*args_pos)
    assert np.allclose(oracle.weighted_abs_v(*args_pos), out_pos, atol=1e-14, rtol=0)
    neg = lambda b: b ^ np.uint16(0x8000)
    args_neg = (x["q"], x["k_cache"], neg(vc_pos), P, T, x["k_new"], neg(vn_pos), mask, scale)
    out_neg, _, _ = tree_attention(*args_neg)
    assert np.allclose(oracle.weighted_abs_v(*args_neg), -out_neg, atol=1e-14, rtol=0)
    # constant values c: the weighted magnitude is |c| whatever the weights
    c = oracle.bf16_round_bits(np.full(x["v_cache"].shape, -0.375, np.float32))
    cn = oracle.bf16_round_bits(np.full(x["v_new"].shape, -0.375, np.float32))
    wc = oracle.weighted_abs_v(x["q"], x["k_cache"], c, P, T, x["k_new"], cn, mask, scale)
    assert np.allclose(wc, 0.375, atol=1e-15, rtol=0)


@pytest.mark.parametrize("seed", range(3))
def test_weighted_abs_v_brute_force_tiny(seed):
    rng = np.random.default_rng(300 + seed)
    M, Hkv, G, D = int(rng.integers(1, 4)), int(rng.integers(1, 3)), int(rng.integers(1, 3)), 4
    P, T = int(rng.integers(0, 4)), int(rng.integers(0, 5))
    Hq = Hkv * G
    x = synth.tree_attn_inputs(M, Hq, Hkv, D, P + T + M, seed + 70)
    mask = rng.integers(0, 2 ** 31, (M, 1)).astype(np.uint32)
    for i in range(M):
        mask[i, 0] |= np.uint32(1 << (T + i))
    scale = 0.9
    wabs = oracle.weighted_abs_v(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, scale)
    f = oracle.bf16_bits_to_f64
    for i in range(M):
        for h in range(Hq):
            g = h // G
            keys, vals = [], []
            for t in range(P + T + M):
                if t >= P and not (int(mask[i, 0]) >> (t - P)) & 1:
                    continue
                src_k = f(x["k_new"][t - P - T, g]) if t >= P + T else f(x["k_cache"][g, t])
                src_v = f(x["v_new"][t - P - T, g]) if t >= P + T else f(x["v_cache"][g, t])
                keys.append(sum(float(a) * float(b) for a, b in zip(f(x["q"][i, h]), src_k)) * scale)
                vals.append([abs(float(v)) for v in src_v])
            mx = max(keys)
            w = [math.exp(s - mx) for s in keys]
            tot = sum(w)
            want = [sum(w[j] * vals[j][d] for j in range(len(w))) / tot for d in range(D)]
            assert np.allclose(wabs[i, h], want, atol=1e-12), (seed, i, h)
