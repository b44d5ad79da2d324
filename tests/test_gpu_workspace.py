"""GPU tests of the per-device workspace the library's calls share: the split-K
completion counters at its start must survive every kind of call (tree attention
included), growth must leave the buffers of live captured graphs valid, and calls
whose needs were reserved must not allocate."""
import math

import numpy as np
import pytest

import oracle
import paper_2509_18344_amd as ss
from paper_2509_18344_amd import synth

from helpers import assert_close, bf16_to_f64, device_projection, run_qlinear

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"


def _projection(N, K, bits, group, seed):
    w = synth.weights_np(N, K, seed, bits, group)
    p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
    q, s16, z16 = oracle.quantize_minmax(w, bits, group)
    return p, (q, s16, z16)


def _qlinear_checked(p, ref, M, seed, what):
    q, s16, z16 = ref
    x = synth.activations(M, p["K"], seed, M)
    y = run_qlinear(p, x.to(DEV))
    torch.cuda.synchronize()
    assert_close(bf16_to_f64(y), oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, p["group"]), what)


def _attention_7b_last_pass(seed):
    """One layer's tree attention at the Qwen2.5-7B shape of the last pass of a depth-48
    tree (6 new tokens, 2048 committed positions, 282 earlier tree tokens)."""
    M, Hq, Hkv, P, T, D = 6, 28, 4, 2048, 282, 128
    S = P + T + M
    x = synth.tree_attn_inputs(M, Hq, Hkv, D, S, seed)
    mask = synth.tree_levels_mask(T, 6, M, seed)
    scale = 1.0 / math.sqrt(D)
    dev = {n: torch.from_numpy(np.ascontiguousarray(x[n]).view(np.int16)).to(DEV)
           for n in ("q", "k_cache", "v_cache", "k_new", "v_new")}
    mk = torch.from_numpy(mask.view(np.int32)).to(DEV)
    out = torch.empty((M, Hq, D), dtype=torch.int16, device=DEV)
    ss.subspec_tree_attention(dev["q"], dev["k_cache"], dev["v_cache"], dev["k_new"], dev["v_new"], mk,
                              M, Hq, Hkv, S, P, T, scale, out)
    torch.cuda.synchronize()
    ref, _, _ = oracle.tree_attention(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"],
                                      mask, scale)
    wabs = oracle.weighted_abs_v(x["q"], x["k_cache"], x["v_cache"], P, T, x["k_new"], x["v_new"], mask, scale)
    got = oracle.bf16_bits_to_f64(out.cpu().numpy().view(np.uint16))
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 2.0 ** -14 * wabs + 1e-6)


def test_attention_leaves_the_split_counters_to_qlinear_and_tree_expand():
    """In a draft pass each layer's attention runs before its projections: the
    attention's partial outputs must not land on the completion counters that a
    split-K qlinear (Qwen2.5-7B q|k|v at M = 64) and the tree expansion rely on."""
    p, ref = _projection(4608, 3584, 4, 128, 600)
    assert ss.subspec_qlinear_plan(64, 4608, 3584, 4, 128)["splits"] > 1
    for rnd in range(2):
        _attention_7b_last_pass(610 + rnd)
        _qlinear_checked(p, ref, 64, 620 + rnd, f"q|k|v M=64 after attention, round {rnd}")
        _attention_7b_last_pass(630 + rnd)
        R, V, k, T = 6, 152064, 6, 0.2
        bits = oracle.bf16_round_bits(np.random.default_rng(640 + rnd).normal(0.0, 3.0, (R, V)).astype(np.float32))
        parent = np.random.default_rng(650 + rnd).uniform(-12.0, 0.0, R).astype(np.float32)
        po = torch.empty(k, dtype=torch.int32, device=DEV)
        to = torch.empty(k, dtype=torch.int32, device=DEV)
        so = torch.empty(k, dtype=torch.float32, device=DEV)
        ss.subspec_tree_expand(torch.from_numpy(bits.view(np.int16)).to(DEV), torch.from_numpy(parent).to(DEV),
                               R, V, T, k, po, to, so)
        torch.cuda.synchronize()
        ref_pi, ref_tok, ref_sc = oracle.tree_expand(bits, parent.astype(np.float64), T, k)
        assert np.all(np.abs(so.cpu().numpy() - ref_sc) <= 2e-4 + 1e-6 * np.abs(ref_sc))
        if oracle.kth_gap(bits, parent.astype(np.float64), T, k) > 8e-4:
            assert set(zip(po.cpu().tolist(), to.cpu().tolist())) == set(zip(ref_pi.tolist(), ref_tok.tolist()))


def test_growth_keeps_the_buffers_of_live_graphs():
    """A graph keeps the workspace address it was captured with.  Growing the
    workspace afterwards (a larger call, or subspec_reserve) must leave that buffer
    allocated until the graph is destroyed: replays after the growth still match the
    oracle, and destroying the graph releases the retired buffer."""
    M, N, K = 40, 1024, 2048
    p, ref = _projection(N, K, 3, 128, 700)
    plan = ss.subspec_qlinear_plan(M, N, K, 3, 128)
    assert plan["splits"] > 1
    # no graph alive: the capture below needs no growth, and buffers retired by
    # earlier tests are freed
    ss.subspec_reserve(plan["workspace_bytes"])
    assert ss.subspec_workspace_info()["retired"] == 0
    q, s16, z16 = ref
    x = synth.activations(M, K, 701).to(DEV)
    y_ref = oracle.qlinear_ref(synth.bf16_bits(x.cpu()), q, s16, z16, 128)
    y = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    launch = [{"x": x, "qweight": p["qweight"], "scales": p["scales"], "zeros": p["zeros"], "y": y, "N": N, "K": K}]
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        g = ss.subspec_stack_capture(launch, 3, 128, M, side)
    try:
        before = ss.subspec_workspace_info()
        ss.subspec_reserve(2 * before["bytes"] + (1 << 20))
        after = ss.subspec_workspace_info()
        assert after["bytes"] > before["bytes"] and after["allocations"] == before["allocations"] + 1
        assert after["retired"] == 1  # the graph's buffer, kept while the graph lives
        for rep in range(3):
            y.zero_()
            ss.subspec_graph_launch(g, side)
            side.synchronize()
            assert_close(bf16_to_f64(y), y_ref, f"replay {rep} after growth")
            # eager work on the grown buffer between replays
            _qlinear_checked(p, ref, M, 702 + rep, f"eager call {rep} after growth")
    finally:
        ss.subspec_graph_destroy(g)
    assert ss.subspec_workspace_info()["retired"] == 0


def test_calls_within_the_reserved_workspace_do_not_allocate():
    """After subspec_reserve(bytes), calls that need at most `bytes` neither grow nor
    replace the workspace (no allocation on the call path)."""
    shapes = [(64, 4608, 3584, 4, 128), (8, 3584, 18944, 4, 128), (128, 2048, 1024, 2, 64)]
    need = max(ss.subspec_qlinear_plan(M, N, K, b, g)["workspace_bytes"] for M, N, K, b, g in shapes)
    need = max(need, ss.subspec_tree_workspace_bytes(6, 152064, 6),
               ss.subspec_tree_attention_workspace_bytes(6, 28, 4, 2048, 282))
    ss.subspec_reserve(need)
    start = ss.subspec_workspace_info()
    assert start["bytes"] >= need
    for i, (M, N, K, b, g) in enumerate(shapes):
        p, ref = _projection(N, K, b, g, 800 + i)
        _qlinear_checked(p, ref, M, 810 + i, f"M={M} N={N} K={K} after reserve")
    _attention_7b_last_pass(820)
    now = ss.subspec_workspace_info()
    assert (now["bytes"], now["allocations"]) == (start["bytes"], start["allocations"])
