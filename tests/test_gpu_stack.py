"""GPU tests of the per-layer launch plan (q|k|v, o, gate|up, down per decoder layer)
and of its HIP-graph capture against the fp64 oracle: small shapes in full, and the
Qwen2.5-7B/32B stacks at their full sizes, every output of the first and the last
layer's launches (the whole stack runs as captured graphs)."""
import numpy as np
import pytest

import oracle
import paper_2509_18344_amd as ss
from paper_2509_18344_amd import prepare, synth
from paper_2509_18344_amd.workloads import WORKLOADS, Proj, fused_layer

from helpers import assert_close, bf16_to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"
TINY = (Proj("q", 256, 256), Proj("k", 256, 64), Proj("v", 256, 64), Proj("o", 256, 256),
        Proj("gate", 256, 512), Proj("up", 256, 512), Proj("down", 512, 256))


def _build(projs, layers, bits, group, cfg, keep_layers, sample):
    """Pack `layers` decoder layers (fused plan).  For the layers in keep_layers, keep
    the fp32 rows (output columns) listed by sample(N) of every fused launch (all of
    them when sample is None)."""
    plan = fused_layer(projs)
    packed, kept = [], {}
    for l in range(layers):
        w = synth.layer_weights(projs, cfg, l)
        groups = [[w["q"], w["k"], w["v"]], [w["o"]], [w["gate"], w["up"]], [w["down"]]]
        layer = []
        for li, parts in enumerate(groups):
            wl = torch.cat(parts, 0) if len(parts) > 1 else parts[0]
            layer.append(prepare.quantize_pack(wl, bits, group))
            if l in keep_layers:
                if sample is None:
                    kept[(l, li)] = (None, wl.cpu().numpy())
                else:
                    cols = sample(plan[li].N)
                    kept[(l, li)] = (cols, wl[torch.as_tensor(cols, device=wl.device)].cpu().numpy())
            del wl
        packed.append(layer)
        del w
    torch.cuda.synchronize()
    return plan, packed, kept


def _acts(plan, layers, M, cfg, outlier_frac=0.0):
    xs, ys = [], []
    for l in range(layers):
        xs.append([synth.activations(M, p.K, cfg, 1000 + l, li, outlier_frac=outlier_frac)
                   for li, p in enumerate(plan)])
        ys.append([torch.empty((M, p.N), dtype=torch.bfloat16, device=DEV) for p in plan])
    return xs, ys


def _launch_list(packed, xs_dev, ys):
    out = []
    for l, layer in enumerate(packed):
        out += prepare.layer_launches(layer, xs_dev[l], ys[l])
    return out


def _check_sampled(kept, xs, ys, bits, group, what):
    for (l, li), (cols, wrows) in kept.items():
        q, s16, z16 = oracle.quantize_minmax(wrows, bits, group)
        y_ref = oracle.qlinear_ref(synth.bf16_bits(xs[l][li]), q, s16, z16, group)
        y = bf16_to_f64(ys[l][li][:, torch.as_tensor(cols, device=DEV)])
        assert_close(y, y_ref, f"{what} layer={l} launch={li}")


@pytest.mark.parametrize("M", [5, 40])
def test_graph_replays_match_eager_and_oracle(M):
    layers, bits, group = 2, 4, 64
    plan, packed, kept = _build(TINY, layers, bits, group, 31, {0, 1}, lambda n: np.arange(n))
    xs, ys = _acts(plan, layers, M, 31)
    xs_dev = [[x.to(DEV) for x in row] for row in xs]
    launches = _launch_list(packed, xs_dev, ys)
    ss.subspec_stack_forward(launches, bits, group, M)
    torch.cuda.synchronize()
    eager = [[y.clone() for y in row] for row in ys]
    _check_sampled(kept, xs, ys, bits, group, "eager")
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        g = ss.subspec_stack_capture(launches, bits, group, M, side)
    try:
        for rep in range(3):
            for row in ys:  # the program's own eager work between replays
                for y in row:
                    y.zero_()
            torch.cuda.synchronize()
            ss.subspec_graph_launch(g, side)
            side.synchronize()
            for l in range(layers):
                for li in range(len(plan)):
                    assert torch.equal(ys[l][li].view(torch.int16), eager[l][li].view(torch.int16)), \
                        (rep, l, li)
    finally:
        ss.subspec_graph_destroy(g)


def _sample_cols(n):
    base = np.linspace(0, n - 1, 21).astype(int)
    return np.unique(np.concatenate([base, [15, 16, n - 16, n - 1]]))


def _check_every_output(w, bits, group, x_bits, y_gpu, what, block=1024):
    """Every output column of one launch against the oracle: the fp32 weights w [N][K]
    are quantized by the oracle in blocks of `block` columns (quantization is per
    column, so a block's codes are the full matrix's), and each block's outputs are
    compared for every M.  x_bits: {M: bf16 bits [M][K]}; y_gpu: {M: float64 [M][N]}."""
    N = w.shape[0]
    for n0 in range(0, N, block):
        n1 = min(N, n0 + block)
        q, s16, z16 = oracle.quantize_minmax(w[n0:n1], bits, group)
        for M, xb in x_bits.items():
            assert_close(y_gpu[M][:, n0:n1], oracle.qlinear_ref(xb, q, s16, z16, group),
                         f"{what} M={M} columns {n0}:{n1}")


def _run_stack_graph(wl, cfg, Ms, keep):
    """Run the whole stack as one captured graph per M; compare every output of the
    launches of the layers in `keep` with the oracle."""
    layers = wl.layers
    plan, packed, kept = _build(wl.projs, layers, wl.bits, wl.group, cfg, keep, None)
    x_bits = {key: {} for key in kept}
    y_gpu = {key: {} for key in kept}
    for M in Ms:
        xs, ys = _acts(plan, layers, M, cfg, wl.outlier_frac)
        xs_dev = [[x.to(DEV) for x in row] for row in xs]
        launches = _launch_list(packed, xs_dev, ys)
        side = torch.cuda.Stream()
        with torch.cuda.stream(side):
            g = ss.subspec_stack_capture(launches, wl.bits, wl.group, M, side)
        try:
            ss.subspec_graph_launch(g, side)
            side.synchronize()
        finally:
            ss.subspec_graph_destroy(g)
        for (l, li) in kept:
            x_bits[(l, li)][M] = synth.bf16_bits(xs[l][li])
            y_gpu[(l, li)][M] = bf16_to_f64(ys[l][li])
        del xs_dev, ys, launches
    del packed
    torch.cuda.empty_cache()
    for (l, li), (_, w) in sorted(kept.items()):
        _check_every_output(w, wl.bits, wl.group, x_bits[(l, li)], y_gpu[(l, li)],
                            f"{wl.key} layer={l} launch={plan[li].name}")


def test_qwen7b_stack_28_layers_m64():
    wl = WORKLOADS["qwen7b_stack"]
    _run_stack_graph(wl, 3, [64], {0, wl.layers - 1})


def test_qwen32b_stack_3bit():
    wl = WORKLOADS["qwen32b_stack"]
    _run_stack_graph(wl, 4, [1, 16, 64, 128], {0, wl.layers - 1})


def test_qwen32b_stack_2bit_outliers_m128():
    wl = WORKLOADS["qwen32b_2bit"]
    _run_stack_graph(wl, 5, [128], {0, wl.layers - 1})


def test_qwen7b_mlp_projections():
    """gate|up (K=3584, N=37888) and down (K=18944, N=3584), 4-bit g128, at
    M in {1, 8, 32, 64}: every output against the oracle."""
    for li, (N, K) in enumerate([(37888, 3584), (3584, 18944)]):
        w = synth.weights_torch(N, K, 2, li)
        p = prepare.quantize_pack(w, 4, 128)
        x_bits, y_gpu = {}, {}
        for M in (1, 8, 32, 64):
            x = synth.activations(M, K, 2, 100 + li, M)
            y = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
            ss.subspec_qlinear(x.to(DEV), p["qweight"], p["scales"], p["zeros"], 4, 128, M, N, K, y)
            x_bits[M] = synth.bf16_bits(x)
            y_gpu[M] = bf16_to_f64(y)
        w_host = w.cpu().numpy()
        cols = _sample_cols(N)
        # the quantizer on these columns is the oracle's, bit for bit
        _, s16, _ = oracle.quantize_minmax(w_host[cols], 4, 128)
        assert np.array_equal(p["scales"][:, torch.as_tensor(cols, device=DEV)].cpu().numpy()
                              .view(np.uint16), s16.view(np.uint16))
        del w, p
        _check_every_output(w_host, 4, 128, x_bits, y_gpu, f"qwen7b mlp N={N} K={K}")
