"""Seeded synthetic inputs shaped like the paper's draft-model workloads.

Only random numbers and their placement live here -- no quantization, packing or
matmul arithmetic -- so both the HIP path and the CPU oracle can take the very
same inputs.  Weights are N(0, 0.02) float32; activations are N(0, 1) rounded to
bfloat16 (round-to-nearest-even), optionally with a fraction of input channels
scaled by 20 before rounding (outlier channels).
"""
from __future__ import annotations

import numpy as np


def seed_of(*keys: int) -> int:
    """A 63-bit seed derived from a tuple of non-negative integers."""
    ss = np.random.SeedSequence([int(k) for k in keys])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & np.uint64(0x7FFF_FFFF_FFFF_FFFF))


def weights_np(N: int, K: int, *keys: int, std: float = 0.02) -> np.ndarray:
    """float32 [N][K] ~ N(0, std^2), generated on the host."""
    rng = np.random.default_rng(np.random.SeedSequence([int(k) for k in keys]))
    return (rng.standard_normal((N, K), dtype=np.float32) * np.float32(std)).astype(np.float32)


def weights_torch(N: int, K: int, *keys: int, device="cuda", std: float = 0.02):
    """float32 [N][K] ~ N(0, std^2), generated directly on ``device`` by torch's
    seeded generator (used for the multi-GB stacks)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed_of(*keys))
    w = torch.randn((N, K), generator=g, device=device, dtype=torch.float32)
    return w.mul_(std)


def outlier_channels(K: int, frac: float, *keys: int) -> np.ndarray:
    """round(frac*K) distinct input channels, chosen by a seeded RNG."""
    n = int(round(frac * K))
    rng = np.random.default_rng(np.random.SeedSequence([int(k) for k in keys] + [7]))
    return np.sort(rng.choice(K, size=n, replace=False))


def activations(M: int, K: int, *keys: int, outlier_frac: float = 0.0,
                outlier_scale: float = 20.0):
    """bfloat16 torch tensor [M][K] (CPU): N(0, 1) float32, outlier channels
    multiplied by ``outlier_scale`` in float32, then rounded to bf16."""
    import torch
    rng = np.random.default_rng(np.random.SeedSequence([int(k) for k in keys]))
    x = rng.standard_normal((M, K), dtype=np.float32)
    if outlier_frac > 0:
        ch = outlier_channels(K, outlier_frac, *keys)
        x[:, ch] *= np.float32(outlier_scale)
    return torch.from_numpy(x).to(torch.bfloat16)


def bf16_bits(t) -> np.ndarray:
    """uint16 bit patterns of a (CPU) bfloat16 tensor."""
    import torch
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def layer_weights(projs, cfg: int, layer: int, device="cuda"):
    """fp32 weights of one decoder layer: {name: [N][K]} for the 7 projections, each
    from its own seeded stream (cfg, layer, projection index)."""
    return {p.name: weights_torch(p.N, p.K, cfg, layer, i, device=device)
            for i, p in enumerate(projs)}


def tree_levels_mask(T: int, k: int, M: int, *keys: int) -> np.ndarray:
    """Ancestor mask of a random draft tree, as uint32 bit rows [M][ceil((T + M) / 32)].

    The T tree tokens already in the cache come in levels of k in cache order (the
    last level may be shorter); each token's parent is a uniformly chosen token of
    the level before, the first level hanging off the prefix.  The M new tokens form
    the next level.  Bit j of row i is set when tree token j (cache position
    prefix + j) is an ancestor of new token i, and bit T + i marks the token itself.
    """
    rng = np.random.default_rng(np.random.SeedSequence([int(x) for x in keys] + [11]))
    parent = np.full(T + M, -1, dtype=np.int64)
    levels = [list(range(s, min(s + k, T))) for s in range(0, T, k)]
    for lv in range(1, len(levels)):
        for j in levels[lv]:
            parent[j] = rng.choice(levels[lv - 1])
    for i in range(M):
        parent[T + i] = rng.choice(levels[-1]) if levels else -1
    W = (T + M + 31) // 32
    mask = np.zeros((M, W), dtype=np.uint32)
    for i in range(M):
        j = T + i
        while j >= 0:
            mask[i, j // 32] |= np.uint32(1 << (j % 32))
            j = parent[j]
    return mask


def tree_attn_inputs(M: int, Hq: int, Hkv: int, D: int, S: int, *keys: int, q_scale: float = 1.0):
    """bf16 bit patterns (uint16) of one layer's tree-attention inputs: q [M][Hq][D]
    (N(0, q_scale^2)), K and V caches [Hkv][S][D], new keys and values [M][Hkv][D]
    (all N(0, 1)); float32 draws rounded to bf16 (round to nearest even)."""
    import torch
    rng = np.random.default_rng(np.random.SeedSequence([int(x) for x in keys] + [13]))

    def bf(shape, s=1.0):
        a = rng.standard_normal(shape, dtype=np.float32) * np.float32(s)
        return bf16_bits(torch.from_numpy(a).to(torch.bfloat16))

    return {"q": bf((M, Hq, D), q_scale), "k_cache": bf((Hkv, S, D)), "v_cache": bf((Hkv, S, D)),
            "k_new": bf((M, Hkv, D)), "v_new": bf((M, Hkv, D))}
