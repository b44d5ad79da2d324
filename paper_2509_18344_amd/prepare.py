"""Building substitute weights on the GPU with the library: quantize (subspec_quantize)
and pack (subspec_qpack) one projection, or several that share their input and are
fused along N (q|k|v, gate|up), plus the per-layer launch list of a decoder layer."""
from __future__ import annotations

from . import _binding as b


def quantize_pack(w, bits: int, group: int, stream=None) -> dict:
    """w: float32 device tensor [N][K] -> packed projection (device tensors)."""
    import torch
    N, K = w.shape
    codes = torch.empty((N, K), dtype=torch.uint8, device=w.device)
    sc = torch.empty((K // group, N), dtype=torch.float16, device=w.device)
    zr = torch.empty((K // group, N), dtype=torch.float16, device=w.device)
    b.subspec_quantize(w, bits, group, N, K, codes, sc, zr, stream)
    qw = torch.empty(b.subspec_qpack_bytes(bits, N, K), dtype=torch.uint8, device=w.device)
    b.subspec_qpack(codes, bits, N, K, qw, stream)
    return {"qweight": qw, "scales": sc, "zeros": zr, "N": N, "K": K, "bits": bits,
            "group": group}


def fused(ws, bits: int, group: int) -> dict:
    """Projections sharing K, concatenated along N (quantization is per column, so
    the result equals the separate projections side by side)."""
    import torch
    return quantize_pack(torch.cat(list(ws), dim=0), bits, group)


def layer_launches(packed, xs, ys):
    """The 4-launch plan of one decoder layer: dicts for subspec_stack_forward."""
    return [{"x": xs[i], "y": ys[i], "qweight": p["qweight"], "scales": p["scales"],
             "zeros": p["zeros"], "N": p["N"], "K": p["K"]} for i, p in enumerate(packed)]
