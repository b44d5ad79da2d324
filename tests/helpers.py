"""Shared helpers of the GPU tests: build one quantized projection on the device with
the library, and the element-wise tolerance check against the oracle."""
import numpy as np

import oracle
import paper_2509_18344_amd as ss
from paper_2509_18344_amd import synth

RTOL, ATOL = 1e-2, 1e-3  # |y - y_ref| <= ATOL + RTOL * |y_ref|, bf16 outputs, fp32 accumulation


def device_projection(w, bits, group):
    """Quantize (subspec_quantize) and pack (subspec_qpack) fp32 weights ``w`` [N][K]
    (a torch tensor on the GPU) with the library; returns device tensors."""
    import torch
    N, K = w.shape
    dev = w.device
    codes = torch.empty((N, K), dtype=torch.uint8, device=dev)
    sc = torch.empty((K // group, N), dtype=torch.float16, device=dev)
    zr = torch.empty((K // group, N), dtype=torch.float16, device=dev)
    ss.subspec_quantize(w, bits, group, N, K, codes, sc, zr)
    qw = torch.empty(ss.subspec_qpack_bytes(bits, N, K), dtype=torch.uint8, device=dev)
    ss.subspec_qpack(codes, bits, N, K, qw)
    return {"codes": codes, "scales": sc, "zeros": zr, "qweight": qw, "N": N, "K": K,
            "bits": bits, "group": group}


def run_qlinear(proj, x, path=ss.SUBSPEC_PATH_AUTO):
    import torch
    M = x.shape[0]
    y = torch.empty((M, proj["N"]), dtype=torch.bfloat16, device=x.device)
    ss.subspec_qlinear_path(x, proj["qweight"], proj["scales"], proj["zeros"], proj["bits"],
                            proj["group"], M, proj["N"], proj["K"], y, path)
    return y


def bf16_to_f64(t):
    return oracle.bf16_bits_to_f64(synth.bf16_bits(t.cpu()))


def assert_close(y_gpu, y_ref, what=""):
    y = np.asarray(y_gpu, dtype=np.float64)
    bad = np.abs(y - y_ref) > ATOL + RTOL * np.abs(y_ref)
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outside tolerance; first at "
                             f"{i}: gpu={y[i]!r} ref={y_ref[i]!r}")
