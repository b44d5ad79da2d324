"""GPU parity of the quantizer with an HQQ-style optimised zero-point: codes, fp16
scales and zeros bit for bit against the oracle (both sides take every rounding
decision in float64 with sums in index order), and the unchanged qlinear kernels on
HQQ-quantized weights against the oracle's product."""
import numpy as np
import pytest

import oracle
import paper_2509_18344_amd as ss
from paper_2509_18344_amd import synth

from helpers import assert_close, bf16_to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _hqq_gpu(w, bits, group):
    N, K = w.shape
    wd = torch.from_numpy(w).cuda()
    codes = torch.empty((N, K), dtype=torch.uint8, device="cuda")
    sc = torch.empty((K // group, N), dtype=torch.float16, device="cuda")
    zr = torch.empty((K // group, N), dtype=torch.float16, device="cuda")
    ss.subspec_quantize_hqq(wd, bits, group, N, K, codes, sc, zr)
    torch.cuda.synchronize()
    return codes, sc, zr


@pytest.mark.parametrize("bits,group,N,K", [(4, 64, 48, 1024), (3, 64, 32, 512), (2, 64, 16, 768),
                                            (4, 128, 40, 1024), (3, 128, 16, 384), (4, 64, 3584, 256)])
def test_hqq_quantizer_bit_exact(bits, group, N, K):
    w = synth.weights_np(N, K, 31, bits, group)
    w[0, :group] = 0.125            # a constant group
    w[1, group:2 * group] = 0.0     # an all-zero group
    codes, sc, zr = _hqq_gpu(w, bits, group)
    q, s16, z16 = oracle.quantize_hqq(w, bits, group)
    assert np.array_equal(codes.cpu().numpy(), q)
    assert np.array_equal(sc.cpu().numpy().view(np.uint16), s16.view(np.uint16))
    assert np.array_equal(zr.cpu().numpy().view(np.uint16), z16.view(np.uint16))
    # the zeros moved for most groups (the optimisation ran), the scales did not
    _, s0, z0 = oracle.quantize_minmax(w, bits, group)
    assert np.array_equal(s16, s0) and (z16 != z0).mean() > 0.3


def test_hqq_weights_through_qlinear():
    bits, group, N, K, M = 4, 64, 512, 1024, 8
    w = synth.weights_np(N, K, 41)
    codes, sc, zr = _hqq_gpu(w, bits, group)
    qw = torch.empty(ss.subspec_qpack_bytes(bits, N, K), dtype=torch.uint8, device="cuda")
    ss.subspec_qpack(codes, bits, N, K, qw)
    x = synth.activations(M, K, 42).cuda()
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    ss.subspec_qlinear(x, qw, sc, zr, bits, group, M, N, K, y)
    torch.cuda.synchronize()
    q, s16, z16 = oracle.quantize_hqq(w, bits, group)
    ref = oracle.qlinear_ref(synth.bf16_bits(x.cpu()), q, s16, z16, group)
    assert_close(bf16_to_f64(y), ref, "qlinear on HQQ weights")
