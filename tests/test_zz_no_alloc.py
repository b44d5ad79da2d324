"""GPU test of subspec_qlinear_noalloc, the allocation-free variant of subspec_qlinear
(its scratch is a fixed array per device inside the library), through the C ABI:
two calls in a row, the second with a smaller input, each against subspec_qlinear's
output and the oracle; a shape whose usual plan needs more scratch than the array
holds; and no use of the growable workspace."""
import numpy as np
import pytest

import oracle
import paper_2509_18344_amd as ss
from paper_2509_18344_amd import synth

from helpers import assert_close, bf16_to_f64, device_projection

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"


def _both(p, x, M):
    """(subspec_qlinear output, subspec_qlinear_noalloc output) for x [M][K]."""
    N, K, bits, group = p["N"], p["K"], p["bits"], p["group"]
    y_ref = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    y_na = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device=DEV)
    ss.subspec_qlinear(x, p["qweight"], p["scales"], p["zeros"], bits, group, M, N, K, y_ref)
    ss.subspec_qlinear_noalloc(x, p["qweight"], p["scales"], p["zeros"], bits, group, M, N, K, y_na)
    torch.cuda.synchronize()
    return y_ref, y_na


def test_noalloc_matches_qlinear_on_two_calls_in_a_row():
    # both plans fit the fixed scratch, so the two entry points run the same launches
    # and must agree bit for bit; each is also checked against the oracle
    cases = [(64, 4608, 3584, 4, 128), (40, 1024, 2048, 3, 128)]  # the second call is smaller
    ws0 = ss.subspec_workspace_info()
    for i, (M, N, K, bits, group) in enumerate(cases):
        plan = ss.subspec_qlinear_plan(M, N, K, bits, group)
        assert plan["splits"] > 1 and 0 < plan["workspace_bytes"] <= ss.SUBSPEC_NOALLOC_SCRATCH_BYTES, plan
        w = synth.weights_np(N, K, 900 + i, bits)
        p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
        q, s16, z16 = oracle.quantize_minmax(w, bits, group)
        x = synth.activations(M, K, 910 + i, M)
        ss.subspec_reserve(plan["workspace_bytes"])  # subspec_qlinear below must not grow it
        ws1 = ss.subspec_workspace_info()
        y_ref, y_na = _both(p, x.to(DEV), M)
        assert torch.equal(y_na.view(torch.int16), y_ref.view(torch.int16)), (M, N, K)
        assert_close(bf16_to_f64(y_na), oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, group),
                     f"noalloc M={M} N={N} K={K}")
        # the allocation-free call neither grew nor replaced the growable workspace
        assert ss.subspec_workspace_info() == ws1
    assert ss.subspec_workspace_info()["allocations"] >= ws0["allocations"]


def test_noalloc_caps_its_splits_to_the_fixed_scratch():
    # Qwen2.5-7B gate|up at M = 128: the usual plan splits the tail column groups six
    # ways (about 116 MB of partial sums); the allocation-free call splits less and
    # agrees with subspec_qlinear within the fp32-accumulation tolerance, and with the
    # oracle on sampled columns
    M, N, K, bits, group = 128, 37888, 3584, 4, 128
    assert ss.subspec_qlinear_plan(M, N, K, bits, group)["workspace_bytes"] > ss.SUBSPEC_NOALLOC_SCRATCH_BYTES
    w = synth.weights_torch(N, K, 920, device=DEV)
    p = device_projection(w, bits, group)
    x = synth.activations(M, K, 921)
    y_ref, y_na = _both(p, x.to(DEV), M)
    assert_close(bf16_to_f64(y_na), bf16_to_f64(y_ref), "noalloc against qlinear, capped splits")
    cols = np.unique(np.concatenate([np.arange(0, N, 997), [N - 16, N - 1]]))
    wc = w[torch.from_numpy(cols).to(DEV)].cpu().numpy()
    q, s16, z16 = oracle.quantize_minmax(wc, bits, group)
    ref = oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, group)
    assert_close(bf16_to_f64(y_na)[:, cols], ref, "noalloc against the oracle, sampled columns")
