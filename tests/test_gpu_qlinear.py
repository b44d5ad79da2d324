"""GPU parity of the HIP path against the fp64 CPU oracle, through the C ABI.

Integer/bit work (quantizer codes, fp16 scale/zero, packing, dequantization) must be
bit-exact; layer outputs must satisfy |y - y_ref| <= 1e-3 + 1e-2 |y_ref| element-wise,
with y_ref computed by the oracle on the exact dequantized weights."""
import numpy as np
import pytest

import oracle
import paper_2509_18344_amd as ss
from paper_2509_18344_amd import synth

from helpers import assert_close, bf16_to_f64, device_projection, run_qlinear

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda"


def _w(N, K, *keys):
    return synth.weights_np(N, K, *keys)


# ------------------------------------------------------------------ preparation

@pytest.mark.parametrize("bits,group", [(4, 64), (4, 128), (3, 128), (3, 64), (2, 64), (2, 128)])
def test_quantize_bit_exact(bits, group):
    N, K = 80, 768
    w = _w(N, K, 100, bits, group)
    # a few adversarial groups: constant, all positive, all negative, tiny range
    w[0, :group] = 0.25
    w[1, :group] = np.linspace(0.5, 2.0, group)
    w[2, :group] = np.linspace(-3.0, -1.0, group)
    w[3, :group] = np.tile((np.arange(group // 4) - 5.0) * 2.0 ** -22, 4)[:group]
    p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
    q, s16, z16 = oracle.quantize_minmax(w, bits, group)
    torch.cuda.synchronize()
    assert np.array_equal(p["codes"].cpu().numpy(), q)
    assert np.array_equal(p["scales"].cpu().numpy().view(np.uint16), s16.view(np.uint16))
    assert np.array_equal(p["zeros"].cpu().numpy().view(np.uint16), z16.view(np.uint16))


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_device_pack_matches_layout(bits):
    N, K = 48, 640
    rng = np.random.default_rng(bits)
    codes = rng.integers(0, 2 ** bits, (N, K)).astype(np.uint8)
    qw = torch.empty(ss.subspec_qpack_bytes(bits, N, K), dtype=torch.uint8, device=DEV)
    ss.subspec_qpack(torch.from_numpy(codes).to(DEV), bits, N, K, qw)
    torch.cuda.synchronize()
    assert np.array_equal(oracle.unpack(qw.cpu().numpy(), bits, N, K), codes)


@pytest.mark.parametrize("bits,group", [(4, 64), (4, 128), (3, 128), (2, 64)])
def test_dequant_bit_exact(bits, group):
    N, K = 64, 512
    w = _w(N, K, 200, bits, group)
    p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
    wf = torch.empty((N, K), dtype=torch.float32, device=DEV)
    wb = torch.empty((N, K), dtype=torch.int16, device=DEV)
    ss.subspec_qdequant(p["qweight"], p["scales"], p["zeros"], bits, group, N, K, wf, wb)
    torch.cuda.synchronize()
    q, s16, z16 = oracle.quantize_minmax(w, bits, group)
    exp_f = oracle.dequant_f32(q, s16, z16, group)
    exp_b = oracle.dequant_bf16_bits(q, s16, z16, group)
    assert np.array_equal(wf.cpu().numpy().view(np.uint32), exp_f.view(np.uint32))
    assert np.array_equal(wb.cpu().numpy().view(np.uint16), exp_b)


# ------------------------------------------------------------------ the layer

SHAPES = [(512, 256), (528, 640), (1040, 1152)]  # tiles x blocks incl. ragged groups/chunks


PATH_MS = {ss.SUBSPEC_PATH_GEMV: [1, 2, 3, 4, 5, 8],
           ss.SUBSPEC_PATH_MFMA16: [1, 8, 16, 17, 33, 64, 100, 128],
           ss.SUBSPEC_PATH_MFMA32: [1, 17, 64, 65, 100, 128]}


@pytest.mark.parametrize("bits,group", [(4, 64), (4, 128), (3, 128), (3, 64), (2, 64), (2, 128)])
@pytest.mark.parametrize("path", list(PATH_MS))
def test_qlinear_matches_oracle(bits, group, path):
    ms = PATH_MS[path]
    for (N, K) in SHAPES:
        w = _w(N, K, 300, N, K, bits, group)
        p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
        q, s16, z16 = oracle.quantize_minmax(w, bits, group)
        for M in ms:
            x = synth.activations(M, K, 301, M, N, K)
            y = run_qlinear(p, x.to(DEV), path)
            y_ref = oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, group)
            assert_close(bf16_to_f64(y), y_ref, f"bits={bits} g={group} path={path} M={M} N={N} K={K}")


@pytest.mark.parametrize("M,bits,group", [(1, 4, 128), (8, 4, 128), (40, 4, 128), (64, 4, 128),
                                          (2, 3, 128), (16, 3, 64), (5, 2, 64), (100, 2, 128)])
def test_qlinear_balanced_tail_split(M, bits, group):
    """More column groups than CUs (276 column groups, of the width the plan uses at
    this M): the groups past a multiple of the CU count run split along K while the
    others run whole; every output is checked against the oracle."""
    K = 1024
    probe = ss.subspec_qlinear_plan(M, 16 * 4096, K, bits, group)
    N = probe["waves"] * probe["tiles_per_wave"] * 16 * 276
    plan = ss.subspec_qlinear_plan(M, N, K, bits, group)
    assert 0 < plan["full_groups"] < plan["col_groups"] and plan["splits"] > 1, plan
    w = _w(N, K, 310, M, bits, group)
    p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
    q, s16, z16 = oracle.quantize_minmax(w, bits, group)
    x = synth.activations(M, K, 311, M, bits)
    ss.subspec_reserve(plan["workspace_bytes"])
    for _ in range(2):  # the completion counters must be back at zero for the second call
        y = run_qlinear(p, x.to(DEV))
        y_ref = oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, group)
        assert_close(bf16_to_f64(y), y_ref, f"tail split M={M} bits={bits} g={group} plan={plan}")


@pytest.mark.parametrize("M,N,bits,group", [(128, 49152, 3, 128), (65, 49168, 3, 128), (100, 49168, 2, 64),
                                            (128, 49152, 2, 128), (64, 49152, 3, 128), (33, 49168, 4, 64),
                                            (48, 49168, 2, 128), (40, 49152, 4, 128), (48, 34832, 4, 128),
                                            (64, 34816, 3, 64)])
def test_qlinear_eight_wavefront_groups(M, N, bits, group):
    """256-column groups of eight wavefronts sharing one x ring (the plan for wide
    launches from M = 33, and from M = 48 where the groups cover only half the CUs:
    64-row tiles up to M = 64, 128-row ones above), including a last group with a
    single 16-column tile (N % 256 = 16): every output against the oracle."""
    K = 384
    plan = ss.subspec_qlinear_plan(M, N, K, bits, group)
    assert plan["mfma_rows"] == 32 and plan["waves"] == 8 and plan["col_groups"] == -(-N // 256), plan
    assert plan["rows"] == (64 if M <= 64 else 128), plan
    w = _w(N, K, 320, M, N, bits, group)
    p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
    q, s16, z16 = oracle.quantize_minmax(w, bits, group)
    x = synth.activations(M, K, 321, M, N, bits)
    y = run_qlinear(p, x.to(DEV))
    y_ref = oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, group)
    assert_close(bf16_to_f64(y), y_ref, f"eight wavefronts M={M} N={N} bits={bits} g={group}")


@pytest.mark.parametrize("M,N,K,bits,group", [(128, 528, 16384, 3, 128), (65, 1040, 16512, 4, 64),
                                              (100, 512, 16512, 2, 128), (33, 1040, 16384, 4, 128),
                                              (64, 528, 16512, 3, 64), (48, 512, 16384, 2, 128)])
def test_qlinear_two_teams(M, N, K, bits, group):
    """Long-K launches (at least 128 k-blocks) on two teams of four wavefronts per
    workgroup, each team on one half of the workgroup's k-blocks (uneven halves when
    the count is odd), summed through LDS, on 64-row tiles up to M = 64 and 128-row
    ones above: every output against the oracle."""
    plan = ss.subspec_qlinear_plan(M, N, K, bits, group)
    assert plan["mfma_rows"] == 32 and plan["teams"] == 2 and plan["waves"] == 8, plan
    assert plan["rows"] == (64 if M <= 64 else 128), plan
    w = _w(N, K, 330, M, N, K, bits, group)
    p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
    q, s16, z16 = oracle.quantize_minmax(w, bits, group)
    x = synth.activations(M, K, 331, M, N, K)
    ss.subspec_reserve(plan["workspace_bytes"])
    for _ in range(2):  # the completion counters must be back at zero for the second call
        y = run_qlinear(p, x.to(DEV))
        y_ref = oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, group)
        assert_close(bf16_to_f64(y), y_ref, f"two teams M={M} N={N} K={K} bits={bits} g={group} plan={plan}")


@pytest.mark.parametrize("M,N,K,bits,group", [(40, 128, 16384, 3, 128), (100, 128, 16384, 4, 64),
                                              (64, 160, 16384, 2, 128)])
def test_qlinear_two_teams_one_block_splits(M, N, K, bits, group):
    """Two teams on splits of a single k-block: team 0 takes the block and team 1 none
    (it loads in-range blocks it never uses and hands zeros to team 0), on 64- and
    128-row tiles, with a last column group of one 32-column block (N = 160): every
    output against the oracle, twice, for the completion counters."""
    plan = ss.subspec_qlinear_plan(M, N, K, bits, group)
    assert plan["teams"] == 2 and plan["blocks_per_split"] == 1 and plan["splits"] == K // 128, plan
    w = _w(N, K, 360, M, N, bits, group)
    p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
    q, s16, z16 = oracle.quantize_minmax(w, bits, group)
    x = synth.activations(M, K, 361, M, N)
    ss.subspec_reserve(plan["workspace_bytes"])
    for _ in range(2):
        y = run_qlinear(p, x.to(DEV))
        y_ref = oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, group)
        assert_close(bf16_to_f64(y), y_ref, f"one-block team splits M={M} N={N} bits={bits} g={group} plan={plan}")


@pytest.mark.parametrize("M,N,K,bits,group", [(33, 1040, 3584, 4, 128), (64, 1040, 3584, 3, 128),
                                              (100, 528, 5120, 2, 64), (128, 1040, 2560, 3, 64),
                                              (65, 4624, 3584, 4, 64)])
def test_qlinear_row_blocks(M, N, K, bits, group):
    """Short 16x16x32 launches from M = 33 run their rows in two blocks along grid y,
    each with its own partial sums and completion counters (the second block holding
    M - rows rows, down to one): every output against the oracle, twice, so that the
    counters of both blocks must be back at zero for the second call."""
    plan = ss.subspec_qlinear_plan(M, N, K, bits, group)
    assert plan["mfma_rows"] == 16 and plan["row_blocks"] == 2 and plan["splits"] > 1, plan
    w = _w(N, K, 350, M, N, K, bits, group)
    p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
    q, s16, z16 = oracle.quantize_minmax(w, bits, group)
    x = synth.activations(M, K, 351, M, N, K)
    ss.subspec_reserve(plan["workspace_bytes"])
    for _ in range(2):
        y = run_qlinear(p, x.to(DEV))
        y_ref = oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, group)
        assert_close(bf16_to_f64(y), y_ref, f"row blocks M={M} N={N} K={K} bits={bits} g={group} plan={plan}")


@pytest.mark.parametrize("bits,group", [(3, 128), (4, 64), (2, 128)])
def test_qlinear_single_block_k(bits, group):
    """K = 128: every split is one k-block starting at block 0, the case in which the
    32x32 kernel's refill of its second ring slot would ask for the sums of group -1
    (held at 0, never used); all three paths against the oracle."""
    N, K = 1040, 128
    w = _w(N, K, 340, bits, group)
    p = device_projection(torch.from_numpy(w).to(DEV), bits, group)
    q, s16, z16 = oracle.quantize_minmax(w, bits, group)
    for path, ms in ((ss.SUBSPEC_PATH_GEMV, (1, 5)), (ss.SUBSPEC_PATH_MFMA16, (3, 64)),
                     (ss.SUBSPEC_PATH_MFMA32, (17, 100, 128))):
        for M in ms:
            x = synth.activations(M, K, 341, M, bits)
            y = run_qlinear(p, x.to(DEV), path)
            y_ref = oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, group)
            assert_close(bf16_to_f64(y), y_ref, f"K=128 bits={bits} g={group} path={path} M={M}")


@pytest.mark.parametrize("path", [ss.SUBSPEC_PATH_GEMV, ss.SUBSPEC_PATH_MFMA16, ss.SUBSPEC_PATH_MFMA32])
def test_qlinear_exact_integer_case(path):
    # s=1, z=0, codes in {0,1}, x in {-1,0,1}: every partial sum is a small integer,
    # so the GPU result must equal the oracle bit for bit.
    M, N, K = (4 if path == ss.SUBSPEC_PATH_GEMV else 32), 64, 256
    rng = np.random.default_rng(5)
    codes = rng.integers(0, 2, (N, K)).astype(np.uint8)
    xi = rng.integers(-1, 2, (M, K)).astype(np.float32)
    qw = torch.empty(ss.subspec_qpack_bytes(4, N, K), dtype=torch.uint8, device=DEV)
    ss.subspec_qpack(torch.from_numpy(codes).to(DEV), 4, N, K, qw)
    sc = torch.ones((K // 128, N), dtype=torch.float16, device=DEV)
    zr = torch.zeros((K // 128, N), dtype=torch.float16, device=DEV)
    x = torch.from_numpy(xi).to(torch.bfloat16)
    y = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    ss.subspec_qlinear_path(x.to(DEV), qw, sc, zr, 4, 128, M, N, K, y, path)
    y_ref = oracle.qlinear_ref(synth.bf16_bits(x), codes, sc.cpu().numpy(), zr.cpu().numpy(), 128)
    assert np.array_equal(bf16_to_f64(y), y_ref)


def test_qlinear_deterministic():
    N, K = 1040, 1152
    w = _w(N, K, 400)
    p = device_projection(torch.from_numpy(w).to(DEV), 3, 128)
    for path, M in [(ss.SUBSPEC_PATH_GEMV, 5), (ss.SUBSPEC_PATH_MFMA16, 40), (ss.SUBSPEC_PATH_MFMA32, 100)]:
        x = synth.activations(M, K, 401, M).to(DEV)
        y1 = run_qlinear(p, x, path)
        y2 = run_qlinear(p, x, path)
        assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


def test_qlinear_outlier_activations():
    # 1% of the input channels scaled by 20 (the aggressive 2-bit workload's inputs)
    N, K = 512, 1280
    w = _w(N, K, 500)
    p = device_projection(torch.from_numpy(w).to(DEV), 2, 64)
    q, s16, z16 = oracle.quantize_minmax(w, 2, 64)
    for M in (4, 128):
        x = synth.activations(M, K, 501, outlier_frac=0.01)
        y = run_qlinear(p, x.to(DEV))
        y_ref = oracle.qlinear_ref(synth.bf16_bits(x), q, s16, z16, 64)
        assert_close(bf16_to_f64(y), y_ref, f"outliers M={M}")


def test_qlinear_does_not_touch_outside_y():
    N, K, M = 512, 256, 3
    w = _w(N, K, 600)
    p = device_projection(torch.from_numpy(w).to(DEV), 4, 64)
    x = synth.activations(M, K, 601).to(DEV)
    guard = torch.full((M * N + 2 * 4096,), -7, dtype=torch.int16, device=DEV)
    y = guard[4096:4096 + M * N].view(torch.bfloat16).view(M, N)
    for path in (ss.SUBSPEC_PATH_GEMV, ss.SUBSPEC_PATH_MFMA16, ss.SUBSPEC_PATH_MFMA32):
        ss.subspec_qlinear_path(x, p["qweight"], p["scales"], p["zeros"], 4, 64, M, N, K, y, path)
        torch.cuda.synchronize()
        assert torch.all(guard[:4096] == -7) and torch.all(guard[4096 + M * N:] == -7)
