"""CPU-only checks of the native library: it loads, exports every entry point the
header declares, validates arguments, plans launches, and its host packer writes
the specified layout (pinned against hand-derived bytes and the oracle's reader)."""
import os
import re

import numpy as np
import pytest

import oracle
import paper_2509_18344_amd as ss
from paper_2509_18344_amd import _binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    lib = ss.load_library()
    header = open(os.path.join(ROOT, "include", "subspec.h")).read()
    names = set(re.findall(r"\b(subspec_[a-z_0-9]+)\s*\(", header))
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n


def test_qpack_bytes():
    assert ss.subspec_qpack_bytes(4, 512, 256) == 512 * 256 // 2
    assert ss.subspec_qpack_bytes(3, 16, 128) == 768
    assert ss.subspec_qpack_bytes(2, 32, 256) == 2048
    assert ss.subspec_qpack_bytes(5, 16, 128) == 0
    assert ss.subspec_qpack_bytes(4, 8, 128) == 0
    assert ss.subspec_qpack_bytes(4, 16, 100) == 0


def _golden_rows(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "unpack_bytes.txt")) as f:
        for ln in f:
            if ln.strip() and not ln.startswith("#"):
                rows.append(ln.split())
    return rows


def test_host_packer_matches_golden_bytes(golden_dir):
    rows = _golden_rows(golden_dir)
    for bits in (2, 3, 4):
        codes = np.zeros((16, 128), np.uint8)
        expect = np.zeros(256 * bits, np.uint8)
        for b, n, k, q, off, val in rows:
            if int(b) != bits:
                continue
            codes[int(n), int(k)] = int(q)
            expect[int(off)] |= int(val, 16)
        out = np.zeros(256 * bits, np.uint8)
        ss.subspec_qpack_host(codes, bits, 16, 128, out)
        assert np.array_equal(out, expect), bits


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_host_packer_round_trip_exhaustive(bits):
    # every code value at every position of a tile, plus a random multi-tile matrix
    N, K = 16, 128
    for v in range(2 ** bits):
        codes = np.full((N, K), v, np.uint8)
        out = np.zeros(N * K * bits // 8, np.uint8)
        ss.subspec_qpack_host(codes, bits, N, K, out)
        assert np.array_equal(oracle.unpack(out, bits, N, K), codes)
    rng = np.random.default_rng(bits)
    for N, K in [(16, 128), (48, 384), (32, 1024)]:
        codes = rng.integers(0, 2 ** bits, (N, K)).astype(np.uint8)
        out = np.zeros(N * K * bits // 8, np.uint8)
        ss.subspec_qpack_host(codes, bits, N, K, out)
        assert np.array_equal(oracle.unpack(out, bits, N, K), codes)


@pytest.mark.parametrize("M,N,K,bits,group,path,err", [
    (1, 512, 256, 5, 64, 0, "EUNSUPPORTED"),
    (1, 512, 256, 4, 32, 0, "EUNSUPPORTED"),
    (1, 512, 200, 4, 64, 0, "EUNSUPPORTED"),
    (1, 520, 256, 4, 64, 0, "EUNSUPPORTED"),
    (0, 512, 256, 4, 64, 0, "EUNSUPPORTED"),
    (129, 512, 256, 4, 64, 0, "EUNSUPPORTED"),
    (9, 512, 256, 4, 64, 1, "EUNSUPPORTED"),
    (4, 512, 256, 4, 64, 7, "EINVAL"),
    (4, -16, 256, 4, 64, 0, "EINVAL"),
    (4, 1 << 20, 1 << 13, 4, 64, 0, "EUNSUPPORTED"),   # N*K > 2^32
    (4, 16, (1 << 24) + 128, 4, 64, 0, "EUNSUPPORTED"),  # K > 2^24
])
def test_plan_rejects_bad_shapes(M, N, K, bits, group, path, err):
    with pytest.raises(ss.SubspecError) as ei:
        ss.subspec_qlinear_plan(M, N, K, bits, group, path)
    assert err in str(ei.value)


def test_plan_choices_are_consistent():
    for M in (1, 2, 3, 4, 5, 8, 9, 16, 17, 32, 33, 64, 65, 100, 128):
        for (N, K) in [(512, 256), (18944, 3584), (3584, 18944), (55296, 5120), (5120, 27648), (7168, 5120)]:
            for bits, group in [(4, 128), (3, 128), (2, 64), (4, 64)]:
                p = ss.subspec_qlinear_plan(M, N, K, bits, group)
                rb = p["row_blocks"]
                # row blocks: 16x16x32 tiles only, each block holding at least one row
                assert rb == 1 or (rb == 2 and p["mfma_rows"] == 16 and p["full_groups"] == 0), p
                assert p["rows"] * rb >= M > p["rows"] * (rb - 1)
                KB = K // 128
                assert p["splits"] >= 1 and p["blocks_per_split"] % p["chunk_blocks"] == 0
                assert (p["splits"] - 1) * p["blocks_per_split"] < KB <= p["splits"] * p["blocks_per_split"]
                # teams split a workgroup's k-blocks (32x32 tiles only); a layout
                # mismatch between the binding and the C struct would show here
                assert p["teams"] == 1 or (p["teams"] == 2 and p["mfma_rows"] == 32 and p["waves"] == 8), p
                cols = p["waves"] // p["teams"] * p["tiles_per_wave"] * 16
                assert p["col_groups"] == -(-N // cols)
                fg = p["full_groups"]
                assert 0 <= fg < p["col_groups"]
                assert p["grid"] == fg + (p["col_groups"] - fg) * p["splits"]
                if fg:
                    # whole groups on a multiple of the CUs; the rest split at most
                    # once per CU
                    assert p["splits"] > 1 and fg % 256 == 0
                    assert (p["col_groups"] - fg) * p["splits"] <= 256
                # completion counters (16384 x 4 bytes), the per-group sums of x the
                # 32x32 kernel reads (fp32 [M][K/group], 256-byte aligned), then the
                # splits' fp32 partial sums
                xs = -(-M * (K // group) * 4 // 256) * 256 if p["mfma_rows"] == 32 else 0
                part_rows = 2 * p["rows"] if rb == 2 else M
                partials = p["splits"] * part_rows * N * 4 if p["splits"] > 1 else 0
                expect = 65536 + xs + partials if (xs or partials) else 0
                assert p["workspace_bytes"] == expect, (M, N, K, bits, group, p)
    # 592 column groups on 256 CUs: 512 whole, the last 80 split three ways
    p = ss.subspec_qlinear_plan(1, 37888, 3584, 4, 128)
    assert (p["col_groups"], p["full_groups"], p["splits"], p["grid"]) == (592, 512, 3, 752)
    # automatic plan: GEMV only for one row (measured crossover), MFMA from M = 2
    assert ss.subspec_qlinear_plan(1, 512, 256, 4, 64)["path"] == ss.SUBSPEC_PATH_GEMV
    assert ss.subspec_qlinear_plan(2, 512, 256, 4, 64)["path"] == ss.SUBSPEC_PATH_MFMA
    assert ss.subspec_qlinear_plan(8, 512, 256, 4, 64, ss.SUBSPEC_PATH_GEMV)["path"] == ss.SUBSPEC_PATH_GEMV
    assert ss.subspec_qlinear_plan(8, 512, 256, 4, 64, ss.SUBSPEC_PATH_MFMA)["path"] == ss.SUBSPEC_PATH_MFMA


def test_mfma_tile_shape_choice():
    """The automatic plan runs 32x32x16 tiles (128 rows) only above M = 64, on launches
    that fill the 256 CUs with whole 128-column groups (two-chunk ring) or split a K of
    at least 192 blocks (four-chunk ring); everything else stays on 16x16x32 tiles.
    Where 256-column groups still cover three quarters of the CUs and K is not split,
    eight wavefronts share a four-chunk ring (if that variant is built for the bit
    width and group), and from M = 33 such launches take 64-row 32x32x16 tiles too.
    Launches whose K spans at least 128 blocks take two teams of four wavefronts per
    workgroup from M = 33 (64-row tiles up to M = 64; the last tuple entry is then minus
    the wavefronts of one team)."""
    def shape(M, N, K, bits=3, group=128, path=ss.SUBSPEC_PATH_AUTO):
        p = ss.subspec_qlinear_plan(M, N, K, bits, group, path)
        return p["mfma_rows"], p["rows"], p["ring_chunks"], p["waves"] // p["teams"] * (1 if p["teams"] == 1 else -1)
    assert shape(128, 55296, 5120) == (32, 128, 4, 8)      # 32B gate|up
    assert shape(128, 55296, 5120, 2, 64) == (32, 128, 4, 8)
    assert shape(128, 55296, 5120, 4, 128) == (32, 128, 2, 4)  # no eight-wavefront 4-bit build
    assert shape(96, 37888, 3584, 4) == (32, 128, 2, 4)     # 7B gate|up: 148 groups of 256
    assert shape(128, 5120, 27648) == (32, 128, 2, -4)     # 32B down: two teams of four
    assert shape(96, 3584, 18944, 4) == (32, 128, 2, -4)   # 7B down
    assert shape(128, 7168, 5120)[0] == 16           # 32B q|k|v
    assert shape(64, 55296, 5120) == (32, 64, 4, 8)        # 32B gate|up, 64-row tiles
    assert shape(33, 55296, 5120, 2, 64) == (32, 64, 4, 8)
    assert shape(48, 55296, 5120, 4, 128) == (32, 64, 4, 8)
    assert shape(32, 55296, 5120)[0] == 16
    assert shape(64, 37888, 3584, 4) == (32, 64, 4, 8)     # 7B gate|up: half-wide, from M = 48
    assert shape(48, 37888, 3584, 4) == (32, 64, 4, 8)
    assert shape(40, 37888, 3584, 4)[0] == 16
    assert shape(64, 5120, 27648) == (32, 64, 2, -4)       # long K: 64-row tiles on two teams
    assert shape(33, 3584, 18944, 4) == (32, 64, 2, -4)
    assert shape(32, 5120, 27648)[0] == 16
    assert shape(64, 7168, 5120)[0] == 16                  # q|k|v
    assert shape(17, 512, 256, path=ss.SUBSPEC_PATH_MFMA32) == (32, 128, 4, 4)
    # 16x16x32 launches whose column groups number fewer than the CUs, with K under
    # 128 blocks, run their rows in two blocks from M = 33 (q|k|v, o); long-K, wide
    # and M <= 32 launches keep one block
    def blocks(M, N, K, bits=3, group=128):
        p = ss.subspec_qlinear_plan(M, N, K, bits, group)
        return p["row_blocks"], p["rows"]
    assert blocks(64, 7168, 5120) == (2, 32)              # 32B q|k|v
    assert blocks(128, 5120, 5120) == (2, 64)             # 32B o
    assert blocks(33, 4608, 3584, 4) == (2, 32)           # 7B q|k|v
    assert blocks(100, 3584, 3584, 4) == (2, 64)          # 7B o
    assert blocks(32, 7168, 5120) == (1, 32)
    assert blocks(64, 5120, 27648) == (1, 64)             # long K
    assert blocks(64, 3584, 18944, 4) == (1, 64)
    assert blocks(40, 37888, 3584, 4) == (1, 64)          # 592 column groups
    assert shape(128, 55296, 5120, path=ss.SUBSPEC_PATH_MFMA16)[0] == 16
    for path in (ss.SUBSPEC_PATH_MFMA16, ss.SUBSPEC_PATH_MFMA32):
        assert ss.subspec_qlinear_plan(40, 512, 256, 4, 64, path)["path"] == ss.SUBSPEC_PATH_MFMA


def test_gemv_plan_refuses_splits_longer_than_its_staging():
    # At 8 rows a GEMV split stages at most 2048 k of x.  With more than 16384 column
    # groups (N > 2^20) the plan cannot split K (one completion counter per group), so
    # K = 2560 would leave 512 k unstaged: refused, never silently wrong.
    N = (1 << 20) + 64
    with pytest.raises(ss.SubspecError, match="EUNSUPPORTED"):
        ss.subspec_qlinear_plan(8, N, 2560, 4, 128, ss.SUBSPEC_PATH_GEMV)
    assert "GEMV" in ss.subspec_last_error()
    # the same shape with K inside one staged span, and the MFMA path, still plan
    p = ss.subspec_qlinear_plan(8, N, 2048, 4, 128, ss.SUBSPEC_PATH_GEMV)
    assert p["splits"] == 1
    assert ss.subspec_qlinear_plan(8, N, 2560, 4, 128, ss.SUBSPEC_PATH_MFMA)["splits"] >= 1
    # below the counter limit the plan splits K instead
    p = ss.subspec_qlinear_plan(8, 65536, 8192, 4, 128, ss.SUBSPEC_PATH_GEMV)
    assert p["splits"] * p["blocks_per_split"] * 128 >= 8192 and p["blocks_per_split"] * 128 <= 2048


def test_noalloc_refuses_shapes_beyond_its_fixed_scratch():
    # 32x32 kernel at M = 128 over K = 4325376 with groups of 64: the sums of x alone
    # (128 x 67584 fp32) exceed the 32 MiB array, so even an unsplit plan cannot fit;
    # the call is refused while planning, before any GPU work
    assert ss.SUBSPEC_NOALLOC_SCRATCH_BYTES == 32 << 20
    with pytest.raises(ss.SubspecError, match="EUNSUPPORTED"):
        ss.subspec_qlinear_noalloc(16, 16, 16, 16, 4, 64, 128, 256, 4325376, 16, stream=0)
    assert "scratch" in ss.subspec_last_error()


def test_qlinear_argument_errors_need_no_gpu():
    with pytest.raises(ss.SubspecError) as ei:
        ss.subspec_qlinear(None, 16, 16, 16, 4, 64, 1, 512, 256, 16, stream=0)
    assert "EINVAL" in str(ei.value) and "null" in ss.subspec_last_error()
    with pytest.raises(ss.SubspecError) as ei:
        ss.subspec_qlinear(16, 16, 16, 24, 4, 64, 1, 512, 256, 16, stream=0)
    assert "aligned" in ss.subspec_last_error()
    with pytest.raises(ss.SubspecError):
        ss.subspec_qlinear_path(16, 16, 16, 16, 4, 64, 9, 512, 256, 16, ss.SUBSPEC_PATH_GEMV, stream=0)
    with pytest.raises(ss.SubspecError):
        ss.subspec_quantize(16, 4, 64, 16, 100, 16, 16, 16, stream=0)


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_binding, "_lib", None)
    monkeypatch.setattr(_binding, "_HERE", str(tmp_path))
    with pytest.raises(RuntimeError, match="missing"):
        _binding.load_library()


def test_tree_expand_argument_errors_need_no_gpu():
    # (R, V, k, T): rejected before any GPU work
    for R, V, k, T, err in [(0, 64, 1, 0.2, "EUNSUPPORTED"), (1025, 64, 1, 0.2, "EUNSUPPORTED"),
                            (2, 100, 1, 0.2, "EUNSUPPORTED"), (2, 64, 0, 0.2, "EUNSUPPORTED"),
                            (2, 64, 33, 0.2, "EUNSUPPORTED"), (1, 8, 9, 0.2, "EUNSUPPORTED"),
                            (2, 64, 4, 0.0, "EINVAL"), (2, 64, 4, -1.0, "EINVAL"),
                            (1000, 1 << 22, 4, 0.2, "EUNSUPPORTED")]:
        with pytest.raises(ss.SubspecError) as ei:
            ss.subspec_tree_expand(16, 16, R, V, T, k, 16, 16, 16, stream=0)
        assert err in str(ei.value), (R, V, k, T)
    with pytest.raises(ss.SubspecError):
        ss.subspec_tree_expand(None, 16, 2, 64, 0.2, 4, 16, 16, 16, stream=0)
    with pytest.raises(ss.SubspecError):
        ss.subspec_tree_expand(24, 16, 2, 64, 0.2, 4, 16, 16, 16, stream=0)
    assert ss.subspec_tree_workspace_bytes(6, 152064, 6) > 65536
    assert ss.subspec_tree_workspace_bytes(6, 100, 6) == 0


def test_tree_plan_shapes():
    # about 512 workgroups, each at least 2048 logits (one 16-byte load per thread)
    # unless the row is shorter; slices are multiples of 8 and cover the row
    assert ss.subspec_tree_plan(6, 152064, 6) == (75, 2032, 8)
    assert ss.subspec_tree_plan(64, 152064, 6) == (8, 19008, 8)
    assert ss.subspec_tree_plan(1, 152064, 6) == (75, 2032, 8)
    assert ss.subspec_tree_plan(1024, 64, 32) == (1, 64, 32)
    assert ss.subspec_tree_plan(37, 4096, 17) == (2, 2048, 32)
    assert ss.subspec_tree_plan(3, 2048, 9)[2] == 16
    for R, V, k in [(1, 8, 1), (6, 1000, 6), (128, 152064, 6), (1000, 2048, 32), (7, 152064, 16)]:
        c, n, _ = ss.subspec_tree_plan(R, V, k)
        assert n % 8 == 0 and (c - 1) * n < V <= c * n and R * c <= 1024, (R, V, k)
    for R, V, k in [(0, 64, 1), (2, 100, 1), (2, 64, 33), (1, 8, 9)]:
        with pytest.raises(ss.SubspecError, match="EUNSUPPORTED"):
            ss.subspec_tree_plan(R, V, k)


def test_tree_attention_plan_and_errors_need_no_gpu():
    # Qwen2.5-7B at the last pass of a depth-48 tree: 2336 keys = 73 tiles of 32,
    # three tiles per range
    assert ss.subspec_tree_attention_plan(6, 28, 4, 2048, 282) == (25, 3)
    for M, Hq, Hkv, P, T in [(6, 28, 4, 0, 0), (1, 1, 1, 0, 0), (6, 40, 8, 30000, 282), (8, 16, 2, 33, 7)]:
        s, t = ss.subspec_tree_attention_plan(M, Hq, Hkv, P, T)
        tiles = -(-(P + T + M) // 32)
        assert t >= 1 and (s - 1) * t < tiles <= s * t, (M, Hq, Hkv, P, T)
        rows_pad = 16 * -(-(Hq // Hkv * M) // 16)
        # the split-K completion counters (64 KiB) stay in front of the partials
        assert ss.subspec_tree_attention_workspace_bytes(M, Hq, Hkv, P, T) == \
            65536 + Hkv * s * rows_pad * (128 + 2) * 4
    for M, Hq, Hkv, P, T in [(6, 30, 4, 10, 0), (0, 28, 4, 10, 0), (10, 28, 4, 10, 0), (6, 28, 4, -1, 0),
                             (64, 1, 1, 0, 1100), (6, 4, 0, 10, 0)]:
        with pytest.raises(ss.SubspecError, match="EUNSUPPORTED"):
            ss.subspec_tree_attention_plan(M, Hq, Hkv, P, T)
        assert ss.subspec_tree_attention_workspace_bytes(M, Hq, Hkv, P, T) == 0
    args = dict(M=6, Hq=28, Hkv=4, S=2400, P=2048, T=282, scale=0.088)

    def call(q=16, kc=16, vc=16, kn=16, vn=16, mask=16, out=16, **kw):
        a = dict(args, **kw)
        return ss.subspec_tree_attention(q, kc, vc, kn, vn, mask, a["M"], a["Hq"], a["Hkv"], a["S"], a["P"],
                                         a["T"], a["scale"], out, stream=0)
    with pytest.raises(ss.SubspecError, match="EINVAL"):
        call(q=None)
    with pytest.raises(ss.SubspecError, match="EINVAL"):
        call(kc=24)
    with pytest.raises(ss.SubspecError, match="EINVAL"):
        call(mask=18)
    with pytest.raises(ss.SubspecError, match="EUNSUPPORTED"):
        call(S=2335)
    with pytest.raises(ss.SubspecError, match="EINVAL"):
        call(scale=float("inf"))


def test_prefetch_argument_errors_need_no_gpu():
    for slot_bytes, slots in [(0, 2), (1024, 1), (1024, 65)]:
        with pytest.raises(ss.SubspecError, match="EINVAL"):
            ss.Prefetcher(slot_bytes, slots)
    lib = ss.load_library()
    import ctypes
    t = ctypes.c_longlong()
    p = ctypes.c_void_p()
    assert lib.subspec_prefetch_begin(None, None, 16, ctypes.byref(t)) == -1  # SUBSPEC_EINVAL
    assert lib.subspec_prefetch_acquire(None, 0, None, ctypes.byref(p)) == -1  # SUBSPEC_EINVAL
    assert lib.subspec_prefetch_release(None, 0, None) == -1  # SUBSPEC_EINVAL
    assert lib.subspec_prefetch_destroy(None) == -1  # SUBSPEC_EINVAL
    assert lib.subspec_prefetch_create(16, 2, None) == -1  # SUBSPEC_EINVAL


def test_quantize_hqq_argument_errors_need_no_gpu():
    with pytest.raises(ss.SubspecError, match="EUNSUPPORTED"):
        ss.subspec_quantize_hqq(16, 5, 64, 16, 128, 16, 16, 16, stream=0)
    with pytest.raises(ss.SubspecError, match="EINVAL"):
        ss.subspec_quantize_hqq(16, 4, 64, 16, 100, 16, 16, 16, stream=0)
    with pytest.raises(ss.SubspecError, match="EINVAL"):
        ss.subspec_quantize_hqq(None, 4, 64, 16, 128, 16, 16, 16, stream=0)
    with pytest.raises(ss.SubspecError, match="EINVAL"):
        ss.subspec_quantize_hqq(16, 4, 64, 16, 128, 24, 16, 16, stream=0)
