"""Pins of the fp64 oracle against facts that do not come from the oracle itself:
hand-derived golden values, closed forms, invariants and exact-rational brute force
(CPU only)."""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

RNG = np.random.default_rng(1234)


def _read_rows(path):
    with open(path) as f:
        return [ln.strip() for ln in f if ln.strip() and not ln.startswith("#")]


# ---------------------------------------------------------------- number formats

def _all_fp16_values():
    bits = np.arange(0x7C00, dtype=np.uint16)  # +0 .. largest finite
    return bits, bits.view(np.float16).astype(np.float64)


def test_fp16_round_is_nearest_even():
    bits, vals = _all_fp16_values()
    samples = np.concatenate([RNG.standard_normal(300) * 0.02, RNG.uniform(0, 16, 300),
                              RNG.uniform(0, 1e-4, 100), vals[1:200] * 1.5,
                              (vals[1000:1100] + vals[1001:1101]) / 2])  # exact ties
    for v in samples:
        a = abs(v)
        i = np.searchsorted(vals, a)
        cands = [j for j in (i - 1, i) if 0 <= j < len(vals)]
        best = min(cands, key=lambda j: (abs(Fraction(vals[j]) - Fraction(a)), int(bits[j]) & 1))
        exp = np.float16(vals[best]) if v >= 0 else -np.float16(vals[best])
        got = oracle.fp16_round(v)
        assert got == exp and np.signbit(got) == np.signbit(exp), v


def test_bf16_round_is_nearest_even():
    xs = np.concatenate([RNG.standard_normal(2000).astype(np.float32),
                         (RNG.standard_normal(200) * 1e-30).astype(np.float32)])
    # exact ties: bf16 value + half an ulp
    base = np.arange(0x3F80, 0x3F80 + 64, dtype=np.uint32) << 16
    ties = (base | 0x8000).view(np.float32)
    xs = np.concatenate([xs, ties])
    got = oracle.bf16_round_bits(xs)
    for x, g in zip(xs, got):
        u = int(np.float32(x).view(np.uint32))
        lo, hi = u >> 16, (u >> 16) + 1
        f = lambda b: Fraction(float(np.uint32(b << 16).view(np.float32)))
        dlo, dhi = abs(f(lo) - Fraction(float(x))), abs(f(hi) - Fraction(float(x)))
        exp = lo if (dlo < dhi or (dlo == dhi and lo % 2 == 0)) else hi
        assert int(g) == exp, x


# ---------------------------------------------------------------- quantizer

def test_quantizer_golden(golden_dir):
    for row in _read_rows(os.path.join(golden_dir, "quant_examples.txt")):
        bits, group, vals, s_hex, z_hex, codes = [c.strip() for c in row.split("|")]
        w = np.array([float(v) for v in vals.split()], dtype=np.float32)[None, :]
        q, s16, z16 = oracle.quantize_minmax(w, int(bits), int(group))
        assert int(s16.view(np.uint16)[0, 0]) == int(s_hex, 16), row
        assert int(z16.view(np.uint16)[0, 0]) == int(z_hex, 16), row
        assert q[0].tolist() == [int(c) for c in codes.split()], row


@pytest.mark.parametrize("bits,group", [(4, 64), (4, 128), (3, 128), (2, 64)])
def test_quantizer_invariants(bits, group):
    N, K = 48, 512
    w = (RNG.standard_normal((N, K)) * 0.02).astype(np.float32)
    q, s16, z16 = oracle.quantize_minmax(w, bits, group)
    qmax = 2 ** bits - 1
    assert q.dtype == np.uint8 and q.shape == (N, K)
    assert s16.shape == (K // group, N) and z16.shape == (K // group, N)
    assert q.max() <= qmax
    deq = oracle.dequant(q, s16, z16, group)
    s_full = np.repeat(s16.astype(np.float64).T, group, axis=1)
    # reconstruction error at most half a step (up to float64 rounding of w/s + z)
    assert np.all(np.abs(w.astype(np.float64) - deq) <= s_full * (0.5 + 1e-12))
    # the group minimum maps to code 0 and the maximum to the top code
    wg = w.reshape(N, K // group, group)
    qg = q.reshape(N, K // group, group)
    idx_min = wg.argmin(axis=2)[..., None]
    idx_max = wg.argmax(axis=2)[..., None]
    assert np.all(np.take_along_axis(qg, idx_min, 2) == 0)
    assert np.all(np.take_along_axis(qg, idx_max, 2) == qmax)
    # idempotent: quantizing the dequantized weights with the same s, z gives q back
    z_full = np.repeat(z16.astype(np.float64).T, group, axis=1)
    q2 = np.clip(np.rint(deq / s_full + z_full), 0, qmax)
    assert np.array_equal(q2, q)


def test_quantizer_edge_groups():
    # all-negative, all-positive, tiny range (an exact fp16-subnormal scale), constant
    rows = [np.linspace(-3.0, -1.0, 64), np.linspace(0.5, 2.0, 64),
            np.tile((np.arange(16) - 5.0) * 2.0 ** -22, 4), np.full(64, -0.75)]
    w = np.array(rows, dtype=np.float32)
    q, s16, z16 = oracle.quantize_minmax(w, 4, 64)
    deq = oracle.dequant(q, s16, z16, 64)
    for r in range(3):
        s = float(s16[0, r])
        assert np.all(np.abs(w[r].astype(np.float64) - deq[r]) <= s * (0.5 + 1e-12)), r
        assert q[r].min() == 0 and q[r].max() == 15, r
    assert s16[0, 2] < np.float16(6.2e-5)  # the scale really is subnormal in fp16
    assert float(s16[0, 3]) == 1.0 and np.all(q[3] == 0) and np.all(deq[3] == -0.75)


# ---------------------------------------------------------------- dequant

def test_dequant_exact_and_canonical_roundings():
    n = 4000
    s_bits = RNG.integers(0x0001, 0x5C00, n).astype(np.uint16)   # incl. subnormals
    z_bits = RNG.integers(0, 0x4C00, n).astype(np.uint16) | (RNG.integers(0, 2, n) << 15).astype(np.uint16)
    q = RNG.integers(0, 16, n).astype(np.uint8)
    s16, z16 = s_bits.view(np.float16)[None, :], z_bits.view(np.float16)[None, :]
    deq = oracle.dequant(q[:, None], s16, z16, 1)[:, 0]
    f32 = oracle.dequant_f32(q[:, None], s16, z16, 1)[:, 0]
    for i in range(n):
        exact = Fraction(float(s16[0, i])) * (int(q[i]) - Fraction(float(z16[0, i])))
        assert Fraction(float(deq[i])) == exact  # no rounding happened in float64
        # float32: nearest float32 to the exact value (brute force over neighbours)
        c = np.float32(float(exact))
        nb = [np.nextafter(c, np.float32(-np.inf)), c, np.nextafter(c, np.float32(np.inf))]
        best = min(nb, key=lambda v: (abs(Fraction(float(v)) - exact), int(np.float32(v).view(np.uint32)) & 1))
        assert f32[i] == best


def test_dequant_special_cases():
    q = np.arange(16, dtype=np.uint8)[None, :].repeat(2, 0)
    s16 = np.array([[1.0, 0.25]], dtype=np.float16)
    z16 = np.array([[0.0, 3.0]], dtype=np.float16)
    deq = oracle.dequant(q, s16, z16, 16)
    assert np.array_equal(deq[0], np.arange(16.0))
    assert np.array_equal(deq[1], 0.25 * (np.arange(16.0) - 3.0))
    bits = oracle.dequant_bf16_bits(q, s16, z16, 16)
    assert np.array_equal(oracle.bf16_bits_to_f64(bits), deq)  # all exactly representable


# ---------------------------------------------------------------- unpack

def test_unpack_golden(golden_dir):
    rows = [list(map(str, r.split())) for r in _read_rows(os.path.join(golden_dir, "unpack_bytes.txt"))]
    for bits in (2, 3, 4):
        sel = [r for r in rows if int(r[0]) == bits]
        buf = np.zeros(256 * bits, dtype=np.uint8)
        expect = np.zeros((16, 128), dtype=np.uint8)
        for _, n, k, q, off, val in sel:
            buf[int(off)] |= int(val, 16)
            expect[int(n), int(k)] = int(q)
        got = oracle.unpack(buf, bits, 16, 128)
        assert np.array_equal(got, expect), bits


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_unpack_is_a_bijection(bits):
    # every code position of a 2x2-tile buffer is read from exactly `bits` distinct bits
    N, K = 32, 256
    nbits = N * K * bits
    base = oracle.unpack(np.zeros(nbits // 8, np.uint8), bits, N, K)
    assert np.all(base == 0)
    hits = np.zeros((N, K), dtype=np.int64)
    for b in range(0, nbits, 7):  # a spread of single set bits
        buf = np.zeros(nbits // 8, np.uint8)
        buf[b // 8] = 1 << (b % 8)
        c = oracle.unpack(buf, bits, N, K)
        nz = np.argwhere(c)
        assert len(nz) == 1, b  # one bit belongs to exactly one code
        v = int(c[tuple(nz[0])])
        assert v & (v - 1) == 0 and v < 2 ** bits  # and is one bit of it
        hits[tuple(nz[0])] += 1
    assert hits.max() <= bits


# ---------------------------------------------------------------- the linear layer

def _bf16_activations(M, K, scale=1.0):
    return oracle.bf16_round_bits((RNG.standard_normal((M, K)) * scale).astype(np.float32))


def test_qlinear_brute_force_fractions():
    M, N, K, G = 3, 16, 128, 64
    w = (RNG.standard_normal((N, K)) * 0.02).astype(np.float32)
    q, s16, z16 = oracle.quantize_minmax(w, 4, G)
    x = _bf16_activations(M, K)
    y = oracle.qlinear_ref(x, q, s16, z16, G)
    xv = oracle.bf16_bits_to_f64(x)
    for m in range(M):
        for n in range(N):
            acc = Fraction(0)
            mag = 0.0
            for k in range(K):
                g = k // G
                wv = Fraction(float(s16[g, n])) * (int(q[n, k]) - Fraction(float(z16[g, n])))
                acc += Fraction(float(xv[m, k])) * wv
                mag += abs(float(xv[m, k]) * float(wv))
            assert abs(Fraction(float(y[m, n])) - acc) <= Fraction(K * mag) * Fraction(2) ** -52


def test_qlinear_one_hot_and_ones():
    N, K, G = 32, 256, 128
    w = (RNG.standard_normal((N, K)) * 0.02).astype(np.float32)
    q, s16, z16 = oracle.quantize_minmax(w, 3, G)
    deq = oracle.dequant(q, s16, z16, G)
    ks = [0, 5, 127, 128, 255]
    x = np.zeros((len(ks), K), dtype=np.float32)
    for i, k in enumerate(ks):
        x[i, k] = 1.0
    y = oracle.qlinear_ref(oracle.bf16_round_bits(x), q, s16, z16, G)
    for i, k in enumerate(ks):
        assert np.array_equal(y[i], deq[:, k])  # orientation: y[., n] = W^[n, k]
    ones = oracle.bf16_round_bits(np.ones((1, K), np.float32))
    y1 = oracle.qlinear_ref(ones, q, s16, z16, G)[0]
    s = s16.astype(np.float64)
    z = z16.astype(np.float64)
    qs = q.astype(np.float64).reshape(N, K // G, G).sum(axis=2).T  # [K/G][N]
    closed = (s * (qs - G * z)).sum(axis=0)
    np.testing.assert_allclose(y1, closed, rtol=1e-13, atol=1e-15)


def test_qlinear_exact_integer_case():
    # s=1, z=0, codes in {0,1}, x in {-1,0,1}: y is a small integer, exactly
    M, N, K = 4, 16, 128
    q = RNG.integers(0, 2, (N, K)).astype(np.uint8)
    xi = RNG.integers(-1, 2, (M, K))
    s16 = np.ones((1, N), np.float16)
    z16 = np.zeros((1, N), np.float16)
    y = oracle.qlinear_ref(oracle.bf16_round_bits(xi.astype(np.float32)), q, s16, z16, 128)
    assert np.array_equal(y, (xi @ q.T.astype(np.int64)).astype(np.float64))


def test_wprec_roundings():
    N, K, G = 16, 128, 64
    w = (RNG.standard_normal((N, K)) * 0.02).astype(np.float32)
    q, s16, z16 = oracle.quantize_minmax(w, 2, G)
    x = _bf16_activations(2, K)
    y_e = oracle.qlinear_ref(x, q, s16, z16, G, "exact")
    y_f = oracle.qlinear_ref(x, q, s16, z16, G, "fp32")
    y_b = oracle.qlinear_ref(x, q, s16, z16, G, "bf16")
    xv = oracle.bf16_bits_to_f64(x)
    wf = oracle.dequant_f32(q, s16, z16, G).astype(np.float64)
    wb = oracle.bf16_bits_to_f64(oracle.dequant_bf16_bits(q, s16, z16, G))
    np.testing.assert_array_equal(y_f, xv @ wf.T)
    np.testing.assert_array_equal(y_b, xv @ wb.T)
    assert np.max(np.abs(y_e - y_f)) < 1e-6 and np.max(np.abs(y_e - y_b)) < 5e-2
