// Weight preparation kernels: min/max quantizer, the quantizer with an HQQ-style
// optimised zero-point, packer into the tile layout and the materialising
// dequantizer (include/subspec.h documents each operation).
#include "device_common.h"
#include "kernels.h"
#include "kernels_hqq.h"

namespace subspec {

// float64 -> IEEE binary16 bits, round to nearest, ties to even, written from the
// format definition: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits,
// subnormals below 2^-14, overflow to infinity.
__device__ __forceinline__ uint16_t f64_to_f16_bits(double d) {
  const uint64_t u = __builtin_bit_cast(uint64_t, d);
  const uint16_t sign = static_cast<uint16_t>((u >> 48) & 0x8000u);
  const int ex = static_cast<int>((u >> 52) & 0x7FF);
  const uint64_t frac = u & ((1ull << 52) - 1);
  if (ex == 0x7FF) return sign | 0x7C00u | (frac ? 0x200u : 0u);  // inf / NaN
  if (ex == 0) return sign;                   // float64 zero or subnormal: |d| < 2^-1022
  const int e = ex - 1023;                    // d = 1.frac * 2^e
  if (e > 15) return sign | 0x7C00u;          // >= 2^16: overflow
  if (e < -25) return sign;                   // < 2^-25: rounds to zero
  const uint64_t sig = (1ull << 52) | frac;   // 53-bit significand
  // Keep 11 bits for normal results; fewer for subnormal ones (quantum 2^-24).
  const int shift = (e >= -14) ? 42 : 42 + (-14 - e);
  uint64_t m = sig >> shift;
  const uint64_t rem = sig & ((1ull << shift) - 1);
  const uint64_t half = 1ull << (shift - 1);
  if (rem > half || (rem == half && (m & 1))) ++m;
  if (e >= -14) {
    // m in [2^10, 2^11]; a carry to 2^11 bumps the exponent (and may reach inf).
    return sign | static_cast<uint16_t>(((e + 15 - 1) << 10) + m);
  }
  return sign | static_cast<uint16_t>(m);     // subnormal (m == 2^10 is the min normal)
}

__device__ __forceinline__ double f16_bits_to_f64(uint16_t h) {
  return static_cast<double>(__builtin_bit_cast(_Float16, h));
}

// One wavefront per (column n, group g).  Lane l holds GROUP/64 consecutive values.
template <int GROUP>
__global__ __launch_bounds__(256) void k_quantize(const float* __restrict__ w, int bits,
                                                  int N, int K, uint8_t* __restrict__ codes,
                                                  uint16_t* __restrict__ sc,
                                                  uint16_t* __restrict__ zr) {
  constexpr int PER = GROUP / kWave;
  const int gpr = K / GROUP;
  const long long gid = static_cast<long long>(blockIdx.x) * 4 + threadIdx.x / kWave;
  if (gid >= static_cast<long long>(N) * gpr) return;  // whole wavefronts exit together
  const int lane = threadIdx.x % kWave;
  const long long n = gid / gpr;
  const int g = static_cast<int>(gid % gpr);
  const float* src = w + n * K + static_cast<long long>(g) * GROUP + lane * PER;
  float v[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) v[i] = src[i];
  float mn = v[0], mx = v[0];
#pragma unroll
  for (int i = 1; i < PER; ++i) { mn = fminf(mn, v[i]); mx = fmaxf(mx, v[i]); }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    mn = fminf(mn, __shfl_xor(mn, off));
    mx = fmaxf(mx, __shfl_xor(mx, off));
  }
  const double wmin = mn, wmax = mx;
  const double qmax = static_cast<double>((1 << bits) - 1);
  uint16_t s16 = f64_to_f16_bits((wmax - wmin) / qmax);
  double s = f16_bits_to_f64(s16);
  const bool degenerate = (wmax == wmin) || (s == 0.0);
  uint16_t z16;
  if (degenerate) {
    s16 = 0x3C00u;
    s = 1.0;
    z16 = f64_to_f16_bits(-wmin);
  } else {
    z16 = f64_to_f16_bits(-wmin / s);
  }
  const double z = f16_bits_to_f64(z16);
  uint8_t* dst = codes + n * K + static_cast<long long>(g) * GROUP + lane * PER;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    double t = static_cast<double>(v[i]) / s + z;
    t = __builtin_rint(t);
    t = t < 0.0 ? 0.0 : (t > qmax ? qmax : t);
    dst[i] = degenerate ? 0 : static_cast<uint8_t>(t);
  }
  if (lane == 0) {
    sc[static_cast<long long>(g) * N + n] = s16;
    zr[static_cast<long long>(g) * N + n] = z16;
  }
}

// HQQ-style zero-point (SubSpec Sec. 4.1 and 5.1 quantize the substitutes with HQQ;
// the rounds follow the cited half-quadratic quantization work).  The scale is the
// min/max scale; starting from the min/max zero, each round quantizes with the
// current zero, shrinks the residual x = w - s (q - z) with the generalised soft
// threshold sign(x) max(|x| - |x|^(p-1) / beta, 0) and refits the zero as the mean of
// q - (w - e) / s; the group's sum of |w - s (q - z)| decides: the best zero is kept
// and a round without improvement ends the search; beta grows by kappa per round.
// The best zero, rounded to fp16, replaces the min/max zero only if it is still
// better in fp16.  Everything in float64 with sums in index order, one thread per
// (column n, group g), so that the rounding decisions are reproducible.
constexpr double kHqqP = 0.7;
constexpr double kHqqBeta = 10.0;
constexpr double kHqqKappa = 1.01;
constexpr int kHqqIters = 20;

// The group's weights sit in LDS, transposed (element i of thread t at [i][t]), so
// the rounds index them without spilling registers and without bank conflicts.
template <int GROUP>
__global__ __launch_bounds__(kWave) void k_quantize_hqq(const float* __restrict__ w, int bits, int N, int K,
                                                       uint8_t* __restrict__ codes, uint16_t* __restrict__ sc,
                                                       uint16_t* __restrict__ zr) {
  __shared__ float wl[GROUP][kWave];
  const int t = threadIdx.x;
  const int gpr = K / GROUP;
  const long long gid = static_cast<long long>(blockIdx.x) * kWave + t;  // g * N + n
  if (gid >= static_cast<long long>(N) * gpr) return;  // no barrier follows
  const long long n = gid % N;
  const int g = static_cast<int>(gid / N);
  const float* src = w + n * K + static_cast<long long>(g) * GROUP;
  float mn = INFINITY, mx = -INFINITY;
  for (int i = 0; i < GROUP; i += 4) {
    const float4 q4 = *reinterpret_cast<const float4*>(src + i);
    wl[i][t] = q4.x;
    wl[i + 1][t] = q4.y;
    wl[i + 2][t] = q4.z;
    wl[i + 3][t] = q4.w;
    mn = fminf(fminf(mn, q4.x), fminf(fminf(q4.y, q4.z), q4.w));
    mx = fmaxf(fmaxf(mx, q4.x), fmaxf(fmaxf(q4.y, q4.z), q4.w));
  }
  const double wmin = mn, wmax = mx;
  const double qmax = static_cast<double>((1 << bits) - 1);
  uint16_t s16 = f64_to_f16_bits((wmax - wmin) / qmax);
  double s = f16_bits_to_f64(s16);
  const bool degenerate = (wmax == wmin) || (s == 0.0);
  uint16_t z16;
  if (degenerate) {
    s16 = 0x3C00u;
    s = 1.0;
    z16 = f64_to_f16_bits(-wmin);
  } else {
    z16 = f64_to_f16_bits(-wmin / s);
  }
  auto code = [&](double x, double z) __attribute__((always_inline)) {
    const double c = __builtin_rint(x / s + z);
    return c < 0.0 ? 0.0 : (c > qmax ? qmax : c);
  };
  auto l1 = [&](double z) __attribute__((always_inline)) {
    double tot = 0.0;
    for (int i = 0; i < GROUP; ++i) {
      const double x = wl[i][t];
      tot += fabs(x - (code(x, z) - z) * s);
    }
    return tot;
  };
  if (!degenerate) {
    const double z0 = f16_bits_to_f64(z16);
    const double e0 = l1(z0);
    double z = z0, best_z = z0, best = e0, beta = kHqqBeta;
    for (int it = 0; it < kHqqIters; ++it) {
      double acc = 0.0;
      for (int i = 0; i < GROUP; ++i) {
        const double x = wl[i][t];
        const double q = code(x, z);
        const double r = x - (q - z) * s;
        const double a = fabs(r);
        const double e = r == 0.0 ? 0.0 : copysign(fmax(a - pow(a, kHqqP - 1.0) / beta, 0.0), r);
        acc += q - (x - e) / s;
      }
      const double z_new = acc / GROUP;
      const double err = l1(z_new);
      if (!(err < best)) break;
      best = err;
      best_z = z_new;
      z = z_new;
      beta = beta * kHqqKappa;
    }
    const uint16_t zb = f64_to_f16_bits(best_z);
    if (l1(f16_bits_to_f64(zb)) < e0) z16 = zb;
  }
  const double zf = f16_bits_to_f64(z16);
  uint8_t* dst = codes + n * K + static_cast<long long>(g) * GROUP;
  for (int i = 0; i < GROUP; i += 16) {
    uint32_t word[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t b = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        b |= (degenerate ? 0u : static_cast<uint32_t>(code(wl[i + 4 * j + k][t], zf))) << (8 * k);
      word[j] = b;
    }
    *reinterpret_cast<uint4*>(dst + i) = make_uint4(word[0], word[1], word[2], word[3]);
  }
  sc[static_cast<long long>(g) * N + n] = s16;
  zr[static_cast<long long>(g) * N + n] = z16;
}

// Packed words of one slice from its 32 codes c[e + 8*j] (k order of the slice).
template <int BITS>
__device__ __forceinline__ void pack_slice_words(const uint32_t c[32], uint32_t* out) {
  constexpr uint32_t mask = (1u << BITS) - 1;
  for (int w = 0; w < BITS; ++w) out[w] = 0;
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    const int j = p / 4, i = p % 4;
    const uint32_t ev = c[8 * j + 2 * i] & mask, od = c[8 * j + 2 * i + 1] & mask;
    if constexpr (BITS == 4) {
      out[p / 4] |= (ev << (4 * (p % 4))) | (od << (16 + 4 * (p % 4)));
    } else if constexpr (BITS == 2) {
      out[p / 8] |= (ev << (2 * (p % 8))) | (od << (16 + 2 * (p % 8)));
    } else {
      if (p < 15) {
        out[p / 5] |= (ev << (3 * (p % 5))) | (od << (16 + 3 * (p % 5)));
      } else {
#pragma unroll
        for (int b = 0; b < 3; ++b)
          out[b] |= (((ev >> b) & 1u) << 15) | (((od >> b) & 1u) << 31);
      }
    }
  }
}

// One thread per (tile, slice).
template <int BITS>
__global__ __launch_bounds__(256) void k_qpack(const uint8_t* __restrict__ codes, int N, int K,
                                               uint8_t* __restrict__ qw) {
  const int KB = K / kTileK;
  const long long tiles = static_cast<long long>(N / kTileN) * KB;
  const long long gidx = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (gidx >= tiles * kWave) return;
  const long long tile = gidx / kWave;
  const int L = static_cast<int>(gidx % kWave);
  const long long nt = tile / KB;
  const int kb = static_cast<int>(tile % KB);
  const long long n = nt * kTileN + L % 16;
  const uint8_t* row = codes + n * K + kb * kTileK + 8 * (L / 16);
  uint32_t c[32];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint2 v = *reinterpret_cast<const uint2*>(row + 32 * j);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      c[8 * j + e] = (v.x >> (8 * e)) & 0xFFu;
      c[8 * j + 4 + e] = (v.y >> (8 * e)) & 0xFFu;
    }
  }
  uint32_t words[BITS];
  pack_slice_words<BITS>(c, words);
  uint32_t* dst = reinterpret_cast<uint32_t*>(qw + (tile * kWave + L) * (4 * BITS));
#pragma unroll
  for (int w = 0; w < BITS; ++w) dst[w] = words[w];
}

// One thread per (tile, slice): unpack with the qlinear kernels' code, then dequant.
template <int BITS>
__global__ __launch_bounds__(256) void k_qdequant(const uint8_t* __restrict__ qw,
                                                  const uint16_t* __restrict__ sc,
                                                  const uint16_t* __restrict__ zr, int group,
                                                  int N, int K, float* __restrict__ wf,
                                                  uint16_t* __restrict__ wb) {
  const int KB = K / kTileK;
  const long long tiles = static_cast<long long>(N / kTileN) * KB;
  const long long gidx = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (gidx >= tiles * kWave) return;
  const long long tile = gidx / kWave;
  const int L = static_cast<int>(gidx % kWave);
  const long long nt = tile / KB;
  const int kb = static_cast<int>(tile % KB);
  const long long n = nt * kTileN + L % 16;
  const Slice<BITS> s = load_slice<BITS>(qw + (tile * kWave + L) * (4 * BITS));
  uint32_t pr[16];
  unpack_pairs<BITS>(s, pr);
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    const int k0 = kb * kTileK + 32 * (p / 4) + 8 * (L / 16) + 2 * (p % 4);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k = k0 + h;
      const float q = static_cast<float>((pr[p] >> (16 * h)) & 0xFFu);
      const long long gi = static_cast<long long>(k / group) * N + n;
      const float sv = half_bits_to_float(sc[gi]);
      const float zv = half_bits_to_float(zr[gi]);
      const float b = -(sv * zv);  // exact: product of two fp16 values
      const float v = __builtin_fmaf(q, sv, b);
      if (wf) wf[n * K + k] = v;
      if (wb) wb[n * K + k] = float_to_bf16_bits(v);
    }
  }
}

hipError_t launch_quantize(const float* w, int bits, int group, int N, int K, uint8_t* codes,
                           uint16_t* sc, uint16_t* zr, hipStream_t st) {
  const long long groups = static_cast<long long>(N) * (K / group);
  const long long blocks = (groups + 3) / 4;
  if (group == 64)
    hipLaunchKernelGGL(k_quantize<64>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, w,
                       bits, N, K, codes, sc, zr);
  else
    hipLaunchKernelGGL(k_quantize<128>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, st, w,
                       bits, N, K, codes, sc, zr);
  return hipGetLastError();
}

hipError_t launch_quantize_hqq(const float* w, int bits, int group, int N, int K, uint8_t* codes,
                               uint16_t* sc, uint16_t* zr, hipStream_t st) {
  const long long groups = static_cast<long long>(N) * (K / group);
  const dim3 grid(static_cast<unsigned>((groups + kWave - 1) / kWave)), block(kWave);
  if (group == 64)
    hipLaunchKernelGGL(k_quantize_hqq<64>, grid, block, 0, st, w, bits, N, K, codes, sc, zr);
  else
    hipLaunchKernelGGL(k_quantize_hqq<128>, grid, block, 0, st, w, bits, N, K, codes, sc, zr);
  return hipGetLastError();
}

hipError_t launch_qpack(const uint8_t* codes, int bits, int N, int K, void* qw, hipStream_t st) {
  const long long threads = static_cast<long long>(N / kTileN) * (K / kTileK) * kWave;
  const dim3 grid(static_cast<unsigned>((threads + 255) / 256));
  uint8_t* out = static_cast<uint8_t*>(qw);
  switch (bits) {
    case 4: hipLaunchKernelGGL(k_qpack<4>, grid, dim3(256), 0, st, codes, N, K, out); break;
    case 3: hipLaunchKernelGGL(k_qpack<3>, grid, dim3(256), 0, st, codes, N, K, out); break;
    default: hipLaunchKernelGGL(k_qpack<2>, grid, dim3(256), 0, st, codes, N, K, out); break;
  }
  return hipGetLastError();
}

hipError_t launch_qdequant(const void* qw, const void* sc, const void* zr, int bits, int group,
                           int N, int K, float* wf, uint16_t* wb, hipStream_t st) {
  const long long threads = static_cast<long long>(N / kTileN) * (K / kTileK) * kWave;
  const dim3 grid(static_cast<unsigned>((threads + 255) / 256));
  const uint8_t* q = static_cast<const uint8_t*>(qw);
  const uint16_t* s = static_cast<const uint16_t*>(sc);
  const uint16_t* z = static_cast<const uint16_t*>(zr);
  switch (bits) {
    case 4: hipLaunchKernelGGL(k_qdequant<4>, grid, dim3(256), 0, st, q, s, z, group, N, K, wf, wb); break;
    case 3: hipLaunchKernelGGL(k_qdequant<3>, grid, dim3(256), 0, st, q, s, z, group, N, K, wf, wb); break;
    default: hipLaunchKernelGGL(k_qdequant<2>, grid, dim3(256), 0, st, q, s, z, group, N, K, wf, wb); break;
  }
  return hipGetLastError();
}

}  // namespace subspec
