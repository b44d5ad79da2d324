// Dispatch of the 32x32x16 qlinear kernel (qmma_kernel.h) over its instantiations.
#include "qmma_kernel.h"

namespace subspec {

static const MmaVariant* find_mma(int waves, int teams, int mb, int nb, int pf, int bits, int group) {
  int n = 0;
  const MmaVariant* v = bits == 2 ? qmma_variants_b2(&n) : bits == 3 ? qmma_variants_b3(&n) : qmma_variants_b4(&n);
  for (int i = 0; i < n; ++i)
    if (v[i].waves == waves && v[i].teams == teams && v[i].mb == mb && v[i].nb == nb && (pf == 0 || v[i].pf == pf) && v[i].bits == bits &&
        v[i].group == group)
      return &v[i];
  return nullptr;
}

bool qmma_variant_exists(int waves, int teams, int mb, int nb, int pf, int bits, int group) {
  return find_mma(waves, teams, mb, nb, pf, bits, group) != nullptr;
}

int qmma_resident_blocks(int waves, int teams, int mb, int nb, int pf, int bits, int group) {
  const MmaVariant* v = find_mma(waves, teams, mb, nb, pf, bits, group);
  if (!v) return 0;
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, reinterpret_cast<const void*>(v->fn),
                                                   waves * kWave, 0) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return blocks;
}

hipError_t launch_qmma(int waves, int teams, int mb, int nb, int pf, int bits, int group, const QArgs& a,
                       int grid, hipStream_t st) {
  const MmaVariant* v = find_mma(waves, teams, mb, nb, pf, bits, group);
  if (!v) return hipErrorInvalidDeviceFunction;
  hipLaunchKernelGGL(v->fn, dim3(grid), dim3(waves * kWave), 0, st, a);
  return hipGetLastError();
}

// Sums of x over every group of k: one wavefront per (row, 512 k); lane l sums the 8
// values at k = 512 s + 8 l (four bf16 dot products with ones), then the G / 8 lanes
// of a group are added with lane exchanges (a fixed order, so the result is the same
// on every call).
template <int GROUP>
__global__ __launch_bounds__(256) void k_xsum(const uint16_t* __restrict__ x, int M, int K, float* __restrict__ out) {
  constexpr int LANES = GROUP / 8;
  const int lane = threadIdx.x % kWave;
  const int segs = (K + 511) / 512;
  const long long wv = static_cast<long long>(blockIdx.x) * 4 + threadIdx.x / kWave;
  if (wv >= static_cast<long long>(M) * segs) return;
  const int m = static_cast<int>(wv / segs), seg = static_cast<int>(wv % segs);
  const int k = seg * 512 + 8 * lane;
  float v = 0.f;
  if (k < K) v = piece_sum(*reinterpret_cast<const u32x4_t*>(x + static_cast<size_t>(m) * K + k), 0.f);
#pragma unroll
  for (int d = 1; d < LANES; d *= 2) v += __shfl_xor(v, d);
  if (k < K && lane % LANES == 0) out[static_cast<size_t>(m) * (K / GROUP) + k / GROUP] = v;
}

hipError_t launch_xsum(const uint16_t* x, int M, int K, int group, float* out, hipStream_t st) {
  const long long waves = static_cast<long long>(M) * ((K + 511) / 512);
  const dim3 grid(static_cast<unsigned>((waves + 3) / 4)), block(256);
  if (group == 64)
    hipLaunchKernelGGL(k_xsum<64>, grid, block, 0, st, x, M, K, out);
  else
    hipLaunchKernelGGL(k_xsum<128>, grid, block, 0, st, x, M, K, out);
  return hipGetLastError();
}

}  // namespace subspec
