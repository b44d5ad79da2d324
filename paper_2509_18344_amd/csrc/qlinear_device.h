// Device-side pieces shared by the qlinear kernels (k_qgemv, k_qgemm_mfma and
// k_qmma): compile-time loops, bf16 dot products, the work assignment of a
// workgroup, buffer resources of the operands, and the split-K completion.
#pragma once

#include <type_traits>
#include <utility>

#include "device_common.h"
#include "kernels.h"

namespace subspec {

// ---------------------------------------------------------------------------
// Small helpers.
// ---------------------------------------------------------------------------

// Calls f(std::integral_constant<int, 0>{}) ... f(integral_constant<int, N-1>{}): ring
// slots indexed by a compile-time constant stay in registers.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ float dot2_bf16(uint32_t xa, uint32_t wb, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, xa),
                                         __builtin_bit_cast(bf16x2_t, wb), acc, false);
}

// Sum of the eight bf16 values of a 16-byte piece (dot products with 1.0 pairs).
__device__ __forceinline__ float piece_sum(const u32x4_t& v, float acc) {
  constexpr uint32_t kOnes = 0x3F803F80u;  // bf16 1.0, 1.0
  acc = dot2_bf16(v.x, kOnes, acc);
  acc = dot2_bf16(v.y, kOnes, acc);
  acc = dot2_bf16(v.z, kOnes, acc);
  return dot2_bf16(v.w, kOnes, acc);
}

// DPP move of a float within rows of 16 lanes (all lanes active).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xF, 0xF, false));
}
constexpr int kDppQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]

// Sum over the lanes of an aligned group of SPAN lanes (SPAN = 1, 2 or 4).
template <int SPAN>
__device__ __forceinline__ float span_reduce(float v) {
  if constexpr (SPAN >= 2) v += dpp_f<kDppQuadXor1>(v);
  if constexpr (SPAN >= 4) v += dpp_f<kDppQuadXor2>(v);
  return v;
}


// ---------------------------------------------------------------------------
// Dequantization constants.
// ---------------------------------------------------------------------------

// Per (column, group): the scale s and the offset c = s * (128 + z) that removes the
// code bias and the zero-point from the group's accumulated x * (128 + q).
__device__ __forceinline__ void scale_and_offset(uint32_t sbits, uint32_t zbits, float& s, float& c) {
  s = half_bits_to_float(static_cast<uint16_t>(sbits));
  const float z = half_bits_to_float(static_cast<uint16_t>(zbits));
  c = s * (kCodeBias + z);
}


// Global operands of one launch as buffer resources.
struct QBuffers {
  __amdgpu_buffer_rsrc_t x, w, s, z, xs;
  __device__ __forceinline__ QBuffers(const QArgs& a, int bits, int group) {
    x = buffer_rsrc(a.x, static_cast<uint32_t>(a.M) * a.K * 2);
    w = buffer_rsrc(a.qw, static_cast<uint32_t>(a.n_tiles) * a.KB * 256 * bits);
    const uint32_t sz = static_cast<uint32_t>(a.K / group) * a.N * 2;
    s = buffer_rsrc(a.sc, sz);
    z = buffer_rsrc(a.zr, sz);
    xs = buffer_rsrc(a.xsum, a.xsum ? static_cast<uint32_t>(a.M) * (a.K / group) * 4 : 0);
  }
};

// The row block of this workgroup (blockIdx.y, see QArgs) as a launch of its own:
// activations, output, partial sums and completion counters rebased, M cut to the
// block's rows.
__device__ __forceinline__ QArgs row_block(const QArgs& in) {
  QArgs a = in;
  if (a.rb_rows > 0) {
    const int r = blockIdx.y, m0 = r * a.rb_rows;
    a.x += static_cast<size_t>(m0) * a.K;
    a.y += static_cast<size_t>(m0) * a.N;
    a.ws += static_cast<size_t>(r) * a.splits * a.rb_rows * a.N;
    a.cnt += r * a.rb_counters;
    a.M = min(a.rb_rows, a.M - m0);
  }
  return a;
}

// ---------------------------------------------------------------------------
// Work of one workgroup (see QArgs): column group ng, k-blocks [kb0, kb_end), and
// its split index among the nsplit workgroups of that column group.
// ---------------------------------------------------------------------------

struct WorkItem {
  int ng, split, nsplit, kb0, kb_end;
  __device__ __forceinline__ explicit WorkItem(const QArgs& a) {
    const int b = blockIdx.x;
    if (b < a.full_groups) {
      ng = b;
      split = 0;
      nsplit = 1;
      kb0 = 0;
      kb_end = a.KB;
    } else {
      const int r = b - a.full_groups;
      ng = a.full_groups + r / a.splits;
      split = r % a.splits;
      nsplit = a.splits;
      kb0 = split * a.blocks_per_split;
      kb_end = min(a.KB, kb0 + a.blocks_per_split);
    }
  }
};

// ---------------------------------------------------------------------------
// Output.  A workgroup that covers all of K writes y directly.  Otherwise every
// workgroup of the column group stores fp32 partial sums ws[split][m][n], and the
// last one to finish adds them in split order and writes y (finish_splitk).  The
// partial sums are written and read with agent-scope cache policy (coherent across
// the XCDs' L2 caches) and each workgroup waits for its own stores before counting
// itself in, so no cache flush or invalidation is needed.
// ---------------------------------------------------------------------------

constexpr int kCachePolicyAgent = 16;  // sc1: coherent at agent scope
constexpr int kFinishBatch = 8;        // partial-sum loads in flight per output quad
// s_waitcnt vmcnt(0), other counters untouched (expcnt 7, lgkmcnt 15).
constexpr int kWaitVmcnt0 = 0x0F70;
// s_waitcnt lgkmcnt(0), other counters untouched (vmcnt 63, expcnt 7).
constexpr int kWaitLgkmcnt0 = 0xC07F;

__device__ __forceinline__ void store_out(const QArgs& a, const WorkItem& wi, int m, int n, float v) {
  const int split = wi.split;
  if (wi.nsplit == 1)
    a.y[static_cast<size_t>(m) * a.N + n] = float_to_bf16_bits(v);
  else
    __hip_atomic_store(a.ws + (static_cast<size_t>(split) * a.M + m) * a.N + n, v, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

// Split-K completion for column group ng (columns [ng*cols, ng*cols + cols) of N,
// split a.splits ways): called by every thread of the workgroup after its partial
// sums are stored.
template <int THREADS>
__device__ __forceinline__ void finish_splitk(const QArgs& a, int ng, int cols) {
  __shared__ int last;
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __syncthreads();
  if (threadIdx.x == 0)
    last = __hip_atomic_fetch_add(a.cnt + ng, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
           static_cast<unsigned>(a.splits - 1);
  __syncthreads();
  if (!last) return;
  const int n0 = ng * cols;
  const int nq = min(cols, a.N - n0) / 4;  // column quads of the group
  const int total = a.M * nq;
  const uint32_t split_bytes = static_cast<uint32_t>(a.M) * a.N * 4;
  const __amdgpu_buffer_rsrc_t ws = buffer_rsrc(a.ws, split_bytes * a.splits);
  auto load = [&](uint32_t off) __attribute__((always_inline)) {
    return __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(ws, off, 0, kCachePolicyAgent));
  };
  // Every read of a partial sum is a trip to the coherent level of the memory
  // system, so a thread takes two quads at a time and issues the loads of up to
  // kFinishBatch splits of both before adding them in split order.  Splits past the
  // last read zeros (an offset past the buffer resource) and leave the sums unchanged.
  constexpr uint32_t kPastEnd = 0xFFFFFFF0u;
  for (int q0 = threadIdx.x; q0 < total; q0 += 2 * THREADS) {
    bool ok[2];
    int m[2], n[2];
    uint32_t off[2];
    f32x4_t acc[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = q0 + i * THREADS;
      ok[i] = q < total;
      const int qc = ok[i] ? q : q0;
      m[i] = qc / nq;
      n[i] = n0 + 4 * (qc % nq);
      off[i] = (static_cast<uint32_t>(m[i]) * a.N + n[i]) * 4;
      acc[i] = load(off[i]);
    }
    for (int sp = 1; sp < a.splits; sp += kFinishBatch) {
      f32x4_t v[2][kFinishBatch];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int u = 0; u < kFinishBatch; ++u)
          v[i][u] = load(sp + u < a.splits ? off[i] + (sp + u) * split_bytes : kPastEnd);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int u = 0; u < kFinishBatch; ++u) acc[i] += v[i][u];
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (!ok[i]) continue;
      const uint32_t lo = static_cast<uint32_t>(float_to_bf16_bits(acc[i][0])) |
                          (static_cast<uint32_t>(float_to_bf16_bits(acc[i][1])) << 16);
      const uint32_t hi = static_cast<uint32_t>(float_to_bf16_bits(acc[i][2])) |
                          (static_cast<uint32_t>(float_to_bf16_bits(acc[i][3])) << 16);
      *reinterpret_cast<uint2*>(a.y + static_cast<size_t>(m[i]) * a.N + n[i]) = make_uint2(lo, hi);
    }
  }
  if (threadIdx.x == 0) __hip_atomic_store(a.cnt + ng, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}


}  // namespace subspec
