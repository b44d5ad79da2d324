// Draft-tree expansion with probability sharpening (SubSpec Sec. 4.2 and App. D).
//
// In each draft pass every leaf i of the tree yields logits l_i over the vocabulary.
// A candidate (i, v) scores  s_i + log softmax(l_i / T)(v)  -- the logarithm of the
// product of the parent's path score and the sharpened conditional probability --
// and the k best candidates over all leaves become the next leaves.  Order: larger
// score first, then the smaller flat index i * V + v.
//
// One launch, two phases.  Workgroup (row i, chunk c) streams its slice of l_i once
// (16-byte loads of eight bf16 logits), keeping per thread an online softmax pair
// (running max m, sum of exp(z - m)) and a sorted list of its k best z = l / T; the
// workgroup merges both and stores them.  The last workgroup to finish (completion
// counter, as in the qlinear split-K) combines the pairs of each row into its
// log-sum-exp, turns every stored candidate into a score and selects the k best.
// Every reduction runs in a fixed order, so results are bit-reproducible.
#include <climits>
#include <cmath>

#include "device_common.h"
#include "kernels.h"

namespace subspec {

namespace {

constexpr int kTreeThreads = 256;
constexpr int kTreeWaves = kTreeThreads / kWave;

// Candidate order: larger value first, then smaller index.
__device__ __forceinline__ bool better(float av, int ai, float bv, int bi) {
  return av > bv || (av == bv && ai < bi);
}

// A thread's KMAX best candidates, best first; empty slots hold (-inf, INT_MAX).
template <int KMAX>
struct TopList {
  float v[KMAX];
  int i[KMAX];
  __device__ __forceinline__ void clear() {
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      v[j] = -INFINITY;
      i[j] = INT_MAX;
    }
  }
  // One pass of compare-exchange down the list keeps it sorted.
  __device__ __forceinline__ void insert(float val, int idx) {
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      const bool b = better(val, idx, v[j], i[j]);
      const float tv = v[j];
      const int ti = i[j];
      v[j] = b ? val : tv;
      i[j] = b ? idx : ti;
      val = b ? tv : val;
      idx = b ? ti : idx;
    }
  }
  __device__ __forceinline__ void pop() {
#pragma unroll
    for (int j = 0; j + 1 < KMAX; ++j) {
      v[j] = v[j + 1];
      i[j] = i[j + 1];
    }
    v[KMAX - 1] = -INFINITY;
    i[KMAX - 1] = INT_MAX;
  }
};

// (m, s) pairs of an online softmax: s = sum of exp(z - m) over the values seen.
__device__ __forceinline__ void softmax_merge(float& m, float& s, float m2, float s2) {
  if (m2 > m) {
    const float t = m;
    m = m2;
    m2 = t;
    const float u = s;
    s = s2;
    s2 = u;
  }
  if (m2 != -INFINITY) s += s2 * __expf(m2 - m);
}

struct TreeShared {
  float wm[kTreeWaves], ws[kTreeWaves];
  float bv[kTreeWaves];
  int bi[kTreeWaves];
  int last;
};

// Workgroup-wide best head of the threads' lists, removed from its owner; k rounds
// give the workgroup's k best in order.  All threads get (value, index).
template <int KMAX>
__device__ __forceinline__ void take_best(TopList<KMAX>& t, TreeShared& sh, float& val, int& idx) {
  float v = t.v[0];
  int i = t.i[0];
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(v, off);
    const int oi = __shfl_xor(i, off);
    if (better(ov, oi, v, i)) {
      v = ov;
      i = oi;
    }
  }
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  if (lane == 0) {
    sh.bv[wave] = v;
    sh.bi[wave] = i;
  }
  __syncthreads();
  val = sh.bv[0];
  idx = sh.bi[0];
#pragma unroll
  for (int w = 1; w < kTreeWaves; ++w)
    if (better(sh.bv[w], sh.bi[w], val, idx)) {
      val = sh.bv[w];
      idx = sh.bi[w];
    }
  __syncthreads();
  if (t.i[0] == idx) t.pop();
}

template <int KMAX>
__global__ __launch_bounds__(kTreeThreads) void k_tree_expand(TreeArgs a) {
  __shared__ TreeShared sh;
  __shared__ float lse_row[kTreeMaxRows];
  const int blk = blockIdx.x;
  const int row = blk / a.chunks, ch = blk % a.chunks;
  const int v0 = ch * a.chunk_len, v1 = min(a.V, v0 + a.chunk_len);

  // Phase 1: this workgroup's slice of row `row`.
  const uint16_t* lrow = a.logits + static_cast<size_t>(row) * a.V;
  float m = -INFINITY, s = 0.f;
  TopList<KMAX> top;
  top.clear();
  for (int v = v0 + static_cast<int>(threadIdx.x) * 8; v < v1; v += kTreeThreads * 8) {
    const u32x4_t q = *reinterpret_cast<const u32x4_t*>(lrow + v);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t w = q[e / 2];
      const float x = __uint_as_float(e % 2 ? (w & 0xFFFF0000u) : (w << 16));  // bf16 -> f32
      const float z = x * a.inv_t;
      if (z > m) {
        s = s * __expf(m - z) + 1.f;
        m = z;
      } else {
        s += __expf(z - m);
      }
      top.insert(z, v + e);
    }
  }
  // (m, s) over the workgroup: lanes, then wavefronts, in a fixed order.
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const float om = __shfl_xor(m, off), os = __shfl_xor(s, off);
    softmax_merge(m, s, om, os);
  }
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  if (lane == 0) {
    sh.wm[wave] = m;
    sh.ws[wave] = s;
  }
  __syncthreads();
  float bm = sh.wm[0], bs = sh.ws[0];
#pragma unroll
  for (int w = 1; w < kTreeWaves; ++w) softmax_merge(bm, bs, sh.wm[w], sh.ws[w]);
  __syncthreads();
  for (int j = 0; j < a.k; ++j) {
    float val;
    int idx;
    take_best(top, sh, val, idx);
    if (threadIdx.x == 0) {
      __hip_atomic_store(a.cand_val + static_cast<size_t>(blk) * a.k + j, val, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.cand_idx + static_cast<size_t>(blk) * a.k + j, idx, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if (threadIdx.x == 0) {
    __hip_atomic_store(a.stat_m + blk, bm, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(a.stat_s + blk, bs, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // Completion: every workgroup waits for its own stores, the last one goes on.
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  __syncthreads();
  if (threadIdx.x == 0)
    sh.last = __hip_atomic_fetch_add(a.cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
              static_cast<unsigned>(gridDim.x - 1);
  __syncthreads();
  if (!sh.last) return;

  // Phase 2: log-sum-exp of every row from its chunks' pairs, in chunk order.
  for (int r = threadIdx.x; r < a.R; r += kTreeThreads) {
    float rm = -INFINITY, rs = 0.f;
    for (int c = 0; c < a.chunks; ++c)
      softmax_merge(rm, rs,
                    __hip_atomic_load(a.stat_m + r * a.chunks + c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
                    __hip_atomic_load(a.stat_s + r * a.chunks + c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    lse_row[r] = rm + __logf(rs);
  }
  __syncthreads();
  // Every stored candidate becomes a score; the k best over all rows are the result.
  top.clear();
  const int per_row = a.chunks * a.k;
  for (int q = threadIdx.x; q < a.R * per_row; q += kTreeThreads) {
    const int r = q / per_row;
    const float z = __hip_atomic_load(a.cand_val + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int v = __hip_atomic_load(a.cand_idx + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (v == INT_MAX) continue;  // an empty slot of a chunk shorter than k
    top.insert(a.parent[r] + (z - lse_row[r]), r * a.V + v);
  }
  for (int j = 0; j < a.k; ++j) {
    float val;
    int idx;
    take_best(top, sh, val, idx);
    if (threadIdx.x == 0) {
      a.out_parent[j] = idx / a.V;
      a.out_token[j] = idx % a.V;
      a.out_score[j] = val;
    }
  }
  if (threadIdx.x == 0) __hip_atomic_store(a.cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

void tree_plan(int R, int V, int* chunks, int* chunk_len) {
  // About two workgroups per CU of the 256, at least 2048 logits each.
  int c = (512 + R - 1) / R;
  const int cmax = (V + 2047) / 2048;
  if (c > cmax) c = cmax;
  if (c < 1) c = 1;
  int len = (V + c - 1) / c;
  len = (len + 7) / 8 * 8;
  *chunk_len = len;
  *chunks = (V + len - 1) / len;
}

size_t tree_workspace_bytes(int R, int V, int k) {
  int chunks = 0, len = 0;
  tree_plan(R, V, &chunks, &len);
  const size_t blocks = static_cast<size_t>(R) * chunks;
  return kSplitCounterBytes + blocks * 2 * sizeof(float) + blocks * k * (sizeof(float) + sizeof(int));
}

hipError_t launch_tree_expand(const TreeArgs& a, hipStream_t st) {
  const dim3 grid(a.R * a.chunks), block(kTreeThreads);
  if (a.k <= 8)
    hipLaunchKernelGGL(k_tree_expand<8>, grid, block, 0, st, a);
  else if (a.k <= 16)
    hipLaunchKernelGGL(k_tree_expand<16>, grid, block, 0, st, a);
  else
    hipLaunchKernelGGL(k_tree_expand<32>, grid, block, 0, st, a);
  return hipGetLastError();
}

}  // namespace subspec
