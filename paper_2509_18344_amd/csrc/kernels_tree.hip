// Draft-tree expansion with probability sharpening (SubSpec Sec. 4.2 and App. D).
//
// In each draft pass every leaf i of the tree yields logits l_i over the vocabulary.
// A candidate (i, v) scores  s_i + log softmax(l_i / T)(v)  -- the logarithm of the
// product of the parent's path score and the sharpened conditional probability --
// and the k best candidates over all leaves become the next leaves.  Order: larger
// score first, then the smaller flat index i * V + v.
//
// One launch, two phases.  Workgroup (row i, chunk c) streams its slice of l_i once
// (16-byte loads of eight bf16 logits, four loads in flight per thread), keeping per thread an online softmax pair
// (running max m, sum of exp(z - m)) and a sorted list of its k best z = l / T; the
// workgroup merges both and stores them.  The last workgroup to finish (completion
// counter, as in the qlinear split-K) combines the pairs of each row into its
// log-sum-exp, turns every stored candidate into a score and selects the k best.
// Every reduction runs in a fixed order, so results are bit-reproducible.
#include <climits>
#include <cmath>

#include "device_common.h"
#include "kernels_tree.h"

namespace subspec {

namespace {

constexpr int kTreeThreads = 256;
constexpr int kTreeWaves = kTreeThreads / kWave;
constexpr int kTreeMaxBlocks = 1024;  // R * chunks never exceeds this (tree_plan)
constexpr int kTreeBatch = 16;        // candidate loads in flight per thread
constexpr int kTreeLoads = 4;         // logit loads in flight per thread
constexpr int kTreeCoherent = 16;     // sc1: coherent at agent scope
constexpr int kTreeCap = 2048;        // candidates ranked at once in LDS

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
  // per-wavefront heads of a selection round; rounds alternate between the two
  // slots, so one barrier per round suffices
  float bv[2][kTreeWaves];
  int bi[2][kTreeWaves];
  int last;
  int n;  // candidates appended to the LDS buffer
  // the k winners of the workgroup, stored to memory after the last round (a store
  // inside a round would make every following barrier wait for it)
  float win_v[kTreeMaxK];
  int win_i[kTreeMaxK];
};

// One step of a wavefront reduction over (value, index) with a DPP lane move.  Rows
// outside ROW_MASK keep their own pair (the move returns it as `old`).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ void dpp_best(float& v, int& i) {
  const int vb = __builtin_bit_cast(int, v);
  const float ov = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(vb, vb, CTRL, ROW_MASK, 0xF, false));
  const int oi = __builtin_amdgcn_update_dpp(i, i, CTRL, ROW_MASK, 0xF, false);
  if (better(ov, oi, v, i)) {
    v = ov;
    i = oi;
  }
}

// The wavefront's best (value, index) in every lane: quads, half rows and rows by
// lane permutations, then rows 0-1 and 2-3 by row broadcasts into lane 63.
__device__ __forceinline__ void wave_best(float& v, int& i) {
  dpp_best<0xB1, 0xF>(v, i);   // quad_perm [1,0,3,2]
  dpp_best<0x4E, 0xF>(v, i);   // quad_perm [2,3,0,1]
  dpp_best<0x141, 0xF>(v, i);  // row_half_mirror
  dpp_best<0x140, 0xF>(v, i);  // row_mirror
  dpp_best<0x142, 0xA>(v, i);  // row_bcast:15 into rows 1 and 3
  dpp_best<0x143, 0xC>(v, i);  // row_bcast:31 into rows 2 and 3
  v = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), kWave - 1));
  i = __builtin_amdgcn_readlane(i, kWave - 1);
}

// Largest value over the wavefront (same lane moves), in every lane.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_max_step(float v) {
  const int vb = __builtin_bit_cast(int, v);
  return fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(vb, vb, CTRL, ROW_MASK, 0xF, false)));
}
__device__ __forceinline__ float wave_max(float v) {
  v = dpp_max_step<0xB1, 0xF>(v);
  v = dpp_max_step<0x4E, 0xF>(v);
  v = dpp_max_step<0x141, 0xF>(v);
  v = dpp_max_step<0x140, 0xF>(v);
  v = dpp_max_step<0x142, 0xA>(v);
  v = dpp_max_step<0x143, 0xC>(v);
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), kWave - 1));
}

// Workgroup-wide best head of the threads' lists, removed from its owner; rounds
// 0..k-1 give the workgroup's k best in order.  All threads get (value, index).
// A thread can write the slot of round j + 2 only after every thread has reached
// the barrier of round j + 1, i.e. has finished reading round j.
template <int KMAX>
__device__ __forceinline__ void take_best(TopList<KMAX>& t, TreeShared& sh, int round, float& val, int& idx) {
  float v = t.v[0];
  int i = t.i[0];
  wave_best(v, i);
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int slot = round & 1;
  if (lane == 0) {
    sh.bv[slot][wave] = v;
    sh.bi[slot][wave] = i;
  }
  __syncthreads();
  val = sh.bv[slot][0];
  idx = sh.bi[slot][0];
#pragma unroll
  for (int w = 1; w < kTreeWaves; ++w)
    if (better(sh.bv[slot][w], sh.bi[slot][w], val, idx)) {
      val = sh.bv[slot][w];
      idx = sh.bi[slot][w];
    }
  if (t.i[0] == idx) t.pop();
}

// A value that at least k of the lanes' heads reach: the largest heads are taken off
// round by round (tied lanes together) until k are counted; -inf if the wavefront
// holds fewer than k finite heads.  Called with every lane active.
__device__ __forceinline__ float wave_kth_head(float h, int k) {
  float th = -INFINITY;
  int cnt = 0;
  while (cnt < k) {
    const float mx = wave_max(h);
    if (mx == -INFINITY) return -INFINITY;
    cnt += __popcll(__ballot(h == mx));
    th = mx;
    h = h == mx ? -INFINITY : h;
  }
  return th;
}

struct Cand {
  float v;
  int i;
};

// The k best of the n (<= kTreeCap) buffered candidates, by rank: each candidate
// counts the candidates better than it (indices are distinct, so ranks are too) and
// the ranks below k take their places; places past n get empty entries.  Ends with
// a barrier.
// The buffer is read two entries per 16-byte load and compared without branches, so
// the loads of an unrolled step are all in flight together.
__device__ __forceinline__ int better01(float av, int ai, float bv, int bi) {
  return static_cast<int>(av > bv) | (static_cast<int>(av == bv) & static_cast<int>(ai < bi));
}
__device__ __forceinline__ void rank_select(const Cand* buf, int n, int k, TreeShared& sh) {
  const int n2 = n & ~1;
  for (int c = threadIdx.x; c < n; c += kTreeThreads) {
    const Cand me = buf[c];
    int r = 0;
#pragma unroll 4
    for (int j = 0; j < n2; j += 2) {
      const float4 w = *reinterpret_cast<const float4*>(buf + j);
      r += better01(w.x, __float_as_int(w.y), me.v, me.i) + better01(w.z, __float_as_int(w.w), me.v, me.i);
    }
    if (n & 1) r += better01(buf[n - 1].v, buf[n - 1].i, me.v, me.i);
    if (r < k) {
      sh.win_v[r] = me.v;
      sh.win_i[r] = me.i;
    }
  }
  for (int t = threadIdx.x; t < k; t += kTreeThreads)
    if (t >= n) {
      sh.win_v[t] = -INFINITY;
      sh.win_i[t] = INT_MAX;
    }
  __syncthreads();
}

// The k best entries of the threads' lists into sh.win_v / sh.win_i, best first.
// A threshold that some wavefront's heads reach k times leaves few entries; those
// are ranked in LDS.  If more than kTreeCap remain (ties), k rounds of take_best.
// Called with every thread active; ends with a barrier.
template <int KMAX>
__device__ __forceinline__ void select_from_lists(TopList<KMAX>& top, TreeShared& sh, Cand* buf, int k) {
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const float th = wave_kth_head(top.v[0], k);
  if (lane == 0) sh.bv[0][wave] = th;
  if (threadIdx.x == 0) sh.n = 0;
  __syncthreads();
  float theta = sh.bv[0][0];
#pragma unroll
  for (int w = 1; w < kTreeWaves; ++w) theta = fmaxf(theta, sh.bv[0][w]);
  // the entries at or above theta are a prefix of each sorted list
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) cnt += top.i[j] != INT_MAX && top.v[j] >= theta ? 1 : 0;
  int off = 0;
  if (cnt) off = atomicAdd(&sh.n, cnt);
#pragma unroll
  for (int j = 0; j < KMAX; ++j)
    if (j < cnt && off + j < kTreeCap) buf[off + j] = Cand{top.v[j], top.i[j]};
  __syncthreads();
  const int n = sh.n;
  if (n <= kTreeCap) {
    rank_select(buf, n, k, sh);
    return;
  }
  for (int j = 0; j < k; ++j) {
    float val;
    int idx;
    take_best(top, sh, j, val, idx);
    if (threadIdx.x == 0) {
      sh.win_v[j] = val;
      sh.win_i[j] = idx;
    }
  }
  __syncthreads();
}

template <int KMAX>
__global__ __launch_bounds__(kTreeThreads) void k_tree_expand(TreeArgs a) {
  __shared__ TreeShared sh;
  __shared__ float lse_row[kTreeMaxRows];
  __shared__ float stat_lds[2 * kTreeMaxBlocks];
  __shared__ float par_lds[kTreeMaxRows];
  __shared__ __align__(16) Cand cbuf[kTreeCap];
  const int blk = blockIdx.x;
  const int row = blk / a.chunks, ch = blk % a.chunks;
  const int v0 = ch * a.chunk_len, v1 = min(a.V, v0 + a.chunk_len);

  // Phase 1: this workgroup's slice of row `row`.
  // kTreeLoads 16-byte loads per thread are in flight before any is used; loads
  // past the chunk read zeros (buffer resource ends at v1) and are skipped.
  const __amdgpu_buffer_rsrc_t lr = buffer_rsrc(a.logits + static_cast<size_t>(row) * a.V, v1 * 2);
  float m = -INFINITY, s = 0.f;
  TopList<KMAX> top;
  top.clear();
  // theta: a value that k of the logits seen by the wavefront reach (the lists keep
  // them), so nothing below it can be among the wavefront's k best.  It is set from
  // the k-th largest of the lanes' maxima of their first eight logits and raised once
  // per batch from the k-th largest of the lanes' list heads; the (divergent)
  // insertions of the logits at or above it stay rare.
  float theta = -INFINITY;
  // The trip count is the same for every lane (wave_max needs all lanes active);
  // each lane skips the logits past the chunk.
  for (int vb0 = v0; vb0 < v1; vb0 += kTreeThreads * 8 * kTreeLoads) {
    const int vb = vb0 + static_cast<int>(threadIdx.x) * 8;
    u32x4_t q[kTreeLoads];
#pragma unroll
    for (int u = 0; u < kTreeLoads; ++u)
      q[u] = __builtin_amdgcn_raw_buffer_load_b128(lr, static_cast<uint32_t>(vb + u * kTreeThreads * 8) * 2,
                                                   0, 0);
#pragma unroll
    for (int u = 0; u < kTreeLoads; ++u) {
      const int v = vb + u * kTreeThreads * 8;
      const bool live = v < v1;
      float z[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t w = q[u][e / 2];
        z[e] = __uint_as_float(e % 2 ? (w & 0xFFFF0000u) : (w << 16)) * a.inv_t;  // bf16 -> f32
      }
      float m8 = z[0];
#pragma unroll
      for (int e = 1; e < 8; ++e) m8 = fmaxf(m8, z[e]);
      if (theta == -INFINITY)  // wave-uniform: until a first bound is found
        theta = wave_kth_head(live ? m8 : -INFINITY, a.k);
      if (!live) continue;
      // online softmax over the eight: one rescale per load
      const float mn = fmaxf(m, m8);
      float add = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) add += __expf(z[e] - mn);
      s = (m == -INFINITY ? 0.f : s * __expf(m - mn)) + add;
      m = mn;
      // the rare logits at or above theta go through one insertion site
      unsigned hit = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) hit |= (z[e] >= theta ? 1u : 0u) << e;
      while (hit) {
        const int e = __builtin_ctz(hit);
        hit &= hit - 1;
        float ze = z[0];
#pragma unroll
        for (int f = 1; f < 8; ++f) ze = e == f ? z[f] : ze;
        if (better(ze, v + e, top.v[KMAX - 1], top.i[KMAX - 1])) top.insert(ze, v + e);
      }
    }
    theta = fmaxf(theta, wave_kth_head(top.v[0], a.k));
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
  select_from_lists(top, sh, cbuf, a.k);
  if (static_cast<int>(threadIdx.x) < a.k) {
    const size_t o = static_cast<size_t>(blk) * a.k + threadIdx.x;
    __hip_atomic_store(a.cand_val + o, sh.win_v[threadIdx.x], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(a.cand_idx + o, sh.win_i[threadIdx.x], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

  // Phase 2.  The workgroups' results are read with the coherent cache policy; each
  // read is a trip to the coherent level of the memory system, so the (m, s) pairs
  // and the first batch of candidates are all requested before anything waits.
  const int nblk = gridDim.x;
  const int per_row = a.chunks * a.k;
  const int total = a.R * per_row;
  const __amdgpu_buffer_rsrc_t rm_ = buffer_rsrc(a.stat_m, nblk * 4);
  const __amdgpu_buffer_rsrc_t rs_ = buffer_rsrc(a.stat_s, nblk * 4);
  const __amdgpu_buffer_rsrc_t rv_ = buffer_rsrc(a.cand_val, total * 4);
  const __amdgpu_buffer_rsrc_t ri_ = buffer_rsrc(a.cand_idx, total * 4);
  float z[kTreeBatch];
  int v[kTreeBatch];
  auto load_batch = [&](int q0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < kTreeBatch; ++u) {  // past the end: zeros, skipped when used
      const uint32_t off = static_cast<uint32_t>(q0 + u * kTreeThreads) * 4;
      z[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rv_, off, 0, kTreeCoherent));
      v[u] = static_cast<int>(__builtin_amdgcn_raw_buffer_load_b32(ri_, off, 0, kTreeCoherent));
    }
  };
  constexpr int kPer = kTreeMaxBlocks / kTreeThreads;
  static_assert(kTreeMaxRows <= kTreeMaxBlocks, "one parent score per block slot");
  const __amdgpu_buffer_rsrc_t rp_ = buffer_rsrc(a.parent, a.R * 4);
  float pm[kPer], ps[kPer], pk[kPer], ph[kPer], pp[kPer];  // per block: (m, s), k-th and first candidate; parents
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int b = threadIdx.x + u * kTreeThreads;
    const uint32_t off = static_cast<uint32_t>(b) * 4;
    pm[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rm_, off, 0, kTreeCoherent));
    ps[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs_, off, 0, kTreeCoherent));
    pk[u] = __uint_as_float(
        __builtin_amdgcn_raw_buffer_load_b32(rv_, static_cast<uint32_t>(b * a.k + a.k - 1) * 4, 0, kTreeCoherent));
    ph[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rv_, static_cast<uint32_t>(b * a.k) * 4, 0, kTreeCoherent));
    pp[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rp_, off, 0, 0));
  }
  load_batch(threadIdx.x);
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int q = threadIdx.x + u * kTreeThreads;
    if (q < nblk) {
      stat_lds[2 * q] = pm[u];
      stat_lds[2 * q + 1] = ps[u];
    }
    if (q < a.R) par_lds[q] = pp[u];
  }
  if (threadIdx.x == 0) sh.n = 0;
  __syncthreads();
  // The log-sum-exp of every row from its chunks' pairs: a group of G lanes per row
  // (G the power of two >= chunks, at most a wavefront), each lane over chunks
  // lane, lane + G, ..., then a butterfly over the group.  Both merges of a
  // butterfly pair give the same bits, so every lane ends with the same pair.
  {
    int G = 1;
    while (G < a.chunks && G < kWave) G <<= 1;
    const int rows_per_pass = kTreeThreads / G;
    const int gl = threadIdx.x % G, gi = threadIdx.x / G;
    for (int r0 = 0; r0 < a.R; r0 += rows_per_pass) {  // the same trip count for all lanes
      const int r = r0 + gi;
      float rm = -INFINITY, rs = 0.f;
      if (r < a.R)
        for (int c = gl; c < a.chunks; c += G)
          softmax_merge(rm, rs, stat_lds[2 * (r * a.chunks + c)], stat_lds[2 * (r * a.chunks + c) + 1]);
      for (int off = 1; off < G; off <<= 1) {
        const float om = __shfl_xor(rm, off), os = __shfl_xor(rs, off);
        softmax_merge(rm, rs, om, os);
      }
      if (r < a.R && gl == 0) lse_row[r] = rm + __logf(rs);
    }
  }
  __syncthreads();
  // theta: a score that k candidates reach, so nothing below it can be among the k
  // best: the best score of any block's k-th candidate (that block alone has k
  // candidates at or above it: a score grows with z within a row, also in rounding),
  // or a value that k lanes' best block heads reach, whichever is larger.
  {
    float tb = -INFINITY, hb = -INFINITY;
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int b = threadIdx.x + u * kTreeThreads;
      if (b < nblk) {
        const int r = b / a.chunks;
        tb = fmaxf(tb, par_lds[r] + (pk[u] - lse_row[r]));
        hb = fmaxf(hb, par_lds[r] + (ph[u] - lse_row[r]));
      }
    }
    tb = fmaxf(wave_max(tb), wave_kth_head(hb, a.k));
    if (lane == 0) sh.wm[wave] = tb;
  }
  __syncthreads();
  float theta2 = sh.wm[0];
#pragma unroll
  for (int w = 1; w < kTreeWaves; ++w) theta2 = fmaxf(theta2, sh.wm[w]);
  // Every stored candidate becomes a score; those at or above theta are kept.
  float sc[kTreeBatch];
  auto score_batch = [&](int q0) __attribute__((always_inline)) -> unsigned {
    unsigned ok = 0;
#pragma unroll
    for (int u = 0; u < kTreeBatch; ++u) {
      const int q = q0 + u * kTreeThreads;
      const bool valid = q < total && v[u] != INT_MAX;  // past the end, or an empty slot
      const int r = valid ? q / per_row : 0;
      sc[u] = par_lds[r] + (z[u] - lse_row[r]);
      v[u] = r * a.V + v[u];
      ok |= (valid && sc[u] >= theta2 ? 1u : 0u) << u;
    }
    return ok;
  };
  auto pick = [&](int u, float& su, int& iu) __attribute__((always_inline)) {
    su = sc[0];
    iu = v[0];
#pragma unroll
    for (int w = 1; w < kTreeBatch; ++w) {
      su = u == w ? sc[w] : su;
      iu = u == w ? v[w] : iu;
    }
  };
  // Usually only a few candidates reach theta: they go to the LDS buffer and are
  // ranked there.
  for (int q0 = threadIdx.x; q0 < total; q0 += kTreeThreads * kTreeBatch) {
    if (q0 != static_cast<int>(threadIdx.x)) load_batch(q0);
    unsigned ok = score_batch(q0);
    if (ok) {
      int off = atomicAdd(&sh.n, __popc(ok));
      while (ok) {
        const int u = __builtin_ctz(ok);
        ok &= ok - 1;
        float su;
        int iu;
        pick(u, su, iu);
        if (off < kTreeCap) cbuf[off] = Cand{su, iu};
        ++off;
      }
    }
  }
  __syncthreads();
  const int n = sh.n;
  if (n <= kTreeCap) {
    rank_select(cbuf, n, a.k, sh);
  } else {
    // More ties than the buffer holds: the same candidates again, through the
    // threads' lists and k rounds of take_best.
    top.clear();
    for (int q0 = threadIdx.x; q0 < total; q0 += kTreeThreads * kTreeBatch) {
      load_batch(q0);
      unsigned ok = score_batch(q0);
      while (ok) {
        const int u = __builtin_ctz(ok);
        ok &= ok - 1;
        float su;
        int iu;
        pick(u, su, iu);
        top.insert(su, iu);
      }
    }
    for (int j = 0; j < a.k; ++j) {
      float val;
      int idx;
      take_best(top, sh, j, val, idx);
      if (threadIdx.x == 0) {
        sh.win_v[j] = val;
        sh.win_i[j] = idx;
      }
    }
    __syncthreads();
  }
  if (static_cast<int>(threadIdx.x) < a.k) {
    const int idx = sh.win_i[threadIdx.x];
    a.out_parent[threadIdx.x] = idx / a.V;
    a.out_token[threadIdx.x] = idx % a.V;
    a.out_score[threadIdx.x] = sh.win_v[threadIdx.x];
  }
  if (threadIdx.x == 0) __hip_atomic_store(a.cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

void tree_plan(int R, int V, int* chunks, int* chunk_len) {
  // About two workgroups per CU of the 256, at least 2048 logits (one 16-byte load
  // per thread) each.
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
