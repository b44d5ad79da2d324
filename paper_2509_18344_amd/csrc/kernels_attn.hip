// Tree attention of the draft model over the shared KV cache (SubSpec Sec. 4.1,
// "Shared KV-Cache"; tree masks as in Sec. 2 and Sec. 4.2).
//
// One draft pass of one decoder layer: M new tree tokens, each with Hq query heads
// grouped onto Hkv key/value heads (G = Hq / Hkv queries share one), attend to the P
// committed positions of the cache, to the tree tokens of earlier passes their mask
// bits allow (cache positions P .. P + T - 1) and to themselves and each other as
// the mask allows (the new keys and values, which also go into the cache at
// P + T .. P + T + M - 1 for the passes that follow).
//
// Kernel 1 (k_attn_partial): workgroup (range s, key/value head g) streams its range
// of keys in tiles of 32 through LDS (keys row-major, values transposed into the
// order the P.V product wants); wavefront t owns query rows 16t .. 16t + 15 of the
// G * M rows of head g (row = local head * M + token).  Per tile and wavefront:
//   S^T = K Q^T        16x16x32 bf16 MFMA, 2 key halves x 4 steps of 32 dimensions
//   online softmax     log2 domain; each lane holds one query's scores (4 keys per
//                      half), the row maximum takes two cross-quarter exchanges
//   O^T += V^T P^T     16x16x32 bf16 MFMA, 8 tiles of 16 dimensions; P is split
//                      into two bf16 terms (hi = bf16(p), lo = bf16(p - hi)), two
//                      MFMAs each, so the probabilities keep 16 significant bits;
//                      P is already in the B-operand layout in registers
// and writes its unnormalised partial output with the running maximum and sum.
// Kernel 2 (k_attn_combine): one workgroup per (token, query head) combines the
// ranges in a fixed order and writes bf16; it also appends the new keys and values
// to the cache (after kernel 1, so nothing in this call reads a slot it writes).
#include <cmath>

#include "device_common.h"
#include "kernels_attn.h"

namespace subspec {

namespace {

constexpr int kAttnThreads = 256;
constexpr int kKRow = kAttnD + 8;     // bf16 per key row in LDS (16 bytes of padding)
constexpr int kVRow = kAttnTile + 8;  // bf16 per dimension row of the transposed values
constexpr int kDepth = 4;             // tiles in flight per thread

// The P.V product takes, in k-slot 8q + r of a lane in quarter q, key 4q + r (r < 4)
// and in slot 8q + 4 + r key 16 + 4q + r: exactly the keys whose scores that lane
// holds after S^T = K Q^T.  Values are stored transposed in this slot order.
__device__ __forceinline__ int value_slot(int key) {
  return key < 16 ? 8 * (key >> 2) + (key & 3) : 8 * ((key - 16) >> 2) + 4 + (key & 3);
}

struct AttnLds {
  alignas(16) uint16_t k[2][kAttnTile][kKRow];
  alignas(16) uint16_t vt[2][kAttnD][kVRow];
  alignas(16) uint32_t mask[kAttnMaskWords];
};

// Visibility of the 32 keys key0 .. key0 + 31 for one query row (bit k: key0 + k):
// committed positions (< P) always, tree positions P + j by bit j of the row's mask,
// nothing at or past k_end.  `row_mask` is the row's W words in LDS.
__device__ __forceinline__ uint32_t tile_visibility(const uint32_t* row_mask, int W, int P, int key0, int k_end) {
  uint32_t vis;
  if (key0 + kAttnTile <= P) {
    vis = ~0u;
  } else if (key0 >= P) {
    const int jb = key0 - P, w = jb >> 5, sh = jb & 31;
    const uint64_t lo = row_mask[w];
    const uint64_t hi = w + 1 < W ? row_mask[w + 1] : 0u;
    vis = static_cast<uint32_t>(((hi << 32) | lo) >> sh);
  } else {  // the tile straddles P: committed keys, then the first tree bits
    const int n = P - key0;  // 1 .. 31
    vis = (row_mask[0] << n) | ((1u << n) - 1u);
  }
  const int live = k_end - key0;  // >= 1
  return live >= kAttnTile ? vis : vis & ((1u << live) - 1u);
}

// A tile's share of one thread: two 16-byte pieces of keys (key c / 16, dimensions
// 8 (c % 16) ..) for c = thread, thread + 256, and a pair of keys' 8 dimensions of
// values (keys 2 (thread % 16) and + 1, dimensions 8 (thread / 16) ..).
struct TileRegs {
  uint4 k[2];
  uint4 v[2];
};

__device__ __forceinline__ const uint16_t* key_row(const AttnArgs& a, const uint16_t* cache,
                                                   const uint16_t* fresh, int g, int pos) {
  const int old = a.P + a.T;
  return pos < old ? cache + (static_cast<size_t>(g) * a.S + pos) * kAttnD
                   : fresh + (static_cast<size_t>(pos - old) * a.Hkv + g) * kAttnD;
}

__device__ __forceinline__ void load_tile(const AttnArgs& a, int g, int key0, int key_end, TileRegs& r) {
  const int t = threadIdx.x;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int c = t + h * kAttnThreads;
    const int pos = key0 + (c >> 4);
    r.k[h] = pos < key_end ? *reinterpret_cast<const uint4*>(key_row(a, a.k_cache, a.k_new, g, pos) + 8 * (c & 15))
                           : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int pos = key0 + 2 * (t & 15) + h;
    r.v[h] = pos < key_end ? *reinterpret_cast<const uint4*>(key_row(a, a.v_cache, a.v_new, g, pos) + 8 * (t >> 4))
                           : make_uint4(0, 0, 0, 0);
  }
}

__device__ __forceinline__ void store_tile(AttnLds& L, int buf, const TileRegs& r) {
  const int t = threadIdx.x;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int c = t + h * kAttnThreads;
    *reinterpret_cast<uint4*>(&L.k[buf][c >> 4][8 * (c & 15)]) = r.k[h];
  }
  // two keys (adjacent slots) of one dimension per 32-bit word
  const int slot = value_slot(2 * (t & 15));
  const int d0 = 8 * (t >> 4);
  const uint32_t a0[4] = {r.v[0].x, r.v[0].y, r.v[0].z, r.v[0].w};
  const uint32_t a1[4] = {r.v[1].x, r.v[1].y, r.v[1].z, r.v[1].w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t lo = __builtin_amdgcn_perm(a1[e], a0[e], 0x05040100u);  // dimension 2e: key, key + 1
    const uint32_t hi = __builtin_amdgcn_perm(a1[e], a0[e], 0x07060302u);  // dimension 2e + 1
    *reinterpret_cast<uint32_t*>(&L.vt[buf][d0 + 2 * e][slot]) = lo;
    *reinterpret_cast<uint32_t*>(&L.vt[buf][d0 + 2 * e + 1][slot]) = hi;
  }
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return static_cast<uint32_t>(float_to_bf16_bits(lo)) | (static_cast<uint32_t>(float_to_bf16_bits(hi)) << 16);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

template <int QT>
__global__ __launch_bounds__(kAttnThreads) void k_attn_partial(AttnArgs a) {
  __shared__ AttnLds L;
  const int s = blockIdx.x, g = blockIdx.y;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int col = lane & 15, quarter = lane >> 4;
  const int G = a.Hq / a.Hkv;
  const int rows = G * a.M;
  const int Ltot = a.P + a.T + a.M;
  const int k_begin = s * a.tiles_per_split * kAttnTile;
  const int k_end = min(Ltot, k_begin + a.tiles_per_split * kAttnTile);
  const int ntiles = (k_end - k_begin + kAttnTile - 1) / kAttnTile;

  // this lane's query row (one per lane and wavefront) and its fragments of q
  const int row = 16 * wave + col;
  const bool live_row = wave < QT && row < rows;
  const int qi = live_row ? row % a.M : 0;
  const int hl = live_row ? row / a.M : 0;
  bf16x8_t qf[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint4 w = make_uint4(0, 0, 0, 0);
    if (live_row)
      w = *reinterpret_cast<const uint4*>(a.q + (static_cast<size_t>(qi) * a.Hq + g * G + hl) * kAttnD + 32 * j +
                                          8 * quarter);
    qf[j] = __builtin_bit_cast(bf16x8_t, w);
  }
  for (int w = threadIdx.x; w < a.M * a.W; w += kAttnThreads) L.mask[w] = a.mask[w];

  float m = -INFINITY, lsum = 0.f;
  f32x4_t o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  TileRegs ring[kDepth];
#pragma unroll
  for (int d = 0; d < kDepth; ++d)
    if (d < ntiles) load_tile(a, g, k_begin + d * kAttnTile, k_end, ring[d]);

  for (int n0 = 0; n0 < ntiles; n0 += kDepth) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      const int n = n0 + d;
      if (n >= ntiles) break;
      const int buf = n & 1;
      // buffer buf was last read two tiles ago, before the previous barrier
      store_tile(L, buf, ring[d]);
      if (n + kDepth < ntiles) load_tile(a, g, k_begin + (n + kDepth) * kAttnTile, k_end, ring[d]);
      __syncthreads();
      if (wave < QT) {
        const int key0 = k_begin + n * kAttnTile;
        // S^T = K Q^T: lane holds keys 16u + 4 quarter + r of its query
        f32x4_t st[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          st[u] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(&L.k[buf][16 * u + col][32 * j + 8 * quarter]);
            st[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[j], st[u], 0, 0, 0);
          }
        }
        // scale, mask (committed positions are always visible), online softmax
        const uint32_t vis = live_row ? tile_visibility(&L.mask[qi * a.W], a.W, a.P, key0, k_end) : 0u;
        float sv[2][4];
        float mx = -INFINITY;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const bool ok = (vis >> (16 * u + 4 * quarter + r)) & 1u;
            sv[u][r] = ok ? st[u][r] * a.scale_log2 : -INFINITY;
            mx = fmaxf(mx, sv[u][r]);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mn = fmaxf(m, mx);
        // raw 2^x (a probability below 2^-126 flushing to zero does not matter)
        const float alpha = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mn);
        // p = hi + lo in bf16; the same two terms feed P.V and the sum
        uint32_t ph[4], pl[4];
        float add = 0.f;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int r = 0; r < 4; r += 2) {
            const float p0 = sv[u][r] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sv[u][r] - mn);
            const float p1 = sv[u][r + 1] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sv[u][r + 1] - mn);
            const uint32_t h = pack_bf16(p0, p1);
            const uint32_t l = pack_bf16(p0 - bf16_lo(h), p1 - bf16_hi(h));
            ph[2 * u + r / 2] = h;
            pl[2 * u + r / 2] = l;
            add += (bf16_lo(h) + bf16_lo(l)) + (bf16_hi(h) + bf16_hi(l));
          }
        lsum = lsum * alpha + add;
        m = mn;
        const bf16x8_t pfh = __builtin_bit_cast(bf16x8_t, make_uint4(ph[0], ph[1], ph[2], ph[3]));
        const bf16x8_t pfl = __builtin_bit_cast(bf16x8_t, make_uint4(pl[0], pl[1], pl[2], pl[3]));
        if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {  // some row's maximum moved
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) o[dt] *= alpha;
        }
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
          const bf16x8_t vf = *reinterpret_cast<const bf16x8_t*>(&L.vt[buf][16 * dt + col][8 * quarter]);
          o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pfh, o[dt], 0, 0, 0);
          o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pfl, o[dt], 0, 0, 0);
        }
      }
    }
  }

  if (wave < QT) {
    // the four quarters hold partial sums of the same query
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
  }
  if (live_row) {  // padding rows are never read
    const size_t base = (static_cast<size_t>(g) * a.splits + s) * a.rows_pad + row;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
      *reinterpret_cast<f32x4_t*>(a.part_o + base * kAttnD + 16 * dt + 4 * quarter) = o[dt];
    if (quarter == 0) {
      a.part_ml[2 * base] = m;
      a.part_ml[2 * base + 1] = lsum;
    }
  }
}

// One workgroup per (token i, query head h), one thread per dimension.  Each range's
// (max, sum) pair is read once into LDS and turned into a weight; the partial
// outputs are then read in batches of independent loads and summed in range order.
__global__ __launch_bounds__(kAttnD) void k_attn_combine(AttnArgs a) {
  __shared__ float sm[kAttnMaxSplits], sl[kAttnMaxSplits];
  constexpr int kBatch = 16;
  const int i = blockIdx.x / a.Hq, h = blockIdx.x % a.Hq;
  const int d = threadIdx.x;
  const int G = a.Hq / a.Hkv;
  const int g = h / G, hl = h % G;
  const int row = hl * a.M + i;
  const int ns = a.splits;
  const size_t base = static_cast<size_t>(g) * ns * a.rows_pad + row;
  for (int s = d; s < ns; s += kAttnD) {
    const size_t b = base + static_cast<size_t>(s) * a.rows_pad;
    sm[s] = a.part_ml[2 * b];
    sl[s] = a.part_ml[2 * b + 1];
  }
  __syncthreads();
  float mmax = -INFINITY;
  for (int s = 0; s < ns; ++s) mmax = fmaxf(mmax, sm[s]);
  __syncthreads();
  for (int s = d; s < ns; s += kAttnD) sm[s] = sm[s] == -INFINITY ? 0.f : exp2f(sm[s] - mmax);
  __syncthreads();
  float den = 0.f, num = 0.f;
  for (int s0 = 0; s0 < ns; s0 += kBatch) {
    float v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      v[u] = s0 + u < ns ? a.part_o[(base + static_cast<size_t>(s0 + u) * a.rows_pad) * kAttnD + d] : 0.f;
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      if (s0 + u < ns) {
        den += sm[s0 + u] * sl[s0 + u];
        num += sm[s0 + u] * v[u];
      }
  }
  a.out[(static_cast<size_t>(i) * a.Hq + h) * kAttnD + d] = float_to_bf16_bits(den > 0.f ? num / den : 0.f);
  // append this token's key and value for head g (once per key/value head)
  if (hl == 0) {
    const size_t dst = (static_cast<size_t>(g) * a.S + a.P + a.T + i) * kAttnD + d;
    const size_t src = (static_cast<size_t>(i) * a.Hkv + g) * kAttnD + d;
    a.k_cache[dst] = a.k_new[src];
    a.v_cache[dst] = a.v_new[src];
  }
}

}  // namespace

void attn_plan(int M, int Hq, int Hkv, int P, int T, int* splits, int* tiles_per_split) {
  (void)Hq;
  const int L = P + T + M;
  const int tiles = (L + kAttnTile - 1) / kAttnTile;
  // at most one workgroup per CU of the 256 and at least three tiles each (all in
  // flight at once): fewer, longer ranges keep the partial outputs small beside the
  // keys and values read (three measured fastest at 2336 keys; two and four were
  // within 4 %, six 20 % slower)
  constexpr int kMinTiles = 3;
  int tps = (tiles * Hkv + 255) / 256;
  if (tps < kMinTiles) tps = kMinTiles;
  if (tps > tiles) tps = tiles;
  *tiles_per_split = tps;
  *splits = (tiles + tps - 1) / tps;
}

size_t attn_workspace_bytes(int M, int Hq, int Hkv, int P, int T) {
  int splits = 0, tps = 0;
  attn_plan(M, Hq, Hkv, P, T, &splits, &tps);
  const int rows_pad = 16 * ((Hq / Hkv * M + 15) / 16);
  const size_t n = static_cast<size_t>(Hkv) * splits * rows_pad;
  // The partials follow the split-K completion counters at the workspace's start.
  return kSplitCounterBytes + n * kAttnD * sizeof(float) + n * 2 * sizeof(float);
}

hipError_t launch_tree_attention(const AttnArgs& a, hipStream_t st) {
  const dim3 grid(a.splits, a.Hkv), block(kAttnThreads);
  switch (a.rows_pad / 16) {
    case 1: hipLaunchKernelGGL(k_attn_partial<1>, grid, block, 0, st, a); break;
    case 2: hipLaunchKernelGGL(k_attn_partial<2>, grid, block, 0, st, a); break;
    case 3: hipLaunchKernelGGL(k_attn_partial<3>, grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL(k_attn_partial<4>, grid, block, 0, st, a); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_attn_combine, dim3(a.M * a.Hq), dim3(kAttnD), 0, st, a);
  return hipGetLastError();
}

}  // namespace subspec
