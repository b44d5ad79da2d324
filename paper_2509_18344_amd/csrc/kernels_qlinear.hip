// The substitute-layer linear y = x * dequant(q, s, z)^T (SubSpec Sec. 4.1) for
// draft-tree batches, as two kernels over one packed layout:
//
//   k_qgemv       M <= 8.  VALU bf16 dot products; the four 16-lane quarters of a
//                 wavefront split K inside every tile and are reduced with cross-row
//                 lane swaps at the end, workgroups split K through a fixed-order
//                 reduction of fp32 partial sums.
//   k_qgemm_mfma  any M.  16x16x32 bf16 MFMA; the A operand (activations) comes
//                 from LDS, the B operand straight from the unpacked codes.
//
// Dequantization is folded into the accumulation.  Within one group the weight is
// affine in the code, W^ = s*(q - z), so for every (row m, column n, group g)
//     sum_{k in g} x*W^ = s * ( sum_{k in g} x*(128+q) - (128+z) * sum_{k in g} x ).
// The kernels feed the exact bf16 values 128+q (one and-or per code pair, see
// device_common.h) to the dot products / matrix cores and apply s and z once per
// (m, n, g).  The effective weights are the exact dequantized values; the only
// roundings are the fp32 accumulation and the final bf16 store.
#include "device_common.h"
#include "kernels.h"

namespace subspec {

// ---------------------------------------------------------------------------
// Activation staging: one chunk (CHUNK blocks of 128 k, all ROWS rows) of x is
// copied to LDS by the whole workgroup together with the per-group sums of x the
// zero-point correction needs.  Double buffered: chunk c+1 is read from global
// memory into registers while chunk c is being consumed.
// ---------------------------------------------------------------------------

template <int ROWS, int CHUNK, int GROUP, bool QUARTER>
struct StageLds {
  static constexpr int CK = CHUNK * kTileK;
  static constexpr int XSTRIDE = CK + 8;  // bf16 per row, +16 bytes against bank conflicts
  static constexpr int GPC = CK / GROUP;  // groups per chunk
  static constexpr int SUMS = QUARTER ? 4 : 1;
  uint16_t x[2][ROWS][XSTRIDE];
  // Sum of x over one group (MFMA) or over the quarter of a group one 16-lane
  // quarter of a wavefront sees (GEMV: k % 32 in [8q, 8q+8)).
  float xsum[2][GPC][ROWS][SUMS];
};

template <int ROWS, int CHUNK>
struct StageRegs {
  static constexpr int C8 = CHUNK * 16;  // 16-byte pieces per row of a chunk
  static constexpr int TOTAL = ROWS * C8;
  static constexpr int NPASS = (TOTAL + kThreadsPerBlock - 1) / kThreadsPerBlock;
  uint4 v[NPASS];
};

template <int ROWS, int CHUNK>
__device__ __forceinline__ void stage_load(StageRegs<ROWS, CHUNK>& r, const QArgs& a, int kb,
                                           int kb_end) {
  using R = StageRegs<ROWS, CHUNK>;
#pragma unroll
  for (int p = 0; p < R::NPASS; ++p) {
    const int i = p * kThreadsPerBlock + threadIdx.x;
    const int row = i / R::C8, c8 = i % R::C8;
    const bool ok = (i < R::TOTAL) && (row < a.M) && (kb + c8 / 16 < kb_end);
    r.v[p] = ok ? *reinterpret_cast<const uint4*>(a.x + static_cast<size_t>(row) * a.K +
                                                  static_cast<size_t>(kb) * kTileK + c8 * 8)
                : make_uint4(0u, 0u, 0u, 0u);
  }
}

__device__ __forceinline__ float bf16lo(uint32_t v) { return __builtin_bit_cast(float, v << 16); }
__device__ __forceinline__ float bf16hi(uint32_t v) { return __builtin_bit_cast(float, v & 0xFFFF0000u); }

// DPP move of a float within 16-lane rows (all lanes active).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xF, 0xF, false));
}
constexpr int kDppQuadXor1 = 0xB1;      // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;      // quad_perm [2,3,0,1]
constexpr int kDppRowRor4 = 0x124;      // row_ror:4
constexpr int kDppRowRor8 = 0x128;      // row_ror:8
constexpr int kDppRowHalfMirror = 0x141;

template <int ROWS, int CHUNK, int GROUP, bool QUARTER>
__device__ __forceinline__ void stage_store(StageLds<ROWS, CHUNK, GROUP, QUARTER>& L, int buf,
                                            const StageRegs<ROWS, CHUNK>& r) {
  using R = StageRegs<ROWS, CHUNK>;
  constexpr int P8 = GROUP / 8;  // 16-byte pieces per group
#pragma unroll
  for (int p = 0; p < R::NPASS; ++p) {
    const int i = p * kThreadsPerBlock + threadIdx.x;
    const int row = i / R::C8, c8 = i % R::C8;
    const uint4 v = r.v[p];
    if (i < R::TOTAL) *reinterpret_cast<uint4*>(&L.x[buf][row][c8 * 8]) = v;
    float s = ((bf16lo(v.x) + bf16hi(v.x)) + (bf16lo(v.y) + bf16hi(v.y))) +
              ((bf16lo(v.z) + bf16hi(v.z)) + (bf16lo(v.w) + bf16hi(v.w)));
    // The pieces of one (row, group) are P8 consecutive lanes of one 16-lane row.
    if constexpr (QUARTER) {
      // quarter q of a group = pieces with c8 % 4 == q
      if constexpr (GROUP == 128) {
        s += dpp_f<kDppRowRor4>(s);
        s += dpp_f<kDppRowRor8>(s);
      } else {
        s += __shfl_xor(s, 4);
      }
      if (i < R::TOTAL && (c8 % P8) < 4) L.xsum[buf][c8 / P8][row][c8 % 4] = s;
    } else {
      s += dpp_f<kDppQuadXor1>(s);
      s += dpp_f<kDppQuadXor2>(s);
      if constexpr (GROUP == 128) {
        s += dpp_f<kDppRowRor4>(s);
        s += dpp_f<kDppRowRor8>(s);
      } else {
        s += dpp_f<kDppRowHalfMirror>(s);
      }
      if (i < R::TOTAL && (c8 % P8) == 0) L.xsum[buf][c8 / P8][row][0] = s;
    }
  }
}

// ---------------------------------------------------------------------------
// Weight stream: every wavefront owns NT tiles (16 columns each) and walks its
// split's k-blocks; one chunk of slices plus the chunk's scale/zero pairs is kept
// in flight ahead of the one being consumed.
// ---------------------------------------------------------------------------

template <int BITS, int NT, int CHUNK, int GPC>
struct WeightRegs {
  Slice<BITS> w[CHUNK][NT];
  uint32_t sz[GPC][NT];  // fp16 scale | fp16 zero << 16
};

template <int BITS, int GROUP, int NT, int CHUNK, int GPC>
__device__ __forceinline__ void load_weights(WeightRegs<BITS, NT, CHUNK, GPC>& r, const QArgs& a,
                                             const uint8_t* const (&wbase)[NT],
                                             const bool (&tok)[NT], const int (&ncol)[NT], int kb,
                                             int kb_end) {
  constexpr int GPB = kTileK / GROUP;
#pragma unroll
  for (int b = 0; b < CHUNK; ++b) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (tok[t] && kb + b < kb_end) {
        r.w[b][t] = load_slice<BITS>(wbase[t] + static_cast<size_t>(kb + b) * (256 * BITS));
      } else {
#pragma unroll
        for (int q = 0; q < BITS; ++q) r.w[b][t].w[q] = 0u;
      }
    }
  }
#pragma unroll
  for (int gc = 0; gc < GPC; ++gc) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const size_t gi = static_cast<size_t>(kb * GPB + gc) * a.N + ncol[t];
      const bool ok = tok[t] && (kb + gc / GPB < kb_end);
      r.sz[gc][t] = ok ? (static_cast<uint32_t>(a.sc[gi]) | (static_cast<uint32_t>(a.zr[gi]) << 16))
                       : 0u;
    }
  }
}

__device__ __forceinline__ void scale_and_offset(uint32_t sz, float& s, float& c) {
  s = half_bits_to_float(static_cast<uint16_t>(sz & 0xFFFFu));
  const float z = half_bits_to_float(static_cast<uint16_t>(sz >> 16));
  c = s * (kCodeBias + z);
}

// ---------------------------------------------------------------------------
// Split-K epilogue shared by both kernels: with one split the result goes straight
// to y; otherwise every workgroup stores fp32 partials and the last one of its
// column group to arrive sums them in split order (so the result does not depend
// on arrival order) and resets the arrival counter for the next call.
// ---------------------------------------------------------------------------

__device__ __forceinline__ void store_out(const QArgs& a, int split, int m, int n, float v) {
  if (a.splits == 1)
    a.y[static_cast<size_t>(m) * a.N + n] = float_to_bf16_bits(v);
  else
    a.ws[(static_cast<size_t>(split) * a.M + m) * a.N + n] = v;
}

__device__ __forceinline__ void finish_splits(const QArgs& a, int ng, int cols_per_group,
                                              unsigned* s_last) {
  if (a.splits == 1) return;
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned prev = atomicAdd(&a.counters[ng], 1u);
    *s_last = (prev == static_cast<unsigned>(a.splits - 1)) ? 1u : 0u;
  }
  __syncthreads();
  if (*s_last == 0u) return;
  __threadfence();
  const int n0 = ng * cols_per_group;
  const int ncols = min(a.N - n0, cols_per_group);
  const int total = a.M * ncols;
  for (int idx = threadIdx.x; idx < total; idx += kThreadsPerBlock) {
    const int m = idx / ncols, n = n0 + idx % ncols;
    float s = 0.0f;
    for (int sp = 0; sp < a.splits; ++sp)
      s += __builtin_nontemporal_load(&a.ws[(static_cast<size_t>(sp) * a.M + m) * a.N + n]);
    a.y[static_cast<size_t>(m) * a.N + n] = float_to_bf16_bits(s);
  }
  if (threadIdx.x == 0) a.counters[ng] = 0u;
}

// ---------------------------------------------------------------------------
// MFMA kernel.
// ---------------------------------------------------------------------------

template <int BITS, int GROUP, int MT, int NT, int CHUNK>
__global__ __launch_bounds__(kThreadsPerBlock) void k_qgemm_mfma(QArgs a) {
  constexpr int ROWS = 16 * MT;
  constexpr int GPB = kTileK / GROUP;  // groups per block
  constexpr int SPG = 4 / GPB;         // 32-k steps per group
  constexpr int GPC = CHUNK * GPB;
  using Lds = StageLds<ROWS, CHUNK, GROUP, false>;
  __shared__ Lds lds;
  __shared__ unsigned s_last;

  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int col = lane & 15, quarter = lane >> 4;
  const int ng = blockIdx.x / a.splits, split = blockIdx.x % a.splits;
  const int nt0 = (ng * kWavesPerBlock + wave) * NT;
  const int kb_begin = split * a.blocks_per_split;
  const int kb_end = min(a.KB, kb_begin + a.blocks_per_split);
  const int nchunks = (kb_end - kb_begin + CHUNK - 1) / CHUNK;

  const uint8_t* wbase[NT];
  bool tok[NT];
  int ncol[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    tok[t] = nt0 + t < a.n_tiles;
    const int ntc = tok[t] ? nt0 + t : 0;
    wbase[t] = a.qw + static_cast<size_t>(ntc) * a.KB * (256 * BITS) + lane * (4 * BITS);
    ncol[t] = ntc * kTileN + col;
  }

  f32x4_t tot[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int t = 0; t < NT; ++t) tot[mt][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  WeightRegs<BITS, NT, CHUNK, GPC> wc, wn;
  StageRegs<ROWS, CHUNK> xr;
  load_weights<BITS, GROUP>(wc, a, wbase, tok, ncol, kb_begin, kb_end);
  stage_load(xr, a, kb_begin, kb_end);
  stage_store(lds, 0, xr);
  __syncthreads();

  for (int c = 0; c < nchunks; ++c) {
    const int kb = kb_begin + c * CHUNK;
    const int buf = c & 1;
    const bool more = c + 1 < nchunks;
    if (more) {
      load_weights<BITS, GROUP>(wn, a, wbase, tok, ncol, kb + CHUNK, kb_end);
      stage_load(xr, a, kb + CHUNK, kb_end);
    }
#pragma unroll
    for (int b = 0; b < CHUNK; ++b) {
      if (kb + b < kb_end) {
        uint32_t pr[NT][16];
#pragma unroll
        for (int t = 0; t < NT; ++t) unpack_pairs<BITS>(wc.w[b][t], pr[t]);
#pragma unroll
        for (int gi = 0; gi < GPB; ++gi) {
          const int gc = b * GPB + gi;
          float sv[NT], cv[NT];
#pragma unroll
          for (int t = 0; t < NT; ++t) scale_and_offset(wc.sz[gc][t], sv[t], cv[t]);
          f32x4_t acc[MT][NT];
#pragma unroll
          for (int js = 0; js < SPG; ++js) {
            const int j = gi * SPG + js;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
              const bf16x8_t A = *reinterpret_cast<const bf16x8_t*>(
                  &lds.x[buf][16 * mt + col][b * kTileK + 32 * j + 8 * quarter]);
#pragma unroll
              for (int t = 0; t < NT; ++t) {
                const uint4 bw = make_uint4(pr[t][4 * j], pr[t][4 * j + 1], pr[t][4 * j + 2],
                                            pr[t][4 * j + 3]);
                const bf16x8_t B = __builtin_bit_cast(bf16x8_t, bw);
                const f32x4_t cin = (js == 0) ? f32x4_t{0.f, 0.f, 0.f, 0.f} : acc[mt][t];
                acc[mt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B, cin, 0, 0, 0);
              }
            }
          }
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const f32x4_t xs =
                *reinterpret_cast<const f32x4_t*>(&lds.xsum[buf][gc][16 * mt + 4 * quarter][0]);
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                float v = __builtin_fmaf(sv[t], acc[mt][t][r], tot[mt][t][r]);
                tot[mt][t][r] = __builtin_fmaf(-cv[t], xs[r], v);
              }
          }
        }
      }
    }
    if (more) stage_store(lds, buf ^ 1, xr);
    __syncthreads();
    wc = wn;
  }

  // D layout of 16x16 MFMA: lane holds column lane%16, rows 4*(lane/16) + r.
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = 16 * mt + 4 * quarter + r;
        if (tok[t] && m < a.M) store_out(a, split, m, ncol[t], tot[mt][t][r]);
      }
  finish_splits(a, ng, kWavesPerBlock * NT * kTileN, &s_last);
}

// ---------------------------------------------------------------------------
// GEMV kernel.
// ---------------------------------------------------------------------------

__device__ __forceinline__ float dot2_bf16(uint32_t xa, uint32_t wb, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, xa),
                                         __builtin_bit_cast(bf16x2_t, wb), acc, false);
}

template <int BITS, int GROUP, int ROWS, int NT, int CHUNK>
__global__ __launch_bounds__(kThreadsPerBlock) void k_qgemv(QArgs a) {
  constexpr int GPB = kTileK / GROUP;
  constexpr int SPG = 4 / GPB;
  constexpr int GPC = CHUNK * GPB;
  using Lds = StageLds<ROWS, CHUNK, GROUP, true>;
  __shared__ Lds lds;
  __shared__ unsigned s_last;

  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int col = lane & 15, quarter = lane >> 4;
  const int ng = blockIdx.x / a.splits, split = blockIdx.x % a.splits;
  const int nt0 = (ng * kWavesPerBlock + wave) * NT;
  const int kb_begin = split * a.blocks_per_split;
  const int kb_end = min(a.KB, kb_begin + a.blocks_per_split);
  const int nchunks = (kb_end - kb_begin + CHUNK - 1) / CHUNK;

  const uint8_t* wbase[NT];
  bool tok[NT];
  int ncol[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    tok[t] = nt0 + t < a.n_tiles;
    const int ntc = tok[t] ? nt0 + t : 0;
    wbase[t] = a.qw + static_cast<size_t>(ntc) * a.KB * (256 * BITS) + lane * (4 * BITS);
    ncol[t] = ntc * kTileN + col;
  }

  float tot[ROWS][NT];
#pragma unroll
  for (int m = 0; m < ROWS; ++m)
#pragma unroll
    for (int t = 0; t < NT; ++t) tot[m][t] = 0.f;

  WeightRegs<BITS, NT, CHUNK, GPC> wc, wn;
  StageRegs<ROWS, CHUNK> xr;
  load_weights<BITS, GROUP>(wc, a, wbase, tok, ncol, kb_begin, kb_end);
  stage_load(xr, a, kb_begin, kb_end);
  stage_store(lds, 0, xr);
  __syncthreads();

  for (int c = 0; c < nchunks; ++c) {
    const int kb = kb_begin + c * CHUNK;
    const int buf = c & 1;
    const bool more = c + 1 < nchunks;
    if (more) {
      load_weights<BITS, GROUP>(wn, a, wbase, tok, ncol, kb + CHUNK, kb_end);
      stage_load(xr, a, kb + CHUNK, kb_end);
    }
#pragma unroll
    for (int b = 0; b < CHUNK; ++b) {
      if (kb + b < kb_end) {
        uint32_t pr[NT][16];
#pragma unroll
        for (int t = 0; t < NT; ++t) unpack_pairs<BITS>(wc.w[b][t], pr[t]);
#pragma unroll
        for (int gi = 0; gi < GPB; ++gi) {
          const int gc = b * GPB + gi;
          float sv[NT], cv[NT];
#pragma unroll
          for (int t = 0; t < NT; ++t) scale_and_offset(wc.sz[gc][t], sv[t], cv[t]);
          float acc[ROWS][NT];
#pragma unroll
          for (int m = 0; m < ROWS; ++m)
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[m][t] = 0.f;
#pragma unroll
          for (int js = 0; js < SPG; ++js) {
            const int j = gi * SPG + js;
#pragma unroll
            for (int m = 0; m < ROWS; ++m) {
              const uint4 xv = *reinterpret_cast<const uint4*>(
                  &lds.x[buf][m][b * kTileK + 32 * j + 8 * quarter]);
#pragma unroll
              for (int t = 0; t < NT; ++t) {
                float v = acc[m][t];
                v = dot2_bf16(xv.x, pr[t][4 * j + 0], v);
                v = dot2_bf16(xv.y, pr[t][4 * j + 1], v);
                v = dot2_bf16(xv.z, pr[t][4 * j + 2], v);
                v = dot2_bf16(xv.w, pr[t][4 * j + 3], v);
                acc[m][t] = v;
              }
            }
          }
#pragma unroll
          for (int m = 0; m < ROWS; ++m) {
            const float xq = lds.xsum[buf][gc][m][quarter];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
              const float v = __builtin_fmaf(sv[t], acc[m][t], tot[m][t]);
              tot[m][t] = __builtin_fmaf(-cv[t], xq, v);
            }
          }
        }
      }
    }
    if (more) stage_store(lds, buf ^ 1, xr);
    __syncthreads();
    wc = wn;
  }

  // Split-K inside the wavefront: the four quarters hold partial sums of the same
  // column over disjoint k; add the partner rows (lane ^ 16, then lane ^ 32).
#pragma unroll
  for (int m = 0; m < ROWS; ++m)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      float v = tot[m][t];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      tot[m][t] = v;
    }
#pragma unroll
  for (int m = 0; m < ROWS; ++m)
#pragma unroll
    for (int t = 0; t < NT; ++t)
      if (tok[t] && (m & 3) == quarter && m < a.M) store_out(a, split, m, ncol[t], tot[m][t]);
  finish_splits(a, ng, kWavesPerBlock * NT * kTileN, &s_last);
}

// ---------------------------------------------------------------------------
// Dispatch table.
// ---------------------------------------------------------------------------

typedef void (*QKernel)(QArgs);

struct Variant {
  int path, rows, nt, chunk, bits, group;
  QKernel fn;
};

#define SUBSPEC_GEMV(B, G, R, T, C) {1, R, T, C, B, G, k_qgemv<B, G, R, T, C>}
#define SUBSPEC_MFMA(B, G, MT, T, C) {2, 16 * MT, T, C, B, G, k_qgemm_mfma<B, G, MT, T, C>}
#define SUBSPEC_BG(X)                                                                    \
  X(4, 128) X(4, 64) X(3, 128) X(3, 64) X(2, 128) X(2, 64)
#define SUBSPEC_GEMV_SET(B, G)                                                          \
  SUBSPEC_GEMV(B, G, 1, 1, 4), SUBSPEC_GEMV(B, G, 2, 1, 4), SUBSPEC_GEMV(B, G, 4, 1, 4), \
      SUBSPEC_GEMV(B, G, 8, 1, 4), SUBSPEC_GEMV(B, G, 1, 2, 4), SUBSPEC_GEMV(B, G, 2, 2, 4), \
      SUBSPEC_GEMV(B, G, 4, 2, 4), SUBSPEC_GEMV(B, G, 8, 2, 4),
#define SUBSPEC_MFMA_SET(B, G)                                                          \
  SUBSPEC_MFMA(B, G, 1, 2, 4), SUBSPEC_MFMA(B, G, 2, 2, 2), SUBSPEC_MFMA(B, G, 4, 2, 2), \
      SUBSPEC_MFMA(B, G, 8, 2, 1),

static const Variant kVariants[] = {SUBSPEC_BG(SUBSPEC_GEMV_SET) SUBSPEC_BG(SUBSPEC_MFMA_SET)};

static QKernel find_variant(const KernelChoice& kc, int bits, int group) {
  for (const Variant& v : kVariants)
    if (v.path == kc.path && v.rows == kc.rows && v.nt == kc.nt && v.chunk == kc.chunk &&
        v.bits == bits && v.group == group)
      return v.fn;
  return nullptr;
}

bool qlinear_variant_exists(const KernelChoice& kc, int bits, int group) {
  return find_variant(kc, bits, group) != nullptr;
}

hipError_t launch_qlinear(const KernelChoice& kc, int bits, int group, const QArgs& a, int grid,
                          hipStream_t st) {
  QKernel fn = find_variant(kc, bits, group);
  if (!fn) return hipErrorInvalidDeviceFunction;
  hipLaunchKernelGGL(fn, dim3(grid), dim3(kThreadsPerBlock), 0, st, a);
  return hipGetLastError();
}

}  // namespace subspec
