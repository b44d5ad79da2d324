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

// Loads are unconditional: out-of-range pieces read a clamped (valid) address and
// are never consumed (blocks past the split are skipped, rows past M never stored),
// so no branch -- and no early wait on the counter of outstanding loads -- is
// placed around them.
template <int ROWS, int CHUNK>
__device__ __forceinline__ void stage_load(StageRegs<ROWS, CHUNK>& r, const QArgs& a, int kb,
                                           int kb_end) {
  using R = StageRegs<ROWS, CHUNK>;
#pragma unroll
  for (int p = 0; p < R::NPASS; ++p) {
    const int i = p * kThreadsPerBlock + threadIdx.x;
    const int row = min(i / R::C8, a.M - 1), c8 = i % R::C8;
    const int kbc = min(kb + c8 / 16, kb_end - 1);
    r.v[p] = *reinterpret_cast<const uint4*>(a.x + static_cast<size_t>(row) * a.K +
                                             static_cast<size_t>(kbc) * kTileK + (c8 % 16) * 8);
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
// split's k-blocks in chunks of CH blocks.  Two chunks of slices and their raw
// fp16 scale/zero values are in flight at any time (ping-pong registers).
// ---------------------------------------------------------------------------

template <int BITS, int NT, int CH, int GPC>
struct WChunk {
  Slice<BITS> w[CH][NT];
  uint32_t s[GPC][NT];  // fp16 bits of the scale
  uint32_t z[GPC][NT];  // fp16 bits of the zero-point
};

// Unconditional loads from clamped addresses (see stage_load): blocks past the end
// of the split re-read its last block and are never consumed.
template <int BITS, int GROUP, int NT, int CH, int GPC>
__device__ __forceinline__ void load_wchunk(WChunk<BITS, NT, CH, GPC>& r, const QArgs& a,
                                            const uint8_t* const (&wbase)[NT],
                                            const int (&ncol)[NT], int kb, int kb_end) {
  constexpr int GPB = kTileK / GROUP;
#pragma unroll
  for (int b = 0; b < CH; ++b) {
    const int kbc = min(kb + b, kb_end - 1);
#pragma unroll
    for (int t = 0; t < NT; ++t)
      r.w[b][t] = load_slice<BITS>(wbase[t] + static_cast<size_t>(kbc) * (256 * BITS));
  }
#pragma unroll
  for (int gc = 0; gc < GPC; ++gc) {
    const int g = min(kb * GPB + gc, kb_end * GPB - 1);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const size_t gi = static_cast<size_t>(g) * a.N + ncol[t];
      r.s[gc][t] = a.sc[gi];
      r.z[gc][t] = a.zr[gi];
    }
  }
}

// Per (column, group): the scale s and the offset c = s * (128 + z) that removes the
// code bias and the zero-point from the group's accumulated x * (128 + q).
__device__ __forceinline__ void scale_and_offset(uint32_t sbits, uint32_t zbits, float& s, float& c) {
  s = half_bits_to_float(static_cast<uint16_t>(sbits));
  const float z = half_bits_to_float(static_cast<uint16_t>(zbits));
  c = s * (kCodeBias + z);
}

// ---------------------------------------------------------------------------
// Output: with one split the result goes straight to y; otherwise each workgroup
// stores fp32 partial sums and k_splitk_reduce (launched next on the same stream,
// so the kernel boundary orders the two) adds them in split order.
// ---------------------------------------------------------------------------

__device__ __forceinline__ void store_out(const QArgs& a, int split, int m, int n, float v) {
  if (a.splits == 1)
    a.y[static_cast<size_t>(m) * a.N + n] = float_to_bf16_bits(v);
  else
    a.ws[(static_cast<size_t>(split) * a.M + m) * a.N + n] = v;
}

// y[m][n] = bf16(sum over s of ws[s][m][n]), s ascending; 4 columns per thread.
__global__ __launch_bounds__(kThreadsPerBlock) void k_splitk_reduce(const float* __restrict__ ws,
                                                                     uint16_t* __restrict__ y,
                                                                     int M, int N, int splits) {
  const size_t quads = static_cast<size_t>(M) * N / 4;
  const size_t i = static_cast<size_t>(blockIdx.x) * kThreadsPerBlock + threadIdx.x;
  if (i >= quads) return;
  const size_t plane = static_cast<size_t>(M) * N / 4;
  const float4* src = reinterpret_cast<const float4*>(ws) + i;
  float4 acc = src[0];
  for (int sp = 1; sp < splits; ++sp) {
    const float4 v = src[sp * plane];
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  const uint32_t lo = static_cast<uint32_t>(float_to_bf16_bits(acc.x)) |
                      (static_cast<uint32_t>(float_to_bf16_bits(acc.y)) << 16);
  const uint32_t hi = static_cast<uint32_t>(float_to_bf16_bits(acc.z)) |
                      (static_cast<uint32_t>(float_to_bf16_bits(acc.w)) << 16);
  reinterpret_cast<uint2*>(y)[i] = make_uint2(lo, hi);
}

// ---------------------------------------------------------------------------
// MFMA kernel.  Workgroup = 4 wavefronts x NT tiles = 64*NT columns, all rows, one
// k-split.  Per chunk of CH blocks: x is staged in LDS (double buffered, one
// barrier per chunk); each wavefront unpacks its tiles' codes straight into B
// operands and runs 16x16x32 bf16 MFMAs against A fragments read from LDS.
// ---------------------------------------------------------------------------

template <int BITS, int GROUP, int MT, int NT, int CH>
struct MfmaBody {
  static constexpr int ROWS = 16 * MT;
  static constexpr int GPB = kTileK / GROUP;  // groups per block
  static constexpr int SPG = 4 / GPB;         // 32-k steps per group
  static constexpr int GPC = CH * GPB;        // groups per chunk
  using Lds = StageLds<ROWS, CH, GROUP, false>;
  using W = WChunk<BITS, NT, CH, GPC>;

  // Consume one chunk (blocks kb..kb+CH-1 of the split, LDS buffer buf).
  static __device__ __forceinline__ void compute(const W& wc, const Lds& lds, int buf, int kb,
                                                 int kb_end, int col, int quarter,
                                                 f32x4_t (&tot)[MT][NT]) {
#pragma unroll
    for (int b = 0; b < CH; ++b) {
      if (kb + b < kb_end) {
        uint32_t pr[NT][16];
#pragma unroll
        for (int t = 0; t < NT; ++t) unpack_pairs<BITS>(wc.w[b][t], pr[t]);
#pragma unroll
        for (int gi = 0; gi < GPB; ++gi) {
          const int gc = b * GPB + gi;
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
          float sv[NT], cv[NT];
#pragma unroll
          for (int t = 0; t < NT; ++t) scale_and_offset(wc.s[gc][t], wc.z[gc][t], sv[t], cv[t]);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const f32x4_t xs =
                *reinterpret_cast<const f32x4_t*>(&lds.xsum[buf][gc][16 * mt + 4 * quarter][0]);
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const float v = __builtin_fmaf(sv[t], acc[mt][t][r], tot[mt][t][r]);
                tot[mt][t][r] = __builtin_fmaf(-cv[t], xs[r], v);
              }
          }
        }
      }
    }
  }
};

template <int BITS, int GROUP, int MT, int NT, int CH>
__global__ __launch_bounds__(kThreadsPerBlock) void k_qgemm_mfma(QArgs a) {
  using Body = MfmaBody<BITS, GROUP, MT, NT, CH>;
  __shared__ typename Body::Lds lds;

  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int col = lane & 15, quarter = lane >> 4;
  const int ng = blockIdx.x / a.splits, split = blockIdx.x % a.splits;
  const int nt0 = (ng * kWavesPerBlock + wave) * NT;
  const int kb_begin = split * a.blocks_per_split;
  const int kb_end = min(a.KB, kb_begin + a.blocks_per_split);
  const int nchunks = (kb_end - kb_begin + CH - 1) / CH;

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

  typename Body::W w0, w1;
  StageRegs<Body::ROWS, CH> xr;
  load_wchunk<BITS, GROUP>(w0, a, wbase, ncol, kb_begin, kb_end);
  load_wchunk<BITS, GROUP>(w1, a, wbase, ncol, kb_begin + CH, kb_end);
  stage_load(xr, a, kb_begin, kb_end);
  stage_store(lds, 0, xr);
  __syncthreads();

  // Straight-line loop body (refills and staging loads are unconditional, clamped
  // past the end of the split) so that every wait on outstanding loads is exact.
  for (int c = 0; c < nchunks; c += 2) {
    const int kb = kb_begin + c * CH;
    stage_load(xr, a, kb + CH, kb_end);
    Body::compute(w0, lds, 0, kb, kb_end, col, quarter, tot);
    load_wchunk<BITS, GROUP>(w0, a, wbase, ncol, kb + 2 * CH, kb_end);
    stage_store(lds, 1, xr);
    __syncthreads();
    stage_load(xr, a, kb + 2 * CH, kb_end);
    Body::compute(w1, lds, 1, kb + CH, kb_end, col, quarter, tot);
    load_wchunk<BITS, GROUP>(w1, a, wbase, ncol, kb + 3 * CH, kb_end);
    stage_store(lds, 0, xr);
    __syncthreads();
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
}

// ---------------------------------------------------------------------------
// GEMV kernel (M <= 8).  Workgroup = 4 wavefronts x NT tiles, one k-split.  The
// split's activations (ROWS x kspan bf16) and the per-quarter group sums of x are
// staged in LDS once; the main loop then streams weights without barriers.  Lane
// (quarter q, column c) accumulates its 8-k slices of every step with bf16 dot
// products; the four quarters are summed at the end (cross-row lane exchange).
// ---------------------------------------------------------------------------

constexpr int kGemvPieces = 8;  // 16-byte activation pieces staged per thread

// Dynamic LDS layout: x [ROWS][kspan + 8] bf16, then xsum [kspan/GROUP][ROWS][4] f32.
__host__ __device__ constexpr int gemv_x_stride(int kspan) { return kspan + 8; }
__host__ __device__ constexpr size_t gemv_xsum_offset(int rows, int kspan) {
  return (static_cast<size_t>(rows) * gemv_x_stride(kspan) * 2 + 15) / 16 * 16;
}
size_t gemv_lds_bytes(int rows, int kspan, int group) {
  return gemv_xsum_offset(rows, kspan) + static_cast<size_t>(kspan / group) * rows * 4 * 4;
}
int gemv_max_kspan(int rows) { return kThreadsPerBlock * kGemvPieces * 8 / rows; }

__device__ __forceinline__ float dot2_bf16(uint32_t xa, uint32_t wb, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, xa),
                                         __builtin_bit_cast(bf16x2_t, wb), acc, false);
}

template <int BITS, int GROUP, int ROWS, int NT, int CH>
struct GemvBody {
  static constexpr int GPB = kTileK / GROUP;
  static constexpr int SPG = 4 / GPB;
  static constexpr int GPC = CH * GPB;
  using W = WChunk<BITS, NT, CH, GPC>;

  // Consume one chunk: local blocks lb..lb+CH-1 of the split (nblk valid).
  static __device__ __forceinline__ void compute(const W& wc, const uint16_t* xl, const float* xsum,
                                                 int xs, int lb, int nblk, int quarter,
                                                 float (&tot)[ROWS][NT]) {
#pragma unroll
    for (int b = 0; b < CH; ++b) {
      if (lb + b < nblk) {
        uint32_t pr[NT][16];
#pragma unroll
        for (int t = 0; t < NT; ++t) unpack_pairs<BITS>(wc.w[b][t], pr[t]);
#pragma unroll
        for (int gi = 0; gi < GPB; ++gi) {
          const int gc = b * GPB + gi;
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
              const uint4 xv = *static_cast<const uint4*>(__builtin_assume_aligned(
                  xl + m * xs + (lb + b) * kTileK + 32 * j + 8 * quarter, 16));
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
          float sv[NT], cv[NT];
#pragma unroll
          for (int t = 0; t < NT; ++t) scale_and_offset(wc.s[gc][t], wc.z[gc][t], sv[t], cv[t]);
          const int g = (lb + b) * GPB + gi;  // group index within the split
#pragma unroll
          for (int m = 0; m < ROWS; ++m) {
            const float xq = xsum[(g * ROWS + m) * 4 + quarter];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
              const float v = __builtin_fmaf(sv[t], acc[m][t], tot[m][t]);
              tot[m][t] = __builtin_fmaf(-cv[t], xq, v);
            }
          }
        }
      }
    }
  }
};

template <int BITS, int GROUP, int ROWS, int NT, int CH>
__global__ __launch_bounds__(kThreadsPerBlock) void k_qgemv(QArgs a) {
  using Body = GemvBody<BITS, GROUP, ROWS, NT, CH>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int col = lane & 15, quarter = lane >> 4;
  const int ng = blockIdx.x / a.splits, split = blockIdx.x % a.splits;
  const int nt0 = (ng * kWavesPerBlock + wave) * NT;
  const int kb_begin = split * a.blocks_per_split;
  const int kb_end = min(a.KB, kb_begin + a.blocks_per_split);
  const int nblk = kb_end - kb_begin;
  const int nchunks = (nblk + CH - 1) / CH;
  const int kspan = a.blocks_per_split * kTileK;
  const int xs = gemv_x_stride(kspan);
  uint16_t* xl = reinterpret_cast<uint16_t*>(smem);
  float* xsum = reinterpret_cast<float*>(smem + gemv_xsum_offset(ROWS, kspan));

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

  // Start the weight stream before staging the activations.
  typename Body::W w0, w1;
  load_wchunk<BITS, GROUP>(w0, a, wbase, ncol, kb_begin, kb_end);
  load_wchunk<BITS, GROUP>(w1, a, wbase, ncol, kb_begin + CH, kb_end);

  // Stage x[0..ROWS)[split] (rows past M repeat row M-1 and are never stored).
  {
    const int p16 = nblk * 16;  // 16-byte pieces per row
    const int total = ROWS * p16;
    uint4 v[kGemvPieces];
#pragma unroll
    for (int p = 0; p < kGemvPieces; ++p) {
      const int i = min(p * kThreadsPerBlock + static_cast<int>(threadIdx.x), total - 1);
      const int row = min(i / p16, a.M - 1), c8 = i % p16;
      v[p] = *reinterpret_cast<const uint4*>(a.x + static_cast<size_t>(row) * a.K +
                                             static_cast<size_t>(kb_begin) * kTileK + c8 * 8);
    }
    constexpr int P8 = GROUP / 8;
#pragma unroll
    for (int p = 0; p < kGemvPieces; ++p) {
      const int i = p * kThreadsPerBlock + threadIdx.x;
      const int row = i / p16, c8 = i % p16;
      if (i < total) *reinterpret_cast<uint4*>(xl + row * xs + c8 * 8) = v[p];
      float s = ((bf16lo(v[p].x) + bf16hi(v[p].x)) + (bf16lo(v[p].y) + bf16hi(v[p].y))) +
                ((bf16lo(v[p].z) + bf16hi(v[p].z)) + (bf16lo(v[p].w) + bf16hi(v[p].w)));
      // quarter q of a group = pieces with c8 % 4 == q; the pieces of one (row,
      // block) are one aligned 16-lane row
      if constexpr (GROUP == 128) {
        s += dpp_f<kDppRowRor4>(s);
        s += dpp_f<kDppRowRor8>(s);
      } else {
        s += __shfl_xor(s, 4);
      }
      if (i < total && (c8 % P8) < 4) xsum[((c8 / P8) * ROWS + row) * 4 + (c8 % 4)] = s;
    }
  }
  __syncthreads();

  float tot[ROWS][NT];
#pragma unroll
  for (int m = 0; m < ROWS; ++m)
#pragma unroll
    for (int t = 0; t < NT; ++t) tot[m][t] = 0.f;

  // The refills are unconditional (clamped past the end of the split) so that the
  // loop body is straight-line and every wait on outstanding loads is exact: a
  // conditional refill would make the compiler wait for all loads in flight.
  for (int c = 0; c < nchunks; c += 2) {
    Body::compute(w0, xl, xsum, xs, c * CH, nblk, quarter, tot);
    load_wchunk<BITS, GROUP>(w0, a, wbase, ncol, kb_begin + (c + 2) * CH, kb_end);
    Body::compute(w1, xl, xsum, xs, (c + 1) * CH, nblk, quarter, tot);
    load_wchunk<BITS, GROUP>(w1, a, wbase, ncol, kb_begin + (c + 3) * CH, kb_end);
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
  const size_t lds = kc.path == 1 ? gemv_lds_bytes(kc.rows, a.blocks_per_split * kTileK, group) : 0;
  hipLaunchKernelGGL(fn, dim3(grid), dim3(kThreadsPerBlock), lds, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  const size_t quads = static_cast<size_t>(a.M) * a.N / 4;
  const unsigned rgrid = static_cast<unsigned>((quads + kThreadsPerBlock - 1) / kThreadsPerBlock);
  hipLaunchKernelGGL(k_splitk_reduce, dim3(rgrid), dim3(kThreadsPerBlock), 0, st, a.ws, a.y, a.M,
                     a.N, a.splits);
  return hipGetLastError();
}

}  // namespace subspec
