// The substitute-layer linear y = x * dequant(q, s, z)^T (SubSpec Sec. 4.1) for
// draft-tree batches, as two kernels over one packed layout:
//
//   k_qgemv       small M.  VALU bf16 dot products; the four 16-lane quarters of a
//                 wavefront split K inside every tile and are summed with cross-row
//                 lane exchanges at the end.
//   k_qgemm_mfma  any M.  16x16x32 bf16 MFMA; the A operand (activations) comes
//                 from LDS, the B operand straight from the unpacked codes.
//
// Both split K across workgroups when a projection has too few columns to fill the
// GPU; the last workgroup of a column group to finish adds the fp32 partial sums in
// split order (finish_splitk).
//
// Dequantization is folded into the accumulation.  Within one group the weight is
// affine in the code, W^ = s*(q - z), so for every (row m, column n, group g)
//     sum_{k in g} x*W^ = s * ( sum_{k in g} x*(128+q) - (128+z) * sum_{k in g} x ).
// The kernels feed the exact bf16 values 128+q (one and-or per code pair, see
// device_common.h) to the dot products / matrix cores and apply s and z once per
// (m, n, g).  The effective weights are the exact dequantized values; the only
// roundings are the fp32 accumulation and the final bf16 store.
#include "qlinear_device.h"

namespace subspec {

// ---------------------------------------------------------------------------
// Activation staging.  The unit of work is a "span": 32 consecutive k of one row
// (four 16-byte pieces) read by one thread, so that the thread can sum its own
// values; the spans of one group of k are G/32 consecutive threads (2 or 4 lanes of
// one DPP quad) and are reduced with one or two quad permutes.  Piece p of a span
// holds the k with k % 32 in [8p, 8p+8): the slice of a group one 16-lane quarter
// of a wavefront multiplies (quarter p).
//
// Loads are unconditional: out-of-range spans read a clamped (valid) address and
// are never consumed (blocks past the split are skipped, rows past M never stored),
// so no branch -- and no early wait on outstanding loads -- surrounds them.
// ---------------------------------------------------------------------------

template <int SPANS_PER_THREAD>
struct SpanRegs {
  u32x4_t v[SPANS_PER_THREAD][4];
};

// Load spans i = p*THREADS + tid (p < SPT) of a rows x (nblk blocks) region starting
// at block kb; a row holds nblk*4 spans.
template <int SPT, int THREADS>
__device__ __forceinline__ void load_spans(SpanRegs<SPT>& r, const QArgs& a, int kb, int kb_end,
                                           int spans_per_row, int total) {
#pragma unroll
  for (int p = 0; p < SPT; ++p) {
    const int i = min(p * THREADS + static_cast<int>(threadIdx.x), total - 1);
    const int row = min(i / spans_per_row, a.M - 1);
    const int sp = i % spans_per_row;
    const int kbc = min(kb + sp / 4, kb_end - 1);
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(a.x + static_cast<size_t>(row) * a.K +
                                                          static_cast<size_t>(kbc) * kTileK +
                                                          (sp % 4) * 32);
#pragma unroll
    for (int q = 0; q < 4; ++q) r.v[p][q] = src[q];
  }
}

// ---------------------------------------------------------------------------
// MFMA kernel.  Workgroup = WAVES wavefronts x NT tiles, all rows, one k-split.  Per
// chunk of CH blocks, x is copied to LDS (double buffered, one barrier per chunk);
// each wavefront unpacks its tiles' codes straight into B operands and runs
// 16x16x32 bf16 MFMAs against A fragments read from LDS.
//
// The zero-point term needs the per-group sums of x.  They are the same for every
// wavefront, so each row tile has one owner wavefront (row tile mt belongs to
// wavefront mt % WAVES) that runs one more MFMA per A fragment with an all-ones B
// operand -- the sums land in the accumulator layout -- and publishes them in LDS.
// They are visible to the other wavefronts after the chunk's barrier, so the term
// -c * sum(x) of a chunk is applied at the start of the next one (the offsets c of
// the chunk are kept in registers until then).
//
// LDS layout of a chunk: 16-byte pieces, row-major [row][block][piece], the 16
// pieces of each (row, block) permuted by piece ^ (row & 15).  Copy-in writes the 16
// pieces of one row per 16 lanes and an A fragment reads one piece of 16 consecutive
// rows per 16 lanes: either way the 16 lanes touch all 64 banks once.
//
// All global reads go through buffer resources: 32-bit offsets from a scalar base,
// and rows past M (offsets past the end of x) read zeros.  Blocks past the split
// read whatever lies there and are never consumed.
// ---------------------------------------------------------------------------

template <int ROWS, int CH, int GPC>
struct MfmaLds {
  u32x4_t x[2][ROWS * CH * 16];
  float xs[2][GPC][ROWS];  // per-group sums of x of the chunk in the same buffer
  f32x4_t sink[kWave];     // target of the lanes that do not publish sums
};


template <int BITS, int GROUP, int MT, int NT, int CH, int WAVES>
struct MfmaBody {
  static constexpr int ROWS = 16 * MT;
  static constexpr int THREADS = WAVES * kWave;
  static constexpr int GPB = kTileK / GROUP;  // groups per block
  static constexpr int SPG = 4 / GPB;         // 32-k steps per group
  static constexpr int GPC = CH * GPB;        // groups per chunk
  static constexpr int PIECES = ROWS * CH * 16;
  static constexpr int PPT = PIECES / THREADS;  // pieces per thread per chunk
  // A-fragment prefetch (see compute) for two or four row tiles with one tile per
  // wavefront: measured -1.7 us on the 7B gate|up at M = 64 and -1 us on down at
  // M = 32.  The two-tile and eight-row-tile variants would need more than 256 VGPRs
  // with it (one wavefront per SIMD), and the one-row-tile one gains nothing.
  static constexpr bool kPrefetchA = (MT == 2 || MT == 4) && NT == 1;
  static_assert(PIECES % THREADS == 0, "a chunk is a whole number of pieces per thread");
  using Lds = MfmaLds<ROWS, CH, GPC>;
  struct W {
    Slice<BITS> w[CH][NT];
    uint32_t s[GPC][NT];  // fp16 bits of the scale
    uint32_t z[GPC][NT];  // fp16 bits of the zero-point
  };
  struct X {
    u32x4_t v[PPT];
  };

  static __device__ __forceinline__ int slot(int row, int b, int piece) {
    return row * (CH * 16) + b * 16 + (piece ^ (row & 15));
  }

  // Weights of blocks kb..kb+CH-1 for the wavefront's tiles; wofs[t] is the byte
  // offset of the lane's slice in block 0 of tile t, col[t] its column.
  static __device__ __forceinline__ void load_w(W& r, const QBuffers& bu, const QArgs& a,
                                                const uint32_t (&wofs)[NT], const int (&col)[NT],
                                                int kb) {
#pragma unroll
    for (int b = 0; b < CH; ++b)
#pragma unroll
      for (int t = 0; t < NT; ++t)
        r.w[b][t] = load_slice<BITS>(bu.w, wofs[t] + static_cast<uint32_t>(kb + b) * (256 * BITS));
#pragma unroll
    for (int gc = 0; gc < GPC; ++gc)
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const uint32_t off = (static_cast<uint32_t>(kb * GPB + gc) * a.N + col[t]) * 2;
        r.s[gc][t] = __builtin_amdgcn_raw_buffer_load_b16(bu.s, off, 0, 0);
        r.z[gc][t] = __builtin_amdgcn_raw_buffer_load_b16(bu.z, off, 0, 0);
      }
  }

  // Coalesced copy of chunk (rows x blocks kb..kb+CH-1) into registers.
  static __device__ __forceinline__ void stage_load(X& r, const QBuffers& bu, int K, int kb) {
#pragma unroll
    for (int p = 0; p < PPT; ++p) {
      const int P = p * THREADS + threadIdx.x;
      const int row = P / (CH * 16), b = (P / 16) % CH, pc = P % 16;
      const uint32_t off =
          (static_cast<uint32_t>(row) * K + static_cast<uint32_t>(kb + b) * kTileK + pc * 8) * 2;
      r.v[p] = __builtin_amdgcn_raw_buffer_load_b128(bu.x, off, 0, 0);
    }
  }

  static __device__ __forceinline__ void stage_store(Lds& L, int buf, const X& r) {
#pragma unroll
    for (int p = 0; p < PPT; ++p) {
      const int P = p * THREADS + threadIdx.x;
      const int row = P / (CH * 16), b = (P / 16) % CH, pc = P % 16;
      L.x[buf][slot(row, b, pc)] = r.v[p];
    }
  }

  // The zero-point term of the previous chunk (LDS buffer buf, first block kb):
  // tot -= c * sum(x) with the offsets c kept from that chunk.
  template <bool FULL>
  static __device__ __forceinline__ void correct(const Lds& L, int buf, int kb, int kb_end, int lane,
                                                 const float (&cprev)[GPC][NT],
                                                 f32x4_t (&tot)[MT][NT]) {
    const int quarter = lane >> 4;
#pragma unroll
    for (int b = 0; b < CH; ++b) {
      if (FULL || kb + b < kb_end) {
#pragma unroll
        for (int gi = 0; gi < GPB; ++gi) {
          const int gc = b * GPB + gi;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const f32x4_t xv = *reinterpret_cast<const f32x4_t*>(&L.xs[buf][gc][16 * mt + 4 * quarter]);
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
              for (int r = 0; r < 4; ++r) tot[mt][t][r] = __builtin_fmaf(-cprev[gc][t], xv[r], tot[mt][t][r]);
          }
        }
      }
    }
  }

  // Consume one chunk (blocks kb..kb+CH-1 of the split, LDS buffer buf): MFMAs per
  // group with the k-steps outermost, so the MT*NT accumulators of a group form
  // independent chains; tot += s * acc when the group is complete.  The wavefront
  // with index DW also sums x over its row tiles DW, DW+WAVES, ... (one ones-MFMA
  // per A fragment it reads anyway) and publishes the group's sums; DW = -1 for a
  // wavefront that owns no row tile.  cnext receives the chunk's offsets c.
  template <bool FULL, int DW>
  static __device__ __forceinline__ void compute(const W& wc, Lds& L, int buf, int kb, int kb_end,
                                                 int lane, f32x4_t (&tot)[MT][NT],
                                                 float (&cnext)[GPC][NT]) {
    constexpr int DUTY = DW < 0 ? 0 : (MT - DW + WAVES - 1) / WAVES;
    const int col = lane & 15, quarter = lane >> 4;
    const bf16x8_t ones = __builtin_bit_cast(
        bf16x8_t, make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u));
    const f32x4_t zero = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int b = 0; b < CH; ++b) {
      if (FULL || kb + b < kb_end) {
        uint32_t pr[NT][16];
#pragma unroll
        for (int t = 0; t < NT; ++t) unpack_pairs<BITS>(wc.w[b][t], pr[t]);
#pragma unroll
        for (int gi = 0; gi < GPB; ++gi) {
          const int gc = b * GPB + gi;
          f32x4_t acc[MT][NT], accx[DUTY > 0 ? DUTY : 1];
          // The group's MFMAs run at raised wave priority, so the other wavefront on
          // the SIMD tends to be in its VALU part (unpack, scale FMAs) meanwhile: the
          // two otherwise fall into step and their MFMA and VALU time add up.
          // Measured: -1.3 us (gate|up M = 64), -1.6 us (down M = 64), -0.7 us (down
          // M = 8, 32); with two row tiles and two tiles per wavefront it cost 1.2 us
          // (gate|up M = 32), so that variant keeps the normal priority.
          constexpr bool kRaisePrio = !(MT == 2 && NT == 2);
          if constexpr (kRaisePrio) __builtin_amdgcn_s_setprio(1);
          // With kPrefetchA the A fragments of the next 32-k step are read before the
          // MFMAs of the current one, and scheduling fences keep the compiler from
          // sinking those reads back next to their first use, so the LDS latency runs
          // under four or eight MFMAs instead of stalling the wavefront.
          bf16x8_t Acur[MT];
          if constexpr (kPrefetchA) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
              Acur[mt] = __builtin_bit_cast(bf16x8_t, L.x[buf][slot(16 * mt + col, b, 4 * (gi * SPG) + quarter)]);
          }
#pragma unroll
          for (int js = 0; js < SPG; ++js) {
            const int j = gi * SPG + js;
            bf16x8_t Anext[MT];
            if constexpr (kPrefetchA) {
              if (js + 1 < SPG) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                  Anext[mt] = __builtin_bit_cast(bf16x8_t, L.x[buf][slot(16 * mt + col, b, 4 * (j + 1) + quarter)]);
              }
              __builtin_amdgcn_sched_barrier(0);
            }
            static_for<MT>([&](auto mtc) __attribute__((always_inline)) {
              constexpr int mt = decltype(mtc)::value;
              const bf16x8_t A = kPrefetchA ? Acur[mt]
                                            : __builtin_bit_cast(bf16x8_t, L.x[buf][slot(16 * mt + col, b, 4 * j + quarter)]);
#pragma unroll
              for (int t = 0; t < NT; ++t) {
                const uint4 bw = make_uint4(pr[t][4 * j], pr[t][4 * j + 1], pr[t][4 * j + 2],
                                            pr[t][4 * j + 3]);
                const bf16x8_t B = __builtin_bit_cast(bf16x8_t, bw);
                acc[mt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    A, B, js == 0 ? zero : acc[mt][t], 0, 0, 0);
              }
              if constexpr (DW >= 0 && mt % WAVES == DW) {
                constexpr int i = mt / WAVES;
                accx[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, ones, js == 0 ? zero : accx[i],
                                                                  0, 0, 0);
              }
            });
            if constexpr (kPrefetchA) {
              __builtin_amdgcn_sched_barrier(0);
              if (js + 1 < SPG) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) Acur[mt] = Anext[mt];
              }
            }
          }
          if constexpr (kRaisePrio) __builtin_amdgcn_s_setprio(0);
          float sv[NT];
#pragma unroll
          for (int t = 0; t < NT; ++t) scale_and_offset(wc.s[gc][t], wc.z[gc][t], sv[t], cnext[gc][t]);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
              for (int r = 0; r < 4; ++r) tot[mt][t][r] = __builtin_fmaf(sv[t], acc[mt][t][r], tot[mt][t][r]);
#pragma unroll
          for (int i = 0; i < DUTY; ++i) {
            // all 16 columns hold the same sums; lanes of column 0 publish them
            f32x4_t* dst = col == 0 ? reinterpret_cast<f32x4_t*>(&L.xs[buf][gc][16 * (DW + WAVES * i) + 4 * quarter])
                                    : &L.sink[lane];
            *dst = accx[i];
          }
        }
      }
    }
  }
};

// Register budget: with four row tiles and one tile per wavefront the kernel is held
// to three wavefronts per SIMD (at most 168 VGPRs; left alone the compiler lands on
// either side of that line), which the planner's residency-aware choices count on.
// The smaller variants fit four or more by themselves.
template <int MT, int NT>
constexpr int mfma_min_waves() {
  return MT == 4 && NT == 1 ? 3 : 1;
}

template <int BITS, int GROUP, int MT, int NT, int CH, int WAVES, int PF>
__global__ __launch_bounds__(WAVES * kWave) __attribute__((amdgpu_waves_per_eu(mfma_min_waves<MT, NT>())))
void k_qgemm_mfma(QArgs args) {
  const QArgs a = row_block(args);
  static_assert(PF % 2 == 0, "the LDS buffer of a chunk follows the ring slot's parity");
  using Body = MfmaBody<BITS, GROUP, MT, NT, CH, WAVES>;
  constexpr int GPC = Body::GPC;
  __shared__ typename Body::Lds lds;

  const int lane = threadIdx.x % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x / kWave));
  const WorkItem wi(a);
  const int ng = wi.ng, kb0 = wi.kb0, kb_end = wi.kb_end;
  const int nchunks = (kb_end - kb0 + CH - 1) / CH;
  const QBuffers bu(a, BITS, GROUP);

  bool ok[NT];
  int col[NT];
  uint32_t wofs[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int nt = (ng * WAVES + wave) * NT + t;
    ok[t] = nt < a.n_tiles;
    const int ntc = ok[t] ? nt : 0;
    col[t] = ntc * kTileN + (lane & 15);
    wofs[t] = static_cast<uint32_t>(ntc) * a.KB * (256 * BITS) + lane * (4 * BITS);
  }

  f32x4_t tot[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int t = 0; t < NT; ++t) tot[mt][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float cprev[GPC][NT];

  // Weights and activations: rings of PF chunks each, refilled in the same order
  // (weights of chunk c+PF, then activations of chunk c+1+PF), so every load is
  // issued PF chunks before it is waited for.  Loads complete in issue order: an
  // activation ring shallower than the weight ring would cap the weights' lead too.
  // Loads of chunks past the split repeat its last chunk (L2 hits, never consumed),
  // so a split shorter than the ring costs no extra memory traffic.
  typename Body::W w[PF];
  typename Body::X x[PF];
  const int kb_last = kb0 + (nchunks - 1) * CH;
  static_for<PF>([&](auto u) __attribute__((always_inline)) {
    Body::load_w(w[u.value], bu, a, wofs, col, min(kb0 + u.value * CH, kb_last));
    Body::stage_load(x[u.value], bu, a.K, min(kb0 + u.value * CH, kb_last));
  });
  Body::stage_store(lds, 0, x[0]);
  Body::stage_load(x[0], bu, a.K, min(kb0 + PF * CH, kb_last));
  // The first chunk's zero-point step reads the sums of "chunk -1": zeros, with
  // zero offsets.
  for (int i = threadIdx.x; i < GPC * Body::ROWS; i += WAVES * kWave) (&lds.xs[1][0][0])[i] = 0.f;
#pragma unroll
  for (int gc = 0; gc < GPC; ++gc)
#pragma unroll
    for (int t = 0; t < NT; ++t) cprev[gc][t] = 0.f;
  __syncthreads();

  // The main loop, for a wavefront whose duty is DW (see MfmaBody::compute).
  auto run = [&](auto dwc) __attribute__((always_inline)) {
    constexpr int DW = decltype(dwc)::value;
    // One chunk: ring slot U holds chunk c+U; the LDS buffer follows the chunk's
    // parity (PF is even).  REFILL = false in the drain.  Every chunk of the steady
    // state is whole (only the split's last one can be partial), so it runs without
    // bounds checks.
    auto step = [&](auto u, int c, auto refill) __attribute__((always_inline)) {
      constexpr int U = decltype(u)::value;
      constexpr int V = (U + 1) % PF;  // slot of chunk c+U+1
      constexpr bool FULL = decltype(refill)::value;
      const int kb = kb0 + (c + U) * CH;
      if constexpr (MT == 1) {
        // One row tile: the MFMAs of the chunk go first and the previous chunk's
        // zero-point term fills their latency (measured faster at M = 8; with more
        // row tiles the MFMA sequence is long enough on its own, and the order there
        // is the other way round).
        float cp[GPC][NT];
#pragma unroll
        for (int g = 0; g < GPC; ++g)
#pragma unroll
          for (int t = 0; t < NT; ++t) cp[g][t] = cprev[g][t];
        Body::template compute<FULL, DW>(w[U], lds, U & 1, kb, kb_end, lane, tot, cprev);
        Body::template correct<FULL>(lds, (U + 1) & 1, kb - CH, kb_end, lane, cp, tot);
      } else {
        Body::template correct<FULL>(lds, (U + 1) & 1, kb - CH, kb_end, lane, cprev, tot);
        Body::template compute<FULL, DW>(w[U], lds, U & 1, kb, kb_end, lane, tot, cprev);
      }
      if constexpr (FULL) Body::load_w(w[U], bu, a, wofs, col, min(kb + PF * CH, kb_last));
      Body::stage_store(lds, (U + 1) & 1, x[V]);
      if constexpr (FULL) Body::stage_load(x[V], bu, a.K, min(kb + (PF + 1) * CH, kb_last));
      __syncthreads();
    };
    // Steady state: straight-line body (every load unconditional) so that each wait
    // on outstanding loads is exact.  Then drain the last (at most PF) chunks without
    // further loads, and apply the last chunk's zero-point term.
    int c = 0;
    for (; c + PF < nchunks; c += PF)
      static_for<PF>([&](auto u) __attribute__((always_inline)) { step(u, c, std::true_type{}); });
    static_for<PF>([&](auto u) __attribute__((always_inline)) { step(u, c, std::false_type{}); });
    Body::template correct<false>(lds, (PF - 1) & 1, kb0 + (c + PF - 1) * CH, kb_end, lane, cprev, tot);
  };
  // A wavefront's duty is a compile-time property of the code it runs, so the duty
  // MFMAs reuse the A fragments of the regular ones: one copy of the main loop per
  // owner wavefront, and one for the wavefronts that own no row tile.
  if constexpr (MT >= WAVES) {
    static_for<WAVES>([&](auto wc) __attribute__((always_inline)) {
      if (wave == decltype(wc)::value) run(wc);
    });
  } else {
    static_for<MT>([&](auto wc) __attribute__((always_inline)) {
      if (wave == decltype(wc)::value) run(wc);
    });
    if (wave >= MT) run(std::integral_constant<int, -1>{});
  }

  // D layout of 16x16 MFMA: lane holds column lane%16, rows 4*(lane/16) + r.  The
  // stores go through a buffer resource over the output (bf16 y, or this split's fp32
  // partial sums) with the whole offset in the vector offset, which the range check
  // covers: rows at or past M and the lanes of a tile past N (given an offset outside
  // the resource) are dropped.  All offsets stay below 2^31 when the tile's rows span
  // less than 2 GiB; larger outputs take per-element stores.
  const int quarter = lane >> 4;
  const bool split = wi.nsplit > 1;
  const uint32_t esz = split ? 4 : 2;
  if (static_cast<uint64_t>(16 * MT) * a.N * esz < (1ull << 31)) {
    const uint32_t rowb = static_cast<uint32_t>(a.N) * esz;
    const uint32_t out_bytes = static_cast<uint32_t>(a.M) * rowb;
    const __amdgpu_buffer_rsrc_t out =
        split ? buffer_rsrc(a.ws + static_cast<size_t>(wi.split) * a.M * a.N, out_bytes) : buffer_rsrc(a.y, out_bytes);
    constexpr uint32_t kOutside = 0x80000000u;
    uint32_t voff[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
      voff[t] = ok[t] ? static_cast<uint32_t>(col[t]) * esz + static_cast<uint32_t>(4 * quarter) * rowb : kOutside;
    auto store_all = [&](auto splitc) __attribute__((always_inline)) {
      constexpr bool SPLIT = decltype(splitc)::value;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const uint32_t off = voff[t] + static_cast<uint32_t>(16 * mt + r) * rowb;
            const float v = tot[mt][t][r];  // a plain value: bit casts of a vector element misbehave
            if constexpr (SPLIT)
              __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), out, off, 0, kCachePolicyAgent);
            else
              __builtin_amdgcn_raw_buffer_store_b16(float_to_bf16_bits(v), out, off, 0, 0);
          }
    };
    if (split)
      store_all(std::true_type{});
    else
      store_all(std::false_type{});
  } else {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = 16 * mt + 4 * quarter + r;
          if (ok[t] && m < a.M) store_out(a, wi, m, col[t], tot[mt][t][r]);
        }
  }
  if (wi.nsplit > 1) finish_splitk<WAVES * kWave>(a, ng, WAVES * NT * kTileN);
}

// ---------------------------------------------------------------------------
// GEMV kernel (small M).  Workgroup = WAVES wavefronts x NT tiles, one k-split.  The
// split's activations (ROWS x kspan bf16) and the per-quarter group sums of x are
// staged in LDS once; the main loop then streams weights without barriers.  Lane
// (quarter q, column c) accumulates its 8-k slices of every step with bf16 dot
// products; the four quarters are summed at the end (cross-row lane exchange).
// ---------------------------------------------------------------------------

constexpr int kGemvSpans = 2;  // 32-k activation spans staged per thread
constexpr size_t kGemvLdsBudget = 48 * 1024;  // dynamic LDS per workgroup (3 fit a CU)
constexpr int kGemvSzRounds = 2;  // (group, 8-column) scale pieces staged per thread

// Dynamic LDS layout: x [ROWS][kspan + 8] bf16, xsum [kspan/GROUP][ROWS][4] f32, then
// sc [kspan/GROUP][cols] (s, c = s * (128 + z)) f32 pairs for the workgroup's columns.
__host__ __device__ constexpr int gemv_x_stride(int kspan) { return kspan + 8; }
__host__ __device__ constexpr size_t gemv_xsum_offset(int rows, int kspan) {
  return (static_cast<size_t>(rows) * gemv_x_stride(kspan) * 2 + 15) / 16 * 16;
}
__host__ __device__ constexpr size_t gemv_sc_offset(int rows, int kspan, int group) {
  return gemv_xsum_offset(rows, kspan) + static_cast<size_t>(kspan / group) * rows * 4 * 4;
}
size_t gemv_lds_bytes(int rows, int kspan, int group, int cols) {
  return gemv_sc_offset(rows, kspan, group) + static_cast<size_t>(kspan / group) * cols * 8;
}
int gemv_max_kspan(int rows, int waves, int group, int cols) {
  const int staged = waves * kWave * kGemvSpans * 32 / rows;  // what the prologue copies
  const size_t per_block = gemv_lds_bytes(rows, kTileK, group, cols) - 16;  // bytes per 128 k
  const int fit = static_cast<int>((kGemvLdsBudget - 16) / per_block) * kTileK;
  const int sz_groups = kGemvSzRounds * waves * kWave / (cols / 8);  // scale pieces staged
  const int sz_fit = sz_groups / (kTileK / group) * kTileK;
  return min(min(staged, sz_fit), max(fit, kTileK));
}

template <int BITS, int NT, int CH>
struct GemvW {
  Slice<BITS> w[CH][NT];
};

template <int BITS, int GROUP, int ROWS, int NT, int CH>
struct GemvBody {
  static constexpr int GPB = kTileK / GROUP;
  static constexpr int SPG = 4 / GPB;
  using W = GemvW<BITS, NT, CH>;

  // Weights of local blocks kb..kb+CH-1 (buffer loads; blocks past the split read
  // the next data and are never consumed).
  static __device__ __forceinline__ void load(W& r, __amdgpu_buffer_rsrc_t wr,
                                              const uint32_t (&wofs)[NT], int kb) {
#pragma unroll
    for (int b = 0; b < CH; ++b)
#pragma unroll
      for (int t = 0; t < NT; ++t)
        r.w[b][t] = load_slice<BITS>(wr, wofs[t] + static_cast<uint32_t>(kb + b) * (256 * BITS));
  }

  // Consume one chunk: local blocks lb..lb+CH-1 of the split (nblk valid).
  static __device__ __forceinline__ void compute(const W& wc, const uint16_t* xl, const float* xsum,
                                                 const float2* sc, int xs, int cols, int lb,
                                                 int nblk, int quarter, const int (&lcol)[NT],
                                                 float (&tot)[ROWS][NT]) {
#pragma unroll
    for (int b = 0; b < CH; ++b) {
      if (lb + b < nblk) {
        uint32_t pr[NT][16];
#pragma unroll
        for (int t = 0; t < NT; ++t) unpack_pairs<BITS>(wc.w[b][t], pr[t]);
#pragma unroll
        for (int gi = 0; gi < GPB; ++gi) {
          float acc[ROWS][NT], acc2[ROWS][NT];
#pragma unroll
          for (int m = 0; m < ROWS; ++m)
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[m][t] = acc2[m][t] = 0.f;
#pragma unroll
          for (int js = 0; js < SPG; ++js) {
            const int j = gi * SPG + js;
#pragma unroll
            for (int m = 0; m < ROWS; ++m) {
              const uint4 xv = *static_cast<const uint4*>(__builtin_assume_aligned(
                  xl + m * xs + (lb + b) * kTileK + 32 * j + 8 * quarter, 16));
#pragma unroll
              for (int t = 0; t < NT; ++t) {
                // two chains per (row, tile) halve the dependent dot-product latency
                float v0 = acc[m][t], v1 = acc2[m][t];
                v0 = dot2_bf16(xv.x, pr[t][4 * j + 0], v0);
                v1 = dot2_bf16(xv.y, pr[t][4 * j + 1], v1);
                v0 = dot2_bf16(xv.z, pr[t][4 * j + 2], v0);
                v1 = dot2_bf16(xv.w, pr[t][4 * j + 3], v1);
                acc[m][t] = v0;
                acc2[m][t] = v1;
              }
            }
          }
          const int g = (lb + b) * GPB + gi;  // group index within the split
          float2 scv[NT];
#pragma unroll
          for (int t = 0; t < NT; ++t) scv[t] = sc[g * cols + lcol[t]];
#pragma unroll
          for (int m = 0; m < ROWS; ++m) {
            const float xq = xsum[(g * ROWS + m) * 4 + quarter];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
              const float v = __builtin_fmaf(scv[t].x, acc[m][t] + acc2[m][t], tot[m][t]);
              tot[m][t] = __builtin_fmaf(-scv[t].y, xq, v);
            }
          }
        }
      }
    }
  }
};

template <int BITS, int GROUP, int ROWS, int NT, int CH, int WAVES, int PF>
__global__ __launch_bounds__(WAVES * kWave) void k_qgemv(QArgs a) {
  constexpr int THREADS = WAVES * kWave;
  constexpr int COLS = WAVES * NT * kTileN;
  constexpr int GPB = kTileK / GROUP;
  using Body = GemvBody<BITS, GROUP, ROWS, NT, CH>;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int quarter = lane >> 4;
  const WorkItem wi(a);
  const int ng = wi.ng, kb0 = wi.kb0, kb_end = wi.kb_end;
  const int nblk = kb_end - kb0;
  const int nchunks = (nblk + CH - 1) / CH;
  const int kspan = a.span_blocks * kTileK;  // LDS layout: the launch's largest span
  const int xs = gemv_x_stride(kspan);
  uint16_t* xl = reinterpret_cast<uint16_t*>(smem);
  float* xsum = reinterpret_cast<float*>(smem + gemv_xsum_offset(ROWS, kspan));
  float2* sc = reinterpret_cast<float2*>(smem + gemv_sc_offset(ROWS, kspan, GROUP));
  const QBuffers bu(a, BITS, GROUP);
  const int n0 = ng * COLS;

  bool ok[NT];
  int col[NT], lcol[NT];
  uint32_t wofs[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int nt = (ng * WAVES + wave) * NT + t;
    ok[t] = nt < a.n_tiles;
    const int ntc = ok[t] ? nt : 0;
    col[t] = ntc * kTileN + (lane & 15);
    lcol[t] = (wave * NT + t) * kTileN + (lane & 15);
    wofs[t] = (static_cast<uint32_t>(ntc) * a.KB + kb0) * (256 * BITS) + lane * (4 * BITS);
  }

  typename Body::W w[PF];
  u32x4_t szs[kGemvSzRounds], szz[kGemvSzRounds];
  // Stage x[0..ROWS)[split] (rows past M repeat row M-1 and are never stored) and the
  // per-quarter group sums: piece q of a span is the quarter-q slice of its 32 k.
  {
    constexpr int SPAN_G = GROUP / 32;
    const int spans_per_row = nblk * 4;
    const int total = ROWS * spans_per_row;
    SpanRegs<kGemvSpans> r;
    load_spans<kGemvSpans, THREADS>(r, a, kb0, kb_end, spans_per_row, total);
    // Scales and zero-points of the split's groups for the workgroup's columns: one
    // (group, 8 columns) piece of s and of z per thread and round, 16-byte loads.
    const int ngroups = nblk * GPB;
#pragma unroll
    for (int p = 0; p < kGemvSzRounds; ++p) {
      const int q = min(p * THREADS + static_cast<int>(threadIdx.x), ngroups * (COLS / 8) - 1);
      const int g = q / (COLS / 8), c8 = q % (COLS / 8);
      const uint32_t off = (static_cast<uint32_t>(kb0 * GPB + g) * a.N + n0 + 8 * c8) * 2;
      szs[p] = __builtin_amdgcn_raw_buffer_load_b128(bu.s, off, 0, 0);
      szz[p] = __builtin_amdgcn_raw_buffer_load_b128(bu.z, off, 0, 0);
    }
    // The whole weight ring is issued right after these (small) loads: they complete
    // in issue order, so the activations still return first, and a short split then
    // waits for one memory latency instead of one per ring refill.  Chunks past the
    // split repeat its last one (L2 hits, never consumed).
    static_for<PF>([&](auto u) __attribute__((always_inline)) {
      Body::load(w[u.value], bu.w, wofs, min(u.value, nchunks - 1) * CH);
    });
#pragma unroll
    for (int p = 0; p < kGemvSpans; ++p) {
      const int i = p * THREADS + threadIdx.x;
      const int row = i / spans_per_row, sp = i % spans_per_row;
      float qs[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) qs[q] = span_reduce<SPAN_G>(piece_sum(r.v[p][q], 0.f));
      if (i < total) {
        u32x4_t* dst = reinterpret_cast<u32x4_t*>(xl + row * xs + sp * 32);
#pragma unroll
        for (int q = 0; q < 4; ++q) dst[q] = r.v[p][q];
        if (sp % SPAN_G == 0)
          *reinterpret_cast<float4*>(xsum + ((sp / SPAN_G) * ROWS + row) * 4) =
              make_float4(qs[0], qs[1], qs[2], qs[3]);
      }
    }
    // Scales and offsets (s, c = s * (128 + z)) of the loaded pieces.
#pragma unroll
    for (int p = 0; p < kGemvSzRounds; ++p) {
      const int q = p * THREADS + threadIdx.x;
      if (q < ngroups * (COLS / 8)) {
        const int g = q / (COLS / 8), c8 = q % (COLS / 8);
        float4* dst = reinterpret_cast<float4*>(sc + g * COLS + 8 * c8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float s0 = half_bits_to_float(static_cast<uint16_t>(szs[p][e]));
          const float s1 = half_bits_to_float(static_cast<uint16_t>(szs[p][e] >> 16));
          const float z0 = half_bits_to_float(static_cast<uint16_t>(szz[p][e]));
          const float z1 = half_bits_to_float(static_cast<uint16_t>(szz[p][e] >> 16));
          dst[e] = make_float4(s0, s0 * (kCodeBias + z0), s1, s1 * (kCodeBias + z1));
        }
      }
    }
  }
  __syncthreads();

  float tot[ROWS][NT];
#pragma unroll
  for (int m = 0; m < ROWS; ++m)
#pragma unroll
    for (int t = 0; t < NT; ++t) tot[m][t] = 0.f;

  // Steady state with unconditional refills, then a load-free drain.
  int c = 0;
  for (; c + PF < nchunks; c += PF) {
    static_for<PF>([&](auto u) __attribute__((always_inline)) {
      constexpr int U = decltype(u)::value;
      Body::compute(w[U], xl, xsum, sc, xs, COLS, (c + U) * CH, nblk, quarter, lcol, tot);
      Body::load(w[U], bu.w, wofs, min(c + U + PF, nchunks - 1) * CH);
    });
  }
  static_for<PF>([&](auto u) __attribute__((always_inline)) {
    Body::compute(w[decltype(u)::value], xl, xsum, sc, xs, COLS, (c + decltype(u)::value) * CH, nblk,
                  quarter, lcol, tot);
  });

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
      if (ok[t] && (m & 3) == quarter && m < a.M) store_out(a, wi, m, col[t], tot[m][t]);
  if (wi.nsplit > 1) finish_splitk<THREADS>(a, ng, COLS);
}

// ---------------------------------------------------------------------------
// Dispatch table.
// ---------------------------------------------------------------------------

typedef void (*QKernel)(QArgs);

struct Variant {
  int path, rows, nt, chunk, waves, prefetch, bits, group;
  QKernel fn;
};

#define SUBSPEC_GEMV(B, G, R, T, C, W, P) {1, R, T, C, W, P, B, G, k_qgemv<B, G, R, T, C, W, P>}
#define SUBSPEC_MFMA(B, G, MT, T, C, W, P) \
  {2, 16 * MT, T, C, W, P, B, G, k_qgemm_mfma<B, G, MT, T, C, W, P>}
#define SUBSPEC_BG(X) X(4, 128) X(4, 64) X(3, 128) X(3, 64) X(2, 128) X(2, 64)
#define SUBSPEC_GEMV_SET(B, G)                                                                \
  SUBSPEC_GEMV(B, G, 1, 1, 2, 4, 2), SUBSPEC_GEMV(B, G, 2, 1, 2, 4, 2),                       \
      SUBSPEC_GEMV(B, G, 4, 1, 4, 4, 2), SUBSPEC_GEMV(B, G, 8, 1, 4, 4, 2),
#define SUBSPEC_MFMA_SET(B, G)                                                                \
  SUBSPEC_MFMA(B, G, 1, 1, 2, 4, 2), SUBSPEC_MFMA(B, G, 1, 2, 2, 4, 2),                       \
      SUBSPEC_MFMA(B, G, 2, 1, 1, 4, 2), SUBSPEC_MFMA(B, G, 2, 2, 1, 4, 2),                   \
      SUBSPEC_MFMA(B, G, 4, 1, 1, 4, 2), SUBSPEC_MFMA(B, G, 4, 2, 1, 4, 4),                   \
      SUBSPEC_MFMA(B, G, 8, 1, 1, 4, 2), SUBSPEC_MFMA(B, G, 8, 2, 1, 4, 2),

static const Variant kVariants[] = {SUBSPEC_BG(SUBSPEC_GEMV_SET) SUBSPEC_BG(SUBSPEC_MFMA_SET)};

static const Variant* find_variant(const KernelChoice& kc, int bits, int group) {
  for (const Variant& v : kVariants)
    if (v.path == kc.path && v.rows == kc.rows && v.nt == kc.nt && v.chunk == kc.chunk &&
        v.waves == kc.waves && v.bits == bits && v.group == group &&
        (kc.prefetch == 0 || v.prefetch == kc.prefetch))
      return &v;
  return nullptr;
}

bool qlinear_variant_exists(const KernelChoice& kc, int bits, int group) {
  return find_variant(kc, bits, group) != nullptr;
}

int qlinear_resident_blocks(const KernelChoice& kc, int bits, int group, size_t dyn_lds) {
  const Variant* v = find_variant(kc, bits, group);
  if (!v) return 0;
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, reinterpret_cast<const void*>(v->fn),
                                                   kc.waves * kWave, dyn_lds) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return blocks;
}

hipError_t launch_qlinear(const KernelChoice& kc, int bits, int group, const QArgs& a, int grid,
                          hipStream_t st) {
  const Variant* v = find_variant(kc, bits, group);
  if (!v) return hipErrorInvalidDeviceFunction;
  const size_t lds = kc.path == 1 ? gemv_lds_bytes(kc.rows, a.span_blocks * kTileK, group,
                                                   kc.waves * kc.nt * kTileN)
                                  : 0;
  hipLaunchKernelGGL(v->fn, dim3(grid, kc.row_blocks), dim3(kc.waves * kWave), lds, st, a);
  return hipGetLastError();
}

}  // namespace subspec
