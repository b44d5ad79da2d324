// The substitute-layer linear y = x * dequant(q, s, z)^T (SubSpec Sec. 4.1) for draft
// batches of 17 to 128 tree tokens, on 32x32x16 bf16 matrix cores (k_qmma).
//
// Roles of the operands: the activations are the A operand (32 rows of x per row
// block, read from LDS), the unpacked codes the B operand (32 columns per column
// block, straight from the weight stream), so a lane's accumulators all belong to one
// output column (lane % 32) and the per-column scale is one register.  A 32x32x16
// instruction keeps the matrix pipe busy for 32 cycles, long enough for about four
// VALU instructions of the same wavefront to issue in its shadow.
//
// Dequantization is folded into the accumulation as in the other kernels: inside a
// group the weight is affine in the code, so for every (row m, column n, group g)
//     sum_{k in g} x*W^ = s*( sum_{k in g} x*(128+q) ) - s*(128+z) * sum_{k in g} x.
// The first term: MFMAs on the exact bf16 values 128+q into a per-group accumulator,
// then tot += s * acc (one FMA per output per group).  The second term for a pair of
// groups at once: one fp32 32x32x2 MFMA with A = the two groups' sums of x and
// B = -s*(128+z) of the two groups (a rank-2 update of the 32x32 output block).
// The sums of x per (row, group) are the same for every workgroup; a small kernel
// (k_xsum) computes them once per call, and each wavefront loads the two it needs per
// row block and pair of groups along with the weights.
//
// Weight fetch: a 32-column block is two 16-column tiles of the packed layout.  The
// B operand of step s (k = 16s ... 16s+15 of a 128-k block) holds, in lanes 0-31, k
// 16s..16s+7 of the block's 32 columns and in lanes 32-63 k 16s+8..16s+15; in tile
// terms lane l takes slice (l % 16) + 16*(2h + l/32) of tile 2cb + (l % 32)/16, with
// h = s % 2, and uses step j = s / 2 of that slice.  Each lane therefore loads two
// slices per block, and every load instruction reads two contiguous runs of 32 slices.
// Every load's per-chunk offset is a scalar (soffset): the lane part of each address
// is computed once.
#pragma once

#include "qlinear_device.h"

namespace subspec {

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

namespace qmma {

typedef __attribute__((address_space(3))) void* LdsPtr;

// LDS of one workgroup: a ring of XB chunks of x per team, each [rows][16 pieces of
// 8 k] with the pieces of row r permuted by piece ^ (r & 15) (the copy-in writes a
// row's 16 pieces per 16 lanes and an A fragment reads one piece of 16 consecutive rows
// per 16 lanes, both conflict free).  The chunk buffers are separate LDS objects on
// purpose: the copy into one runs while another is read, and only distinct objects let
// the compiler see that those reads need not wait for the copy.

// Code pair P (0..15) of a slice: two bf16 values 128 + q (see device_common.h).
template <int BITS, int P>
__device__ __forceinline__ uint32_t code_pair(const Slice<BITS>& s) {
  if constexpr (BITS == 4) {
    return and_or(s.w[P / 4] >> (4 * (P % 4)), 0x000F000Fu, kPairBias);
  } else if constexpr (BITS == 2) {
    return and_or(s.w[P / 8] >> (2 * (P % 8)), 0x00030003u, kPairBias);
  } else if constexpr (P < 15) {
    return and_or(s.w[P / 5] >> (3 * (P % 5)), 0x00070007u, kPairBias);
  } else {
    uint32_t p = and_or(s.w[0] >> 15, 0x00010001u, kPairBias);
    p = and_or(s.w[1] >> 14, 0x00020002u, p);
    return and_or(s.w[2] >> 13, 0x00040004u, p);
  }
}

// B operand of 32-k step J of a slice: pairs 4J .. 4J+3 (8 consecutive k).
template <int BITS, int J>
__device__ __forceinline__ bf16x8_t b_operand(const Slice<BITS>& s) {
  const u32x4_t v = {code_pair<BITS, 4 * J>(s), code_pair<BITS, 4 * J + 1>(s), code_pair<BITS, 4 * J + 2>(s),
                     code_pair<BITS, 4 * J + 3>(s)};
  return __builtin_bit_cast(bf16x8_t, v);
}

template <int BITS>
__device__ __forceinline__ Slice<BITS> load_slice_s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  Slice<BITS> s;
  if constexpr (BITS == 4) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kStreamPolicy);
    s.w[0] = v[0]; s.w[1] = v[1]; s.w[2] = v[2]; s.w[3] = v[3];
  } else if constexpr (BITS == 2) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, kStreamPolicy);
    s.w[0] = v[0]; s.w[1] = v[1];
  } else {
    const auto v = __builtin_amdgcn_raw_buffer_load_b96(r, voff, soff, kStreamPolicy);
    s.w[0] = v[0]; s.w[1] = v[1]; s.w[2] = v[2];
  }
  return s;
}

template <int BITS, int GROUP, int MB, int NB, int WAVES>
struct MmaBody {
  static constexpr int ROWS = 32 * MB;
  static constexpr int GPC = kTileK / GROUP;  // groups per 128-k chunk
  static constexpr int SPG = 8 / GPC;         // 16-k steps per group
  static constexpr int XCH = ROWS * 16;       // 16-byte pieces per chunk buffer
  static constexpr int DMA = ROWS / (4 * WAVES);  // x copy loads per wavefront per chunk
  static_assert(DMA * 4 * WAVES == ROWS, "each copy load fills four rows");

  // One ring slot: the chunk's two slices per column block and the fp16 scale and
  // zero-point of the lane's column for each of the chunk's groups.
  struct W {
    Slice<BITS> w[NB][2];
    uint16_t s[GPC][NB];  // raw fp16 bits, converted only when the group is applied
    uint16_t z[GPC][NB];
    float xs[MB];         // sums of x of a pair of groups (see load_w): row 32 i + lane % 32
  };

  // Lane parts of every address, fixed for the whole launch.
  struct Lanes {
    uint32_t w[NB][2];     // slice byte offsets in block 0 of the column block's tiles
    uint32_t sz[NB];       // byte offset of the lane's column in a row of scales
    uint32_t x;            // byte offset of the lane's first copied piece in chunk 0
    int a;                 // LDS piece index of the lane's A row in row block 0, piece 0
    uint32_t xs;           // byte offset of x-sum (row lane % 32, group lane / 32)
  };

  static __device__ __forceinline__ int slot(int row, int piece) { return row * 16 + (piece ^ (row & 15)); }

  // Chunk kb's weights, scales and zero-points, and the sums of x of groups fg (lanes
  // 0-31) and fg + 1 (lanes 32-63) for each row block; ng = K / GROUP groups per row.
  static __device__ __forceinline__ void load_w(W& r, const QBuffers& bu, const Lanes& ln, int N, int kb, int fg,
                                                int ng) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        r.w[nb][h] = load_slice_s<BITS>(bu.w, ln.w[nb][h], static_cast<uint32_t>(kb) * (256 * BITS));
#pragma unroll
    for (int gi = 0; gi < GPC; ++gi) {
      const uint32_t soff = static_cast<uint32_t>(kb * GPC + gi) * N * 2;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        r.s[gi][nb] = __builtin_amdgcn_raw_buffer_load_b16(bu.s, ln.sz[nb], soff, 0);
        r.z[gi][nb] = __builtin_amdgcn_raw_buffer_load_b16(bu.z, ln.sz[nb], soff, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < MB; ++i)
      r.xs[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                              bu.xs, ln.xs + static_cast<uint32_t>(32 * i) * ng * 4,
                                              static_cast<uint32_t>(fg) * 4, 0));
  }

  // Copy chunk kb of x (all ROWS rows; rows past M read zeros) straight from memory
  // into an LDS buffer: each load instruction fills 1 KB (four consecutive rows) with
  // 16 bytes per lane in lane order, so lane l writes position l % 16 of its row and
  // fetches the piece that the swizzle puts there.  Load j of wavefront w covers rows
  // 4w + 4*WAVES*j + (0..3): a lane keeps the same row % 16, hence the same swizzled
  // piece, in all of its loads.  The row part of the offset stays in the lane offset,
  // which the buffer's range check covers (rows past M read zeros); the chunk's
  // position in the row is the scalar offset.
  static __device__ __forceinline__ void stage(u32x4_t* xb, const QBuffers& bu, const Lanes& ln, int K, int kb,
                                               int wave) {
#pragma unroll
    for (int j = 0; j < DMA; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(bu.x, (LdsPtr)(xb + (4 * wave + 4 * WAVES * j) * 16), 16,
                                               ln.x + static_cast<uint32_t>(j) * (8 * WAVES) * K,
                                               static_cast<uint32_t>(kb) * (kTileK * 2), 0, 0);
  }

  // One chunk (x buffer X, ring slot wc).  The A fragments of the next step are read
  // before the current step's MFMAs, so the LDS latency runs under them (16 more
  // registers at four row blocks, still within two wavefronts per SIMD once the sums
  // of x come from the pre-pass).  cneg[gi][nb] receives -s*(128+z) of the chunk's
  // groups.
  static __device__ __forceinline__ void compute(const W& wc, const u32x4_t* X, int lane, const Lanes& ln,
                                                 f32x16_t (&tot)[MB][NB], float (&cneg)[GPC][NB]) {
    const int r32 = lane & 31, hi = lane >> 5;
    const f32x16_t zero = {};
    // Row 32 i + r32, piece p lives at ln.a + 512 i + (p ^ (r32 & 15)).
    auto read_a = [&](int i, int piece) __attribute__((always_inline)) {
      return __builtin_bit_cast(bf16x8_t, X[ln.a + 512 * i + (piece ^ (r32 & 15))]);
    };
    bf16x8_t A[MB];
#pragma unroll
    for (int i = 0; i < MB; ++i) A[i] = read_a(i, hi);
    static_for<GPC>([&](auto gic) __attribute__((always_inline)) {
      constexpr int gi = decltype(gic)::value;
      f32x16_t acc[MB][NB];
      static_for<SPG>([&](auto ssc) __attribute__((always_inline)) {
        constexpr int SS = decltype(ssc)::value;
        constexpr int S = gi * SPG + SS;  // 16-k step within the chunk
        bf16x8_t An[MB];
        if constexpr (S + 1 < 8) {
#pragma unroll
          for (int i = 0; i < MB; ++i) An[i] = read_a(i, 2 * (S + 1) + hi);
        }
        bf16x8_t B[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) B[nb] = b_operand<BITS, S / 2>(wc.w[nb][S % 2]);
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            acc[i][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[i], B[nb], SS == 0 ? zero : acc[i][nb], 0, 0, 0);
        if constexpr (S + 1 < 8) {
#pragma unroll
          for (int i = 0; i < MB; ++i) A[i] = An[i];
        }
        // Keep each step's unpacking and the next step's reads next to its MFMAs:
        // hoisting a whole chunk's worth of them costs more registers than two
        // wavefronts per SIMD leave.
        __builtin_amdgcn_sched_barrier(0);
      });
      float sv[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        sv[nb] = half_bits_to_float(wc.s[gi][nb]);
        const float z = half_bits_to_float(wc.z[gi][nb]);
        cneg[gi][nb] = -(sv[nb] * (kCodeBias + z));
      }
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) tot[i][nb][r] = __builtin_fmaf(sv[nb], acc[i][nb][r], tot[i][nb][r]);
    });
  }

  // Zero-point term of a pair of groups: lanes 0-31 carry the first group, lanes
  // 32-63 the second; xs[i] is the sum of x of the lane's row in block i and the
  // lane half's group, cop is -s*(128+z) of the lane half's group.  tot += X * C as
  // one fp32 32x32x2 MFMA per output block.
  static __device__ __forceinline__ void apply_pair(const float (&xs)[MB], const float (&cop)[NB],
                                                    f32x16_t (&tot)[MB][NB]) {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        tot[i][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(xs[i], cop[nb], tot[i][nb], 0, 0, 0);
  }
};

// Barrier between chunks.  Each wavefront first reads one element of the buffer the
// next chunk uses: the compiler then waits for this wavefront's copy into that buffer
// (and, loads completing in order, for everything issued before it), but not for the
// copies and weight loads issued after it, which a fenced __syncthreads() would drain.
// LDS writes (the x sums) and reads are complete at the lgkmcnt wait; the empty
// assembly statements keep the compiler from moving LDS accesses across the barrier.
__device__ __forceinline__ void chunk_barrier(const u32x4_t* next, uint32_t& touch) {
  touch ^= next[threadIdx.x & 63].x;
  __builtin_amdgcn_s_waitcnt(kWaitLgkmcnt0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// XB: depth of the x ring and of each wavefront's weight ring, in 128-k chunks.  The
// barrier after chunk c waits for the copy of chunk c + 1, issued XB - 1 chunks
// earlier; the only weight load issued before that copy and not yet needed is the one
// for chunk c + 1 itself, so every weight load has XB - 1 chunks to arrive.
// WAVES: wavefronts per workgroup, one 32-column block each (NB = 1).  TEAMS = 1: all
// of them share the workgroup's x ring.  TEAMS = 2: two teams of four wavefronts on
// the same four column blocks, each with an x ring of its own, take the first and the
// second half of the workgroup's k-blocks, and add their sums through LDS in team
// order at the end (twice the wavefronts per column group without more partial sums).
template <int BITS, int GROUP, int MB, int NB, int XB, int WAVES, int TEAMS>
// Four wavefronts: two workgroups per CU (two wavefronts per SIMD) fit the LDS of a
// two-chunk ring; a deeper ring takes one workgroup per CU and may use the SIMD's
// whole register file.  Eight wavefronts: one workgroup per CU, two per SIMD.
__global__ __launch_bounds__(WAVES * kWave)
__attribute__((amdgpu_waves_per_eu(WAVES == 8 || XB <= 2 ? 2 : 1))) void k_qmma(QArgs a) {
  static_assert(XB % 2 == 0 && XB >= 2 && XB <= 6, "chunk parity (pairs of 128-k groups) follows the ring slot");
  static_assert(WAVES == 4 || WAVES == 8, "wavefronts per workgroup");
  static_assert(TEAMS == 1 || (TEAMS == 2 && WAVES == 8 && XB == 2 && (MB == 2 || MB == 4) && NB == 1),
                "two teams of four wavefronts with two-chunk rings");
  constexpr int TW = WAVES / TEAMS;  // wavefronts per team (its column blocks)
  using Body = MmaBody<BITS, GROUP, MB, NB, TW>;
  constexpr int GPC = Body::GPC;
  constexpr int XCH = Body::XCH;
  constexpr int PF = XB;
  constexpr int NBUF = XB * TEAMS;  // LDS chunk buffers; team t uses [t * XB, t * XB + XB)
  static_assert(NBUF <= 8, "LDS chunk buffers");
  __shared__ u32x4_t xb0[XCH], xb1[XCH], xb2[NBUF > 2 ? XCH : 1], xb3[NBUF > 3 ? XCH : 1],
      xb4[NBUF > 4 ? XCH : 1], xb5[NBUF > 5 ? XCH : 1], xb6[NBUF > 6 ? XCH : 1], xb7[NBUF > 7 ? XCH : 1];
  // Chunk buffer I, selected at compile time: separate LDS objects, so that the
  // compiler can tell the buffers' accesses apart.
  auto lds = [&](auto ic) __attribute__((always_inline)) -> u32x4_t* {
    constexpr int I = decltype(ic)::value;
    static_assert(I < NBUF, "chunk buffer index");
    if constexpr (I == 0) return xb0;
    else if constexpr (I == 1) return xb1;
    else if constexpr (I == 2) return xb2;
    else if constexpr (I == 3) return xb3;
    else if constexpr (I == 4) return xb4;
    else if constexpr (I == 5) return xb5;
    else if constexpr (I == 6) return xb6;
    else return xb7;
  };

  const int lane = threadIdx.x % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x / kWave));
  const int team = wave / TW, tw = wave % TW;
  const int r32 = lane & 31, hi = lane >> 5;
  const WorkItem wi(a);
  const int ng = wi.ng;
  // The team's k-blocks: team 0 the first half of the workgroup's (rounded up), team 1
  // the rest (possibly none).  Both run team 0's number of chunk steps, so that their
  // barriers pair up; a team past its last chunk skips the arithmetic.
  const int nwg = wi.kb_end - wi.kb0;
  const int h0 = TEAMS == 1 ? nwg : (nwg + 1) / 2;
  const int kb0 = wi.kb0 + (team == 0 ? 0 : h0);
  const int nchunks = team == 0 ? h0 : nwg - h0;
  const int nsteps = h0;
  const int last = nchunks - 1;
  const int ngroups = a.K / GROUP;
  const QBuffers bu(a, BITS, GROUP);
  // Block of the team's chunk c, held inside the workgroup's range: loads past the
  // team's last chunk repeat it (L2 hits, never used).
  auto blk = [&](int c) __attribute__((always_inline)) {
    return min(kb0 + max(min(c, last), 0), wi.kb_end - 1);
  };

  // Column blocks of this wavefront: 32 columns each, tiles 2cb and 2cb + 1.  A
  // block past N (half of the last one when N % 32 == 16) reads a valid tile and is
  // never stored.
  typename Body::Lanes ln;
  bool ok[NB];
  int col[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int cb = (ng * TW + tw) * NB + nb;
    const int t = 2 * cb + (r32 >> 4);
    ok[nb] = t < a.n_tiles;
    const int tc = ok[nb] ? t : a.n_tiles - 1;
    col[nb] = tc * kTileN + (lane & 15);
    ln.sz[nb] = static_cast<uint32_t>(col[nb]) * 2;
#pragma unroll
    for (int h = 0; h < 2; ++h)
      ln.w[nb][h] = static_cast<uint32_t>(tc) * a.KB * (256 * BITS) + ((lane & 15) + 16 * (2 * h + hi)) * (4 * BITS);
  }
  {
    const int row = 4 * tw + (lane >> 4), pc = (lane & 15) ^ (row & 15);
    ln.x = (static_cast<uint32_t>(row) * a.K + pc * 8) * 2;
    ln.a = r32 * 16;
    ln.xs = (static_cast<uint32_t>(r32) * ngroups + hi) * 4;
  }

  f32x16_t tot[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) tot[i][nb] = f32x16_t{};

  // The first group of the pair whose x sums chunk c's ring slot carries: with groups
  // of 64 its own two groups; with groups of 128 the pair (c - 1, c) for odd c and
  // (c, c + 1) for even c (used only when c is the team's last chunk, then alone).  A
  // refill past the last chunk can ask for group -1 of the workgroup's first block,
  // which it never uses: held at 0, since the scalar offset of a buffer load is not
  // range checked.
  auto pair_first = [&](int c, int parity) __attribute__((always_inline)) {
    const int kb = blk(c);
    return GPC == 2 ? 2 * kb : parity ? max(kb - 1, 0) : kb;
  };

  uint32_t touch = 0;
  // The main loop of team T (a compile-time constant, so that its ring buffers are
  // distinct LDS objects the compiler can tell apart).
  auto run = [&](auto tc) __attribute__((always_inline)) {
    constexpr int T = decltype(tc)::value;
    // ring slot I of team T: chunk c in slot c % XB
    auto ring = [&](auto ic) __attribute__((always_inline)) -> u32x4_t* {
      return lds(std::integral_constant<int, T * XB + decltype(ic)::value % XB>{});
    };
    // Prologue: chunks 0 .. XB - 2 of x and of the weights in flight.  Unconditional
    // loads keep the compiler's count of outstanding loads exact.
    typename Body::W w[PF];
    static_for<XB - 1>([&](auto u) __attribute__((always_inline)) {
      constexpr int U = decltype(u)::value;
      Body::stage(ring(u), bu, ln, a.K, blk(U), tw);
      Body::load_w(w[U], bu, ln, a.N, blk(U), pair_first(U, U & 1), ngroups);
    });
    chunk_barrier(ring(std::integral_constant<int, 0>{}), touch);

    float cfirst[NB];  // 128-k groups: -s*(128+z) of the first group of an open pair

    // One chunk cc (ring slot U = cc % XB, parity U): start the copy of chunk
    // cc + XB - 1 of x (into the buffer chunk cc - 1 used) and the refill of the weight
    // slot chunk cc - 1 used, then the chunk's MFMAs and, once a pair of groups is
    // complete, its zero-point term.
    auto step = [&](auto u, int cc) __attribute__((always_inline)) {
      constexpr int U = decltype(u)::value;
      const int cn = cc + XB - 1;
      Body::stage(ring(std::integral_constant<int, (U + XB - 1) % XB>{}), bu, ln, a.K, blk(cn), tw);
      Body::load_w(w[(U + PF - 1) % PF], bu, ln, a.N, blk(cn), pair_first(cn, (U + PF - 1) & 1), ngroups);
      if (TEAMS == 1 || cc < nchunks) {
        float cneg[GPC][NB];
        Body::compute(w[U], ring(u), lane, ln, tot, cneg);
        float cop[NB];
        if constexpr (GPC == 2) {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) cop[nb] = hi ? cneg[1][nb] : cneg[0][nb];
          Body::apply_pair(w[U].xs, cop, tot);
        } else if constexpr (U % 2 == 1) {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) cop[nb] = hi ? cneg[0][nb] : cfirst[nb];
          Body::apply_pair(w[U].xs, cop, tot);
        } else {
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) cfirst[nb] = cneg[0][nb];
          if (cc == last) {  // an odd number of chunks: the last group pairs with nothing
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) cop[nb] = hi ? 0.f : cneg[0][nb];
            Body::apply_pair(w[U].xs, cop, tot);
          }
        }
      }
      chunk_barrier(ring(std::integral_constant<int, (U + 1) % XB>{}), touch);
    };
    for (int c = 0; c < nsteps; c += XB)
      static_for<XB>([&](auto u) __attribute__((always_inline)) {
        if (c + decltype(u)::value < nsteps) step(u, c + decltype(u)::value);
      });
  };
  if constexpr (TEAMS == 1) {
    run(std::integral_constant<int, 0>{});
  } else {
    if (team == 0)
      run(std::integral_constant<int, 0>{});
    else
      run(std::integral_constant<int, 1>{});
  }
  // `touch` (an xor of the touched values) only keeps the touching reads alive.
  if (touch == 0x7FC00001u && a.M < 0) a.y[0] = 0;

  if constexpr (TEAMS == 2) {
    // Team 1 hands its sums to team 0 through the LDS of its ring (4 wavefronts x MB
    // row blocks x 16 registers x 64 lanes, the size of two of its chunk buffers: each
    // holds MB / 2 row blocks).  Copies into the rings issued past the last chunk may
    // still be landing, so every wavefront first waits for its own.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
    constexpr int PER = MB / 2;  // row blocks per buffer
    float* red0 = reinterpret_cast<float*>(lds(std::integral_constant<int, XB>{}));      // row blocks [0, PER)
    float* red1 = reinterpret_cast<float*>(lds(std::integral_constant<int, XB + 1>{}));  // row blocks [PER, MB)
    auto at = [&](int i, int r) __attribute__((always_inline)) {
      return ((tw * PER + i % PER) * 16 + r) * kWave + lane;
    };
    if (team == 1) {
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) (i < PER ? red0 : red1)[at(i, r)] = tot[i][0][r];
    }
    __syncthreads();
    if (team == 0) {
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) tot[i][0][r] += (i < PER ? red0 : red1)[at(i, r)];
    }
  }

  // D layout of the 32x32 MFMA: lane l holds column l % 32 and, in register r, row
  // 8 * (r / 4) + 4 * (l / 32) + r % 4 of the block.  The stores go through a buffer
  // resource over the output (bf16 y, or this split's fp32 partial sums) with the
  // whole offset in the vector offset, which the range check covers (the scalar
  // offset is not checked): rows at or past M fall outside the resource and are
  // dropped, and so are the lanes of a column block past N, given an offset outside
  // it.  All offsets stay below 2^31 (no wrap-around into the range) when the tile's
  // rows span less than 2 GiB; larger outputs take per-element stores.
  if (team == 0) {
    const bool split = wi.nsplit > 1;
    const uint32_t esz = split ? 4 : 2;
    const uint64_t out_bytes = static_cast<uint64_t>(a.M) * a.N * esz;
    if (static_cast<uint64_t>(32 * MB) * a.N * esz < (1ull << 31)) {
      const uint32_t rowb = static_cast<uint32_t>(a.N) * esz;
      const __amdgpu_buffer_rsrc_t out =
          split ? buffer_rsrc(a.ws + static_cast<size_t>(wi.split) * a.M * a.N, static_cast<uint32_t>(out_bytes))
                : buffer_rsrc(a.y, static_cast<uint32_t>(out_bytes));
      constexpr uint32_t kOutside = 0x80000000u;
      uint32_t voff[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        voff[nb] = ok[nb] ? static_cast<uint32_t>(col[nb]) * esz + static_cast<uint32_t>(4 * hi) * rowb : kOutside;
      auto store_all = [&](auto splitc) __attribute__((always_inline)) {
        constexpr bool SPLIT = decltype(splitc)::value;
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const uint32_t off = voff[nb] + static_cast<uint32_t>(32 * i + 8 * (r / 4) + (r % 4)) * rowb;
              const float v = tot[i][nb][r];  // a plain value: bit casts of a vector element misbehave
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
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int m = 32 * i + 8 * (r / 4) + 4 * hi + (r % 4);
            if (ok[nb] && m < a.M) store_out(a, wi, m, col[nb], tot[i][nb][r]);
          }
    }
  }
  if (wi.nsplit > 1) finish_splitk<WAVES * kWave>(a, ng, TW * NB * 32);
}

}  // namespace qmma

typedef void (*QmmaKernel)(QArgs);

struct MmaVariant {
  int mb, nb, pf, waves, teams, bits, group;  // pf: depth of the x and weight rings (k_qmma's XB)
  QmmaKernel fn;
};

// The instantiations of one bit width (kernels_qmma_b<bits>.hip).
const MmaVariant* qmma_variants_b2(int* n);
const MmaVariant* qmma_variants_b3(int* n);
const MmaVariant* qmma_variants_b4(int* n);

}  // namespace subspec
