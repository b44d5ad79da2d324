// Host-visible launchers of the library's kernels (internal; the public ABI is
// include/subspec.h).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace subspec {

constexpr int kTileN = 16;    // output columns per tile
constexpr int kTileK = 128;   // inputs per tile (one "block")
constexpr int kWave = 64;

// Everything a qlinear kernel needs; filled by the host dispatcher from a plan.
struct QArgs {
  const uint16_t* x;      // bf16 [M][K]
  const uint8_t* qw;      // tile layout
  const uint16_t* sc;     // fp16 [K/group][N]
  const uint16_t* zr;     // fp16 [K/group][N]
  uint16_t* y;            // bf16 [M][N]
  float* ws;              // fp32 [splits][M][N] partial sums (splits > 1)
  unsigned* cnt;          // per column group: workgroups done (zero between launches)
  const float* xsum;      // k_qmma: fp32 [M][K/group] per-group sums of x (k_xsum)
  int M, N, K;
  int KB;                 // K / 128
  int n_tiles;            // N / 16
  // Work assignment: workgroups [0, full_groups) each take one whole column group;
  // the remaining column groups are split `splits` ways (blocks_per_split 128-k
  // blocks each), one workgroup per (column group, split).
  int full_groups;
  int splits;
  int blocks_per_split;
  int span_blocks;        // largest k-block count of one workgroup (GEMV LDS layout)
  // Row blocks (launch grid y > 1, 16x16x32 kernel): workgroups with blockIdx.y = r
  // take rows [r * rb_rows, r * rb_rows + rb_rows) as a launch of their own, with
  // their own partial sums (splits * rb_rows * N floats per block) and completion
  // counters (rb_counters per block).  rb_rows = 0: one block of all M rows.
  int rb_rows;
  int rb_counters;
};

struct KernelChoice {
  int path;    // 1 = GEMV, 2 = MFMA
  int rows;    // GEMV: 1, 2, 4, 8; MFMA: 16 * m-tiles (shape 16) or 32 * m-blocks (shape 32)
  int nt;      // tiles per wavefront
  int chunk;   // 128-k blocks per LDS stage
  int waves;   // wavefronts per workgroup (4 or 8)
  int prefetch = 0;  // ring depth in chunks; 0 = the variant table's choice
  int shape = 0;     // MFMA path: 16 = k_qgemm_mfma (16x16x32), 32 = k_qmma (32x32x16)
  int teams = 1;     // k_qmma: wavefront teams splitting the workgroup's K range
  int row_blocks = 1;  // k_qgemm_mfma: row blocks of `rows` rows each (launch grid y)
};

hipError_t launch_qlinear(const KernelChoice& kc, int bits, int group, const QArgs& a,
                          int grid, hipStream_t st);  // grid: workgroups per row block
bool qlinear_variant_exists(const KernelChoice& kc, int bits, int group);
// Workgroups of this variant that fit on one compute unit (0 if unknown, e.g. no GPU).
int qlinear_resident_blocks(const KernelChoice& kc, int bits, int group, size_t dyn_lds);
// GEMV path: the whole split's activations and the scales/offsets of its groups live
// in LDS, so a split may span at most gemv_max_kspan inputs; gemv_lds_bytes is the
// dynamic LDS of one workgroup (cols = columns of the workgroup).
int gemv_max_kspan(int rows, int waves, int group, int cols);
size_t gemv_lds_bytes(int rows, int kspan, int group, int cols);

// The 32x32x16 kernel (k_qmma): `waves` wavefronts per workgroup (4 or 8) in `teams`
// teams that split its K range (1 or 2), mb 32-row blocks, nb 32-column blocks per
// wavefront, a ring of pf chunks.
bool qmma_variant_exists(int waves, int teams, int mb, int nb, int pf, int bits, int group);
int qmma_resident_blocks(int waves, int teams, int mb, int nb, int pf, int bits, int group);
hipError_t launch_qmma(int waves, int teams, int mb, int nb, int pf, int bits, int group, const QArgs& a,
                       int grid, hipStream_t st);
// The sums of x over every group of k that k_qmma needs: out[m][g] = sum over the
// group's k of x[m][k] (fp32), x bf16 [M][K].
hipError_t launch_xsum(const uint16_t* x, int M, int K, int group, float* out, hipStream_t st);

hipError_t launch_quantize(const float* w, int bits, int group, int N, int K, uint8_t* codes,
                           uint16_t* sc, uint16_t* zr, hipStream_t st);
hipError_t launch_qpack(const uint8_t* codes, int bits, int N, int K, void* qw, hipStream_t st);
hipError_t launch_qdequant(const void* qw, const void* sc, const void* zr, int bits, int group,
                           int N, int K, float* wf, uint16_t* wb, hipStream_t st);

// Split-K workspace: kSplitCounters zeroed counters, then the fp32 partial sums.
constexpr int kSplitCounters = 16384;
constexpr size_t kSplitCounterBytes = kSplitCounters * sizeof(unsigned);

// The allocation-free qlinear entry point's scratch: one fixed array per device
// (completion counters, x sums, partial sums), defined in noalloc.hip.
constexpr size_t kNoAllocScratchBytes = size_t(32) << 20;
// Device address of the current device's scratch array, looked up on the first call
// per device, which also zeroes the completion counters on `st` and waits for them.
// That first call is refused (hipErrorStreamCaptureUnsupported) while `st` is being
// captured; later calls do no GPU work and no allocation.
hipError_t noalloc_scratch(hipStream_t st, void** out);

}  // namespace subspec
