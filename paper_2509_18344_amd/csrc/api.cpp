// C ABI of the library (include/subspec.h): argument validation, launch planning,
// the per-device split-K workspace, the host packer and error reporting.
#include "subspec.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <cstring>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "kernels.h"
#include "kernels_tree.h"
#include "kernels_attn.h"
#include "kernels_hqq.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(SUBSPEC_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_bits_group(int bits, int group) {
  if (bits < 2 || bits > 4) return fail(SUBSPEC_EUNSUPPORTED, "bits=%d: must be 2, 3 or 4", bits);
  if (group != 64 && group != 128)
    return fail(SUBSPEC_EUNSUPPORTED, "group=%d: must be 64 or 128", group);
  return SUBSPEC_OK;
}

int check_tiles(int N, int K) {
  if (N <= 0 || K <= 0) return fail(SUBSPEC_EINVAL, "N=%d, K=%d: must be positive", N, K);
  if (N % subspec::kTileN) return fail(SUBSPEC_EUNSUPPORTED, "N=%d: must be a multiple of 16", N);
  if (K % subspec::kTileK) return fail(SUBSPEC_EUNSUPPORTED, "K=%d: must be a multiple of 128", K);
  // The kernels address every operand with 32-bit byte offsets.
  if (static_cast<long long>(N) * K > (1ll << 32))
    return fail(SUBSPEC_EUNSUPPORTED, "N*K=%lld too large (at most 2^32)", static_cast<long long>(N) * K);
  if (K > (1 << 24)) return fail(SUBSPEC_EUNSUPPORTED, "K=%d too large (at most 2^24)", K);
  return SUBSPEC_OK;
}

constexpr int kMaxRows = 128;
constexpr int kGemvMaxRows = 8;
// Measured on the Qwen2.5-7B MLP shapes (4-bit g128) with kernel traces and SQ
// counters: the GEMV path's VALU work grows with M (dot products per row) while the
// 16-row MFMA tile's does not, and the MFMA path is faster from M = 2 on (gate|up:
// 15.9 against 17.2 us at M = 2, 17.4 against 52.1 us at M = 6).
constexpr int kAutoGemvMaxRows = 1;

// --- launch planning --------------------------------------------------------

// Every planning choice below has a default measured on the 7B MLP shapes; the
// fields exist so that measurement sweeps can override them (SUBSPEC_TUNE).  None of
// them changes what is computed.
struct Tuning {
  int gemv_max_m = kAutoGemvMaxRows;  // largest M the automatic plan sends to the GEMV path
  int target_blocks = 0;          // workgroups to aim for; 0 = the per-CU target below
  int gemv_nt = 1;                // tiles per GEMV wavefront
  int gemv_waves = 4;             // wavefronts per GEMV workgroup
  int gemv_ch = 0;                // 128-k blocks per GEMV ring stage; 0 = choose per M
  int gemv_pf = 0;                // ring depth in stages; 0 = the variant's
  int mfma_nt = 0;                // tiles per MFMA wavefront; 0 = choose per shape
  int mfma_ch = 0;                // 128-k blocks per MFMA chunk; 0 = choose per M
  int mfma_pf = 0;                // MFMA ring depth in chunks; 0 = the variant's
  int wg_per_cu = 0;              // split-K target workgroups per CU; 0 = two
  int tail = 1;                   // split only the column groups past a multiple of the CUs
  int fill_cus = 2;               // partial-sum cap still gives each CU this many workgroups
  int splits = 0;                 // 0 = choose per shape
  int partial_div = 2;            // split-K partial traffic may reach weight bytes / this
  // Largest M the automatic MFMA plan keeps on 16x16x32 tiles (k_qgemm_mfma) in all
  // cases; above it, k_qmma where it measured faster (see make_plan).
  int mma16_max_m = 64;
  int mma_nb = 0;                 // 32x32 kernel: 32-column blocks per wavefront; 0 = choose
  int mma_shape = 0;              // automatic MFMA plans: 16 or 32 forces the tile shape
  int mma_waves = 0;              // 32x32 kernel: wavefronts per workgroup (4 or 8); 0 = choose
  // Smallest M at which wide launches take the 32x32 kernel's 64-row eight-wavefront
  // tiles instead of 16x16x32 ones (0 = never).
  int mma8_min_m = 33;
  int mma8_half_min_m = 48;       // the same where 256-column groups cover only half the CUs
  int mma_teams = 0;              // 32x32 kernel, long-K launches: 1 = one team, 2 = two; 0 = choose
  int teams64_min_m = 33;         // long-K launches from this M up to 64: 64-row two-team 32x32 tiles
  int row_split = 0;              // 16x16x32 tiles: 1 = two row blocks where possible, 2 = never; 0 = choose
};

// Optional overrides for measurement sweeps: SUBSPEC_TUNE="gemv_max_m=4,target=512,...".
const Tuning& tuning() {
  static Tuning t = [] {
    Tuning r;
    const char* env = std::getenv("SUBSPEC_TUNE");
    if (!env) return r;
    std::string s(env);
    size_t pos = 0;
    while (pos < s.size()) {
      size_t end = s.find(',', pos);
      if (end == std::string::npos) end = s.size();
      std::string kv = s.substr(pos, end - pos);
      size_t eq = kv.find('=');
      if (eq != std::string::npos) {
        const std::string k = kv.substr(0, eq);
        const int v = std::atoi(kv.c_str() + eq + 1);
        if (k == "gemv_max_m") r.gemv_max_m = v;
        else if (k == "target") r.target_blocks = v;
        else if (k == "gemv_nt") r.gemv_nt = v;
        else if (k == "gemv_waves") r.gemv_waves = v;
        else if (k == "gemv_ch") r.gemv_ch = v;
        else if (k == "gemv_pf") r.gemv_pf = v;
        else if (k == "mfma_nt") r.mfma_nt = v;
        else if (k == "mfma_ch") r.mfma_ch = v;
        else if (k == "mfma_pf") r.mfma_pf = v;
        else if (k == "wg_per_cu") r.wg_per_cu = v;
        else if (k == "tail") r.tail = v;
        else if (k == "fill_cus") r.fill_cus = v;
        else if (k == "splits") r.splits = v;
        else if (k == "partial_div") r.partial_div = v;
        else if (k == "mma16_max_m") r.mma16_max_m = v;
        else if (k == "mma_nb") r.mma_nb = v;
        else if (k == "mma_shape") r.mma_shape = v;
        else if (k == "mma_waves") r.mma_waves = v;
        else if (k == "mma8_min_m") r.mma8_min_m = v;
        else if (k == "mma8_half_min_m") r.mma8_half_min_m = v;
        else if (k == "mma_teams") r.mma_teams = v;
        else if (k == "row_split") r.row_split = v;
        else if (k == "teams64_min_m") r.teams64_min_m = v;
      }
      pos = end + 1;
    }
    return r;
  }();
  return t;
}

// Compute units of the current device (256 on MI355X; the fallback when no GPU is
// present keeps host-only planning deterministic).
int device_cus() {
  static int cus = [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
      (void)hipGetLastError();
      return 256;
    }
    return n;
  }();
  return cus;
}

// Bytes of the per-group sums of x the 32x32 kernel reads (fp32 [M][K/group]),
// rounded up to 256.
size_t xsum_bytes(const subspec::KernelChoice& c, int M, int K, int group) {
  if (c.shape != 32) return 0;
  return (static_cast<size_t>(M) * (K / group) * sizeof(float) + 255) & ~size_t(255);
}

// ws_cap bounds the workspace the plan may use (the allocation-free entry point's
// fixed scratch array): the split count shrinks to fit, and a plan that cannot fit
// even unsplit is refused.
int make_plan(int M, int N, int K, int bits, int group, int path, subspec_plan* p,
              subspec::KernelChoice* kc, size_t ws_cap = SIZE_MAX) {
  int rc = check_bits_group(bits, group);
  if (rc) return rc;
  rc = check_tiles(N, K);
  if (rc) return rc;
  if (M < 1 || M > kMaxRows) return fail(SUBSPEC_EUNSUPPORTED, "M=%d: must be in 1..%d", M, kMaxRows);
  const Tuning& tu = tuning();
  if (path == SUBSPEC_PATH_AUTO) path = (M <= tu.gemv_max_m) ? SUBSPEC_PATH_GEMV : SUBSPEC_PATH_MFMA;
  const int KB = K / subspec::kTileK;
  // 32x32x16 tiles (k_qmma, 128 rows, 128 columns per workgroup) against 16x16x32
  // (k_qgemm_mfma).  Measured on the Qwen2.5-7B/32B stacks at M = 96 and 128, k_qmma
  // wins where its workgroups fill every CU without splitting K (gate|up: 7B 52.8
  // against 66.0 us, 32B 3-bit 98.0 against 122.0 us at M = 96) and, one workgroup per
  // CU with a four-chunk ring, on splits of a long K (32B down, K = 27648: 65.7
  // against 68.2 us); on the short split launches (q|k|v, o; 7B down, K = 18944) the
  // 16x16x32 kernel is faster (7B o at M = 128: 25.8 against 32.0 us).
  const bool wide = (N + 127) / 128 >= device_cus();
  const bool long_k = KB >= 128;
  // 256-column groups (eight wavefronts of the 32x32 kernel) still cover three
  // quarters (wide8) or half (half8) of the CUs.
  const bool wide8 = (N + 255) / 256 * 4 >= 3 * device_cus();
  const bool half8 = (N + 255) / 256 * 2 >= device_cus();
  if (path == SUBSPEC_PATH_MFMA) {
    // Below mma16_max_m, wide unsplit launches still take 64-row 32x32 tiles from
    // mma8_min_m on: 32B gate|up 48.7 against 53.4 us at M = 33, 51.6 against 55.1 at
    // 48, 53.9 against 59.0 at 64; where 256-column groups cover only half the CUs,
    // from mma8_half_min_m on (7B gate|up, 148 groups: 32.8 against 34.5 us at M = 48,
    // 35.1 against 37.3 at 64, but 32.4 against 31.1 at 33); the short launches stay on
    // 16x16x32 (q|k|v at M = 64 27.2 against 19.0 us).  Long-K launches take 64-row
    // tiles on two teams of four wavefronts from teams64_min_m (below): 32B down 34.5
    // against 39.3 us at M = 48 and 39.6 against 41.5 at 64, 2-bit g64 36.0 against 43.9
    // and 40.2 against 46.1; the 7B down about even (25.7 against 25.2 at 48, 26.8
    // against 27.5 at 64); at M = 32, with half of each tile empty, 30.7 against 27.3.
    const bool tiles64 = tu.mma8_min_m > 0 && M >= tu.mma8_min_m && (half8 && !wide8 ? M >= tu.mma8_half_min_m : wide8) &&
                         !long_k;
    const bool teams64 = tu.teams64_min_m > 0 && long_k && M >= tu.teams64_min_m && M <= 64;
    const bool use32 =
        tu.mma_shape ? tu.mma_shape == 32 : (M > tu.mma16_max_m && (wide || long_k)) || tiles64 || teams64;
    path = use32 ? SUBSPEC_PATH_MFMA32 : SUBSPEC_PATH_MFMA16;
  }
  subspec::KernelChoice c{}, c8{};
  bool use8 = false;  // 32x32 kernel: the eight-wavefront variant (c8) where it exists
  c.waves = 4;
  if (path == SUBSPEC_PATH_GEMV) {
    if (M > kGemvMaxRows) return fail(SUBSPEC_EUNSUPPORTED, "GEMV path needs M <= 8 (M=%d)", M);
    c.path = 1;
    c.rows = M <= 1 ? 1 : M <= 2 ? 2 : M <= 4 ? 4 : 8;
    c.nt = tu.gemv_nt;
    c.waves = tu.gemv_waves;
    // A shallow ring (two stages of two blocks for one or two rows) keeps register
    // use low enough for more resident waves; measured faster than deeper rings.
    c.chunk = tu.gemv_ch ? tu.gemv_ch : c.rows <= 2 ? 2 : 4;
    c.prefetch = tu.gemv_pf;
  } else if (path == SUBSPEC_PATH_MFMA32) {
    // 32x32x16 matrix cores (k_qmma): four row blocks of 32 (two up to M = 64), four
    // wavefronts of one 32-column block each, one 128-k chunk per LDS stage.  The ring
    // is two chunks deep (two workgroups per CU) when whole column groups fill the
    // device, four deep (one workgroup per CU, more loads in flight each) otherwise;
    // the eight-wavefront and two-team forms below replace it where they measured
    // faster.
    c.path = 2;
    c.shape = 32;
    c.rows = M <= 64 ? 64 : 128;
    c.nt = 2 * (tu.mma_nb ? tu.mma_nb : 1);
    c.chunk = 1;
    c.prefetch = tu.mfma_pf ? tu.mfma_pf : wide ? 2 : 4;
    // Eight wavefronts of one 32-column block each share one x ring four chunks deep
    // (one workgroup of 256 columns per CU): each wavefront then has three chunks of
    // weights in flight instead of one.  Taken where 256-column groups still cover
    // three quarters of the CUs and K is not split (32B gate|up, N = 55296, M = 128:
    // 90.9 against 98.0 us at 3 bits, 97.1 against 103.1 at 2 bits; slower on the 7B
    // gate|up's 148 groups and on the split 32B down projection).  Up to M = 64 the
    // tiles are 64 rows (two row blocks), built for eight wavefronts only.
    c8 = c;
    c8.waves = 8;
    c8.prefetch = tu.mfma_pf ? tu.mfma_pf : 4;
    use8 = tu.mma_waves == 8 || (!tu.mma_waves && (wide8 || (half8 && c.rows == 64)) && !long_k);
    // Long-K launches (split along K, not wide enough for whole groups) take two teams
    // of four wavefronts per workgroup, each on half of the workgroup's k-blocks: two
    // wavefronts per SIMD at the same number of splits (32B down, K = 27648: 61.5
    // against 63.8 us at M = 128, 54.7 against 58.7 at 96; 7B down, K = 18944: 40.5
    // against 45.7 on 16x16x32 tiles at M = 128).  Each team's ring stays two chunks
    // deep: four-chunk rings of 64 rows (128 KB of LDS) measured no faster (32B down
    // 35.2 against 34.5 us at M = 48, 41.3 against 39.6 at 64).
    const bool teams = tu.mma_teams ? tu.mma_teams == 2 : long_k;
    if (!use8 && teams) {
      c8 = c;
      c8.waves = 8;
      c8.teams = 2;
      c8.prefetch = 2;
      use8 = true;
    }
  } else if (path == SUBSPEC_PATH_MFMA16) {
    c.path = 2;
    c.shape = 16;
    const int mt = M <= 16 ? 1 : M <= 32 ? 2 : M <= 64 ? 4 : 8;
    c.rows = 16 * mt;
    // LDS holds two chunks of rows x (128*chunk) activations (at most 64 KB).  Short
    // ring stages (256 k for one row tile, 128 k beyond) keep register use low enough
    // for a third resident workgroup; measured faster than longer stages.
    c.chunk = tu.mfma_ch ? tu.mfma_ch : mt == 1 ? 2 : 1;
    c.prefetch = tu.mfma_pf;
    c.nt = tu.mfma_nt ? tu.mfma_nt : 1;
  } else {
    return fail(SUBSPEC_EINVAL, "path=%d: unknown", path);
  }
  auto variant_exists = [&](const subspec::KernelChoice& k) {
    return k.shape == 32 ? subspec::qmma_variant_exists(k.waves, k.teams, k.rows / 32, k.nt / 2, k.prefetch, bits,
                                                        group)
                         : subspec::qlinear_variant_exists(k, bits, group);
  };
  if (use8 && (tu.mma_waves == 8 || variant_exists(c8))) c = c8;
  if (c.shape == 32 && c.rows == 64 && !variant_exists(c)) c.rows = 128;  // no 64-row build
  if (!variant_exists(c))
    return fail(SUBSPEC_EUNSUPPORTED, "no kernel for path=%d rows=%d nt=%d chunk=%d waves=%d bits=%d group=%d",
                c.path, c.rows, c.nt, c.chunk, c.waves, bits, group);

  // Workgroups that fit on the device at once (one residency round).
  auto resident_of = [&](const subspec::KernelChoice& k) {
    if (tu.target_blocks > 0) return tu.target_blocks;
    size_t lds = 0;
    if (k.path == 1) {
      const int cols = k.waves / k.teams * k.nt * subspec::kTileN;
      lds = subspec::gemv_lds_bytes(k.rows, std::min(K, subspec::gemv_max_kspan(k.rows, k.waves, group, cols)),
                                    group, cols);
    }
    int per_cu = k.shape == 32 ? subspec::qmma_resident_blocks(k.waves, k.teams, k.rows / 32, k.nt / 2,
                                                               k.prefetch, bits, group)
                               : subspec::qlinear_resident_blocks(k, bits, group, lds);
    if (per_cu <= 0) per_cu = 2;
    return per_cu * device_cus();
  };
  auto groups_of = [&](const subspec::KernelChoice& k) {
    const int cols = k.waves / k.teams * k.nt * subspec::kTileN;
    return (N + cols - 1) / cols;
  };
  int resident = resident_of(c);
  // Two tiles per wavefront halve the workgroups, and each A fragment read from LDS
  // feeds two MFMAs.  At two row tiles that LDS traffic is what bounds a workgroup, so
  // two tiles win whenever they still leave every CU a column group and two
  // wavefronts per SIMD (measured on the 7B gate|up at M = 32).  At four row tiles the
  // one-tile kernel reads its A fragments a step ahead and is faster (7B gate|up at
  // M = 64: 36.7 against 38.4 us); at eight row tiles the two-tile variant fits one
  // wavefront per SIMD and loses.  Otherwise two tiles only pay when the one-tile
  // launch would need a second residency round.
  if (c.path == 2 && c.shape == 16 && !tu.mfma_nt) {
    subspec::KernelChoice c2 = c;
    c2.nt = 2;
    if (subspec::qlinear_variant_exists(c2, bits, group)) {
      const int r2 = resident_of(c2);
      const long long rounds1 = (groups_of(c) + resident - 1) / resident;
      const long long rounds2 = (groups_of(c2) + r2 - 1) / r2;
      const bool lds_bound = c.rows == 32 && groups_of(c2) >= device_cus() && r2 >= 2 * device_cus();
      if (lds_bound || (groups_of(c) > resident && rounds2 < rounds1)) {
        c = c2;
        resident = r2;
      }
    }
  }
  // Row blocks: the 16x16x32 kernel's rows in two blocks of half the tile height, each
  // a launch of its own along grid y with its own partial sums and counters.  Each
  // weight tile is then read by two workgroups, but a launch that has to split K needs
  // half the splits for the same number of workgroups, and the last workgroup of a
  // column group, which adds the partial sums alone, reads a quarter of them.  Taken
  // for tiles of 64 rows or more on launches that split a K of under 128 blocks
  // (q|k|v and o): 32B q|k|v 16.4 against 19.4 us at M = 64, 26.6 against 31.4 at 128,
  // o 13.6 against 17.2 and 21.9 against 27.4; 7B q|k|v 11.3 against 17.1 at M = 64.
  // Slower on the long-K down (32B at M = 64: 44.1 against 40.8 us) and on gate|up at
  // M = 32 (32.2 against 24.9), which keep one block.
  const bool split_rows = tu.row_split ? tu.row_split == 1
                                       : c.rows >= 64 && !long_k && groups_of(c) < device_cus();
  if (c.path == 2 && c.shape == 16 && split_rows && c.rows >= 32 && M > c.rows / 2) {
    subspec::KernelChoice cr = c;
    cr.rows = c.rows / 2;
    cr.row_blocks = 2;
    cr.chunk = tu.mfma_ch ? tu.mfma_ch : cr.rows == 16 ? 2 : 1;
    if (variant_exists(cr)) c = cr;
  }
  const int cols_per_group = c.waves / c.teams * c.nt * subspec::kTileN;
  const int col_groups = groups_of(c);
  const int units = col_groups * c.row_blocks;  // workgroups of one split
  const long long part_rows = c.row_blocks > 1 ? static_cast<long long>(c.row_blocks) * c.rows : M;
  const int chunks = (KB + c.chunk - 1) / c.chunk;

  // Split K across workgroups only as far as a target workgroup count reaches, and
  // only while the fp32 partial sums (written once, read once) stay a modest fraction
  // of the weight bytes.  The target is two workgroups per CU (or one residency
  // round, if smaller): their waves already keep enough loads in flight, and further
  // splits only add partial traffic (measured on the 7B MLP with both paths: 592
  // column groups run faster unsplit than split in two, 56 faster in 9 splits than
  // in 13).
  const int per_cu_target = tu.wg_per_cu ? tu.wg_per_cu : 2;
  const int target = tu.target_blocks ? resident : std::min(resident, per_cu_target * device_cus());
  int splits = std::max(1, target / units);
  const double wbytes = static_cast<double>(N) * K * bits / 8 + 4.0 * N * (K / group);
  const double per_split = 8.0 * M * N;
  int cap = tu.partial_div > 0 ? std::max(1, static_cast<int>(wbytes / (tu.partial_div * per_split)))
                               : splits;
  // The cap never leaves a CU with fewer than two workgroups: at large M a
  // workgroup's own issue rate, not HBM, bounds it, and partial sums cost less than
  // idle CUs (7B q|k|v at M = 64: 72 workgroups took as long as gate|up).
  if (tu.fill_cus) cap = std::max(cap, (device_cus() * tu.fill_cus + units - 1) / units);
  splits = std::min(splits, cap);
  if (tu.splits > 0) splits = tu.splits;
  if (c.path == 1) {
    // the split's activations must fit the GEMV kernel's LDS staging
    const int max_chunks = std::max(1, subspec::gemv_max_kspan(c.rows, c.waves, group, cols_per_group) /
                                           subspec::kTileK / c.chunk);
    const int min_splits = (chunks + max_chunks - 1) / max_chunks;
    if (splits < min_splits) splits = min_splits;
  }
  // Split-K needs a completion counter per column group and 32-bit offsets into the
  // partial sums.
  const long long split_bytes = 4ll * part_rows * N;
  auto fit_offsets = [&](int sp) {
    if (sp > 1 && split_bytes * sp >= (1ll << 31))
      sp = std::max(1, static_cast<int>(((1ll << 31) - 1) / split_bytes));
    return sp;
  };
  if (units > subspec::kSplitCounters) splits = 1;
  const size_t fixed_ws = subspec::kSplitCounterBytes + xsum_bytes(c, M, K, group);
  auto fit_cap = [&](int sp) {
    if (sp > 1 && ws_cap != SIZE_MAX) {
      const size_t room = ws_cap > fixed_ws ? ws_cap - fixed_ws : 0;
      const size_t most = room / (static_cast<size_t>(4) * part_rows * N);
      if (static_cast<size_t>(sp) > most) sp = static_cast<int>(std::max<size_t>(1, most));
    }
    return sp;
  };
  splits = fit_cap(fit_offsets(splits));

  // Balanced tail.  With col_groups = base * CUs + rem (base >= 1), whole column groups
  // alone leave rem CUs one group ahead of the rest (592 groups on 256 CUs: 80 CUs run
  // three, 176 run two).  Instead the first base * CUs groups run whole and the last
  // rem are split CUs / rem ways, so no CU gets more than base groups plus one part of
  // a split one.  (A GEMV workgroup that runs a whole group stages all of K.)
  int full_groups = 0;
  const int cus = device_cus();
  if (splits == 1 && tu.tail && !tu.splits && c.row_blocks == 1 && col_groups <= subspec::kSplitCounters &&
      (c.path != 1 || K <= subspec::gemv_max_kspan(c.rows, c.waves, group, cols_per_group))) {
    const int base = col_groups / cus, rem = col_groups % cus;
    const int ts = fit_cap(fit_offsets(std::min(rem ? cus / rem : 0, chunks)));
    if (base >= 1 && ts >= 2) {
      full_groups = base * cus;
      splits = ts;
    }
  }
  if (splits > chunks) splits = chunks;
  int chunks_per_split = (chunks + splits - 1) / splits;
  const int blocks_per_split = chunks_per_split * c.chunk;
  splits = (KB + blocks_per_split - 1) / blocks_per_split;
  if (splits == 1) full_groups = 0;
  if (c.path == 1) {
    // The clamps above (counter count, 32-bit partial offsets) can undo the GEMV
    // minimum split count; a split that spans more of K than the kernel stages in LDS
    // would read unstaged activations, so such shapes are refused.
    const int span = subspec::gemv_max_kspan(c.rows, c.waves, group, cols_per_group);
    const long long split_k = static_cast<long long>(splits == 1 ? KB : blocks_per_split) * subspec::kTileK;
    if (std::min<long long>(split_k, K) > span)
      return fail(SUBSPEC_EUNSUPPORTED,
                  "GEMV path: M=%d N=%d K=%d needs splits of at most %d k, but the plan can only "
                  "split %d ways (%d column groups)", M, N, K, span, splits, col_groups);
  }
  p->path = c.path == 1 ? SUBSPEC_PATH_GEMV : SUBSPEC_PATH_MFMA;
  p->mfma_rows = c.path == 2 ? c.shape : 0;
  p->teams = c.teams;
  p->row_blocks = c.row_blocks;
  p->rows = c.rows;
  p->tiles_per_wave = c.nt;
  p->waves = c.waves;
  p->chunk_blocks = c.chunk;
  p->ring_chunks = c.prefetch;
  p->col_groups = col_groups;
  p->full_groups = full_groups;
  p->splits = splits;
  p->blocks_per_split = blocks_per_split;
  p->grid = full_groups + (col_groups - full_groups) * splits;
  // Workspace: split-K completion counters, then (32x32 kernel) the per-group sums of
  // x, then the splits' fp32 partial sums.
  p->workspace_bytes = 0;
  if (splits > 1 || c.shape == 32)
    p->workspace_bytes = subspec::kSplitCounterBytes + xsum_bytes(c, M, K, group) +
                         (splits > 1 ? static_cast<size_t>(splits) * part_rows * N * sizeof(float) : 0);
  if (p->workspace_bytes > ws_cap)
    return fail(SUBSPEC_EUNSUPPORTED, "M=%d N=%d K=%d: needs %zu bytes of scratch even unsplit, above the "
                "%zu available", M, N, K, p->workspace_bytes, ws_cap);
  if (kc) *kc = c;
  return SUBSPEC_OK;
}

// A call's plan depends only on (device, M, N, K, bits, group, path, workspace cap)
// and the process's tuning, so each thread keeps the plans it has made: repeated
// calls (every draft pass repeats the same shapes) skip the planner and its occupancy
// queries.  Failed plans are not kept.
struct PlanKey {
  int dev, M, N, K, bits, group, path;
  size_t cap;
  bool operator==(const PlanKey& o) const {
    return dev == o.dev && M == o.M && N == o.N && K == o.K && bits == o.bits && group == o.group &&
           path == o.path && cap == o.cap;
  }
};
struct PlanKeyHash {
  size_t operator()(const PlanKey& k) const {
    size_t h = static_cast<size_t>(k.cap);
    for (int v : {k.dev, k.M, k.N, k.K, k.bits, k.group, k.path}) h = h * 1000003u ^ static_cast<size_t>(v);
    return h;
  }
};
struct CachedPlan {
  subspec_plan plan;
  subspec::KernelChoice kc;
};
constexpr size_t kPlanCacheEntries = 4096;  // a full cache is cleared, not evicted entry by entry

int make_plan_cached(int M, int N, int K, int bits, int group, int path, subspec_plan* p,
                     subspec::KernelChoice* kc, size_t ws_cap) {
  thread_local std::unordered_map<PlanKey, CachedPlan, PlanKeyHash> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    dev = -1;
  }
  const PlanKey key{dev, M, N, K, bits, group, path, ws_cap};
  const auto it = cache.find(key);
  if (it != cache.end()) {
    *p = it->second.plan;
    *kc = it->second.kc;
    return SUBSPEC_OK;
  }
  const int rc = make_plan(M, N, K, bits, group, path, p, kc, ws_cap);
  if (rc) return rc;
  if (cache.size() >= kPlanCacheEntries) cache.clear();
  cache.emplace(key, CachedPlan{*p, *kc});
  return SUBSPEC_OK;
}

// --- per-device workspace -----------------------------------------------------

struct Workspace {
  void* ptr = nullptr;
  size_t bytes = 0;
  int graphs = 0;                // live captured graphs made on this device
  std::vector<void*> retired;    // earlier buffers: queued kernels or graphs may still use them
  unsigned long long allocations = 0;
};
std::mutex g_ws_mutex;
std::vector<Workspace> g_ws;

int current_device(int* dev) {
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  return SUBSPEC_OK;
}

Workspace& workspace_of(int dev) {  // caller holds g_ws_mutex
  if (static_cast<int>(g_ws.size()) <= dev) g_ws.resize(dev + 1);
  return g_ws[dev];
}

// Frees the retired buffers of `w`; the caller has synchronised the device.
int free_retired(Workspace& w) {
  int rc = SUBSPEC_OK;
  for (void* p : w.retired) {
    const hipError_t e = hipFree(p);
    if (e != hipSuccess && rc == SUBSPEC_OK) rc = hip_fail(e, "hipFree(retired workspace)");
  }
  w.retired.clear();
  return rc;
}

// Returns the device's workspace, grown to `bytes` if needed.  Growth allocates a new
// buffer (at least twice the old size, so retired buffers total less than the live
// one), zeroes its completion counters on `st` and waits for that stream only.  The
// old buffer is retired, not freed: kernels queued on other streams and captured
// graphs may still use it.  Growth is refused while `st` is being captured.
int get_workspace(size_t bytes, hipStream_t st, void** out) {
  int dev = 0;
  int rc = current_device(&dev);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(g_ws_mutex);
  Workspace& w = workspace_of(dev);
  if (w.bytes >= bytes) {
    *out = w.ptr;
    return SUBSPEC_OK;
  }
  if (st != nullptr) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    hipError_t e = hipStreamIsCapturing(st, &cs);
    if (e != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
    if (cs != hipStreamCaptureStatusNone)
      return fail(SUBSPEC_ECAPTURE, "workspace must grow to %zu bytes during stream capture; call "
                  "subspec_reserve() first", bytes);
  }
  size_t nb = std::max({bytes, 2 * w.bytes, size_t(1) << 20});
  nb = (nb + 0xFFFFF) & ~size_t(0xFFFFF);
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, nb);
  if (e != hipSuccess) return hip_fail(e, "hipMalloc(workspace)");
  // The split-K completion counters start at zero; every launch leaves them at zero.
  e = hipMemsetAsync(p, 0, subspec::kSplitCounterBytes, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) {
    (void)hipFree(p);
    return hip_fail(e, "zeroing the workspace counters");
  }
  if (w.ptr) w.retired.push_back(w.ptr);
  w.ptr = p;
  w.bytes = nb;
  ++w.allocations;
  *out = p;
  return SUBSPEC_OK;
}

// --- host packer (the same layout as the device packer) ----------------------

template <int BITS>
void pack_slice_host(const uint32_t c[32], uint32_t* out) {
  const uint32_t mask = (1u << BITS) - 1;
  for (int w = 0; w < BITS; ++w) out[w] = 0;
  for (int p = 0; p < 16; ++p) {
    const int j = p / 4, i = p % 4;
    const uint32_t ev = c[8 * j + 2 * i] & mask, od = c[8 * j + 2 * i + 1] & mask;
    if (BITS == 4) {
      out[p / 4] |= (ev << (4 * (p % 4))) | (od << (16 + 4 * (p % 4)));
    } else if (BITS == 2) {
      out[p / 8] |= (ev << (2 * (p % 8))) | (od << (16 + 2 * (p % 8)));
    } else if (p < 15) {
      out[p / 5] |= (ev << (3 * (p % 5))) | (od << (16 + 3 * (p % 5)));
    } else {
      for (int b = 0; b < 3; ++b) out[b] |= (((ev >> b) & 1u) << 15) | (((od >> b) & 1u) << 31);
    }
  }
}

template <int BITS>
void pack_host(const uint8_t* codes, int N, int K, uint8_t* out) {
  const int KB = K / subspec::kTileK;
  uint32_t c[32], words[BITS];
  for (long long nt = 0; nt < N / subspec::kTileN; ++nt)
    for (int kb = 0; kb < KB; ++kb)
      for (int L = 0; L < 64; ++L) {
        const long long n = nt * subspec::kTileN + L % 16;
        const uint8_t* row = codes + n * K + kb * subspec::kTileK + 8 * (L / 16);
        for (int j = 0; j < 4; ++j)
          for (int e = 0; e < 8; ++e) c[8 * j + e] = row[32 * j + e];
        pack_slice_host<BITS>(c, words);
        uint8_t* dst = out + ((nt * KB + kb) * 64 + L) * (4 * BITS);
        std::memcpy(dst, words, 4 * BITS);  // little-endian host
      }
}

// noalloc: take the scratch from the library's fixed per-device array (no allocation,
// splits capped to its size) instead of the growable workspace.
int qlinear_impl(const void* x, const void* qweight, const void* scales, const void* zeros,
                 int bits, int group, int M, int N, int K, void* y, int path, hipStream_t st,
                 bool noalloc = false) {
  subspec_plan p;
  subspec::KernelChoice kc;
  int rc = make_plan_cached(M, N, K, bits, group, path, &p, &kc,
                            noalloc ? subspec::kNoAllocScratchBytes : SIZE_MAX);
  if (rc) return rc;
  if (!x || !qweight || !scales || !zeros || !y) return fail(SUBSPEC_EINVAL, "null pointer argument");
  if (!aligned16(x) || !aligned16(qweight) || !aligned16(scales) || !aligned16(zeros) || !aligned16(y))
    return fail(SUBSPEC_EINVAL, "device pointers must be 16-byte aligned");
  subspec::QArgs a{};
  a.x = static_cast<const uint16_t*>(x);
  a.qw = static_cast<const uint8_t*>(qweight);
  a.sc = static_cast<const uint16_t*>(scales);
  a.zr = static_cast<const uint16_t*>(zeros);
  a.y = static_cast<uint16_t*>(y);
  a.M = M;
  a.N = N;
  a.K = K;
  a.KB = K / subspec::kTileK;
  a.n_tiles = N / subspec::kTileN;
  a.full_groups = p.full_groups;
  a.splits = p.splits;
  a.blocks_per_split = p.blocks_per_split;
  a.span_blocks = p.full_groups > 0 ? a.KB : p.blocks_per_split;
  if (kc.row_blocks > 1) {
    a.rb_rows = kc.rows;
    a.rb_counters = p.col_groups;
  }
  if (p.workspace_bytes) {
    void* ws = nullptr;
    if (noalloc) {
      const hipError_t e = subspec::noalloc_scratch(st, &ws);
      if (e == hipErrorStreamCaptureUnsupported)
        return fail(SUBSPEC_ECAPTURE, "subspec_qlinear_noalloc: the first call on a device sets up its scratch "
                    "array and must not be captured");
      if (e != hipSuccess) return hip_fail(e, "scratch array set-up");
    } else {
      rc = get_workspace(p.workspace_bytes, st, &ws);
      if (rc) return rc;
    }
    char* base = static_cast<char*>(ws);
    const size_t xsb = xsum_bytes(kc, M, K, group);
    a.cnt = reinterpret_cast<unsigned*>(base);
    a.xsum = xsb ? reinterpret_cast<const float*>(base + subspec::kSplitCounterBytes) : nullptr;
    a.ws = reinterpret_cast<float*>(base + subspec::kSplitCounterBytes + xsb);
  }
  hipError_t e = hipSuccess;
  if (kc.shape == 32) {
    e = subspec::launch_xsum(a.x, M, K, group, const_cast<float*>(a.xsum), st);
    if (e == hipSuccess)
      e = subspec::launch_qmma(kc.waves, kc.teams, kc.rows / 32, kc.nt / 2, kc.prefetch, bits, group, a, p.grid,
                               st);
  } else {
    e = subspec::launch_qlinear(kc, bits, group, a, p.grid, st);
  }
  if (e != hipSuccess) return hip_fail(e, "qlinear launch");
  return SUBSPEC_OK;
}

}  // namespace

extern "C" {

size_t subspec_qpack_bytes(int bits, int N, int K) {
  if (bits < 2 || bits > 4 || N <= 0 || K <= 0 || N % subspec::kTileN || K % subspec::kTileK) return 0;
  return static_cast<size_t>(N) * K / 8 * bits;
}

int subspec_quantize(const float* w, int bits, int group, int N, int K, uint8_t* codes,
                     uint16_t* scales, uint16_t* zeros, hipStream_t stream) {
  int rc = check_bits_group(bits, group);
  if (rc) return rc;
  if (N <= 0 || K <= 0 || K % group) return fail(SUBSPEC_EINVAL, "N=%d K=%d group=%d: bad shape", N, K, group);
  if (!w || !codes || !scales || !zeros) return fail(SUBSPEC_EINVAL, "null pointer argument");
  if (!aligned16(w) || !aligned16(codes) || !aligned16(scales) || !aligned16(zeros))
    return fail(SUBSPEC_EINVAL, "device pointers must be 16-byte aligned");
  hipError_t e = subspec::launch_quantize(w, bits, group, N, K, codes, scales, zeros, stream);
  if (e != hipSuccess) return hip_fail(e, "quantize launch");
  return SUBSPEC_OK;
}

int subspec_quantize_hqq(const float* w, int bits, int group, int N, int K, uint8_t* codes,
                         uint16_t* scales, uint16_t* zeros, hipStream_t stream) {
  int rc = check_bits_group(bits, group);
  if (rc) return rc;
  if (N <= 0 || K <= 0 || K % group) return fail(SUBSPEC_EINVAL, "N=%d K=%d group=%d: bad shape", N, K, group);
  if (!w || !codes || !scales || !zeros) return fail(SUBSPEC_EINVAL, "null pointer argument");
  if (!aligned16(w) || !aligned16(codes) || !aligned16(scales) || !aligned16(zeros))
    return fail(SUBSPEC_EINVAL, "device pointers must be 16-byte aligned");
  hipError_t e = subspec::launch_quantize_hqq(w, bits, group, N, K, codes, scales, zeros, stream);
  if (e != hipSuccess) return hip_fail(e, "quantize_hqq launch");
  return SUBSPEC_OK;
}

int subspec_qpack(const uint8_t* codes, int bits, int N, int K, void* qweight, hipStream_t stream) {
  if (bits < 2 || bits > 4) return fail(SUBSPEC_EUNSUPPORTED, "bits=%d: must be 2, 3 or 4", bits);
  int rc = check_tiles(N, K);
  if (rc) return rc;
  if (!codes || !qweight) return fail(SUBSPEC_EINVAL, "null pointer argument");
  if (!aligned16(codes) || !aligned16(qweight)) return fail(SUBSPEC_EINVAL, "device pointers must be 16-byte aligned");
  hipError_t e = subspec::launch_qpack(codes, bits, N, K, qweight, stream);
  if (e != hipSuccess) return hip_fail(e, "qpack launch");
  return SUBSPEC_OK;
}

int subspec_qpack_host(const uint8_t* codes, int bits, int N, int K, void* qweight) {
  if (bits < 2 || bits > 4) return fail(SUBSPEC_EUNSUPPORTED, "bits=%d: must be 2, 3 or 4", bits);
  int rc = check_tiles(N, K);
  if (rc) return rc;
  if (!codes || !qweight) return fail(SUBSPEC_EINVAL, "null pointer argument");
  uint8_t* out = static_cast<uint8_t*>(qweight);
  if (bits == 4) pack_host<4>(codes, N, K, out);
  else if (bits == 3) pack_host<3>(codes, N, K, out);
  else pack_host<2>(codes, N, K, out);
  return SUBSPEC_OK;
}

int subspec_qlinear(const void* x, const void* qweight, const void* scales, const void* zeros,
                    int bits, int group, int M, int N, int K, void* y, hipStream_t stream) {
  return qlinear_impl(x, qweight, scales, zeros, bits, group, M, N, K, y, SUBSPEC_PATH_AUTO, stream);
}

int subspec_qlinear_noalloc(const void* x, const void* qweight, const void* scales, const void* zeros,
                            int bits, int group, int M, int N, int K, void* y, hipStream_t stream) {
  return qlinear_impl(x, qweight, scales, zeros, bits, group, M, N, K, y, SUBSPEC_PATH_AUTO, stream, true);
}

int subspec_qlinear_path(const void* x, const void* qweight, const void* scales, const void* zeros,
                         int bits, int group, int M, int N, int K, void* y, int path,
                         hipStream_t stream) {
  return qlinear_impl(x, qweight, scales, zeros, bits, group, M, N, K, y, path, stream);
}

int subspec_qlinear_plan(int M, int N, int K, int bits, int group, int path, subspec_plan* plan) {
  if (!plan) return fail(SUBSPEC_EINVAL, "null plan pointer");
  return make_plan(M, N, K, bits, group, path, plan, nullptr);
}

int subspec_qdequant(const void* qweight, const void* scales, const void* zeros, int bits,
                     int group, int N, int K, float* w_f32, uint16_t* w_bf16, hipStream_t stream) {
  int rc = check_bits_group(bits, group);
  if (rc) return rc;
  rc = check_tiles(N, K);
  if (rc) return rc;
  if (!qweight || !scales || !zeros) return fail(SUBSPEC_EINVAL, "null pointer argument");
  if (!w_f32 && !w_bf16) return SUBSPEC_OK;
  hipError_t e = subspec::launch_qdequant(qweight, scales, zeros, bits, group, N, K, w_f32, w_bf16, stream);
  if (e != hipSuccess) return hip_fail(e, "qdequant launch");
  return SUBSPEC_OK;
}

int subspec_stack_forward(const subspec_proj* projs, int nproj, int bits, int group, int M,
                          hipStream_t stream) {
  if (!projs || nproj < 0) return fail(SUBSPEC_EINVAL, "bad projection list");
  for (int i = 0; i < nproj; ++i) {
    const subspec_proj& p = projs[i];
    const int rc = qlinear_impl(p.x, p.qweight, p.scales, p.zeros, bits, group, M, p.N, p.K, p.y,
                                SUBSPEC_PATH_AUTO, stream);
    if (rc) return rc;
  }
  return SUBSPEC_OK;
}

struct subspec_graph {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  int device = 0;  // its workspace buffers stay allocated while it lives
};

int subspec_stack_capture(const subspec_proj* projs, int nproj, int bits, int group, int M,
                          hipStream_t stream, subspec_graph** out) {
  if (!out) return fail(SUBSPEC_EINVAL, "null graph pointer");
  *out = nullptr;
  if (!projs || nproj <= 0) return fail(SUBSPEC_EINVAL, "bad projection list");
  if (stream == nullptr) return fail(SUBSPEC_EINVAL, "capture needs a non-null stream");
  // Plan every launch first: argument errors surface before capture, and the
  // workspace is grown (allocation is not capturable) to the largest need.
  size_t need = 0;
  for (int i = 0; i < nproj; ++i) {
    subspec_plan p;
    const int rc = make_plan(M, projs[i].N, projs[i].K, bits, group, SUBSPEC_PATH_AUTO, &p, nullptr);
    if (rc) return rc;
    need = std::max(need, p.workspace_bytes);
  }
  if (need) {
    void* ws = nullptr;
    const int rc = get_workspace(need, nullptr, &ws);
    if (rc) return rc;
  }
  hipError_t e = hipStreamBeginCapture(stream, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) return hip_fail(e, "hipStreamBeginCapture");
  const int rc = subspec_stack_forward(projs, nproj, bits, group, M, stream);
  hipGraph_t graph = nullptr;
  e = hipStreamEndCapture(stream, &graph);
  if (rc) {
    if (graph) (void)hipGraphDestroy(graph);  // the capture error is the one reported
    return rc;
  }
  if (e != hipSuccess) return hip_fail(e, "hipStreamEndCapture");
  hipGraphExec_t exec = nullptr;
  e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  if (e != hipSuccess) {
    (void)hipGraphDestroy(graph);  // the instantiation error is the one reported
    return hip_fail(e, "hipGraphInstantiate");
  }
  subspec_graph* g = new subspec_graph;
  g->graph = graph;
  g->exec = exec;
  int dev = 0;
  (void)hipGetDevice(&dev);
  g->device = dev;
  {
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    ++workspace_of(dev).graphs;
  }
  *out = g;
  return SUBSPEC_OK;
}

int subspec_graph_launch(subspec_graph* g, hipStream_t stream) {
  if (!g || !g->exec) return fail(SUBSPEC_EINVAL, "null graph");
  hipError_t e = hipGraphLaunch(g->exec, stream);
  if (e != hipSuccess) return hip_fail(e, "hipGraphLaunch");
  return SUBSPEC_OK;
}

int subspec_graph_destroy(subspec_graph* g) {
  if (!g) return SUBSPEC_OK;
  hipError_t e1 = hipDeviceSynchronize();
  hipError_t e2 = g->exec ? hipGraphExecDestroy(g->exec) : hipSuccess;
  hipError_t e3 = g->graph ? hipGraphDestroy(g->graph) : hipSuccess;
  int rc = SUBSPEC_OK;
  {
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    Workspace& w = workspace_of(g->device);
    // The last graph of the device is gone and the device is idle: nothing can still
    // reference a retired buffer.
    if (--w.graphs == 0 && e1 == hipSuccess) rc = free_retired(w);
  }
  delete g;
  if (e1 != hipSuccess) return hip_fail(e1, "hipDeviceSynchronize");
  if (e2 != hipSuccess) return hip_fail(e2, "hipGraphExecDestroy");
  if (e3 != hipSuccess) return hip_fail(e3, "hipGraphDestroy");
  return rc;
}

size_t subspec_tree_workspace_bytes(int R, int V, int k) {
  if (R < 1 || R > subspec::kTreeMaxRows || V < 8 || V % 8 || k < 1 || k > subspec::kTreeMaxK)
    return 0;
  return subspec::tree_workspace_bytes(R, V, k);
}

namespace {

// Shape checks shared by the tree-attention entry points ("" when supported).
const char* attn_shape_error(int M, int Hq, int Hkv, int P, int T) {
  if (Hkv < 1 || Hq < Hkv || Hq % Hkv) return "Hq must be a positive multiple of Hkv";
  if (M < 1 || static_cast<long long>(Hq / Hkv) * M > subspec::kAttnMaxRows)
    return "need 1 <= M and (Hq / Hkv) * M <= 64";
  if (P < 0 || T < 0 || static_cast<long long>(P) + T + M >= (1ll << 30)) return "P, T out of range";
  const long long W = (static_cast<long long>(T) + M + 31) / 32;
  if (M * W > subspec::kAttnMaskWords) return "M * ceil((T + M) / 32) must be at most 2048";
  return "";
}

}  // namespace

int subspec_tree_attention_plan(int M, int Hq, int Hkv, int P, int T, int* splits, int* tiles_per_split) {
  if (!splits || !tiles_per_split) return fail(SUBSPEC_EINVAL, "null pointer argument");
  const char* why = attn_shape_error(M, Hq, Hkv, P, T);
  if (*why) return fail(SUBSPEC_EUNSUPPORTED, "tree_attention: %s", why);
  subspec::attn_plan(M, Hq, Hkv, P, T, splits, tiles_per_split);
  return SUBSPEC_OK;
}

size_t subspec_tree_attention_workspace_bytes(int M, int Hq, int Hkv, int P, int T) {
  if (*attn_shape_error(M, Hq, Hkv, P, T)) return 0;
  return subspec::attn_workspace_bytes(M, Hq, Hkv, P, T);
}

int subspec_tree_attention(const void* q, void* k_cache, void* v_cache, const void* k_new,
                           const void* v_new, const uint32_t* mask, int M, int Hq, int Hkv,
                           int S, int P, int T, float scale, void* out, hipStream_t stream) {
  if (!q || !k_cache || !v_cache || !k_new || !v_new || !mask || !out)
    return fail(SUBSPEC_EINVAL, "null pointer argument");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(k_new) ||
      !aligned16(v_new) || !aligned16(out))
    return fail(SUBSPEC_EINVAL, "q, caches, new keys/values and out must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(mask) & 3u) return fail(SUBSPEC_EINVAL, "mask must be 4-byte aligned");
  const char* why = attn_shape_error(M, Hq, Hkv, P, T);
  if (*why) return fail(SUBSPEC_EUNSUPPORTED, "tree_attention: %s", why);
  if (static_cast<long long>(P) + T + M > S)
    return fail(SUBSPEC_EUNSUPPORTED, "tree_attention: P + T + M = %lld exceeds S = %d",
                static_cast<long long>(P) + T + M, S);
  if (!std::isfinite(scale)) return fail(SUBSPEC_EINVAL, "scale must be finite");
  void* ws = nullptr;
  const int rc = get_workspace(subspec::attn_workspace_bytes(M, Hq, Hkv, P, T), stream, &ws);
  if (rc) return rc;
  subspec::AttnArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k_cache = static_cast<uint16_t*>(k_cache);
  a.v_cache = static_cast<uint16_t*>(v_cache);
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.mask = mask;
  a.M = M;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.S = S;
  a.P = P;
  a.T = T;
  a.W = (T + M + 31) / 32;
  a.scale_log2 = scale * 1.4426950408889634f;
  subspec::attn_plan(M, Hq, Hkv, P, T, &a.splits, &a.tiles_per_split);
  if (a.splits > subspec::kAttnMaxSplits)
    return fail(SUBSPEC_EUNSUPPORTED, "tree_attention: %d key ranges exceed %d", a.splits, subspec::kAttnMaxSplits);
  a.rows_pad = 16 * ((Hq / Hkv * M + 15) / 16);
  const size_t n = static_cast<size_t>(Hkv) * a.splits * a.rows_pad;
  // The first kSplitCounterBytes of the workspace are the split-K completion counters
  // that qlinear and tree_expand rely on being zero: the partials go after them.
  a.part_o = reinterpret_cast<float*>(static_cast<char*>(ws) + subspec::kSplitCounterBytes);
  a.part_ml = a.part_o + n * subspec::kAttnD;
  a.out = static_cast<uint16_t*>(out);
  const hipError_t e = subspec::launch_tree_attention(a, stream);
  if (e != hipSuccess) return hip_fail(e, "tree_attention launch");
  return SUBSPEC_OK;
}

int subspec_tree_plan(int R, int V, int k, int* chunks, int* chunk_len, int* list_len) {
  if (!chunks || !chunk_len || !list_len) return fail(SUBSPEC_EINVAL, "null pointer argument");
  if (R < 1 || R > subspec::kTreeMaxRows || V < 8 || V % 8 || k < 1 || k > subspec::kTreeMaxK ||
      static_cast<long long>(R) * V >= (1LL << 31) || k > static_cast<long long>(R) * V)
    return fail(SUBSPEC_EUNSUPPORTED, "tree_plan: (R, V, k) out of the supported range");
  subspec::tree_plan(R, V, chunks, chunk_len);
  *list_len = k <= 8 ? 8 : k <= 16 ? 16 : 32;
  return SUBSPEC_OK;
}

int subspec_tree_expand(const void* logits, const float* parent_logp, int R, int V,
                        float temperature, int k, int* parent_out, int* token_out,
                        float* score_out, hipStream_t stream) {
  if (!logits || !parent_logp || !parent_out || !token_out || !score_out)
    return fail(SUBSPEC_EINVAL, "null pointer argument");
  if (!aligned16(logits)) return fail(SUBSPEC_EINVAL, "logits must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(parent_logp) | reinterpret_cast<uintptr_t>(parent_out) |
       reinterpret_cast<uintptr_t>(token_out) | reinterpret_cast<uintptr_t>(score_out)) & 3u)
    return fail(SUBSPEC_EINVAL, "scores and outputs must be 4-byte aligned");
  if (R < 1 || R > subspec::kTreeMaxRows)
    return fail(SUBSPEC_EUNSUPPORTED, "R=%d: must be in 1..%d", R, subspec::kTreeMaxRows);
  if (V < 8 || V % 8) return fail(SUBSPEC_EUNSUPPORTED, "V=%d: must be a positive multiple of 8", V);
  if (static_cast<long long>(R) * V >= (1ll << 31))
    return fail(SUBSPEC_EUNSUPPORTED, "R*V=%lld: must be below 2^31", static_cast<long long>(R) * V);
  if (k < 1 || k > subspec::kTreeMaxK || static_cast<long long>(k) > static_cast<long long>(R) * V)
    return fail(SUBSPEC_EUNSUPPORTED, "k=%d: must be in 1..%d and at most R*V", k, subspec::kTreeMaxK);
  if (!(temperature > 0.f) || !std::isfinite(temperature) || !std::isfinite(1.f / temperature))
    return fail(SUBSPEC_EINVAL, "temperature must be positive and finite");
  void* ws = nullptr;
  const int rc = get_workspace(subspec::tree_workspace_bytes(R, V, k), stream, &ws);
  if (rc) return rc;
  subspec::TreeArgs a{};
  a.logits = static_cast<const uint16_t*>(logits);
  a.parent = parent_logp;
  a.R = R;
  a.V = V;
  a.k = k;
  a.inv_t = 1.f / temperature;
  subspec::tree_plan(R, V, &a.chunks, &a.chunk_len);
  const size_t blocks = static_cast<size_t>(R) * a.chunks;
  char* base = static_cast<char*>(ws);
  a.cnt = reinterpret_cast<unsigned*>(base);
  char* p = base + subspec::kSplitCounterBytes;
  a.stat_m = reinterpret_cast<float*>(p);
  a.stat_s = a.stat_m + blocks;
  a.cand_val = a.stat_s + blocks;
  a.cand_idx = reinterpret_cast<int*>(a.cand_val + blocks * k);
  a.out_parent = parent_out;
  a.out_token = token_out;
  a.out_score = score_out;
  const hipError_t e = subspec::launch_tree_expand(a, stream);
  if (e != hipSuccess) return hip_fail(e, "tree_expand launch");
  return SUBSPEC_OK;
}

int subspec_reserve(size_t bytes) {
  void* p = nullptr;
  int rc = get_workspace(bytes, nullptr, &p);
  if (rc) return rc;
  int dev = 0;
  rc = current_device(&dev);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(g_ws_mutex);
  Workspace& w = workspace_of(dev);
  if (w.graphs > 0 || w.retired.empty()) return SUBSPEC_OK;
  const hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  return free_retired(w);
}

int subspec_workspace_info(size_t* bytes, int* retired, unsigned long long* allocations) {
  int dev = 0;
  const int rc = current_device(&dev);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(g_ws_mutex);
  const Workspace& w = workspace_of(dev);
  if (bytes) *bytes = w.bytes;
  if (retired) *retired = static_cast<int>(w.retired.size());
  if (allocations) *allocations = w.allocations;
  return SUBSPEC_OK;
}

const char* subspec_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"

// --- cross-layer asynchronous weight prefetch (Sec. 4.3, App. E) ---------------------

struct subspec_prefetch {
  struct Slot {
    void* dev = nullptr;
    hipEvent_t copied = nullptr;  // recorded on the copy stream after the copy
    hipEvent_t freed = nullptr;   // recorded on the releasing stream
    long long ticket = -1;        // ticket in the slot, -1 if never used
    bool held = false;            // begun and not yet released
    bool freed_recorded = false;
  };
  int device = 0;
  size_t slot_bytes = 0;
  hipStream_t copy = nullptr;
  std::vector<Slot> slots;
  long long next = 0;
};

namespace {

void prefetch_teardown(subspec_prefetch* pf) {
  if (pf->copy) (void)hipStreamSynchronize(pf->copy);
  for (auto& s : pf->slots) {
    if (s.dev) (void)hipFree(s.dev);
    if (s.copied) (void)hipEventDestroy(s.copied);
    if (s.freed) (void)hipEventDestroy(s.freed);
  }
  if (pf->copy) (void)hipStreamDestroy(pf->copy);
  delete pf;
}

// The slot that holds `ticket`, or null (with the error set).
subspec_prefetch::Slot* prefetch_slot(subspec_prefetch* pf, long long ticket) {
  if (ticket < 0 || ticket >= pf->next) {
    fail(SUBSPEC_EINVAL, "prefetch: ticket %lld was not begun", ticket);
    return nullptr;
  }
  auto& s = pf->slots[ticket % static_cast<long long>(pf->slots.size())];
  if (s.ticket != ticket || !s.held) {
    fail(SUBSPEC_EINVAL, "prefetch: ticket %lld is released or its slot was reused", ticket);
    return nullptr;
  }
  return &s;
}

int prefetch_device_check(const subspec_prefetch* pf) {
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != pf->device) return fail(SUBSPEC_EINVAL, "prefetch: created on device %d, called on %d", pf->device, dev);
  return SUBSPEC_OK;
}

}  // namespace

int subspec_prefetch_create(size_t slot_bytes, int slots, subspec_prefetch** out) {
  if (!out) return fail(SUBSPEC_EINVAL, "null pointer argument");
  *out = nullptr;
  if (slot_bytes == 0 || slots < 2 || slots > 64)
    return fail(SUBSPEC_EINVAL, "prefetch: need slot_bytes > 0 and 2 <= slots <= 64");
  auto* pf = new subspec_prefetch();
  pf->slot_bytes = slot_bytes;
  hipError_t e = hipGetDevice(&pf->device);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&pf->copy, hipStreamNonBlocking);
  pf->slots.resize(slots);
  for (auto& s : pf->slots) {
    if (e == hipSuccess) e = hipMalloc(&s.dev, slot_bytes);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&s.copied, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&s.freed, hipEventDisableTiming);
  }
  if (e != hipSuccess) {
    prefetch_teardown(pf);
    return hip_fail(e, "prefetch_create");
  }
  *out = pf;
  return SUBSPEC_OK;
}

int subspec_prefetch_destroy(subspec_prefetch* pf) {
  if (!pf) return fail(SUBSPEC_EINVAL, "null pointer argument");
  prefetch_teardown(pf);
  return SUBSPEC_OK;
}

int subspec_prefetch_begin(subspec_prefetch* pf, const void* host_src, size_t bytes, long long* ticket) {
  if (!pf || !host_src || !ticket) return fail(SUBSPEC_EINVAL, "null pointer argument");
  if (bytes == 0 || bytes > pf->slot_bytes)
    return fail(SUBSPEC_EINVAL, "prefetch: %zu bytes do not fit a slot of %zu", bytes, pf->slot_bytes);
  int rc = prefetch_device_check(pf);
  if (rc) return rc;
  hipPointerAttribute_t attr{};
  if (hipPointerGetAttributes(&attr, host_src) != hipSuccess || attr.type != hipMemoryTypeHost) {
    (void)hipGetLastError();
    return fail(SUBSPEC_EINVAL, "prefetch: host source must be pinned host memory");
  }
  const long long t = pf->next;
  auto& s = pf->slots[t % static_cast<long long>(pf->slots.size())];
  if (s.held)
    return fail(SUBSPEC_EINVAL, "prefetch: slot of ticket %lld still holds ticket %lld (release it first)", t,
                s.ticket);
  hipError_t e = hipSuccess;
  if (s.freed_recorded) e = hipStreamWaitEvent(pf->copy, s.freed, 0);
  if (e == hipSuccess) e = hipMemcpyAsync(s.dev, host_src, bytes, hipMemcpyHostToDevice, pf->copy);
  if (e == hipSuccess) e = hipEventRecord(s.copied, pf->copy);
  if (e != hipSuccess) return hip_fail(e, "prefetch_begin");
  s.ticket = t;
  s.held = true;
  pf->next = t + 1;
  *ticket = t;
  return SUBSPEC_OK;
}

int subspec_prefetch_acquire(subspec_prefetch* pf, long long ticket, hipStream_t compute, void** dev_ptr) {
  if (!pf || !dev_ptr) return fail(SUBSPEC_EINVAL, "null pointer argument");
  int rc = prefetch_device_check(pf);
  if (rc) return rc;
  auto* s = prefetch_slot(pf, ticket);
  if (!s) return SUBSPEC_EINVAL;
  const hipError_t e = hipStreamWaitEvent(compute, s->copied, 0);
  if (e != hipSuccess) return hip_fail(e, "prefetch_acquire");
  *dev_ptr = s->dev;
  return SUBSPEC_OK;
}

int subspec_prefetch_release(subspec_prefetch* pf, long long ticket, hipStream_t compute) {
  if (!pf) return fail(SUBSPEC_EINVAL, "null pointer argument");
  int rc = prefetch_device_check(pf);
  if (rc) return rc;
  auto* s = prefetch_slot(pf, ticket);
  if (!s) return SUBSPEC_EINVAL;
  const hipError_t e = hipEventRecord(s->freed, compute);
  if (e != hipSuccess) return hip_fail(e, "prefetch_release");
  s->held = false;
  s->freed_recorded = true;
  return SUBSPEC_OK;
}
