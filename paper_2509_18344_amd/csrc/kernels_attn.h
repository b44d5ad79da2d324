// Host-visible launcher of the draft model's tree attention over the shared KV cache
// (internal; the public ABI is include/subspec.h).
#pragma once

#include "kernels.h"

namespace subspec {

constexpr int kAttnD = 128;           // head dimension (Qwen2.5 models)
constexpr int kAttnTile = 32;         // keys per tile
constexpr int kAttnMaxRows = 64;      // query rows per key/value head: (Hq / Hkv) * M
constexpr int kAttnMaskWords = 2048;  // M * ceil((T + M) / 32)
constexpr int kAttnMaxSplits = 512;   // key ranges per head (attn_plan gives at most 256)

struct AttnArgs {
  const uint16_t* q;      // bf16 [M][Hq][D]
  uint16_t* k_cache;      // bf16 [Hkv][S][D]
  uint16_t* v_cache;      // bf16 [Hkv][S][D]
  const uint16_t* k_new;  // bf16 [M][Hkv][D]
  const uint16_t* v_new;  // bf16 [M][Hkv][D]
  const uint32_t* mask;   // [M][W] bit rows over the tree tokens
  int M, Hq, Hkv, S, P, T, W;
  float scale_log2;       // scale * log2(e)
  int splits;             // key ranges per key/value head
  int tiles_per_split;    // 32-key tiles per range
  int rows_pad;           // 16 * ceil((Hq / Hkv) * M / 16)
  float* part_o;          // [Hkv][splits][rows_pad][D] unnormalised partial outputs
  float* part_ml;         // [Hkv][splits][rows_pad][2] running max (log2 domain), sum
  uint16_t* out;          // bf16 [M][Hq][D]
};

void attn_plan(int M, int Hq, int Hkv, int P, int T, int* splits, int* tiles_per_split);
size_t attn_workspace_bytes(int M, int Hq, int Hkv, int P, int T);
hipError_t launch_tree_attention(const AttnArgs& a, hipStream_t st);

}  // namespace subspec
