// Host-visible launcher of the draft-tree expansion kernel (internal; the public ABI
// is include/subspec.h).
#pragma once

#include "kernels.h"

namespace subspec {

// Draft-tree expansion (kernels_tree.hip): logits bf16 [R][V], path scores fp32 [R].
constexpr int kTreeMaxRows = 1024;
constexpr int kTreeMaxK = 32;
struct TreeArgs {
  const uint16_t* logits;
  const float* parent;
  int R, V, k;
  float inv_t;            // 1 / temperature
  int chunks, chunk_len;  // workgroups per row and the logits each one covers
  float* stat_m;          // [R * chunks] running maxima
  float* stat_s;          // [R * chunks] sums of exp(z - m)
  float* cand_val;        // [R * chunks][k] best z of each workgroup
  int* cand_idx;          // [R * chunks][k] their tokens
  unsigned* cnt;          // completion counter (zero between launches)
  int* out_parent;
  int* out_token;
  float* out_score;
};
void tree_plan(int R, int V, int* chunks, int* chunk_len);
size_t tree_workspace_bytes(int R, int V, int k);
hipError_t launch_tree_expand(const TreeArgs& a, hipStream_t st);

}  // namespace subspec
