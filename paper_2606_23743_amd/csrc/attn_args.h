// Arguments of the bf16 attention kernels (sparse and dense), kept in a header
// of their own so that a record of measurements can tell whether the kernel
// sources changed.
#pragma once

#include <cstdint>

namespace sva {

// Arguments shared by the attention kernels.
struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* kv_idx;
  const int32_t* kv_count;
  void* out;
  float* lse;
  int N, nB, kmax, n_rows;
  float scale_log2;   // c * log2(e)
  int frame_blocks;   // query blocks per frame of the latent grid, rounded (>= 1)
};

}  // namespace sva
