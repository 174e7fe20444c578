// Internal interface of the prefill attention that pools its key tiles on the
// fly (arXiv 2607.06827, Sec. III-C: in training the pooling of Eq. 4 runs
// inside the forward pass).  One launch reads the raw K/V, pools every key
// tile it needs in registers (the same steps as the pooling kernel, so the
// same bits), attends over it under the causal mask over compressed positions
// and writes each pooled row to the paged cache once.
#pragma once

#include "kernels.hpp"

namespace skv {

struct PrefillFusedArgs {
  PrefillArgs at;     // the attention; at.k_pages / at.v_pages are the cache written
  void* k_pages;      // the same pools, written
  void* v_pages;
  const void* k_raw;  // [B][S][Hkv][D] with element strides
  const void* v_raw;
  int64_t stride_b, stride_s, stride_h;
  int raw_len;
  const float* gate;       // [Hkv][D] or null (zero gate)
  int32_t* cache_len_out;  // may be null
};

// Query rows per block of the pooling variant (sizes num_tiles).
int prefill_fused_rows_per_tile(int group);
// bf16 only; head_dim 64 or 128.
hipError_t launch_prefill_fused(const PrefillFusedArgs& a, int head_dim, int group, int batch,
                                hipStream_t s);

}  // namespace skv
