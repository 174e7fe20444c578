// Internal interface between the C-ABI host layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"
#include "spans.hpp"

namespace skv {

// Window pooling into the paged cache (Sec. III-B, Eq. 4).
struct PoolArgs {
  const void* k_raw;
  const void* v_raw;
  int64_t stride_b, stride_s, stride_h;  // elements
  int raw_len;
  const int32_t* prefix_len;
  const int32_t* speech_len;
  const int32_t* suffix_len;
  int w_eff;
  const float* gate;  // [Hkv][D] or null (zero gate)
  void* k_pages;
  void* v_pages;
  const int32_t* table;
  PagedView pv;
  int32_t* cache_len_out;  // may be null
  int max_out;             // bound on the compressed length (grid size)
  SegmentTable segs;       // several speech runs per sequence when segs.seg_start is set
};

// Window pooling of whole hidden states (HS Compression, Sec. IV-A method
// (4); the pooling of Eq. 4 applied to the hidden state).
struct PoolHiddenArgs {
  const void* h;
  int64_t stride_b, stride_s;  // elements
  int raw_len;
  const int32_t* prefix_len;
  const int32_t* speech_len;
  const int32_t* suffix_len;
  int w;
  const float* gate;  // [hidden] or null (zero gate)
  void* out;
  int64_t out_stride_b, out_stride_s;  // elements
  int out_cap;        // rows per sequence in out
  int32_t* out_len;   // may be null
  int max_out;        // bound on the compressed length (grid size)
};

// Split-K decode attention (Sec. III-B, Eq. 5; Sec. III-C).
struct DecodeArgs {
  const void* q;
  void* k_pages;
  void* v_pages;
  const int32_t* table;
  PagedView pv;
  const int32_t* cache_len;
  int max_len;
  const void* k_new;
  const void* v_new;
  float scale_log2;  // scale * log2(e)
  int num_splits;
  void* out;
  float* ws_o;   // [B][Hq][splits][D] unnormalised partial outputs
  float* ws_ml;  // [B][Hq][splits][2] running max (log2 units) and sum
};

// Full-resolution-query attention over the compressed cache (Eq. 5 + mask).
struct PrefillArgs {
  const void* q;
  void* out;
  float* lse;
  const void* k_pages;
  const void* v_pages;
  const int32_t* table;
  PagedView pv;
  const int32_t* prefix_len;
  const int32_t* speech_len;
  const int32_t* suffix_len;
  int w_eff;
  int mask_mode;
  int q_len;
  int num_tiles;  // query tiles per (sequence, KV head)
  int num_q_heads;
  float scale_log2;
  SegmentTable segs;  // several speech runs per sequence when segs.seg_start is set
};

// dtype: 0 = fp32, 1 = bf16.  Each launcher returns the launch status.
hipError_t launch_pool(const PoolArgs& a, int dtype, int head_dim, int batch, hipStream_t s);
// blocks per sequence of launch_pool's grid (at most INT32_MAX for a launch)
int64_t pool_grid_blocks(int max_out, int kv_heads, int head_dim);
bool pool_hidden_supported(int hidden);
hipError_t launch_pool_hidden(const PoolHiddenArgs& a, int dtype, int hidden, int batch,
                              hipStream_t s);
hipError_t launch_decode(const DecodeArgs& a, int dtype, int head_dim, int group, int batch,
                         hipStream_t s);
hipError_t launch_decode_merge(const DecodeArgs& a, int dtype, int head_dim, int num_q_heads,
                               int batch, hipStream_t s);
int prefill_rows_per_tile(int group);
hipError_t launch_prefill(const PrefillArgs& a, int dtype, int head_dim, int group, int batch,
                          hipStream_t s);

// Launch a kernel whose only parameter is one argument struct.
template <typename A>
inline hipError_t launch_struct(void (*kernel)(A), dim3 grid, dim3 block, hipStream_t s, A args) {
  void* argv[] = {&args};
  return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv, 0, s);
}

}  // namespace skv
