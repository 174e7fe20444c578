// Internal interface of the backward (training) kernels: gradients of the
// attention over the compressed cache (Eq. 5 under the causal mask over
// compressed positions) and of the window pooling (Eq. 4), which training
// optimises jointly with the model (arXiv 2607.06827, Sec. III-C).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"
#include "spans.hpp"

namespace skv {

struct PrefillBwdArgs {
  const void* q;       // [B][q_len][Hq][D]
  const void* out;     // forward output, same layout
  const void* dout;    // gradient of the output, same layout
  const float* lse;    // [B][Hq][q_len], natural log
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
  int num_q_heads;
  int num_q_tiles;    // query tiles per (sequence, KV head), dQ kernel
  int num_key_tiles;  // key blocks per (sequence, KV head), dK/dV kernel
  float scale;
  float scale_log2;
  float* delta;       // [B][Hq][q_len]: rowsum(dO * O), written by the dQ kernel
  void* dq;           // [B][q_len][Hq][D], element type of q
  float* dk_hat;      // [B][hat_cap][Hkv][D] fp32
  float* dv_hat;
  int hat_cap;
  SegmentTable segs;  // several speech runs per sequence when segs.seg_start is set
};

// Window pooling backward (Eq. 4): raw K/V gradients and the gate's.
struct PoolBwdArgs {
  const void* k_raw;
  const void* v_raw;
  int64_t stride_b, stride_s, stride_h;  // elements, shared by the raw gradients
  int raw_len;
  const int32_t* prefix_len;
  const int32_t* speech_len;
  const int32_t* suffix_len;
  int w_eff;
  int kv_heads;
  const float* gate;    // [Hkv][D] or null (zero gate)
  const float* dk_hat;  // [B][hat_cap][Hkv][D] fp32
  const float* dv_hat;
  int hat_cap;
  void* dk_raw;
  void* dv_raw;
  float* du_part;       // [batch][blocks_per_seq][Hkv][D] per-block partial gate gradients
  float* du;            // [Hkv][D] or null
  int max_out;          // bound on the compressed length
  int slots_per_block;
  int blocks_per_seq;
  SegmentTable segs;    // several speech runs per sequence when segs.seg_start is set
};

int prefill_bwd_rows_per_tile(int dtype, int group);
int prefill_bwd_keys_per_block(int dtype, int head_dim);  // keys of one dK/dV block
hipError_t launch_prefill_bwd(const PrefillBwdArgs& a, int dtype, int head_dim, int group,
                              int batch, hipStream_t s);
// Slots of one sequence a pooling-backward block covers (a multiple of the
// slots one pass of 256 threads covers), and so the size of the partial
// gate-gradient buffer; 0 when (kv_heads, head_dim) is not supported.
int pool_bwd_slots_per_block(int batch, int max_out, int kv_heads, int head_dim);
// The launch's slots per block and blocks per (sequence, head): sized from
// min(max_out, hat_cap), the slots that can hold work, and never more blocks
// than the workspace of pool_bwd_slots_per_block holds.  Arguments must have
// passed pool_bwd_slots_per_block.
void pool_bwd_grid(int batch, int max_out, int hat_cap, int kv_heads, int head_dim, int* spb, int* blocks);
hipError_t launch_pool_bwd(const PoolBwdArgs& a, int dtype, int head_dim, int batch,
                           hipStream_t s);

}  // namespace skv
