// Device helpers shared by the SpeechKV kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace skv {

typedef unsigned short bf16_bits;  // raw bf16 storage

// ------------------------------------------------------------------ numerics

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

typedef __bf16 bf16x2_hw __attribute__((ext_vector_type(2)));

// Round-to-nearest-even fp32 -> bf16 with v_cvt_pk_bf16_f32 (bit-identical to
// the textbook RNE bit manipulation, NaN stays NaN); two values per
// instruction, the first in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_hw v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint32_t f32_to_bf16(float f) { return pack_bf16x2(f, 0.f) & 0xffffu; }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

// ------------------------------------------------------ 8-element row chunks
// Every kernel moves head_dim rows in chunks of 8 elements: 16 bytes of bf16
// or 32 bytes of fp32.

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <typename T>
struct Chunk;

template <>
struct Chunk<bf16_bits> {
  uint4 raw;  // 8 bf16
  __device__ __forceinline__ void load(const bf16_bits* p) { raw = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void store(bf16_bits* p) const { *reinterpret_cast<uint4*>(p) = raw; }
  // non-temporal store: for rows no later access of this kernel touches
  __device__ __forceinline__ void store_nt(bf16_bits* p) const {
    const u32x4_t v = {raw.x, raw.y, raw.z, raw.w};
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t*>(p));
  }
  __device__ __forceinline__ void zero() { raw = make_uint4(0, 0, 0, 0); }
  __device__ __forceinline__ void to_float(float* f) const {
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ __forceinline__ void from_float(const float* f) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(f[2 * i], f[2 * i + 1]);
    raw = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

template <>
struct Chunk<float> {
  float4 a, b;  // 8 fp32
  __device__ __forceinline__ void load(const float* p) {
    a = reinterpret_cast<const float4*>(p)[0];
    b = reinterpret_cast<const float4*>(p)[1];
  }
  __device__ __forceinline__ void store(float* p) const {
    reinterpret_cast<float4*>(p)[0] = a;
    reinterpret_cast<float4*>(p)[1] = b;
  }
  __device__ __forceinline__ void store_nt(float* p) const {
    const f32x4_t va = {a.x, a.y, a.z, a.w}, vb = {b.x, b.y, b.z, b.w};
    __builtin_nontemporal_store(va, reinterpret_cast<f32x4_t*>(p));
    __builtin_nontemporal_store(vb, reinterpret_cast<f32x4_t*>(p) + 1);
  }
  __device__ __forceinline__ void zero() {
    a = make_float4(0.f, 0.f, 0.f, 0.f);
    b = a;
  }
  __device__ __forceinline__ void to_float(float* f) const {
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
    f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
  __device__ __forceinline__ void from_float(const float* f) {
    a = make_float4(f[0], f[1], f[2], f[3]);
    b = make_float4(f[4], f[5], f[6], f[7]);
  }
};

// -------------------------------------------------------- lane reductions
// DPP row operations act inside rows of 16 lanes.  After the four steps
// below every lane of a 16-lane row (8-lane group for kLanes = 8) holds the
// row's sum.

// Every pattern used here reads a lane of the same row that exists, so the
// "old" operand never shows and bound_ctrl only spares a register copy.
template <int kCtrl>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), kCtrl, 0xf, 0xf, true));
}

constexpr int kDppQuadXor1 = 0xB1;    // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;    // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <- 7 - i within 8
constexpr int kDppMirror = 0x140;     // lane i <- 15 - i within 16
constexpr int kDppRowRor8 = 0x128;    // lane i <- (i + 8) mod 16 within 16 (= i ^ 8)
constexpr int kDppRowBcast0 = 0x150;  // row_newbcast:n (+ n): lane n of each row to the row

// s_waitcnt immediate (CDNA layout: vmcnt bits 3:0 and 15:14, expcnt 6:4,
// lgkmcnt 11:8) that waits for every outstanding vector-memory operation and
// leaves the other counters alone
constexpr int kWaitVmcnt0 = 0x0F70;

template <int kLanes>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(kLanes == 8 || kLanes == 16, "group of 8 or 16 lanes");
  x += dpp<kDppQuadXor1>(x);
  x += dpp<kDppQuadXor2>(x);
  x += dpp<kDppHalfMirror>(x);
  if (kLanes == 16) x += dpp<kDppMirror>(x);
  return x;
}

__device__ __forceinline__ float xor_shuffle(float x, int mask) { return __shfl_xor(x, mask, 64); }

// ----------------------------------------------------------- paged cache
struct PagedView {
  int64_t num_pages;
  int page_shift;      // log2(page_size)
  int max_pages;       // per sequence
  int kv_heads;
};

// Element offset of row `slot` of (page, head) in a [pages][heads][page][D] pool.
template <int D>
__device__ __forceinline__ int64_t page_row(int64_t page, int head, int slot, const PagedView& pv) {
  return (((page * pv.kv_heads + head) << pv.page_shift) + slot) * (int64_t)D;
}

// Page holding cache slot c of sequence b, or -1 when the table entry is out
// of range (the caller then skips the row).
__device__ __forceinline__ int64_t page_of(const int32_t* __restrict__ table, int b, int c,
                                           const PagedView& pv) {
  int idx = c >> pv.page_shift;
  if (idx >= pv.max_pages) return -1;
  int64_t page = table[(int64_t)b * pv.max_pages + idx];
  return (page >= 0 && page < pv.num_pages) ? page : -1;
}

}  // namespace skv
