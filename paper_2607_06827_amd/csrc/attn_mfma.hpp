// MFMA building blocks shared by the prefill attention kernels and their
// backward (arXiv 2607.06827, Sec. III-B, Eq. 5 under the causal mask over
// compressed positions): operand types and loads of the 32x32 bf16 / fp32
// MFMAs, the visibility rule n_vis(p), the block shapes and the exchange with
// the partner lane of the 32x32 C layout.
#pragma once

#include "common.hpp"
#include "spans.hpp"

namespace skv {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned short u16x8_t __attribute__((ext_vector_type(8)));
typedef unsigned short u16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

template <typename T>
struct Mfma;

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t* lds_s16x4_ptr;

template <>
struct Mfma<bf16_bits> {
  static constexpr int kPack = 8;    // elements per lane per operand
  static constexpr int kRowV = 160;  // V row stride in elements (80 words = 16 mod 64 banks)
  typedef bf16x8_t Frag;
  static __device__ __forceinline__ f32x16_t mma(Frag a, Frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ Frag load(const bf16_bits* p) {
    return __builtin_bit_cast(Frag, *reinterpret_cast<const u16x8_t*>(p));
  }
  static __device__ __forceinline__ Frag zero() { return __builtin_bit_cast(Frag, u16x8_t{0, 0, 0, 0, 0, 0, 0, 0}); }
  // A operand of O^T += V^T P^T for keys 16kk.. and head-dim block db, read
  // from the row-major V tile with the gfx950 LDS transpose read.  In MFMA
  // order lane (m = lane%32, h = lane/32) needs column m's keys 16kk + 4h +
  // {0..3} and 16kk + 8 + 4h + {0..3} (the key order of the S^T C layout).
  // ds_read_b64_tr_b16 gives lane i of a 16-lane group element (row 4r +
  // i/4, column i%4) of the 16 x 4 block its lanes point at, so lane j of
  // group g points at key 16kk + 4(g/2) + j/4 (+8 for the second read),
  // elements 32db + 16(g%2) + 4(j%4) .. +3.
  // (kRow: row stride of the tile in elements; any row-major [key][d] tile
  // in LDS can be read transposed this way)
  template <int kRow = kRowV>
  static __device__ __forceinline__ Frag load_v(const bf16_bits* sv, int kk, int db, int lane) {
    const int g = lane >> 4, j = lane & 15;
    const bf16_bits* p = sv + (16 * kk + 4 * (g >> 1) + (j >> 2)) * kRow + 32 * db + 16 * (g & 1) + 4 * (j & 3);
    const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)p);
    const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)(p + 8 * kRow));
    const u16x8_t v = {(unsigned short)lo[0], (unsigned short)lo[1], (unsigned short)lo[2], (unsigned short)lo[3],
                       (unsigned short)hi[0], (unsigned short)hi[1], (unsigned short)hi[2], (unsigned short)hi[3]};
    return __builtin_bit_cast(Frag, v);
  }
  // round-to-nearest-even pack of 8 probabilities (v_cvt_pk_bf16_f32)
  static __device__ __forceinline__ Frag pack_p(const float* p) {
    Frag f;
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = (__bf16)p[i];
    return f;
  }
  // four output values of one row, rounded to bf16, stored as 8 bytes
  static __device__ __forceinline__ void store4(bf16_bits* dst, float a, float b, float c, float d) {
    bf16x4_t v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
    *reinterpret_cast<bf16x4_t*>(dst) = v;
  }
};

template <>
struct Mfma<float> {
  static constexpr int kPack = 1;
  static constexpr int kRowV = 160;  // V row stride in elements (160 words = 32 mod 64 banks)
  typedef float Frag;
  static __device__ __forceinline__ f32x16_t mma(Frag a, Frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ Frag load(const float* p) { return *p; }
  static __device__ __forceinline__ Frag zero() { return 0.f; }
  // A operand of O^T += V^T P^T: lane (m = lane%32, hg = lane/32) takes key
  // 8*(kk/4) + 4*hg + (kk%4) (the key order of the S^T C layout), column m
  // of head-dim block db, from the row-major V tile
  template <int kRow = kRowV>
  static __device__ __forceinline__ Frag load_v(const float* sv, int kk, int db, int lane) {
    const int hg = lane >> 5, m = lane & 31;
    return sv[(8 * (kk / 4) + 4 * hg + (kk % 4)) * kRow + 32 * db + m];
  }
  static __device__ __forceinline__ Frag pack_p(const float* p) { return p[0]; }
  static __device__ __forceinline__ void store4(float* dst, float a, float b, float c, float d) {
    *reinterpret_cast<float4*>(dst) = make_float4(a, b, c, d);
  }
};

template <int G>
struct PrefillShape {
  static constexpr int kRowBlocks = G >= 4 ? 1 : 4 / G;
  static constexpr int kWaves = G * kRowBlocks;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kRows = 32 * kRowBlocks;
};

__device__ __forceinline__ float partner_max(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto p = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}

__device__ __forceinline__ float partner_sum(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto p = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

}  // namespace skv
