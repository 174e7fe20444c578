// MFMA building blocks shared by the prefill attention kernels and their
// backward (arXiv 2607.06827, Sec. III-B, Eq. 5 under the causal mask over
// compressed positions): operand types and loads of the 32x32 bf16 / fp32
// MFMAs, untracked global-to-LDS staging with explicit waits, the block
// shapes and the exchange with the partner lane of the 32x32 C layout.
#pragma once

#include <type_traits>

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

// ------------------------------------------------- LDS staging and waits

typedef __attribute__((address_space(3))) void* lds_void_ptr;
typedef __attribute__((address_space(1))) void* global_void_ptr;

// Byte address of an LDS object (the 32-bit LDS address space).
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)(lds_void_ptr)p; }

// 16 bytes per lane from sbase + voff (bytes; sbase wave-uniform) into LDS at
// lds + 16 * lane, issued from inline assembly so that the compiler neither
// counts nor waits for it: the caller waits with an explicit vector-memory
// count.  (The compiler cannot tell which LDS object a transposed read
// touches, and with tracked direct loads it waits for all of them before every
// such read.)
__device__ __forceinline__ void lds_dma16(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}

// 4 bytes per lane from the per-lane address p into LDS at lds + 4 * lane,
// untracked like lds_dma16.
__device__ __forceinline__ void lds_dma4(const void* p, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off" : : "v"(p), "s"(lds) : "memory", "m0");
}

// 16 bytes at p + kOff into r, untracked like lds_dma16: the caller waits
// explicitly before r is read.
template <int kOff, typename F>
__device__ __forceinline__ void untracked_load16(F& r, const void* p) {
  static_assert(sizeof(F) == 16, "16-byte fragment");
  asm volatile("global_load_dwordx4 %0, %1, off offset:%2" : "=v"(r) : "v"(p), "i"(kOff) : "memory");
}

// s_waitcnt immediate: at most n vector-memory operations outstanding, LDS
// and scalar loads complete (CDNA layout: vmcnt bits 3:0 and 15:14, lgkmcnt
// 11:8, expcnt 6:4 left at its maximum)
constexpr int wait_vm_lgkm0(int n) { return 0x0070 | (n & 15) | ((n >> 4) << 14); }

// f(integral_constant<int, i>) for i = 0 .. n-1, unrolled at compile time
template <int n, int i = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (i < n) {
    f(std::integral_constant<int, i>());
    static_for<n, i + 1>(f);
  }
}

// Full barrier with no memory fence: waits until at most vm of the wave's
// (untracked) vector-memory operations are in flight and its LDS reads are
// done, then joins the block.  Compiler and scheduler fences on both sides
// keep every LDS access on its side.
template <int kVm>
__device__ __forceinline__ void bare_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(kVm));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Work item of block bid in a grid of nblk = P x T blocks over P pairs
// (sequence, KV head) x T query tiles, the work of a tile growing with its
// index.  XCD x (= bid mod 8) runs the items of a contiguous range of pairs,
// whose tiles then share that XCD's L2 copy of the pairs' K/V; each pair's
// tiles run heaviest first, pair after pair, so that heavy and light blocks
// share the CUs throughout.  A grid of at most three rounds of blocks on the
// 256 CUs (three 4-wave blocks each) ends with whatever its last round
// holds: there, when the pairs split evenly over the XCDs, an XCD takes them
// in groups of kTileGroupPairs, the heaviest tile of each pair of a group
// first, then the next heaviest, so that the blocks to start last are the
// lightest (1596 x 471, b = 8: -7%; the 60 s stack's 6656-block grids run
// faster pair after pair).
constexpr int kTileGroupPairs = 8;
constexpr int kHeaviestFirstBlocks = 3 * 3 * 256;
__device__ __forceinline__ void query_tile_item(int bid, int nblk, int T, int& pair, int& tile) {
  const int xcd = bid & 7, per = nblk >> 3, rem = nblk & 7;
  const int local = bid >> 3;
  if (nblk <= kHeaviestFirstBlocks && rem == 0 && per % T == 0) {
    const int np = per / T;                          // pairs per XCD
    const int grp = local / (kTileGroupPairs * T);   // group of pairs
    const int in = local - grp * kTileGroupPairs * T;
    const int gp = min(kTileGroupPairs, np - grp * kTileGroupPairs);  // pairs in this group
    pair = xcd * np + grp * kTileGroupPairs + in % gp;
    tile = T - 1 - in / gp;
  } else {
    const int item = xcd * per + min(xcd, rem) + local;
    pair = item / T;
    tile = T - 1 - item % T;
  }
}

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
