// Attainable HBM read bandwidth on this device, measured beside the
// published peak: a non-temporal streaming read of two equal buffers (the
// shape of a decode launch, which reads a K and a V pool).  Each wave reads a
// contiguous range of both buffers as whole 1 KB wave-wide loads, `depth`
// loads per buffer in flight.  It moves the bytes and does nothing else, so
// its rate is a ceiling for any kernel that must read the same bytes once.
//
// Benchmark infrastructure only: built into its own library, loaded by the
// benchmark script, and not part of the SpeechKV interface.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 stream_load(const char* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// Wave q reads bytes [q * per_wave, min((q + 1) * per_wave, bytes)) of a and
// of b; per_wave and bytes are multiples of 1 KB.
template <int kDepth>
__global__ void stream_read_kernel(const char* __restrict__ a, const char* __restrict__ b,
                                   size_t per_wave, size_t bytes, uint32_t* sink) {
  const int lane = threadIdx.x & 63;
  const size_t wave = (size_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
  const size_t lo = wave * per_wave;
  const size_t hi = lo + per_wave < bytes ? lo + per_wave : bytes;
  u32x4 acc = {0, 0, 0, 0};
  size_t off = lo;
  for (; off + 1024 * kDepth <= hi; off += 1024 * kDepth) {
    u32x4 x[kDepth], y[kDepth];
#pragma unroll
    for (int i = 0; i < kDepth; ++i) {
      x[i] = stream_load(a + off + 1024 * i + 16 * lane);
      y[i] = stream_load(b + off + 1024 * i + 16 * lane);
    }
#pragma unroll
    for (int i = 0; i < kDepth; ++i) acc ^= x[i] ^ y[i];
  }
  for (; off + 1024 <= hi; off += 1024) acc ^= stream_load(a + off + 16 * lane) ^ stream_load(b + off + 16 * lane);
  // keeps the loads alive; the pattern never occurs in practice, and a write
  // here would be harmless anyway
  if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9e3779b9u) sink[0] = 1;
}

}  // namespace

// Reads `bytes` (a positive multiple of 1024) of each of a and b with
// `blocks` x `threads` (threads a multiple of 64, at most 1024) and depth in
// {1, 2, 4, 8}.  sink: device uint32, never written in practice.  Returns 0,
// -1 for bad arguments, or the HIP error of the launch.
extern "C" int skv_stream_read(const void* a, const void* b, size_t bytes, int blocks, int threads,
                               int depth, void* sink, void* stream) {
  if (!a || !b || !sink || bytes == 0 || bytes % 1024 || blocks < 1 || threads < 64 ||
      threads > 1024 || threads % 64)
    return -1;
  const size_t waves = (size_t)blocks * (threads / 64);
  size_t per_wave = (bytes + waves - 1) / waves;
  per_wave = (per_wave + 1023) / 1024 * 1024;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const char* pa = static_cast<const char*>(a);
  const char* pb = static_cast<const char*>(b);
  uint32_t* k = static_cast<uint32_t*>(sink);
  switch (depth) {
    case 1: hipLaunchKernelGGL(stream_read_kernel<1>, dim3(blocks), dim3(threads), 0, s, pa, pb, per_wave, bytes, k); break;
    case 2: hipLaunchKernelGGL(stream_read_kernel<2>, dim3(blocks), dim3(threads), 0, s, pa, pb, per_wave, bytes, k); break;
    case 4: hipLaunchKernelGGL(stream_read_kernel<4>, dim3(blocks), dim3(threads), 0, s, pa, pb, per_wave, bytes, k); break;
    case 8: hipLaunchKernelGGL(stream_read_kernel<8>, dim3(blocks), dim3(threads), 0, s, pa, pb, per_wave, bytes, k); break;
    default: return -1;
  }
  return (int)hipGetLastError();
}
