// One lane's share of the learned window pooling of Eq. 4 (arXiv 2607.06827,
// Sec. III-B): kLanes consecutive lanes own one (slot, KV head) unit, each
// lane 8 consecutive elements of the key and value rows.  The window's
// frames are taken in groups of four; the softmax over the gate logits
// u . k_j runs online over the groups (log2 units), and the same weights pool
// the keys and the values.  Both the pooling kernel and the prefill kernel
// that pools its key tiles on the fly use these steps, so the two produce the
// same bits for every pooled row.
#pragma once

#include "common.hpp"
#include "spans.hpp"

namespace skv {

template <typename T, int kLanes>
struct WindowPool {
  static constexpr float kLog2e = 1.4426950408889634f;
  float m, l, ak[8], av[8];

  __device__ __forceinline__ void init() {
    m = neg_inf();
    l = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) ak[i] = av[i] = 0.f;
  }

  // Frames f0 .. f0+3 of a window of `frames` rows; frames past the window
  // (their chunks may hold anything finite) get weight 0.  Without a gate
  // every logit is 0: uniform averaging.
  template <bool kGate>
  __device__ __forceinline__ void add4(const Chunk<T> (&kc)[4], const Chunk<T> (&vc)[4],
                                       const float (&u)[8], int f0, int frames) {
    // every operation rounds on its own (only the explicit fmaf are fused),
    // whatever code surrounds the call: the two kernels that use these steps
    // then agree bit for bit
#pragma clang fp contract(off)
    // (rows are converted to fp32 where they are used, which is exact, so
    // that four converted rows never need to be live at once)
    float s[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      float part = 0.f;
      if constexpr (kGate) {
        float kf[8];
        kc[t].to_float(kf);
#pragma unroll
        for (int i = 0; i < 8; ++i) part = __builtin_fmaf(u[i], kf[i], part);
        part = group_sum<kLanes>(part);
      }
      s[t] = f0 + t < frames ? part * kLog2e : neg_inf();  // log2 units
    }
    const float mn = fmaxf(m, fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])));
    const float corr = fast_exp2(m - mn);  // m = -inf on the first group gives 0
    l *= corr;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      ak[i] *= corr;
      av[i] *= corr;
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const float p = fast_exp2(s[t] - mn);
      float kf[8], vf[8];
      kc[t].to_float(kf);
      vc[t].to_float(vf);
      l += p;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        ak[i] = __builtin_fmaf(p, kf[i], ak[i]);
        av[i] = __builtin_fmaf(p, vf[i], av[i]);
      }
    }
    m = mn;
  }

  // Normalised pooled rows, rounded once to the element type.
  __device__ __forceinline__ void finish(Chunk<T>& ko, Chunk<T>& vo) {
#pragma clang fp contract(off)
    const float inv = 1.f / l;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      ak[i] *= inv;
      av[i] *= inv;
    }
    ko.from_float(ak);
    vo.from_float(av);
  }
};

}  // namespace skv
