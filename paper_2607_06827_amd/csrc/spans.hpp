// Where the rows of a sequence come from, and from which full-resolution
// position each compressed key is visible (arXiv 2607.06827, Sec. III-B:
// Eq. 4 pools each window of w speech frames, text rows are kept, and the
// causal mask over compressed positions keeps attention causal).
//
// Two forms of sequence, each a "span view" with the same interface:
//   OneRun   [P text | T speech | N text], in closed form;
//   Runs     any number of segments [text_len[i] text | speech_len[i]
//            speech], each speech run pooled in windows that start at its
//            own first frame (a multi-turn input), by a scan over the
//            sequence's segments.
// A view answers: rows() and clen() (raw and compressed lengths), slot(c)
// (first raw row and frame count of compressed slot c; one frame for a text
// row), visible(p, mode) (how many compressed keys row p sees: they are a
// prefix of the cache, as the position a key becomes visible at grows with
// c) and visible_from(c, mode) (that position).  Mask modes: 0 = a window is visible from its last frame, 1 = from its
// first frame.
#pragma once

#include "common.hpp"

namespace skv {

struct SlotSource {
  int first, frames;
  __device__ __forceinline__ SlotSource() : first(0), frames(1) {}
  // slot c of one run with P text rows, T frames in nW windows of w, then text
  __device__ __forceinline__ SlotSource(int c, int P, int T, int nW, int w) {
    const bool text_before = c < P, text_after = c >= P + nW;
    first = text_before ? c : text_after ? P + T + (c - P - nW) : P + (c - P) * w;
    frames = (text_before || text_after) ? 1 : min(w, P + T - first);
  }
};

// Number of compressed keys visible from full-resolution row p of one run.
__device__ __forceinline__ int visible_keys(int p, int P, int T, int nW, int w, int mode) {
  if (p < P) return p + 1;
  const int t = p - P;
  if (t < T) {
    if (mode == 1) return P + t / w + 1;        // window visible from its first frame
    return (t == T - 1) ? P + nW : P + (t + 1) / w;  // ... from its last frame
  }
  return P + nW + (t - T) + 1;
}

// Full-resolution row from which compressed key c of one run is visible.
__device__ __forceinline__ int key_visible_from(int c, int P, int T, int nW, int w, int mode) {
  if (c < P) return c;
  if (c < P + nW) {
    const int i = c - P;
    if (mode == 1) return P + i * w;
    return min(P + (i + 1) * w, P + T) - 1;
  }
  return P + T + (c - P - nW);
}

// Several speech runs per sequence (segments in a table).
struct SegmentTable {
  const int32_t* seg_start = nullptr;   // [batch + 1]: sequence b owns segments [seg_start[b], seg_start[b+1])
  const int32_t* text_len = nullptr;    // [num_segments]
  const int32_t* speech_len = nullptr;  // [num_segments]
  int num_segments = 0;
  int max_segs = 0;                     // bound on the segments of one sequence (loop bound)
  int max_rows = 0;                     // bound on the rows of one sequence
};

struct OneRun {
  int P, T, N, w, nW;
  __device__ __forceinline__ OneRun(int p, int t, int n, int w_)
      : P(max(p, 0)), T(max(t, 0)), N(max(n, 0)), w(w_), nW((T + w_ - 1) / w_) {}
  __device__ __forceinline__ int rows() const { return P + T + N; }
  __device__ __forceinline__ int clen() const { return P + nW + N; }
  __device__ __forceinline__ SlotSource slot(int c) const { return SlotSource(c, P, T, nW, w); }
  __device__ __forceinline__ int visible(int p, int mode) const {
    return visible_keys(p, P, T, nW, w, mode);
  }
  __device__ __forceinline__ int visible_from(int c, int mode) const {
    return key_visible_from(c, P, T, nW, w, mode);
  }
};

// The segments of one sequence, read from the table with every device value
// clamped: at most max_segs segments, lengths >= 0, and no more than
// max_rows rows in all (a segment that would pass it is cut there), so every
// position the view returns lies in [0, max_rows].
struct Runs {
  const int32_t* text;
  const int32_t* speech;
  int s0, s1;   // segment range
  int w;
  int rows_, clen_;
  int max_rows;

  __device__ __forceinline__ Runs(const SegmentTable& t, int b, int w_) {
    text = t.text_len;
    speech = t.speech_len;
    w = w_;
    max_rows = t.max_rows;
    s0 = min(max(t.seg_start[b], 0), t.num_segments);
    s1 = min(max(t.seg_start[b + 1], s0), min(t.num_segments, s0 + t.max_segs));
    int r = 0, c = 0;
    for (int i = s0; i < s1; ++i) {
      int tl, sl;
      lengths(i, r, tl, sl);
      r += tl + sl;
      c += tl + (sl + w - 1) / w;
    }
    rows_ = r;
    clen_ = c;
  }
  // lengths of segment i given the r rows before it, cut at max_rows
  __device__ __forceinline__ void lengths(int i, int r, int& tl, int& sl) const {
    tl = min(max(text[i], 0), max_rows - r);
    sl = min(max(speech[i], 0), max_rows - r - tl);
  }
  __device__ __forceinline__ int rows() const { return rows_; }
  __device__ __forceinline__ int clen() const { return clen_; }

  __device__ __forceinline__ SlotSource slot(int c) const {
    SlotSource s;
    int r = 0, cc = 0;
    for (int i = s0; i < s1; ++i) {
      int tl, sl;
      lengths(i, r, tl, sl);
      const int nw = (sl + w - 1) / w;
      if (c < cc + tl) {
        s.first = r + (c - cc);
        s.frames = 1;
        return s;
      }
      if (c < cc + tl + nw) {
        const int f = (c - cc - tl) * w;
        s.first = r + tl + f;
        s.frames = min(w, sl - f);
        return s;
      }
      r += tl + sl;
      cc += tl + nw;
    }
    s.first = max(r - 1, 0);  // past the sequence: its last row (never stored)
    s.frames = 1;
    return s;
  }

  __device__ __forceinline__ int visible(int p, int mode) const {
    int r = 0, cc = 0;
    for (int i = s0; i < s1; ++i) {
      int tl, sl;
      lengths(i, r, tl, sl);
      const int nw = (sl + w - 1) / w;
      if (p < r + tl) return cc + (p - r) + 1;
      if (p < r + tl + sl) {
        const int f = p - r - tl;
        if (mode == 1) return cc + tl + f / w + 1;
        return cc + tl + (f == sl - 1 ? nw : (f + 1) / w);
      }
      r += tl + sl;
      cc += tl + nw;
    }
    return cc;
  }

  // row from which key c is visible (past the sequence: its row count)
  __device__ __forceinline__ int visible_from(int c, int mode) const {
    int r = 0, cc = 0;
    for (int i = s0; i < s1; ++i) {
      int tl, sl;
      lengths(i, r, tl, sl);
      const int nw = (sl + w - 1) / w;
      if (c < cc + tl) return r + (c - cc);
      if (c < cc + tl + nw) {
        const int f = (c - cc - tl) * w;
        return r + tl + (mode == 1 ? f : min(f + w, sl) - 1);
      }
      r += tl + sl;
      cc += tl + nw;
    }
    return r;
  }
};

// One run's three lengths, requested in one batch of scalar loads: one round
// trip before anything that depends on them, where the compiler had waited
// for each load in turn (blocks of a few steps spend a good part of their
// time in that prologue).  b must be uniform over the wave, as it is in every
// kernel here (it comes from the block index; the compiler cannot always tell,
// hence the readfirstlane).
__device__ __forceinline__ OneRun one_run_now(const int32_t* prefix, const int32_t* speech,
                                              const int32_t* suffix, int b, int w) {
  b = __builtin_amdgcn_readfirstlane(b);
  int p, t, n;
  asm volatile(
      "s_load_dword %0, %3, 0x0\n\t"
      "s_load_dword %1, %4, 0x0\n\t"
      "s_load_dword %2, %5, 0x0\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&s"(p), "=&s"(t), "=&s"(n)
      : "s"(prefix + b), "s"(speech + b), "s"(suffix + b)
      : "memory");
  return OneRun(p, t, n, w);
}

// The span view of sequence b: the segment table when kRuns, else the
// one-run spans of the argument struct.
template <bool kRuns, typename A>
__device__ __forceinline__ auto span_view(const A& a, int b, int w) {
  if constexpr (kRuns)
    return Runs(a.segs, b, w);
  else
    return one_run_now(a.prefix_len, a.speech_len, a.suffix_len, b, w);
}

}  // namespace skv
