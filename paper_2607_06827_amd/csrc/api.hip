// C-ABI host layer of libspeechkv: argument validation, grid sizing and
// dispatch to the kernels.  Every check runs before the first HIP call, so a
// call that returns an error has enqueued nothing.  No allocation and no
// synchronisation.  The only global state is the per-device address of the
// static scratch array of speechkv_decode_attn_noalloc, set once per device.
#include "../../include/speechkv.h"

#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include "kernels.hpp"
#include "kernels_bwd.hpp"
#include "kernels_fused.hpp"

// Split partials of speechkv_decode_attn_noalloc.  Each GPU holds its own
// copy for the life of the process; every call on that GPU shares it.  The
// name is a host-side stand-in for the array, never a device address: host
// code uses only the address hipGetSymbolAddress returns for the current
// device, kept per device below.
static __device__ __align__(256) unsigned char scratch[SPEECHKV_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxGrid = 65535;
constexpr int kMaxRows = 2147483647 - SPEECHKV_MAX_WINDOW;  // ceil(T / w) stays in int32

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int elt_size(int dtype) { return dtype == SPEECHKV_DTYPE_BF16 ? 2 : 4; }

int log2_exact(int x) {
  int s = 0;
  while ((1 << s) < x) ++s;
  return (1 << s) == x ? s : -1;
}

// Checks shared by every call on the cache description.
int check_cache(const speechkv_paged_kv* c) {
  if (!c || !c->k_pages || !c->v_pages || !c->block_table) return SPEECHKV_ERR_INVALID_ARG;
  if (c->num_pages < 1 || c->max_pages_per_seq < 1 || c->num_kv_heads < 1)
    return SPEECHKV_ERR_INVALID_ARG;
  if (c->dtype != SPEECHKV_DTYPE_F32 && c->dtype != SPEECHKV_DTYPE_BF16) return SPEECHKV_ERR_UNSUPPORTED;
  if (c->head_dim != 64 && c->head_dim != 128) return SPEECHKV_ERR_UNSUPPORTED;
  if (c->page_size < 8 || c->page_size > 256 || log2_exact(c->page_size) < 0)
    return SPEECHKV_ERR_UNSUPPORTED;
  if (c->num_kv_heads > kMaxGrid) return SPEECHKV_ERR_UNSUPPORTED;
  if ((int64_t)c->max_pages_per_seq * c->page_size > INT32_MAX) return SPEECHKV_ERR_INVALID_ARG;
  if (!aligned16(c->k_pages) || !aligned16(c->v_pages)) return SPEECHKV_ERR_INVALID_ARG;
  return SPEECHKV_OK;
}

int check_spans(const speechkv_spans* s) {
  if (!s || !s->prefix_len || !s->speech_len || !s->suffix_len) return SPEECHKV_ERR_INVALID_ARG;
  if (s->max_speech_len < 0 || s->max_total_len < 0 || s->max_speech_len > s->max_total_len)
    return SPEECHKV_ERR_INVALID_ARG;
  return SPEECHKV_OK;
}

int check_segments(const speechkv_segments* g) {
  if (!g || !g->seg_start || !g->text_len || !g->speech_len) return SPEECHKV_ERR_INVALID_ARG;
  if (g->num_segments < 0 || g->max_segments < 0 || g->max_segments > SPEECHKV_MAX_SEGMENTS ||
      g->max_total_len < 0)
    return SPEECHKV_ERR_INVALID_ARG;
  return SPEECHKV_OK;
}

skv::SegmentTable table_of(const speechkv_segments* g) {
  skv::SegmentTable t;
  t.seg_start = g->seg_start;
  t.text_len = g->text_len;
  t.speech_len = g->speech_len;
  t.num_segments = g->num_segments;
  t.max_segs = g->max_segments;
  t.max_rows = g->max_total_len;
  return t;
}

// The one-run span arguments of a segment-table call: the kernels read the
// table instead, and these pointers stay unread.
speechkv_spans spans_of(const speechkv_segments* g) {
  speechkv_spans s;
  s.prefix_len = g->seg_start;
  s.speech_len = g->seg_start;
  s.suffix_len = g->seg_start;
  s.max_speech_len = 0;
  s.max_total_len = g->max_total_len;
  return s;
}

skv::PagedView view_of(const speechkv_paged_kv* c) {
  skv::PagedView v;
  v.num_pages = c->num_pages;
  v.page_shift = log2_exact(c->page_size);
  v.max_pages = c->max_pages_per_seq;
  v.kv_heads = c->num_kv_heads;
  return v;
}

int group_of(int num_q_heads, int num_kv_heads) {
  if (num_q_heads < 1 || num_q_heads % num_kv_heads) return -1;
  const int g = num_q_heads / num_kv_heads;
  return (g == 1 || g == 2 || g == 4 || g == 8) ? g : -1;
}

int64_t page_pool_bytes(const speechkv_paged_kv* c) {
  return (int64_t)c->num_pages * c->num_kv_heads * c->page_size * c->head_dim * elt_size(c->dtype);
}

bool overlaps(const void* a, int64_t na, const void* b, int64_t nb) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + (uintptr_t)nb && b0 < a0 + (uintptr_t)na;
}

int status_of(hipError_t e) { return e == hipSuccess ? SPEECHKV_OK : SPEECHKV_ERR_HIP; }

// A byte range of one argument; a null pointer takes no part in the checks.
struct Region {
  const void* p;
  int64_t n;
};

// True when a written region overlaps a read region or another written one.
bool aliased(const Region* wr, int nw, const Region* rd, int nr) {
  for (int i = 0; i < nw; ++i) {
    if (!wr[i].p) continue;
    for (int k = 0; k < nr; ++k)
      if (rd[k].p && overlaps(wr[i].p, wr[i].n, rd[k].p, rd[k].n)) return true;
    for (int k = i + 1; k < nw; ++k)
      if (wr[k].p && overlaps(wr[i].p, wr[i].n, wr[k].p, wr[k].n)) return true;
  }
  return false;
}

constexpr int kMaxDevices = 256;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mutex;

// Device address of the current device's copy of `scratch`, looked up once
// per device (with that device current) and kept.
hipError_t device_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress((void**)&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return e;
      if (!p) return hipErrorInvalidSymbol;
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return hipSuccess;
}

}  // namespace

extern "C" {

int64_t speechkv_compressed_len(int32_t prefix_len, int32_t speech_len, int32_t suffix_len,
                                int32_t w, int32_t layer, int32_t l0) {
  if (prefix_len < 0 || speech_len < 0 || suffix_len < 0 || w < 1 || layer < 0 || l0 < 0) return -1;
  const int64_t weff = layer >= l0 ? w : 1;
  return (int64_t)prefix_len + (speech_len + weff - 1) / weff + suffix_len;
}

int64_t speechkv_compressed_len_segments(const int32_t* text_len, const int32_t* speech_len,
                                         int32_t num_segments, int32_t w, int32_t layer,
                                         int32_t l0) {
  if (num_segments < 0 || (num_segments > 0 && (!text_len || !speech_len)) || w < 1 || layer < 0 ||
      l0 < 0)
    return -1;
  const int64_t weff = layer >= l0 ? w : 1;
  int64_t n = 0;
  for (int32_t i = 0; i < num_segments; ++i) {
    if (text_len[i] < 0 || speech_len[i] < 0) return -1;
    n += (int64_t)text_len[i] + (speech_len[i] + weff - 1) / weff;
  }
  return n;
}

int32_t speechkv_decode_num_splits(int32_t batch, int32_t num_kv_heads, int32_t max_cache_len) {
  if (batch < 1 || num_kv_heads < 1 || max_cache_len < 0) return -1;
  // Pick the split count with the smallest estimated launch time, among
  // powers of two (measured faster than the counts between them).  Model,
  // fitted to a sweep on MI355X over 1-64 sequences and 126-7788 keys with
  // bf16 rows of 128 (512 bytes of K and V per key and KV head): a 4-wave
  // block streams its range at ~0.016 us per key after ~1 us of fixed cost;
  // a launch moves at most ~6.5 TB/s; more than one split adds ~4 us (the
  // merge launch and the extra blocks' fixed costs; any value from 2.5 to
  // 4.5 us picks the same counts on the sweep, the larger one keeps marginal
  // short caches whole).  Short caches are therefore not split (the merge costs
  // more than the parallelism saves), long caches of few sequences are.
  // Each split keeps at least 16 groups of 4 keys (four per wave), and the
  // grid at most ~1024 blocks.
  const double units = (double)batch * num_kv_heads;
  const double L = max_cache_len;
  const double t_stream = units * L * 512.0 / 6.5e6;  // us at the bandwidth bound
  const int64_t groups = ((int64_t)max_cache_len + 3) / 4;
  const int64_t by_grid = std::max<int64_t>(1, (int64_t)((1024.0 + units - 1.0) / units));
  const int64_t s_max = std::max<int64_t>(1, std::min<int64_t>({32, groups / 16, by_grid}));
  int32_t best = 1;
  double best_t = 0.0;
  for (int64_t s = 1; s <= s_max; s *= 2) {
    const double t = std::max(1.0 + 0.016 * L / (double)s, t_stream) + (s > 1 ? 4.0 : 0.0);
    if (s == 1 || t < best_t) {
      best = (int32_t)s;
      best_t = t;
    }
  }
  return best;
}

size_t speechkv_decode_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                       int32_t head_dim, int32_t max_cache_len, int32_t num_splits) {
  if (batch < 1 || num_q_heads < 1 || num_kv_heads < 1 || head_dim < 1 || max_cache_len < 0 ||
      num_splits < 0)
    return 0;
  const int32_t s = num_splits ? num_splits : speechkv_decode_num_splits(batch, num_kv_heads, max_cache_len);
  if (s <= 1) return 0;
  const size_t rows = (size_t)batch * num_q_heads * s;
  size_t o_bytes = rows * head_dim * sizeof(float);
  o_bytes = (o_bytes + 255) & ~(size_t)255;
  return o_bytes + rows * 2 * sizeof(float);
}

const char* speechkv_status_string(int status) {
  switch (status) {
    case SPEECHKV_OK: return "ok";
    case SPEECHKV_ERR_INVALID_ARG: return "invalid argument";
    case SPEECHKV_ERR_UNSUPPORTED: return "unsupported dtype, head_dim, group size or page size";
    case SPEECHKV_ERR_WORKSPACE: return "workspace missing or too small";
    case SPEECHKV_ERR_ALIAS: return "a buffer written overlaps one read or another written";
    case SPEECHKV_ERR_HIP: return "HIP runtime error";
    case SPEECHKV_ERR_SCRATCH: return "the problem needs more than the library's static scratch holds";
    default: return "unknown status";
  }
}

const char* speechkv_version(void) { return "0.1.0"; }

// speechkv_pool_kv and speechkv_pool_kv_segments (segs set: several runs)
static int pool_kv_impl(const void* k_raw, const void* v_raw, int64_t stride_b, int64_t stride_s,
                        int64_t stride_h, int32_t batch, int32_t raw_len, const speechkv_spans* spans,
                        const skv::SegmentTable* segs, int32_t w, const float* gate_u, int32_t layer,
                        int32_t l0, const speechkv_paged_kv* cache, int32_t* cache_len_out,
                        void* stream) {
  if (!k_raw || !v_raw) return SPEECHKV_ERR_INVALID_ARG;
  int st = check_cache(cache);
  if (st) return st;
  if ((st = check_spans(spans))) return st;
  if (batch < 1 || batch > kMaxGrid || raw_len < 1 || raw_len > kMaxRows || w < 1 ||
      w > SPEECHKV_MAX_WINDOW || layer < 0 || l0 < 0)
    return SPEECHKV_ERR_INVALID_ARG;
  if (stride_b < 0 || stride_s < 0 || stride_h < 0) return SPEECHKV_ERR_INVALID_ARG;
  if (spans->max_total_len > raw_len) return SPEECHKV_ERR_INVALID_ARG;
  const int esz = elt_size(cache->dtype);
  const int D = cache->head_dim;
  const int64_t per16 = 16 / esz;  // elements per 16 bytes
  if (stride_b % per16 || stride_s % per16 || stride_h % per16) return SPEECHKV_ERR_INVALID_ARG;
  if (!aligned16(k_raw) || !aligned16(v_raw)) return SPEECHKV_ERR_INVALID_ARG;
  if (gate_u && !aligned16(gate_u)) return SPEECHKV_ERR_INVALID_ARG;
  // byte extent of the raw tensors versus the pool they are written into
  const int64_t last = (int64_t)(batch - 1) * stride_b + (int64_t)(raw_len - 1) * stride_s +
                       (int64_t)(cache->num_kv_heads - 1) * stride_h + D;
  const int64_t raw_bytes = last * esz;
  const int64_t pool_bytes = page_pool_bytes(cache);
  // the pools and the lengths written may not overlap what is read (raw K/V,
  // gate, block table, span lengths) or each other
  const int64_t lens = (int64_t)batch * 4;
  const Region rd[] = {{k_raw, raw_bytes}, {v_raw, raw_bytes},
                       {gate_u, (int64_t)cache->num_kv_heads * D * 4},
                       {cache->block_table, (int64_t)batch * cache->max_pages_per_seq * 4},
                       {spans->prefix_len, lens}, {spans->speech_len, lens},
                       {spans->suffix_len, lens}};
  const Region wr[] = {{cache->k_pages, pool_bytes}, {cache->v_pages, pool_bytes},
                       {cache_len_out, lens}};
  if (aliased(wr, 3, rd, 7)) return SPEECHKV_ERR_ALIAS;
  if (skv::pool_grid_blocks(spans->max_total_len, cache->num_kv_heads, D) > INT32_MAX)
    return SPEECHKV_ERR_UNSUPPORTED;
  skv::PoolArgs a;
  a.k_raw = k_raw;
  a.v_raw = v_raw;
  a.stride_b = stride_b;
  a.stride_s = stride_s;
  a.stride_h = stride_h;
  a.raw_len = raw_len;
  a.prefix_len = spans->prefix_len;
  a.speech_len = spans->speech_len;
  a.suffix_len = spans->suffix_len;
  a.w_eff = layer >= l0 ? w : 1;
  a.gate = gate_u;
  a.k_pages = cache->k_pages;
  a.v_pages = cache->v_pages;
  a.table = cache->block_table;
  a.pv = view_of(cache);
  a.cache_len_out = cache_len_out;
  a.max_out = spans->max_total_len;
  if (segs) a.segs = *segs;
  return status_of(skv::launch_pool(a, cache->dtype, D, batch, static_cast<hipStream_t>(stream)));
}

int speechkv_pool_kv(const void* k_raw, const void* v_raw, int64_t stride_b, int64_t stride_s,
                     int64_t stride_h, int32_t batch, int32_t raw_len, const speechkv_spans* spans,
                     int32_t w, const float* gate_u, int32_t layer, int32_t l0,
                     const speechkv_paged_kv* cache, int32_t* cache_len_out, void* stream) {
  return pool_kv_impl(k_raw, v_raw, stride_b, stride_s, stride_h, batch, raw_len, spans, nullptr, w,
                      gate_u, layer, l0, cache, cache_len_out, stream);
}

int speechkv_pool_kv_segments(const void* k_raw, const void* v_raw, int64_t stride_b,
                              int64_t stride_s, int64_t stride_h, int32_t batch, int32_t raw_len,
                              const speechkv_segments* segs, int32_t w, const float* gate_u,
                              int32_t layer, int32_t l0, const speechkv_paged_kv* cache,
                              int32_t* cache_len_out, void* stream) {
  const int st = check_segments(segs);
  if (st) return st;
  const speechkv_spans sp = spans_of(segs);
  const skv::SegmentTable t = table_of(segs);
  return pool_kv_impl(k_raw, v_raw, stride_b, stride_s, stride_h, batch, raw_len, &sp, &t, w,
                      gate_u, layer, l0, cache, cache_len_out, stream);
}

int speechkv_pool_hidden(const void* h, int64_t stride_b, int64_t stride_s, int32_t batch,
                         int32_t raw_len, int32_t hidden, int32_t dtype, const speechkv_spans* spans,
                         int32_t w, const float* gate_u, void* out, int64_t out_stride_b,
                         int64_t out_stride_s, int32_t out_capacity, int32_t* out_len, void* stream) {
  if (!h || !out) return SPEECHKV_ERR_INVALID_ARG;
  int st = check_spans(spans);
  if (st) return st;
  if (dtype != SPEECHKV_DTYPE_F32 && dtype != SPEECHKV_DTYPE_BF16) return SPEECHKV_ERR_UNSUPPORTED;
  if (!skv::pool_hidden_supported(hidden)) return SPEECHKV_ERR_UNSUPPORTED;
  if (batch < 1 || batch > kMaxGrid || raw_len < 1 || raw_len > kMaxRows || w < 1 ||
      w > SPEECHKV_MAX_WINDOW)
    return SPEECHKV_ERR_INVALID_ARG;
  if (stride_b < 0 || stride_s < 0 || out_stride_b < 0 || out_stride_s < 0) return SPEECHKV_ERR_INVALID_ARG;
  if (spans->max_total_len > raw_len || out_capacity < 1) return SPEECHKV_ERR_INVALID_ARG;
  const int esz = elt_size(dtype);
  const int64_t per16 = 16 / esz;
  if (stride_b % per16 || stride_s % per16 || out_stride_b % per16 || out_stride_s % per16)
    return SPEECHKV_ERR_INVALID_ARG;
  if (!aligned16(h) || !aligned16(out) || (gate_u && !aligned16(gate_u))) return SPEECHKV_ERR_INVALID_ARG;
  const int64_t in_bytes =
      ((int64_t)(batch - 1) * stride_b + (int64_t)(raw_len - 1) * stride_s + hidden) * esz;
  const int64_t out_bytes =
      ((int64_t)(batch - 1) * out_stride_b + (int64_t)(out_capacity - 1) * out_stride_s + hidden) * esz;
  if (overlaps(h, in_bytes, out, out_bytes)) return SPEECHKV_ERR_ALIAS;
  skv::PoolHiddenArgs a;
  a.h = h;
  a.stride_b = stride_b;
  a.stride_s = stride_s;
  a.raw_len = raw_len;
  a.prefix_len = spans->prefix_len;
  a.speech_len = spans->speech_len;
  a.suffix_len = spans->suffix_len;
  a.w = w;
  a.gate = gate_u;
  a.out = out;
  a.out_stride_b = out_stride_b;
  a.out_stride_s = out_stride_s;
  a.out_cap = out_capacity;
  a.out_len = out_len;
  // no output row at or past min(max_total_len, out_capacity) is written
  a.max_out = spans->max_total_len < out_capacity ? spans->max_total_len : out_capacity;
  return status_of(skv::launch_pool_hidden(a, dtype, hidden, batch, static_cast<hipStream_t>(stream)));
}

// Checks and launches of speechkv_decode_attn.  `workspace` holds the split
// partials when the step is split; its size has been checked by the caller.
static int decode_attn_impl(const void* q, int32_t batch, int32_t num_q_heads,
                            const speechkv_paged_kv* cache, const int32_t* cache_len,
                            int32_t max_cache_len, const void* k_new, const void* v_new,
                            float scale, int32_t splits, void* out, void* workspace, size_t need,
                            void* stream) {
  const int group = group_of(num_q_heads, cache->num_kv_heads);
  const int esz = elt_size(cache->dtype);
  const int D = cache->head_dim;
  // nothing written (out, the split partials, and the pools when the new
  // token is stored) may overlap anything read or another written region
  const int64_t qo_bytes = (int64_t)batch * num_q_heads * D * esz;
  const int64_t new_bytes = (int64_t)batch * cache->num_kv_heads * D * esz;
  const int64_t pool_bytes = page_pool_bytes(cache);
  const int64_t table_bytes = (int64_t)batch * cache->max_pages_per_seq * 4;
  // (the pools count as written when the new token is stored, else as read)
  const bool store = k_new != nullptr;
  const Region rd[] = {{q, qo_bytes}, {k_new, new_bytes}, {v_new, new_bytes},
                       {cache_len, (int64_t)batch * 4}, {cache->block_table, table_bytes},
                       {store ? nullptr : cache->k_pages, pool_bytes},
                       {store ? nullptr : cache->v_pages, pool_bytes}};
  const Region wr[] = {{out, qo_bytes}, {need ? workspace : nullptr, (int64_t)need},
                       {store ? cache->k_pages : nullptr, pool_bytes},
                       {store ? cache->v_pages : nullptr, pool_bytes}};
  if (aliased(wr, 4, rd, 7)) return SPEECHKV_ERR_ALIAS;
  skv::DecodeArgs a;
  a.q = q;
  a.k_pages = cache->k_pages;
  a.v_pages = cache->v_pages;
  a.table = cache->block_table;
  a.pv = view_of(cache);
  a.cache_len = cache_len;
  a.max_len = max_cache_len;
  a.k_new = k_new;
  a.v_new = v_new;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.num_splits = splits;
  a.out = out;
  a.ws_o = nullptr;
  a.ws_ml = nullptr;
  if (splits > 1) {
    const size_t rows = (size_t)batch * num_q_heads * splits;
    size_t o_bytes = rows * cache->head_dim * sizeof(float);
    o_bytes = (o_bytes + 255) & ~(size_t)255;
    a.ws_o = static_cast<float*>(workspace);
    a.ws_ml = reinterpret_cast<float*>(static_cast<char*>(workspace) + o_bytes);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = skv::launch_decode(a, cache->dtype, cache->head_dim, group, batch, s);
  if (e != hipSuccess) return SPEECHKV_ERR_HIP;
  if (splits > 1) e = skv::launch_decode_merge(a, cache->dtype, cache->head_dim, num_q_heads, batch, s);
  return status_of(e);
}

// Argument checks of both decode entry points; on success *splits holds the
// split count and *need the workspace bytes it takes.
static int check_decode(const void* q, int32_t batch, int32_t num_q_heads,
                        const speechkv_paged_kv* cache, const int32_t* cache_len,
                        int32_t max_cache_len, const void* k_new, const void* v_new, float scale,
                        int32_t num_splits, const void* out, int32_t* splits, size_t* need) {
  if (!q || !out || !cache_len) return SPEECHKV_ERR_INVALID_ARG;
  int st = check_cache(cache);
  if (st) return st;
  if (batch < 1 || batch > kMaxGrid || max_cache_len < 0 || num_splits < 0 || num_splits > kMaxGrid)
    return SPEECHKV_ERR_INVALID_ARG;
  if ((k_new == nullptr) != (v_new == nullptr)) return SPEECHKV_ERR_INVALID_ARG;
  if (!(scale > 0.f) || scale > 3.0e38f) return SPEECHKV_ERR_INVALID_ARG;  // finite, > 0
  if ((int64_t)max_cache_len > (int64_t)cache->max_pages_per_seq * cache->page_size)
    return SPEECHKV_ERR_INVALID_ARG;
  const int group = group_of(num_q_heads, cache->num_kv_heads);
  if (num_q_heads < 1 || num_q_heads % cache->num_kv_heads) return SPEECHKV_ERR_INVALID_ARG;
  if (group < 0) return SPEECHKV_ERR_UNSUPPORTED;
  if (!aligned16(q) || !aligned16(out) || (k_new && (!aligned16(k_new) || !aligned16(v_new))))
    return SPEECHKV_ERR_INVALID_ARG;
  *splits = num_splits ? num_splits
                       : speechkv_decode_num_splits(batch, cache->num_kv_heads, max_cache_len);
  *need = speechkv_decode_workspace_bytes(batch, num_q_heads, cache->num_kv_heads,
                                          cache->head_dim, max_cache_len, *splits);
  return SPEECHKV_OK;
}

int speechkv_decode_attn(const void* q, int32_t batch, int32_t num_q_heads,
                         const speechkv_paged_kv* cache, const int32_t* cache_len,
                         int32_t max_cache_len, const void* k_new, const void* v_new, float scale,
                         int32_t num_splits, void* out, void* workspace, size_t workspace_bytes,
                         void* stream) {
  int32_t splits = 0;
  size_t need = 0;
  const int st = check_decode(q, batch, num_q_heads, cache, cache_len, max_cache_len, k_new, v_new,
                              scale, num_splits, out, &splits, &need);
  if (st) return st;
  if (need && (!workspace || workspace_bytes < need || !aligned16(workspace))) return SPEECHKV_ERR_WORKSPACE;
  return decode_attn_impl(q, batch, num_q_heads, cache, cache_len, max_cache_len, k_new, v_new,
                          scale, splits, out, workspace, need, stream);
}

int speechkv_decode_attn_noalloc(const void* q, int32_t batch, int32_t num_q_heads,
                                 const speechkv_paged_kv* cache, const int32_t* cache_len,
                                 int32_t max_cache_len, const void* k_new, const void* v_new,
                                 float scale, int32_t num_splits, void* out, void* stream) {
  int32_t splits = 0;
  size_t need = 0;
  const int st = check_decode(q, batch, num_q_heads, cache, cache_len, max_cache_len, k_new, v_new,
                              scale, num_splits, out, &splits, &need);
  if (st) return st;
  if (need > (size_t)SPEECHKV_NOALLOC_SCRATCH_BYTES) return SPEECHKV_ERR_SCRATCH;
  void* ws = nullptr;
  if (need) {
    const hipError_t e = device_scratch(&ws);
    if (e != hipSuccess) return SPEECHKV_ERR_HIP;
  }
  return decode_attn_impl(q, batch, num_q_heads, cache, cache_len, max_cache_len, k_new, v_new,
                          scale, splits, out, ws, need, stream);
}

// speechkv_prefill_attn and speechkv_prefill_attn_segments (segs set)
static int prefill_attn_impl(const void* q, int32_t batch, int32_t num_q_heads, int32_t q_len,
                             const speechkv_paged_kv* cache, const speechkv_spans* spans,
                             const skv::SegmentTable* segs, int32_t w, int32_t layer, int32_t l0,
                             int32_t mask_mode, float scale, void* out, float* lse, void* stream) {
  if (!q || !out) return SPEECHKV_ERR_INVALID_ARG;
  int st = check_cache(cache);
  if (st) return st;
  if ((st = check_spans(spans))) return st;
  if (batch < 1 || q_len < 1 || q_len > kMaxRows || w < 1 || w > SPEECHKV_MAX_WINDOW ||
      layer < 0 || l0 < 0)
    return SPEECHKV_ERR_INVALID_ARG;
  if (mask_mode != SPEECHKV_MASK_WINDOW_END && mask_mode != SPEECHKV_MASK_WINDOW_START)
    return SPEECHKV_ERR_INVALID_ARG;
  if (spans->max_total_len > q_len) return SPEECHKV_ERR_INVALID_ARG;
  if (!(scale > 0.f) || scale > 3.0e38f) return SPEECHKV_ERR_INVALID_ARG;  // finite, > 0
  if (num_q_heads < 1 || num_q_heads % cache->num_kv_heads) return SPEECHKV_ERR_INVALID_ARG;
  const int group = group_of(num_q_heads, cache->num_kv_heads);
  if (group < 0) return SPEECHKV_ERR_UNSUPPORTED;
  if (!aligned16(q) || !aligned16(out) || (lse && (reinterpret_cast<uintptr_t>(lse) & 3u)))
    return SPEECHKV_ERR_INVALID_ARG;
  // out and lse may not overlap what is read (queries, pools, block table,
  // span lengths) or each other
  const int64_t qo_bytes =
      (int64_t)batch * q_len * num_q_heads * cache->head_dim * elt_size(cache->dtype);
  const int64_t pool_bytes = page_pool_bytes(cache);
  const int64_t lens = (int64_t)batch * 4;
  const Region rd[] = {{q, qo_bytes}, {cache->k_pages, pool_bytes}, {cache->v_pages, pool_bytes},
                       {cache->block_table, (int64_t)batch * cache->max_pages_per_seq * 4},
                       {spans->prefix_len, lens}, {spans->speech_len, lens},
                       {spans->suffix_len, lens}};
  const Region wr[] = {{out, qo_bytes}, {lse, (int64_t)batch * num_q_heads * q_len * 4}};
  if (aliased(wr, 2, rd, 7)) return SPEECHKV_ERR_ALIAS;
  if (spans->max_total_len == 0) return SPEECHKV_OK;
  const int rows_per_tile = skv::prefill_rows_per_tile(group);
  const int64_t tiles = (spans->max_total_len + rows_per_tile - 1) / rows_per_tile;
  if ((int64_t)batch * cache->num_kv_heads * tiles > INT32_MAX) return SPEECHKV_ERR_INVALID_ARG;
  skv::PrefillArgs a;
  a.q = q;
  a.out = out;
  a.lse = lse;
  a.k_pages = cache->k_pages;
  a.v_pages = cache->v_pages;
  a.table = cache->block_table;
  a.pv = view_of(cache);
  a.prefix_len = spans->prefix_len;
  a.speech_len = spans->speech_len;
  a.suffix_len = spans->suffix_len;
  a.w_eff = layer >= l0 ? w : 1;
  a.mask_mode = mask_mode;
  a.q_len = q_len;
  a.num_tiles = (int)tiles;
  a.num_q_heads = num_q_heads;
  a.scale_log2 = scale * 1.4426950408889634f;
  if (segs) a.segs = *segs;
  return status_of(skv::launch_prefill(a, cache->dtype, cache->head_dim, group, batch,
                                       static_cast<hipStream_t>(stream)));
}

int speechkv_prefill_attn(const void* q, int32_t batch, int32_t num_q_heads, int32_t q_len,
                          const speechkv_paged_kv* cache, const speechkv_spans* spans, int32_t w,
                          int32_t layer, int32_t l0, int32_t mask_mode, float scale, void* out,
                          float* lse, void* stream) {
  return prefill_attn_impl(q, batch, num_q_heads, q_len, cache, spans, nullptr, w, layer, l0,
                           mask_mode, scale, out, lse, stream);
}

int speechkv_prefill_attn_segments(const void* q, int32_t batch, int32_t num_q_heads,
                                   int32_t q_len, const speechkv_paged_kv* cache,
                                   const speechkv_segments* segs, int32_t w, int32_t layer,
                                   int32_t l0, int32_t mask_mode, float scale, void* out,
                                   float* lse, void* stream) {
  const int st = check_segments(segs);
  if (st) return st;
  const speechkv_spans sp = spans_of(segs);
  const skv::SegmentTable t = table_of(segs);
  return prefill_attn_impl(q, batch, num_q_heads, q_len, cache, &sp, &t, w, layer, l0, mask_mode,
                           scale, out, lse, stream);
}

int speechkv_pool_prefill_attn(const void* q, int32_t batch, int32_t num_q_heads, int32_t q_len,
                               const void* k_raw, const void* v_raw, int64_t stride_b,
                               int64_t stride_s, int64_t stride_h, int32_t raw_len,
                               const speechkv_spans* spans, int32_t w, const float* gate_u,
                               int32_t layer, int32_t l0, const speechkv_paged_kv* cache,
                               int32_t* cache_len_out, int32_t mask_mode, float scale, void* out,
                               float* lse, void* stream) {
  if (!q || !out || !k_raw || !v_raw) return SPEECHKV_ERR_INVALID_ARG;
  int st = check_cache(cache);
  if (st) return st;
  if ((st = check_spans(spans))) return st;
  if (cache->dtype != SPEECHKV_DTYPE_BF16) return SPEECHKV_ERR_UNSUPPORTED;
  if (batch < 1 || batch > kMaxGrid || q_len < 1 || q_len > kMaxRows || raw_len < 1 ||
      raw_len > kMaxRows || w < 1 || w > SPEECHKV_MAX_WINDOW || layer < 0 || l0 < 0)
    return SPEECHKV_ERR_INVALID_ARG;
  if (mask_mode != SPEECHKV_MASK_WINDOW_END && mask_mode != SPEECHKV_MASK_WINDOW_START)
    return SPEECHKV_ERR_INVALID_ARG;
  if (spans->max_total_len > q_len || spans->max_total_len > raw_len) return SPEECHKV_ERR_INVALID_ARG;
  if (!(scale > 0.f) || scale > 3.0e38f) return SPEECHKV_ERR_INVALID_ARG;  // finite, > 0
  if (num_q_heads < 1 || num_q_heads % cache->num_kv_heads) return SPEECHKV_ERR_INVALID_ARG;
  const int group = group_of(num_q_heads, cache->num_kv_heads);
  if (group < 0) return SPEECHKV_ERR_UNSUPPORTED;
  if (stride_b < 0 || stride_s < 0 || stride_h < 0) return SPEECHKV_ERR_INVALID_ARG;
  const int esz = elt_size(cache->dtype);
  const int D = cache->head_dim;
  const int64_t per16 = 16 / esz;
  if (stride_b % per16 || stride_s % per16 || stride_h % per16) return SPEECHKV_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(out) || !aligned16(k_raw) || !aligned16(v_raw) ||
      (gate_u && !aligned16(gate_u)) || (lse && (reinterpret_cast<uintptr_t>(lse) & 3u)))
    return SPEECHKV_ERR_INVALID_ARG;
  // nothing written (pages, out, lse) may overlap anything read (q, raw K/V,
  // gate) or another written region
  const int64_t raw_bytes = ((int64_t)(batch - 1) * stride_b + (int64_t)(raw_len - 1) * stride_s +
                             (int64_t)(cache->num_kv_heads - 1) * stride_h + D) * esz;
  const int64_t qo_bytes = (int64_t)batch * q_len * num_q_heads * D * esz;
  const int64_t lse_bytes = (int64_t)batch * num_q_heads * q_len * 4;
  const int64_t pool_bytes = page_pool_bytes(cache);
  const int64_t gate_bytes = (int64_t)cache->num_kv_heads * D * 4;
  const void* rd[] = {q, k_raw, v_raw, gate_u};
  const int64_t rd_n[] = {qo_bytes, raw_bytes, raw_bytes, gate_bytes};
  const void* wr[] = {cache->k_pages, cache->v_pages, out, lse};
  const int64_t wr_n[] = {pool_bytes, pool_bytes, qo_bytes, lse_bytes};
  for (int i = 0; i < 4; ++i) {
    if (!wr[i]) continue;
    for (int j = 0; j < 4; ++j)
      if (rd[j] && overlaps(wr[i], wr_n[i], rd[j], rd_n[j])) return SPEECHKV_ERR_ALIAS;
    for (int j = i + 1; j < 4; ++j)
      if (wr[j] && overlaps(wr[i], wr_n[i], wr[j], wr_n[j])) return SPEECHKV_ERR_ALIAS;
  }
  const int rows_per_tile = skv::prefill_fused_rows_per_tile(group);
  // at least one tile per (sequence, head): tile 0 writes cache_len_out
  int64_t tiles = (spans->max_total_len + rows_per_tile - 1) / rows_per_tile;
  if (tiles < 1) tiles = 1;
  if ((int64_t)batch * cache->num_kv_heads * tiles > INT32_MAX) return SPEECHKV_ERR_INVALID_ARG;
  skv::PrefillFusedArgs f;
  skv::PrefillArgs& a = f.at;
  a.q = q;
  a.out = out;
  a.lse = lse;
  a.k_pages = cache->k_pages;
  a.v_pages = cache->v_pages;
  a.table = cache->block_table;
  a.pv = view_of(cache);
  a.prefix_len = spans->prefix_len;
  a.speech_len = spans->speech_len;
  a.suffix_len = spans->suffix_len;
  a.w_eff = layer >= l0 ? w : 1;
  a.mask_mode = mask_mode;
  a.q_len = q_len;
  a.num_tiles = (int)tiles;
  a.num_q_heads = num_q_heads;
  a.scale_log2 = scale * 1.4426950408889634f;
  f.k_pages = cache->k_pages;
  f.v_pages = cache->v_pages;
  f.k_raw = k_raw;
  f.v_raw = v_raw;
  f.stride_b = stride_b;
  f.stride_s = stride_s;
  f.stride_h = stride_h;
  f.raw_len = raw_len;
  f.gate = gate_u;
  f.cache_len_out = cache_len_out;
  return status_of(skv::launch_prefill_fused(f, D, group, batch, static_cast<hipStream_t>(stream)));
}

size_t speechkv_prefill_attn_bwd_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t q_len) {
  if (batch < 1 || num_q_heads < 1 || q_len < 1) return 0;
  return (size_t)batch * num_q_heads * q_len * sizeof(float);
}

// speechkv_prefill_attn_bwd and speechkv_prefill_attn_bwd_segments (segs set)
static int prefill_attn_bwd_impl(const void* q, int32_t batch, int32_t num_q_heads, int32_t q_len,
                                 const speechkv_paged_kv* cache, const speechkv_spans* spans,
                                 const skv::SegmentTable* segs, int32_t w, int32_t layer, int32_t l0,
                                 int32_t mask_mode, float scale, const void* out, const float* lse,
                                 const void* dout, void* dq, float* dk_hat, float* dv_hat,
                                 int32_t hat_capacity, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  if (!q || !out || !lse || !dout || !dq || !dk_hat || !dv_hat) return SPEECHKV_ERR_INVALID_ARG;
  int st = check_cache(cache);
  if (st) return st;
  if ((st = check_spans(spans))) return st;
  if (batch < 1 || q_len < 1 || q_len > kMaxRows || w < 1 || w > SPEECHKV_MAX_WINDOW ||
      layer < 0 || l0 < 0 || hat_capacity < 1)
    return SPEECHKV_ERR_INVALID_ARG;
  if (mask_mode != SPEECHKV_MASK_WINDOW_END && mask_mode != SPEECHKV_MASK_WINDOW_START)
    return SPEECHKV_ERR_INVALID_ARG;
  if (spans->max_total_len > q_len) return SPEECHKV_ERR_INVALID_ARG;
  if (!(scale > 0.f) || scale > 3.0e38f) return SPEECHKV_ERR_INVALID_ARG;
  if (num_q_heads < 1 || num_q_heads % cache->num_kv_heads) return SPEECHKV_ERR_INVALID_ARG;
  const int group = group_of(num_q_heads, cache->num_kv_heads);
  if (group < 0) return SPEECHKV_ERR_UNSUPPORTED;
  const size_t need = speechkv_prefill_attn_bwd_workspace_bytes(batch, num_q_heads, q_len);
  if (!workspace || workspace_bytes < need) return SPEECHKV_ERR_WORKSPACE;
  if (!aligned16(q) || !aligned16(out) || !aligned16(dout) || !aligned16(dq) || !aligned16(dk_hat) ||
      !aligned16(dv_hat) || !aligned16(workspace) || (reinterpret_cast<uintptr_t>(lse) & 3u))
    return SPEECHKV_ERR_INVALID_ARG;
  const int esz = elt_size(cache->dtype);
  const int64_t qbytes = (int64_t)batch * q_len * num_q_heads * cache->head_dim * esz;
  const int64_t hbytes = (int64_t)batch * hat_capacity * cache->num_kv_heads * cache->head_dim * 4;
  // outputs must not overlap each other or the inputs they are computed from
  const void* outs[4] = {dq, dk_hat, dv_hat, workspace};
  const int64_t osz[4] = {qbytes, hbytes, hbytes, (int64_t)need};
  const void* ins[4] = {q, out, dout, lse};
  const int64_t isz[4] = {qbytes, qbytes, qbytes, (int64_t)batch * num_q_heads * q_len * 4};
  for (int i = 0; i < 4; ++i) {
    for (int k = i + 1; k < 4; ++k)
      if (overlaps(outs[i], osz[i], outs[k], osz[k])) return SPEECHKV_ERR_ALIAS;
    for (int k = 0; k < 4; ++k)
      if (overlaps(outs[i], osz[i], ins[k], isz[k])) return SPEECHKV_ERR_ALIAS;
    if (overlaps(outs[i], osz[i], cache->k_pages, page_pool_bytes(cache)) ||
        overlaps(outs[i], osz[i], cache->v_pages, page_pool_bytes(cache)))
      return SPEECHKV_ERR_ALIAS;
  }
  if (spans->max_total_len == 0) return SPEECHKV_OK;
  const int rows_per_tile = skv::prefill_bwd_rows_per_tile(cache->dtype, group);
  const int64_t q_tiles = (spans->max_total_len + rows_per_tile - 1) / rows_per_tile;
  const int64_t keys = spans->max_total_len < hat_capacity ? spans->max_total_len : hat_capacity;
  const int keys_per_block = skv::prefill_bwd_keys_per_block(cache->dtype, cache->head_dim);
  const int64_t key_tiles = (keys + keys_per_block - 1) / keys_per_block;
  if ((int64_t)batch * cache->num_kv_heads * q_tiles > INT32_MAX ||
      (int64_t)batch * cache->num_kv_heads * key_tiles > INT32_MAX)
    return SPEECHKV_ERR_INVALID_ARG;
  skv::PrefillBwdArgs a;
  a.q = q;
  a.out = out;
  a.dout = dout;
  a.lse = lse;
  a.k_pages = cache->k_pages;
  a.v_pages = cache->v_pages;
  a.table = cache->block_table;
  a.pv = view_of(cache);
  a.prefix_len = spans->prefix_len;
  a.speech_len = spans->speech_len;
  a.suffix_len = spans->suffix_len;
  a.w_eff = layer >= l0 ? w : 1;
  a.mask_mode = mask_mode;
  a.q_len = q_len;
  a.num_q_heads = num_q_heads;
  a.num_q_tiles = (int)q_tiles;
  a.num_key_tiles = (int)key_tiles;
  a.scale = scale;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.delta = static_cast<float*>(workspace);
  a.dq = dq;
  a.dk_hat = dk_hat;
  a.dv_hat = dv_hat;
  a.hat_cap = hat_capacity;
  if (segs) a.segs = *segs;
  return status_of(skv::launch_prefill_bwd(a, cache->dtype, cache->head_dim, group, batch,
                                           static_cast<hipStream_t>(stream)));
}

int speechkv_prefill_attn_bwd(const void* q, int32_t batch, int32_t num_q_heads, int32_t q_len,
                              const speechkv_paged_kv* cache, const speechkv_spans* spans, int32_t w,
                              int32_t layer, int32_t l0, int32_t mask_mode, float scale,
                              const void* out, const float* lse, const void* dout, void* dq,
                              float* dk_hat, float* dv_hat, int32_t hat_capacity, void* workspace,
                              size_t workspace_bytes, void* stream) {
  return prefill_attn_bwd_impl(q, batch, num_q_heads, q_len, cache, spans, nullptr, w, layer, l0,
                               mask_mode, scale, out, lse, dout, dq, dk_hat, dv_hat, hat_capacity,
                               workspace, workspace_bytes, stream);
}

int speechkv_prefill_attn_bwd_segments(const void* q, int32_t batch, int32_t num_q_heads,
                                       int32_t q_len, const speechkv_paged_kv* cache,
                                       const speechkv_segments* segs, int32_t w, int32_t layer,
                                       int32_t l0, int32_t mask_mode, float scale, const void* out,
                                       const float* lse, const void* dout, void* dq,
                                       float* dk_hat, float* dv_hat, int32_t hat_capacity,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  const int st = check_segments(segs);
  if (st) return st;
  const speechkv_spans sp = spans_of(segs);
  const skv::SegmentTable t = table_of(segs);
  return prefill_attn_bwd_impl(q, batch, num_q_heads, q_len, cache, &sp, &t, w, layer, l0,
                               mask_mode, scale, out, lse, dout, dq, dk_hat, dv_hat, hat_capacity,
                               workspace, workspace_bytes, stream);
}

size_t speechkv_pool_kv_bwd_workspace_bytes(int32_t batch, int32_t max_total_len,
                                            int32_t num_kv_heads, int32_t head_dim) {
  if (batch < 1 || max_total_len < 0 || num_kv_heads < 1) return 0;
  const int spb = skv::pool_bwd_slots_per_block(batch, max_total_len, num_kv_heads, head_dim);
  if (spb == 0) return 0;
  const int64_t blocks = max_total_len > 0 ? (max_total_len + spb - 1) / spb : 1;
  return (size_t)batch * blocks * num_kv_heads * head_dim * sizeof(float);
}

// speechkv_pool_kv_bwd and speechkv_pool_kv_bwd_segments (segs set)
static int pool_kv_bwd_impl(const void* k_raw, const void* v_raw, int64_t stride_b, int64_t stride_s,
                            int64_t stride_h, int32_t batch, int32_t raw_len, int32_t num_kv_heads,
                            int32_t head_dim, int32_t dtype, const speechkv_spans* spans,
                            const skv::SegmentTable* segs, int32_t w, const float* gate_u,
                            int32_t layer, int32_t l0, const float* dk_hat, const float* dv_hat,
                            int32_t hat_capacity, void* dk_raw, void* dv_raw, float* du,
                            void* workspace, size_t workspace_bytes, void* stream) {
  if (!k_raw || !v_raw || !dk_hat || !dv_hat || !dk_raw || !dv_raw) return SPEECHKV_ERR_INVALID_ARG;
  int st = check_spans(spans);
  if (st) return st;
  if (dtype != SPEECHKV_DTYPE_F32 && dtype != SPEECHKV_DTYPE_BF16) return SPEECHKV_ERR_UNSUPPORTED;
  if (head_dim != 64 && head_dim != 128) return SPEECHKV_ERR_UNSUPPORTED;
  if (num_kv_heads < 1 || batch < 1) return SPEECHKV_ERR_INVALID_ARG;
  if (num_kv_heads > kMaxGrid) return SPEECHKV_ERR_UNSUPPORTED;
  if (spans->max_total_len > raw_len) return SPEECHKV_ERR_INVALID_ARG;
  const int spb = skv::pool_bwd_slots_per_block(batch, spans->max_total_len, num_kv_heads, head_dim);
  if (spb == 0) return SPEECHKV_ERR_UNSUPPORTED;
  if (batch < 1 || batch > kMaxGrid || raw_len < 1 || raw_len > kMaxRows || w < 1 ||
      w > SPEECHKV_MAX_WINDOW || layer < 0 || l0 < 0 || hat_capacity < 1)
    return SPEECHKV_ERR_INVALID_ARG;
  if (stride_b < 0 || stride_s < 0 || stride_h < 0) return SPEECHKV_ERR_INVALID_ARG;
  if (spans->max_total_len > raw_len) return SPEECHKV_ERR_INVALID_ARG;
  const int esz = elt_size(dtype);
  const int64_t per16 = 16 / esz;
  if (stride_b % per16 || stride_s % per16 || stride_h % per16) return SPEECHKV_ERR_INVALID_ARG;
  if (!aligned16(k_raw) || !aligned16(v_raw) || !aligned16(dk_raw) || !aligned16(dv_raw) ||
      !aligned16(dk_hat) || !aligned16(dv_hat) || (gate_u && !aligned16(gate_u)) || (du && !aligned16(du)))
    return SPEECHKV_ERR_INVALID_ARG;
  const size_t need = du ? speechkv_pool_kv_bwd_workspace_bytes(batch, spans->max_total_len,
                                                                num_kv_heads, head_dim)
                         : 0;
  if (du && (!workspace || workspace_bytes < need || !aligned16(workspace))) return SPEECHKV_ERR_WORKSPACE;
  const int64_t raw_bytes = ((int64_t)(batch - 1) * stride_b + (int64_t)(raw_len - 1) * stride_s +
                             (int64_t)(num_kv_heads - 1) * stride_h + head_dim) * esz;
  const int64_t hbytes = (int64_t)batch * hat_capacity * num_kv_heads * head_dim * 4;
  const int64_t ubytes = (int64_t)num_kv_heads * head_dim * 4;
  const void* outs[4] = {dk_raw, dv_raw, du, du ? workspace : nullptr};
  const int64_t osz[4] = {raw_bytes, raw_bytes, ubytes, (int64_t)need};
  const void* ins[5] = {k_raw, v_raw, dk_hat, dv_hat, gate_u};
  const int64_t isz[5] = {raw_bytes, raw_bytes, hbytes, hbytes, ubytes};
  for (int i = 0; i < 4; ++i) {
    if (!outs[i]) continue;
    for (int k = i + 1; k < 4; ++k)
      if (outs[k] && overlaps(outs[i], osz[i], outs[k], osz[k])) return SPEECHKV_ERR_ALIAS;
    for (int k = 0; k < 5; ++k)
      if (ins[k] && overlaps(outs[i], osz[i], ins[k], isz[k])) return SPEECHKV_ERR_ALIAS;
  }
  skv::PoolBwdArgs a;
  a.k_raw = k_raw;
  a.v_raw = v_raw;
  a.stride_b = stride_b;
  a.stride_s = stride_s;
  a.stride_h = stride_h;
  a.raw_len = raw_len;
  a.prefix_len = spans->prefix_len;
  a.speech_len = spans->speech_len;
  a.suffix_len = spans->suffix_len;
  a.w_eff = layer >= l0 ? w : 1;
  a.kv_heads = num_kv_heads;
  a.gate = gate_u;
  a.dk_hat = dk_hat;
  a.dv_hat = dv_hat;
  a.hat_cap = hat_capacity;
  a.dk_raw = dk_raw;
  a.dv_raw = dv_raw;
  a.du = du;
  a.du_part = du ? static_cast<float*>(workspace) : nullptr;
  a.max_out = spans->max_total_len;
  skv::pool_bwd_grid(batch, spans->max_total_len, hat_capacity, num_kv_heads, head_dim, &a.slots_per_block,
                     &a.blocks_per_seq);
  if (segs) a.segs = *segs;
  return status_of(skv::launch_pool_bwd(a, dtype, head_dim, batch, static_cast<hipStream_t>(stream)));
}

int speechkv_pool_kv_bwd(const void* k_raw, const void* v_raw, int64_t stride_b, int64_t stride_s,
                         int64_t stride_h, int32_t batch, int32_t raw_len, int32_t num_kv_heads,
                         int32_t head_dim, int32_t dtype, const speechkv_spans* spans, int32_t w,
                         const float* gate_u, int32_t layer, int32_t l0, const float* dk_hat,
                         const float* dv_hat, int32_t hat_capacity, void* dk_raw, void* dv_raw,
                         float* du, void* workspace, size_t workspace_bytes, void* stream) {
  return pool_kv_bwd_impl(k_raw, v_raw, stride_b, stride_s, stride_h, batch, raw_len, num_kv_heads,
                          head_dim, dtype, spans, nullptr, w, gate_u, layer, l0, dk_hat, dv_hat,
                          hat_capacity, dk_raw, dv_raw, du, workspace, workspace_bytes, stream);
}

int speechkv_pool_kv_bwd_segments(const void* k_raw, const void* v_raw, int64_t stride_b,
                                  int64_t stride_s, int64_t stride_h, int32_t batch,
                                  int32_t raw_len, int32_t num_kv_heads, int32_t head_dim,
                                  int32_t dtype, const speechkv_segments* segs, int32_t w,
                                  const float* gate_u, int32_t layer, int32_t l0,
                                  const float* dk_hat, const float* dv_hat, int32_t hat_capacity,
                                  void* dk_raw, void* dv_raw, float* du, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  const int st = check_segments(segs);
  if (st) return st;
  const speechkv_spans sp = spans_of(segs);
  const skv::SegmentTable t = table_of(segs);
  return pool_kv_bwd_impl(k_raw, v_raw, stride_b, stride_s, stride_h, batch, raw_len, num_kv_heads,
                          head_dim, dtype, &sp, &t, w, gate_u, layer, l0, dk_hat, dv_hat,
                          hat_capacity, dk_raw, dv_raw, du, workspace, workspace_bytes, stream);
}

}  // extern "C"
