// Full-resolution queries attending over the compressed cache under the
// causal mask over compressed positions (arXiv 2607.06827, Sec. III-B, Eq. 5
// and the mask described after it; Sec. III-C: the same computation runs on
// the fly in training).
//
// Mask.  Key c is visible from full-resolution position tau(c): prefix keys at
// their own position, pooled window i at its last frame (WINDOW_END) or first
// frame (WINDOW_START), suffix key m at P + T + m.  tau is increasing, so row
// p sees the prefix [0, n_vis(p)) of the cache: a query tile needs only the
// key tiles below n_vis of its last row, and only the tiles that straddle the
// n_vis of some row of a wave are masked element by element.  With several
// speech runs per sequence (kRuns) the same holds run by run, and n_vis comes
// from a scan of the sequence's segments (spans.hpp).
//
// Tiling (wave64, 32x32 MFMA).  A block owns one (sequence, KV head) and 32*RB
// query rows for all G query heads of the group (G*RB waves, RB = max(1, 4/G)),
// so every K/V tile staged in LDS serves G*RB waves.  Each wave holds its 32
// query rows in registers and, per 32-key tile, computes
//     S^T = K Q^T            (keys x queries; A = K tile, B = Q^T)
// so that the C layout puts one query per lane column.  The online softmax
// then runs per lane (row max exchanged with the partner lane l^32 by a
// permlane swap, rescaling only when the max grows by more than 2^8), and the
// probabilities already sit in the B-operand layout of
//     O^T += V^T P^T          (A = V^T tile from LDS, B = P^T)
// with the key order of the C layout carried into the V reads.  bf16 uses
// v_mfma_f32_32x32x16_bf16 (8 elements per lane per operand), fp32 uses
// v_mfma_f32_32x32x2_f32 (1 element), both accumulating in fp32.
//
// K and V tiles are both staged row-major in LDS behind a branch-free
// pipeline with one barrier per tile.  fp32: double-buffered, block-table
// entries three tiles ahead, K/V rows two tiles ahead in registers (whole
// 256-byte rows per wave-wide load), LDS one tile ahead.  bf16: three
// buffers filled straight from the paged cache by direct loads two tiles
// ahead, entries three tiles ahead as scalar loads.  The bf16 V^T operand
// comes from the row-major V tile through the gfx950 LDS transpose read
// (ds_read_b64_tr_b16), so no register transpose is needed at staging; row
// strides or swizzles put every staging write and operand read on distinct
// banks.  The output tile goes back through LDS so that rows leave as
// 16-byte stores.
//
// Blocks are remapped so that the eight XCDs each run a contiguous range of
// (sequence, head, tile) items: tiles of one (b, g) share that XCD's L2 copy
// of the compressed K/V.  Heavy tiles (late rows) are issued first.
#include <type_traits>

#include "attn_mfma.hpp"
#include "kernels.hpp"
#include "kernels_fused.hpp"
#include "pool_window.hpp"

namespace skv {

namespace {

// Running maxima may lag the true maximum by up to 2^kSlack in the exponent
// before the accumulators are rescaled; the final division by the weight sum
// makes the choice of reference exact.
constexpr float kSlack = 8.f;

template <typename T, int D, int G, bool kRuns>
__global__ __launch_bounds__(PrefillShape<G>::kThreads) void prefill_kernel(PrefillArgs a) {
  typedef Mfma<T> M;
  typedef typename M::Frag Frag;
  constexpr int kThreads = PrefillShape<G>::kThreads;
  constexpr int kWaves = PrefillShape<G>::kWaves;
  constexpr int kRows = PrefillShape<G>::kRows;
  constexpr int kKeys = 32;                       // keys per tile
  constexpr int kPack = M::kPack;
  constexpr int kStep = 2 * kPack;                // head-dim elements per QK MFMA
  constexpr int kQChunks = D / kStep;
  constexpr int kElems16 = 16 / (int)sizeof(T);   // elements per 16-byte chunk
  constexpr int kChunksPerRow = D / kElems16;
  constexpr int kRowK = D + kElems16;             // padded K row (elements)
  constexpr int kRowV = M::kRowV;                 // padded V^T row (elements)
  constexpr int kItems = kKeys * kChunksPerRow;  // staging work: (key, 16-byte chunk)
  constexpr int kItemsPerThread = (kItems + kThreads - 1) / kThreads;
  constexpr int kTileK = kKeys * kRowK, kTileV = kKeys * kRowV;
  constexpr int kRowO = D + kElems16;             // padded output row (elements)
  constexpr float kLn2 = 0.6931471805599453f;
  // the output tiles of all waves go through the staging buffers when they fit
  constexpr bool kStageOut = kWaves * 32 * kRowO <= 2 * (kTileK + kTileV);

  __shared__ __attribute__((aligned(16))) T s_buf[2 * (kTileK + kTileV)];

  // XCD-aware, heaviest-first item order
  int pair, tile;
  query_tile_item(blockIdx.x, gridDim.x, a.num_tiles, pair, tile);
  const int heads = a.pv.kv_heads;
  const int g = pair % heads;
  const int b = pair / heads;

  const int w = a.w_eff;
  const auto sp = span_view<kRuns>(a, b, w);
  const int rows = min(sp.rows(), a.q_len);
  const int clen = min(sp.clen(), a.pv.max_pages << a.pv.page_shift);
  const int p0 = tile * kRows;
  if (p0 >= rows) return;
  const int kmax = min(sp.visible(min(p0 + kRows, rows) - 1, a.mask_mode), clen);

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = g * G + wave % G;
  const int col = lane & 31, hg = lane >> 5;
  const int wrow0 = p0 + (wave / G) * 32;  // first row of this wave
  const int p = wrow0 + col;
  const bool qvalid = p < rows;
  const int nvis = qvalid ? min(sp.visible(p, a.mask_mode), clen) : 0;
  // keys every valid row of the wave sees (n_vis grows with the row)
  const int nvis_lo = wrow0 < rows ? min(sp.visible(wrow0, a.mask_mode), clen) : 0;
  const int hq = a.num_q_heads;
  const int slot_mask = (1 << a.pv.page_shift) - 1;


  f32x16_t o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
  float m_run = neg_inf(), l_run = 0.f;

  const T* kpool = static_cast<const T*>(a.k_pages);
  const T* vpool = static_cast<const T*>(a.v_pages);
  const int ntiles = (kmax + kKeys - 1) / kKeys;

  // Staging pipeline, branch-free so that every wait covers exactly the loads
  // it needs: the block-table entries of tile t are loaded at the start of
  // tile t-3, the K/V rows of tile t at the start of tile t-2 (two register
  // sets), and tile t is written to LDS at the end of tile t-1 (two LDS
  // buffers).  Each thread owns staging items (key, 16-byte chunk), chunks
  // fastest, so each wave-wide load reads whole rows and each LDS row write
  // covers all banks once.  K and V are both staged row-major.  Tiles past
  // the last one load clamped, in-range addresses and are never read.
  const int32_t* table_row = a.table + (int64_t)b * a.pv.max_pages;
  const int64_t num_pages = a.pv.num_pages;
  const int shift = a.pv.page_shift;
  int pg[2][kItemsPerThread];  // table entries, by tile parity
  uint4 rk[2][kItemsPerThread], rv[2][kItemsPerThread];  // by tile parity
  uint32_t okm[2];  // bit it: item it holds a valid key
  auto item_key = [&](int it) { return (tid + it * kThreads) / kChunksPerRow; };  // key within the tile
  auto item_chunk = [&](int it) { return (tid + it * kThreads) % kChunksPerRow; };
  auto table_load = [&](int kt, int* pgs) {
#pragma unroll
    for (int it = 0; it < kItemsPerThread; ++it)
      pgs[it] = table_row[min((kt * kKeys + item_key(it)) >> shift, a.pv.max_pages - 1)];
  };
  auto fetch = [&](int kt, const int* pgs, uint4* rks, uint4* rvs, uint32_t& oks) {
    oks = 0;
#pragma unroll
    for (int it = 0; it < kItemsPerThread; ++it) {
      const int key = kt * kKeys + item_key(it);
      const int page = pgs[it];
      const bool ok = key < kmax && page >= 0 && page < num_pages;
      oks |= ok ? 1u << it : 0u;
      const int64_t off = page_row<D>(ok ? page : 0, g, key & slot_mask, a.pv) + item_chunk(it) * kElems16;
      rks[it] = *reinterpret_cast<const uint4*>(kpool + off);
      rvs[it] = *reinterpret_cast<const uint4*>(vpool + off);
    }
  };
  auto stage = [&](int buf, const uint4* rks, const uint4* rvs, uint32_t oks) {
    T* sk = s_buf + buf * (kTileK + kTileV);
    T* sv = sk + kTileK;
#pragma unroll
    for (int it = 0; it < kItemsPerThread; ++it) {
      if (tid + it * kThreads >= kItems) continue;
      const int key = item_key(it), ch = item_chunk(it);
      // rows of keys past the visible range (or of a bad table entry) are
      // zero: their V would otherwise meet a zero weight as 0 * garbage
      // (masked word by word, so that the rows stay in registers)
      const uint32_t m = 0u - ((oks >> it) & 1u);
      const uint4 kv = rks[it], vv = rvs[it];
      *reinterpret_cast<uint4*>(&sk[key * kRowK + ch * kElems16]) = make_uint4(kv.x & m, kv.y & m, kv.z & m, kv.w & m);
      *reinterpret_cast<uint4*>(&sv[key * kRowV + ch * kElems16]) = make_uint4(vv.x & m, vv.y & m, vv.z & m, vv.w & m);
    }
  };

  // prologue: tables of tiles 0..2, K/V of tiles 0 and 1, then this lane's
  // query row (the B operand of S^T = K Q^T), then tile 0 into LDS.  The
  // memory counter is in order: issued after the first fetches, the query
  // loads arrive while tile 0 is in flight instead of delaying it.
  table_load(0, pg[0]);
  table_load(1, pg[1]);
  fetch(0, pg[0], rk[0], rv[0], okm[0]);
  table_load(2, pg[0]);
  fetch(1, pg[1], rk[1], rv[1], okm[1]);
  // (rows past the end read row 0 of the sequence: finite, never stored)
  __builtin_amdgcn_sched_barrier(0);  // keep this issue order
  Frag qf[kQChunks];
  const T* qrow = static_cast<const T*>(a.q) + (((int64_t)b * a.q_len + (qvalid ? p : 0)) * hq + h) * D;
#pragma unroll
  for (int kc = 0; kc < kQChunks; ++kc) qf[kc] = M::load(qrow + kc * kStep + hg * kPack);
  __builtin_amdgcn_sched_barrier(0);
  stage(0, rk[0], rv[0], okm[0]);
  __syncthreads();
  // tile 0 needs the queries, and every load of the prologue was issued
  // before them; one wait here leaves nothing of the prologue pending at the
  // loop head, where it would make every iteration's waits conservative
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);

  // one tile of the steady state; kPar = kt & 1 (compile-time register sets)
  auto tile_step = [&](int kt, auto par) {
    constexpr int kPar = decltype(par)::value;
    constexpr int kOther = 1 - kPar;
    table_load(kt + 3, pg[kOther]);                          // tile kt+3: parity of kt+1
    fetch(kt + 2, pg[kPar], rk[kPar], rv[kPar], okm[kPar]);  // tile kt+2: parity of kt
    const int kb = kt * kKeys;
    const T* sk = s_buf + kPar * (kTileK + kTileV);
    const T* sv = sk + kTileK;
    if (kt < ntiles) {  // (the loop runs an even number of steps)
      // S^T tile: row = key (8*(i/4) + 4*hg + i%4), column = this lane's query
      f32x16_t st;
  #pragma unroll
      for (int i = 0; i < 16; ++i) st[i] = 0.f;
      const T* krow = &sk[col * kRowK + hg * kPack];
  #pragma unroll
      for (int kc = 0; kc < kQChunks; ++kc) st = M::mma(M::load(krow + kc * kStep), qf[kc], st);

      float pr[16];
      float mt = neg_inf();
      const bool masked = kb + kKeys > nvis_lo;  // uniform over the wave
      if (masked) {
  #pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kb + 8 * (i / 4) + 4 * hg + (i % 4);
          pr[i] = key < nvis ? st[i] : neg_inf();
          mt = fmaxf(mt, pr[i]);
        }
      } else {
  #pragma unroll
        for (int i = 0; i < 16; ++i) {
          pr[i] = st[i];
          mt = fmaxf(mt, pr[i]);
        }
      }
      mt = partner_max(mt) * a.scale_log2;  // the scale is > 0
      if (mt > m_run + kSlack) {
        const float corr = fast_exp2(m_run - mt);
        l_run *= corr;
  #pragma unroll
        for (int db = 0; db < D / 32; ++db)
  #pragma unroll
          for (int i = 0; i < 16; ++i) o[db][i] *= corr;
        m_run = mt;
      }
      float sum = 0.f;
  #pragma unroll
      for (int i = 0; i < 16; ++i) {
        pr[i] = fast_exp2(__builtin_fmaf(pr[i], a.scale_log2, -m_run));
        if (masked) pr[i] = m_run == neg_inf() ? 0.f : pr[i];  // nothing visible yet
        sum += pr[i];
      }
      l_run += sum;

      // O^T += V^T P^T over the 32 keys of the tile
  #pragma unroll
      for (int kk = 0; kk < kKeys / kStep; ++kk) {
        const Frag pf = M::pack_p(pr + kk * kPack);
  #pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const Frag vf = M::load_v(sv, kk, db, lane);
          o[db] = M::mma(vf, pf, o[db]);
        }
      }
    }
    stage(kOther, rk[kOther], rv[kOther], okm[kOther]);  // tile kt+1 (never read past the end)
    __syncthreads();
  };
  // two steps per iteration so that the register sets are compile-time; the
  // loads and stores of a step past the last tile are harmless
  for (int kt = 0; kt < ntiles; kt += 2) {
    tile_step(kt, std::integral_constant<int, 0>());
    tile_step(kt + 1, std::integral_constant<int, 1>());
  }

  const float l_tot = partner_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (hg == 0 && a.lse && qvalid)
    a.lse[((int64_t)b * hq + h) * a.q_len + p] = l_tot > 0.f ? (m_run + __log2f(l_tot)) * kLn2 : neg_inf();

  if (!kStageOut) {  // direct stores of the C layout: four values per row
    if (qvalid) {
      T* orow = static_cast<T*>(a.out) + (((int64_t)b * a.q_len + p) * hq + h) * D;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int ig = 0; ig < 4; ++ig)
          M::store4(orow + db * 32 + 8 * ig + 4 * hg, o[db][4 * ig] * inv, o[db][4 * ig + 1] * inv,
                    o[db][4 * ig + 2] * inv, o[db][4 * ig + 3] * inv);
    }
    return;
  }
  // output: through LDS, one 32 x D tile per wave, then 16-byte row stores
  // (the barrier after the last tile has freed the staging buffers)
  T* so = s_buf + wave * 32 * kRowO;
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int ig = 0; ig < 4; ++ig)
      M::store4(&so[col * kRowO + db * 32 + 8 * ig + 4 * hg], o[db][4 * ig] * inv, o[db][4 * ig + 1] * inv,
                o[db][4 * ig + 2] * inv, o[db][4 * ig + 3] * inv);
  __syncthreads();
  constexpr int kLanesPerRow = D / kElems16;      // 16-byte chunks per row
  constexpr int kRowsPerPass = 64 / kLanesPerRow;
  const int rsub = lane / kLanesPerRow, cch = lane % kLanesPerRow;
#pragma unroll
  for (int r0 = 0; r0 < 32; r0 += kRowsPerPass) {
    const int rr = r0 + rsub;
    const int out_row = wrow0 + rr;
    if (out_row < rows) {
      const uint4 v = *reinterpret_cast<const uint4*>(&so[rr * kRowO + cch * kElems16]);
      *reinterpret_cast<uint4*>(static_cast<T*>(a.out) + (((int64_t)b * a.q_len + out_row) * hq + h) * D +
                                cch * kElems16) = v;
    }
  }
}

// bf16 prefill with the K/V tiles moved straight from the paged cache into
// LDS by the gfx950 direct loads (global_load_lds_dwordx4): no staging
// registers, no staging writes.  A wave-wide direct load fills 1 KB of LDS
// in lane order, so tile rows are unpadded (D elements) and 16-byte chunks
// are XOR-swizzled within a row instead: chunk c of row r sits at position
// c ^ swz(r), with swz_k(r) = r mod 16 (the QK reads of 16 rows at one
// chunk hit distinct banks) and swz_v(r) = (r mod 4) * 4 (the transposed PV
// reads of 4 rows x 4 chunks hit distinct banks).  The loading lane picks the
// global chunk that belongs at its LDS position.  Keys past the visible range
// load a visible row (finite data that the mask gives zero weight).  Tile
// buffers are 256-byte aligned, so a lane's fragment addresses differ from
// one base register by an XOR of the swizzled chunk bits (see attend_tile).
template <int D>
struct LdsSwz {
  static constexpr int kChunks = D / 8;  // 16-byte chunks per row
  static __device__ __forceinline__ int k(int row) { return row & (kChunks >= 16 ? 15 : kChunks - 1); }
  static __device__ __forceinline__ int v(int row) { return (row % (kChunks / 4)) << 2; }
};

// One 32-key tile of the online softmax for the 32 query rows of a wave
// (bf16).  sk / sv: the swizzled row-major K and V tiles in LDS; qf: the
// wave's query fragments (B operand of S^T = K Q^T); kb: first key of the
// tile; nvis: keys this lane's row sees, nvis_lo: keys every row of the wave
// sees.  The K fragments are read three ahead of the S chain, the first V
// fragments during the softmax and the rest one ahead of the P.V chain.
template <int D>
__device__ __forceinline__ void attend_tile(const bf16_bits* sk, const bf16_bits* sv,
                                            const bf16x8_t (&qf)[D / 16], f32x16_t (&o)[D / 32],
                                            float& m_run, float& l_run, int kb, int nvis, int nvis_lo,
                                            int lane, float scale_log2) {
  typedef Mfma<bf16_bits> M;
  typedef M::Frag Frag;
  typedef LdsSwz<D> Swz;
  typedef __attribute__((address_space(3))) const u16x8_t* lds_frag_ptr;
  constexpr int kKeys = 32;
  constexpr int kStep = 16;                 // head-dim elements per QK MFMA
  constexpr int kQChunks = D / kStep;
  constexpr int kVFrags = (kKeys / kStep) * (D / 32);
  const int col = lane & 31, hg = lane >> 5;

  // S^T tile: row = key (8*(i/4) + 4*hg + i%4), column = this lane's query.
  // K fragment kc of this lane is row col, 16-byte chunk (2kc + hg) ^ swz(col)
  // = 2kc ^ c0 with c0 = hg ^ swz(col): byte address a0 ^ 32kc.
  uint32_t a0 = lds_addr(sk + col * D) + ((uint32_t)(hg ^ Swz::k(col)) << 4);
  asm volatile("" : "+v"(a0));  // one address register, not one per fragment
  auto kfrag = [&](int kc) __attribute__((always_inline)) {
    return __builtin_bit_cast(Frag, *(lds_frag_ptr)(uintptr_t)(a0 ^ (uint32_t)(32 * kc)));
  };
  f32x16_t st;
#pragma unroll
  for (int i = 0; i < 16; ++i) st[i] = 0.f;
  constexpr int kAhead = kQChunks >= 3 ? 3 : kQChunks;
  Frag kbuf[kAhead];
#pragma unroll
  for (int j = 0; j < kAhead; ++j) kbuf[j] = kfrag(j);
#pragma unroll
  for (int kc = 0; kc < kQChunks; ++kc) {
    const Frag cur = kbuf[kc % kAhead];
    if (kc + kAhead < kQChunks) kbuf[kc % kAhead] = kfrag(kc + kAhead);
    st = M::mma(cur, qf[kc], st);
  }
  __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);  // DS reads
#pragma unroll
  for (int kc = 0; kc + kAhead < kQChunks; ++kc) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, kAhead, 0);

  // A operand of O^T += V^T P^T through the LDS transpose read (see
  // Mfma<bf16_bits>::load_v): lane (vg, vj) reads key rows 16kk + 4(vg/2) +
  // vj/4 (and +8), elements 32db + 16(vg%2) + 4(vj%4) .. +3, whose 16-byte
  // chunk 4db + c1 sits at (4db + c1) ^ swz_v(row) = 4(db ^ s) + c1 (s =
  // swz_v(row)/4, the same for both rows and every kk): byte address va ^
  // 64db plus a constant for kk and the second row.
  const int vg = lane >> 4, vj = lane & 15;
  const int vr = 4 * (vg >> 1) + (vj >> 2);
  uint32_t va = lds_addr(sv + vr * D) +
                (uint32_t)((((Swz::v(vr) >> 2) * 4 + 2 * (vg & 1) + ((vj & 3) >> 1)) << 4) | ((vj & 1) << 3));
  asm volatile("" : "+v"(va));
  auto vfrag = [&](int idx) __attribute__((always_inline)) {
    const int kk = idx / (D / 32), db = idx % (D / 32);
    const uint32_t al = (va ^ (uint32_t)(64 * db)) + (uint32_t)(kk * 16 * D * 2);
    const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)(uintptr_t)al);
    const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)(uintptr_t)(al + 8 * D * 2));
    const u16x8_t v = {(unsigned short)lo[0], (unsigned short)lo[1], (unsigned short)lo[2], (unsigned short)lo[3],
                       (unsigned short)hi[0], (unsigned short)hi[1], (unsigned short)hi[2], (unsigned short)hi[3]};
    return __builtin_bit_cast(Frag, v);
  };
  Frag vbuf[2] = {vfrag(0), vfrag(1)};
  __builtin_amdgcn_sched_barrier(0);  // (issued before the softmax)

  float pr[16];
  float mt = neg_inf();
  if (kb + kKeys > nvis_lo) {  // uniform: the tile straddles some row's bound
    const int lim = nvis - kb - 4 * hg;  // element i is visible iff 8(i/4) + i%4 < lim
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      pr[i] = 8 * (i / 4) + (i % 4) < lim ? st[i] : neg_inf();
      mt = fmaxf(mt, pr[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      pr[i] = st[i];
      mt = fmaxf(mt, pr[i]);
    }
  }
  mt = partner_max(mt) * scale_log2;  // the scale is > 0
  if (mt > m_run + kSlack) {
    if (m_run != neg_inf()) {  // (before the first visible key o and l are still 0)
      const float corr = fast_exp2(m_run - mt);
      l_run *= corr;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[db][i] *= corr;
    }
    m_run = mt;
  }
  // a row that sees no key yet has m_run = -inf and every logit -inf:
  // reference 0 turns each weight into exp2(-inf) = 0
  const float m_use = m_run == neg_inf() ? 0.f : m_run;
  // the sum is of the unrounded weights, so that the log-sum-exp output
  // gives weights that sum to 1 when the backward recomputes them
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    pr[i] = fast_exp2(__builtin_fmaf(pr[i], scale_log2, -m_use));
    sum += pr[i];
  }
  l_run += sum;

  // O^T += V^T P^T over the 32 keys (the key order of the C layout carried
  // into the V reads), one V fragment ahead of each MFMA
#pragma unroll
  for (int kk = 0; kk < kKeys / kStep; ++kk) {
    const Frag pf = M::pack_p(pr + kk * 8);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const int idx = kk * (D / 32) + db;
      const Frag cur = vbuf[idx & 1];
      if (idx + 2 < kVFrags) vbuf[idx & 1] = vfrag(idx + 2);
      o[db] = M::mma(cur, pf, o[db]);
    }
  }
#pragma unroll
  for (int idx = 0; idx + 2 < kVFrags; ++idx) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 2, 1);
}

// Normalises the wave's 32 x D output tile, writes its LSE and stores it:
// through so (a 32-row tile area of LDS no other wave uses, rows swizzled
// like K) as 16-byte row stores, or straight from the C layout (so = null).
template <int D>
__device__ __forceinline__ void finish_rows(f32x16_t (&o)[D / 32], float m_run, float l_run, bf16_bits* so,
                                            const PrefillArgs& a, int b, int h, int wrow0, int rows, int lane) {
  typedef Mfma<bf16_bits> M;
  typedef LdsSwz<D> Swz;
  constexpr float kLn2 = 0.6931471805599453f;
  const int col = lane & 31, hg = lane >> 5;
  const int p = wrow0 + col;
  const int hq = a.num_q_heads;
  const float l_tot = partner_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (hg == 0 && a.lse && p < rows)
    a.lse[((int64_t)b * hq + h) * a.q_len + p] = l_tot > 0.f ? (m_run + __log2f(l_tot)) * kLn2 : neg_inf();
  bf16_bits* out = static_cast<bf16_bits*>(a.out);
  if (so == nullptr) {  // direct stores of the C layout: four values of a row
    if (p < rows) {
      bf16_bits* orow = out + (((int64_t)b * a.q_len + p) * hq + h) * D;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int ig = 0; ig < 4; ++ig)
          M::store4(orow + db * 32 + 8 * ig + 4 * hg, o[db][4 * ig] * inv, o[db][4 * ig + 1] * inv,
                    o[db][4 * ig + 2] * inv, o[db][4 * ig + 3] * inv);
    }
    return;
  }
  const int oswz = Swz::k(col);
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int ig = 0; ig < 4; ++ig)
      M::store4(so + col * D + (((4 * db + ig) ^ oswz) << 3) + 4 * hg, o[db][4 * ig] * inv,
                o[db][4 * ig + 1] * inv, o[db][4 * ig + 2] * inv, o[db][4 * ig + 3] * inv);
  __syncthreads();  // (the same wave reads its tile back: orders its LDS traffic)
  constexpr int kChunks = Swz::kChunks;
  constexpr int kRowsPerPass = 64 / kChunks;
#pragma unroll
  for (int r0 = 0; r0 < 32; r0 += kRowsPerPass) {
    const int rr = r0 + lane / kChunks, cch = lane % kChunks;
    const int out_row = wrow0 + rr;
    if (out_row < rows) {
      // (non-temporal: the output is written once and not read by this kernel)
      const uint4 v = *reinterpret_cast<const uint4*>(so + rr * D + ((cch ^ Swz::k(rr)) << 3));
      __builtin_nontemporal_store(u32x4_t{v.x, v.y, v.z, v.w},
                                  reinterpret_cast<u32x4_t*>(out + (((int64_t)b * a.q_len + out_row) * hq + h) * D + cch * 8));
    }
  }
}

// bf16 prefill from the paged cache.  Pipeline over three tile buffers (each
// a 256-byte-aligned LDS array): at step t the block loads the block-table
// entries of tile t+3 (scalar loads) and the K/V rows of tile t+2 (direct
// loads into the buffer tile t-1 used), computes tile t, then waits until
// tile t+1 has landed in every wave's part and joins the block, so every
// tile's loads have two steps to arrive.  The queries are loaded once, first
// of all (their rows do not depend on the span lengths), so they travel
// during the span and block-table round trips.
template <int D, int G, bool kRuns>
__global__ __launch_bounds__(PrefillShape<G>::kThreads, 3) void prefill_kernel_lds(PrefillArgs a) {
  typedef bf16_bits T;
  typedef Mfma<T> M;
  typedef M::Frag Frag;
  typedef LdsSwz<D> Swz;
  constexpr int kWaves = PrefillShape<G>::kWaves;
  constexpr int kRows = PrefillShape<G>::kRows;
  constexpr int kKeys = 32;                        // keys per tile
  constexpr int kQChunks = D / 16;
  constexpr int kChunks = Swz::kChunks;
  constexpr int kRowsPerLoad = 64 / kChunks;       // rows one wave-wide direct load fills
  constexpr int kLoads = kKeys / kRowsPerLoad;     // direct loads per tile and matrix
  constexpr int kLoadsPerWave = kLoads >= kWaves ? kLoads / kWaves : 1;
  static_assert(kLoads % kWaves == 0 || kWaves % kLoads == 0, "loads must split evenly over waves");
  constexpr int kVm = 2 * kLoadsPerWave;           // direct loads per tile of a loading wave
  constexpr int kTile = kKeys * D;                 // elements of one tile

  __shared__ __attribute__((aligned(256))) T s_k0[kTile];
  __shared__ __attribute__((aligned(256))) T s_k1[kTile];
  __shared__ __attribute__((aligned(256))) T s_k2[kTile];
  __shared__ __attribute__((aligned(256))) T s_v0[kTile];
  __shared__ __attribute__((aligned(256))) T s_v1[kTile];
  __shared__ __attribute__((aligned(256))) T s_v2[kTile];

  // XCD-aware, heaviest-first item order
  int pair, tile;
  query_tile_item(blockIdx.x, gridDim.x, a.num_tiles, pair, tile);
  const int heads = a.pv.kv_heads;
  const int g = pair % heads;
  const int b = pair / heads;

  const int p0 = tile * kRows;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = g * G + wave % G;
  const int col = lane & 31, hg = lane >> 5;
  const int wrow0 = p0 + (wave / G) * 32;  // first row of this wave
  const int p = wrow0 + col;
  const int hq = a.num_q_heads;
  // the queries: their rows do not depend on the span lengths, so with one
  // run they go first and are in flight during the span and block-table
  // round trips (a row past the tensor reads its last row: in range, never
  // stored).  A segment table is scanned with loads the compiler tracks, and
  // its waits would take these untracked loads along: there they follow the
  // scans, behind tile 0.
  Frag qf[kQChunks];
  auto load_queries = [&](int row) __attribute__((always_inline)) {
    const T* qrow = static_cast<const T*>(a.q) + (((int64_t)b * a.q_len + row) * hq + h) * D + hg * 8;
    static_for<kQChunks>([&](auto kc) { untracked_load16<decltype(kc)::value * 16 * 2>(qf[decltype(kc)::value], qrow); });
    __builtin_amdgcn_sched_barrier(0);
  };
  if constexpr (!kRuns) load_queries(min(p, a.q_len - 1));

  const auto sp = span_view<kRuns>(a, b, a.w_eff);
  const int rows = min(sp.rows(), a.q_len);
  const int clen = min(sp.clen(), a.pv.max_pages << a.pv.page_shift);
  if (p0 >= rows) {
    // the query loads land before the wave ends (with one run they were
    // issued above; an asm statement ahead of a segment scan would turn its
    // scalar loads into vector loads)
    if constexpr (!kRuns) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    return;
  }
  const int kmax = min(sp.visible(min(p0 + kRows, rows) - 1, a.mask_mode), clen);
  const int kclamp = max(kmax - 1, 0);  // last visible key: the row loaded for keys past kmax

  const bool qvalid = p < rows;
  const int nvis = qvalid ? min(sp.visible(p, a.mask_mode), clen) : 0;
  // keys every valid row of the wave sees (n_vis grows with the row)
  const int nvis_lo = wrow0 < rows ? min(sp.visible(wrow0, a.mask_mode), clen) : 0;
  const int slot_mask = (1 << a.pv.page_shift) - 1;
  const int shift = a.pv.page_shift;
  const int64_t num_pages = a.pv.num_pages;
  const int32_t* table_row = a.table + (int64_t)b * a.pv.max_pages;
  const T* kpool = static_cast<const T*>(a.k_pages);
  const T* vpool = static_cast<const T*>(a.v_pages);
  const int ntiles = (kmax + kKeys - 1) / kKeys;
  // this wave's direct loads: load i fills rows [row0(i), +kRowsPerLoad) of a tile
  const bool loads = kLoads >= kWaves || wave < kLoads;
  auto load_row0 = [&](int i) { return (kLoads >= kWaves ? wave * kLoadsPerWave + i : wave) * kRowsPerLoad; };
  const int lrow = lane / kChunks, lpos = lane % kChunks;  // row within the load, LDS chunk position

  f32x16_t o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
  float m_run = neg_inf(), l_run = 0.f;

  // A wave's direct loads of a tile fill kWaveRows <= 8 consecutive keys,
  // aligned to that count, and pages hold at least 8: its keys (each clamped
  // to kclamp) all lie in the page of min(first key, kclamp), so the wave
  // needs one block-table entry per tile, a wave-uniform index.  The entry is
  // read through the constant address space, a scalar load (no kernel writes
  // the table while this one runs), and the page bases are scalar.
  constexpr int kWaveRows = kLoadsPerWave * kRowsPerLoad;
  static_assert(kWaveRows <= 8, "one page holds a wave's rows of a tile");
  const int wrow_load = loads ? load_row0(0) : 0;
  typedef __attribute__((address_space(4))) const int32_t* const_ptr;
  auto table_load = [&](int kt) __attribute__((always_inline)) {
    const int row0 = min(kt * kKeys + wrow_load, kclamp);
    return ((const_ptr)table_row)[min(row0 >> shift, a.pv.max_pages - 1)];
  };
  // byte addresses: page p of KV head g starts at pool + p * page_bytes +
  // g * head_bytes; the V pool is the K pool plus a fixed distance
  const uint64_t head_bytes = (uint64_t)D * sizeof(T) << shift;
  const uint64_t page_bytes = head_bytes * heads;
  const uintptr_t kpool_g = (uintptr_t)kpool + (uint64_t)g * head_bytes;
  const uintptr_t v_minus_k = (uintptr_t)vpool - (uintptr_t)kpool;
  const uint32_t npages = (uint32_t)num_pages;
  auto tile_load = [&](int kt, int e, T* sk, T* sv) __attribute__((always_inline)) {
    if (!loads) return;
    const uint32_t page = (uint32_t)e < npages ? (uint32_t)e : 0u;  // a bad entry reads an in-range page
    const uintptr_t kbase = kpool_g + (uint64_t)page * page_bytes;  // uniform
    const uintptr_t vbase = kbase + v_minus_k;
#pragma unroll
    for (int i = 0; i < kLoadsPerWave; ++i) {
      const int row = load_row0(i) + lrow;
      const int key = min(kt * kKeys + row, kclamp);
      const uint32_t in_page = (uint32_t)((key & slot_mask) * D * 2);  // bytes
      lds_dma16((const void*)kbase, in_page + ((lpos ^ Swz::k(row)) << 4), lds_addr(sk + load_row0(i) * D));
      lds_dma16((const void*)vbase, in_page + ((lpos ^ Swz::v(row)) << 4), lds_addr(sv + load_row0(i) * D));
    }
  };

  // prologue (the queries are already in flight): tables of tiles 0..2,
  // tile 0, tile 1; then wait for the queries and tile 0 (tile 1 may stay in
  // flight)
  int pg[3] = {table_load(0), table_load(1), table_load(2)};  // entries by tile mod 3
  tile_load(0, pg[0], s_k0, s_v0);  // (also for a block without tiles: in range, never read)
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (kRuns) load_queries(qvalid ? p : 0);  // behind tile 0, after every segment scan
  if (ntiles > 1 && loads) {
    tile_load(1, pg[1], s_k1, s_v1);
    bare_barrier<kVm>();
  } else {
    // (a wave that loads no tile rows has only its query loads in flight:
    // it waits for all of them)
    bare_barrier<0>();
  }
  // A row past the sequence read before the span lengths were known may hold
  // anything: zero it (its queries have landed), so that its scores are 0 and
  // never force the online softmax to rescale.
  if constexpr (!kRuns) {
    if (!qvalid) {
#pragma unroll
      for (int kc = 0; kc < kQChunks; ++kc) qf[kc] = Frag{};
    }
  }

  // step kt; kPar = kt mod 3 selects buffers and table registers at compile
  // time.  Tiles past the last one are neither loaded nor computed: the last
  // two steps wait for everything in flight instead.
  auto tile_step = [&](int kt, auto par) {
    constexpr int kPar = decltype(par)::value;
    constexpr int kNext2 = (kPar + 2) % 3;
    T* const sk = kPar == 0 ? s_k0 : kPar == 1 ? s_k1 : s_k2;
    T* const sv = kPar == 0 ? s_v0 : kPar == 1 ? s_v1 : s_v2;
    const bool more = kt + 2 < ntiles;  // uniform
    if (more) {
      tile_load(kt + 2, pg[kNext2], kNext2 == 0 ? s_k0 : kNext2 == 1 ? s_k1 : s_k2,
                kNext2 == 0 ? s_v0 : kNext2 == 1 ? s_v1 : s_v2);  // into the buffer tile kt-1 used
      if (kt + 3 < ntiles) pg[kPar] = table_load(kt + 3);
    }
    attend_tile<D>(sk, sv, qf, o, m_run, l_run, kt * kKeys, nvis, nvis_lo, lane, a.scale_log2);
    // tile kt+1 has landed in every wave's part once each wave has at most
    // the loads of tile kt+2 in flight; every wave is then done with buffer
    // kPar, which the next step refills
    if (more) bare_barrier<kVm>();
    else bare_barrier<0>();
  };
  // three steps per iteration so that buffers and registers are compile-time
  for (int kt = 0; kt < ntiles; kt += 3) {
    tile_step(kt, std::integral_constant<int, 0>());
    if (kt + 1 >= ntiles) break;
    tile_step(kt + 1, std::integral_constant<int, 1>());
    if (kt + 2 >= ntiles) break;
    tile_step(kt + 2, std::integral_constant<int, 2>());
  }

  // output: one 32 x D tile per wave through the tile buffers, idle since the
  // last step's barrier (or the prologue's, without tiles) left no load in
  // flight and no wave reading them
  T* so = wave == 0 ? s_k0 : wave == 1 ? s_k1 : wave == 2 ? s_k2 : wave == 3 ? s_v0 : wave == 4 ? s_v1 : s_v2;
  finish_rows<D>(o, m_run, l_run, kWaves <= 6 ? so : nullptr, a, b, h, wrow0, rows, lane);
}

// Block shape of the pooling variant: eight waves whatever the group size, so
// a block owns 256/G query rows.  Every block pools each key tile it reads,
// so taller blocks pool each tile fewer times over the whole grid, and eight
// waves share the work of a tile (one pass of D/8-lane units at D = 128).
template <int G>
struct FusedShape {
  static constexpr int kRowBlocks = 8 / G;
  static constexpr int kWaves = 8;
  static constexpr int kThreads = 512;
  static constexpr int kRows = 32 * kRowBlocks;
};

// bf16 prefill that reads the raw K/V and pools each key tile on the fly
// (Sec. III-C) with the pooling kernel's steps (pool_window.hpp), D/8 lanes
// per (slot, head) unit: the first four frames of every window of tile t+1
// are loaded before the MFMAs of tile t and pooled after them, straight into
// the other of two LDS buffers in the layout the direct loads give.  The
// block holding a sequence's last query rows (which see every key) also
// stores each pooled row into the paged cache, and pools the rows no query
// sees, so the cache ends up as the pooling kernel would have written it.
// Two waves per SIMD: the first frames of the next tile's windows are held
// in registers across a step.
template <int D, int G>
__global__ __launch_bounds__(FusedShape<G>::kThreads, 2) void prefill_kernel_fused(PrefillFusedArgs args) {
  const PrefillArgs& a = args.at;
  typedef bf16_bits T;
  typedef Mfma<T> M;
  typedef M::Frag Frag;
  typedef LdsSwz<D> Swz;
  constexpr int kWaves = FusedShape<G>::kWaves;
  constexpr int kRows = FusedShape<G>::kRows;
  constexpr int kKeys = 32;                        // keys per tile
  constexpr int kQChunks = D / 16;
  constexpr int kTile = kKeys * D;                 // elements of one tile

  __shared__ __attribute__((aligned(256))) T s_k0[kTile];
  __shared__ __attribute__((aligned(256))) T s_k1[kTile];
  __shared__ __attribute__((aligned(256))) T s_v0[kTile];
  __shared__ __attribute__((aligned(256))) T s_v1[kTile];

  // XCD-aware, heaviest-first item order
  int pair, tile;
  query_tile_item(blockIdx.x, gridDim.x, a.num_tiles, pair, tile);
  const int heads = a.pv.kv_heads;
  const int g = pair % heads;
  const int b = pair / heads;

  const int w = a.w_eff;
  const auto sp = span_view<false>(a, b, w);
  const int rows = min(sp.rows(), a.q_len);
  const int clen = min(sp.clen(), a.pv.max_pages << a.pv.page_shift);
  const int p0 = tile * kRows;
  if (tile == 0 && g == 0 && threadIdx.x == 0 && args.cache_len_out) args.cache_len_out[b] = sp.clen();
  if (p0 >= rows) return;
  const int kmax = min(sp.visible(min(p0 + kRows, rows) - 1, a.mask_mode), clen);
  const int kclamp = max(kmax - 1, 0);  // last visible key: the row pooled for keys past kmax

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = g * G + wave % G;
  const int col = lane & 31, hg = lane >> 5;
  const int wrow0 = p0 + (wave / G) * 32;  // first row of this wave
  const int p = wrow0 + col;
  const bool qvalid = p < rows;
  const int nvis = qvalid ? min(sp.visible(p, a.mask_mode), clen) : 0;
  const int nvis_lo = wrow0 < rows ? min(sp.visible(wrow0, a.mask_mode), clen) : 0;
  const int hq = a.num_q_heads;
  const int slot_mask = (1 << a.pv.page_shift) - 1;
  const int shift = a.pv.page_shift;
  const int64_t num_pages = a.pv.num_pages;
  const int32_t* table_row = a.table + (int64_t)b * a.pv.max_pages;
  const int ntiles = (kmax + kKeys - 1) / kKeys;

  // on-the-fly pooling: D/8 lanes per (slot, head) unit, one unit per key of
  // the tile; the first kPoolWaves waves pool, lane pj-th chunk of unit
  // pslot.  The first four frames of each unit's window are staged by direct
  // loads into this wave's own LDS area (lane i's 16 bytes of frame t at K:
  // 2t KB + 16 i, V: 2t+1 KB + 16 i), so they cost no registers across the
  // MFMAs and each lane reads back only what it loaded.
  constexpr int kLanes = D / 8;
  constexpr int kPoolWaves = kKeys / (64 / kLanes);
  static_assert(kPoolWaves <= kWaves, "one pass of the pooling waves covers a tile");
  const int pj = lane % kLanes;
  const int pslot = wave * (64 / kLanes) + lane / kLanes;
  const bool pool_wave = wave < kPoolWaves;  // uniform over the wave
  const bool writer = p0 + kRows >= rows;   // holds the last rows: sees every key
  int fsrc = 0, ffr = 1, fent = 0;          // the unit's first raw row, frames, page
  float u[8];
  __shared__ __attribute__((aligned(16))) T s_stage[kPoolWaves * 8 * 512];
  T* const stage = s_stage + (pool_wave ? wave : 0) * 8 * 512;
  const T* kr = static_cast<const T*>(args.k_raw) + b * args.stride_b + g * args.stride_h + 8 * pj;
  const T* vr = static_cast<const T*>(args.v_raw) + b * args.stride_b + g * args.stride_h + 8 * pj;
  const int64_t raw_stride = args.stride_s;
  const int raw_last = args.raw_len - 1;
  if (args.gate) {  // without a gate every logit is 0 (uniform averaging)
    const float4* gp = reinterpret_cast<const float4*>(args.gate + (int64_t)g * D + 8 * pj);
    const float4 u0 = gp[0], u1 = gp[1];
    u[0] = u0.x; u[1] = u0.y; u[2] = u0.z; u[3] = u0.w;
    u[4] = u1.x; u[5] = u1.y; u[6] = u1.z; u[7] = u1.w;
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) u[i] = 0.f;
  }
  auto raw_at = [&](int s) __attribute__((always_inline)) { return (int64_t)min(s, raw_last) * raw_stride; };
  // stage the first four frames of unit (slot min(c0 + pslot, cmax), this
  // head); frames past a window repeat its last one; w = 1 needs one frame
  auto pool_fetch = [&](int c0, int cmax) __attribute__((always_inline)) {
    if (!pool_wave) return;
    const int c = min(c0 + pslot, cmax);
    const SlotSource sl = sp.slot(c);
    fsrc = sl.first;
    ffr = sl.frames;
    fent = writer ? table_row[min(c >> shift, a.pv.max_pages - 1)] : 0;
    const int nt = w == 1 ? 1 : 4;  // uniform
    for (int t = 0; t < nt; ++t) {
      const int64_t o = raw_at(sl.first + min(t, sl.frames - 1));
      __builtin_amdgcn_global_load_lds((global_void_ptr)(kr + o), (lds_void_ptr)(stage + 2 * t * 512), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((global_void_ptr)(vr + o), (lds_void_ptr)(stage + (2 * t + 1) * 512), 16, 0, 0);
    }
  };
  // the unit's pooled rows from the staged frames (and the later frames of
  // windows longer than four); a text row or one-frame window is its raw row
  auto pool_rows = [&](Chunk<T>& ko, Chunk<T>& vo) __attribute__((always_inline)) {
    // the wave's own direct loads must have landed before it reads them back:
    // the compiler does not order LDS-DMA writes against later LDS reads, so
    // wait explicitly, fenced on both sides for the optimiser and scheduler
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    Chunk<T> kc[4], vc[4];
    const int nt = w == 1 ? 1 : 4;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (t < nt) {
        kc[t].raw = *reinterpret_cast<const uint4*>(stage + 2 * t * 512 + 8 * lane);
        vc[t].raw = *reinterpret_cast<const uint4*>(stage + (2 * t + 1) * 512 + 8 * lane);
      }
    }
    ko = kc[0];
    vo = vc[0];
    if (w > 1) {
      WindowPool<T, kLanes> wp;
      wp.init();
      wp.template add4<true>(kc, vc, u, 0, ffr);
      for (int f0 = 4; f0 < ffr; f0 += 4) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int64_t o = raw_at(fsrc + min(f0 + t, ffr - 1));
          kc[t].load(kr + o);
          vc[t].load(vr + o);
        }
        wp.template add4<true>(kc, vc, u, f0, ffr);
      }
      Chunk<T> pk, pv;
      wp.finish(pk, pv);
      if (ffr > 1) {
        ko = pk;
        vo = pv;
      }
    }
  };
  // cache row c of this head, when it exists, has a valid page and its
  // source rows lie inside the raw tensor (as the pooling kernel checks)
  auto cache_store = [&](int c, const Chunk<T>& ko, const Chunk<T>& vo) __attribute__((always_inline)) {
    if (c < clen && fent >= 0 && fent < num_pages && fsrc + ffr <= raw_last + 1) {
      const int64_t off = page_row<D>(fent, g, c & slot_mask, a.pv) + 8 * pj;
      ko.store(static_cast<T*>(args.k_pages) + off);
      vo.store(static_cast<T*>(args.v_pages) + off);
    }
  };
  // pool key tile kt into LDS; the writer also stores its visible rows
  auto pool_tile = [&](int kt, T* sk, T* sv) __attribute__((always_inline)) {
    if (!pool_wave) return;
    Chunk<T> ko, vo;
    pool_rows(ko, vo);
    const int r = pslot;
    ko.store(sk + r * D + ((pj ^ Swz::k(r)) << 3));
    vo.store(sv + r * D + ((pj ^ Swz::v(r)) << 3));
    if (writer && kt * kKeys + r < kmax) cache_store(kt * kKeys + r, ko, vo);
  };

  f32x16_t o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
  float m_run = neg_inf(), l_run = 0.f;

  // prologue: stage tile 0's frames, load this lane's query row (rows past
  // the end read row 0: finite, never stored), pool tile 0
  if (ntiles > 0) pool_fetch(0, kclamp);
  __builtin_amdgcn_sched_barrier(0);
  Frag qf[kQChunks];
  {
    const T* qrow = static_cast<const T*>(a.q) + (((int64_t)b * a.q_len + (qvalid ? p : 0)) * hq + h) * D;
#pragma unroll
    for (int kc = 0; kc < kQChunks; ++kc) qf[kc] = M::load(qrow + kc * 16 + hg * 8);
  }
  if (ntiles > 0) pool_tile(0, s_k0, s_v0);
  __syncthreads();

  // step kt: stage the frames of tile kt+1, attend to tile kt, pool tile kt+1
  // into the other buffer; kPar = kt & 1 selects buffers at compile time
  auto tile_step = [&](int kt, auto par) {
    constexpr int kPar = decltype(par)::value;
    T* const sk = kPar ? s_k1 : s_k0;
    T* const sv = kPar ? s_v1 : s_v0;
    const bool pool_next = kt + 1 < ntiles;  // uniform
    if (pool_next) pool_fetch((kt + 1) * kKeys, kclamp);  // pooled after this tile's MFMAs
    if (kt < ntiles) attend_tile<D>(sk, sv, qf, o, m_run, l_run, kt * kKeys, nvis, nvis_lo, lane, a.scale_log2);
    if (pool_next) pool_tile(kt + 1, kPar ? s_k0 : s_k1, kPar ? s_v0 : s_v1);
    __syncthreads();
  };
  for (int kt = 0; kt < ntiles; kt += 2) {
    tile_step(kt, std::integral_constant<int, 0>());
    tile_step(kt + 1, std::integral_constant<int, 1>());
  }
  // cache rows no query of this sequence sees: pooled and stored by the writer
  if (writer) {
    for (int c0 = kmax; c0 < clen; c0 += kKeys) {
      pool_fetch(c0, clen - 1);
      if (pool_wave) {
        Chunk<T> ko, vo;
        pool_rows(ko, vo);
        cache_store(c0 + pslot, ko, vo);
      }
    }
  }
  static_assert(kWaves > 4, "eight waves store their rows from the C layout");
  finish_rows<D>(o, m_run, l_run, nullptr, a, b, h, wrow0, rows, lane);
}

template <typename T, int D, bool kRuns>
hipError_t launch_prefill_d(const PrefillArgs& a, int group, int batch, hipStream_t s) {
  const unsigned items = (unsigned)(batch * a.pv.kv_heads * a.num_tiles);
  switch (group) {
    case 1: return launch_struct(prefill_kernel<T, D, 1, kRuns>, dim3(items), dim3(PrefillShape<1>::kThreads), s, a);
    case 2: return launch_struct(prefill_kernel<T, D, 2, kRuns>, dim3(items), dim3(PrefillShape<2>::kThreads), s, a);
    case 4: return launch_struct(prefill_kernel<T, D, 4, kRuns>, dim3(items), dim3(PrefillShape<4>::kThreads), s, a);
    default: return launch_struct(prefill_kernel<T, D, 8, kRuns>, dim3(items), dim3(PrefillShape<8>::kThreads), s, a);
  }
}

template <int D, bool kRuns>
hipError_t launch_prefill_lds(const PrefillArgs& a, int group, int batch, hipStream_t s) {
  const unsigned items = (unsigned)(batch * a.pv.kv_heads * a.num_tiles);
  switch (group) {
    case 1: return launch_struct(prefill_kernel_lds<D, 1, kRuns>, dim3(items), dim3(PrefillShape<1>::kThreads), s, a);
    case 2: return launch_struct(prefill_kernel_lds<D, 2, kRuns>, dim3(items), dim3(PrefillShape<2>::kThreads), s, a);
    case 4: return launch_struct(prefill_kernel_lds<D, 4, kRuns>, dim3(items), dim3(PrefillShape<4>::kThreads), s, a);
    default: return launch_struct(prefill_kernel_lds<D, 8, kRuns>, dim3(items), dim3(PrefillShape<8>::kThreads), s, a);
  }
}

template <int D>
hipError_t launch_prefill_fused_d(const PrefillFusedArgs& args, int group, int batch, hipStream_t s) {
  const PrefillArgs& a = args.at;
  const unsigned items = (unsigned)(batch * a.pv.kv_heads * a.num_tiles);
  switch (group) {
    case 1: return launch_struct(prefill_kernel_fused<D, 1>, dim3(items), dim3(FusedShape<1>::kThreads), s, args);
    case 2: return launch_struct(prefill_kernel_fused<D, 2>, dim3(items), dim3(FusedShape<2>::kThreads), s, args);
    case 4: return launch_struct(prefill_kernel_fused<D, 4>, dim3(items), dim3(FusedShape<4>::kThreads), s, args);
    default: return launch_struct(prefill_kernel_fused<D, 8>, dim3(items), dim3(FusedShape<8>::kThreads), s, args);
  }
}

}  // namespace

int prefill_rows_per_tile(int group) {
  switch (group) {
    case 1: return PrefillShape<1>::kRows;
    case 2: return PrefillShape<2>::kRows;
    case 4: return PrefillShape<4>::kRows;
    default: return PrefillShape<8>::kRows;
  }
}

hipError_t launch_prefill(const PrefillArgs& a, int dtype, int head_dim, int group, int batch,
                          hipStream_t s) {
  const bool runs = a.segs.seg_start != nullptr;
  if (dtype == 1) {
    if (head_dim == 128)
      return runs ? launch_prefill_lds<128, true>(a, group, batch, s)
                  : launch_prefill_lds<128, false>(a, group, batch, s);
    return runs ? launch_prefill_lds<64, true>(a, group, batch, s)
                : launch_prefill_lds<64, false>(a, group, batch, s);
  }
  if (head_dim == 128)
    return runs ? launch_prefill_d<float, 128, true>(a, group, batch, s)
                : launch_prefill_d<float, 128, false>(a, group, batch, s);
  return runs ? launch_prefill_d<float, 64, true>(a, group, batch, s)
              : launch_prefill_d<float, 64, false>(a, group, batch, s);
}

int prefill_fused_rows_per_tile(int group) {
  switch (group) {
    case 1: return FusedShape<1>::kRows;
    case 2: return FusedShape<2>::kRows;
    case 4: return FusedShape<4>::kRows;
    default: return FusedShape<8>::kRows;
  }
}

hipError_t launch_prefill_fused(const PrefillFusedArgs& a, int head_dim, int group, int batch,
                                hipStream_t s) {
  if (head_dim == 128) return launch_prefill_fused_d<128>(a, group, batch, s);
  return launch_prefill_fused_d<64>(a, group, batch, s);
}

}  // namespace skv
