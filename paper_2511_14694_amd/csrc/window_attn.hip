// Window attention over [retained summary cache ; window] (focus_window_attn).
//
// C(t) mask: for window w of sequence b, query row i (0 <= i < T_w) of head h
// attends to every cache row j < C_w and to window rows u <= i: the visibility
// set C(t) of Appendix A.1, which is also the mask of the masked-parallel form
// (A.1, "Cross-window consistency").  One launch may cover any set of windows
// of any sequences; each window only reads the cache rows its predecessors
// retained.
//
// k-mer-local mask (Section 3.2, "Visibility and summarization rule"): query
// row i sees the earlier-or-equal rows of its own k-mer, the earlier summaries
// of its window and the carried boundary (cache row C_w - 1).  The keys are
// visited as a gathered summary list [boundary ; the window's summaries] and
// then only the window tiles that hold the block's k-mers; a two-sided mask
// keeps each row's own k-mer.
//
// bf16 path under C(t) (the hot one, attn_ct): one workgroup = 8 waves x 32
// query rows of one (window, head), two waves per SIMD; keys arrive in 64-key
// tiles copied global -> LDS directly through four LDS stages, and each wave
// runs a one-sub-tile (32 keys) software pipeline:
//   S^T = K Q^T   v_mfma_f32_32x32x16_bf16: each lane ends up holding one
//                 query's scores for 16 keys of a 32-key block, so the row
//                 max / row sum are lane-local plus one exchange with lane^32;
//                 the next sub-tile's scores are issued on the MFMA pipe while
//                 the VALU does this sub-tile's softmax;
//   softmax       exp2 domain, running max with lazy rescaling: the output
//                 accumulator is rescaled only when a row's max grows by more
//                 than 2^8, which keeps exp2 arguments <= 8 and is exact;
//   O^T += V^T P^T  the same MFMA; P comes straight from the S^T accumulator
//                 (rounded to bf16), V^T is read from LDS with the gfx950
//                 transposing read ds_read_b64_tr_b16.
// The cache's tiles start 64 ceil(C_w / 64) - C_w rows before cache row 0, so
// its one partial tile is the first key tile and every tile from there to the
// block's diagonal is full and unmasked: those steps run a branch-free body.
// Both LDS tiles are XOR-swizzled so that the MFMA operand reads are free of
// bank conflicts.  Blocks are dealt out so that all query tiles of one
// (window, head) land on the same XCD (sharing K/V through its L2) and the
// listed windows are started in list order (last window = largest cache first
// by default).
//
// The k-mer-local mask (attn_kl) uses the same MFMA scheme without the
// software pipeline: one workgroup of 4 waves streams all query tiles of a
// (window, head), each wave copying its share of 32-key tiles through five
// LDS stages.
//
// Summary queries (the FOCUS adapter's attention): under C(t) several windows'
// summaries share one workgroup (attn_sq_block); otherwise the bf16 kernel
// above runs with one wave of 32 summary slots per (window, head).
//
// f32 path: a plain VALU kernel (4 lanes per query row, exact online softmax),
// used for the float32 checks; it is not tuned.
#include "common.h"

#include <math.h>

namespace {

using focus::bf16x4;
using focus::bf16x8;
using focus::f32x16;
using focus::u32x4;

constexpr float kLn2 = 0.69314718055994531f;
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kMinit = -1.0e30f;  // finite start of the running max (no inf - inf)
constexpr float kLazy = 8.0f;       // rescale when the max grows by > 2^8

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) void lds_void;

// Waves per workgroup of the bf16 kernels (each wave owns 32 query rows):
// eight under C(t), where a workgroup streams thousands of keys; four under the
// k-mer-local mask (attn_kl), where a query tile visits a handful of key tiles.
constexpr int kBf16Waves = 8;
constexpr int kBf16WavesKL = 4;
// attn_kl at head_dim 128: waves per workgroup and LDS stages (8 waves and 8
// stages, one workgroup per CU: 8.41 vs 7.86 ms at 1 Mb)
constexpr int kKlWaves128 = 4, kKlStages128 = 4;

struct Item {
  int64_t list_idx;
  int h;
  int qt;
  bool valid;
};

// Block -> (listed window, head, query tile).  Blocks go round robin over the
// XCDs.  When H is a multiple of the XCD count, XCD x owns heads x, x + 8, ...
// and walks them one at a time, each over all listed windows in list order:
// the workgroups that run together on an XCD then stream the same cache rows
// of one head at about the same time, so each row is fetched into its L2 once
// for all of them.  Otherwise pair p = list_idx * H + h goes to XCD p % 8, in
// increasing p.  The QT query tiles of a pair go last-first (under the causal
// window mask the last tile sees the most keys, and starting the longest
// workgroups first shortens the tail of a launch).
//
// Two orders of an XCD's blocks (H a multiple of 8):
// * ROUNDS = false: a pair's query tiles are consecutive blocks (they share
//   the window's K/V through the XCD's L2 while they run together);
// * ROUNDS = true: kRound consecutive blocks (one per compute unit of the XCD)
//   are one query tile of kRound pairs, the next kRound the next query tile of
//   the same pairs.  The hardware hands an XCD's blocks to its compute units in
//   a fixed rotation, so with the first order each compute unit always gets
//   the same query tile, and the ones with short tiles wait every round for
//   the ones with long tiles (per-workgroup timestamps: ~12 us idle per
//   workgroup at 1 Mb).  With one tile per round the workgroups of a round
//   last about equally long.  It pays where the arithmetic dominates (the C(t)
//   attention: 1 Mb 88.6 -> 86.7 ms, 100 kb 2.70 -> 2.58 ms); the HBM-bound
//   k-mer-local launch loses more from the scattered K/V reuse (9.6 -> 10.5 ms)
//   and keeps the first order.
constexpr int64_t kRound = 32;  // compute units per XCD on MI355X (256 / 8)
template <bool ROUNDS = false>
__device__ inline Item map_block(int64_t bid, int64_t n_pairs, int H, int QT) {
  const int x = (int)(bid % focus::kXcds);
  const int64_t s = bid / focus::kXcds;
  Item it;
  it.qt = QT - 1 - (int)(s % QT);
  int64_t j = s / QT;  // this XCD's j-th pair
  if (H % focus::kXcds == 0) {
    bool in_range = true;
    if (ROUNDS) {
      const int64_t npx = n_pairs / focus::kXcds;  // pairs of this XCD
      const int64_t c = s / (kRound * QT), r = s % (kRound * QT);
      const int64_t m = min(kRound, npx - c * kRound);  // pairs in this group of rounds
      in_range = m > 0 && r < m * QT;
      j = c * kRound + (in_range ? r % m : 0);
      it.qt = QT - 1 - (in_range ? (int)(r / m) : 0);
    }
    const int64_t nwl = n_pairs / H;  // listed windows
    const int64_t hl = nwl > 0 ? j / nwl : 0;
    it.valid = in_range && nwl > 0 && hl < H / focus::kXcds;
    it.list_idx = nwl > 0 ? j % nwl : 0;
    it.h = (int)(hl * focus::kXcds + x);
  } else {
    const int64_t p = j * focus::kXcds + x;
    it.valid = p < n_pairs;
    it.list_idx = p / H;
    it.h = (int)(p % H);
  }
  return it;
}

__device__ inline int64_t listed_window(const focus_attn_desc& d, int64_t li) {
  return d.win_ids ? (int64_t)d.win_ids[li] : d.totals.n_windows - 1 - li;
}

// ------------------------------------------------------------------ bf16 MFMA

template <int D, int W, int BK = 64>
struct Cfg {
  static constexpr int kWaves = W;                        // 32 query rows per wave
  static constexpr int kBQ = 32 * W;                      // query rows per block
  static constexpr int kBK = BK;                          // keys per tile
  static constexpr int kSt = BK / 32;                     // 32-key MFMA blocks per tile
  static constexpr int kThreads = 64 * W;
  static constexpr int kRB = D * 2;                       // bytes per row
  static constexpr int kTile = kBK * kRB;                 // bytes per tile per tensor
  static constexpr int kCh16 = kRB / 16;                  // 16-byte chunks per row
  static constexpr int kLoads = kBK * kCh16 / kThreads;   // chunks per thread per tensor
  static constexpr int kKsteps = D / 16;                  // MFMA k-steps of QK^T
  static constexpr int kDtiles = D / 32;                  // 32-row blocks of O^T
};

// K tile: 16-byte chunk c of row r sits at chunk c ^ (r mod chunks-per-row).
template <int D>
__device__ inline int k_off(int r, int c16) {
  constexpr int kRB = D * 2, kCh16 = kRB / 16;
  return r * kRB + ((c16 ^ (r % kCh16)) << 4);
}
// V tile: 64-byte granule g of row r sits at granule g ^ f(r), with f chosen
// so that the four rows one transposing read touches per half-wave fall into
// four different 64-byte bank groups.
template <int D>
__device__ inline int v_off(int r, int byte) {
  const int f = D == 128 ? (r & 3) : ((r >> 1) & 1);
  return r * (D * 2) + ((((byte >> 6) ^ f)) << 6) + (byte & 63);
}

// Summary-query mode (the FOCUS adapter attention of eq. focus-attn): the
// queries of a window are its summary tokens only; query slot j is summary
// win_sum_off[w] + j at window row sum_tok[...] - win_tok_off[w], and q / o /
// lse rows are indexed by global summary index - base.
struct SumQ {
  const int32_t* win_nsum;
  const int64_t* win_sum_off;
  const int64_t* sum_tok;
  const void* q;
  void* o;
  float* lse;
  int64_t base, rows;
};

// Key split (C(t), bf16): when a launch has fewer workgroups than the device
// has compute units (one window per call), each (window, head, query tile)
// item is split into n workgroups over consecutive ranges of its key tiles.
// Each writes its rows' unnormalised float32 output and (running max, sum) in
// the exp2 domain to the workspace, [split][listed window][row][head][D] and
// [split][listed window][row][head][2]; attn_combine merges them.
struct Split {
  int n;        // 1 = no split
  float* po;    // partial outputs
  float* pml;   // (max, sum) pairs
  int64_t rows; // rows per listed window in the workspace (max window tokens)
  int64_t nwl;  // listed windows
};
constexpr Split kNoSplit = {1, nullptr, nullptr, 0, 0};

// Summary queries (the FOCUS adapter's attention) under C(t) (KL false) or
// the k-mer-local mask (KL true), where attn_sq_block does not apply: W waves
// of 32 summary slots per (window, head), 64-key tiles through two LDS stages.
// (The window attention itself is attn_ct under C(t) and attn_kl under the
// k-mer-local mask.)
template <int D, int W, bool KL, bool SQ>
__global__ __launch_bounds__(64 * W, W == 1 ? 1 : 2) void attn_bf16(focus_attn_desc d, float sc, int64_t n_pairs,
                                                                     int QT, SumQ sq) {
  static_assert(SQ, "the window attention is attn_ct (C(t)) or attn_kl (k-mer-local)");
  using C = Cfg<D, W, 64>;
  // K and V tile buffers as separate arrays, referenced statically by a loop
  // unrolled by the stage count: the compiler can then tell a tile being read
  // from the ones being filled, and waits for the copies only where it must.
  __shared__ __attribute__((aligned(1024))) char kbuf0[C::kTile], kbuf1[C::kTile];
  __shared__ __attribute__((aligned(1024))) char vbuf0[C::kTile], vbuf1[C::kTile];

  const int tid = threadIdx.x;
  const Item it = map_block(blockIdx.x, n_pairs, d.n_heads, QT);
  if (!it.valid) return;
  const int64_t gw = listed_window(d, it.list_idx);
  if (gw < 0 || gw >= d.totals.n_windows) {
    if (tid == 0 && it.qt == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
    return;
  }
  const int T = d.win_ntok[gw];
  const int q0 = it.qt * C::kBQ;
  const int nq = sq.win_nsum[gw];        // query slots of the window: its summaries
  const int64_t s0 = sq.win_sum_off[gw];  // the window's first summary
  if (q0 >= nq) return;
  const int Cw = d.win_cache_off[gw];
  const int b = d.win_seq[gw];
  const int64_t tok0 = d.win_tok_off[gw] - d.qkv_tok_base;
  if (b < 0 || b >= d.batch || Cw < 0 || Cw > d.cache_cap || tok0 < 0 || tok0 + T > d.qkv_rows || nq > T ||
      s0 < sq.base || s0 + nq > sq.base + sq.rows) {
    if (tid == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
    return;
  }
  // window row of query slot j (clamped to the last slot)
  auto qpos = [&](int j) -> int {
    j = min(j, nq - 1);
    const int64_t r = sq.sum_tok[s0 + j] - d.win_tok_off[gw];
    return (int)(r < 0 ? 0 : r >= T ? T - 1 : r);
  };
  const int H = d.n_heads, Hkv = d.n_kv_heads, h = it.h;
  const int hk = h / (H / Hkv);
  const int nwk = qpos(q0 + C::kBQ - 1) + 1;  // window keys any query of this tile can see
  // C(t): keys are visited as nct tiles of cache rows [0, Cw) followed by nwt
  // tiles of window rows [0, nwk); only the last tile of each phase is partial.
  // k-mer-local: the first nct tiles hold the summary list [carried boundary
  // (cache row Cw - 1) ; the window's nsum summaries], gathered row by row;
  // the window tiles start at tile tw0, the one holding the first row of the
  // k-mer of the block's first query.
  int kw = 0, nsum = 0, tw0 = 0;
  if constexpr (KL) {
    kw = d.win_kmer ? d.win_kmer[gw] : d.kmer_uniform;
    if (kw < 0) {
      if (tid == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
      return;
    }
    nsum = kw > 0 ? (T + kw) / (kw + 1) : 0;
    // first row of the k-mer of the tile's first query (summary j closes k-mer j)
    tw0 = kw > 0 ? q0 * (kw + 1) / C::kBK : 0;
  }
  const int nct = KL ? (nsum + C::kBK) / C::kBK : (Cw + C::kBK - 1) / C::kBK;
  const int nwt = (nwk + C::kBK - 1) / C::kBK - tw0;
  // This workgroup's tiles [tb, tb + ntiles) of the item's nct + nwt.
  const int ntiles = nct + nwt;

  const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
  const int js = q0 + wave * 32 + l32;  // this lane's query slot
  const int qi = qpos(js);              // and its row inside the window
  const int wq_lo = qpos(q0 + wave * 32), wq_hi = qpos(q0 + wave * 32 + 31);
  const bool wave_live = q0 + wave * 32 < nq;
  // k-mer-local: this lane's k-mer index jq inside the window and that
  // k-mer's first row qlo; klo_w: first row of the wave's first k-mer.
  int jq = 0, qlo = 0, klo_w = 0;
  if constexpr (KL) {
    if (kw > 0) {
      jq = min(js, nq - 1);
      qlo = jq * (kw + 1);
      klo_w = min(q0 + wave * 32, nq - 1) * (kw + 1);
    }
  }

  // Q^T as the B operand: lane holds query l32, head_dim [16s + 8g, 16s + 8g + 8).
  bf16x8 qf[C::kKsteps];
  {
    const int64_t qrow = s0 + min(js, nq - 1) - sq.base;
    const bf16x8* qp = reinterpret_cast<const bf16x8*>(reinterpret_cast<const __bf16*>(sq.q) + (qrow * H + h) * D);
#pragma unroll
    for (int s = 0; s < C::kKsteps; ++s) qf[s] = qp[2 * s + g];
  }

  // Tiles move global -> LDS directly (global_load_lds_dwordx4: one wave
  // instruction fills 1 KB of LDS, lane l its 16 bytes at offset 16 l), so no
  // registers or LDS writes are spent on staging.  Wave-load i of wave w fills
  // tile rows (w kDma + i) kRPK + lane / kCh16; the lane at 16-byte slot p of
  // a row fetches the global chunk the swizzled layout keeps there.  Tile base
  // pointers are uniform; per-lane parts are 32-bit byte offsets.  The last
  // tile of a phase clamps its rows to the last valid one (extra rows are
  // masked; the clamp keeps reads inside the buffers).
  constexpr int kRPK = 1024 / C::kRB;
  constexpr int kDma = C::kTile / 1024 / C::kWaves;
  static_assert(kDma >= 1 && C::kTile % (1024 * C::kWaves) == 0, "tile must split into 1 KB wave loads");
  const uint32_t row_bytes = (uint32_t)(Hkv * D * 2);
  uint32_t rowb[kDma], kchunk[kDma], vchunk[kDma];
#pragma unroll
  for (int i = 0; i < kDma; ++i) {
    const int r = (wave * kDma + i) * kRPK + lane / C::kCh16;
    const int p = lane % C::kCh16;
    const int f = D == 128 ? (r & 3) : ((r >> 1) & 1);
    rowb[i] = (uint32_t)r * row_bytes;
    kchunk[i] = (uint32_t)((p ^ (r % C::kCh16)) * 16);
    vchunk[i] = (uint32_t)((((p >> 2) ^ f) * 4 + (p & 3)) * 16);
  }
  const char* kwin = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(d.k) + (tok0 * Hkv + hk) * D);
  const char* vwin = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(d.v) + (tok0 * Hkv + hk) * D);
  const char* kcache = reinterpret_cast<const char*>(
      reinterpret_cast<const __bf16*>(d.cache_k) + ((int64_t)b * d.cache_cap * Hkv + hk) * D);
  const char* vcache = reinterpret_cast<const char*>(
      reinterpret_cast<const __bf16*>(d.cache_v) + ((int64_t)b * d.cache_cap * Hkv + hk) * D);

  // Tile x lives in buffers x & 1.
  auto issue_tile = [&](int t, char* kbuf, char* vbuf) {
    if constexpr (KL) {
      if (t < nct) {
        // Summary-list entry R = 64 t + r: R = 0 is the carried boundary, R >= 1
        // the window's summary R - 1 at window row R (k + 1) - 1 (the last one at
        // T - 1).  Rows past the list repeat its last entry (masked).
        char* kl = kbuf + wave * kDma * 1024;
        char* vl = vbuf + wave * kDma * 1024;
#pragma unroll
        for (int i = 0; i < kDma; ++i) {
          const int r = (wave * kDma + i) * kRPK + lane / C::kCh16;
          const int R = min(t * C::kBK + r, nsum);
          const bool boundary = R == 0 && Cw > 0;
          const int wrow = R == 0 ? 0 : min(R * (kw + 1) - 1, T - 1);
          const char* kp = boundary ? kcache + (int64_t)(Cw - 1) * row_bytes : kwin + (int64_t)wrow * row_bytes;
          const char* vp = boundary ? vcache + (int64_t)(Cw - 1) * row_bytes : vwin + (int64_t)wrow * row_bytes;
          const char* ks = kp + kchunk[i];
          const char* vs = vp + vchunk[i];
          __builtin_amdgcn_global_load_lds(ks, (lds_void*)(kl + i * 1024), 16, 0, 0);
          __builtin_amdgcn_global_load_lds(vs, (lds_void*)(vl + i * 1024), 16, 0, 0);
        }
        return;
      }
    }
    const bool in_cache = t < nct;
    const int row0 = in_cache ? t * C::kBK : (t - nct + tw0) * C::kBK;
    const int nvalid = (in_cache ? Cw : nwk) - row0;
    const char* kb = (in_cache ? kcache : kwin) + (int64_t)row0 * row_bytes;
    const char* vb = (in_cache ? vcache : vwin) + (int64_t)row0 * row_bytes;
    char* kl = kbuf + wave * kDma * 1024;
    char* vl = vbuf + wave * kDma * 1024;
    const uint32_t last = (uint32_t)(nvalid - 1) * row_bytes;
#pragma unroll
    for (int i = 0; i < kDma; ++i) {
      const uint32_t rb = nvalid >= C::kBK ? rowb[i] : min(rowb[i], last);
      const uint32_t ko = rb + kchunk[i], vo = rb + vchunk[i];
      __builtin_amdgcn_global_load_lds(kb + ko, (lds_void*)(kl + i * 1024), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(vb + vo, (lds_void*)(vl + i * 1024), 16, 0, 0);
    }
  };

  f32x16 oacc[C::kDtiles];
#pragma unroll
  for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[dt][v] = 0.f;
  float m_run = kMinit, l_run = 0.f;

  // transposing-read coordinates: lane = 16 * grp + 4 * ri + bq
  const int grp = lane >> 4, ri = (lane >> 2) & 3, bq = lane & 3;

  auto compute_tile = [&](int t, const char* kl, const char* vl) {
    // Key kk of the tile (0 .. kBK - 1) is visible to this lane's query iff kk <= lim:
    // cache tiles hide only rows past Cw, window tiles are causal.
    const bool in_cache = t < nct;  // (k-mer-local: the summary list)
    const int row0 = in_cache ? t * C::kBK : (t - nct + tw0) * C::kBK;
    const bool live = wave_live && (in_cache || (row0 <= wq_hi && (!KL || row0 + C::kBK > klo_w)));
    const bool need_mask = KL || (in_cache ? row0 + C::kBK > Cw : row0 + C::kBK - 1 > wq_lo);
    // visible tile keys: lo <= kk <= lim (lo only for k-mer-local)
    const int lim = KL ? (in_cache ? jq - row0 : qi - row0) : (in_cache ? Cw - row0 - 1 : qi - row0);
    const int lo = KL ? (in_cache ? (Cw > 0 ? 0 : 1) - row0 : qlo - row0) : 0;
    if (live) {
      // S^T = K Q^T: the tile's 32-key blocks as independent MFMA chains,
      // each K operand read one k-step ahead of its MFMA.
      f32x16 sacc[C::kSt];
#pragma unroll
      for (int st = 0; st < C::kSt; ++st)
#pragma unroll
        for (int v = 0; v < 16; ++v) sacc[st][v] = 0.f;
      // Per-lane LDS offsets are rebuilt each step behind an empty asm
      // statement: not hoisted out of the loop once per buffer (registers),
      // and one offset from the buffer, so the compiler still tells the
      // buffers apart.  K row 32 st + l32, chunk 2 s + g sits at chunk
      // (2 s + g) ^ (l32 mod kCh16) = 2 s ^ kx.
      const int kx = g ^ (l32 & (C::kCh16 - 1));
      auto kread = [&](int s, int st) {
        int ko = l32 * C::kRB + (((2 * s) ^ kx) << 4);
        asm volatile("" : "+v"(ko));
        return *reinterpret_cast<const bf16x8*>(kl + (ko + st * 32 * C::kRB));
      };
      bf16x8 ka[C::kSt], kn[C::kSt];
#pragma unroll
      for (int st = 0; st < C::kSt; ++st) ka[st] = kread(0, st);
#pragma unroll
      for (int s = 0; s < C::kKsteps; ++s) {
        if (s + 1 < C::kKsteps) {
#pragma unroll
          for (int st = 0; st < C::kSt; ++st) kn[st] = kread(s + 1, st);
        }
#pragma unroll
        for (int st = 0; st < C::kSt; ++st) sacc[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[st], qf[s], sacc[st], 0, 0, 0);
#pragma unroll
        for (int st = 0; st < C::kSt; ++st) ka[st] = kn[st];
      }
      // sacc[st][v] = score of query qi with tile key 32 st + 8 (v/4) + 4 g + v%4
      if (need_mask) {
        const int lim_g = lim - 4 * g, lo_g = lo - 4 * g;
#pragma unroll
        for (int st = 0; st < C::kSt; ++st)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int kk = st * 32 + (v >> 2) * 8 + (v & 3);
            if (kk > lim_g || (KL && kk < lo_g)) sacc[st][v] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int st = 0; st < C::kSt; ++st)
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[st][v]);
      {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
        mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));  // with lane ^ 32
      }
      const float m_new = fmaxf(m_run, mx * sc);
      if (__any(m_new - m_run > kLazy)) {
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) oacc[dt][v] *= alpha;
        m_run = m_new;
      }
      float psum = 0.f;
#pragma unroll
      for (int st = 0; st < C::kSt; ++st)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float p = __builtin_amdgcn_exp2f(fmaf(sacc[st][v], sc, -m_run));
          sacc[st][v] = p;
          psum += p;
        }
      l_run += psum;
#pragma unroll
      for (int st = 0; st < C::kSt; ++st) {
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          bf16x8 pb;
#pragma unroll
          for (int v = 0; v < 8; ++v) pb[v] = (__bf16)sacc[st][8 * m + v];
          // keys of B slot v: 32 st + 16 m + 8 (v/4) + 4 g + v%4
          // V^T operand: row 32 st + 16 m + 4 (grp / 2) + ri (+ 8 for the
          // upper half), byte 64 dt + 32 (grp & 1) + 8 bq of it, whose 64-byte
          // granule sits at dt ^ f (f = ri, or ri / 2 for D = 64)
          const int r0 = (st * 32 + 16 * m) * C::kRB;
#pragma unroll
          for (int dt = 0; dt < C::kDtiles; ++dt) {
            int vo = (4 * (grp >> 1) + ri) * C::kRB + 32 * (grp & 1) + 8 * bq +
                     ((dt ^ (D == 128 ? ri : (ri >> 1) & 1)) << 6);
            asm volatile("" : "+v"(vo));
            const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vl + (vo + r0)));
            const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vl + (vo + r0 + 8 * C::kRB)));
            const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, oacc[dt], 0, 0, 0);
          }
        }
      }
    }
  };

  // The barrier closing each step also waits for the next tile's copies.
  issue_tile(0, kbuf0, vbuf0);
  __syncthreads();
  for (int t = 0; t < ntiles; t += 2) {
    if (t + 1 < ntiles) issue_tile(t + 1, kbuf1, vbuf1);
    compute_tile(t, kbuf0, vbuf0);
    __syncthreads();
    if (t + 1 >= ntiles) break;
    if (t + 2 < ntiles) issue_tile(t + 2, kbuf0, vbuf0);
    compute_tile(t + 1, kbuf1, vbuf1);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (js < nq) {
    const float inv = 1.f / l_tot;
    const int64_t orow = s0 + js - sq.base;
    __bf16* op = reinterpret_cast<__bf16*>(sq.o) + (orow * H + h) * D;
#pragma unroll
    for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        // oacc[dt][4 v4 + e] = O[qi][32 dt + 8 v4 + 4 g + e]
        uint2 w;
        w.x = focus::pack_bf16x2(oacc[dt][4 * v4 + 0] * inv, oacc[dt][4 * v4 + 1] * inv);
        w.y = focus::pack_bf16x2(oacc[dt][4 * v4 + 2] * inv, oacc[dt][4 * v4 + 3] * inv);
        *reinterpret_cast<uint2*>(op + 32 * dt + 8 * v4 + 4 * g) = w;
      }
    if (g == 0 && sq.lse) sq.lse[orow * H + h] = (m_run + log2f(l_tot)) * kLn2;
  }
}

// ------------------------------------------------- bf16 MFMA, k-mer-local

// The k-mer-local kernel below issues its global -> LDS copies as inline
// assembly, so the compiler does not track them: with the compiler-visible
// copy in this loop's control flow it conservatively waits for every copy in
// flight before a step's LDS reads, which would leave one tile in flight
// instead of three.  The kernel's own waits (a vmcnt wait and a barrier that
// close each step) order every LDS read after the copies it needs.
//
// 16 bytes per lane from src to LDS byte lds + 16 lane (one wave: 1 KB); lds
// goes in M0, which the compiler writes just before, so the copy waits one
// cycle for it (s_nop 0).
__device__ __forceinline__ void copy_to_lds(const void* src, uint32_t lds) {
  asm volatile(
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off"
      :
      : "v"(src), "{m0}"(lds)
      : "memory");
}
__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  typedef const __attribute__((address_space(3))) char lds_char;
  return (uint32_t)(uintptr_t)(lds_char*)p;
}

// q[s] = p[2 s] (16 bytes each, 32 bytes apart) for s < NS, returned only once
// every vector memory operation of this wave has completed (the wait is part
// of the statement, so the compiler tracks no load in flight into q).
template <int NS>
__device__ __forceinline__ void load_q_now(const bf16x8* p, bf16x8 (&q)[NS]) {
  static_assert(NS == 4 || NS == 8, "head_dim 64 or 128");
  u32x4 r[NS];
  if constexpr (NS == 8) {
    asm volatile(
        "global_load_dwordx4 %0, %8, off\n\t"
        "global_load_dwordx4 %1, %8, off offset:32\n\t"
        "global_load_dwordx4 %2, %8, off offset:64\n\t"
        "global_load_dwordx4 %3, %8, off offset:96\n\t"
        "global_load_dwordx4 %4, %8, off offset:128\n\t"
        "global_load_dwordx4 %5, %8, off offset:160\n\t"
        "global_load_dwordx4 %6, %8, off offset:192\n\t"
        "global_load_dwordx4 %7, %8, off offset:224\n\t"
        "s_waitcnt vmcnt(0)"
        : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7])
        : "v"(p)
        : "memory");
  } else {
    asm volatile(
        "global_load_dwordx4 %0, %4, off\n\t"
        "global_load_dwordx4 %1, %4, off offset:32\n\t"
        "global_load_dwordx4 %2, %4, off offset:64\n\t"
        "global_load_dwordx4 %3, %4, off offset:96\n\t"
        "s_waitcnt vmcnt(0)"
        : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3])
        : "v"(p)
        : "memory");
  }
#pragma unroll
  for (int s = 0; s < NS; ++s) q[s] = __builtin_bit_cast(bf16x8, r[s]);
}

// The same loads without the wait: q is written when the loads land.  The
// compiler sees q as written here, so nothing may read, copy or spill it
// before wait_loaded (below) has run; the kernel reads it only after that.
template <int NS>
__device__ __forceinline__ void load_q_async(const bf16x8* p, bf16x8 (&q)[NS]) {
  static_assert(NS == 4 || NS == 8, "head_dim 64 or 128");
  u32x4 r[NS];
  if constexpr (NS == 8) {
    asm volatile(
        "global_load_dwordx4 %0, %8, off\n\t"
        "global_load_dwordx4 %1, %8, off offset:32\n\t"
        "global_load_dwordx4 %2, %8, off offset:64\n\t"
        "global_load_dwordx4 %3, %8, off offset:96\n\t"
        "global_load_dwordx4 %4, %8, off offset:128\n\t"
        "global_load_dwordx4 %5, %8, off offset:160\n\t"
        "global_load_dwordx4 %6, %8, off offset:192\n\t"
        "global_load_dwordx4 %7, %8, off offset:224"
        : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7])
        : "v"(p)
        : "memory");
  } else {
    asm volatile(
        "global_load_dwordx4 %0, %4, off\n\t"
        "global_load_dwordx4 %1, %4, off offset:32\n\t"
        "global_load_dwordx4 %2, %4, off offset:64\n\t"
        "global_load_dwordx4 %3, %4, off offset:96"
        : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3])
        : "v"(p)
        : "memory");
  }
#pragma unroll
  for (int s = 0; s < NS; ++s) q[s] = __builtin_bit_cast(bf16x8, r[s]);
}

// Wait until at most N of this wave's vector memory operations are
// outstanding, as an update of q: reads of q cannot be scheduled before it.
template <int N, int NS>
__device__ __forceinline__ void wait_loaded(bf16x8 (&q)[NS]) {
  static_assert(NS == 4 || NS == 8, "head_dim 64 or 128");
  u32x4 r[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) r[s] = __builtin_bit_cast(u32x4, q[s]);
  if constexpr (NS == 8) {
    asm volatile("s_waitcnt vmcnt(%8)"
                 : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]), "+v"(r[7])
                 : "n"(N));
  } else {
    asm volatile("s_waitcnt vmcnt(%4)" : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]) : "n"(N));
  }
#pragma unroll
  for (int s = 0; s < NS; ++s) q[s] = __builtin_bit_cast(bf16x8, r[s]);
}

// The k-mer-local window attention (Section 3.2 rule): one workgroup streams a
// whole (window, head).  Its 4 waves x 32 rows take the window's 128-row query
// tiles one after another, and the key tiles of all of them form one stream of
// 32-key tiles through four LDS stages, three in flight while one is computed;
// a one-tile summary list stays in LDS for all query tiles (80 KB in all: two
// workgroups fill a compute unit's LDS).
// Query tile q visits the gathered summary list [carried boundary ; the
// window's summaries] and then the window tiles from the one holding the first
// row of its first k-mer up to its last row, with a two-sided mask keeping each
// row's own k-mer.  The copies run three tiles ahead across query-tile
// boundaries (every step copies one tile; past the end of the stream the last
// tile again, into a stage nobody reads any more, so every wait is the same),
// and the next query tile's Q loads while this one is computed.  A workgroup
// pays the start-up latency once per window rather than once per query tile.
template <int D, int W, int NST>
__global__ __launch_bounds__(64 * W, 8 / W) void attn_kl(focus_attn_desc d, float sc, int64_t n_pairs) {
  using C = Cfg<D, W, 32>;
  static_assert(NST >= 3, "at least two tiles in flight");
  __shared__ __attribute__((aligned(1024))) char kb[NST][C::kTile];
  __shared__ __attribute__((aligned(1024))) char vb[NST][C::kTile];
  __shared__ __attribute__((aligned(1024))) char kls[C::kTile], vls[C::kTile];  // resident summary list

  const int tid = threadIdx.x;
  // Block -> (listed window, head), heads fastest: the workgroups running at
  // one time read the same token rows of a few windows (each head its slice
  // of every row), which HBM serves far better than one head's slice of many
  // windows (10.7 vs 7.9 ms at 1 Mb).
  if ((int64_t)blockIdx.x >= n_pairs) return;
  Item it;
  it.list_idx = (int64_t)blockIdx.x / d.n_heads;
  it.h = (int)((int64_t)blockIdx.x % d.n_heads);
  const int64_t gw = listed_window(d, it.list_idx);
  if (gw < 0 || gw >= d.totals.n_windows) {
    if (tid == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
    return;
  }
  const int T = d.win_ntok[gw];
  if (T <= 0) return;
  const int Cw = d.win_cache_off[gw];
  const int b = d.win_seq[gw];
  const int64_t tok0 = d.win_tok_off[gw] - d.qkv_tok_base;
  const int kw = d.win_kmer ? d.win_kmer[gw] : d.kmer_uniform;
  if (b < 0 || b >= d.batch || Cw < 0 || Cw > d.cache_cap || tok0 < 0 || tok0 + T > d.qkv_rows || kw < 0) {
    if (tid == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
    return;
  }
  const int H = d.n_heads, Hkv = d.n_kv_heads, h = it.h;
  const int hk = h / (H / Hkv);
  const int nsum = kw > 0 ? (T + kw) / (kw + 1) : 0;
  const int nct = (nsum + C::kBK) / C::kBK;  // tiles of the summary list (boundary + nsum)
  const int nqt = (T + C::kBQ - 1) / C::kBQ;
  // A one-tile summary list (up to 31 summaries: k >= 32 at windows of 1000)
  // is copied once and stays in LDS; a longer one is streamed again for each
  // query tile (nl of its tiles in the stream).
  const bool resident = nct == 1;
  const int nl = resident ? 0 : nct;
  // Query tile q: its first window tile (the one holding the first row of its
  // first k-mer), the window keys it can see and its tile count.
  auto tw0_of = [&](int q) { return kw > 0 ? q * C::kBQ / (kw + 1) * (kw + 1) / C::kBK : 0; };
  auto nwk_of = [&](int q) { return min(q * C::kBQ + C::kBQ, T); };
  auto ntiles_of = [&](int q) { return nl + (nwk_of(q) + C::kBK - 1) / C::kBK - tw0_of(q); };
  int nsteps = 0;
  for (int q = 0; q < nqt; ++q) nsteps += ntiles_of(q);

  const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
  constexpr int kRPK = 1024 / C::kRB;
  constexpr int kDma = C::kTile / 1024 / C::kWaves;
  static_assert(kDma >= 1 && C::kTile % (1024 * C::kWaves) == 0, "tile must split into 1 KB wave loads");
  constexpr int kPer = 2 * kDma;  // copies a wave issues per tile
  const uint32_t row_bytes = (uint32_t)(Hkv * D * 2);
  uint32_t rowb[kDma], kchunk[kDma], vchunk[kDma];
#pragma unroll
  for (int i = 0; i < kDma; ++i) {
    const int r = (wave * kDma + i) * kRPK + lane / C::kCh16;
    const int p = lane % C::kCh16;
    const int f = D == 128 ? (r & 3) : ((r >> 1) & 1);
    rowb[i] = (uint32_t)r * row_bytes;
    kchunk[i] = (uint32_t)((p ^ (r % C::kCh16)) * 16);
    vchunk[i] = (uint32_t)((((p >> 2) ^ f) * 4 + (p & 3)) * 16);
  }
  const char* kwin = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(d.k) + (tok0 * Hkv + hk) * D);
  const char* vwin = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(d.v) + (tok0 * Hkv + hk) * D);
  const char* kcache = reinterpret_cast<const char*>(
      reinterpret_cast<const __bf16*>(d.cache_k) + ((int64_t)b * d.cache_cap * Hkv + hk) * D);
  const char* vcache = reinterpret_cast<const char*>(
      reinterpret_cast<const __bf16*>(d.cache_v) + ((int64_t)b * d.cache_cap * Hkv + hk) * D);
  const __bf16* qwin = reinterpret_cast<const __bf16*>(d.q) + (tok0 * H + h) * D;
  __bf16* owin = reinterpret_cast<__bf16*>(d.o) + (tok0 * H + h) * D;

  // Q^T of query tile q as the B operand: lane holds query row
  // 128 q + 32 wave + l32 (clamped to the window), head_dim [16s + 8g, +8).
  auto q_row = [&](int q) __attribute__((always_inline)) {
    const int r = min(q * C::kBQ + wave * 32 + l32, T - 1);
    return reinterpret_cast<const bf16x8*>(qwin + (int64_t)r * H * D) + g;
  };

  // Issue side: the next tile of the stream (query tile iq, its tile it_).
  int iq = 0, it_ = 0, i_tw0 = tw0_of(0), i_nwk = nwk_of(0), i_nt = ntiles_of(0);
  // Summary-list entry R = 32 t + r: R = 0 is the carried boundary, R >= 1
  // the window's summary R - 1 at window row R (k + 1) - 1 (the last one at
  // T - 1).  Rows past the list repeat its last entry (masked).
  auto list_src = [&](int t, const char** ks, const char** vs) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kDma; ++i) {
      const int r = (wave * kDma + i) * kRPK + lane / C::kCh16;
      const int R = min(t * C::kBK + r, nsum);
      const bool boundary = R == 0 && Cw > 0;
      const int wrow = R == 0 ? 0 : min(R * (kw + 1) - 1, T - 1);
      ks[i] = (boundary ? kcache + (int64_t)(Cw - 1) * row_bytes : kwin + (int64_t)wrow * row_bytes) + kchunk[i];
      vs[i] = (boundary ? vcache + (int64_t)(Cw - 1) * row_bytes : vwin + (int64_t)wrow * row_bytes) + vchunk[i];
    }
  };
  // This wave's share of a tile: one copy pair per 1 KB.
  auto copy_tile = [&](const char* const* ks, const char* const* vs, char* kbuf, char* vbuf)
      __attribute__((always_inline)) {
    const uint32_t kl = lds_addr(kbuf) + wave * kDma * 1024;
    const uint32_t vl = lds_addr(vbuf) + wave * kDma * 1024;
#pragma unroll
    for (int i = 0; i < kDma; ++i) {
      copy_to_lds(ks[i], kl + i * 1024);
      copy_to_lds(vs[i], vl + i * 1024);
    }
  };
  auto issue_next = [&](char* kbuf, char* vbuf) __attribute__((always_inline)) {
    const char* ks[kDma];
    const char* vs[kDma];
    if (it_ < nl) {
      list_src(it_, ks, vs);
    } else {
      const int row0 = (it_ - nl + i_tw0) * C::kBK;
      const int nvalid = i_nwk - row0;
      const char* kb = kwin + (int64_t)row0 * row_bytes;
      const char* vb = vwin + (int64_t)row0 * row_bytes;
      const uint32_t last = (uint32_t)(nvalid - 1) * row_bytes;
#pragma unroll
      for (int i = 0; i < kDma; ++i) {
        const uint32_t rb = nvalid >= C::kBK ? rowb[i] : min(rowb[i], last);
        ks[i] = kb + (rb + kchunk[i]);
        vs[i] = vb + (rb + vchunk[i]);
      }
    }
    copy_tile(ks, vs, kbuf, vbuf);
    if (it_ + 1 < i_nt) {
      ++it_;
    } else if (iq + 1 < nqt) {
      ++iq;
      it_ = 0;
      i_tw0 = tw0_of(iq);
      i_nwk = nwk_of(iq);
      i_nt = ntiles_of(iq);
    }  // else: the stream has ended; the last tile is copied again
  };

  // Compute side: query tile cq, its tile ct; this lane's row qi, its k-mer
  // index jq and that k-mer's first row qlo; klo_w: first row of the wave's
  // first k-mer.
  int cq = 0, ct = 0, c_tw0 = tw0_of(0), c_nt = ntiles_of(0);
  int wq_lo = 0, qi = 0, jq = 0, qlo = 0, klo_w = 0;
  bool wave_live = false;
  auto set_q = [&](int q) __attribute__((always_inline)) {
    wq_lo = q * C::kBQ + wave * 32;
    qi = wq_lo + l32;
    wave_live = wq_lo < T;
    jq = kw > 0 ? qi / (kw + 1) : 0;
    qlo = jq * (kw + 1);
    klo_w = kw > 0 ? wq_lo / (kw + 1) * (kw + 1) : 0;
  };

  f32x16 oacc[C::kDtiles];
#pragma unroll
  for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[dt][v] = 0.f;
  float m_run = kMinit, l_run = 0.f;
  bf16x8 qf[C::kKsteps], qn[C::kKsteps];
  const int grp = lane >> 4, ri = (lane >> 2) & 3, bq = lane & 3;

  // One tile of keys: the summary list's entries row0 .. row0 + 31 (in_list),
  // else window rows row0 .. row0 + 31.
  auto compute_tile = [&](const char* kl, const char* vl, bool in_list, int row0) __attribute__((always_inline)) {
    const bool live = wave_live && (in_list || (row0 <= wq_lo + 31 && row0 + C::kBK > klo_w));
    // visible tile keys: lo <= kk <= lim
    const int lim = in_list ? jq - row0 : qi - row0;
    const int lo = in_list ? (Cw > 0 ? 0 : 1) - row0 : qlo - row0;
    if (!live) return;
    f32x16 sacc;
#pragma unroll
    for (int v = 0; v < 16; ++v) sacc[v] = 0.f;
    const int kx = g ^ (l32 & (C::kCh16 - 1));
    auto kread = [&](int s) {
      int ko = l32 * C::kRB + (((2 * s) ^ kx) << 4);
      asm volatile("" : "+v"(ko));
      return *reinterpret_cast<const bf16x8*>(kl + ko);
    };
    bf16x8 ka = kread(0), kn;
#pragma unroll
    for (int s = 0; s < C::kKsteps; ++s) {
      if (s + 1 < C::kKsteps) kn = kread(s + 1);
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[s], sacc, 0, 0, 0);
      ka = kn;
    }
    // sacc[v] = score of query qi with tile key 8 (v/4) + 4 g + v%4
    {
      const int lim_g = lim - 4 * g, lo_g = lo - 4 * g;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int kk = (v >> 2) * 8 + (v & 3);
        if (kk > lim_g || kk < lo_g) sacc[v] = -INFINITY;
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[v]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));  // with lane ^ 32
    }
    const float m_new = fmaxf(m_run, mx * sc);
    if (__any(m_new - m_run > kLazy)) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[dt][v] *= alpha;
      m_run = m_new;
    }
    float psum = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const float p = __builtin_amdgcn_exp2f(fmaf(sacc[v], sc, -m_run));
      sacc[v] = p;
      psum += p;
    }
    l_run += psum;
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      bf16x8 pb;
#pragma unroll
      for (int v = 0; v < 8; ++v) pb[v] = (__bf16)sacc[8 * m + v];
      const int r0 = 16 * m * C::kRB;
#pragma unroll
      for (int dt = 0; dt < C::kDtiles; ++dt) {
        int vo = (4 * (grp >> 1) + ri) * C::kRB + 32 * (grp & 1) + 8 * bq + ((dt ^ (D == 128 ? ri : (ri >> 1) & 1)) << 6);
        asm volatile("" : "+v"(vo));
        const bf16x4 lo4 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vl + (vo + r0)));
        const bf16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vl + (vo + r0 + 8 * C::kRB)));
        const bf16x8 a = __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7);
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, oacc[dt], 0, 0, 0);
      }
    }
  };

  // O and LSE of the finished query tile.
  auto finish_q = [&]() __attribute__((always_inline)) {
    float l_tot;
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l_run), __float_as_uint(l_run), false, false);
      l_tot = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);  // with lane ^ 32
    }
    if (wave_live) {
      if (qi < T) {
        const float inv = 1.f / l_tot;
        __bf16* op = owin + (int64_t)qi * H * D + 4 * g;
        // oacc[dt][4 v4 + e] = O[qi][32 dt + 8 v4 + 4 g + e]
        auto w2 = [&](int dt, int v4) {
          uint2 w;
          w.x = focus::pack_bf16x2(oacc[dt][4 * v4 + 0] * inv, oacc[dt][4 * v4 + 1] * inv);
          w.y = focus::pack_bf16x2(oacc[dt][4 * v4 + 2] * inv, oacc[dt][4 * v4 + 3] * inv);
          return w;
        };
#pragma unroll
        for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
          for (int v4 = 0; v4 < 4; ++v4) *reinterpret_cast<uint2*>(op + 32 * dt + 8 * v4) = w2(dt, v4);
        if (g == 0 && d.lse) d.lse[(tok0 + qi) * H + h] = (m_run + log2f(l_tot)) * kLn2;
      }
    }
#pragma unroll
    for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
      for (int v = 0; v < 16; ++v) oacc[dt][v] = 0.f;
    m_run = kMinit;
    l_run = 0.f;
  };

  // Step u: copies of tile u + 3 into the stage tile u - 1 left, tile u
  // computed (after the resident summary list, at a query tile's first
  // step), then this wave waits until its copies of tile u + 1 have landed
  // (those of u + 2 and u + 3 may stay in flight; O stores issued after them
  // only make the wait stricter) and the barrier makes that true for every
  // wave's share.
  auto wait_next = [&]() __attribute__((always_inline)) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    constexpr int kYounger = (NST - 2) * kPer;
    __builtin_amdgcn_s_waitcnt((kYounger & 15) | ((kYounger >> 4) << 14) | (7 << 4) | (15 << 8));
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
  };
  auto step = [&](int u, const char* kc, const char* vc, char* kn_, char* vn_) __attribute__((always_inline)) {
    issue_next(kn_, vn_);
    // First tile of query tile cq: the next one's Q starts loading, after this
    // step's copies.
    if (ct == 0 && cq + 1 < nqt) load_q_async<C::kKsteps>(q_row(cq + 1), qn);
    if (ct == 0 && resident) compute_tile(kls, vls, true, 0);
    compute_tile(kc, vc, ct < nl, ct < nl ? ct * C::kBK : (ct - nl + c_tw0) * C::kBK);
    if (++ct == c_nt) {
      if (cq + 1 < nqt) {
        // Every query tile but the last streams at least four tiles, so at
        // least three steps' copies were issued after that Q: once no more
        // than the copies of the three tiles in flight are outstanding, it has
        // landed.
        wait_loaded<(NST - 1) * kPer>(qn);
#pragma unroll
        for (int s = 0; s < C::kKsteps; ++s) qf[s] = qn[s];
      }
      finish_q();
      if (cq + 1 < nqt) {
        ++cq;
        ct = 0;
        c_tw0 = tw0_of(cq);
        c_nt = ntiles_of(cq);
        set_q(cq);
      }
    }
    if (u + 1 < nsteps) wait_next();
  };

  load_q_now<C::kKsteps>(q_row(0), qf);
  set_q(0);
  if (resident) {
    const char* ks[kDma];
    const char* vs[kDma];
    list_src(0, ks, vs);
    copy_tile(ks, vs, kls, vls);
  }
#pragma unroll
  for (int j = 0; j < NST - 1; ++j) issue_next(kb[j], vb[j]);
  wait_next();  // the summary list and tile 0 have landed
  for (int u = 0; u < nsteps; u += NST) {
#pragma unroll
    for (int j = 0; j < NST; ++j) {
      if (u + j >= nsteps) break;
      step(u + j, kb[j], vb[j], kb[(j + NST - 1) % NST], vb[(j + NST - 1) % NST]);
    }
  }
  // No copy may still be writing this workgroup's LDS when it ends (and the
  // last O stores complete).
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
}

// ------------------------------------------- bf16 MFMA, C(t), pipelined waves

// The C(t) window attention: one workgroup = 8 waves x 32 query rows of one
// (window, head), two waves per SIMD (up to 256 registers each).  Keys arrive
// in 64-key tiles through four LDS stages (copies issued by every wave, three
// tiles ahead, spread over the step); each wave walks the keys in 32-key
// sub-tiles with a one-sub-tile software pipeline:
//   V^T operands of sub-tile j are read from LDS;
//   S_{j+1} = K_{j+1} Q^T is issued on the MFMA pipe (its K operands were read
//     one sub-tile earlier), and runs while the VALU does the softmax of S_j;
//   the K operands of sub-tile j + 2 are read;
//   O^T += V_j^T P_j^T.
// So every LDS operand is read about one sub-tile before its MFMA, and the
// exponentials of one sub-tile overlap the score MFMAs of the next.  A
// barrier closes every 64-key step; at its end each wave waits only for the
// copies of the tile the next step starts reading.
template <int D>
struct CtCfg {
  static constexpr int kWaves = 8;
  static constexpr int kBQ = 32 * kWaves;                // query rows per block
  static constexpr int kBK = 64;                         // keys per LDS tile
  static constexpr int kRB = D * 2;                      // bytes per row
  static constexpr int kTile = kBK * kRB;                // bytes per tile per tensor
  static constexpr int kCh16 = kRB / 16;                 // 16-byte chunks per row
  static constexpr int kKsteps = D / 16;                 // MFMA k-steps of QK^T
  static constexpr int kDtiles = D / 32;                 // 32-row blocks of O^T
  static constexpr int kRPK = 1024 / kRB;                // tile rows per 1 KB wave copy
  static constexpr int kDma = kTile / 1024 / kWaves;     // wave copies per tile, tensor and wave
  static constexpr int kPerStep = 2 * kDma;              // copies a wave issues per step
};

template <int D>
__global__ __launch_bounds__(512, 2) void attn_ct(
    focus_attn_desc d, float sc, int64_t n_pairs, int QT, Split sp) {
  using C = CtCfg<D>;
  static_assert(C::kDma >= 1 && C::kTile % (1024 * C::kWaves) == 0, "tile must split into 1 KB wave loads");
  // Four K and four V stages as separate arrays, every reference static (the
  // step loop is unrolled four times): the compiler then tells the buffer a
  // read uses from the ones being filled.
  __shared__ __attribute__((aligned(1024))) char kb0[C::kTile], kb1[C::kTile], kb2[C::kTile], kb3[C::kTile];
  __shared__ __attribute__((aligned(1024))) char vb0[C::kTile], vb1[C::kTile], vb2[C::kTile], vb3[C::kTile];

  const int tid = threadIdx.x;
  int64_t bid = blockIdx.x;
  int split = 0;
  if (sp.n > 1) {
    const int64_t r = bid / focus::kXcds;
    split = (int)(r % sp.n);
    bid = (r / sp.n) * focus::kXcds + bid % focus::kXcds;
  }
  const Item it = map_block<true>(bid, n_pairs, d.n_heads, QT);
  if (!it.valid) return;
  const int64_t gw = listed_window(d, it.list_idx);
  if (gw < 0 || gw >= d.totals.n_windows) {
    if (tid == 0 && it.qt == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
    return;
  }
  const int T = d.win_ntok[gw];
  const int q0 = it.qt * C::kBQ;
  if (q0 >= T) return;
  const int Cw = d.win_cache_off[gw];
  const int b = d.win_seq[gw];
  const int64_t tok0 = d.win_tok_off[gw] - d.qkv_tok_base;
  if (b < 0 || b >= d.batch || Cw < 0 || Cw > d.cache_cap || tok0 < 0 || tok0 + T > d.qkv_rows) {
    if (tid == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
    return;
  }
  const int H = d.n_heads, Hkv = d.n_kv_heads, h = it.h;
  const int hk = h / (H / Hkv);
  const int nwk = min(T, q0 + C::kBQ);  // window keys any query of this block sees
  // keys: nct tiles of cache rows [0, Cw), then nwt tiles of window rows [0, nwk)
  const int nct = (Cw + C::kBK - 1) / C::kBK;
  const int nwt = (nwk + C::kBK - 1) / C::kBK;
  const int tb = (int)((int64_t)split * (nct + nwt) / sp.n);
  const int ntiles = (int)((int64_t)(split + 1) * (nct + nwt) / sp.n) - tb;

  // (the wave index through readfirstlane: the compiler then keeps everything
  // derived from it in scalar registers and branches on it with scalar tests)
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, l32 = lane & 31, g = lane >> 5;
  const int qi = q0 + wave * 32 + l32;
  const int wq_lo = q0 + wave * 32, wq_hi = min(wq_lo + 31, T - 1);
  const bool wave_live = wq_lo < T;

  // Q^T as the B operand: lane holds query l32, head_dim [16 s + 8 g, +8).
  bf16x8 qf[C::kKsteps];
  {
    const bf16x8* qp = reinterpret_cast<const bf16x8*>(reinterpret_cast<const __bf16*>(d.q) +
                                                       ((tok0 + min(qi, T - 1)) * H + h) * D);
#pragma unroll
    for (int s = 0; s < C::kKsteps; ++s) qf[s] = qp[2 * s + g];
  }

  // Copies: wave copy i of this wave fills tile rows (wave kDma + i) kRPK +
  // lane / kCh16; the lane at 16-byte slot p of a row fetches the global chunk
  // the swizzled layout keeps there (K: chunk c of row r at c ^ (r mod kCh16);
  // V: 64-byte granule x of row r at x ^ f(r)).  The last tile of a phase
  // clamps its rows to the last valid one (the extra rows are masked).
  const uint32_t row_bytes = (uint32_t)(Hkv * D * 2);
  uint32_t rowb[C::kDma], kchunk[C::kDma], vchunk[C::kDma];
#pragma unroll
  for (int i = 0; i < C::kDma; ++i) {
    const int r = (wave * C::kDma + i) * C::kRPK + lane / C::kCh16;
    const int p = lane % C::kCh16;
    const int f = D == 128 ? (r & 3) : ((r >> 1) & 1);
    rowb[i] = (uint32_t)r * row_bytes;
    kchunk[i] = (uint32_t)((p ^ (r % C::kCh16)) * 16);
    vchunk[i] = (uint32_t)((((p >> 2) ^ f) * 4 + (p & 3)) * 16);
  }
  const char* kwin = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(d.k) + (tok0 * Hkv + hk) * D);
  const char* vwin = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(d.v) + (tok0 * Hkv + hk) * D);
  const char* kcache = reinterpret_cast<const char*>(
      reinterpret_cast<const __bf16*>(d.cache_k) + ((int64_t)b * d.cache_cap * Hkv + hk) * D);
  const char* vcache = reinterpret_cast<const char*>(
      reinterpret_cast<const __bf16*>(d.cache_v) + ((int64_t)b * d.cache_cap * Hkv + hk) * D);
  // Key stream: nct cache tiles, then the window tiles.  The cache tiles start
  // pad = 64 nct - C_w rows before cache row 0, so the one partial cache tile
  // is tile 0 (its first pad rows are not keys) and every later tile up to
  // the block's diagonal is full and unmasked.  Copy sources: tile tg starts
  // at (tg < nct ? cache - pad rows : window - nct tiles) + tg tiles.  Wave
  // copy i of a tile (K and V) into (kbuf, vbuf); a partial tile clamps its
  // rows into [lo, last], the valid ones.
  const int pad = nct * C::kBK - Cw;
  const int64_t tstride = (int64_t)C::kBK * row_bytes;
  const char* kcache_b = kcache - (int64_t)pad * row_bytes;
  const char* vcache_b = vcache - (int64_t)pad * row_bytes;
  const char* kwin_b = kwin - nct * tstride;
  const char* vwin_b = vwin - nct * tstride;
  const int wfull = nct + nwk / C::kBK;        // window tiles in [nct, wfull) are full
  struct Src {
    const char* k;
    const char* v;
    uint32_t lo, last;  // byte offsets of the tile's first and last valid rows
    bool full;
  };
  auto tile_src = [&](int u) __attribute__((always_inline)) {
    const int tg = tb + u;
    const bool in_cache = tg < nct;
    Src r;
    r.k = (in_cache ? kcache_b : kwin_b) + tg * tstride;
    r.v = (in_cache ? vcache_b : vwin_b) + tg * tstride;
    r.full = in_cache ? (tg > 0 || pad == 0) : tg < wfull;
    r.lo = (uint32_t)(in_cache && tg == 0 ? pad : 0) * row_bytes;
    r.last = (uint32_t)(in_cache ? C::kBK - 1 : min(C::kBK, nwk - (tg - nct) * C::kBK) - 1) * row_bytes;
    return r;
  };
  auto issue = [&](const Src& sr, char* kbuf, char* vbuf, int i, bool clamp) __attribute__((always_inline)) {
    const uint32_t rb = clamp ? min(max(rowb[i], sr.lo), sr.last) : rowb[i];
    const char* ks = sr.k + (rb + kchunk[i]);
    const char* vs = sr.v + (rb + vchunk[i]);
    char* kl = kbuf + (wave * C::kDma + i) * 1024;
    char* vl = vbuf + (wave * C::kDma + i) * 1024;
    __builtin_amdgcn_global_load_lds(ks, (lds_void*)kl, 16, 0, 0);
    __builtin_amdgcn_global_load_lds(vs, (lds_void*)vl, 16, 0, 0);
  };

  // Sub-tile j (32 keys) = half j & 1 of local tile j >> 1, i.e. global
  // sub-tile J = 2 tb + j: stream rows [32 J, 32 J + 32), cache row
  // 32 J + r - pad while J < 2 nct, then window row 32 (J - 2 nct) + r.  This
  // wave computes sub-tiles j < jlive (the window rows past its last query
  // are skipped).  Masks: the rows of tile 0 below pad, and the window rows
  // past the query (from the wave's first diagonal sub-tile, wmask, on).
  const int J0 = 2 * tb;
  const int jlive = wave_live ? min(2 * (tb + ntiles), 2 * nct + (wq_hi >> 5) + 1) - J0 : 0;
  const int wmask = 2 * nct + (wq_lo >> 5);
  auto need_mask = [&](int J) { return 32 * J < pad || J >= wmask; };

  // LDS operand offsets (lane parts; buffers and sub-tile rows are immediates).
  // K row 32 half + l32, chunk 2 s + g sits at chunk (2 s + g) ^ (l32 mod kCh16).
  int kofs[C::kKsteps];
  {
    const int kx = g ^ (l32 & (C::kCh16 - 1));
#pragma unroll
    for (int s = 0; s < C::kKsteps; ++s) kofs[s] = l32 * C::kRB + (((2 * s) ^ kx) << 4);
  }
  // V^T operand: lane = 16 grp + 4 ri + bq reads row 4 (grp / 2) + ri (+ 16 m,
  // + 8 for the upper half) of the sub-tile, bytes 64 dt + 32 (grp & 1) + 8 bq,
  // whose 64-byte granule sits at dt ^ f (f = ri, or ri / 2 for D = 64).
  int vofs[C::kDtiles];
  {
    const int grp = lane >> 4, ri = (lane >> 2) & 3, bq = lane & 3;
    const int f = D == 128 ? ri : (ri >> 1) & 1;
#pragma unroll
    for (int dt = 0; dt < C::kDtiles; ++dt)
      vofs[dt] = (4 * (grp >> 1) + ri) * C::kRB + 32 * (grp & 1) + 8 * bq + ((dt ^ f) << 6);
  }
  // Keeps the offsets opaque to loop-invariant code motion, so the compiler
  // folds buffer and row into the instructions' immediate offsets instead of
  // holding one address register per (buffer, operand).
  auto pin_offsets = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < C::kKsteps; ++s) asm volatile("" : "+v"(kofs[s]));
#pragma unroll
    for (int dt = 0; dt < C::kDtiles; ++dt) asm volatile("" : "+v"(vofs[dt]));
  };

  bf16x8 kop[C::kKsteps];
  auto read_k = [&](const char* kbuf, int half) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < C::kKsteps; ++s)
      kop[s] = *reinterpret_cast<const bf16x8*>(kbuf + (kofs[s] + half * 32 * C::kRB));
  };
  f32x16 sacc[2];
  auto qk = [&](f32x16& acc) __attribute__((always_inline)) {
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] = 0.f;
#pragma unroll
    for (int s = 0; s < C::kKsteps; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[s], qf[s], acc, 0, 0, 0);
  };

  f32x16 oacc[C::kDtiles];
#pragma unroll
  for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[dt][v] = 0.f;
  float m_run = kMinit, l_run = 0.f;

  // One sub-tile iteration (see the header).  half = j & 1 is a constant
  // after inlining; kc / vc hold tile j >> 1, kn tile (j >> 1) + 1; copies of
  // tile u + 3 go to (kcp, vcp).
  auto sub = [&](int j, const int half, const bool fast, const char* vc, const char* kn, char* kcp, char* vcp,
                 int u, const Src& src) __attribute__((always_inline)) {
    const bool lj = fast || j < jlive, lj1 = fast || j + 1 < jlive;
    // A wave keeps at most 15 LDS reads in flight (the counter's range), so
    // the 16 V^T reads go in two halves around the score MFMAs, and the 8 K
    // reads follow the softmax's row maximum.  The reads are unconditional (a
    // dead sub-tile reads a stale but valid buffer), so the compiler's
    // counter waits stay exact.
    bf16x8 vop[2 * C::kDtiles];
    auto read_v = [&](int m) __attribute__((always_inline)) {
#pragma unroll
      for (int dt = 0; dt < C::kDtiles; ++dt) {
        const char* p = vc + (vofs[dt] + (32 * half + 16 * m) * C::kRB);
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p);
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 8 * C::kRB));
        vop[m * C::kDtiles + dt] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    };
    read_v(0);
    // S_{j+1}: its K operands were read one sub-tile earlier
    if (lj1) qk(sacc[half ^ 1]);
    read_v(1);
    if (fast || u + 3 < ntiles) {
#pragma unroll
      for (int i = 0; i < C::kDma; ++i)
        if ((i & 1) == half) issue(src, kcp, vcp, i, !fast && !src.full);
    }
    if (lj) {
      f32x16& s = sacc[half];
      const int J = J0 + j;
      if (!fast && need_mask(J)) {
        // s[v] = score of query qi with sub-tile key 8 (v/4) + 4 g + v%4
        if (J < 2 * nct) {
          const int lo_g = pad - 32 * J - 4 * g;  // rows of tile 0 before cache row 0
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if ((v >> 2) * 8 + (v & 3) < lo_g) s[v] = -INFINITY;
        } else {
          const int lim_g = qi - 32 * (J - 2 * nct) - 4 * g;
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if ((v >> 2) * 8 + (v & 3) > lim_g) s[v] = -INFINITY;
        }
      }
      float mx = s[0];
#pragma unroll
      for (int v = 1; v < 16; ++v) mx = fmaxf(mx, s[v]);
      {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
        mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));  // with lane ^ 32
      }
      const float m_new = fmaxf(m_run, mx * sc);
      if (__any(m_new - m_run > kLazy)) {
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
          for (int v = 0; v < 16; ++v) oacc[dt][v] *= alpha;
        m_run = m_new;
      }
    }
    // K operands of sub-tile j + 2
    read_k(kn, half);
    if (lj) {
      f32x16& s = sacc[half];
      float psum = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[v], sc, -m_run));
        s[v] = p;
        psum += p;
      }
      l_run += psum;
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        bf16x8 pb;
#pragma unroll
        for (int v = 0; v < 8; ++v) pb[v] = (__bf16)s[8 * m + v];
#pragma unroll
        for (int dt = 0; dt < C::kDtiles; ++dt)
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[m * C::kDtiles + dt], pb, oacc[dt], 0, 0, 0);
      }
    }
  };

  // vmcnt(n): this wave's copies older than its last n have landed
  auto wait_copies = [&](bool keep_one_step) __attribute__((always_inline)) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    constexpr int kVm = C::kPerStep;
    if (keep_one_step)
      __builtin_amdgcn_s_waitcnt((kVm & 15) | ((kVm >> 4) << 14) | (7 << 4) | (15 << 8));
    else
      __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));  // vmcnt(0)
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
  };
  // step u: sub-tiles 2u, 2u + 1 from tile u (V in vc); K of tile u + 1
  // (kn); copies of tile u + 3 into (kcp, vcp), the buffers tile u - 1 left.
  // A clean step (fast = true) has every sub-tile live and unmasked for every
  // wave and copies a full tile; it runs without any branch but the softmax's
  // rescaling test.
  auto step = [&](int u, const char* vc, const char* kn, char* kcp, char* vcp, const bool fast)
      __attribute__((always_inline)) {
    pin_offsets();
    Src src;
    if (fast) {
      const int tg = tb + u + 3;
      const int64_t off = (int64_t)tg * tstride;
      const bool c = tg < nct;
      src.k = (c ? kcache_b : kwin_b) + off;
      src.v = (c ? vcache_b : vwin_b) + off;
      src.lo = 0;
      src.last = 0;
      src.full = true;
    } else {
      src = tile_src(u + 3);
    }
    sub(2 * u, 0, fast, vc, kn, kcp, vcp, u, src);
    sub(2 * u + 1, 1, fast, vc, kn, kcp, vcp, u, src);
    // step u + 1 reads K of tile u + 2: wait for it (tile u + 3 may stay in flight)
    wait_copies(fast || u + 3 < ntiles);
  };

  // The scale arrives by a scalar load whose first use is inside the loop;
  // using it here puts the wait for that load before the loop instead of
  // (conservatively) at the top of every iteration.
  asm volatile("" ::"v"(sc));
  // Clean steps: tiles tb + u fully visible to the block's first query (the
  // cache tiles past a partial tile 0, the window tiles below the block's
  // rows) whose copy, tile u + 3, is a full tile; they form one run
  // [u0, u1).  Tile u sits in stage (u - u0) mod 4, so the run starts on stage
  // 0; a partial tile 0 (u0 = 1) takes stage 3 and the general step.  The
  // run goes in rounds of four, its last (u1 - u0) mod 4 steps and the
  // diagonal band after it in the general loop.
  const int u0 = (tb == 0 && pad > 0 && ntiles > 0) ? 1 : 0;
  const int u1 = max(u0, min(min(nct + (q0 + 1) / C::kBK, wfull - 3) - tb, ntiles - 3));
  const int nclean = (u1 - u0) & ~3;
  // prologue: tiles 0..2 in flight, wait for 0 and 1
  {
    const Src s0 = tile_src(0), s1 = tile_src(1), s2 = tile_src(2);
    if (u0 == 0) {
#pragma unroll
      for (int i = 0; i < C::kDma; ++i) {
        if (ntiles > 0) issue(s0, kb0, vb0, i, !s0.full);
        if (ntiles > 1) issue(s1, kb1, vb1, i, !s1.full);
        if (ntiles > 2) issue(s2, kb2, vb2, i, !s2.full);
      }
      wait_copies(ntiles > 2);
      read_k(kb0, 0);
      if (0 < jlive) qk(sacc[0]);
      read_k(kb0, 1);
    } else {
#pragma unroll
      for (int i = 0; i < C::kDma; ++i) {
        issue(s0, kb3, vb3, i, true);
        if (ntiles > 1) issue(s1, kb0, vb0, i, !s1.full);
        if (ntiles > 2) issue(s2, kb1, vb1, i, !s2.full);
      }
      wait_copies(ntiles > 2);
      read_k(kb3, 0);
      if (0 < jlive) qk(sacc[0]);
      read_k(kb3, 1);
    }
  }
  // Let every scalar load land before the loop (lgkmcnt(0) once): a scalar
  // load still pending there would make the compiler wait for all LDS reads
  // at every counter wait inside the loop.
  __builtin_amdgcn_s_waitcnt(0xC07F);
  int u = 0;
  if (u0 > 0) {
    step(0, vb3, kb0, kb2, vb2, false);
    u = 1;
  }
  for (; u < u0 + nclean; u += 4) {
    step(u, vb0, kb1, kb3, vb3, true);
    step(u + 1, vb1, kb2, kb0, vb0, true);
    step(u + 2, vb2, kb3, kb1, vb1, true);
    step(u + 3, vb3, kb0, kb2, vb2, true);
  }
  for (; u < ntiles; u += 4) {
    step(u, vb0, kb1, kb3, vb3, false);
    if (u + 1 >= ntiles) break;
    step(u + 1, vb1, kb2, kb0, vb0, false);
    if (u + 2 >= ntiles) break;
    step(u + 2, vb2, kb3, kb1, vb1, false);
    if (u + 3 >= ntiles) break;
    step(u + 3, vb3, kb0, kb2, vb2, false);
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (sp.n > 1) {
    // key split: the unnormalised output and (max, sum) of this tile range
    if (qi < T && qi < sp.rows) {
      const int64_t pidx = (((int64_t)split * sp.nwl + it.list_idx) * sp.rows + qi) * H + h;
      float* op = sp.po + pidx * D;
#pragma unroll
      for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4)
          *reinterpret_cast<float4*>(op + 32 * dt + 8 * v4 + 4 * g) =
              make_float4(oacc[dt][4 * v4], oacc[dt][4 * v4 + 1], oacc[dt][4 * v4 + 2], oacc[dt][4 * v4 + 3]);
      if (g == 0) *reinterpret_cast<float2*>(sp.pml + pidx * 2) = make_float2(m_run, l_tot);
    }
    return;
  }
  if (qi < T) {
    const float inv = 1.f / l_tot;
    const int64_t orow = tok0 + qi;
    __bf16* op = reinterpret_cast<__bf16*>(d.o) + (orow * H + h) * D;
#pragma unroll
    for (int dt = 0; dt < C::kDtiles; ++dt)
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        // oacc[dt][4 v4 + e] = O[qi][32 dt + 8 v4 + 4 g + e]
        uint2 w;
        w.x = focus::pack_bf16x2(oacc[dt][4 * v4 + 0] * inv, oacc[dt][4 * v4 + 1] * inv);
        w.y = focus::pack_bf16x2(oacc[dt][4 * v4 + 2] * inv, oacc[dt][4 * v4 + 3] * inv);
        *reinterpret_cast<uint2*>(op + 32 * dt + 8 * v4 + 4 * g) = w;
      }
    if (g == 0 && d.lse) d.lse[orow * H + h] = (m_run + log2f(l_tot)) * kLn2;
  }
}

// --------------------------------------- bf16 MFMA, summary queries under C(t)

// The adapter attention under C(t) (eq. focus-attn with the summary tokens as
// the only queries), many windows per workgroup: G listed windows in a row put
// their summaries in the workgroup's 32 W query slots (window k's B_k
// summaries at slots off_k .. off_k + B_k - 1, off_k = B_0 + ... + B_{k-1};
// wave w holds slots 32 w .. 32 w + 31).  For each run of the group's windows
// on one sequence:
//   cache phase   the W waves stream that sequence's cache rows [0, max C)
//                 once, in 64-row stages through two shared LDS stages, every
//                 wave copying its share and a barrier closing each stage; a
//                 row is visible to a slot while it is below the C_w of the
//                 slot's own window (the caches of the windows of one sequence
//                 are prefixes of each other), so the cache crosses into LDS
//                 once per 32 W slots instead of once per window;
//   window phase  each wave, on its own, streams rows [0, last summary's row]
//                 of each window it holds slots of, 32 rows at a time through
//                 its private LDS region, visible to that window's slots up to
//                 the slot's own row.  A tile's operands go to registers
//                 before the next tile is copied into the same region, so the
//                 copy overlaps the tile's arithmetic.
// Every summary of a window must see the window's rows up to its own, and the
// last summary ends the window: the window phase reads essentially every K/V
// row once, which bounds the kernel by HBM.  A slot that holds no summary has a
// zero query and sees every key (its result is dropped), so it forces no
// masking.
template <int D, int W>
__global__ __launch_bounds__(64 * W, 2) void attn_sq_block(focus_attn_desc d, float sc, int64_t n_pairs, int64_t nwl,
                                                          int G, int wpw, SumQ sq) {
  static_assert(W == 4 || W == 8, "four or eight waves");
  constexpr int kSlots = 32 * W;
  constexpr int kBK = 32, kRB = D * 2, kTile = kBK * kRB, kCh16 = kRB / 16;
  constexpr int kKsteps = D / 16, kDtiles = D / 32;
  constexpr int kRPK = 1024 / kRB;             // rows per 1 KB wave copy
  constexpr int kTileCopies = kTile / 1024;    // wave copies per 32-row tile and tensor
  constexpr int kStage = 2 * kTile;            // a 64-row stage of one tensor = one region
  constexpr int kStageCopies = kStage / 1024;
  constexpr int kUnused = W == 8 ? 2 * kTile : 16;
  // one region per wave: [K tile | V tile] in the window phase; in the cache
  // phase regions 0 / 1 are K / V of stage 0 and regions 2 / 3 of stage 1
  __shared__ __attribute__((aligned(1024))) char rg0[2 * kTile], rg1[2 * kTile], rg2[2 * kTile], rg3[2 * kTile];
  __shared__ __attribute__((aligned(1024))) char rg4[kUnused], rg5[kUnused], rg6[kUnused], rg7[kUnused];
  // per window of the group: token and summary offsets, window id, C_w,
  // sequence, summaries, slot offset, rows of the window phase
  __shared__ int64_t wg_tok0[kSlots], wg_s0[kSlots];
  __shared__ int wg_win[kSlots], wg_C[kSlots], wg_b[kSlots], wg_ns[kSlots], wg_off[kSlots + 1], wg_nwk[kSlots];
  __shared__ int bad_any;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, l32 = lane & 31, g = lane >> 5;
  const Item it = map_block(blockIdx.x, n_pairs, d.n_heads, 1);
  if (!it.valid) return;
  const int H = d.n_heads, Hkv = d.n_kv_heads, h = it.h;
  const int hk = h / (H / Hkv);
  const int64_t li0 = it.list_idx * G;
  const int nk = (int)min((int64_t)G, nwl - li0);  // windows in this group
  if (nk <= 0) return;

  // thread k < nk reads window k's description; slot offsets by a prefix sum
  if (tid == 0) bad_any = 0;
  __syncthreads();
  if (tid < nk) {
    const int64_t gw = listed_window(d, li0 + tid);
    bool bad = gw < 0 || gw >= d.totals.n_windows;
    if (!bad) {
      const int T = d.win_ntok[gw], C = d.win_cache_off[gw], b = d.win_seq[gw], ns = sq.win_nsum[gw];
      const int64_t tok0 = d.win_tok_off[gw] - d.qkv_tok_base, s0 = sq.win_sum_off[gw];
      bad = b < 0 || b >= d.batch || C < 0 || C > d.cache_cap || tok0 < 0 || tok0 + T > d.qkv_rows || ns < 0 ||
            ns > T || s0 < sq.base || s0 + ns > sq.base + sq.rows;
      if (!bad) {
        wg_win[tid] = (int)gw;
        wg_tok0[tid] = tok0;
        wg_s0[tid] = s0;
        wg_C[tid] = C;
        wg_b[tid] = b;
        wg_ns[tid] = ns;
        int nwk = 0;
        if (ns > 0) {
          const int64_t r = sq.sum_tok[s0 + ns - 1] - d.win_tok_off[gw];
          nwk = (int)(r < 0 ? 0 : r >= T ? T - 1 : r) + 1;
        }
        wg_nwk[tid] = nwk;
      }
    }
    if (bad) bad_any = 1;
  }
  __syncthreads();
  if (tid == 0 && !bad_any) {
    // wpw > 0: wpw whole windows per wave (window k opens wave k / wpw at its
    // first slot), so that no window's rows are streamed by two waves;
    // wpw = 0: the summaries packed one after the other
    int off = 0;
    for (int k = 0; k < nk; ++k) {
      if (wpw > 0 && k % wpw == 0) off = 32 * (k / wpw);
      wg_off[k] = off;
      off += wg_ns[k];
      if (wpw > 0 && off > 32 * (k / wpw + 1)) bad_any = 1;  // a window past its wave's slots
    }
    wg_off[nk] = off;
    if (off > kSlots) bad_any = 1;  // more summaries than slots
  }
  __syncthreads();
  if (bad_any) {
    if (tid == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
    return;
  }

  // this lane's slot: window kl (the last window whose offset is <= slot),
  // its summary s (global index) and the summary's window row pos
  const int slot = wave * 32 + l32;
  int kl = -1, pos = 0;
  int64_t s = 0;
  if (slot < wg_off[nk]) {
    int lo = 0, hi = nk - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (wg_off[mid] <= slot) lo = mid; else hi = mid - 1;
    }
    kl = slot - wg_off[lo] < wg_ns[lo] ? lo : -1;  // else a slot between two waves' windows
  }
  if (kl >= 0) {
    s = wg_s0[kl] + (slot - wg_off[kl]);
    const int64_t r = sq.sum_tok[s] - d.win_tok_off[wg_win[kl]];
    pos = (int)min(max(r, (int64_t)0), (int64_t)wg_nwk[kl] - 1);
  }
  const int Cl = kl >= 0 ? wg_C[kl] : 0;
  constexpr int kAll = 1 << 30;
  // the windows this wave holds slots of: [kw_lo, kw_hi]
  int kw_lo = kl < 0 ? kAll : kl, kw_hi = kl;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    kw_lo = min(kw_lo, __shfl_xor(kw_lo, o));
    kw_hi = max(kw_hi, __shfl_xor(kw_hi, o));
  }
  kw_lo = __builtin_amdgcn_readfirstlane(kw_lo);
  kw_hi = __builtin_amdgcn_readfirstlane(kw_hi);

  // Q^T as the B operand: lane holds slot l32, head_dim [16 k + 8 g, +8)
  bf16x8 qf[kKsteps];
#pragma unroll
  for (int k = 0; k < kKsteps; ++k)
#pragma unroll
    for (int e = 0; e < 8; ++e) qf[k][e] = (__bf16)0.f;
  if (kl >= 0) {
    const bf16x8* qp =
        reinterpret_cast<const bf16x8*>(reinterpret_cast<const __bf16*>(sq.q) + ((s - sq.base) * H + h) * D);
#pragma unroll
    for (int k = 0; k < kKsteps; ++k) qf[k] = qp[2 * k + g];
  }

  const uint32_t row_bytes = (uint32_t)(Hkv * D * 2);
  // wave copy i of a run of rows starting at row0 (nvalid rows real, the rest
  // repeat the last one): rows i kRPK + lane / kCh16, swizzled as k_off / v_off
  // lay them out, into K at kt and V at vt
  auto copy_one = [&](const char* kbase, const char* vbase, int row0, int nvalid, char* kt, char* vt, int i)
      __attribute__((always_inline)) {
    const int r = i * kRPK + lane / kCh16;
    const int p = lane % kCh16;
    const int f = D == 128 ? (r & 3) : ((r >> 1) & 1);
    const uint32_t rb = (uint32_t)min(r, nvalid - 1 - row0) * row_bytes;
    const char* kb = kbase + (int64_t)row0 * row_bytes;
    const char* vb = vbase + (int64_t)row0 * row_bytes;
    const char* ks = kb + (rb + (uint32_t)((p ^ (r % kCh16)) * 16));
    const char* vs = vb + (rb + (uint32_t)((((p >> 2) ^ f) * 4 + (p & 3)) * 16));
    char* kd = kt + i * 1024;
    char* vd = vt + i * 1024;
    __builtin_amdgcn_global_load_lds(ks, (lds_void*)kd, 16, 0, 0);
    __builtin_amdgcn_global_load_lds(vs, (lds_void*)vd, 16, 0, 0);
  };

  f32x16 oacc[kDtiles];
#pragma unroll
  for (int dt = 0; dt < kDtiles; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[dt][v] = 0.f;
  float m_run = kMinit, l_run = 0.f;
  const int grp = lane >> 4, ri = (lane >> 2) & 3, bq = lane & 3;

  // operands of one 32-row tile (K at kt, V at vt) into registers.  The
  // per-lane LDS offsets are computed once and kept opaque, so that every read
  // is a base, this offset and an immediate (V rows 16 m + 8 hi only add a
  // constant: the swizzle of v_off depends on the row mod 4).
  int kofs[kKsteps], vofs[kDtiles];
#pragma unroll
  for (int k = 0; k < kKsteps; ++k) {
    kofs[k] = k_off<D>(l32, 2 * k + g);
    asm volatile("" : "+v"(kofs[k]));
  }
#pragma unroll
  for (int dt = 0; dt < kDtiles; ++dt) {
    vofs[dt] = v_off<D>(4 * (grp >> 1) + ri, 2 * (32 * dt + 16 * (grp & 1) + 4 * bq));
    asm volatile("" : "+v"(vofs[dt]));
  }
  bf16x8 kop[kKsteps], vop[2 * kDtiles];
  auto read_ops = [&](const char* kt, const char* vt) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kKsteps; ++k) kop[k] = *reinterpret_cast<const bf16x8*>(kt + kofs[k]);
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int dt = 0; dt < kDtiles; ++dt) {
        // keys of B slot v: 16 m + 8 (v/4) + 4 g + v%4
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vt + vofs[dt] + 16 * m * kRB));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vt + vofs[dt] + (16 * m + 8) * kRB));
        vop[m * kDtiles + dt] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
  };
  // one tile from the registers: tile key kk is visible to this lane iff kk <= lim
  auto compute = [&](int lim, bool need_mask) __attribute__((always_inline)) {
    f32x16 sacc;
#pragma unroll
    for (int v = 0; v < 16; ++v) sacc[v] = 0.f;
#pragma unroll
    for (int k = 0; k < kKsteps; ++k) sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[k], qf[k], sacc, 0, 0, 0);
    // sacc[v] = score of slot l32 with tile key 8 (v/4) + 4 g + v%4
    if (need_mask) {
      const int lim_g = lim - 4 * g;
#pragma unroll
      for (int v = 0; v < 16; ++v)
        if ((v >> 2) * 8 + (v & 3) > lim_g) sacc[v] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[v]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));  // with lane ^ 32
    }
    const float m_new = fmaxf(m_run, mx * sc);
    if (__any(m_new - m_run > kLazy)) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < kDtiles; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[dt][v] *= alpha;
      m_run = m_new;
    }
    float psum = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const float p = __builtin_amdgcn_exp2f(fmaf(sacc[v], sc, -m_run));
      sacc[v] = p;
      psum += p;
    }
    l_run += psum;
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      bf16x8 pb;
#pragma unroll
      for (int v = 0; v < 8; ++v) pb[v] = (__bf16)sacc[8 * m + v];
#pragma unroll
      for (int dt = 0; dt < kDtiles; ++dt)
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[m * kDtiles + dt], pb, oacc[dt], 0, 0, 0);
    }
  };
  // over this wave's lanes with a real summary (hi_l != kAll): min and max of hi_l
  auto wave_range = [&](int hi_l, int& hi_min, int& hi_max) __attribute__((always_inline)) {
    int a = hi_l, b = hi_l == kAll ? -1 : hi_l;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      a = min(a, __shfl_xor(a, o));
      b = max(b, __shfl_xor(b, o));
    }
    hi_min = __builtin_amdgcn_readfirstlane(a);
    hi_max = __builtin_amdgcn_readfirstlane(b);
  };
  // the two 32-row tiles of a 64-row cache stage (K at kst, V at vst)
  auto stage_compute = [&](const char* kst, const char* vst, int row0, int hi_l, int hi_min, int hi_max)
      __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int r0 = row0 + j * kBK;
      if (hi_max >= r0) {
        read_ops(kst + j * kTile, vst + j * kTile);
        compute(hi_l - r0, r0 + kBK - 1 > hi_min);
      }
    }
  };
  constexpr int kVm0 = (7 << 4) | (15 << 8);  // s_waitcnt vmcnt(0)

  char* myreg = wave == 0 ? rg0 : wave == 1 ? rg1 : wave == 2 ? rg2 : rg3;
  if constexpr (W == 8)
    if (wave >= 4) myreg = wave == 4 ? rg4 : wave == 5 ? rg5 : wave == 6 ? rg6 : rg7;
  const char* kwin_all = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(d.k) + (int64_t)hk * D);
  const char* vwin_all = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(d.v) + (int64_t)hk * D);
  for (int k0 = 0; k0 < nk;) {
    // run [k0, k1) of windows on sequence b
    // (values read from LDS are the same in every lane: readfirstlane keeps
    // them, and the addresses built from them, in scalar registers)
    const int b = __builtin_amdgcn_readfirstlane(wg_b[k0]);
    int k1 = k0 + 1, cmax = wg_C[k0];
    while (k1 < nk && wg_b[k1] == b) cmax = max(cmax, wg_C[k1++]);
    k1 = __builtin_amdgcn_readfirstlane(k1);
    cmax = __builtin_amdgcn_readfirstlane(cmax);
    // ---- cache phase, shared by the W waves
    __syncthreads();  // every wave is past its window phase: regions 0-3 may be refilled
    if (cmax > 0) {
      const char* kc = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(d.cache_k) +
                                                     ((int64_t)b * d.cache_cap * Hkv + hk) * D);
      const char* vc = reinterpret_cast<const char*>(reinterpret_cast<const __bf16*>(d.cache_v) +
                                                     ((int64_t)b * d.cache_cap * Hkv + hk) * D);
      const int hi_l = kl < 0 ? kAll : (kl >= k0 && kl < k1) ? Cl - 1 : -1;
      int hi_min, hi_max;
      wave_range(hi_l, hi_min, hi_max);
      const int nst = (cmax + 2 * kBK - 1) / (2 * kBK);
      for (int i = wave; i < kStageCopies; i += W) copy_one(kc, vc, 0, cmax, rg0, rg1, i);
      __builtin_amdgcn_s_waitcnt(kVm0);
      __syncthreads();
      for (int t = 0; t < nst; t += 2) {
        if (t + 1 < nst)
          for (int i = wave; i < kStageCopies; i += W) copy_one(kc, vc, (t + 1) * 2 * kBK, cmax, rg2, rg3, i);
        stage_compute(rg0, rg1, t * 2 * kBK, hi_l, hi_min, hi_max);
        __builtin_amdgcn_s_waitcnt(kVm0);
        __syncthreads();
        if (t + 1 >= nst) break;
        if (t + 2 < nst)
          for (int i = wave; i < kStageCopies; i += W) copy_one(kc, vc, (t + 2) * 2 * kBK, cmax, rg0, rg1, i);
        stage_compute(rg2, rg3, (t + 1) * 2 * kBK, hi_l, hi_min, hi_max);
        __builtin_amdgcn_s_waitcnt(kVm0);
        __syncthreads();
      }
    }
    // the last barrier above also ends every read of the stages: the regions
    // belong to their waves again
    // ---- window phase: this wave's windows of the run, on its own, as one
    // stream of 32-row tiles (the next window's first tile is copied while
    // the current window's last tile is computed)
    {
      const int kend = min(k1, kw_hi + 1);
      struct Win {
        int k, ntl, hi_l, hi_min;
        const char* kw;
        const char* vw;
        int nrows;
      };
      // the first window from k on that has rows for this wave's slots
      auto find = [&](int k, Win& x) __attribute__((always_inline)) {
        x.k = kend;
        for (; k < kend; ++k) {
          const int nrows = __builtin_amdgcn_readfirstlane(wg_nwk[k]);
          const int hi_l = kl < 0 ? kAll : kl == k ? pos : -1;
          int hi_min, hi_max;
          wave_range(hi_l, hi_min, hi_max);
          if (hi_max < 0 || nrows <= 0) continue;
          const int64_t tok0 = wg_tok0[k];
          const int64_t tok0_s =
              (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(tok0 >> 32)) << 32) |
                        (uint32_t)__builtin_amdgcn_readfirstlane((int)tok0));
          x.k = k;
          x.ntl = (min(nrows, hi_max + 1) + kBK - 1) / kBK;
          x.hi_l = hi_l;
          x.hi_min = hi_min;
          x.kw = kwin_all + tok0_s * row_bytes;
          x.vw = vwin_all + tok0_s * row_bytes;
          x.nrows = nrows;
          return;
        }
      };
      auto issue_tile = [&](const Win& x, int t) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < kTileCopies; ++i) copy_one(x.kw, x.vw, t * kBK, x.nrows, myreg, myreg + kTile, i);
      };
      Win cur;
      find(max(k0, kw_lo), cur);
      if (cur.k < kend) issue_tile(cur, 0);
      while (cur.k < kend) {
        Win nxt;
        nxt.k = kend;
        for (int t = 0; t < cur.ntl; ++t) {
          __builtin_amdgcn_s_waitcnt(kVm0);  // tile t has landed
          read_ops(myreg, myreg + kTile);
          __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): its operands are in registers
          if (t + 1 < cur.ntl) {
            issue_tile(cur, t + 1);
          } else {
            find(cur.k + 1, nxt);
            if (nxt.k < kend) issue_tile(nxt, 0);
          }
          compute(cur.hi_l - t * kBK, t * kBK + kBK - 1 > cur.hi_min);
        }
        cur = nxt;
      }
    }
    k0 = k1;
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (kl >= 0) {
    const float inv = 1.f / l_tot;
    const int64_t orow = s - sq.base;
    __bf16* op = reinterpret_cast<__bf16*>(sq.o) + (orow * H + h) * D;
#pragma unroll
    for (int dt = 0; dt < kDtiles; ++dt)
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        // oacc[dt][4 v4 + e] = O[slot][32 dt + 8 v4 + 4 g + e]
        uint2 w;
        w.x = focus::pack_bf16x2(oacc[dt][4 * v4 + 0] * inv, oacc[dt][4 * v4 + 1] * inv);
        w.y = focus::pack_bf16x2(oacc[dt][4 * v4 + 2] * inv, oacc[dt][4 * v4 + 3] * inv);
        *reinterpret_cast<uint2*>(op + 32 * dt + 8 * v4 + 4 * g) = w;
      }
    if (g == 0 && sq.lse) sq.lse[orow * H + h] = (m_run + log2f(l_tot)) * kLn2;
  }
}

// ------------------------------------------------- bf16 key-split merge

// Merges the key-split partials of every (listed window, row, head): with
// M = max_s m_s and w_s = 2^(m_s - M), O = sum_s w_s o_s / sum_s w_s l_s and
// LSE = (M + log2 sum_s w_s l_s) ln 2 (m, l in the exp2 domain, as the split
// workgroups left them).  D / 4 lanes per (row, head), four outputs each; the
// windows the attention kernel skipped (rows outside the buffers) are skipped
// here too.
template <int D>
__global__ __launch_bounds__(256) void attn_combine(focus_attn_desc d, Split sp) {
  constexpr int kL = D / 4;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t item = gid / kL;
  const int c = (int)(gid % kL);
  const int H = d.n_heads;
  const int64_t li = item / (sp.rows * H);
  if (li >= sp.nwl) return;
  const int qi = (int)(item / H % sp.rows), h = (int)(item % H);
  const int64_t gw = listed_window(d, li);
  if (gw < 0 || gw >= d.totals.n_windows) return;
  const int T = d.win_ntok[gw];
  const int Cw = d.win_cache_off[gw];
  const int b = d.win_seq[gw];
  const int64_t tok0 = d.win_tok_off[gw] - d.qkv_tok_base;
  if (qi >= T || b < 0 || b >= d.batch || Cw < 0 || Cw > d.cache_cap || tok0 < 0 || tok0 + T > d.qkv_rows) return;
  const int64_t stride = sp.nwl * sp.rows * H;  // (row, head) entries per split
  const int64_t p0 = (li * sp.rows + qi) * H + h;
  float mx = kMinit;
  for (int s = 0; s < sp.n; ++s) mx = fmaxf(mx, sp.pml[2 * (p0 + s * stride)]);
  float l = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s = 0; s < sp.n; ++s) {
    const int64_t p = p0 + s * stride;
    const float w = __builtin_amdgcn_exp2f(sp.pml[2 * p] - mx);
    l += w * sp.pml[2 * p + 1];
    const float4 o = *reinterpret_cast<const float4*>(sp.po + p * D + 4 * c);
    acc.x += w * o.x;
    acc.y += w * o.y;
    acc.z += w * o.z;
    acc.w += w * o.w;
  }
  const float inv = 1.f / l;
  uint2 out;
  out.x = focus::pack_bf16x2(acc.x * inv, acc.y * inv);
  out.y = focus::pack_bf16x2(acc.z * inv, acc.w * inv);
  const int64_t orow = tok0 + qi;
  *reinterpret_cast<uint2*>(reinterpret_cast<__bf16*>(d.o) + (orow * H + h) * D + 4 * c) = out;
  if (c == 0 && d.lse) d.lse[orow * H + h] = (mx + log2f(l)) * kLn2;
}

// ----------------------------------------------------------------- f32 VALU

template <int D, bool KL>
__global__ __launch_bounds__(256) void attn_f32(focus_attn_desc d, float sc, int64_t n_pairs, int QT, SumQ) {
  constexpr int kBQ = 64, kBK = 32, kF4 = D / 4, kPer = D / 16;  // float4 per row / per lane
  __shared__ float4 ks[kBK][kF4];
  __shared__ float4 vs[kBK][kF4];

  const int tid = threadIdx.x;
  const Item it = map_block(blockIdx.x, n_pairs, d.n_heads, QT);
  if (!it.valid) return;
  const int64_t gw = listed_window(d, it.list_idx);
  if (gw < 0 || gw >= d.totals.n_windows) {
    if (tid == 0 && it.qt == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
    return;
  }
  const int T = d.win_ntok[gw];
  const int q0 = it.qt * kBQ;
  if (q0 >= T) return;
  const int Cw = d.win_cache_off[gw];
  const int b = d.win_seq[gw];
  const int64_t tok0 = d.win_tok_off[gw] - d.qkv_tok_base;
  if (b < 0 || b >= d.batch || Cw < 0 || Cw > d.cache_cap || tok0 < 0 || tok0 + T > d.qkv_rows) {
    if (tid == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
    return;
  }
  const int H = d.n_heads, Hkv = d.n_kv_heads, h = it.h;
  const int hk = h / (H / Hkv);
  const int nkeys = Cw + min(T, q0 + kBQ);
  const int qi = q0 + (tid >> 2), sub = tid & 3;
  int kw = 0;
  if constexpr (KL) {
    kw = d.win_kmer ? d.win_kmer[gw] : d.kmer_uniform;
    if (kw < 0) {
      if (tid == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
      return;
    }
  }
  // key j of [cache ; window] is visible to this lane's query
  auto visible = [&](int j) {
    if (!KL) return j < Cw || j - Cw <= qi;
    if (j < Cw) return j == Cw - 1;  // only the carried boundary
    const int u = j - Cw;
    if (u > qi) return false;
    if (kw == 0) return true;
    const bool summary = u % (kw + 1) == kw || u == T - 1;
    return summary || u / (kw + 1) == qi / (kw + 1);
  };
  const int64_t row_f4 = (int64_t)Hkv * kF4;

  float4 qv[kPer], ov[kPer];
  {
    const float4* qp = reinterpret_cast<const float4*>(d.q) + (tok0 + min(qi, T - 1)) * H * kF4 + h * kF4;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      qv[i] = qp[4 * i + sub];
      ov[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  const float4* kwin = reinterpret_cast<const float4*>(d.k) + tok0 * row_f4 + hk * kF4;
  const float4* vwin = reinterpret_cast<const float4*>(d.v) + tok0 * row_f4 + hk * kF4;
  const float4* kcache = reinterpret_cast<const float4*>(d.cache_k) + (int64_t)b * d.cache_cap * row_f4 + hk * kF4;
  const float4* vcache = reinterpret_cast<const float4*>(d.cache_v) + (int64_t)b * d.cache_cap * row_f4 + hk * kF4;

  float m = kMinit, l = 0.f;
  for (int j0 = 0; j0 < nkeys; j0 += kBK) {
    __syncthreads();
    for (int c = tid; c < kBK * kF4; c += 256) {
      const int r = c / kF4, c4 = c % kF4, j = j0 + r;
      float4 kx = make_float4(0.f, 0.f, 0.f, 0.f), vx = kx;
      if (j < Cw) {
        kx = kcache[(int64_t)j * row_f4 + c4];
        vx = vcache[(int64_t)j * row_f4 + c4];
      } else if (j < nkeys) {
        kx = kwin[(int64_t)(j - Cw) * row_f4 + c4];
        vx = vwin[(int64_t)(j - Cw) * row_f4 + c4];
      }
      ks[r][c4] = kx;
      vs[r][c4] = vx;
    }
    __syncthreads();
    const int kend = min(kBK, nkeys - j0);
    for (int kk = 0; kk < kend; ++kk) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const float4 kx = ks[kk][4 * i + sub];
        s = fmaf(qv[i].x, kx.x, s);
        s = fmaf(qv[i].y, kx.y, s);
        s = fmaf(qv[i].z, kx.z, s);
        s = fmaf(qv[i].w, kx.w, s);
      }
      s = focus::sum4(s) * sc;
      const int j = j0 + kk;
      if (visible(j)) {
        const float m_new = fmaxf(m, s);
        const float corr = __builtin_amdgcn_exp2f(m - m_new);
        const float p = __builtin_amdgcn_exp2f(s - m_new);
        l = l * corr + p;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
          const float4 vx = vs[kk][4 * i + sub];
          ov[i].x = fmaf(p, vx.x, ov[i].x * corr);
          ov[i].y = fmaf(p, vx.y, ov[i].y * corr);
          ov[i].z = fmaf(p, vx.z, ov[i].z * corr);
          ov[i].w = fmaf(p, vx.w, ov[i].w * corr);
        }
        m = m_new;
      }
    }
  }
  if (qi < T) {
    const float inv = 1.f / l;
    float4* op = reinterpret_cast<float4*>(d.o) + (tok0 + qi) * H * kF4 + h * kF4;
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      op[4 * i + sub] = make_float4(ov[i].x * inv, ov[i].y * inv, ov[i].z * inv, ov[i].w * inv);
    if (sub == 0 && d.lse) d.lse[(tok0 + qi) * H + h] = (m + log2f(l)) * kLn2;
  }
}

// Query tile rows of a launch: 32 per computing wave (bf16), 64 (f32).
int attn_rows_per_tile(const focus_attn_desc* d) {
  return d->dtype == FOCUS_BF16 ? 32 * (d->mask == FOCUS_MASK_KMER_LOCAL ? kBf16WavesKL : kBf16Waves) : 64;
}

// Key splits of a C(t) bf16 launch (1 = none): as many as still fit the
// (window, head, query tile) items in one round of workgroups, one per CU,
// at most 16 and with at least 8 key tiles per split.
int attn_split_count(const focus_attn_desc* d) {
  if (d->dtype != FOCUS_BF16 || d->mask != FOCUS_MASK_CT || d->n_heads <= 0) return 1;
  const focus_layout_totals& t = d->totals;
  const int64_t nwl = d->win_ids ? d->n_win : t.n_windows;
  if (nwl <= 0 || t.max_window_tokens <= 0 || t.max_window_cache < 0) return 1;
  const int64_t items = nwl * d->n_heads * focus::ceil_div(t.max_window_tokens, attn_rows_per_tile(d));
  const int64_t tiles = focus::ceil_div(t.max_window_cache, 64) + focus::ceil_div(t.max_window_tokens, 64);
  int64_t n = focus::device_cus() / items;
  n = n < tiles / 8 ? n : tiles / 8;
  n = n < 16 ? n : 16;
  return n < 2 ? 1 : (int)n;
}

size_t attn_split_bytes(const focus_attn_desc* d, int n) {
  if (n < 2) return 0;
  const focus_layout_totals& t = d->totals;
  const int64_t nwl = d->win_ids ? d->n_win : t.n_windows;
  const int64_t rows = focus::ceil_div(t.max_window_tokens, attn_rows_per_tile(d)) * attn_rows_per_tile(d);
  return (size_t)n * nwl * rows * d->n_heads * (d->head_dim + 2) * sizeof(float);
}

}  // namespace

extern "C" size_t focus_window_attn_workspace(const focus_attn_desc* d) {
  if (!d) return 0;
  return attn_split_bytes(d, attn_split_count(d));
}

extern "C" focus_status focus_window_attn(const focus_attn_desc* d, focus_stream_t stream) {
  if (!d) return FOCUS_E_NULL;
  if (d->dtype != FOCUS_BF16 && d->dtype != FOCUS_F32) return FOCUS_E_DTYPE;
  if (d->mask != FOCUS_MASK_CT && d->mask != FOCUS_MASK_KMER_LOCAL) return FOCUS_E_ARG;
  if (d->mask == FOCUS_MASK_KMER_LOCAL && !d->win_kmer && d->kmer_uniform < 0) return FOCUS_E_ARG;
  if (d->n_heads <= 0 || d->n_kv_heads <= 0 || d->batch < 0 || d->cache_cap < 0 ||
      d->qkv_rows < 0 || (d->win_ids && d->n_win < 0) || !(d->softmax_scale == d->softmax_scale))
    return FOCUS_E_ARG;
  if (d->head_dim != 64 && d->head_dim != 128) return FOCUS_E_UNSUPPORTED;
  if (d->n_heads % d->n_kv_heads) return FOCUS_E_SHAPE;
  const focus_layout_totals& t = d->totals;
  if (t.n_windows < 0 || t.max_window_tokens < 0 || t.max_window_cache < 0) return FOCUS_E_SHAPE;
  const int64_t nwl = d->win_ids ? d->n_win : t.n_windows;
  if (nwl == 0 || t.max_window_tokens == 0) return FOCUS_OK;
  if (!d->win_seq || !d->win_ntok || !d->win_cache_off || !d->win_tok_off || !d->q || !d->k ||
      !d->v || !d->o)
    return FOCUS_E_NULL;
  if (t.max_window_cache > 0 && (!d->cache_k || !d->cache_v)) return FOCUS_E_NULL;
  if (!focus::aligned16(d->q) || !focus::aligned16(d->k) || !focus::aligned16(d->v) ||
      !focus::aligned16(d->o) || !focus::aligned16(d->cache_k) || !focus::aligned16(d->cache_v) ||
      (reinterpret_cast<uintptr_t>(d->lse) & 3u))
    return FOCUS_E_ARG;
  if (!d->win_ids && t.max_window_cache > d->cache_cap) return FOCUS_E_CAPACITY;

  const float scale = d->softmax_scale > 0.f ? d->softmax_scale : 1.0f / sqrtf((float)d->head_dim);
  const float sc = scale * kLog2e;
  const int64_t n_pairs = nwl * d->n_heads;
  const bool kl = d->mask == FOCUS_MASK_KMER_LOCAL;
  const int waves = kl ? kBf16WavesKL : kBf16Waves;
  const int bq = attn_rows_per_tile(d);
  const int threads = d->dtype == FOCUS_BF16 ? 64 * waves : 256;
  const int64_t qt = focus::ceil_div(t.max_window_tokens, bq);
  // Key split when the workspace allows it (else one workgroup per item).
  Split sp = kNoSplit;
  const int n_split = attn_split_count(d);
  const size_t split_bytes = attn_split_bytes(d, n_split);
  if (n_split > 1 && d->workspace && focus::aligned16(d->workspace) && d->workspace_bytes >= split_bytes) {
    sp.n = n_split;
    sp.rows = qt * bq;
    sp.nwl = nwl;
    sp.po = reinterpret_cast<float*>(d->workspace);
    sp.pml = sp.po + (int64_t)n_split * nwl * sp.rows * d->n_heads * d->head_dim;
  }
  const int64_t blocks = focus::ceil_div(n_pairs, focus::kXcds) * focus::kXcds * qt * sp.n;
  if (blocks * threads >= ((int64_t)1 << 32) || qt > INT32_MAX) return FOCUS_E_SHAPE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const dim3 grid((uint32_t)blocks), block(threads);
#define FOCUS_ATTN_LAUNCH(KERNEL) hipLaunchKernelGGL(KERNEL, grid, block, 0, s, *d, sc, n_pairs, (int)qt, SumQ{})
#define FOCUS_CT_LAUNCH(KERNEL) hipLaunchKernelGGL(KERNEL, grid, block, 0, s, *d, sc, n_pairs, (int)qt, sp)
// k-mer-local bf16: one workgroup per (window, head), looping over its query tiles.
#define FOCUS_KL_LAUNCH(KERNEL, W) hipLaunchKernelGGL(KERNEL, dim3((uint32_t)n_pairs), dim3(64 * (W)), 0, s, *d, sc, n_pairs)
#define FOCUS_F32_LAUNCH(KERNEL) hipLaunchKernelGGL(KERNEL, grid, block, 0, s, *d, sc, n_pairs, (int)qt, SumQ{})
  if (d->dtype == FOCUS_BF16) {
    if (d->head_dim == 128) {
      if (kl) FOCUS_KL_LAUNCH((attn_kl<128, kKlWaves128, kKlStages128>), kKlWaves128); else FOCUS_CT_LAUNCH((attn_ct<128>));
    } else {
      if (kl) FOCUS_KL_LAUNCH((attn_kl<64, 4, 4>), 4); else FOCUS_CT_LAUNCH((attn_ct<64>));
    }
    if (sp.n > 1) {
      const int64_t lanes = sp.nwl * sp.rows * d->n_heads * (d->head_dim / 4);
      const int64_t cblocks = focus::ceil_div(lanes, 256);
      if (cblocks > INT32_MAX) return FOCUS_E_SHAPE;
      if (d->head_dim == 128)
        hipLaunchKernelGGL((attn_combine<128>), dim3((uint32_t)cblocks), dim3(256), 0, s, *d, sp);
      else
        hipLaunchKernelGGL((attn_combine<64>), dim3((uint32_t)cblocks), dim3(256), 0, s, *d, sp);
    }
  } else {
    if (d->head_dim == 128) {
      if (kl) FOCUS_F32_LAUNCH((attn_f32<128, true>)); else FOCUS_F32_LAUNCH((attn_f32<128, false>));
    } else {
      if (kl) FOCUS_F32_LAUNCH((attn_f32<64, true>)); else FOCUS_F32_LAUNCH((attn_f32<64, false>));
    }
  }
#undef FOCUS_ATTN_LAUNCH
#undef FOCUS_CT_LAUNCH
#undef FOCUS_F32_LAUNCH
  return focus::launch_status();
}

// FOCUS adapter attention (Appendix A eq. focus-attn): the summary tokens of
// every listed window attend over [cache ; window] under C(t) or the
// k-mer-local rule (C(t): many windows per workgroup; k-mer-local: one wave
// of 32 summary slots per (window, head)).
extern "C" focus_status focus_adapter_attn(const focus_adapter_desc* a, focus_stream_t stream) {
  if (!a) return FOCUS_E_NULL;
  if (a->dtype != FOCUS_BF16) return a->dtype == FOCUS_F32 ? FOCUS_E_UNSUPPORTED : FOCUS_E_DTYPE;
  if (a->mask != FOCUS_MASK_CT && a->mask != FOCUS_MASK_KMER_LOCAL) return FOCUS_E_ARG;
  if (a->mask == FOCUS_MASK_KMER_LOCAL && !a->win_kmer && a->kmer_uniform < 0) return FOCUS_E_ARG;
  if (a->n_heads <= 0 || a->n_kv_heads <= 0 || a->batch < 0 || a->cache_cap < 0 || a->kv_rows < 0 ||
      a->sum_rows < 0 || (a->win_ids && a->n_win < 0) || !(a->softmax_scale == a->softmax_scale))
    return FOCUS_E_ARG;
  if (a->head_dim != 64 && a->head_dim != 128) return FOCUS_E_UNSUPPORTED;
  if (a->n_heads % a->n_kv_heads) return FOCUS_E_SHAPE;
  const focus_layout_totals& t = a->totals;
  if (t.n_windows < 0 || t.max_window_summaries < 0 || t.max_window_cache < 0) return FOCUS_E_SHAPE;
  const int64_t nwl = a->win_ids ? a->n_win : t.n_windows;
  if (nwl == 0 || t.max_window_summaries == 0) return FOCUS_OK;
  if (!a->win_seq || !a->win_ntok || !a->win_cache_off || !a->win_tok_off || !a->win_nsum ||
      !a->win_sum_off || !a->sum_tok || !a->q_sum || !a->k || !a->v || !a->o_sum)
    return FOCUS_E_NULL;
  if (t.max_window_cache > 0 && (!a->cache_k || !a->cache_v)) return FOCUS_E_NULL;
  if (!focus::aligned16(a->q_sum) || !focus::aligned16(a->k) || !focus::aligned16(a->v) ||
      !focus::aligned16(a->o_sum) || !focus::aligned16(a->cache_k) || !focus::aligned16(a->cache_v) ||
      (reinterpret_cast<uintptr_t>(a->lse_sum) & 3u))
    return FOCUS_E_ARG;
  if (!a->win_ids && t.max_window_cache > a->cache_cap) return FOCUS_E_CAPACITY;

  focus_attn_desc d = {};
  d.totals = t;
  d.dtype = a->dtype;
  d.n_heads = a->n_heads;
  d.n_kv_heads = a->n_kv_heads;
  d.head_dim = a->head_dim;
  d.softmax_scale = a->softmax_scale;
  d.mask = a->mask;
  d.batch = a->batch;
  d.kmer_uniform = a->kmer_uniform;
  d.n_win = a->n_win;
  d.win_ids = a->win_ids;
  d.win_seq = a->win_seq;
  d.win_ntok = a->win_ntok;
  d.win_cache_off = a->win_cache_off;
  d.win_tok_off = a->win_tok_off;
  d.win_kmer = a->win_kmer;
  d.k = a->k;
  d.v = a->v;
  d.qkv_tok_base = a->kv_tok_base;
  d.qkv_rows = a->kv_rows;
  d.cache_k = a->cache_k;
  d.cache_v = a->cache_v;
  d.cache_cap = a->cache_cap;
  d.err = a->err;
  const SumQ sq = {a->win_nsum, a->win_sum_off, a->sum_tok, a->q_sum, a->o_sum, a->lse_sum, a->sum_base, a->sum_rows};

  const float scale = a->softmax_scale > 0.f ? a->softmax_scale : 1.0f / sqrtf((float)a->head_dim);
  const float sc = scale * kLog2e;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool kl = a->mask == FOCUS_MASK_KMER_LOCAL;
  constexpr int kSqWaves = 8;
  if (!kl && t.max_window_summaries <= 32 * kSqWaves) {
    // C(t): G windows per workgroup of kSqWaves waves; whole windows per wave
    // while a window fits one wave's 32 slots
    const int wpw = t.max_window_summaries <= 32 ? (int)(32 / t.max_window_summaries) : 0;
    const int G = wpw > 0 ? kSqWaves * wpw : (int)(32 * kSqWaves / t.max_window_summaries);
    const int64_t n_groups = focus::ceil_div(nwl, G);
    const int64_t n_pairs_g = n_groups * a->n_heads;
    const int64_t blocks_g = focus::ceil_div(n_pairs_g, focus::kXcds) * focus::kXcds;
    if (blocks_g * 64 * kSqWaves >= ((int64_t)1 << 32)) return FOCUS_E_SHAPE;
    const dim3 grid((uint32_t)blocks_g), block(64 * kSqWaves);
    if (a->head_dim == 128)
      hipLaunchKernelGGL((attn_sq_block<128, kSqWaves>), grid, block, 0, s, d, sc, n_pairs_g, nwl, G, wpw, sq);
    else
      hipLaunchKernelGGL((attn_sq_block<64, kSqWaves>), grid, block, 0, s, d, sc, n_pairs_g, nwl, G, wpw, sq);
    return focus::launch_status();
  }
  const int64_t n_pairs = nwl * a->n_heads;
  const int64_t qt = focus::ceil_div(t.max_window_summaries, 32);
  const int64_t blocks = focus::ceil_div(n_pairs, focus::kXcds) * focus::kXcds * qt;
  if (blocks * 64 >= ((int64_t)1 << 32) || qt > INT32_MAX) return FOCUS_E_SHAPE;
  const dim3 grid((uint32_t)blocks), block(64);
#define FOCUS_SQ_LAUNCH(KERNEL) hipLaunchKernelGGL(KERNEL, grid, block, 0, s, d, sc, n_pairs, (int)qt, sq)
  if (a->head_dim == 128) {
    if (kl) FOCUS_SQ_LAUNCH((attn_bf16<128, 1, true, true>)); else FOCUS_SQ_LAUNCH((attn_bf16<128, 1, false, true>));
  } else {
    if (kl) FOCUS_SQ_LAUNCH((attn_bf16<64, 1, true, true>)); else FOCUS_SQ_LAUNCH((attn_bf16<64, 1, false, true>));
  }
#undef FOCUS_SQ_LAUNCH
  return focus::launch_status();
}
