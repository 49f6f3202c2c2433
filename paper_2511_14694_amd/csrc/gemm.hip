// bf16 matrix product on the matrix cores (focus_gemm):
//     C[i, n] = alpha * sum_k A[r(i), k] * B[k, n],   r(i) = a_rows ? a_rows[i] : i
// with float32 accumulation, for the projections around the attention (the
// FOCUS adapter's W_Q / W_K / W_V / W_O of eq. focus-attn, and the layer's
// Q/K/V projection).  a_rows gathers A's rows, so the summary tokens' queries
// are projected without first copying their hidden states.
//
// Two tile shapes (the large one is described at gemm_bf16_wide).  The
// general one: one workgroup = 4 waves = a 128 x 128 tile of C; each wave owns
// 64 x 64 as 2 x 2 blocks of v_mfma_f32_32x32x16_bf16.  K advances 64 at a
// time through LDS, double-buffered, copied global -> LDS directly
// (global_load_lds, 16 B per lane; the A copy gathers rows per lane).  A is
// read with ds_read_b128 from 128-byte rows whose 16-byte chunks are
// XOR-swizzled by row; B (row-major [K, N]) is read k-major with the
// transposing ds_read_b64_tr_b16 from 256-byte rows whose 64-byte granules are
// XOR-swizzled, as the attention's V.
#include "common.h"

namespace {

using focus::bf16x4;
using focus::bf16x8;
using focus::f32x16;

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kBM = 128, kBN = 128, kBKk = 64;   // C tile, K step
constexpr int kThreads = 256;
constexpr int kGroupM = 16;                      // A row stripes per sweep of B
constexpr int kARow = kBKk * 2;                  // bytes per A tile row (128)
constexpr int kBRow = kBN * 2;                   // bytes per B tile row (256)
constexpr int kATile = kBM * kARow;              // 16 KB
constexpr int kBTile = kBKk * kBRow;             // 16 KB

__device__ inline int a_off(int r, int c16) { return r * kARow + ((c16 ^ (r & 7)) << 4); }
__device__ inline int b_off(int r, int byte) { return r * kBRow + (((byte >> 6) ^ (r & 3)) << 6) + (byte & 63); }

// Epilogues: col(c) is evaluated once per column a lane stores; the call
// operator once per element of C with its row, column, float32 value, (kPair)
// the value of its column partner col ^ 1, and the column's col(c).

// C = alpha * A B, stored as bf16 or f32.
struct PlainEpi {
  static constexpr bool kPair = false;
  struct Col {};
  void* c;
  int64_t ldc;
  int32_t c_dtype;
  float alpha;
  __device__ Col col(int64_t) const { return {}; }
  __device__ void operator()(int64_t row, int64_t col, float x, float, Col) const {
    if (c_dtype == FOCUS_BF16)
      reinterpret_cast<__bf16*>(c)[row * ldc + col] = (__bf16)(x * alpha);
    else
      reinterpret_cast<float*>(c)[row * ldc + col] = x * alpha;
  }
  // columns col (even) and col + 1 of a row
  __device__ void pair(int64_t row, int64_t col, float x0, float x1, Col) const {
    const int64_t i = row * ldc + col;
    if (c_dtype == FOCUS_BF16 && !(i & 1)) {
      reinterpret_cast<uint32_t*>(c)[i >> 1] = focus::pack_bf16x2(x0 * alpha, x1 * alpha);
    } else {
      (*this)(row, col, x0, x1, Col{});
      (*this)(row, col + 1, x1, x0, Col{});
    }
  }
};

// The layer's Q/K/V projection: columns [Q heads | K heads | V heads]; RoPE on
// Q and K at the token's position in its augmented stream (the summary tokens
// hold real positions), interleaved pairs (2i, 2i + 1) rotated by
// pos * theta^(-2i/D).  The angle is taken in revolutions,
// pos * theta^(-2i/D) / 2 pi, whose fraction is what the hardware sine and
// cosine need: the per-pair rate is held as a 64-bit binary fraction (from its
// float64 value), so the fraction of pos * rate is the top 32 bits of a
// 32 x 64-bit integer product (two 32-bit multiplies) — exact to 2^-32 of a
// revolution for any position.  K and V rows of summary tokens also go
// straight to their cache row (the compaction pass, fused into the store).
struct QkvEpi {
  static constexpr bool kPair = true;
  struct Col {
    int seg;          // 0 Q, 1 K, 2 V
    int64_t c;        // column inside its tensor row
    bool rot;         // rotated (a Q or K column, theta given)
    bool odd;
    uint32_t r_hi, r_lo;  // revolutions per position of the pair, as a 64-bit fraction
  };
  int32_t H, Hkv, D, batch;
  double log2_theta;   // <= 0: no rotation
  void* q;
  void* k;
  void* v;
  const int32_t* tok_pos;
  const uint8_t* tok_kind;
  const int32_t* tok_kmer;
  const int32_t* tok_win;
  const int32_t* win_seq;
  int64_t tok_base;
  void* cache_k;
  void* cache_v;
  int64_t cache_cap;
  int32_t* cache_len;
  int32_t* err;
  __device__ Col col(int64_t col) const {
    const int64_t qc = (int64_t)H * D, kc = (int64_t)Hkv * D;
    Col r;
    r.seg = col < qc ? 0 : col < qc + kc ? 1 : 2;
    r.c = r.seg == 0 ? col : r.seg == 1 ? col - qc : col - qc - kc;
    const int dd = (int)(r.c % D);
    r.odd = dd & 1;
    r.rot = r.seg < 2 && log2_theta > 0.0;
    const double rev = r.rot ? exp2(-(2.0 * (dd >> 1) / D) * log2_theta) * 0.15915494309189533577 : 0.0;
    const double hi = floor(rev * 4294967296.0);
    r.r_hi = (uint32_t)hi;
    r.r_lo = (uint32_t)((rev * 4294967296.0 - hi) * 4294967296.0);
    return r;
  }
  // fraction of tok_pos[t] * rate, in revolutions, [0, 1]
  __device__ float turn(int64_t t, const Col& cl) const {
    const uint32_t pos = (uint32_t)tok_pos[t];
    const uint32_t f = __umulhi(pos, cl.r_lo) + pos * cl.r_hi;
    return (float)f * 2.3283064365386963e-10f;  // 2^-32
  }
  __device__ void operator()(int64_t row, int64_t, float x, float xp, const Col& cl) const {
    const int64_t t = tok_base + row;
    const int64_t qc = (int64_t)H * D, kc = (int64_t)Hkv * D;
    const int seg = cl.seg;
    const int64_t c = cl.c;
    float y = x;
    if (cl.rot) {
      const float r = turn(t, cl);
      const float sn = __builtin_amdgcn_sinf(r), cs = __builtin_amdgcn_cosf(r);
      // (e, o) -> (e cos - o sin, e sin + o cos); the partner holds the other half
      y = cl.odd ? fmaf(xp, sn, x * cs) : fmaf(-xp, sn, x * cs);
    }
    const __bf16 yb = (__bf16)y;
    __bf16* dst = reinterpret_cast<__bf16*>(seg == 0 ? q : seg == 1 ? k : v);
    dst[row * (seg == 0 ? qc : kc) + c] = yb;
    if (seg > 0 && cache_k && tok_kind[t] == FOCUS_TOK_SUMMARY) {
      const int32_t cr = tok_kmer[t];
      const int32_t b = win_seq[tok_win[t]];
      if (cr < 0 || cr >= cache_cap || b < 0 || b >= batch) {
        focus::raise_err(err, FOCUS_ERR_CAPACITY);
        return;
      }
      __bf16* cdst = reinterpret_cast<__bf16*>(seg == 1 ? cache_k : cache_v);
      cdst[((int64_t)b * cache_cap + cr) * kc + c] = yb;
      if (seg == 1 && c == 0 && cache_len) atomicMax(cache_len + b, cr + 1);
    }
  }
  // columns c (even, described by cl) and c + 1 of a row: one rotation, and
  // both values in one 4-byte store
  __device__ void pair(int64_t row, int64_t, float x0, float x1, const Col& cl) const {
    const int64_t t = tok_base + row;
    const int64_t qc = (int64_t)H * D, kc = (int64_t)Hkv * D;
    const int seg = cl.seg;
    const int64_t c = cl.c;
    float y0 = x0, y1 = x1;
    if (cl.rot) {
      const float r = turn(t, cl);
      const float sn = __builtin_amdgcn_sinf(r), cs = __builtin_amdgcn_cosf(r);
      y0 = fmaf(-x1, sn, x0 * cs);
      y1 = fmaf(x0, sn, x1 * cs);
    }
    const uint32_t w = focus::pack_bf16x2(y0, y1);
    uint32_t* dst = reinterpret_cast<uint32_t*>(seg == 0 ? q : seg == 1 ? k : v);
    dst[(row * (seg == 0 ? qc : kc) + c) >> 1] = w;
    if (seg > 0 && cache_k && tok_kind[t] == FOCUS_TOK_SUMMARY) {
      const int32_t cr = tok_kmer[t];
      const int32_t b = win_seq[tok_win[t]];
      if (cr < 0 || cr >= cache_cap || b < 0 || b >= batch) {
        focus::raise_err(err, FOCUS_ERR_CAPACITY);
        return;
      }
      uint32_t* cdst = reinterpret_cast<uint32_t*>(seg == 1 ? cache_k : cache_v);
      cdst[(((int64_t)b * cache_cap + cr) * kc + c) >> 1] = w;
      if (seg == 1 && c == 0 && cache_len) atomicMax(cache_len + b, cr + 1);
    }
  }
};

template <class Epi>
__global__ __launch_bounds__(kThreads, 2) void gemm_bf16(focus_gemm_desc d, int64_t m_tiles, Epi epi) {
  __shared__ __attribute__((aligned(1024))) char abuf0[kATile], abuf1[kATile];
  __shared__ __attribute__((aligned(1024))) char bbuf0[kBTile], bbuf1[kBTile];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
  // Grouped order: kGroupM row stripes of A sweep every column tile before the
  // next group starts, so A is read from HBM about once and B (the weights)
  // stays in the last-level cache.
  const int64_t n_tiles = d.n / kBN, per_group = (int64_t)kGroupM * n_tiles;
  const int64_t grp0 = blockIdx.x / per_group, in_grp = blockIdx.x % per_group;
  const int64_t gm_rows = min((int64_t)kGroupM, m_tiles - grp0 * kGroupM);
  const int64_t mt = grp0 * kGroupM + in_grp % gm_rows, nt = in_grp / gm_rows;
  const int64_t m0 = mt * kBM, n0 = nt * kBN;
  const int wm = (wave & 1) * 64, wn = (wave >> 1) * 64;   // this wave's 64 x 64 in the tile

  // Copy plan: A tile = 16 wave-loads of 1 KB (8 rows x 128 B), 4 per wave;
  // B tile = 16 wave-loads (4 rows x 256 B), 4 per wave.  Lane p of a row
  // fetches the global chunk the swizzled layout keeps at its slot.
  const char* A = reinterpret_cast<const char*>(d.a);
  const char* B = reinterpret_cast<const char*>(d.b);
  const int64_t a_ld = d.lda * 2, b_ld = d.ldb * 2;
  const char* a_src[4];
  uint32_t b_col[4];
  int brow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = (wave * 4 + i) * 8 + (lane >> 3), p = lane & 7;   // A tile row, 16-B slot
    const int64_t gm = min(m0 + r, d.m - 1);                         // ragged M: repeat the last row
    int64_t ar = d.a_rows ? d.a_rows[gm] : gm;
    if (ar < 0 || ar >= d.a_nrows) {
      focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
      ar = 0;
    }
    a_src[i] = A + ar * a_ld + ((p ^ (r & 7)) << 4);
    brow[i] = (wave * 4 + i) * 4 + (lane >> 4);                      // B tile row
    const int pb = lane & 15;                                        // its 16-B slot
    b_col[i] = (uint32_t)((((pb >> 2) ^ (brow[i] & 3)) * 4 + (pb & 3)) * 16);
  }

  auto issue = [&](int64_t k0, char* ab, char* bb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const char* ga = a_src[i] + k0 * 2;
      __builtin_amdgcn_global_load_lds(ga, (lds_void*)(ab + (wave * 4 + i) * 1024), 16, 0, 0);
      const char* gb = B + (k0 + brow[i]) * b_ld + n0 * 2 + b_col[i];
      __builtin_amdgcn_global_load_lds(gb, (lds_void*)(bb + (wave * 4 + i) * 1024), 16, 0, 0);
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // transposing-read coordinates: lane = 16 * grp + 4 * ri + bq
  const int grp = lane >> 4, ri = (lane >> 2) & 3, bq = lane & 3;
  auto compute = [&](const char* ab, const char* bb) {
#pragma unroll
    for (int s = 0; s < kBKk / 16; ++s) {
      bf16x8 af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = *reinterpret_cast<const bf16x8*>(ab + a_off(wm + 32 * i + l32, 2 * s + g));
      // B operand in the natural k order of the A operand: lane (n, g) holds
      // B[16 s + 8 g + e][n], e = 0..7.  Each transposing read gives a lane one
      // column of the 4 rows its quad points at: rows 16 s + 8 g + ri (e < 4),
      // then 4 further down (e >= 4).
      const int kb = 16 * s + 8 * (grp >> 1) + ri;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col_byte = 2 * (wn + 32 * j + 16 * (grp & 1) + 4 * bq);
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(bb + b_off(kb, col_byte)));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(bb + b_off(kb + 4, col_byte)));
        bf[j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
  };

  const int64_t nk = d.k / kBKk;
  issue(0, abuf0, bbuf0);
  __syncthreads();
  for (int64_t t = 0; t < nk; t += 2) {
    if (t + 1 < nk) issue((t + 1) * kBKk, abuf1, bbuf1);
    compute(abuf0, bbuf0);
    __syncthreads();
    if (t + 1 >= nk) break;
    if (t + 2 < nk) issue((t + 2) * kBKk, abuf0, bbuf0);
    compute(abuf1, bbuf1);
    __syncthreads();
  }

  // acc[i][j][v] = C[m0 + wm + 32 i + 8 (v / 4) + 4 g + v % 4][n0 + wn + 32 j + l32];
  // column col ^ 1 sits in lane ^ 1 (DPP quad swap, taken before any branch)
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int64_t col = n0 + wn + 32 * j + l32;
    const typename Epi::Col cl = epi.col(col);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t row = m0 + wm + 32 * i + 8 * (v >> 2) + 4 * g + (v & 3);
        const float x = acc[i][j][v];
        const float xp = Epi::kPair ? focus::dpp_xor1(x) : 0.f;
        if (row < d.m) epi(row, col, x, xp, cl);
      }
  }
}


// Large products (N a multiple of 256, M >= 256, K a multiple of 128): one
// workgroup = 8 waves = a 256 x 256 tile of C, each wave 128 x 64 as 4 x 2
// blocks of v_mfma_f32_32x32x16_bf16.  Per 16-deep k-step a wave reads 4 A and
// 2 B operands from LDS for 8 MFMAs (the 128 x 128 tile's 64 x 64 waves read
// 2 + 2 for 4); two waves per SIMD, so one's LDS reads and barrier waits
// overlap the other's MFMAs (four waves of 128 x 128, one per SIMD, ran 7 %
// slower).  K advances 32 at a time through four
// LDS stages (A 256 x 64 B + B 32 x 512 B = 32 KB each): the copies of step
// t + 3 start in step t, so a copy has three steps to land, and a step ends on
// a partial wait (only the two younger steps' copies in flight) plus a barrier.
// A rows are 64 bytes: 16-byte chunk c of row r sits at c ^ ((r / 4) mod 4), so
// the 8 rows one quarter-wave reads fall into distinct bank groups; B rows are
// 512 bytes, 64-byte granules XOR-swizzled by (row mod 4) as above.
constexpr int kBM2 = 256, kBN2 = 256, kBK2 = 32;
constexpr int kARow2 = kBK2 * 2;                 // bytes per A tile row (64)
constexpr int kBRow2 = kBN2 * 2;                 // bytes per B tile row (512)
constexpr int kATile2 = kBM2 * kARow2;           // 16 KB
constexpr int kBTile2 = kBK2 * kBRow2;           // 16 KB
constexpr int kStage2 = kATile2 + kBTile2;       // A then B
constexpr int kThreadsWide = 512;

template <class Epi>
__global__ __launch_bounds__(kThreadsWide, 1) void gemm_bf16_wide(focus_gemm_desc d, int64_t m_tiles, Epi epi) {
  // One array per stage: the compiler tracks the copies in flight per array.
  __shared__ __attribute__((aligned(1024))) char st0[kStage2], st1[kStage2], st2[kStage2], st3[kStage2];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
  const int64_t n_tiles = d.n / kBN2, per_group = (int64_t)kGroupM * n_tiles;
  const int64_t grp0 = blockIdx.x / per_group, in_grp = blockIdx.x % per_group;
  const int64_t gm_rows = min((int64_t)kGroupM, m_tiles - grp0 * kGroupM);
  const int64_t mt = grp0 * kGroupM + in_grp % gm_rows, nt = in_grp / gm_rows;
  const int64_t m0 = mt * kBM2, n0 = nt * kBN2;
  const int wm = (wave & 1) * 128, wn = (wave >> 1) * 64;  // this wave's 128 x 64 in the tile

  // Copy plan: A tile = 16 wave-loads of 1 KB (16 rows x 64 B), 2 per wave;
  // B tile = 16 wave-loads (2 rows x 512 B), 2 per wave.  Lane p of a row
  // fetches the global chunk the swizzled layout keeps at its slot.
  const char* A = reinterpret_cast<const char*>(d.a);
  const char* B = reinterpret_cast<const char*>(d.b);
  const int64_t a_ld = d.lda * 2, b_ld = d.ldb * 2;
  const char* a_src[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (wave * 2 + i) * 16 + (lane >> 2), p = lane & 3;  // A tile row, 16-B slot
    const int64_t gm = min(m0 + r, d.m - 1);                         // ragged M: repeat the last row
    int64_t ar = d.a_rows ? d.a_rows[gm] : gm;
    if (ar < 0 || ar >= d.a_nrows) {
      focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
      ar = 0;
    }
    a_src[i] = A + ar * a_ld + ((p ^ ((r >> 2) & 3)) << 4);
  }
  // B tile row of wave-load i: (wave * 2 + i) * 2 + lane / 32 (row mod 4
  // alternates with i); slot lane % 32
  const int pb = lane & 31;
  const int brow0 = wave * 4 + (lane >> 5);
  const uint32_t b_col0 = (uint32_t)((((pb >> 2) ^ (brow0 & 3)) * 4 + (pb & 3)) * 16);
  const uint32_t b_col1 = (uint32_t)((((pb >> 2) ^ ((brow0 + 2) & 3)) * 4 + (pb & 3)) * 16);
  const char* b_src = B + (int64_t)brow0 * b_ld + n0 * 2;

  // wave copy pair i (A rows and B rows) of the step at k0 into a stage
  auto issue_pair = [&](int64_t k0, char* stage, int i) {
    __builtin_amdgcn_global_load_lds(a_src[i] + k0 * 2, (lds_void*)(stage + (wave * 2 + i) * 1024), 16, 0, 0);
    const char* gb = b_src + (k0 + 2 * i) * b_ld + ((i & 1) ? b_col1 : b_col0);
    __builtin_amdgcn_global_load_lds(gb, (lds_void*)(stage + kATile2 + (wave * 2 + i) * 1024), 16, 0, 0);
  };
  auto issue = [&](int64_t k0, char* stage) {
#pragma unroll
    for (int i = 0; i < 2; ++i) issue_pair(k0, stage, i);
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // Computes the step in `stage` and starts the copies of the step at k_nxt
  // into `nxt`, one pair after every 4 MFMAs of the first k-step: a wave that
  // sends all its copies at once stalls until the address unit has taken them.
  auto compute = [&](const char* stage, int64_t k_nxt, char* nxt) {
    // Per-lane LDS offsets, rebuilt each step behind an empty asm statement
    // (not hoisted per stage; one offset from each stage, so the compiler can
    // tell the stage being read from the ones being filled).
    //   A: row wm + 32 i + l32, chunk 2 s + g at (2 s + g) ^ ((l32 / 4) mod 4)
    //   B: transposing read of rows 16 s + 8 (grp / 2) + ri (+ 4), byte
    //      2 (wn + 32 j + 16 (grp & 1) + 4 bq), granule ((wn / 32 + j) ^ ri)
    const int grp = lane >> 4, ri = (lane >> 2) & 3, bq = lane & 3;
    int ao[2], bo[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      ao[s] = (wm + l32) * kARow2 + (((2 * s + g) ^ ((l32 >> 2) & 3)) << 4);
      asm volatile("" : "+v"(ao[s]));
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      bo[j] = kATile2 + (8 * (grp >> 1) + ri) * kBRow2 + ((((wn >> 5) + j) ^ ri) << 6) + 32 * (grp & 1) + 8 * bq;
      asm volatile("" : "+v"(bo[j]));
    }
    // Operands of k-step s + 1 are read while the 8 MFMAs of k-step s run.
    bf16x8 af[2][4], bf[2][2];
    auto load = [&](int s, int buf) {
#pragma unroll
      for (int i = 0; i < 4; ++i) af[buf][i] = *reinterpret_cast<const bf16x8*>(stage + (ao[s] + 32 * i * kARow2));
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(stage + (bo[j] + 16 * s * kBRow2)));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(stage + (bo[j] + (16 * s + 4) * kBRow2)));
        bf[buf][j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    };
    load(0, 0);
    load(1, 1);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s][i], bf[s][j], acc[i][j], 0, 0, 0);
        if (s == 0 && (i & 1)) {
          __builtin_amdgcn_sched_barrier(0);
          issue_pair(k_nxt, nxt, i >> 1);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };

  // Step t: start the copies of step t + 3 (past the end, of the last step
  // again: every step starts the same number, and that stage is not read
  // again), compute step t, wait until step t + 1 has landed, barrier.
  const int64_t nk = d.k / kBK2;
  auto end_step = [&]() {
    constexpr int kVm = 2 * 4;  // two younger steps of 4 wave copies: vmcnt(8) expcnt(7) lgkmcnt(0)
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt((kVm & 15) | ((kVm >> 4) << 14) | (7 << 4) | (0 << 8));
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
  };
  auto step = [&](int64_t t, const char* cur, char* nxt) {
    compute(cur, min(t + 3, nk - 1) * kBK2, nxt);
    end_step();
  };
  issue(0, st0);
  issue(min((int64_t)1, nk - 1) * kBK2, st1);
  issue(min((int64_t)2, nk - 1) * kBK2, st2);
  __syncthreads();
  // nk is a multiple of 4 (a partial round would need exits inside the
  // loop, around which the compiler moves the accumulators out of the AGPRs)
  for (int64_t t = 0; t < nk; t += 4) {
    step(t, st0, st3);
    step(t + 1, st1, st0);
    step(t + 2, st2, st1);
    step(t + 3, st3, st2);
  }
  __builtin_amdgcn_s_waitcnt(0);  // no copy into LDS outlives the block
  __syncthreads();                // and no wave still reads a stage

  // Epilogue through LDS: each wave parks 64 x 64 of its float32 results
  // (half its tile) in half a stage, then walks them two rows at a time (one
  // per half-wave), a lane taking two adjacent columns (a RoPE pair): the
  // epilogue code appears once and every store of a row is contiguous.
  // Same-wave LDS accesses complete in order, so no barrier is needed between
  // the writes and the reads.
  //   acc[i][j][v] = C[m0 + wm + 32 i + 8 (v / 4) + 4 g + v % 4][n0 + wn + 32 j + l32]
  float* ct = reinterpret_cast<float*>((wave >> 1) == 0 ? st0 : (wave >> 1) == 1 ? st1 : (wave >> 1) == 2 ? st2 : st3) +
              (wave & 1) * 64 * 64;
  const int half = lane >> 5, cl32 = lane & 31;
  const int64_t c0 = n0 + wn + 2 * cl32;
  const typename Epi::Col cl0 = epi.col(c0);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
#pragma unroll
    for (int i2 = 0; i2 < 2; ++i2)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          ct[(32 * i2 + 8 * (v >> 2) + 4 * g + (v & 3)) * 64 + 32 * j + l32] = acc[2 * h + i2][j][v];
    const int64_t rows = min((int64_t)64, d.m - (m0 + wm + 64 * h));
    for (int r = half; r < rows; r += 2) {
      const float2 x = reinterpret_cast<const float2*>(ct)[r * 32 + cl32];
      const int64_t row = m0 + wm + 64 * h + r;
      epi.pair(row, c0, x.x, x.y, cl0);
    }
  }
}

// Launch C = A B (+ epilogue) with the wide tile where N and M allow.
template <class Epi>
focus_status launch_gemm(const focus_gemm_desc& d, const Epi& epi, focus_stream_t stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (d.n % kBN2 == 0 && d.m >= kBM2 && d.k % (4 * kBK2) == 0) {
    const int64_t m_tiles = focus::ceil_div(d.m, kBM2), n_tiles = d.n / kBN2;
    if (m_tiles * n_tiles > INT32_MAX) return FOCUS_E_SHAPE;
    hipLaunchKernelGGL(gemm_bf16_wide<Epi>, dim3((uint32_t)(m_tiles * n_tiles)), dim3(kThreadsWide), 0, s, d, m_tiles, epi);
  } else {
    const int64_t m_tiles = focus::ceil_div(d.m, kBM), n_tiles = d.n / kBN;
    if (m_tiles * n_tiles > INT32_MAX) return FOCUS_E_SHAPE;
    hipLaunchKernelGGL(gemm_bf16<Epi>, dim3((uint32_t)(m_tiles * n_tiles)), dim3(kThreads), 0, s, d, m_tiles, epi);
  }
  return focus::launch_status();
}
}  // namespace

extern "C" focus_status focus_gemm(const focus_gemm_desc* d, focus_stream_t stream) {
  if (!d) return FOCUS_E_NULL;
  if (d->c_dtype != FOCUS_BF16 && d->c_dtype != FOCUS_F32) return FOCUS_E_DTYPE;
  if (d->m < 0 || d->n < 0 || d->k < 0 || !(d->alpha == d->alpha)) return FOCUS_E_ARG;
  if (d->m == 0 || d->n == 0) return FOCUS_OK;
  if (d->k == 0 || d->k % kBKk || d->n % kBN) return FOCUS_E_UNSUPPORTED;
  if (!d->a || !d->b || !d->c) return FOCUS_E_NULL;
  if (d->lda < d->k || d->ldb < d->n || d->ldc < d->n || d->lda % 8 || d->ldb % 8) return FOCUS_E_ARG;
  if (d->a_nrows < (d->a_rows ? 1 : d->m)) return FOCUS_E_ARG;
  if (!focus::aligned16(d->a) || !focus::aligned16(d->b) || (reinterpret_cast<uintptr_t>(d->c) & 3u) ||
      (reinterpret_cast<uintptr_t>(d->a_rows) & 7u))
    return FOCUS_E_ARG;
  const PlainEpi epi = {d->c, d->ldc, d->c_dtype, d->alpha};
  return launch_gemm(*d, epi, stream);
}

extern "C" focus_status focus_qkv_project(const focus_qkv_desc* q, focus_stream_t stream) {
  if (!q) return FOCUS_E_NULL;
  if (q->dtype != FOCUS_BF16) return q->dtype == FOCUS_F32 ? FOCUS_E_UNSUPPORTED : FOCUS_E_DTYPE;
  if (q->n_heads <= 0 || q->n_kv_heads <= 0 || q->d_model <= 0 || q->batch < 0 || q->n_rows < 0 ||
      q->tok_base < 0 || !(q->rope_theta == q->rope_theta) || (q->rope_theta > 0.f && q->rope_theta <= 1.f))
    return FOCUS_E_ARG;
  if (q->head_dim != 64 && q->head_dim != 128) return FOCUS_E_UNSUPPORTED;
  if (q->n_heads % q->n_kv_heads) return FOCUS_E_SHAPE;
  const int64_t n = ((int64_t)q->n_heads + 2 * q->n_kv_heads) * q->head_dim;
  if (n % kBN || q->d_model % kBKk) return FOCUS_E_UNSUPPORTED;
  if (q->tok_base + q->n_rows > q->totals.n_tokens) return FOCUS_E_SHAPE;
  if (q->n_rows == 0) return FOCUS_OK;
  if (!q->hidden || !q->w_qkv || !q->q || !q->k || !q->v || !q->tok_pos) return FOCUS_E_NULL;
  if (q->cache_k && (!q->cache_v || !q->tok_kind || !q->tok_kmer || !q->tok_win || !q->win_seq))
    return FOCUS_E_NULL;
  if (q->cache_k && q->cache_cap < q->totals.max_cache_per_seq && q->tok_base == 0 && q->n_rows == q->totals.n_tokens)
    return FOCUS_E_CAPACITY;
  if (!focus::aligned16(q->hidden) || !focus::aligned16(q->w_qkv)) return FOCUS_E_ARG;
  // pairs of bf16 columns are stored as one 4-byte word
  if ((reinterpret_cast<uintptr_t>(q->q) | reinterpret_cast<uintptr_t>(q->k) | reinterpret_cast<uintptr_t>(q->v) |
       reinterpret_cast<uintptr_t>(q->cache_k) | reinterpret_cast<uintptr_t>(q->cache_v)) & 3u)
    return FOCUS_E_ARG;
  focus_gemm_desc g = {};
  g.m = q->n_rows;
  g.n = n;
  g.k = q->d_model;
  g.a = q->hidden;
  g.lda = q->d_model;
  g.a_nrows = q->n_rows;
  g.b = q->w_qkv;
  g.ldb = n;
  g.err = q->err;
  QkvEpi e;
  e.H = q->n_heads;
  e.Hkv = q->n_kv_heads;
  e.D = q->head_dim;
  e.batch = q->batch;
  e.log2_theta = q->rope_theta > 0.f ? log2((double)q->rope_theta) : 0.0;
  e.q = q->q;
  e.k = q->k;
  e.v = q->v;
  e.tok_pos = q->tok_pos;
  e.tok_kind = q->tok_kind;
  e.tok_kmer = q->tok_kmer;
  e.tok_win = q->tok_win;
  e.win_seq = q->win_seq;
  e.tok_base = q->tok_base;
  e.cache_k = q->cache_k;
  e.cache_v = q->cache_v;
  e.cache_cap = q->cache_cap;
  e.cache_len = q->cache_len;
  e.err = q->err;
  return launch_gemm(g, e, stream);
}
