// Summary-token layout and index metadata (focus_layout).
//
// Appendix A cuts each sequence of L bases into windows of W bases (the last
// one clipped), and inserts B_w = ceil(n_w / k_w) summary tokens into window w,
// one at the right boundary of every k_w-base k-mer (Section 3.2), a trailing
// partial k-mer included.  The cache rows window w sees are the C_w summaries
// retained from the earlier windows of its sequence.
//
// Two launches:
//   layout_windows  one workgroup; scans over sequences and windows (the number
//                   of windows is small: 1 000 per megabase at W = 1 000)
//   layout_tokens   four augmented tokens per thread; a closed form places a
//                   token inside its window: with groups of k_w bases + 1
//                   summary, token i of the window is in group i / (k_w + 1),
//                   and it is that group's summary when its offset equals the
//                   group's base count (k_w, or the remainder for the last group)
#include "common.h"

namespace {

constexpr int kScanThreads = 1024;
constexpr int kScanWaves = kScanThreads / 64;
constexpr int kTokThreads = 256;
constexpr int kTokPerThread = 4;

// Exclusive scan of one int64 per thread across the workgroup; *total gets the
// workgroup sum.  Every thread must call it.
__device__ int64_t block_exclusive_scan(int64_t x, int64_t* total) {
  __shared__ int64_t wsum[kScanWaves];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int64_t incl = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int64_t y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (lane == 63) wsum[wid] = incl;
  __syncthreads();
  if (wid == 0) {
    int64_t s = lane < kScanWaves ? wsum[lane] : 0;
#pragma unroll
    for (int off = 1; off < kScanWaves; off <<= 1) {
      int64_t y = __shfl_up(s, off, 64);
      if (lane >= off) s += y;
    }
    if (lane < kScanWaves) wsum[lane] = s;
  }
  __syncthreads();
  const int64_t base = wid > 0 ? wsum[wid - 1] : 0;
  *total = wsum[kScanWaves - 1];
  __syncthreads();
  return base + incl - x;
}

__device__ inline int64_t ceil_div_d(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Largest b in [0, batch) with cu[b] <= x (sequences with no windows share
// their cu value with the next sequence, which is the one that owns x).
__device__ int32_t owner_seq(const int64_t* cu, int32_t batch, int64_t x) {
  int32_t lo = 0, hi = batch - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= x) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ inline int32_t window_kmer(const focus_layout_desc& d, int64_t gw) {
  return d.kmer ? d.kmer[gw] : d.kmer_uniform;
}

__global__ __launch_bounds__(kScanThreads) void layout_windows(focus_layout_desc d) {
  const int tid = threadIdx.x;
  const int64_t W = d.window_nt;
  __shared__ int bad;
  if (tid == 0) bad = 0;
  __syncthreads();

  // Windows per sequence -> cu_windows.
  int64_t carry = 0;
  for (int64_t b0 = 0; b0 < d.batch; b0 += kScanThreads) {
    const int64_t b = b0 + tid;
    int64_t L = b < d.batch ? d.seq_nt[b] : 0;
    if (L < 0) { bad = 1; L = 0; }
    int64_t tot;
    const int64_t ex = block_exclusive_scan(ceil_div_d(L, W), &tot);
    if (b < d.batch) d.cu_windows[b] = carry + ex;
    carry += tot;
  }
  if (tid == 0) d.cu_windows[d.batch] = carry;
  const int64_t NW = carry;
  __syncthreads();
  if (NW != d.totals.n_windows || bad) {
    // Leave every planned window empty so that layout_tokens writes nothing.
    for (int64_t gw = tid; gw < d.totals.n_windows; gw += kScanThreads) d.win_ntok[gw] = 0;
    if (tid == 0) focus::raise_err(d.err, FOCUS_ERR_PLAN);
    return;
  }

  // Per-window sizes and the three running offsets (tokens, summaries, bases).
  int64_t tok_carry = 0, sum_carry = 0, base_carry = 0;
  for (int64_t w0 = 0; w0 < NW; w0 += kScanThreads) {
    const int64_t gw = w0 + tid;
    const bool valid = gw < NW;
    int32_t b = 0;
    int64_t n = 0, B = 0;
    if (valid) {
      b = owner_seq(d.cu_windows, d.batch, gw);
      const int64_t w = gw - d.cu_windows[b];
      const int64_t L = d.seq_nt[b];
      n = (L - w * W) < W ? (L - w * W) : W;
      int64_t k = window_kmer(d, gw);
      if (k < 0) { bad = 1; k = 0; }
      B = k > 0 ? ceil_div_d(n, k) : 0;
      if (n + B > d.totals.max_window_tokens) bad = 1;
    }
    int64_t tot_t, tot_s, tot_n;
    const int64_t ex_t = block_exclusive_scan(n + B, &tot_t);
    const int64_t ex_s = block_exclusive_scan(B, &tot_s);
    const int64_t ex_n = block_exclusive_scan(n, &tot_n);
    if (valid) {
      d.win_seq[gw] = b;
      d.win_nt[gw] = (int32_t)n;
      d.win_nsum[gw] = (int32_t)B;
      d.win_ntok[gw] = (int32_t)(n + B);
      d.win_tok_off[gw] = tok_carry + ex_t;
      d.win_sum_off[gw] = sum_carry + ex_s;
      d.win_base_off[gw] = base_carry + ex_n;
    }
    // Windows of one workgroup see each other's global writes after a barrier.
    __syncthreads();
    if (valid) d.win_cache_off[gw] = (int32_t)(d.win_sum_off[gw] - d.win_sum_off[d.cu_windows[b]]);
    tok_carry += tot_t;
    sum_carry += tot_s;
    base_carry += tot_n;
    __syncthreads();
  }
  if (tok_carry != d.totals.n_tokens || sum_carry != d.totals.n_summaries || bad) {
    for (int64_t gw = tid; gw < NW; gw += kScanThreads) d.win_ntok[gw] = 0;
    if (tid == 0) focus::raise_err(d.err, FOCUS_ERR_PLAN);
  }

  for (int64_t b = tid; b < d.batch; b += kScanThreads) {
    const int64_t fw = d.cu_windows[b];
    d.cu_tokens[b] = fw < NW ? d.win_tok_off[fw] : tok_carry;
    d.cu_summaries[b] = fw < NW ? d.win_sum_off[fw] : sum_carry;
  }
  if (tid == 0) {
    d.cu_tokens[d.batch] = tok_carry;
    d.cu_summaries[d.batch] = sum_carry;
  }
}

// Token i of window gw (i < T_w checked by the caller).
__device__ inline void layout_token(const focus_layout_desc& d, int64_t gw, int64_t i) {
  const int64_t n = d.win_nt[gw];
  const int64_t B = d.win_nsum[gw];
  const int64_t tok = d.win_tok_off[gw] + i;
  if (tok >= d.totals.n_tokens) {
    focus::raise_err(d.err, FOCUS_ERR_PLAN);
    return;
  }
  int64_t k = window_kmer(d, gw);
  if (k < 0) k = 0;

  bool summary = false;
  int64_t group = -1, base_in_win = i;
  if (k > 0) {
    group = i / (k + 1);
    const int64_t r = i - group * (k + 1);
    const int64_t group_bases = group < B - 1 ? k : n - (B - 1) * k;
    summary = r == group_bases;
    base_in_win = group * k + r;
  }
  const int32_t b = d.win_seq[gw];
  if (b < 0 || b >= d.batch) {
    focus::raise_err(d.err, FOCUS_ERR_PLAN);
    return;
  }
  d.tok_pos[tok] = (int32_t)(d.win_tok_off[gw] - d.cu_tokens[b] + i);
  d.tok_win[tok] = (int32_t)gw;
  d.tok_kind[tok] = summary ? FOCUS_TOK_SUMMARY : FOCUS_TOK_BASE;
  const int64_t base = summary ? -1 : d.win_base_off[gw] + base_in_win;
  d.tok_base[tok] = base;
  d.tok_kmer[tok] = k > 0 ? (int32_t)(d.win_cache_off[gw] + group) : -1;
  if (summary) {
    const int64_t s = d.win_sum_off[gw] + group;
    if (s < d.totals.n_summaries) d.sum_tok[s] = tok;
    else focus::raise_err(d.err, FOCUS_ERR_PLAN);
  }
  if (d.bases && d.token_ids) d.token_ids[tok] = summary ? d.summary_token_id : (int32_t)d.bases[base];
  if (d.tok_next_base) {
    // pi(t): the window's bases up to and including t, plus its first base
    // (a summary follows the bases of its k-mer); -1 past the sequence's end
    const int64_t end = d.win_base_off[d.cu_windows[b]] + d.seq_nt[b];
    const int64_t nb = d.win_base_off[gw] + base_in_win + (summary ? 0 : 1);
    d.tok_next_base[tok] = nb < end ? nb : -1;
  }
}

// One workgroup per (window, tile of kTokPerThread * kTokThreads tokens); a
// thread places kTokPerThread tokens, kTokThreads apart, so the window's
// descriptor loads are paid once per tile rather than once per token.
__global__ __launch_bounds__(kTokThreads) void layout_tokens(focus_layout_desc d, int32_t tiles) {
  const int64_t gw = blockIdx.x / tiles;
  if (gw >= d.totals.n_windows) return;
  const int64_t T = d.win_ntok[gw];
  const int64_t i0 = (int64_t)(blockIdx.x % tiles) * kTokPerThread * kTokThreads + threadIdx.x;
#pragma unroll
  for (int r = 0; r < kTokPerThread; ++r) {
    const int64_t i = i0 + (int64_t)r * kTokThreads;
    if (i < T) layout_token(d, gw, i);
  }
}

}  // namespace

extern "C" focus_status focus_layout(const focus_layout_desc* d, focus_stream_t stream) {
  if (!d) return FOCUS_E_NULL;
  const focus_layout_totals& t = d->totals;
  if (d->batch < 0 || d->window_nt <= 0 || (!d->kmer && d->kmer_uniform < 0)) return FOCUS_E_ARG;
  if (t.n_windows < 0 || t.n_tokens < 0 || t.n_summaries < 0 || t.max_window_tokens < 0 ||
      t.n_windows > INT32_MAX || t.n_tokens > (int64_t)INT32_MAX * 64 ||
      t.max_window_tokens > INT32_MAX / 2)
    return FOCUS_E_SHAPE;
  if ((d->batch > 0 && !d->seq_nt) || !d->cu_windows || !d->cu_tokens || !d->cu_summaries)
    return FOCUS_E_NULL;
  if (t.n_windows > 0 && (!d->win_seq || !d->win_nt || !d->win_nsum || !d->win_ntok ||
                          !d->win_cache_off || !d->win_tok_off || !d->win_sum_off ||
                          !d->win_base_off))
    return FOCUS_E_NULL;
  if (t.n_tokens > 0 && (!d->tok_pos || !d->tok_kmer || !d->tok_win || !d->tok_kind || !d->tok_base))
    return FOCUS_E_NULL;
  if (t.n_summaries > 0 && !d->sum_tok) return FOCUS_E_NULL;
  if (d->bases && !d->token_ids) return FOCUS_E_NULL;

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(layout_windows, dim3(1), dim3(kScanThreads), 0, s, *d);
  focus_status st = focus::launch_status();
  if (st != FOCUS_OK) return st;
  if (t.n_windows > 0 && t.max_window_tokens > 0) {
    const int64_t tiles = focus::ceil_div(t.max_window_tokens, (int64_t)kTokThreads * kTokPerThread);
    const int64_t blocks = t.n_windows * tiles;
    if (blocks > INT32_MAX) return FOCUS_E_SHAPE;
    hipLaunchKernelGGL(layout_tokens, dim3((uint32_t)blocks), dim3(kTokThreads), 0, s, *d,
                       (int32_t)tiles);
    st = focus::launch_status();
  }
  return st;
}
