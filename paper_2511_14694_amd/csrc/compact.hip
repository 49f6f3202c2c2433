// Retained-KV compaction (focus_compact_kv).
//
// After window w, FOCUS keeps only the K/V rows of its B_w summary tokens and
// appends them to its sequence's cache at rows [C_w, C_w + B_w) (Appendix A
// "KV compression and budget"); ordinary rows are simply not copied.
//
// One workgroup per retained row copies that row's K and V (n_kv_heads x
// head_dim elements each, 8 KB per tensor at 32 x 128 bf16) with 16-byte
// loads and stores; a launch covering every window of a 1 Mb sequence moves
// 10 000 rows.  The copy is HBM bound: it reads and writes each retained byte
// once and touches nothing else.
#include "common.h"

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

// Window holding global summary s: the largest window whose first summary is
// <= s (windows without summaries share their offset with the next window).
__device__ int64_t owner_window(const int64_t* sum_off, int64_t n_windows, int64_t s) {
  int64_t lo = 0, hi = n_windows - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (sum_off[mid] <= s) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__global__ __launch_bounds__(kThreads) void compact_rows(focus_compact_desc d, int64_t row_chunks) {
  int64_t gw, s;
  if (d.win_ids) {
    const int64_t per = d.totals.max_window_summaries;
    const int64_t li = blockIdx.x / per, j = blockIdx.x % per;
    gw = d.win_ids[li];
    if (gw < 0 || gw >= d.totals.n_windows) {
      if (threadIdx.x == 0 && j == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
      return;
    }
    if (j >= d.win_nsum[gw]) return;
    s = d.win_sum_off[gw] + j;
  } else {
    s = blockIdx.x;
    gw = owner_window(d.win_sum_off, d.totals.n_windows, s);
  }
  const int64_t j = s - d.win_sum_off[gw];
  const int64_t B = d.win_nsum[gw];
  const int32_t b = d.win_seq[gw];
  const int64_t row = d.win_cache_off[gw] + j;
  const int64_t src = d.sum_tok[s] - d.kv_tok_base;
  if (b < 0 || b >= d.batch || j < 0 || j >= B || src < 0 || src >= d.kv_rows) {
    if (threadIdx.x == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
    return;
  }
  if (row < 0 || row >= d.cache_cap) {
    if (threadIdx.x == 0) focus::raise_err(d.err, FOCUS_ERR_CAPACITY);
    return;
  }
  const focus::u32x4* sk = reinterpret_cast<const focus::u32x4*>(d.k) + src * row_chunks;
  const focus::u32x4* sv = reinterpret_cast<const focus::u32x4*>(d.v) + src * row_chunks;
  focus::u32x4* dk = reinterpret_cast<focus::u32x4*>(d.cache_k) + ((int64_t)b * d.cache_cap + row) * row_chunks;
  focus::u32x4* dv = reinterpret_cast<focus::u32x4*>(d.cache_v) + ((int64_t)b * d.cache_cap + row) * row_chunks;
  for (int64_t c0 = 0; c0 < row_chunks; c0 += kThreads * kUnroll) {
    focus::u32x4 rk[kUnroll], rv[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t c = c0 + u * kThreads + threadIdx.x;
      if (c < row_chunks) {
        rk[u] = __builtin_nontemporal_load(sk + c);
        rv[u] = __builtin_nontemporal_load(sv + c);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t c = c0 + u * kThreads + threadIdx.x;
      if (c < row_chunks) {
        __builtin_nontemporal_store(rk[u], dk + c);
        __builtin_nontemporal_store(rv[u], dv + c);
      }
    }
  }
  if (d.cache_len && threadIdx.x == 0 && j == B - 1) atomicMax(d.cache_len + b, (int32_t)(row + 1));
}

}  // namespace

extern "C" focus_status focus_compact_kv(const focus_compact_desc* d, focus_stream_t stream) {
  if (!d) return FOCUS_E_NULL;
  const int64_t eb = focus::elt_bytes(d->dtype);
  if (eb == 0) return FOCUS_E_DTYPE;
  if (d->head_dim != 64 && d->head_dim != 128) return FOCUS_E_UNSUPPORTED;
  if (d->n_kv_heads <= 0 || d->batch < 0 || d->cache_cap < 0 || d->kv_rows < 0 ||
      (d->win_ids && d->n_win < 0))
    return FOCUS_E_ARG;
  const focus_layout_totals& t = d->totals;
  if (t.n_windows < 0 || t.n_summaries < 0 || t.max_window_summaries < 0 ||
      (t.n_summaries > 0 && t.n_windows == 0))
    return FOCUS_E_SHAPE;
  const int64_t items = d->win_ids ? d->n_win * t.max_window_summaries : t.n_summaries;
  if (items == 0) return FOCUS_OK;
  if (!d->win_seq || !d->win_nsum || !d->win_cache_off || !d->win_sum_off || !d->sum_tok ||
      !d->k || !d->v || !d->cache_k || !d->cache_v)
    return FOCUS_E_NULL;
  if (!focus::aligned16(d->k) || !focus::aligned16(d->v) || !focus::aligned16(d->cache_k) ||
      !focus::aligned16(d->cache_v))
    return FOCUS_E_ARG;
  if (!d->win_ids && t.max_cache_per_seq > d->cache_cap) return FOCUS_E_CAPACITY;
  if (items > INT32_MAX) return FOCUS_E_SHAPE;
  const int64_t row_chunks = (int64_t)d->n_kv_heads * d->head_dim * eb / 16;
  hipLaunchKernelGGL(compact_rows, dim3((uint32_t)items), dim3(kThreads), 0,
                     reinterpret_cast<hipStream_t>(stream), *d, row_chunks);
  return focus::launch_status();
}
