// The FOCUS adapter update of the summary tokens at one layer (Appendix A eq.
// focus-attn): projections on the matrix cores (focus_gemm), the adapter's
// retained K/V of the summary tokens (focus_compact_kv), the summary-query
// attention (focus_adapter_attn) and the output projection, enqueued back to
// back on one stream with every intermediate in the caller's workspace.
#include "common.h"

namespace {

size_t round256(size_t x) { return (x + 255) / 256 * 256; }

struct Parts {
  size_t k, v, ck, cv, q, a, total;
};

Parts parts(const focus_adapter_layer_desc* d) {
  const size_t nt = (size_t)d->totals.n_tokens, ns = (size_t)d->totals.n_summaries;
  const size_t kv_row = (size_t)d->n_kv_heads * d->head_dim * 2, q_row = (size_t)d->n_heads * d->head_dim * 2;
  const size_t cap = (size_t)(d->totals.max_cache_per_seq > 0 ? d->totals.max_cache_per_seq : 1);
  Parts p;
  size_t o = 0;
  p.k = o; o += round256(nt * kv_row);
  p.v = o; o += round256(nt * kv_row);
  p.ck = o; o += round256((size_t)d->batch * cap * kv_row);
  p.cv = o; o += round256((size_t)d->batch * cap * kv_row);
  p.q = o; o += round256(ns * q_row);
  p.a = o; o += round256(ns * q_row);
  p.total = o;
  return p;
}

focus_status validate(const focus_adapter_layer_desc* d) {
  if (d->dtype != FOCUS_BF16) return d->dtype == FOCUS_F32 ? FOCUS_E_UNSUPPORTED : FOCUS_E_DTYPE;
  if (d->n_heads <= 0 || d->n_kv_heads <= 0 || d->d_model <= 0 || d->batch < 0 || d->totals.n_tokens < 0 ||
      d->totals.n_summaries < 0)
    return FOCUS_E_ARG;
  if (d->head_dim != 64 && d->head_dim != 128) return FOCUS_E_UNSUPPORTED;
  if (d->n_heads % d->n_kv_heads) return FOCUS_E_SHAPE;
  if (d->d_model % 128 || ((int64_t)d->n_heads * d->head_dim) % 128 || ((int64_t)d->n_kv_heads * d->head_dim) % 128)
    return FOCUS_E_UNSUPPORTED;
  return FOCUS_OK;
}

}  // namespace

extern "C" size_t focus_adapter_layer_workspace(const focus_adapter_layer_desc* d) {
  if (!d || validate(d) != FOCUS_OK) return 0;
  return parts(d).total;
}

extern "C" focus_status focus_adapter_layer(const focus_adapter_layer_desc* d, focus_stream_t stream) {
  if (!d) return FOCUS_E_NULL;
  focus_status st = validate(d);
  if (st != FOCUS_OK) return st;
  if (d->totals.n_summaries == 0) return FOCUS_OK;
  if (!d->hidden || !d->w_q || !d->w_k || !d->w_v || !d->w_o || !d->out || !d->workspace || !d->win_seq ||
      !d->win_ntok || !d->win_cache_off || !d->win_tok_off || !d->win_nsum || !d->win_sum_off || !d->sum_tok)
    return FOCUS_E_NULL;
  const Parts p = parts(d);
  if (d->workspace_bytes < p.total) return FOCUS_E_WORKSPACE;
  if (!focus::aligned16(d->workspace) || !focus::aligned16(d->out)) return FOCUS_E_ARG;
  char* ws = reinterpret_cast<char*>(d->workspace);
  const int64_t nt = d->totals.n_tokens, ns = d->totals.n_summaries;
  const int64_t hq = (int64_t)d->n_heads * d->head_dim, hkv = (int64_t)d->n_kv_heads * d->head_dim;
  const int64_t cap = d->totals.max_cache_per_seq > 0 ? d->totals.max_cache_per_seq : 1;

  // K and V of every token
  focus_gemm_desc g = {};
  g.m = nt;
  g.n = hkv;
  g.k = d->d_model;
  g.a = d->hidden;
  g.lda = d->d_model;
  g.a_nrows = nt;
  g.ldb = hkv;
  g.ldc = hkv;
  g.c_dtype = FOCUS_BF16;
  g.alpha = 1.f;
  g.err = d->err;
  g.b = d->w_k;
  g.c = ws + p.k;
  if ((st = focus_gemm(&g, stream)) != FOCUS_OK) return st;
  g.b = d->w_v;
  g.c = ws + p.v;
  if ((st = focus_gemm(&g, stream)) != FOCUS_OK) return st;

  // the adapter's retained K/V: the summary tokens' rows, per sequence
  focus_compact_desc c = {};
  c.totals = d->totals;
  c.dtype = FOCUS_BF16;
  c.n_kv_heads = d->n_kv_heads;
  c.head_dim = d->head_dim;
  c.batch = d->batch;
  c.win_seq = d->win_seq;
  c.win_nsum = d->win_nsum;
  c.win_cache_off = d->win_cache_off;
  c.win_sum_off = d->win_sum_off;
  c.sum_tok = d->sum_tok;
  c.k = ws + p.k;
  c.v = ws + p.v;
  c.kv_rows = nt;
  c.cache_k = ws + p.ck;
  c.cache_v = ws + p.cv;
  c.cache_cap = cap;
  c.err = d->err;
  if ((st = focus_compact_kv(&c, stream)) != FOCUS_OK) return st;

  // Q of the summary tokens only (rows gathered through sum_tok)
  g.m = ns;
  g.n = hq;
  g.a_rows = d->sum_tok;
  g.b = d->w_q;
  g.ldb = hq;
  g.c = ws + p.q;
  g.ldc = hq;
  if ((st = focus_gemm(&g, stream)) != FOCUS_OK) return st;

  focus_adapter_desc a = {};
  a.totals = d->totals;
  a.dtype = FOCUS_BF16;
  a.n_heads = d->n_heads;
  a.n_kv_heads = d->n_kv_heads;
  a.head_dim = d->head_dim;
  a.softmax_scale = d->softmax_scale;
  a.mask = d->mask;
  a.batch = d->batch;
  a.kmer_uniform = d->kmer_uniform;
  a.win_seq = d->win_seq;
  a.win_ntok = d->win_ntok;
  a.win_cache_off = d->win_cache_off;
  a.win_tok_off = d->win_tok_off;
  a.win_kmer = d->win_kmer;
  a.win_nsum = d->win_nsum;
  a.win_sum_off = d->win_sum_off;
  a.sum_tok = d->sum_tok;
  a.q_sum = ws + p.q;
  a.sum_rows = ns;
  a.k = ws + p.k;
  a.v = ws + p.v;
  a.kv_rows = nt;
  a.cache_k = ws + p.ck;
  a.cache_v = ws + p.cv;
  a.cache_cap = cap;
  a.o_sum = ws + p.a;
  a.err = d->err;
  if ((st = focus_adapter_attn(&a, stream)) != FOCUS_OK) return st;

  // out = A W_O
  g.m = ns;
  g.n = d->d_model;
  g.k = hq;
  g.a = ws + p.a;
  g.lda = hq;
  g.a_rows = nullptr;
  g.a_nrows = ns;
  g.b = d->w_o;
  g.ldb = d->d_model;
  g.c = d->out;
  g.ldc = d->d_model;
  return focus_gemm(&g, stream);
}
