// Library-wide entry points: version, status strings, struct sizes and the
// host-side layout plan.
#include "common.h"

extern "C" int32_t focus_abi_version(void) { return FOCUS_ABI_VERSION; }

extern "C" const char* focus_status_str(focus_status s) {
  switch (s) {
    case FOCUS_OK: return "ok";
    case FOCUS_E_NULL: return "required pointer is NULL";
    case FOCUS_E_ARG: return "argument out of range or pointer misaligned";
    case FOCUS_E_SHAPE: return "inconsistent sizes";
    case FOCUS_E_DTYPE: return "unknown dtype";
    case FOCUS_E_UNSUPPORTED: return "unsupported configuration";
    case FOCUS_E_WORKSPACE: return "workspace missing or too small";
    case FOCUS_E_CAPACITY: return "cache capacity too small";
    case FOCUS_E_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

extern "C" int64_t focus_struct_size(int32_t which) {
  switch (which) {
    case 0: return sizeof(focus_layout_totals);
    case 1: return sizeof(focus_layout_desc);
    case 2: return sizeof(focus_compact_desc);
    case 3: return sizeof(focus_attn_desc);
    case 4: return sizeof(focus_decode_desc);
    case 5: return sizeof(focus_fidelity_desc);
    case 6: return sizeof(focus_gemm_desc);
    case 7: return sizeof(focus_adapter_desc);
    case 8: return sizeof(focus_adapter_layer_desc);
    case 9: return sizeof(focus_qkv_desc);
    case 10: return sizeof(focus_decode_sched);
    default: return -1;
  }
}

// Totals of the layout (Appendix A window and B_w definitions): every window
// of sequence b covers min(W, L_b - wW) bases and holds ceil(n_w / k_w)
// summaries, T_w = n_w + B_w tokens, and sees the C_w summaries of the
// windows before it.
extern "C" focus_status focus_layout_plan(int32_t batch, const int64_t* seq_nt, int32_t window_nt,
                                          const int32_t* kmer, int32_t kmer_uniform,
                                          focus_layout_totals* out) {
  if (!out || (batch > 0 && !seq_nt)) return FOCUS_E_NULL;
  if (batch < 0 || window_nt <= 0 || (!kmer && kmer_uniform < 0)) return FOCUS_E_ARG;
  focus_layout_totals t = {};
  const int64_t W = window_nt;
  for (int32_t b = 0; b < batch; ++b) {
    if (seq_nt[b] < 0) return FOCUS_E_ARG;
    const int64_t L = seq_nt[b];
    const int64_t nwin = focus::ceil_div(L, W);
    int64_t cache = 0;
    for (int64_t w = 0; w < nwin; ++w) {
      const int64_t k = kmer ? kmer[t.n_windows] : kmer_uniform;
      if (k < 0) return FOCUS_E_ARG;
      const int64_t n = (L - w * W) < W ? (L - w * W) : W;
      const int64_t B = k > 0 ? focus::ceil_div(n, k) : 0;
      if (n + B > t.max_window_tokens) t.max_window_tokens = n + B;
      if (B > t.max_window_summaries) t.max_window_summaries = B;
      if (cache > t.max_window_cache) t.max_window_cache = cache;
      cache += B;
      t.n_tokens += n + B;
      t.n_summaries += B;
      t.n_windows += 1;
    }
    if (cache > t.max_cache_per_seq) t.max_cache_per_seq = cache;
  }
  *out = t;
  return FOCUS_OK;
}
