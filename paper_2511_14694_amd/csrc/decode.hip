// One-token decode over [retained summary cache ; current window]
// (focus_decode_step; Appendix A.2 streaming inference).
//
// Three launches per step, all state in device memory:
//   decode_append   a summary token's K/V goes to the cache, a base token's to
//                   the window buffer; the matching length is bumped
//   decode_partial  split-K: one workgroup per (sequence, chunk of split_keys
//                   rows) reads those rows for every head -- contiguous 8 KB
//                   K and V rows at 32 x 128 bf16 -- and writes an unnormalised
//                   partial (running max, sum, output) per head
//   decode_combine  one workgroup per (sequence, head) merges the partials
//                   with log-sum-exp weights and writes o and lse; the first
//                   head's workgroup empties the window buffer when the token
//                   closed its window (the key count comes from the workspace,
//                   so no workgroup reads the length it resets)
// The step reads every cached byte exactly once, so it is HBM bound: a thread
// owns 16 elements of one head (32 B per row in bf16) and the 8 (head_dim 128)
// or 4 (64) threads of a head reduce their dot products with DPP.
#include "common.h"

#include <math.h>

#include <algorithm>
#include <mutex>

namespace {

constexpr float kLn2 = 0.69314718055994531f;
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kMinit = -1.0e30f;
constexpr int kEpt = 16;    // elements of one head per thread
constexpr int kThreads = 256;

template <typename T> struct Elt;
// kU4: 16-byte loads per kEpt elements; kChunk: keys loaded per online-softmax
// update (bounded by registers: kChunk * kU4 * 2 uint4 per thread; for bf16 the
// 16-key chunk fills the 256 VGPRs of a one-wave-per-SIMD launch, which keeps
// the most loads in flight).
template <> struct Elt<__bf16> {
  static constexpr int kU4 = kEpt * 2 / 16;
  static constexpr int kChunk = 16;
  __device__ static void unpack(const uint4* src, float* out) {
#pragma unroll
    for (int i = 0; i < kU4; ++i) {
      const uint4 w = src[i];
      out[8 * i + 0] = focus::bf16_lo(w.x); out[8 * i + 1] = focus::bf16_hi(w.x);
      out[8 * i + 2] = focus::bf16_lo(w.y); out[8 * i + 3] = focus::bf16_hi(w.y);
      out[8 * i + 4] = focus::bf16_lo(w.z); out[8 * i + 5] = focus::bf16_hi(w.z);
      out[8 * i + 6] = focus::bf16_lo(w.w); out[8 * i + 7] = focus::bf16_hi(w.w);
    }
  }
  __device__ static void store(const float* x, void* dst) {
    uint4* p = reinterpret_cast<uint4*>(dst);
#pragma unroll
    for (int i = 0; i < kU4; ++i)
      p[i] = make_uint4(focus::pack_bf16x2(x[8 * i + 0], x[8 * i + 1]), focus::pack_bf16x2(x[8 * i + 2], x[8 * i + 3]),
                        focus::pack_bf16x2(x[8 * i + 4], x[8 * i + 5]), focus::pack_bf16x2(x[8 * i + 6], x[8 * i + 7]));
  }
};
template <> struct Elt<float> {
  static constexpr int kU4 = kEpt * 4 / 16;
  static constexpr int kChunk = 4;
  __device__ static void unpack(const uint4* src, float* out) {
#pragma unroll
    for (int i = 0; i < kU4; ++i) {
      const uint4 w = src[i];
      out[4 * i + 0] = __uint_as_float(w.x); out[4 * i + 1] = __uint_as_float(w.y);
      out[4 * i + 2] = __uint_as_float(w.z); out[4 * i + 3] = __uint_as_float(w.w);
    }
  }
  __device__ static void store(const float* x, void* dst) {
    float4* p = reinterpret_cast<float4*>(dst);
#pragma unroll
    for (int i = 0; i < kU4; ++i) p[i] = make_float4(x[4 * i], x[4 * i + 1], x[4 * i + 2], x[4 * i + 3]);
  }
};

__device__ inline int clamp_len(const int32_t* len, int b, int64_t cap) {
  const int64_t x = len[b];
  return (int)(x < 0 ? 0 : x > cap ? cap : x);
}

template <int TPH>
__device__ inline float head_sum(float x) {
  return TPH == 8 ? focus::sum8(x) : focus::sum4(x);
}

// Appends this step's K/V row of sequence blockIdx.x (bytes: row_u4 uint4s).
__global__ __launch_bounds__(256) void decode_append(focus_decode_desc d, int64_t row_u4) {
  const int b = blockIdx.x;
  const bool summary = d.kind[b] & FOCUS_STEP_SUMMARY;
  __shared__ int64_t row;
  if (threadIdx.x == 0) {
    const int64_t len = summary ? d.cache_len[b] : d.win_len[b];
    const int64_t cap = summary ? d.cache_cap : d.win_cap;
    row = (len >= 0 && len < cap) ? len : -1;
    if (row < 0) focus::raise_err(d.err, FOCUS_ERR_CAPACITY);
  }
  __syncthreads();
  if (row < 0) return;
  uint4* dk = reinterpret_cast<uint4*>(summary ? d.cache_k : d.win_k);
  uint4* dv = reinterpret_cast<uint4*>(summary ? d.cache_v : d.win_v);
  const int64_t cap = summary ? d.cache_cap : d.win_cap;
  const int64_t dst = ((int64_t)b * cap + row) * row_u4;
  const uint4* sk = reinterpret_cast<const uint4*>(d.k_new) + (int64_t)b * row_u4;
  const uint4* sv = reinterpret_cast<const uint4*>(d.v_new) + (int64_t)b * row_u4;
  for (int64_t c = threadIdx.x; c < row_u4; c += blockDim.x) {
    dk[dst + c] = sk[c];
    dv[dst + c] = sv[c];
  }
  __syncthreads();
  if (threadIdx.x == 0) (summary ? d.cache_len : d.win_len)[b] = (int32_t)(row + 1);
}

// Partial attention of one (sequence, split, group of kThreads / TPH heads).
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void decode_partial(focus_decode_desc d, float sc, int split,
                                                           int n_split, float* ws_o, float* ws_ml,
                                                           int32_t* ws_n) {
  constexpr int TPH = D / kEpt;
  constexpr int HPB = kThreads / TPH;
  const int n_hg = (d.n_heads + HPB - 1) / HPB;
  const int hg = blockIdx.x % n_hg;
  const int c = (blockIdx.x / n_hg) % n_split, b = blockIdx.x / (n_hg * n_split);
  const int H = d.n_heads, Hkv = d.n_kv_heads;
  const int h = hg * HPB + threadIdx.x / TPH, sub = threadIdx.x % TPH;
  if (h >= H) return;
  const int clen = clamp_len(d.cache_len, b, d.cache_cap);
  const int wlen = clamp_len(d.win_len, b, d.win_cap);
  const int n = clen + wlen;
  // the key count goes to the workspace, so the combine never reads win_len
  // (which it resets at a window end)
  if (c == 0 && hg == 0 && threadIdx.x == 0) ws_n[b] = n;
  const int jb = c * split;
  if (jb >= n) return;
  const int je = min(n, jb + split);
  const int hk = h / (H / Hkv);
  constexpr int kU4 = Elt<T>::kU4;
  constexpr int kChunk = Elt<T>::kChunk;
  const int64_t row_u4 = (int64_t)Hkv * D * sizeof(T) / 16;
  const int64_t my_u4 = ((int64_t)hk * D + sub * kEpt) * sizeof(T) / 16;

  float q[kEpt], o[kEpt];
  Elt<T>::unpack(reinterpret_cast<const uint4*>(d.q) + (((int64_t)b * H + h) * D + sub * kEpt) * sizeof(T) / 16, q);
#pragma unroll
  for (int e = 0; e < kEpt; ++e) {
    q[e] *= sc;
    o[e] = 0.f;
  }
  const uint4* kc = reinterpret_cast<const uint4*>(d.cache_k) + (int64_t)b * d.cache_cap * row_u4 + my_u4;
  const uint4* vc = reinterpret_cast<const uint4*>(d.cache_v) + (int64_t)b * d.cache_cap * row_u4 + my_u4;
  const uint4* kw = reinterpret_cast<const uint4*>(d.win_k) + (int64_t)b * d.win_cap * row_u4 + my_u4;
  const uint4* vw = reinterpret_cast<const uint4*>(d.win_v) + (int64_t)b * d.win_cap * row_u4 + my_u4;

  float m = kMinit, l = 0.f;
  for (int j0 = jb; j0 < je; j0 += kChunk) {
    uint4 kr[kChunk][kU4], vr[kChunk][kU4];
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      const int j = min(j0 + u, je - 1);
      const uint4* kp = j < clen ? kc + (int64_t)j * row_u4 : kw + (int64_t)(j - clen) * row_u4;
      const uint4* vp = j < clen ? vc + (int64_t)j * row_u4 : vw + (int64_t)(j - clen) * row_u4;
#pragma unroll
      for (int i = 0; i < kU4; ++i) {
        kr[u][i] = kp[i];
        vr[u][i] = vp[i];
      }
    }
    float s[kChunk];
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      float kx[kEpt];
      Elt<T>::unpack(kr[u], kx);
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < kEpt; ++e) acc = fmaf(q[e], kx[e], acc);
      s[u] = head_sum<TPH>(acc);
      if (j0 + u >= je) s[u] = -INFINITY;
    }
    float mx = s[0];
#pragma unroll
    for (int u = 1; u < kChunk; ++u) mx = fmaxf(mx, s[u]);
    const float m_new = fmaxf(m, mx);
    const float alpha = __builtin_amdgcn_exp2f(m - m_new);
    l *= alpha;
#pragma unroll
    for (int e = 0; e < kEpt; ++e) o[e] *= alpha;
    m = m_new;
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      const float p = __builtin_amdgcn_exp2f(s[u] - m);
      l += p;
      float vx[kEpt];
      Elt<T>::unpack(vr[u], vx);
#pragma unroll
      for (int e = 0; e < kEpt; ++e) o[e] = fmaf(p, vx[e], o[e]);
    }
  }
  const int64_t slot = ((int64_t)b * n_split + c) * H + h;
  float4* wo = reinterpret_cast<float4*>(ws_o + slot * D + sub * kEpt);
#pragma unroll
  for (int i = 0; i < kEpt / 4; ++i) wo[i] = make_float4(o[4 * i], o[4 * i + 1], o[4 * i + 2], o[4 * i + 3]);
  if (sub == 0) {
    ws_ml[2 * slot] = m;
    ws_ml[2 * slot + 1] = l;
  }
}

// Log-sum-exp merge of the partials of one (sequence, head): block
// (b * H + h), one thread per output element.  The key count comes from the
// workspace; block (b, 0) then empties the window buffer at a window end.
template <typename T, int D>
__global__ __launch_bounds__(D) void decode_combine(focus_decode_desc d, int split, int n_split,
                                                    const float* ws_o, const float* ws_ml,
                                                    const int32_t* ws_n) {
  const int H = d.n_heads;
  const int b = blockIdx.x / H, h = blockIdx.x % H, e = threadIdx.x;
  const int ns = (ws_n[b] + split - 1) / split;
  const int64_t slot0 = (int64_t)b * n_split * H + h;
  float M = kMinit;
  for (int c = 0; c < ns; ++c) M = fmaxf(M, ws_ml[2 * (slot0 + (int64_t)c * H)]);
  float L = 0.f, o = 0.f;
  for (int c = 0; c < ns; ++c) {
    const int64_t slot = slot0 + (int64_t)c * H;
    const float w = __builtin_amdgcn_exp2f(ws_ml[2 * slot] - M);
    L = fmaf(ws_ml[2 * slot + 1], w, L);
    o = fmaf(ws_o[slot * D + e], w, o);
  }
  o = L > 0.f ? o / L : 0.f;
  reinterpret_cast<T*>(d.o)[((int64_t)b * H + h) * D + e] = (T)o;
  if (e == 0 && d.lse) d.lse[(int64_t)b * H + h] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
  if (e == 0 && h == 0 && (d.kind[b] & FOCUS_STEP_WINDOW_END)) d.win_len[b] = 0;
}

int auto_split(int64_t batch, int64_t cap) {
  // About 7/8 as many workgroups as compute units for a full cache: a single
  // round of long-running workgroups.  Once the count passes the CU count, a
  // partial second round leaves most CUs idle at the end (batch 16 x 11 000
  // keys on 256 CUs: 272 workgroups read 56 % of HBM bandwidth, 208-240 read
  // 71-75 %, 704 read 68 %).
  const int64_t target = std::max(1, focus::device_cus() * 7 / 8);
  int64_t s = focus::ceil_div(batch * cap, target);
  s = focus::ceil_div(s, 16) * 16;
  return (int)(s < 16 ? 16 : s > (1 << 30) ? (1 << 30) : s);
}

struct Plan {
  int split;
  int n_split;
  size_t ws_bytes;
  size_t ml_offset;
  size_t n_offset;
};

Plan make_plan(const focus_decode_desc* d) {
  Plan p;
  const int64_t cap = d->cache_cap + d->win_cap;
  p.split = d->split_keys > 0 ? d->split_keys : auto_split(d->batch, cap);
  p.n_split = (int)focus::ceil_div(cap > 0 ? cap : 1, p.split);
  const size_t slots = (size_t)d->batch * p.n_split * d->n_heads;
  p.ml_offset = slots * d->head_dim * sizeof(float);
  p.n_offset = p.ml_offset + slots * 2 * sizeof(float);
  p.ws_bytes = p.n_offset + (((size_t)d->batch * sizeof(int32_t) + 15) / 16) * 16;
  return p;
}

focus_status validate(const focus_decode_desc* d) {
  if (d->dtype != FOCUS_BF16 && d->dtype != FOCUS_F32) return FOCUS_E_DTYPE;
  if (d->batch < 0 || d->n_heads <= 0 || d->n_kv_heads <= 0 || d->cache_cap < 0 || d->win_cap < 0 ||
      d->split_keys < 0 || (d->split_keys % 16) || !(d->softmax_scale == d->softmax_scale))
    return FOCUS_E_ARG;
  if (d->head_dim != 64 && d->head_dim != 128) return FOCUS_E_UNSUPPORTED;
  if (d->n_heads % d->n_kv_heads) return FOCUS_E_SHAPE;
  if (d->cache_cap + d->win_cap > INT32_MAX / 2) return FOCUS_E_SHAPE;
  return FOCUS_OK;
}

}  // namespace

extern "C" size_t focus_decode_workspace(const focus_decode_desc* d) {
  if (!d || validate(d) != FOCUS_OK) return 0;
  return make_plan(d).ws_bytes;
}

namespace {

// Checks every argument except the workspace; fills the plan.
focus_status check_step(const focus_decode_desc* d, Plan* p) {
  if (!d) return FOCUS_E_NULL;
  focus_status st = validate(d);
  if (st != FOCUS_OK) return st;
  if (d->batch == 0) return FOCUS_OK;
  if (!d->q || !d->k_new || !d->v_new || !d->kind || !d->cache_k || !d->cache_v || !d->cache_len ||
      !d->win_k || !d->win_v || !d->win_len || !d->o)
    return FOCUS_E_NULL;
  if (!focus::aligned16(d->q) || !focus::aligned16(d->k_new) || !focus::aligned16(d->v_new) ||
      !focus::aligned16(d->cache_k) || !focus::aligned16(d->cache_v) || !focus::aligned16(d->win_k) ||
      !focus::aligned16(d->win_v) || !focus::aligned16(d->o) || (reinterpret_cast<uintptr_t>(d->lse) & 3u))
    return FOCUS_E_ARG;
  *p = make_plan(d);
  const int hpb = kThreads / (d->head_dim / kEpt);
  const int64_t blocks = (int64_t)d->batch * p->n_split * focus::ceil_div(d->n_heads, hpb);
  if (blocks > INT32_MAX / kThreads) return FOCUS_E_SHAPE;
  return FOCUS_OK;
}

// Enqueues the three launches of a step with the partials in ws (at least
// p.ws_bytes, 16-byte aligned).
focus_status launch_step(const focus_decode_desc* d, const Plan& p, void* ws, hipStream_t s) {
  focus_status st;
  const int hpb = kThreads / (d->head_dim / kEpt);
  const int64_t blocks = (int64_t)d->batch * p.n_split * focus::ceil_div(d->n_heads, hpb);
  const int64_t eb = focus::elt_bytes(d->dtype);
  const int64_t row_u4 = (int64_t)d->n_kv_heads * d->head_dim * eb / 16;
  hipLaunchKernelGGL(decode_append, dim3(d->batch), dim3(256), 0, s, *d, row_u4);
  if ((st = focus::launch_status()) != FOCUS_OK) return st;

  const float scale = d->softmax_scale > 0.f ? d->softmax_scale : 1.0f / sqrtf((float)d->head_dim);
  const float sc = scale * kLog2e;
  float* ws_o = reinterpret_cast<float*>(ws);
  float* ws_ml = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + p.ml_offset);
  int32_t* ws_n = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(ws) + p.n_offset);
  const dim3 block(kThreads);
#define FOCUS_DECODE_LAUNCH(T, D)                                                                  \
  hipLaunchKernelGGL((decode_partial<T, D>), dim3((uint32_t)blocks), block, 0, s, *d, sc, p.split, \
                     p.n_split, ws_o, ws_ml, ws_n);                                                \
  if ((st = focus::launch_status()) != FOCUS_OK) return st;                                       \
  hipLaunchKernelGGL((decode_combine<T, D>), dim3(d->batch * d->n_heads), dim3(D), 0, s, *d,       \
                     p.split, p.n_split, ws_o, ws_ml, ws_n);
  if (d->dtype == FOCUS_BF16) {
    if (d->head_dim == 128) { FOCUS_DECODE_LAUNCH(__bf16, 128) } else { FOCUS_DECODE_LAUNCH(__bf16, 64) }
  } else {
    if (d->head_dim == 128) { FOCUS_DECODE_LAUNCH(float, 128) } else { FOCUS_DECODE_LAUNCH(float, 64) }
  }
#undef FOCUS_DECODE_LAUNCH
  return focus::launch_status();
}

}  // namespace

extern "C" focus_status focus_decode_step(const focus_decode_desc* d, focus_stream_t stream) {
  Plan p;
  const focus_status st = check_step(d, &p);
  if (st != FOCUS_OK || d->batch == 0) return st;
  if (!d->workspace || d->workspace_bytes < p.ws_bytes) return FOCUS_E_WORKSPACE;
  if (!focus::aligned16(d->workspace)) return FOCUS_E_ARG;
  return launch_step(d, p, d->workspace, reinterpret_cast<hipStream_t>(stream));
}

// ------------------------------------------------------- decode schedule

namespace {

// Cadence of window j of sequence b (a negative one raises BOUNDS, counts as 0).
__device__ inline int sched_kmer(const focus_decode_sched& s, int b, int j) {
  int k = s.kmer_uniform;
  if (s.kmer) k = s.kmer[(int64_t)b * s.kmer_stride + min(max(j, 0), s.kmer_stride - 1)];
  if (k < 0) {
    focus::raise_err(s.err, FOCUS_ERR_BOUNDS);
    k = 0;
  }
  return k;
}

// The insertion rule for one token of a sequence whose window j holds nw
// bases with nk of them in the open k-mer: returns its FOCUS_STEP_* bits and
// advances (j, nw, nk) past it.
__device__ inline uint8_t sched_advance(const focus_decode_sched& s, int b, int& j, int& nw, int& nk) {
  const int W = s.window_nt;
  const int k = sched_kmer(s, b, j);
  uint8_t kind = 0;
  bool end;
  if (k > 0 && (nk == k || (nw == W && nk > 0))) {
    kind = FOCUS_STEP_SUMMARY;
    nk = 0;
    end = nw == W;
  } else {
    ++nw;
    ++nk;
    end = k == 0 && nw == W;
  }
  if (end) {
    kind |= FOCUS_STEP_WINDOW_END;
    ++j;
    nw = 0;
    nk = 0;
  }
  return kind;
}

// One thread per sequence.  start: walk tokens[b] tokens from the start of
// window win_index[b]; otherwise derive the next token's kind.
__global__ __launch_bounds__(256) void decode_sched(focus_decode_sched s, bool start) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= s.batch) return;
  int j = s.win_index[b], nw, nk;
  if (start) {
    nw = nk = 0;
    int summaries = 0;
    const int n = max(s.tokens[b], 0);
    for (int t = 0; t < n; ++t) summaries += sched_advance(s, b, j, nw, nk) & FOCUS_STEP_SUMMARY;
    if (s.summaries) s.summaries[b] = summaries;
  } else {
    nw = s.bases_in_window[b];
    nk = s.bases_in_kmer[b];
    s.kind[b] = sched_advance(s, b, j, nw, nk);
  }
  s.win_index[b] = j;
  s.bases_in_window[b] = nw;
  s.bases_in_kmer[b] = nk;
}

focus_status launch_sched(const focus_decode_sched* s, bool start, focus_stream_t stream) {
  if (!s) return FOCUS_E_NULL;
  if (s->batch < 0 || s->window_nt < 1 || (!s->kmer && s->kmer_uniform < 0) || (s->kmer && s->kmer_stride < 1))
    return FOCUS_E_ARG;
  if (s->batch == 0) return FOCUS_OK;
  if (!s->win_index || !s->bases_in_window || !s->bases_in_kmer || (start ? !s->tokens : !s->kind))
    return FOCUS_E_NULL;
  hipLaunchKernelGGL(decode_sched, dim3((uint32_t)focus::ceil_div(s->batch, 256)), dim3(256), 0,
                     reinterpret_cast<hipStream_t>(stream), *s, start);
  return focus::launch_status();
}

}  // namespace

extern "C" focus_status focus_decode_sched_start(const focus_decode_sched* s, focus_stream_t stream) {
  return launch_sched(s, true, stream);
}

extern "C" focus_status focus_decode_next_kind(const focus_decode_sched* s, focus_stream_t stream) {
  return launch_sched(s, false, stream);
}

// ------------------------------------------------ allocation-free variant

// The partials of focus_decode_step_noalloc live in this array: one copy per
// device, held until the process ends.  Host code never passes the array's
// name to a kernel (on the host it is only a stand-in for the symbol): the
// device address comes from hipGetSymbolAddress, looked up once per device
// with that device current.
static __device__ __align__(256) char scratch[FOCUS_DECODE_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of this device's scratch array (looked up on first use).
focus_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return FOCUS_E_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return FOCUS_E_HIP;
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return FOCUS_OK;
}

}  // namespace

extern "C" focus_status focus_decode_step_noalloc(const focus_decode_desc* d, focus_stream_t stream) {
  Plan p;
  focus_status st = check_step(d, &p);
  if (st != FOCUS_OK || d->batch == 0) return st;
  if (p.ws_bytes > (size_t)FOCUS_DECODE_SCRATCH_BYTES) return FOCUS_E_WORKSPACE;
  void* ws = nullptr;
  if ((st = scratch_address(&ws)) != FOCUS_OK) return st;
  return launch_step(d, p, ws, reinterpret_cast<hipStream_t>(stream));
}
