// Fidelity metrics between two next-base distributions (focus_fidelity):
// L1, L2, Hellinger, Jensen-Shannon and KL(p || q) of the Metrics appendix,
// after clipping both distributions at 1e-12 and renormalising, per position;
// optionally the per-sequence mean of each metric.
//
// Bound by HBM: every input element is read once.  Rows of up to 8 categories
// (the four nucleotides) take one thread per position with the whole row in
// registers; longer rows (a byte-level vocabulary) take one wave per position,
// each lane holding up to 16 of the row's elements, with wave reductions.
// Logarithms are base 2 (v_log_f32) scaled by ln 2 once per sum.
#include "common.h"

#include <math.h>

namespace {

constexpr float kClip = 1e-12f;
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kLn2 = 0.69314718055994531f;
constexpr int kSmallV = 8;       // rows up to this long: one thread per position
constexpr int kMaxPerLane = 16;  // wave path: elements per lane, vocab <= 1024
constexpr int kThreads = 256;

template <typename T> __device__ inline float ld(const T* p, int64_t i);
template <> __device__ inline float ld<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ inline float ld<__bf16>(const __bf16* p, int64_t i) { return (float)p[i]; }

// Wave-wide sum / max, the result in every lane: DPP inside rows of 16 lanes
// (quad swaps, then the half-row and row mirrors), one swizzle across the two
// rows of each half-wave, and v_permlane32_swap across the halves.
__device__ inline float dpp_mirror16(float x) {  // lane i <-> lane 15-i within 16
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false));
}
__device__ inline float wave_sum(float x) {
  x = focus::sum8(x);
  x += dpp_mirror16(x);
  x += __shfl_xor(x, 16);
  const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
}
__device__ inline float wave_max(float x) {
  x = fmaxf(x, focus::dpp_xor1(x));
  x = fmaxf(x, focus::dpp_xor2(x));
  x = fmaxf(x, focus::dpp_half_mirror(x));
  x = fmaxf(x, dpp_mirror16(x));
  x = fmaxf(x, __shfl_xor(x, 16));
  const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
}

// Accumulates the metric sums of one pair of clipped, renormalised
// probabilities: |d|, d^2, (sqrt p - sqrt q)^2, the JS terms and the KL term
// (the last two in log2 units).
struct Sums {
  float l1 = 0.f, l2 = 0.f, h = 0.f, js = 0.f, kl = 0.f;
  __device__ void add(float p, float q) {
    const float d = p - q;
    l1 += fabsf(d);
    l2 = fmaf(d, d, l2);
    const float s = __builtin_amdgcn_sqrtf(p) - __builtin_amdgcn_sqrtf(q);  // p, q clipped: no denormals
    h = fmaf(s, s, h);
    const float lp = __builtin_amdgcn_logf(p), lq = __builtin_amdgcn_logf(q);
    const float lm = __builtin_amdgcn_logf(0.5f * (p + q));
    js += p * (lp - lm) + q * (lq - lm);
    kl = fmaf(p, lp - lq, kl);
  }
  __device__ void store(float* out) const {
    out[FOCUS_FID_L1] = l1;
    out[FOCUS_FID_L2] = sqrtf(l2);
    out[FOCUS_FID_HELLINGER] = sqrtf(0.5f * h);
    out[FOCUS_FID_JS] = 0.5f * kLn2 * js;
    out[FOCUS_FID_KL] = kLn2 * kl;
  }
};

// One thread per position, vocab <= kSmallV.
template <typename T>
__global__ __launch_bounds__(kThreads) void fid_rows_small(focus_fidelity_desc d) {
  const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (t >= d.n_pos) return;
  const int V = d.vocab;
  const T* pr = reinterpret_cast<const T*>(d.p) + t * V;
  const T* qr = reinterpret_cast<const T*>(d.q) + t * V;
  float p[kSmallV], q[kSmallV];
  float mp = -INFINITY, mq = -INFINITY;
#pragma unroll
  for (int i = 0; i < kSmallV; ++i) {
    p[i] = i < V ? ld(pr, i) : 0.f;
    q[i] = i < V ? ld(qr, i) : 0.f;
    if (i < V) {
      mp = fmaxf(mp, p[i]);
      mq = fmaxf(mq, q[i]);
    }
  }
  float sp = 0.f, sq = 0.f;
#pragma unroll
  for (int i = 0; i < kSmallV; ++i) {
    if (i < V) {
      if (d.input_kind == FOCUS_FID_LOGITS) {
        p[i] = __builtin_amdgcn_exp2f((p[i] - mp) * kLog2e);
        q[i] = __builtin_amdgcn_exp2f((q[i] - mq) * kLog2e);
      }
      sp += p[i];
      sq += q[i];
    }
  }
  // finish the softmax (logits only), clip, renormalise
  if (d.input_kind != FOCUS_FID_LOGITS) sp = sq = 1.f;
  float cp = 0.f, cq = 0.f;
#pragma unroll
  for (int i = 0; i < kSmallV; ++i) {
    if (i < V) {
      p[i] = fmaxf(p[i] / sp, kClip);
      q[i] = fmaxf(q[i] / sq, kClip);
      cp += p[i];
      cq += q[i];
    }
  }
  Sums m;
#pragma unroll
  for (int i = 0; i < kSmallV; ++i)
    if (i < V) m.add(p[i] / cp, q[i] / cq);
  m.store(d.out + t * FOCUS_FID_N);
}

// Four categories (the nucleotides), rows 16-byte (float) or 8-byte (bf16)
// aligned: one thread per position, each row in one load, and the softmax,
// clip and renormalisation by reciprocals (one division per row instead of one
// per element).  Contraction is off: a product fused into one side of p - q
// but not the other would break the exact zero of identical rows.
template <typename T>
__global__ __launch_bounds__(kThreads) void fid_rows4(focus_fidelity_desc d) {
#pragma clang fp contract(off)
  const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (t >= d.n_pos) return;
  float p[4], q[4];
  if constexpr (sizeof(T) == 4) {
    const float4 a = reinterpret_cast<const float4*>(d.p)[t];
    const float4 b = reinterpret_cast<const float4*>(d.q)[t];
    p[0] = a.x, p[1] = a.y, p[2] = a.z, p[3] = a.w;
    q[0] = b.x, q[1] = b.y, q[2] = b.z, q[3] = b.w;
  } else {
    const uint2 a = reinterpret_cast<const uint2*>(d.p)[t];
    const uint2 b = reinterpret_cast<const uint2*>(d.q)[t];
    const uint32_t wa[2] = {a.x, a.y}, wb[2] = {b.x, b.y};
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      p[2 * i] = __uint_as_float(wa[i] << 16);
      p[2 * i + 1] = __uint_as_float(wa[i] & 0xFFFF0000u);
      q[2 * i] = __uint_as_float(wb[i] << 16);
      q[2 * i + 1] = __uint_as_float(wb[i] & 0xFFFF0000u);
    }
  }
  if (d.input_kind == FOCUS_FID_LOGITS) {
    const float mp = fmaxf(fmaxf(p[0], p[1]), fmaxf(p[2], p[3]));
    const float mq = fmaxf(fmaxf(q[0], q[1]), fmaxf(q[2], q[3]));
    float sp = 0.f, sq = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p[i] = __builtin_amdgcn_exp2f((p[i] - mp) * kLog2e);
      q[i] = __builtin_amdgcn_exp2f((q[i] - mq) * kLog2e);
      sp += p[i];
      sq += q[i];
    }
    const float rp = 1.f / sp, rq = 1.f / sq;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p[i] *= rp;
      q[i] *= rq;
    }
  }
  float cp = 0.f, cq = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    p[i] = fmaxf(p[i], kClip);
    q[i] = fmaxf(q[i], kClip);
    cp += p[i];
    cq += q[i];
  }
  const float rcp = 1.f / cp, rcq = 1.f / cq;
  Sums m;
#pragma unroll
  for (int i = 0; i < 4; ++i) m.add(p[i] * rcp, q[i] * rcq);
  m.store(d.out + t * FOCUS_FID_N);
}

// One wave per position, kSmallV < vocab <= 64 * NPL (NPL = 8 or 16).  VEC: the row is
// read 16 bytes per lane per load (kVec elements), else one element per load.
// Logarithms of the clipped, renormalised probabilities come straight from the
// logits (log2 p = (x - max) log2 e - log2 sum, or log2 of the clip); the
// mixture's logarithm is built from them, and no division is left per element.
template <typename T, bool VEC, int NPL, bool FULL>
__global__ __launch_bounds__(kThreads) void fid_rows_wave(focus_fidelity_desc d) {
  constexpr int kVec = 16 / sizeof(T);
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (t >= d.n_pos) return;
  const int V = d.vocab;
  const bool logits = d.input_kind == FOCUS_FID_LOGITS;
  const T* pr = reinterpret_cast<const T*>(d.p) + t * V;
  const T* qr = reinterpret_cast<const T*>(d.q) + t * V;
  auto elem = [&](int k) { return VEC ? (k / kVec) * 64 * kVec + lane * kVec + k % kVec : lane + 64 * k; };
  // FULL: vocab == 64 NPL, every element of every lane is in the row
  bool ok[NPL];
#pragma unroll
  for (int k = 0; k < NPL; ++k) ok[k] = FULL || elem(k) < V;
  float xp[NPL], xq[NPL];
  if constexpr (VEC) {
#pragma unroll
    for (int c = 0; c < NPL / kVec; ++c) {
      const int i0 = c * 64 * kVec + lane * kVec;
      uint4 wp = make_uint4(0, 0, 0, 0), wq = wp;
      if (i0 < V) {
        wp = *reinterpret_cast<const uint4*>(pr + i0);
        wq = *reinterpret_cast<const uint4*>(qr + i0);
      }
      const T* ep = reinterpret_cast<const T*>(&wp);
      const T* eq = reinterpret_cast<const T*>(&wq);
#pragma unroll
      for (int j = 0; j < kVec; ++j) {
        xp[c * kVec + j] = (float)ep[j];
        xq[c * kVec + j] = (float)eq[j];
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      const int i = elem(k);
      xp[k] = i < V ? ld(pr, i) : 0.f;
      xq[k] = i < V ? ld(qr, i) : 0.f;
    }
  }
  float mp = -INFINITY, mq = -INFINITY;
  if (logits) {
#pragma unroll
    for (int k = 0; k < NPL; ++k)
      if (ok[k]) {
        mp = fmaxf(mp, xp[k]);
        mq = fmaxf(mq, xq[k]);
      }
    mp = wave_max(mp);
    mq = wave_max(mq);
  }
  // p = softmax(x) (logits) or x (probabilities); then the clip
  float p[NPL], q[NPL];
  float sp = 0.f, sq = 0.f;
#pragma unroll
  for (int k = 0; k < NPL; ++k) {
    p[k] = logits ? __builtin_amdgcn_exp2f((xp[k] - mp) * kLog2e) : xp[k];
    q[k] = logits ? __builtin_amdgcn_exp2f((xq[k] - mq) * kLog2e) : xq[k];
    if (ok[k]) {
      sp += p[k];
      sq += q[k];
    }
  }
  float rp = 1.f, rq = 1.f, lsp = 0.f, lsq = 0.f;
  if (logits) {
    sp = wave_sum(sp);
    sq = wave_sum(sq);
    rp = 1.f / sp;
    rq = 1.f / sq;
    lsp = __builtin_amdgcn_logf(sp);
    lsq = __builtin_amdgcn_logf(sq);
  }
  float cp = 0.f, cq = 0.f;
#pragma unroll
  for (int k = 0; k < NPL; ++k) {
    p[k] = fmaxf(p[k] * rp, kClip);
    q[k] = fmaxf(q[k] * rq, kClip);
    if (ok[k]) {
      cp += p[k];
      cq += q[k];
    }
  }
  cp = wave_sum(cp);
  cq = wave_sum(cq);
  const float rcp = 1.f / cp, rcq = 1.f / cq;
  const float lcp = __builtin_amdgcn_logf(cp), lcq = __builtin_amdgcn_logf(cq);
  const float lclip = __builtin_amdgcn_logf(kClip);
  float l1 = 0.f, l2 = 0.f, h = 0.f, js = 0.f, kl = 0.f;
#pragma unroll
  for (int k = 0; k < NPL; ++k) {
    if (!ok[k]) continue;
    const float pn = p[k] * rcp, qn = q[k] * rcq;
    float lp, lq;
    if (logits) {
      lp = (p[k] > kClip ? (xp[k] - mp) * kLog2e - lsp : lclip) - lcp;
      lq = (q[k] > kClip ? (xq[k] - mq) * kLog2e - lsq : lclip) - lcq;
    } else {
      lp = __builtin_amdgcn_logf(pn);
      lq = __builtin_amdgcn_logf(qn);
    }
    const float dd = pn - qn;
    l1 += fabsf(dd);
    l2 = fmaf(dd, dd, l2);
    // pn, qn >= 1e-12 / 1.x after the clip: no denormals, so the bare
    // v_sqrt_f32 (no denormal scaling around it) is exact to its ulp
    const float sd = __builtin_amdgcn_sqrtf(pn) - __builtin_amdgcn_sqrtf(qn);
    h = fmaf(sd, sd, h);
    // log2 m from lp and lq (exactly lp when lp == lq, so identical inputs
    // give an exact zero): m = 2^max * (1 + 2^-|lp - lq|) / 2
    const float lm = fmaxf(lp, lq) + __builtin_amdgcn_logf(0.5f + 0.5f * __builtin_amdgcn_exp2f(-fabsf(lp - lq)));
    js += pn * (lp - lm) + qn * (lq - lm);
    kl = fmaf(pn, lp - lq, kl);
  }
  Sums m;
  m.l1 = wave_sum(l1);
  m.l2 = wave_sum(l2);
  m.h = wave_sum(h);
  m.js = wave_sum(js);
  m.kl = wave_sum(kl);
  if (lane == 0) m.store(d.out + t * FOCUS_FID_N);
}

// Sums / extrema over the 32 lanes of a half-wave, the result in each of them.
__device__ inline float half_sum(float x) {
  x = focus::sum8(x);
  x += dpp_mirror16(x);
  return x + __shfl_xor(x, 16);
}
__device__ inline float half_max(float x) {
  x = fmaxf(x, focus::dpp_xor1(x));
  x = fmaxf(x, focus::dpp_xor2(x));
  x = fmaxf(x, focus::dpp_half_mirror(x));
  x = fmaxf(x, dpp_mirror16(x));
  return fmaxf(x, __shfl_xor(x, 16));
}
__device__ inline float half_min(float x) { return -half_max(-x); }

// Logits rows with 64 < vocab <= 32 NPL read 16 bytes per lane per load: half
// a wave (32 lanes) per position, two positions per wave.
//
// Fewer operations per element than fid_rows_wave:
// * e = 2^((x - max) log2(e) / 2) is the square root of the unnormalised
//   probability: p = e^2 rp (rp = 1 / sum e^2) and sqrt(p) = e sqrt(rp), so
//   one exponential per element gives both, and the Hellinger term needs no
//   square root;
// * when the smallest probability of both rows is at least twice the clip
//   (decided from the row minimum of the logits), the clip changes nothing and
//   the renormalised sum is 1: that pass is skipped.  Otherwise the clip and
//   the renormalisation are applied as in fid_rows_wave;
// * log2 p and log2 q come from the logits, and the mixture's logarithm from
//   r = log2 q - log2 p: log2 m - log2 p = max(r, 0) + log2((1 + 2^-|r|) / 2),
//   so the JS term is q r - (p + q) that (exactly zero when p = q).
template <typename T, int NPL, bool FULL>
__global__ __launch_bounds__(kThreads) void fid_logits_half(focus_fidelity_desc d) {
  // every fused multiply-add below is written out: a product contracted into
  // one side of p - q but not the other would break the exact zero of p = q
#pragma clang fp contract(off)
  constexpr int kVec = 16 / sizeof(T);
  static_assert(NPL % kVec == 0, "whole 16-byte loads per lane");
  constexpr float kH = 0.5f * kLog2e;
  const int lane = threadIdx.x & 31;
  const int64_t t = (int64_t)blockIdx.x * (kThreads / 32) + (threadIdx.x >> 5);
  if (t >= d.n_pos) return;  // a whole half-wave: the cross-lane steps stay inside a half
  const int V = d.vocab;
  const T* pr = reinterpret_cast<const T*>(d.p) + t * V;
  const T* qr = reinterpret_cast<const T*>(d.q) + t * V;
  bool ok[NPL];
  float xp[NPL], xq[NPL];
#pragma unroll
  for (int c = 0; c < NPL / kVec; ++c) {
    const int i0 = c * 32 * kVec + lane * kVec;
    uint4 wp = make_uint4(0, 0, 0, 0), wq = wp;
    if (FULL || i0 < V) {
      wp = *reinterpret_cast<const uint4*>(pr + i0);
      wq = *reinterpret_cast<const uint4*>(qr + i0);
    }
    const T* ep = reinterpret_cast<const T*>(&wp);
    const T* eq = reinterpret_cast<const T*>(&wq);
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
      ok[c * kVec + j] = FULL || i0 < V;
      xp[c * kVec + j] = (float)ep[j];
      xq[c * kVec + j] = (float)eq[j];
    }
  }
  float mp = -INFINITY, mq = -INFINITY, np_ = INFINITY, nq = INFINITY;
#pragma unroll
  for (int k = 0; k < NPL; ++k)
    if (ok[k]) {
      mp = fmaxf(mp, xp[k]);
      mq = fmaxf(mq, xq[k]);
      np_ = fminf(np_, xp[k]);
      nq = fminf(nq, xq[k]);
    }
  mp = half_max(mp);
  mq = half_max(mq);
  np_ = half_min(np_);
  nq = half_min(nq);
  const float mph = mp * kH, mqh = mq * kH;
  // y = log2 of the unnormalised probability, halved; e = 2^y
  float yp[NPL], yq[NPL], ep[NPL], eq[NPL];
  float sp = 0.f, sq = 0.f;
#pragma unroll
  for (int k = 0; k < NPL; ++k) {
    yp[k] = fmaf(xp[k], kH, -mph);
    yq[k] = fmaf(xq[k], kH, -mqh);
    ep[k] = __builtin_amdgcn_exp2f(yp[k]);
    eq[k] = __builtin_amdgcn_exp2f(yq[k]);
    if (ok[k]) {
      sp = fmaf(ep[k], ep[k], sp);
      sq = fmaf(eq[k], eq[k], sq);
    }
  }
  sp = half_sum(sp);
  sq = half_sum(sq);
  const float rp = 1.f / sp, rq = 1.f / sq;
  const float lsp = __builtin_amdgcn_logf(sp), lsq = __builtin_amdgcn_logf(sq);
  const float emp = __builtin_amdgcn_exp2f(fmaf(np_, kH, -mph)), emq = __builtin_amdgcn_exp2f(fmaf(nq, kH, -mqh));
  const bool fast = emp * emp * rp >= 2.f * kClip && emq * emq * rq >= 2.f * kClip;

  float l1 = 0.f, l2 = 0.f, h = 0.f, js = 0.f, kl = 0.f;
  // one pair: probabilities pn, qn, their square roots a, b and base-2 logs lp, lq
  auto add = [&](float pn, float qn, float a, float b, float lp, float lq) __attribute__((always_inline)) {
    const float dd = pn - qn;
    l1 += fabsf(dd);
    l2 = fmaf(dd, dd, l2);
    const float sd = a - b;
    h = fmaf(sd, sd, h);
    const float r = lq - lp;
    kl = fmaf(pn, -r, kl);
    const float g = fmaxf(r, 0.f) + __builtin_amdgcn_logf(fmaf(0.5f, __builtin_amdgcn_exp2f(-fabsf(r)), 0.5f));
    js = fmaf(qn, r, js);
    js = fmaf(-(pn + qn), g, js);
  };
  if (fast) {
    const float srp = __builtin_amdgcn_sqrtf(rp), srq = __builtin_amdgcn_sqrtf(rq);
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      if (!ok[k]) continue;
      const float a = ep[k] * srp, b = eq[k] * srq;
      add(a * a, b * b, a, b, fmaf(yp[k], 2.f, -lsp), fmaf(yq[k], 2.f, -lsq));
    }
  } else {
    // the clip at 1e-12 and the renormalisation, as in fid_rows_wave
    float p[NPL], q[NPL];
    float cp = 0.f, cq = 0.f;
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      p[k] = fmaxf(ep[k] * ep[k] * rp, kClip);
      q[k] = fmaxf(eq[k] * eq[k] * rq, kClip);
      if (ok[k]) {
        cp += p[k];
        cq += q[k];
      }
    }
    cp = half_sum(cp);
    cq = half_sum(cq);
    const float rcp = 1.f / cp, rcq = 1.f / cq;
    const float lcp = __builtin_amdgcn_logf(cp), lcq = __builtin_amdgcn_logf(cq);
    const float lclip = __builtin_amdgcn_logf(kClip);
#pragma unroll
    for (int k = 0; k < NPL; ++k) {
      if (!ok[k]) continue;
      const float pn = p[k] * rcp, qn = q[k] * rcq;
      const float lp = (p[k] > kClip ? fmaf(yp[k], 2.f, -lsp) : lclip) - lcp;
      const float lq = (q[k] > kClip ? fmaf(yq[k], 2.f, -lsq) : lclip) - lcq;
      // pn, qn >= 1e-12 / 1.x: no denormals for the bare v_sqrt_f32
      add(pn, qn, __builtin_amdgcn_sqrtf(pn), __builtin_amdgcn_sqrtf(qn), lp, lq);
    }
  }
  Sums m;
  m.l1 = half_sum(l1);
  m.l2 = half_sum(l2);
  m.h = half_sum(h);
  m.js = half_sum(js);
  m.kl = half_sum(kl);
  if (lane == 0) m.store(d.out + t * FOCUS_FID_N);
}

// Mean of each metric over a sequence's positions: one workgroup per
// sequence, a fixed-order tree sum (deterministic).
__global__ __launch_bounds__(kThreads) void fid_seq_mean(focus_fidelity_desc d) {
  const int b = blockIdx.x;
  __shared__ float red[FOCUS_FID_N][kThreads];
  const int64_t t0 = d.cu_pos[b], t1 = d.cu_pos[b + 1];
  const bool ok = t0 >= 0 && t1 >= t0 && t1 <= d.n_pos;
  if (!ok && threadIdx.x == 0) focus::raise_err(d.err, FOCUS_ERR_BOUNDS);
  float acc[FOCUS_FID_N] = {0.f, 0.f, 0.f, 0.f, 0.f};
  if (ok)
    for (int64_t t = t0 + threadIdx.x; t < t1; t += kThreads)
#pragma unroll
      for (int m = 0; m < FOCUS_FID_N; ++m) acc[m] += d.out[t * FOCUS_FID_N + m];
#pragma unroll
  for (int m = 0; m < FOCUS_FID_N; ++m) red[m][threadIdx.x] = acc[m];
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s)
#pragma unroll
      for (int m = 0; m < FOCUS_FID_N; ++m) red[m][threadIdx.x] += red[m][threadIdx.x + s];
    __syncthreads();
  }
  if ((int)threadIdx.x < FOCUS_FID_N) {
    const int64_t n = ok ? t1 - t0 : 0;
    d.seq_mean[(int64_t)b * FOCUS_FID_N + threadIdx.x] = n > 0 ? red[threadIdx.x][0] / (float)n : 0.f;
  }
}

}  // namespace

extern "C" focus_status focus_fidelity(const focus_fidelity_desc* d, focus_stream_t stream) {
  if (!d) return FOCUS_E_NULL;
  if (d->dtype != FOCUS_BF16 && d->dtype != FOCUS_F32) return FOCUS_E_DTYPE;
  if (d->input_kind != FOCUS_FID_LOGITS && d->input_kind != FOCUS_FID_PROBS) return FOCUS_E_ARG;
  if (d->n_pos < 0 || d->vocab < 1 || d->n_seq < 0) return FOCUS_E_ARG;
  if (d->vocab > 64 * kMaxPerLane) return FOCUS_E_UNSUPPORTED;
  const bool want_mean = d->n_seq > 0 && d->seq_mean;
  if (want_mean && (!d->cu_pos || (d->n_pos > 0 && !d->out))) return FOCUS_E_ARG;
  if (d->n_pos > 0 && (!d->p || !d->q || !d->out)) return FOCUS_E_NULL;
  const uintptr_t ea = (uintptr_t)focus::elt_bytes(d->dtype) - 1;
  if ((reinterpret_cast<uintptr_t>(d->p) & ea) || (reinterpret_cast<uintptr_t>(d->q) & ea) ||
      (reinterpret_cast<uintptr_t>(d->out) & 3u) || (reinterpret_cast<uintptr_t>(d->seq_mean) & 3u) ||
      (reinterpret_cast<uintptr_t>(d->cu_pos) & 7u))
    return FOCUS_E_ARG;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (d->n_pos > 0) {
    const bool small = d->vocab <= kSmallV;
    const int64_t per_block = small ? kThreads : kThreads / 64;
    const int64_t blocks = focus::ceil_div(d->n_pos, per_block);
    if (blocks > INT32_MAX) return FOCUS_E_SHAPE;
    const dim3 grid((uint32_t)blocks), block(kThreads);
    // 16-byte row loads when every row starts 16-byte aligned
    const int64_t eb = focus::elt_bytes(d->dtype);
    const bool vec = (d->vocab * eb) % 16 == 0 && focus::aligned16(d->p) && focus::aligned16(d->q);
    const bool wide = d->vocab > 512;
#define FOCUS_FID_WAVE(T)                                                                        \
  if (wide) {                                                                                    \
    if (vec && d->vocab == 1024) hipLaunchKernelGGL((fid_rows_wave<T, true, 16, true>), grid, block, 0, s, *d);   \
    else if (vec) hipLaunchKernelGGL((fid_rows_wave<T, true, 16, false>), grid, block, 0, s, *d);  \
    else hipLaunchKernelGGL((fid_rows_wave<T, false, 16, false>), grid, block, 0, s, *d);          \
  } else {                                                                                       \
    if (vec && d->vocab == 512) hipLaunchKernelGGL((fid_rows_wave<T, true, 8, true>), grid, block, 0, s, *d);     \
    else if (vec) hipLaunchKernelGGL((fid_rows_wave<T, true, 8, false>), grid, block, 0, s, *d);   \
    else hipLaunchKernelGGL((fid_rows_wave<T, false, 8, false>), grid, block, 0, s, *d);           \
  }
    // logits rows of 64 < vocab <= 512 with 16-byte loads: two positions per wave
    const bool half = vec && d->input_kind == FOCUS_FID_LOGITS && d->vocab > 64 && d->vocab <= 512;
    const dim3 grid_h((uint32_t)focus::ceil_div(d->n_pos, kThreads / 32));
#define FOCUS_FID_HALF(T)                                                                                  \
  if (d->vocab == 512) hipLaunchKernelGGL((fid_logits_half<T, 16, true>), grid_h, block, 0, s, *d);         \
  else if (d->vocab > 256) hipLaunchKernelGGL((fid_logits_half<T, 16, false>), grid_h, block, 0, s, *d);    \
  else if (d->vocab == 256) hipLaunchKernelGGL((fid_logits_half<T, 8, true>), grid_h, block, 0, s, *d);     \
  else hipLaunchKernelGGL((fid_logits_half<T, 8, false>), grid_h, block, 0, s, *d);
    // four categories, rows aligned for one load each
    const bool rows4 = d->vocab == 4 && (reinterpret_cast<uintptr_t>(d->p) % (4 * eb)) == 0 &&
                       (reinterpret_cast<uintptr_t>(d->q) % (4 * eb)) == 0;
    if (d->dtype == FOCUS_BF16) {
      if (rows4) hipLaunchKernelGGL(fid_rows4<__bf16>, grid, block, 0, s, *d);
      else if (small) hipLaunchKernelGGL(fid_rows_small<__bf16>, grid, block, 0, s, *d);
      else if (half) { FOCUS_FID_HALF(__bf16) }
      else { FOCUS_FID_WAVE(__bf16) }
    } else {
      if (rows4) hipLaunchKernelGGL(fid_rows4<float>, grid, block, 0, s, *d);
      else if (small) hipLaunchKernelGGL(fid_rows_small<float>, grid, block, 0, s, *d);
      else if (half) { FOCUS_FID_HALF(float) }
      else { FOCUS_FID_WAVE(float) }
    }
#undef FOCUS_FID_WAVE
#undef FOCUS_FID_HALF
    focus_status st = focus::launch_status();
    if (st != FOCUS_OK) return st;
  }
  if (want_mean) {
    hipLaunchKernelGGL(fid_seq_mean, dim3(d->n_seq), dim3(kThreads), 0, s, *d);
    return focus::launch_status();
  }
  return FOCUS_OK;
}
