// Internal helpers shared by the FOCUS HIP sources (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "focus.h"

namespace focus {

// ---------------------------------------------------------------- host side

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline int64_t elt_bytes(int32_t dtype) {
  return dtype == FOCUS_BF16 ? 2 : dtype == FOCUS_F32 ? 4 : 0;
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

inline focus_status launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? FOCUS_OK : FOCUS_E_HIP;
}

// Number of XCDs (each with its own L2) blocks are dealt over, round robin.
constexpr int kXcds = 8;

// Compute units of the current device (256 if the query fails).
inline int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  return cus;
}

// --------------------------------------------------------------- device side

__device__ inline void raise_err(int32_t* err, int32_t bit) {
  if (err) atomicOr(err, bit);
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// bf16 -> f32 is exact: the bf16 bits are the high half of the f32.
__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// f32 -> bf16 bits, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 r;
  r[0] = (__bf16)lo;
  r[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, r);
}

// Cross-lane sums inside aligned groups of 4 / 8 lanes (DPP, no LDS traffic).
__device__ inline float dpp_xor1(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));
}
__device__ inline float dpp_xor2(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));
}
__device__ inline float dpp_half_mirror(float x) {  // lane i <-> lane 7-i within 8
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false));
}
__device__ inline float sum4(float x) {
  x += dpp_xor1(x);
  x += dpp_xor2(x);
  return x;
}
__device__ inline float sum8(float x) {
  x = sum4(x);
  x += dpp_half_mirror(x);
  return x;
}

}  // namespace focus
