// Internal helpers shared by the FlashLoop HIP sources: status plumbing and exact numeric conversions.
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdarg>

#include "flashloop.h"

namespace fl {

// ---- host-side status ------------------------------------------------------------------------------
int set_error(int status, const char* fmt, ...);
int check_launch(const char* what);

#define FL_REQUIRE(cond, status, ...)                     \
  do {                                                    \
    if (!(cond)) return ::fl::set_error((status), __VA_ARGS__); \
  } while (0)

#define FL_API_BEGIN try {
#define FL_API_END                                                              \
  }                                                                             \
  catch (...) {                                                                 \
    return ::fl::set_error(FL_E_INTERNAL, "unexpected C++ exception");         \
  }

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// The optional index-list check (fl_set_index_checks / FL_CHECK_INDICES): n_lists lists of len entries,
// each strictly ascending within [lo, hi); FL_E_RANGE otherwise.  Synchronizes `st` and copies the lists to
// the host, so it is a debugging aid; FL_OK without any work when the check is off.
bool index_checks_on();
int check_index_lists(const char* fn, const char* name, const int32_t* list, int64_t n_lists, int len, int lo,
                      int hi, hipStream_t st);
// With the checks on: FL_E_RANGE unless every bf16 value of x[0..n) has magnitude <= 65504 (fits fp16).
int check_f16_range(const char* fn, const char* name, const uint16_t* x, int64_t n, hipStream_t st);
#define FL_CHECK_LIST(fn, name, list, n_lists, len, lo, hi, st)                                   \
  do {                                                                                            \
    const int fl_rc_ = ::fl::check_index_lists((fn), (name), (list), (n_lists), (len), (lo), (hi), (st)); \
    if (fl_rc_ != FL_OK) return fl_rc_;                                                           \
  } while (0)

// Top-k of `segments` key rows (fl_select.hip): segment s selects the k largest of keys[s * key_stride +
// 0..n-1] (ties to the lower position), writes their ids (cand[s * cand_stride + p], or id_base + p)
// ascending at out[s * out_stride + n_prefix ..], ids 0..n_prefix-1 first, and optionally the slot map.
int launch_topk(int segments, const float* keys, int64_t key_stride, int n, int k, const int32_t* cand,
                int64_t cand_stride, int id_base, int32_t* out, int64_t out_stride, int n_prefix,
                int32_t* slot, int slot_n, hipStream_t st);

// ---- device numerics -------------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// fp32 -> bf16 bit pattern, round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

// Bit pattern of a double that is exactly a finite binary16 value.
__device__ __forceinline__ uint32_t f16_bits_of_exact(double v) {
  uint32_t sign = signbit(v) ? 0x8000u : 0u;
  double a = fabs(v);
  if (a == 0.0) return sign;
  if (a < 0x1p-14) return sign | (uint32_t)(a * 0x1p24);      // subnormal: multiple of 2^-24
  int e;
  double m = frexp(a, &e);                                     // a = m * 2^e, m in [0.5, 1)
  uint32_t mant = (uint32_t)((m * 2.0 - 1.0) * 1024.0);        // exact
  return sign | ((uint32_t)(e - 1 + 15) << 10) | mant;
}

// Largest finite binary16 value <= x, saturating at -65504; a zero result is +0.
__device__ __forceinline__ double f16_down_value(double x) {
  if (x >= 65504.0) return 65504.0;
  if (x <= -65504.0) return -65504.0;
  double a = fabs(x);
  int sh = 24;                          // x * 2^sh counts fp16 spacings (2^-24 below the normal range)
  if (a >= 0x1p-14) {
    int e;
    frexp(a, &e);                       // a in [2^(e-1), 2^e): spacing 2^(e - 11) in that binade
    sh = 11 - e;
  }
  // floor(x / spacing) * spacing with both scalings as exponent shifts (exact: no division)
  const double v = ldexp(floor(ldexp(x, sh)), -sh);
  return v + 0.0;                            // -0 -> +0
}

__device__ __forceinline__ double f16_up_value(double x) {
  return -f16_down_value(-x) + 0.0;
}

// 64-lane wave reductions (xor butterflies).
__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ int wave_sum_i32(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

}  // namespace fl
