// Building blocks shared by the attention kernels: buffer descriptors and LDS-DMA, waits and barriers,
// bf16 packing, cross-lane reductions of one query row, and the LDS layout of a column tile.
#pragma once

#include "fl_common.h"

#include <climits>

namespace fl {

constexpr int kBN = 32;            // columns per tile
// cache policy of the tile loads: non-temporal (the "nt" bit, 2 on gfx950); measured a few percent
// faster than the default policy on the 32K workload
constexpr int kDmaPolicy = 2;

typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
constexpr uint32_t kOOB = 0x80000000u;   // beyond every descriptor's range (ranges stay <= 2^31)
constexpr int kPad = INT_MAX;            // column id of a padding entry: fails every visibility test
#define FL_LDS(p) ((__attribute__((address_space(3))) void*)(p))
#define FL_LDS4(p) ((__attribute__((address_space(3))) i16x4*)(p))

__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// s_waitcnt vmcnt(n) with every other counter left alone (gfx9 encoding).
#define FL_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (7 << 4) | (15 << 8) | ((((n) >> 4) & 3) << 14))
// LDS traffic done, then a workgroup barrier without a memory fence (LDS-DMA waits are explicit).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
}

__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, f16x2));
}
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// two fp32 values to bf16 (round to nearest even), packed low | high << 16
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, bf16x2));
}

// max / sum of a lane and lane ^ 32 (the two half-waves hold disjoint columns of the same row)
__device__ __forceinline__ float xor32_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_add(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// One ring slot: the LDS-DMA target of one tile.  Column ids and flags live in separate arrays (never
// a DMA target), so the compiler's LDS-DMA tracking does not order them behind pending tile loads.
template <int D>
struct Slot {
  uint16_t k[kBN * D];     // row c at c*D, 16-byte chunks permuted (swz16_f, swz32_f)
  uint16_t v[kBN * D];     // same layout; converted in place from bf16 to fp16 before use
};

// Tile rows in LDS: the 16-byte chunk ch of row c sits at chunk position ch ^ g(c) (the LDS-DMA lanes
// fetch their global chunks in that order).  LDS reads are served 256 bytes (64 banks, 16 groups of 16
// bytes) at a time, so g spreads the rows one read instruction touches over the 16 groups.  For the
// 16x16x32 kernels: g is a bijection on 16 consecutive rows (the K reads: 16 rows x 16 B) whose halves
// g(c) >> 1 are distinct on 8 consecutive rows (the transposed V reads: 8 rows x 32 B).
template <int D>
__device__ __forceinline__ int swz16_f(int c) {
  if constexpr (D == 128) return ((c & 7) << 1) | ((c >> 3) & 1);
  else return (((c >> 1) & 3) << 1) | ((c >> 3) & 1);   // 128-byte rows: two rows share a 256-byte line
}
// For the 32x32x16 reads of loop_attn_kernel: a bijection on 16 consecutive rows (K: 16 rows x 16 B) whose
// quarters g(c) >> 2 are distinct on 4 consecutive rows (transposed V: 4 rows x 64 B).
template <int D>
__device__ __forceinline__ int swz32_f(int c) {
  if constexpr (D == 128) return ((c & 3) << 2) | ((c >> 2) & 3);
  else return (((c >> 1) & 1) << 2) | ((c >> 2) & 3);
}

__device__ __forceinline__ float xor16_max(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor16_add(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// max / sum over the four 16-lane rows of the wave (the lanes that hold one query row)
__device__ __forceinline__ float row4_max(float x) { return xor32_max(xor16_max(x)); }
__device__ __forceinline__ float row4_add(float x) { return xor32_add(xor16_add(x)); }

// max(x, y) for non-NaN inputs (-inf included) as a median with +inf; pinf holds +inf as a kernel
// argument, so the median is not folded back into a maximum with its NaN-quieting steps
__device__ __forceinline__ float fmax_nn(float x, float y, float pinf) { return __builtin_amdgcn_fmed3f(x, y, pinf); }

// Whether the segment kernels (fl_seg_attn.hip) cover a shape.
bool seg_supported(int k, int c_list, int window, int N, int d);

// Teams per workgroup of the segment kernel a shape takes (bh = B * H): 0 outside seg_supported, 1 for the
// one-team kernels, 2 for the two-team ones.  The launchers below choose by it.
int seg_teams(int k, int c_list, int window, int N, int d, int bh);

// Segment kernel of the subtract pass over the previous loop's state; FL_E_UNSUPPORTED without a launch
// outside seg_supported.
int launch_seg_sub(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, const uint16_t* v16,
                   const int32_t* rows, int k,
                   const int32_t* cols, int c_list, int window, int B, int N, int H, int d, float sm_scale,
                   const float* lse_ref, float* term_out, float* mass_out, hipStream_t st);

// Segment kernel of the add pass over current caches (fl_seg_attn.hip); FL_E_UNSUPPORTED without a launch
// when the shape is outside what it covers.
int launch_seg_cur(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, const uint16_t* v16,
                   const int32_t* rows, int k,
                   const int32_t* cols, int c_list, int window, int B, int N, int H, int d, float sm_scale,
                   float* lse_ref, float* o, const float* term_prev, const float* mass_prev,
                   const int32_t* slot_prev, int k_prev, float* term_out, float* mass_out, hipStream_t st);

}  // namespace fl
