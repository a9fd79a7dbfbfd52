// Cross-loop K/V residual codec: Section 4.3, Eq. 4; Appendix D.3, Eq. 8; quantizer of Appendix E.
//
// All kernels stream rows with 16-byte loads: one thread owns 8 consecutive channels of a row, so codes
// of those channels form one 2/4/8-byte word (LSB-first packing) and metadata loads are 2 or 16 bytes.
//   quant_token   (keys, per-channel groups of G packed rows): a 256-thread workgroup owns one group of
//                 rows x 256 channels; 8 row slices reduce min/max through LDS, then the same threads
//                 encode their rows from registers (no second pass over HBM).
//   quant_channel (values, per-token groups of G channels): the G/8 threads of a group reduce min/max
//                 with lane shuffles.
//   dequant       rebuilds bf16(x_hat + z + q*s) rows, compact or in place.
// Both quantizers optionally write the reconstructed rows (fusing the compact dequantization).
#include "fl_common.h"

namespace fl {

struct Row8 {
  float v[8];
};

__device__ __forceinline__ Row8 load_bf16x8(const uint16_t* p) {
  uint4 w = *reinterpret_cast<const uint4*>(p);
  const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
  Row8 r;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    r.v[2 * t] = __uint_as_float(ws[t] << 16);
    r.v[2 * t + 1] = __uint_as_float(ws[t] & 0xFFFF0000u);
  }
  return r;
}

__device__ __forceinline__ void store_bf16x8(uint16_t* p, const Row8& r) {
  uint32_t ws[4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
    ws[t] = f32_to_bf16_rne(r.v[2 * t]) | (f32_to_bf16_rne(r.v[2 * t + 1]) << 16);
  *reinterpret_cast<uint4*>(p) = make_uint4(ws[0], ws[1], ws[2], ws[3]);
}

// Two fp32 values to packed fp16 (round to nearest even; v_cvt_pk_f16_f32, the conversion the attention
// kernels apply to bf16 value rows in LDS).
__device__ __forceinline__ uint32_t f16x2_bits(float a, float b) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){a, b}, h2));
}

// Eight bf16 values (as packed bits) to fp16.
__device__ __forceinline__ uint4 bf16x8_to_f16(uint4 w) {
  const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
  uint32_t o[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) o[t] = f16x2_bits(__uint_as_float(ws[t] << 16), __uint_as_float(ws[t] & 0xFFFF0000u));
  return make_uint4(o[0], o[1], o[2], o[3]);
}

// The fp16 copy of a row chunk as store_bf16x8 writes it: each value rounded to bf16 first, then to fp16.
__device__ __forceinline__ void store_f16x8_of_bf16(uint16_t* p, const Row8& r) {
  uint32_t o[4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
    o[t] = f16x2_bits(__uint_as_float(f32_to_bf16_rne(r.v[2 * t]) << 16),
                      __uint_as_float(f32_to_bf16_rne(r.v[2 * t + 1]) << 16));
  *reinterpret_cast<uint4*>(p) = make_uint4(o[0], o[1], o[2], o[3]);
}

// Reciprocal of a metadata scale for encode1 (within 1 ulp; s is an fp16 value, so 1/s is a normal fp32).
__device__ __forceinline__ float scale_rcp(float s) { return __builtin_amdgcn_rcpf(s); }

// Encode one value: q = clamp(rint(fp32(fp32(delta - z) / s)), 0, qmax), 0 when s == 0, with rs = scale_rcp(s).
// No division: q1 = a rs, e = a - q1 s (one fma, exact), q2 = e rs + q1 (one fma) is Markstein's correction
// step (P. Markstein, IBM J. Res. Dev. 34(1), 1990), within |a/s| 2^-45 of a/s.  The scale s is an fp16
// value (at most 11 significant bits) and a an fp32 value, so a - (m + 1/2) s is a multiple of a power of
// two that keeps a/s either exactly at a half-integer m + 1/2 or more than half an ulp away from it (by
// 2^-11 of that half ulp at least): rint(q2) is rint of the correctly rounded quotient, the IEEE division's
// code, bit for bit (checked in exact arithmetic on the host, ties and fp32 neighbours of every boundary).
__device__ __forceinline__ uint32_t encode1(float delta, float z, float s, float rs, int qmax) {
  const float a = delta - z;
  const float q1 = a * rs;
  const float e = __builtin_fmaf(-q1, s, a);
  float t = __builtin_fmaf(e, rs, q1);
  t = __builtin_rintf(t);
  t = fminf(fmaxf(t, 0.0f), (float)qmax);
  return s == 0.0f ? 0u : (uint32_t)t;
}

template <int BITS>
__device__ __forceinline__ void store_codes8(uint8_t* dst, const uint32_t q[8]) {
  if constexpr (BITS == 8) {
    uint32_t lo = q[0] | (q[1] << 8) | (q[2] << 16) | (q[3] << 24);
    uint32_t hi = q[4] | (q[5] << 8) | (q[6] << 16) | (q[7] << 24);
    *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
  } else {
    uint32_t w = 0;
#pragma unroll
    for (int t = 0; t < 8; ++t) w |= q[t] << (t * BITS);
    if constexpr (BITS == 4) *reinterpret_cast<uint32_t*>(dst) = w;
    else *reinterpret_cast<uint16_t*>(dst) = (uint16_t)w;
  }
}

template <int BITS>
__device__ __forceinline__ void load_codes8(const uint8_t* src, uint32_t q[8]) {
  constexpr uint32_t mask = (1u << BITS) - 1u;
  if constexpr (BITS == 8) {
    uint2 w = *reinterpret_cast<const uint2*>(src);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      q[t] = (w.x >> (8 * t)) & mask;
      q[t + 4] = (w.y >> (8 * t)) & mask;
    }
  } else {
    uint32_t w = (BITS == 4) ? *reinterpret_cast<const uint32_t*>(src)
                             : (uint32_t)*reinterpret_cast<const uint16_t*>(src);
#pragma unroll
    for (int t = 0; t < 8; ++t) q[t] = (w >> (t * BITS)) & mask;
  }
}

// Group metadata from fp32 min/max: z = fp16 down(min), s = fp16 up((max - z) / qmax), both fp64.
__device__ __forceinline__ void group_meta(float mn, float mx, int qmax, double& z, double& s) {
  z = f16_down_value((double)mn);
  s = f16_up_value(((double)mx - z) / (double)qmax);
}

// ---- keys: per-channel groups along packed rows ----------------------------------------------------
// A workgroup of 256 threads = S row slices x CH chunks of 8 channels; each slice holds RPS = G/S rows.
// S = min(G, 32), so a group of 64 rows spreads over 32 slices and a workgroup covers 64 channels.

// out_rows: compact [B, k, HD] rows, or (commit) the cache rows idx of x_ref itself, written in place
// (every element is read before the same thread writes it, after the workgroup's reduction).
// Body of one workgroup: channel block bx, row group g, batch b.
template <int BITS, int S, int RPS>
__device__ __forceinline__ void quant_token_body(
    const uint16_t* __restrict__ x_cur, const uint16_t* x_ref,
    const int32_t* __restrict__ idx, int k, int N, int HD, int G, uint8_t* __restrict__ codes,
    uint16_t* __restrict__ scale, uint16_t* __restrict__ zero, uint16_t* out_rows, bool commit,
    int bx, int g, int b) {
  constexpr int CH = 256 / S;          // chunks of 8 channels per workgroup
  __shared__ float s_mn[S][CH * 8];
  __shared__ float s_mx[S][CH * 8];
  __shared__ float s_z[CH * 8];
  __shared__ float s_s[CH * 8];
  constexpr int qmax = (1 << BITS) - 1;
  const int slice = threadIdx.x / CH, chunk = threadIdx.x % CH;
  const int c0 = bx * (CH * 8) + chunk * 8;
  const bool ch_ok = c0 < HD;
  const int ng = (k + G - 1) / G;

  float dl[RPS][8];
  uint4 ref_raw[RPS];
  int64_t roff[RPS];                   // element offset of each row in x_ref
  float mn[8], mx[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) { mn[t] = INFINITY; mx[t] = -INFINITY; }
#pragma unroll
  for (int j = 0; j < RPS; ++j) {
    const int p = g * G + slice * RPS + j;
    ref_raw[j] = make_uint4(0, 0, 0, 0);
    roff[j] = 0;
    if (ch_ok && p < k) {
      const int64_t i = idx ? (int64_t)idx[(int64_t)b * k + p] : (int64_t)p;
      const int64_t off = ((int64_t)b * N + i) * HD + c0;
      roff[j] = off;
      Row8 c = load_bf16x8(x_cur + off);
      Row8 r{};
      if (x_ref) {
        ref_raw[j] = *reinterpret_cast<const uint4*>(x_ref + off);
        r = load_bf16x8(x_ref + off);
      }
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        dl[j][t] = c.v[t] - r.v[t];
        mn[t] = fminf(mn[t], dl[j][t]);
        mx[t] = fmaxf(mx[t], dl[j][t]);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    s_mn[slice][chunk * 8 + t] = mn[t];
    s_mx[slice][chunk * 8 + t] = mx[t];
  }
  __syncthreads();
  if (threadIdx.x < CH * 8) {
    const int ch = threadIdx.x;   // one thread per channel
    const int c = bx * (CH * 8) + ch;
    float a = INFINITY, bb = -INFINITY;
#pragma unroll
    for (int sl = 0; sl < S; ++sl) {
      a = fminf(a, s_mn[sl][ch]);
      bb = fmaxf(bb, s_mx[sl][ch]);
    }
    double z = 0.0, s = 0.0;
    if (c < HD) {
      group_meta(a, bb, qmax, z, s);
      const int64_t m = ((int64_t)b * ng + g) * HD + c;
      zero[m] = (uint16_t)f16_bits_of_exact(z);
      scale[m] = (uint16_t)f16_bits_of_exact(s);
    }
    s_z[ch] = (float)z;
    s_s[ch] = (float)s;
  }
  __syncthreads();
  if (!ch_ok) return;
  float z8[8], s8[8], r8[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    z8[t] = s_z[chunk * 8 + t];
    s8[t] = s_s[chunk * 8 + t];
    r8[t] = scale_rcp(s8[t]);
  }
  const int row_bytes = HD * BITS / 8;
#pragma unroll
  for (int j = 0; j < RPS; ++j) {
    const int p = g * G + slice * RPS + j;
    if (p >= k) break;
    uint32_t q[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) q[t] = encode1(dl[j][t], z8[t], s8[t], r8[t], qmax);
    store_codes8<BITS>(codes + ((int64_t)b * k + p) * row_bytes + c0 * BITS / 8, q);
    if (out_rows) {
      const uint32_t rw[4] = {ref_raw[j].x, ref_raw[j].y, ref_raw[j].z, ref_raw[j].w};
      Row8 o;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        float ref = (t & 1) ? __uint_as_float(rw[t >> 1] & 0xFFFF0000u) : __uint_as_float(rw[t >> 1] << 16);
        float dq = z8[t] + (float)q[t] * s8[t];     // q * s exact in fp32: one rounding
        o.v[t] = ref + dq;
      }
      store_bf16x8(out_rows + (commit ? roff[j] : ((int64_t)b * k + p) * HD + c0), o);
    }
  }
}

template <int BITS, int S, int RPS>
__global__ __launch_bounds__(256) void quant_token_kernel(
    const uint16_t* __restrict__ x_cur, const uint16_t* x_ref,
    const int32_t* __restrict__ idx, int k, int N, int HD, int G, uint8_t* __restrict__ codes,
    uint16_t* __restrict__ scale, uint16_t* __restrict__ zero, uint16_t* out_rows, bool commit) {
  quant_token_body<BITS, S, RPS>(x_cur, x_ref, idx, k, N, HD, G, codes, scale, zero, out_rows, commit,
                                 blockIdx.x, blockIdx.y, blockIdx.z);
}

// ---- values: per-token groups of G channels ----------------------------------------------------------
// out_rows as for quant_token_kernel (each element is read and written by one thread).
// Body of one thread: 8-channel chunk `local` of the k * HD / 8 chunks of batch b.
template <int BITS>
__device__ __forceinline__ void quant_channel_body(
    const uint16_t* __restrict__ x_cur, const uint16_t* x_ref,
    const int32_t* __restrict__ idx, int k, int N, int HD, int G, uint8_t* __restrict__ codes,
    uint16_t* __restrict__ scale, uint16_t* __restrict__ zero, uint16_t* out_rows, bool commit,
    int64_t local, int b, uint16_t* out_f16 = nullptr) {
  constexpr int qmax = (1 << BITS) - 1;
  const int chunks = HD / 8;
  const bool ok = local < (int64_t)k * chunks;
  const int p = ok ? (int)(local / chunks) : 0;
  const int chunk = ok ? (int)(local % chunks) : 0;
  const int c0 = chunk * 8;
  float dl[8];
  uint4 ref_raw = make_uint4(0, 0, 0, 0);
  float mn = INFINITY, mx = -INFINITY;
  int64_t roff = 0;
  if (ok) {
    const int64_t i = idx ? (int64_t)idx[(int64_t)b * k + p] : (int64_t)p;
    const int64_t off = ((int64_t)b * N + i) * HD + c0;
    roff = off;
    Row8 c = load_bf16x8(x_cur + off);
    Row8 r{};
    if (x_ref) {
      ref_raw = *reinterpret_cast<const uint4*>(x_ref + off);
      r = load_bf16x8(x_ref + off);
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      dl[t] = c.v[t] - r.v[t];
      mn = fminf(mn, dl[t]);
      mx = fmaxf(mx, dl[t]);
    }
  }
  // reduce across the G/8 consecutive lanes of the group (groups never straddle a wave)
  for (int off = 1; off < G / 8; off <<= 1) {
    mn = fminf(mn, __shfl_xor(mn, off, 64));
    mx = fmaxf(mx, __shfl_xor(mx, off, 64));
  }
  if (!ok) return;
  double z, s;
  group_meta(mn, mx, qmax, z, s);
  if ((chunk % (G / 8)) == 0) {
    const int64_t m = ((int64_t)b * k + p) * (HD / G) + c0 / G;
    zero[m] = (uint16_t)f16_bits_of_exact(z);
    scale[m] = (uint16_t)f16_bits_of_exact(s);
  }
  const float z32 = (float)z, s32 = (float)s, r32 = scale_rcp(s32);
  uint32_t q[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) q[t] = encode1(dl[t], z32, s32, r32, qmax);
  store_codes8<BITS>(codes + ((int64_t)b * k + p) * (HD * BITS / 8) + c0 * BITS / 8, q);
  if (out_rows) {
    const uint32_t rw[4] = {ref_raw.x, ref_raw.y, ref_raw.z, ref_raw.w};
    Row8 o;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      float ref = (t & 1) ? __uint_as_float(rw[t >> 1] & 0xFFFF0000u) : __uint_as_float(rw[t >> 1] << 16);
      o.v[t] = ref + (z32 + (float)q[t] * s32);
    }
    store_bf16x8(out_rows + (commit ? roff : ((int64_t)b * k + p) * HD + c0), o);
    if (out_f16) store_f16x8_of_bf16(out_f16 + roff, o);   // (commit only: the cache row's fp16 copy)
  }
}

template <int BITS>
__global__ __launch_bounds__(256) void quant_channel_kernel(
    const uint16_t* __restrict__ x_cur, const uint16_t* x_ref,
    const int32_t* __restrict__ idx, int k, int N, int HD, int G, uint8_t* __restrict__ codes,
    uint16_t* __restrict__ scale, uint16_t* __restrict__ zero, uint16_t* out_rows, bool commit) {
  quant_channel_body<BITS>(x_cur, x_ref, idx, k, N, HD, G, codes, scale, zero, out_rows, commit,
                           (int64_t)blockIdx.x * blockDim.x + threadIdx.x, blockIdx.y);
}

// ---- keys and values in one launch -------------------------------------------------------------------
// The first kx * ky * B workgroups run the key body (token axis), the rest the value body (channel
// axis), so the two short streams share one launch instead of two dependent ones.
struct QuantKV {
  const uint16_t* k_cur;
  const uint16_t* k_ref;
  const uint16_t* v_cur;
  const uint16_t* v_ref;
  const int32_t* idx;
  uint8_t* k_codes;
  uint16_t* k_scale;
  uint16_t* k_zero;
  uint8_t* v_codes;
  uint16_t* v_scale;
  uint16_t* v_zero;
  uint16_t* k_rows;
  uint16_t* v_rows;
  uint16_t* v_f16;     // optional (commit): fp16 copy of the value cache, rows idx rewritten
  int k, N, HD, G;
  int kx, ky, vx;      // key workgroups per (row group, batch) and row groups; value workgroups per batch
  int commit;
};

template <int BITS, int S, int RPS>
__global__ __launch_bounds__(256) void quant_kv_kernel(QuantKV a) {
  const int nkb = a.kx * a.ky;
  const int blk = blockIdx.x;
  const int b = blk / (nkb + a.vx);
  const int r = blk - b * (nkb + a.vx);
  if (r < nkb) {
    quant_token_body<BITS, S, RPS>(a.k_cur, a.k_ref, a.idx, a.k, a.N, a.HD, a.G, a.k_codes, a.k_scale,
                                   a.k_zero, a.k_rows, a.commit != 0, r % a.kx, r / a.kx, b);
  } else {
    quant_channel_body<BITS>(a.v_cur, a.v_ref, a.idx, a.k, a.N, a.HD, a.G, a.v_codes, a.v_scale, a.v_zero,
                             a.v_rows, a.commit != 0, (int64_t)(r - nkb) * 256 + threadIdx.x, b, a.v_f16);
  }
}

// ---- bits = 16: the payload is the raw state ---------------------------------------------------------
__global__ __launch_bounds__(256) void passthrough_kernel(const uint16_t* __restrict__ x_cur,
                                                          const int32_t* __restrict__ idx, int k,
                                                          int N, int HD, uint8_t* __restrict__ codes,
                                                          uint16_t* __restrict__ out_rows, bool commit) {
  const int chunks = HD / 8;
  const int64_t local = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int b = blockIdx.y;
  if (local >= (int64_t)k * chunks) return;
  const int p = (int)(local / chunks), c0 = (int)(local % chunks) * 8;
  const int64_t i = idx ? (int64_t)idx[(int64_t)b * k + p] : (int64_t)p;
  uint4 w = *reinterpret_cast<const uint4*>(x_cur + ((int64_t)b * N + i) * HD + c0);
  *reinterpret_cast<uint4*>(codes + (((int64_t)b * k + p) * HD + c0) * 2) = w;
  if (out_rows)
    *reinterpret_cast<uint4*>(out_rows + (commit ? ((int64_t)b * N + i) * HD : ((int64_t)b * k + p) * HD) + c0) = w;
}

// ---- dequantization / reconstruction ------------------------------------------------------------------
// One thread: 8-channel chunk `local` of the k * HD / 8 chunks of batch b.
template <int BITS, int AXIS>
__device__ __forceinline__ void dequant_body(
    const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scale,
    const uint16_t* __restrict__ zero, const int32_t* __restrict__ idx, int k, int N, int HD, int G,
    uint16_t* x_hat, uint16_t* out_rows, int64_t local, int b) {
  const int chunks = HD / 8;
  if (local >= (int64_t)k * chunks) return;
  const int p = (int)(local / chunks), c0 = (int)(local % chunks) * 8;
  const int64_t i = idx ? (int64_t)idx[(int64_t)b * k + p] : (int64_t)p;
  const int64_t xoff = ((int64_t)b * N + i) * HD + c0;
  uint16_t* dst = out_rows ? out_rows + ((int64_t)b * k + p) * HD + c0 : x_hat + xoff;
  if constexpr (BITS == 16) {
    *reinterpret_cast<uint4*>(dst) =
        *reinterpret_cast<const uint4*>(codes + (((int64_t)b * k + p) * HD + c0) * 2);
  } else {
    uint32_t q[8];
    load_codes8<BITS>(codes + ((int64_t)b * k + p) * (HD * BITS / 8) + c0 * BITS / 8, q);
    float z8[8], s8[8];
    if constexpr (AXIS == FL_AXIS_TOKEN) {
      const int ng = (k + G - 1) / G;
      const int64_t m = ((int64_t)b * ng + p / G) * HD + c0;
      uint4 zw = *reinterpret_cast<const uint4*>(zero + m);
      uint4 sw = *reinterpret_cast<const uint4*>(scale + m);
      const uint32_t za[4] = {zw.x, zw.y, zw.z, zw.w}, sa[4] = {sw.x, sw.y, sw.z, sw.w};
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        z8[t] = f16_bits_to_f32((t & 1) ? (za[t >> 1] >> 16) : (za[t >> 1] & 0xFFFFu));
        s8[t] = f16_bits_to_f32((t & 1) ? (sa[t >> 1] >> 16) : (sa[t >> 1] & 0xFFFFu));
      }
    } else {
      const int64_t m = ((int64_t)b * k + p) * (HD / G) + c0 / G;
      const float z = f16_bits_to_f32(zero[m]), s = f16_bits_to_f32(scale[m]);
#pragma unroll
      for (int t = 0; t < 8; ++t) { z8[t] = z; s8[t] = s; }
    }
    Row8 x = load_bf16x8(x_hat + xoff);
    Row8 o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o.v[t] = x.v[t] + (z8[t] + (float)q[t] * s8[t]);
    store_bf16x8(dst, o);
  }
}

template <int BITS, int AXIS>
__global__ __launch_bounds__(256) void dequant_kernel(
    const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scale,
    const uint16_t* __restrict__ zero, const int32_t* __restrict__ idx, int k, int N, int HD, int G,
    uint16_t* x_hat, uint16_t* out_rows) {
  dequant_body<BITS, AXIS>(codes, scale, zero, idx, k, N, HD, G, x_hat, out_rows,
                           (int64_t)blockIdx.x * blockDim.x + threadIdx.x, blockIdx.y);
}

// Keys (token axis) in workgroups [0, half) and values (channel axis) in [half, 2 half) of one launch.
struct DequantKV {
  const uint8_t* k_codes;
  const uint16_t* k_scale;
  const uint16_t* k_zero;
  const uint8_t* v_codes;
  const uint16_t* v_scale;
  const uint16_t* v_zero;
  const int32_t* idx;
  uint16_t* k_hat;
  uint16_t* v_hat;
  uint16_t* k_rows;
  uint16_t* v_rows;
  int k, N, HD, G, half;
};

template <int BITS>
__global__ __launch_bounds__(256) void dequant_kv_kernel(DequantKV a) {
  const int bx = blockIdx.x;
  if (bx < a.half)
    dequant_body<BITS, FL_AXIS_TOKEN>(a.k_codes, a.k_scale, a.k_zero, a.idx, a.k, a.N, a.HD, a.G, a.k_hat,
                                      a.k_rows, (int64_t)bx * 256 + threadIdx.x, blockIdx.y);
  else
    dequant_body<BITS, FL_AXIS_CHANNEL>(a.v_codes, a.v_scale, a.v_zero, a.idx, a.k, a.N, a.HD, a.G, a.v_hat,
                                        a.v_rows, (int64_t)(bx - a.half) * 256 + threadIdx.x, blockIdx.y);
}

static int check_codec_args(const char* fn, const void* codes, const void* a, int k, int B, int N,
                            int H, int d, int bits, int group, int axis, bool need_meta,
                            const void* scale, const void* zero, const void* idx) {
  FL_REQUIRE((codes || k == 0) && a, FL_E_NULL, "%s: codes and the state pointer are required", fn);
  FL_REQUIRE(B >= 1 && N >= 1 && H >= 1, FL_E_SHAPE, "%s: need B, N, H >= 1", fn);
  FL_REQUIRE(d == 64 || d == 128, FL_E_SHAPE, "%s: head dim %d not in {64, 128}", fn, d);
  FL_REQUIRE((int64_t)N * H * d < ((int64_t)1 << 31), FL_E_SHAPE, "%s: N * H * d too large", fn);
  FL_REQUIRE(idx != nullptr || k == N || k == 0, FL_E_SHAPE, "%s: without idx, k must equal N", fn);
  FL_REQUIRE(k >= 0 && k <= N, FL_E_RANGE, "%s: k=%d outside [0, N]", fn, k);
  FL_REQUIRE(bits == 2 || bits == 4 || bits == 8 || bits == 16, FL_E_UNSUPPORTED,
             "%s: bits=%d not in {2, 4, 8, 16}", fn, bits);
  FL_REQUIRE(axis == FL_AXIS_TOKEN || axis == FL_AXIS_CHANNEL, FL_E_UNSUPPORTED, "%s: bad axis %d", fn, axis);
  if (bits != 16) {
    FL_REQUIRE(group >= 8 && group <= 128 && group % 8 == 0 && (group & (group - 1)) == 0,
               FL_E_UNSUPPORTED, "%s: group=%d must be a power of two in [8, 128]", fn, group);
    FL_REQUIRE(axis == FL_AXIS_TOKEN || d % group == 0, FL_E_SHAPE,
               "%s: CHANNEL axis needs group | d (group=%d, d=%d)", fn, group, d);
    if (need_meta && k > 0) FL_REQUIRE(scale && zero, FL_E_NULL, "%s: scale and zero are required", fn);
  }
  return FL_OK;
}

static int residual_quant(const char* fn, const uint16_t* x_cur, const uint16_t* x_ref, const int32_t* idx,
                          int k, int B, int N, int H, int d, int bits, int group, int axis, uint8_t* codes,
                          uint16_t* scale, uint16_t* zero, uint16_t* out_rows, bool commit, void* stream) {
  int rc = check_codec_args(fn, codes, x_cur, k, B, N, H, d, bits, group, axis, true, scale, zero, idx);
  if (rc != FL_OK) return rc;
  if (k == 0) return FL_OK;
  hipStream_t st = as_stream(stream);
  FL_CHECK_LIST(fn, "idx", idx, B, k, 0, N, st);
  const int HD = H * d;
  if (bits == 16) {
    dim3 grid((unsigned)(((int64_t)k * (HD / 8) + 255) / 256), B);
    passthrough_kernel<<<grid, 256, 0, st>>>(x_cur, idx, k, N, HD, codes, out_rows, commit);
    return check_launch("passthrough_kernel");
  }
  if (axis == FL_AXIS_TOKEN) {
    const int slices = group < 32 ? group : 32;
    const int cw = 256 / slices * 8;                      // channels per workgroup
    dim3 grid((HD + cw - 1) / cw, (k + group - 1) / group, B);
#define FL_QT(BB, SS, RR)                                                                          \
  quant_token_kernel<BB, SS, RR><<<grid, 256, 0, st>>>(x_cur, x_ref, idx, k, N, HD, group, codes, \
                                                       scale, zero, out_rows, commit)
#define FL_QT_BITS(BB)                                   \
  switch (group) {                                       \
    case 8: FL_QT(BB, 8, 1); break;                      \
    case 16: FL_QT(BB, 16, 1); break;                    \
    case 32: FL_QT(BB, 32, 1); break;                    \
    case 64: FL_QT(BB, 32, 2); break;                    \
    default: FL_QT(BB, 32, 4); break;                    \
  }
    if (bits == 2) { FL_QT_BITS(2) } else if (bits == 4) { FL_QT_BITS(4) } else { FL_QT_BITS(8) }
#undef FL_QT_BITS
#undef FL_QT
    return check_launch("quant_token_kernel");
  }
  dim3 grid((unsigned)(((int64_t)k * (HD / 8) + 255) / 256), B);
#define FL_QC(BB) \
  quant_channel_kernel<BB><<<grid, 256, 0, st>>>(x_cur, x_ref, idx, k, N, HD, group, codes, scale, zero, out_rows, commit)
  if (bits == 2) FL_QC(2);
  else if (bits == 4) FL_QC(4);
  else FL_QC(8);
#undef FL_QC
  return check_launch("quant_channel_kernel");
}

// Keys (token axis) and values (channel axis) with one bit width and group size.  out rows: compact
// k_rows / v_rows (each optional), or with commit the rows idx of k_ref / v_ref in place.
// ---- fp16 copy of rows of a bf16 [B, N, HD] tensor (all rows, or rows idx) ------------------------------
__global__ __launch_bounds__(256) void f16_rows_kernel(const uint16_t* __restrict__ x, const int32_t* __restrict__ idx,
                                                       int k, int N, int HD, uint16_t* __restrict__ y) {
  const int b = blockIdx.y;
  const int chunks = HD / 8;
  const int64_t local = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (local >= (int64_t)k * chunks) return;
  const int p = (int)(local / chunks), c = (int)(local % chunks);
  const int64_t i = idx ? (int64_t)idx[(int64_t)b * k + p] : (int64_t)p;
  const int64_t off = ((int64_t)b * N + i) * HD + (int64_t)c * 8;
  *reinterpret_cast<uint4*>(y + off) = bf16x8_to_f16(*reinterpret_cast<const uint4*>(x + off));
}

static int launch_f16_rows(const uint16_t* x, const int32_t* idx, int k, int B, int N, int HD, uint16_t* y,
                           hipStream_t st) {
  if (k == 0) return FL_OK;
  dim3 grid((unsigned)(((int64_t)k * (HD / 8) + 255) / 256), B);
  f16_rows_kernel<<<grid, 256, 0, st>>>(x, idx, k, N, HD, y);
  return check_launch("f16_rows_kernel");
}

static int residual_quant_kv(const char* fn, const uint16_t* k_cur, uint16_t* k_ref, const uint16_t* v_cur,
                             uint16_t* v_ref, const int32_t* idx, int k, int B, int N, int H, int d, int bits,
                             int group, uint8_t* k_codes, uint16_t* k_scale, uint16_t* k_zero, uint8_t* v_codes,
                             uint16_t* v_scale, uint16_t* v_zero, uint16_t* k_rows, uint16_t* v_rows, bool commit,
                             uint16_t* v_f16,
                             void* stream) {
  int rc = check_codec_args(fn, k_codes, k_cur, k, B, N, H, d, bits, group, FL_AXIS_TOKEN, true, k_scale,
                            k_zero, idx);
  if (rc != FL_OK) return rc;
  rc = check_codec_args(fn, v_codes, v_cur, k, B, N, H, d, bits, group, FL_AXIS_CHANNEL, true, v_scale, v_zero,
                        idx);
  if (rc != FL_OK) return rc;
  if (k == 0) return FL_OK;
  if (bits == 16) {   // raw payload: two copy launches
    rc = residual_quant(fn, k_cur, k_ref, idx, k, B, N, H, d, bits, group, FL_AXIS_TOKEN, k_codes, k_scale,
                        k_zero, commit ? k_ref : k_rows, commit, stream);
    if (rc != FL_OK) return rc;
    rc = residual_quant(fn, v_cur, v_ref, idx, k, B, N, H, d, bits, group, FL_AXIS_CHANNEL, v_codes, v_scale,
                        v_zero, commit ? v_ref : v_rows, commit, stream);
    if (rc != FL_OK || !v_f16) return rc;
    return launch_f16_rows(v_ref, idx, k, B, N, H * d, v_f16, as_stream(stream));
  }
  const int HD = H * d;
  const int slices = group < 32 ? group : 32;
  const int cw = 256 / slices * 8;
  QuantKV a;
  a.k_cur = k_cur; a.k_ref = k_ref; a.v_cur = v_cur; a.v_ref = v_ref; a.idx = idx;
  a.k_codes = k_codes; a.k_scale = k_scale; a.k_zero = k_zero;
  a.v_codes = v_codes; a.v_scale = v_scale; a.v_zero = v_zero;
  a.k_rows = commit ? k_ref : k_rows;
  a.v_rows = commit ? v_ref : v_rows;
  a.v_f16 = commit ? v_f16 : nullptr;
  a.k = k; a.N = N; a.HD = HD; a.G = group;
  a.kx = (HD + cw - 1) / cw;
  a.ky = (k + group - 1) / group;
  a.vx = (int)(((int64_t)k * (HD / 8) + 255) / 256);
  a.commit = commit ? 1 : 0;
  const int64_t blocks = ((int64_t)a.kx * a.ky + a.vx) * B;
  FL_REQUIRE(blocks < ((int64_t)1 << 31), FL_E_SHAPE, "%s: grid too large", fn);
  hipStream_t st = as_stream(stream);
  FL_CHECK_LIST(fn, "idx", idx, B, k, 0, N, st);
#define FL_QKV(BB, SS, RR) quant_kv_kernel<BB, SS, RR><<<(unsigned)blocks, 256, 0, st>>>(a)
#define FL_QKV_BITS(BB)                                   \
  switch (group) {                                        \
    case 8: FL_QKV(BB, 8, 1); break;                      \
    case 16: FL_QKV(BB, 16, 1); break;                    \
    case 32: FL_QKV(BB, 32, 1); break;                    \
    case 64: FL_QKV(BB, 32, 2); break;                    \
    default: FL_QKV(BB, 32, 4); break;                    \
  }
  if (bits == 2) { FL_QKV_BITS(2) } else if (bits == 4) { FL_QKV_BITS(4) } else { FL_QKV_BITS(8) }
#undef FL_QKV_BITS
#undef FL_QKV
  return check_launch("quant_kv_kernel");
}


// The most recent tokens stay in bf16 (Appendix E): rows i >= N - tail among the active rows are stored as
// the exact X^(r) rows, in the caches and/or the compact rows (their codes are formed with the others).
// idx ascends, so only its last min(k, tail) entries can be tail rows: one thread per 16-byte chunk of those.
__global__ __launch_bounds__(256) void keep_recent_kernel(const uint16_t* __restrict__ x_cur,
                                                          const int32_t* __restrict__ idx, int k, int N, int HD,
                                                          int lo, int n_last, uint16_t* cache, uint16_t* rows) {
  const int b = blockIdx.y;
  const int chunks = HD / 8;
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (x >= (int64_t)n_last * chunks) return;
  const int p = k - n_last + (int)(x / chunks);
  const int c = (int)(x % chunks);
  const int i = idx ? idx[(int64_t)b * k + p] : p;
  if (i < lo) return;
  const uint4 v = *reinterpret_cast<const uint4*>(x_cur + ((int64_t)b * N + i) * HD + c * 8);
  if (cache) *reinterpret_cast<uint4*>(cache + ((int64_t)b * N + i) * HD + c * 8) = v;
  if (rows) *reinterpret_cast<uint4*>(rows + ((int64_t)b * k + p) * HD + c * 8) = v;
}

}  // namespace fl

using namespace fl;

extern "C" int fl_kv_residual_quant(const uint16_t* x_cur, const uint16_t* x_ref, const int32_t* idx,
                                    int k, int B, int N, int H, int d, int bits, int group, int axis,
                                    uint8_t* codes, uint16_t* scale, uint16_t* zero,
                                    uint16_t* out_rows, void* stream) {
  FL_API_BEGIN
  FL_REQUIRE(!(out_rows && out_rows == x_ref && idx), FL_E_SHAPE,
             "fl_kv_residual_quant: out_rows may alias x_ref only when idx is NULL");
  return residual_quant("fl_kv_residual_quant", x_cur, x_ref, idx, k, B, N, H, d, bits, group, axis, codes,
                        scale, zero, out_rows, false, stream);
  FL_API_END
}

extern "C" int fl_kv_residual_quant_commit(const uint16_t* x_cur, uint16_t* x_hat, const int32_t* idx, int k,
                                           int B, int N, int H, int d, int bits, int group, int axis,
                                           uint8_t* codes, uint16_t* scale, uint16_t* zero, void* stream) {
  FL_API_BEGIN
  FL_REQUIRE(x_hat != nullptr, FL_E_NULL, "fl_kv_residual_quant_commit: x_hat is required");
  return residual_quant("fl_kv_residual_quant_commit", x_cur, x_hat, idx, k, B, N, H, d, bits, group, axis,
                        codes, scale, zero, x_hat, true, stream);
  FL_API_END
}

extern "C" int fl_kv_residual_quant_kv(const uint16_t* k_cur, uint16_t* k_ref, const uint16_t* v_cur,
                                       uint16_t* v_ref, const int32_t* idx, int k, int B, int N, int H, int d,
                                       int bits, int group, uint8_t* k_codes, uint16_t* k_scale, uint16_t* k_zero,
                                       uint8_t* v_codes, uint16_t* v_scale, uint16_t* v_zero, uint16_t* k_rows,
                                       uint16_t* v_rows, int mode, void* stream) {
  FL_API_BEGIN
  const char* fn = "fl_kv_residual_quant_kv";
  FL_REQUIRE(mode == FL_DQ_COMPACT || mode == FL_DQ_COMMIT, FL_E_UNSUPPORTED, "%s: bad mode %d", fn, mode);
  if (mode == FL_DQ_COMMIT) {
    FL_REQUIRE(k_ref && v_ref, FL_E_NULL, "%s: COMMIT needs k_ref and v_ref", fn);
    FL_REQUIRE(!k_rows && !v_rows, FL_E_NULL, "%s: COMMIT needs k_rows == v_rows == NULL", fn);
    FL_REQUIRE(k_ref != v_ref, FL_E_SHAPE, "%s: COMMIT needs distinct key and value caches", fn);
  } else {
    FL_REQUIRE(!(k_rows && k_rows == k_ref && idx) && !(v_rows && v_rows == v_ref && idx), FL_E_SHAPE,
               "%s: rows may alias the reference only when idx is NULL", fn);
  }
  FL_REQUIRE(k == 0 || k_codes != v_codes, FL_E_SHAPE, "%s: key and value codes must be distinct buffers", fn);
  return residual_quant_kv(fn, k_cur, k_ref, v_cur, v_ref, idx, k, B, N, H, d, bits, group, k_codes, k_scale,
                           k_zero, v_codes, v_scale, v_zero, k_rows, v_rows, mode == FL_DQ_COMMIT, nullptr, stream);
  FL_API_END
}

extern "C" int fl_kv_residual_quant_kv_v16(const uint16_t* k_cur, uint16_t* k_ref, const uint16_t* v_cur,
                                           uint16_t* v_ref, uint16_t* v_f16, const int32_t* idx, int k, int B, int N,
                                           int H, int d, int bits, int group, uint8_t* k_codes, uint16_t* k_scale,
                                           uint16_t* k_zero, uint8_t* v_codes, uint16_t* v_scale, uint16_t* v_zero,
                                           void* stream) {
  FL_API_BEGIN
  const char* fn = "fl_kv_residual_quant_kv_v16";
  FL_REQUIRE(k_ref && v_ref && v_f16, FL_E_NULL, "%s: k_ref, v_ref and v_f16 are required", fn);
  FL_REQUIRE(k_ref != v_ref && (const void*)v_f16 != (const void*)v_ref && (const void*)v_f16 != (const void*)k_ref,
             FL_E_SHAPE, "%s: the key cache, the value cache and its fp16 copy must be distinct", fn);
  FL_REQUIRE(k == 0 || k_codes != v_codes, FL_E_SHAPE, "%s: key and value codes must be distinct buffers", fn);
  return residual_quant_kv(fn, k_cur, k_ref, v_cur, v_ref, idx, k, B, N, H, d, bits, group, k_codes, k_scale,
                           k_zero, v_codes, v_scale, v_zero, nullptr, nullptr, true, v_f16, stream);
  FL_API_END
}

extern "C" int fl_kv_f16_rows(const uint16_t* x, const int32_t* idx, int k, int B, int N, int H, int d,
                              uint16_t* x_f16, void* stream) {
  FL_API_BEGIN
  const char* fn = "fl_kv_f16_rows";
  FL_REQUIRE(x && x_f16, FL_E_NULL, "%s: x and x_f16 are required", fn);
  FL_REQUIRE((const void*)x != (const void*)x_f16, FL_E_SHAPE, "%s: x_f16 may not alias x", fn);
  FL_REQUIRE(B >= 1 && N >= 1 && H >= 1 && d >= 8 && d % 8 == 0, FL_E_SHAPE,
             "%s: need B, N, H >= 1 and d a multiple of 8", fn);
  FL_REQUIRE(k >= 0 && k <= N, FL_E_RANGE, "%s: k=%d outside [0, N]", fn, k);
  if (k == 0) return FL_OK;               // (an empty index list may come as NULL)
  FL_REQUIRE(idx || k == N, FL_E_RANGE, "%s: k=%d with idx NULL (every row: k = N)", fn, k);
  const hipStream_t st = as_stream(stream);
  if (idx) FL_CHECK_LIST(fn, "idx", idx, B, k, 0, N, st);
  return launch_f16_rows(x, idx, k, B, N, H * d, x_f16, st);
  FL_API_END
}

extern "C" int fl_kv_residual_dequant_kv(const uint8_t* k_codes, const uint16_t* k_scale, const uint16_t* k_zero,
                                         const uint8_t* v_codes, const uint16_t* v_scale, const uint16_t* v_zero,
                                         const int32_t* idx, int k, int B, int N, int H, int d, int bits, int group,
                                         int mode, uint16_t* k_hat, uint16_t* v_hat, uint16_t* k_rows,
                                         uint16_t* v_rows, void* stream) {
  FL_API_BEGIN
  const char* fn = "fl_kv_residual_dequant_kv";
  int rc = check_codec_args(fn, k_codes, k_hat, k, B, N, H, d, bits, group, FL_AXIS_TOKEN, true, k_scale, k_zero,
                            idx);
  if (rc != FL_OK) return rc;
  rc = check_codec_args(fn, v_codes, v_hat, k, B, N, H, d, bits, group, FL_AXIS_CHANNEL, true, v_scale, v_zero, idx);
  if (rc != FL_OK) return rc;
  FL_REQUIRE(mode == FL_DQ_COMPACT || mode == FL_DQ_COMMIT, FL_E_UNSUPPORTED, "%s: bad mode %d", fn, mode);
  FL_REQUIRE(mode == FL_DQ_COMMIT ? (!k_rows && !v_rows) : (k_rows && v_rows), FL_E_NULL,
             "%s: COMPACT needs k_rows and v_rows, COMMIT needs both NULL", fn);
  FL_REQUIRE(mode == FL_DQ_COMPACT || k_hat != v_hat, FL_E_SHAPE, "%s: COMMIT needs distinct caches", fn);
  if (k == 0) return FL_OK;
  const int64_t half = ((int64_t)k * (H * d / 8) + 255) / 256;
  FL_REQUIRE(2 * half < ((int64_t)1 << 31), FL_E_SHAPE, "%s: grid too large", fn);
  DequantKV a;
  a.k_codes = k_codes; a.k_scale = k_scale; a.k_zero = k_zero;
  a.v_codes = v_codes; a.v_scale = v_scale; a.v_zero = v_zero;
  a.idx = idx; a.k_hat = k_hat; a.v_hat = v_hat;
  a.k_rows = mode == FL_DQ_COMMIT ? nullptr : k_rows;
  a.v_rows = mode == FL_DQ_COMMIT ? nullptr : v_rows;
  a.k = k; a.N = N; a.HD = H * d; a.G = group; a.half = (int)half;
  dim3 grid((unsigned)(2 * half), B);
  hipStream_t st = as_stream(stream);
  FL_CHECK_LIST("fl_kv_residual_dequant_kv", "idx", idx, B, k, 0, N, st);
  if (bits == 16) {   // raw payload: both axes copy the same way
    dequant_kv_kernel<16><<<grid, 256, 0, st>>>(a);
  } else if (bits == 2) {
    dequant_kv_kernel<2><<<grid, 256, 0, st>>>(a);
  } else if (bits == 4) {
    dequant_kv_kernel<4><<<grid, 256, 0, st>>>(a);
  } else {
    dequant_kv_kernel<8><<<grid, 256, 0, st>>>(a);
  }
  return check_launch("dequant_kv_kernel");
  FL_API_END
}

extern "C" int fl_kv_residual_dequant(const uint8_t* codes, const uint16_t* scale, const uint16_t* zero,
                                      const int32_t* idx, int k, int B, int N, int H, int d, int bits,
                                      int group, int axis, int mode, uint16_t* x_hat,
                                      uint16_t* out_rows, void* stream) {
  FL_API_BEGIN
  int rc = check_codec_args("fl_kv_residual_dequant", codes, x_hat, k, B, N, H, d, bits, group, axis,
                            true, scale, zero, idx);
  if (rc != FL_OK) return rc;
  FL_REQUIRE(mode == FL_DQ_COMPACT || mode == FL_DQ_COMMIT, FL_E_UNSUPPORTED,
             "fl_kv_residual_dequant: bad mode %d", mode);
  FL_REQUIRE(mode == FL_DQ_COMMIT ? out_rows == nullptr : out_rows != nullptr, FL_E_NULL,
             "fl_kv_residual_dequant: COMPACT needs out_rows, COMMIT needs out_rows == NULL");
  if (k == 0) return FL_OK;
  const int HD = H * d;
  dim3 grid((unsigned)(((int64_t)k * (HD / 8) + 255) / 256), B);
  hipStream_t st = as_stream(stream);
  FL_CHECK_LIST("fl_kv_residual_dequant", "idx", idx, B, k, 0, N, st);
#define FL_DQ(BB, AA) \
  dequant_kernel<BB, AA><<<grid, 256, 0, st>>>(codes, scale, zero, idx, k, N, HD, group, x_hat, out_rows)
  if (bits == 16) FL_DQ(16, 0);
  else if (axis == FL_AXIS_TOKEN) {
    if (bits == 2) FL_DQ(2, FL_AXIS_TOKEN); else if (bits == 4) FL_DQ(4, FL_AXIS_TOKEN); else FL_DQ(8, FL_AXIS_TOKEN);
  } else {
    if (bits == 2) FL_DQ(2, FL_AXIS_CHANNEL); else if (bits == 4) FL_DQ(4, FL_AXIS_CHANNEL); else FL_DQ(8, FL_AXIS_CHANNEL);
  }
#undef FL_DQ
  return check_launch("dequant_kernel");
  FL_API_END
}

extern "C" int fl_kv_keep_recent(const uint16_t* x_cur, const int32_t* idx, int k, int B, int N, int H, int d,
                                 int tail, uint16_t* cache, uint16_t* rows, void* stream) {
  FL_API_BEGIN
  FL_REQUIRE(x_cur, FL_E_NULL, "fl_kv_keep_recent: x_cur is required");
  FL_REQUIRE(cache || rows, FL_E_NULL, "fl_kv_keep_recent: cache or rows is required");
  FL_REQUIRE(B >= 1 && N >= 1 && H >= 1, FL_E_SHAPE, "fl_kv_keep_recent: need B, N, H >= 1");
  FL_REQUIRE(d >= 8 && d % 8 == 0, FL_E_SHAPE, "fl_kv_keep_recent: d=%d must be a positive multiple of 8", d);
  FL_REQUIRE((int64_t)N * H * d < ((int64_t)1 << 40), FL_E_SHAPE, "fl_kv_keep_recent: N * H * d too large");
  FL_REQUIRE(k >= 0 && k <= N, FL_E_RANGE, "fl_kv_keep_recent: k=%d outside [0, N]", k);
  FL_REQUIRE(idx || k == N, FL_E_SHAPE, "fl_kv_keep_recent: without idx, k must equal N");
  FL_REQUIRE(tail >= 0, FL_E_RANGE, "fl_kv_keep_recent: tail must be >= 0");
  const int n_last = std::min(k, tail);
  if (n_last == 0) return FL_OK;
  const int HD = H * d;
  const int64_t work = (int64_t)n_last * (HD / 8);
  dim3 grid((unsigned)((work + 255) / 256), B);
  FL_CHECK_LIST("fl_kv_keep_recent", "idx", idx, B, k, 0, N, as_stream(stream));
  keep_recent_kernel<<<grid, 256, 0, as_stream(stream)>>>(x_cur, idx, k, N, HD, std::max(0, N - tail), n_last,
                                                          cache, rows);
  return check_launch("keep_recent_kernel");
  FL_API_END
}
