// Token selection (Section 4.1; Appendix D.1, Eq. 5) and column-list selection (Appendix D.2, Eq. 6).
//
// score_rows: one wave per candidate row streams the four bf16 rows (K and V, current and previous)
//   with non-temporal 16-byte loads, forms fp32 differences, accumulates squared norms in fp64,
//   reduces across the wave and writes the fp32 key.  HBM-bound: 4 * D * 2 bytes per candidate.
//   When the budget keeps every candidate (k = n_cand, nested loops with a constant budget), extra
//   workgroups of the same launch write the selection itself: the candidates and their slot map.
// topk_select: one 1024-thread workgroup per segment runs the radix top-k of fl_topk.h.
#include "fl_common.h"
#include "fl_topk.h"

namespace fl {

constexpr int kScoreWaves = 4;

// 16-byte load marked non-temporal: each state row is read once per pass, so it should not displace
// cached data (measured: the pass streams about 15% faster than with ordinary loads)
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 stream_load16(const uint16_t* p) {
  const u32x4v w = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(p));
  return make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ void accum_pair(uint4 c, uint4 p, double& num, double& den) {
  const uint32_t cw[4] = {c.x, c.y, c.z, c.w};
  const uint32_t pw[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float c0 = __uint_as_float(cw[t] << 16), c1 = __uint_as_float(cw[t] & 0xFFFF0000u);
    float p0 = __uint_as_float(pw[t] << 16), p1 = __uint_as_float(pw[t] & 0xFFFF0000u);
    double d0 = (double)(c0 - p0), d1 = (double)(c1 - p1);   // fp32 difference, then exact widen
    num += d0 * d0;
    num += d1 * d1;
    den += (double)c0 * (double)c0;
    den += (double)c1 * (double)c1;
  }
}

// take_all (k == n_cand): workgroups past the scoring ones write the selection itself, which keeps every
// candidate: idx = the candidates, and slot[j] = j's position among them (binary search) or -1.
__global__ __launch_bounds__(64 * kScoreWaves) void score_rows_kernel(
    const uint16_t* __restrict__ k_cur, const uint16_t* __restrict__ k_prev,
    const uint16_t* __restrict__ v_cur, const uint16_t* __restrict__ v_prev, int N, int D,
    const int32_t* __restrict__ cand, int n_cand, int normalize, double eps,
    float* __restrict__ out_key, int score_blocks, int32_t* __restrict__ take_idx,
    int32_t* __restrict__ take_slot) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.y;
  if ((int)blockIdx.x >= score_blocks) {
    const int64_t t = (int64_t)(blockIdx.x - score_blocks) * blockDim.x + threadIdx.x;
    const int32_t* cp = cand ? cand + (int64_t)b * n_cand : nullptr;
    if (t < n_cand) take_idx[(int64_t)b * n_cand + t] = cp ? cp[t] : (int32_t)t;
    if (take_slot && t < N) {
      int pos = (int)t;                    // all rows are candidates without a list
      if (cp) {
        int lo = 0, hi = n_cand;
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (cp[mid] < (int)t) lo = mid + 1; else hi = mid;
        }
        pos = (lo < n_cand && cp[lo] == (int)t) ? lo : -1;
      }
      take_slot[(int64_t)b * N + t] = pos;
    }
    return;
  }
  const int p = blockIdx.x * kScoreWaves + (threadIdx.x >> 6);
  if (p >= n_cand) return;
  const int64_t row = cand ? (int64_t)cand[(int64_t)b * n_cand + p] : (int64_t)p;
  const int64_t base = ((int64_t)b * N + row) * D;
  double num = 0.0, den = 0.0;
#pragma unroll 4
  for (int e = lane * 8; e < D; e += 512) {
    uint4 kc = stream_load16(k_cur + base + e);
    uint4 kp = stream_load16(k_prev + base + e);
    uint4 vc = make_uint4(0, 0, 0, 0), vp = make_uint4(0, 0, 0, 0);
    if (v_cur) {
      vc = stream_load16(v_cur + base + e);
      vp = stream_load16(v_prev + base + e);
    }
    accum_pair(kc, kp, num, den);
    accum_pair(vc, vp, num, den);
  }
  num = wave_sum_f64(num);
  den = wave_sum_f64(den);
  if (lane == 0) {
    double s = normalize ? sqrt(num) / (sqrt(den) + eps) : sqrt(num);
    out_key[(int64_t)b * n_cand + p] = (float)s;
  }
}

// Segment s = blockIdx.x: keys at keys + s key_stride, ids from cand + s cand_stride (or id_base + p),
// output at out + s out_stride, slot map at slot + s slot_n.
template <int M>
__global__ __launch_bounds__(kTopkThreads) void topk_select_kernel(
    const float* __restrict__ keys, int64_t key_stride, int n, int k,
    const int32_t* __restrict__ cand, int64_t cand_stride, int id_base,
    int32_t* __restrict__ out, int64_t out_stride, int n_prefix,
    int32_t* __restrict__ slot, int slot_n) {
  const int s = blockIdx.x;
  topk_block<M>(keys + (int64_t)s * key_stride, n, k, cand ? cand + (int64_t)s * cand_stride : nullptr, id_base,
                out + (int64_t)s * out_stride, n_prefix, slot ? slot + (int64_t)s * slot_n : nullptr, slot_n);
}

int launch_topk(int segments, const float* keys, int64_t key_stride, int n, int k,
                       const int32_t* cand, int64_t cand_stride, int id_base, int32_t* out,
                       int64_t out_stride, int n_prefix, int32_t* slot, int slot_n,
                       hipStream_t st) {
  const int per = (n + kTopkThreads - 1) / kTopkThreads;
  dim3 grid(segments), block(kTopkThreads);
#define FL_TOPK(MM)                                                                          \
  topk_select_kernel<MM><<<grid, block, 0, st>>>(keys, key_stride, n, k, cand, cand_stride, \
                                                 id_base, out, out_stride, n_prefix, slot,  \
                                                 slot_n)
  if (per <= 1) FL_TOPK(1);
  else if (per <= 2) FL_TOPK(2);
  else if (per <= 4) FL_TOPK(4);
  else if (per <= 8) FL_TOPK(8);
  else if (per <= 16) FL_TOPK(16);
  else if (per <= 32) FL_TOPK(32);
  else if (per <= 64) FL_TOPK(64);
  else return set_error(FL_E_SHAPE, "top-k over %d keys exceeds the 65536 supported", n);
#undef FL_TOPK
  return check_launch("topk_select_kernel");
}

}  // namespace fl

using namespace fl;

extern "C" int fl_select_tokens(const uint16_t* k_cur, const uint16_t* k_prev,
                                const uint16_t* v_cur, const uint16_t* v_prev, int B, int N, int D,
                                const int32_t* cand, int n_cand, int k, int normalize, double eps,
                                float* out_key, int32_t* out_idx, int32_t* out_slot, void* stream) {
  FL_API_BEGIN
  FL_REQUIRE(k_cur && k_prev && out_key, FL_E_NULL, "fl_select_tokens: k_cur, k_prev and out_key are required");
  FL_REQUIRE((v_cur == nullptr) == (v_prev == nullptr), FL_E_NULL,
             "fl_select_tokens: v_cur and v_prev must both be set or both be NULL");
  FL_REQUIRE(B >= 1 && N >= 1 && D >= 8 && D % 8 == 0, FL_E_SHAPE,
             "fl_select_tokens: need B, N >= 1 and D a positive multiple of 8 (B=%d N=%d D=%d)", B, N, D);
  FL_REQUIRE((int64_t)N * D < (int64_t)1 << 40, FL_E_SHAPE, "fl_select_tokens: N * D too large");
  FL_REQUIRE(cand != nullptr || n_cand == N, FL_E_SHAPE,
             "fl_select_tokens: without a candidate list n_cand must equal N");
  FL_REQUIRE(n_cand >= 0 && n_cand <= N, FL_E_RANGE, "fl_select_tokens: n_cand=%d outside [0, N]", n_cand);
  FL_REQUIRE(n_cand <= 65536, FL_E_SHAPE, "fl_select_tokens: n_cand=%d exceeds 65536", n_cand);
  FL_REQUIRE(k >= 0 && k <= n_cand, FL_E_RANGE, "fl_select_tokens: k=%d outside [0, n_cand=%d]", k, n_cand);
  FL_REQUIRE(k == 0 || out_idx, FL_E_NULL, "fl_select_tokens: out_idx is required when k > 0");
  FL_REQUIRE(eps >= 0.0, FL_E_RANGE, "fl_select_tokens: eps must be >= 0");
  hipStream_t st = as_stream(stream);
  FL_CHECK_LIST("fl_select_tokens", "cand", cand, B, n_cand, 0, N, st);
  // k == n_cand keeps every candidate: the scoring launch also writes the selection (no top-k launch)
  const bool take_all = k == n_cand && k > 0;
  if (n_cand > 0) {
    const int score_blocks = (n_cand + kScoreWaves - 1) / kScoreWaves;
    const int fill_blocks = take_all ? (N + 64 * kScoreWaves - 1) / (64 * kScoreWaves) : 0;
    dim3 grid(score_blocks + fill_blocks, B), block(64 * kScoreWaves);
    score_rows_kernel<<<grid, block, 0, st>>>(k_cur, k_prev, v_cur, v_prev, N, D, cand, n_cand,
                                              normalize, eps, out_key, score_blocks, out_idx, out_slot);
    int rc = check_launch("score_rows_kernel");
    if (rc != FL_OK) return rc;
  }
  if (take_all) return FL_OK;
  if (k == 0 && !out_slot) return FL_OK;
  return launch_topk(B, out_key, n_cand, n_cand, k, cand, n_cand, 0, out_idx, k, 0, out_slot, N, st);
  FL_API_END
}

extern "C" int fl_select_columns(const float* col_key, int B, int H, int N, int n_sink, int t,
                                 int32_t* cols, void* stream) {
  FL_API_BEGIN
  FL_REQUIRE(B >= 1 && H >= 1 && N >= 1, FL_E_SHAPE, "fl_select_columns: need B, H, N >= 1");
  FL_REQUIRE(n_sink >= 0, FL_E_RANGE, "fl_select_columns: n_sink must be >= 0");
  const int ns = n_sink < N ? n_sink : N;
  FL_REQUIRE(t >= 0 && t <= N - ns, FL_E_RANGE, "fl_select_columns: t=%d outside [0, N - n_sink]", t);
  FL_REQUIRE(N - ns <= 65536, FL_E_SHAPE, "fl_select_columns: N - n_sink exceeds 65536");
  if (ns + t == 0) return FL_OK;          // an empty list: nothing to write (cols may be NULL)
  FL_REQUIRE(col_key && cols, FL_E_NULL, "fl_select_columns: col_key and cols are required");
  return launch_topk(B * H, col_key + ns, N, N - ns, t, nullptr, 0, ns, cols, ns + t, ns, nullptr, 0,
                     as_stream(stream));
  FL_API_END
}
