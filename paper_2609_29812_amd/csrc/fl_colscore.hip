// Column statistic of a dense source loop (Appendix D.2, Eq. 6 with all causal keys and cached mass 1,
// summed over the rows of a prefill), in fp64 so that the fp32 keys the column top-k ranks are the
// correctly rounded values of the exact statistic up to fp64 rounding.
//
// Two passes, both "a register-resident vector against LDS-staged vectors":
//   pass 1 (rows)    : a thread pair owns query row i (each thread half of the dims); K rows are staged
//                      32 at a time; l_ij = sigma * sum_e q_ie k_je and an online fp64 logsumexp over
//                      j <= i give lse_i (stored in the workspace);
//   pass 2 (columns) : a thread pair owns key column j; Q rows and their lse are staged 32 at a time and
//                      col_j = sum_{i >= j} exp(l_ij - lse_i) is accumulated in ascending i.
// Products of bf16 values are exact in fp64; every sum runs in a fixed order (deterministic).
#include "fl_common.h"

namespace fl {

constexpr int kCsThreads = 256;
constexpr int kCsOwn = kCsThreads / 2;   // rows (pass 1) or columns (pass 2) per workgroup
constexpr int kCsTile = 32;

template <int D>
__device__ __forceinline__ void stage_f64(double (*tile)[D], const uint16_t* src, int64_t row_stride,
                                          int first, int N) {
  for (int q = threadIdx.x; q < kCsTile * D; q += kCsThreads) {
    const int r = q / D, e = q % D;
    const int idx = first + r;
    tile[r][e] = idx < N ? (double)bf16_to_f32(src[(int64_t)idx * row_stride + e]) : 0.0;
  }
}

template <int D, bool COLUMNS>
__global__ __launch_bounds__(kCsThreads) void colscore_kernel(const uint16_t* __restrict__ q,
                                                              const uint16_t* __restrict__ kc, int N,
                                                              int H, double sigma,
                                                              double* __restrict__ lse,
                                                              float* __restrict__ col_key) {
  __shared__ double tile[kCsTile][D];
  __shared__ double tile_lse[kCsTile];
  constexpr int HALF = D / 2;
  const int h = blockIdx.y, b = blockIdx.z;
  const int me = blockIdx.x * kCsOwn + (threadIdx.x >> 1);
  const int half = threadIdx.x & 1;
  const bool ok = me < N;
  const int64_t stride = (int64_t)H * D;
  const uint16_t* qbase = q + (int64_t)b * N * stride + (int64_t)h * D;
  const uint16_t* kbase = kc + (int64_t)b * N * stride + (int64_t)h * D;
  double* lse_bh = lse + ((int64_t)b * H + h) * N;

  double v[HALF];
  {
    const uint16_t* src = (COLUMNS ? kbase : qbase) + (int64_t)(ok ? me : 0) * stride + half * HALF;
#pragma unroll
    for (int e = 0; e < HALF; ++e) v[e] = ok ? (double)bf16_to_f32(src[e]) : 0.0;
  }

  if (!COLUMNS) {
    const int last = min(N, (int)(blockIdx.x + 1) * kCsOwn) - 1;
    double m = -INFINITY, s = 0.0;
    for (int t0 = 0; t0 <= last; t0 += kCsTile) {
      stage_f64<D>(tile, kbase, stride, t0, N);
      __syncthreads();
      for (int jj = 0; jj < kCsTile; ++jj) {
        const int j = t0 + jj;
        double dot = 0.0;
#pragma unroll
        for (int e = 0; e < HALF; ++e) dot = fma(v[e], tile[jj][half * HALF + e], dot);
        const double other = __shfl_xor(dot, 1, 64);
        const double full = half ? other + dot : dot + other;   // lower half first
        if (ok && j <= me) {
          const double l = sigma * full;
          if (l > m) {
            s = s * exp(m - l) + 1.0;
            m = l;
          } else {
            s += exp(l - m);
          }
        }
      }
      __syncthreads();
    }
    if (ok && half == 0) lse_bh[me] = m + log(s);
  } else {
    const int first = blockIdx.x * kCsOwn;
    double acc = 0.0;
    for (int t0 = first; t0 < N; t0 += kCsTile) {
      stage_f64<D>(tile, qbase, stride, t0, N);
      if (threadIdx.x < kCsTile) tile_lse[threadIdx.x] = (t0 + (int)threadIdx.x) < N ? lse_bh[t0 + threadIdx.x] : 0.0;
      __syncthreads();
      for (int ii = 0; ii < kCsTile; ++ii) {
        const int i = t0 + ii;
        double dot = 0.0;
#pragma unroll
        for (int e = 0; e < HALF; ++e) dot = fma(v[e], tile[ii][half * HALF + e], dot);
        const double other = __shfl_xor(dot, 1, 64);
        const double full = half ? other + dot : dot + other;
        if (ok && i < N && i >= me) acc += exp(sigma * full - tile_lse[ii]);
      }
      __syncthreads();
    }
    if (ok && half == 0) col_key[((int64_t)b * H + h) * N + me] = (float)acc;
  }
}

}  // namespace fl

using namespace fl;

extern "C" size_t fl_column_scores_ws(int B, int N, int H) {
  if (B < 1 || N < 1 || H < 1) return 0;
  return (size_t)B * (size_t)H * (size_t)N * sizeof(double);
}

extern "C" int fl_column_scores(const uint16_t* q, const uint16_t* k_cache, int B, int N, int H, int d,
                                float* col_key, void* ws, size_t ws_bytes, void* stream) {
  FL_API_BEGIN
  FL_REQUIRE(q && k_cache && col_key, FL_E_NULL, "fl_column_scores: q, k_cache and col_key are required");
  FL_REQUIRE(B >= 1 && N >= 1 && H >= 1, FL_E_SHAPE, "fl_column_scores: need B, N, H >= 1");
  FL_REQUIRE(d == 64 || d == 128, FL_E_SHAPE, "fl_column_scores: head dim %d not in {64, 128}", d);
  FL_REQUIRE((int64_t)N * H * d < ((int64_t)1 << 31), FL_E_SHAPE, "fl_column_scores: N * H * d too large");
  FL_REQUIRE(ws && ws_bytes >= fl_column_scores_ws(B, N, H), FL_E_WORKSPACE,
             "fl_column_scores: workspace of %zu bytes required", fl_column_scores_ws(B, N, H));
  hipStream_t st = as_stream(stream);
  const double sigma = 1.0 / std::sqrt((double)d);
  double* lse = static_cast<double*>(ws);
  dim3 grid((N + kCsOwn - 1) / kCsOwn, H, B);
  if (d == 128) {
    colscore_kernel<128, false><<<grid, kCsThreads, 0, st>>>(q, k_cache, N, H, sigma, lse, col_key);
    int rc = check_launch("colscore_kernel(rows)");
    if (rc != FL_OK) return rc;
    colscore_kernel<128, true><<<grid, kCsThreads, 0, st>>>(q, k_cache, N, H, sigma, lse, col_key);
  } else {
    colscore_kernel<64, false><<<grid, kCsThreads, 0, st>>>(q, k_cache, N, H, sigma, lse, col_key);
    int rc = check_launch("colscore_kernel(rows)");
    if (rc != FL_OK) return rc;
    colscore_kernel<64, true><<<grid, kCsThreads, 0, st>>>(q, k_cache, N, H, sigma, lse, col_key);
  }
  return check_launch("colscore_kernel(columns)");
  FL_API_END
}
