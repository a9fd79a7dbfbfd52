// Column statistics in fp64, so that the fp32 keys a top-k ranks are the correctly rounded values of the
// exact statistic up to fp64 rounding:
//   * the dense source loop's statistic (Appendix D.2, Eq. 6 with all causal keys and cached mass 1, summed
//     over the rows of a prefill), in two passes: the rows' log-normalisers, then the column sums;
//   * the statistic that prunes a list for a smaller budget (Section 4.2): the mass the updated rows give
//     each list entry, from their stored reference log-normalisers.
// The dot products run on v_mfma_f64_16x16x4 (products of bf16 values are exact in fp64); every sum runs
// in a fixed order (deterministic).
#include "fl_common.h"

namespace fl {

constexpr int kCsRows = 32;               // vectors staged per step
typedef double f64x4 __attribute__((ext_vector_type(4)));

// Which (row, column) of a v_mfma_f64_16x16x4 product each of a lane's four accumulator elements holds,
// read off two index products (A = row index in k-column 0 against B = 1 in k-row 0, and the transposed
// pair), clamped so that the indices stay in range whatever the products hold.
__device__ __forceinline__ void mfma_f64_layout(int l16, int kq, int (&row)[4], int (&col)[4]) {
  const f64x4 zero = {0.0, 0.0, 0.0, 0.0};
  const f64x4 r = __builtin_amdgcn_mfma_f64_16x16x4f64(kq == 0 ? (double)l16 : 0.0, kq == 0 ? 1.0 : 0.0, zero, 0, 0, 0);
  const f64x4 c = __builtin_amdgcn_mfma_f64_16x16x4f64(kq == 0 ? 1.0 : 0.0, kq == 0 ? (double)l16 : 0.0, zero, 0, 0, 0);
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    row[t] = min(max((int)r[t], 0), 15);
    col[t] = min(max((int)c[t], 0), 15);
  }
}

// Dense column statistic in two passes, the fp64 dot products on v_mfma_f64_16x16x4 (products of bf16 values
// are exact in fp64).  A wave owns 16 vectors of one side in registers (lane l holds dim 4s + l / 16 of vector
// l % 16 for step s), a workgroup 64 of them; the other side is staged 32 vectors at a time in LDS as fp64.
//   pass 1 (ROWS)  : the wave's 16 query rows against the staged K columns j <= i: per accumulator element
//                    an online (max, sum) in fp64; the 16 partial pairs of a row are merged in column order;
//   pass 2 (!ROWS) : the wave's 16 K columns against the staged query rows i >= j and their lse_i:
//                    col_j = sum exp(l_ij - lse_i), the 16 partials of a column added in row order.
// Every sum runs in a fixed order (deterministic).
template <int D, bool ROWS>
__global__ __launch_bounds__(256) void colscore_kernel(const uint16_t* __restrict__ q,
                                                       const uint16_t* __restrict__ kc, int N, int H,
                                                       double sigma, double* __restrict__ lse,
                                                       float* __restrict__ col_key) {
  constexpr int QS = D + 1;               // padded stride (doubles): the 16 vectors of a read spread over banks
  constexpr int KSTEPS = D / 4;
  __shared__ double st[kCsRows * QS];
  __shared__ double st_lse[kCsRows];
  __shared__ double red_m[4][16][17];
  __shared__ double red_s[4][16][17];
  const int h = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, kq = lane >> 4;
  const int64_t stride = (int64_t)H * D;
  const uint16_t* qbase = q + (int64_t)b * N * stride + (int64_t)h * D;
  const uint16_t* kbase = kc + (int64_t)b * N * stride + (int64_t)h * D;
  double* lse_bh = lse + ((int64_t)b * H + h) * N;
  const int v0 = blockIdx.x * 64 + wave * 16;          // first of the wave's own vectors
  const bool wave_ok = v0 < N;

  double reg[KSTEPS];                                   // own vectors (query rows or key columns)
  {
    const int v = v0 + l16;
    const uint16_t* src = (ROWS ? qbase : kbase) + (int64_t)(v < N ? v : 0) * stride + kq;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) reg[s] = v < N ? (double)bf16_to_f32(src[4 * s]) : 0.0;
  }
  int el_r[4], el_c[4];                   // element t: staged vector el_r (A side), own vector el_c (B side)
  mfma_f64_layout(l16, kq, el_r, el_c);
  // staged range: pass 1 columns 0 .. last own row; pass 2 rows from the workgroup's first column on
  const int wg_first = blockIdx.x * 64;
  const int s_begin = ROWS ? 0 : wg_first;
  const int s_end = ROWS ? min(N, wg_first + 64) : N;
  double m[4], acc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) { m[t] = -INFINITY; acc[t] = 0.0; }
  for (int t0 = s_begin; t0 < s_end; t0 += kCsRows) {
    for (int x = threadIdx.x; x < kCsRows * D; x += 256) {
      const int r = x / D, dd = x % D;
      const int v = t0 + r;
      st[r * QS + dd] = v < s_end ? (double)bf16_to_f32((ROWS ? kbase : qbase)[(int64_t)v * stride + dd]) : 0.0;
    }
    if (!ROWS && threadIdx.x < kCsRows) {
      const int v = t0 + (int)threadIdx.x;
      st_lse[threadIdx.x] = v < s_end ? lse_bh[v] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int half = 0; half < kCsRows / 16; ++half) {
      const int sv0 = t0 + 16 * half;                   // first staged vector of this 16
      // uniform: pass 1 needs staged columns <= the wave's last row, pass 2 staged rows >= its first column
      const bool useful = wave_ok && sv0 < s_end && (ROWS ? sv0 <= v0 + 15 : sv0 + 15 >= v0);
      if (useful) {
        f64x4 d4 = {0.0, 0.0, 0.0, 0.0};
        const double* sa = st + (16 * half + l16) * QS + kq;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) d4 = __builtin_amdgcn_mfma_f64_16x16x4f64(sa[4 * s], reg[s], d4, 0, 0, 0);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int sv = sv0 + el_r[t];                  // staged vector
          const int ov = v0 + el_c[t];                   // own vector
          const double l = sigma * d4[t];
          if (ROWS) {
            if (sv < s_end && ov < N && sv <= ov) {      // column sv of row ov
              if (l > m[t]) {
                acc[t] = acc[t] * exp(m[t] - l) + 1.0;
                m[t] = l;
              } else {
                acc[t] += exp(l - m[t]);
              }
            }
          } else {
            if (sv < s_end && ov < N && sv >= ov) acc[t] += exp(l - st_lse[16 * half + el_r[t]]);   // row sv
          }
        }
      }
    }
    __syncthreads();
  }
  // merge the 16 partials of each own vector in staged-slot order
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    red_m[wave][el_c[t]][el_r[t]] = m[t];
    red_s[wave][el_c[t]][el_r[t]] = acc[t];
  }
  __syncthreads();
  const int v = v0 + lane;
  if (lane < 16 && v < N) {
    if (ROWS) {
      double mm = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) mm = fmax(mm, red_m[wave][lane][r]);
      double ss = 0.0;
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (red_s[wave][lane][r] > 0.0) ss += red_s[wave][lane][r] * exp(red_m[wave][lane][r] - mm);
      lse_bh[v] = mm + log(ss);
    } else {
      double ss = 0.0;
#pragma unroll
      for (int r = 0; r < 16; ++r) ss += red_s[wave][lane][r];
      col_key[((int64_t)b * H + h) * N + v] = (float)ss;
    }
  }
}

// Statistic of the list entries for pruning a shrinking list (Section 4.2; Appendix D.2, Eq. 6 with a
// sparse source): entry j of the (b, h) list gets sum_{i updated, i >= j} exp(sigma q_i . k_j - lse_ref_i),
// the loop-r probability mass it receives from the updated rows, each row's probabilities recovered from
// its reference log-normaliser.  The dot products are fp64 MFMAs (v_mfma_f64_16x16x4): a wave owns 16
// entries (their K rows as the B operand, in registers: lane l holds dim 4s + l / 16 of entry l % 16 for
// step s), a workgroup 64 entries and one chunk of kPruneChunk updated rows, staged 32 rows at a time in
// LDS as fp64 (the A operand: row l % 16, dim 4s + l / 16).  Which accumulator element is which (row,
// entry) is read off two index products at the start, so the epilogue does not depend on the output
// layout.  The chunk partials (fp64, fixed order) are added in chunk order by prune_sum_kernel.
constexpr int kPruneChunk = 256;
constexpr int kPruneEnt = 64;             // entries per workgroup (16 per wave)
constexpr int kPruneRows = 32;            // rows staged per step

template <int D>
__global__ __launch_bounds__(256) void prune_mass_kernel(const uint16_t* __restrict__ q,
                                                         const uint16_t* __restrict__ kc,
                                                         const int32_t* __restrict__ rows, int k,
                                                         const int32_t* __restrict__ cols, int c_list, int ns,
                                                         const float* __restrict__ lse_ref, int N, int H,
                                                         double sigma, int n_chunks, double* __restrict__ part) {
  constexpr int QS = D + 1;               // padded row stride (doubles): the 16 rows of a read spread over banks
  constexpr int KSTEPS = D / 4;
  __shared__ double qt[kPruneRows * QS];
  __shared__ double q_lse[kPruneRows];
  __shared__ int q_row[kPruneRows];
  __shared__ double red[4][16][17];       // per wave: accumulators by (entry, row) for the ordered sum
  __shared__ int s_rows[kPruneChunk];     // the chunk's updated rows
  __shared__ int s_cnt[4];
  const int h = blockIdx.y % H, chunk = blockIdx.y / H, b = blockIdx.z;
  const int n_ent = c_list - ns;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, kq = lane >> 4;
  const int64_t stride = (int64_t)H * D;
  const int32_t* cl = cols + ((int64_t)b * H + h) * c_list + ns;
  const int32_t* rp = rows + (int64_t)b * k;
  const int p_end = min(k, (chunk + 1) * kPruneChunk);
  const int e_wave = blockIdx.x * kPruneEnt + wave * 16;     // first entry of this wave
  const bool wave_ok = e_wave < n_ent;
  const int j_first = wave_ok ? cl[e_wave] : INT_MAX;        // entries ascend

  // B operand: dims 4s + kq of entry e_wave + l16 (zero past the list's end)
  double kb[KSTEPS];
  {
    const int e = e_wave + l16;
    const bool ok = e < n_ent;
    const uint16_t* src = kc + ((int64_t)b * N + (ok ? cl[e] : 0)) * stride + (int64_t)h * D + kq;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) kb[s] = ok ? (double)bf16_to_f32(src[4 * s]) : 0.0;
  }
  // which (row, entry) each accumulator element holds: D = A B with A = row index in k-column 0, B = 1 in
  // k-row 0 gives the row; the transposed pair gives the entry
  int el_row[4], el_ent[4];
  mfma_f64_layout(l16, kq, el_row, el_ent);
  int el_j[4];                             // column id of each element's entry (INT_MAX past the end)
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int e = e_wave + el_ent[t];
    el_j[t] = e < n_ent ? cl[e] : INT_MAX;
  }
  // the chunk's rows into LDS, and the first one that can see the workgroup's first entry (rows and
  // entries ascend: the rows before it are counted with one ballot per wave)
  const int p0 = chunk * kPruneChunk;
  static_assert(kPruneChunk == 256, "one row of the chunk per thread");
  {
    const int j0 = cl[blockIdx.x * kPruneEnt];
    const int p = p0 + (int)threadIdx.x;
    const int i = p < p_end ? rp[p] : INT_MAX;
    s_rows[threadIdx.x] = i;
    const uint64_t before = __builtin_amdgcn_ballot_w64(i < j0);
    if (lane == 0) s_cnt[wave] = __builtin_popcountll(before);
  }
  __syncthreads();
  const int first = p0 + s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int t0 = first; t0 < p_end; t0 += kPruneRows) {
    for (int x = threadIdx.x; x < kPruneRows * D; x += 256) {
      const int r = x / D, dd = x % D;
      const int p = t0 + r;
      qt[r * QS + dd] = p < p_end ? (double)bf16_to_f32(q[((int64_t)b * N + s_rows[p - p0]) * stride + (int64_t)h * D + dd]) : 0.0;
    }
    if (threadIdx.x < kPruneRows) {
      const int p = t0 + (int)threadIdx.x;
      const int i = p < p_end ? s_rows[p - p0] : -1;
      q_row[threadIdx.x] = i;
      q_lse[threadIdx.x] = p < p_end ? (double)lse_ref[((int64_t)b * N + i) * H + h] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int half = 0; half < kPruneRows / 16; ++half) {
      // uniform: skip 16 rows that all come before this wave's first entry
      const int last_row = q_row[min(16 * half + 15, p_end - t0 - 1)];
      if (wave_ok && last_row >= j_first) {
        f64x4 d4 = {0.0, 0.0, 0.0, 0.0};
        const double* qa = qt + (16 * half + l16) * QS + kq;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) d4 = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[4 * s], kb[s], d4, 0, 0, 0);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int r = 16 * half + el_row[t];
          const int i = q_row[r];                                // -1 past the chunk's last row
          if (i >= el_j[t]) acc[t] += exp(sigma * d4[t] - q_lse[r]);
        }
      }
    }
    __syncthreads();
  }
  // ordered sum over the rows held by the wave's lanes: accumulators by (entry, row group), then entry-wise
#pragma unroll
  for (int t = 0; t < 4; ++t) red[wave][el_ent[t]][el_row[t]] = acc[t];
  __syncthreads();
  if (lane < 16 && wave_ok && e_wave + lane < n_ent) {
    double s = 0.0;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += red[wave][lane][r];
    part[(((int64_t)b * H + h) * n_chunks + chunk) * n_ent + e_wave + lane] = s;
  }
}

// key[b, h, e] = fp32 of the chunks' partial sums of entry e, added in chunk order
__global__ __launch_bounds__(256) void prune_sum_kernel(const double* __restrict__ part, int n_chunks, int n_ent,
                                                        int64_t n_seg, float* __restrict__ key) {
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (x >= n_seg * n_ent) return;
  const int64_t seg = x / n_ent, e = x % n_ent;
  double s = 0.0;
  for (int c = 0; c < n_chunks; ++c) s += part[(seg * n_chunks + c) * n_ent + e];
  key[x] = (float)s;
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
  dim3 grid((N + 63) / 64, H, B);
  if (d == 128) {
    colscore_kernel<128, true><<<grid, 256, 0, st>>>(q, k_cache, N, H, sigma, lse, col_key);
    int rc = check_launch("colscore_kernel(rows)");
    if (rc != FL_OK) return rc;
    colscore_kernel<128, false><<<grid, 256, 0, st>>>(q, k_cache, N, H, sigma, lse, col_key);
  } else {
    colscore_kernel<64, true><<<grid, 256, 0, st>>>(q, k_cache, N, H, sigma, lse, col_key);
    int rc = check_launch("colscore_kernel(rows)");
    if (rc != FL_OK) return rc;
    colscore_kernel<64, false><<<grid, 256, 0, st>>>(q, k_cache, N, H, sigma, lse, col_key);
  }
  return check_launch("colscore_kernel(columns)");
  FL_API_END
}

extern "C" size_t fl_prune_columns_ws(int B, int H, int k, int c_list, int n_sink) {
  if (B < 1 || H < 1 || k < 0 || c_list < 1 || n_sink < 0) return 0;
  const int n_ent = c_list - std::min(n_sink, c_list);
  const int n_chunks = std::max(1, (k + kPruneChunk - 1) / kPruneChunk);
  return (size_t)B * H * n_chunks * n_ent * sizeof(double);
}

extern "C" int fl_prune_columns(const uint16_t* q, const uint16_t* k_cache, const int32_t* rows, int k,
                                const int32_t* cols, int c_list, const float* lse_ref, int B, int N, int H,
                                int d, double sm_scale, int n_sink, int t_next, float* col_key,
                                int32_t* cols_next, void* ws, size_t ws_bytes, void* stream) {
  FL_API_BEGIN
  FL_REQUIRE(q && k_cache && cols && lse_ref && cols_next, FL_E_NULL,
             "fl_prune_columns: q, k_cache, cols, lse_ref and cols_next are required");
  FL_REQUIRE(B >= 1 && N >= 1 && H >= 1, FL_E_SHAPE, "fl_prune_columns: need B, N, H >= 1");
  FL_REQUIRE(d == 64 || d == 128, FL_E_SHAPE, "fl_prune_columns: head dim %d not in {64, 128}", d);
  FL_REQUIRE((int64_t)N * H * d < ((int64_t)1 << 31), FL_E_SHAPE, "fl_prune_columns: N * H * d too large");
  FL_REQUIRE(k >= 0 && k <= N, FL_E_RANGE, "fl_prune_columns: k=%d outside [0, N]", k);
  FL_REQUIRE(k == 0 || rows, FL_E_NULL, "fl_prune_columns: rows are required when k > 0");
  FL_REQUIRE(c_list >= 1 && c_list <= N, FL_E_RANGE, "fl_prune_columns: c_list=%d outside [1, N]", c_list);
  FL_REQUIRE(n_sink >= 0, FL_E_RANGE, "fl_prune_columns: n_sink must be >= 0");
  const int ns = std::min(n_sink, c_list);
  const int n_ent = c_list - ns;
  FL_REQUIRE(t_next >= 0 && t_next <= n_ent, FL_E_RANGE, "fl_prune_columns: t_next=%d outside [0, %d]", t_next,
             n_ent);
  FL_REQUIRE(n_ent <= 65536, FL_E_SHAPE, "fl_prune_columns: %d list entries after the sinks exceed 65536", n_ent);
  FL_REQUIRE(n_ent == 0 || col_key, FL_E_NULL, "fl_prune_columns: col_key is required when entries follow the sinks");
  FL_REQUIRE(sm_scale > 0.0 && std::isfinite(sm_scale), FL_E_RANGE, "fl_prune_columns: sm_scale must be > 0");
  const size_t need = fl_prune_columns_ws(B, H, k, c_list, n_sink);
  FL_REQUIRE(need == 0 || (ws && ws_bytes >= need), FL_E_WORKSPACE,
             "fl_prune_columns: workspace of %zu bytes required", need);
  hipStream_t st = as_stream(stream);
  FL_CHECK_LIST("fl_prune_columns", "rows", rows, B, k, 0, N, st);
  FL_CHECK_LIST("fl_prune_columns", "cols", cols, (int64_t)B * H, c_list, 0, N, st);
  if (n_ent == 0) {                       // the list is all sinks: it is kept as it is
    if (hipMemcpyAsync(cols_next, cols, (size_t)B * H * ns * sizeof(int32_t), hipMemcpyDeviceToDevice, st) !=
        hipSuccess)
      return set_error(FL_E_HIP, "fl_prune_columns: copy of the sinks failed");
    return FL_OK;
  }
  const int n_chunks = std::max(1, (k + kPruneChunk - 1) / kPruneChunk);
  FL_REQUIRE((int64_t)H * n_chunks <= 65535, FL_E_SHAPE, "fl_prune_columns: H * ceil(k / %d) above 65535",
             kPruneChunk);
  double* part = static_cast<double*>(ws);
  dim3 grid((n_ent + kPruneEnt - 1) / kPruneEnt, H * n_chunks, B);
  if (d == 128)
    prune_mass_kernel<128><<<grid, 256, 0, st>>>(q, k_cache, rows, k, cols, c_list, ns, lse_ref, N, H, sm_scale,
                                                 n_chunks, part);
  else
    prune_mass_kernel<64><<<grid, 256, 0, st>>>(q, k_cache, rows, k, cols, c_list, ns, lse_ref, N, H, sm_scale,
                                                n_chunks, part);
  int rc = check_launch("prune_mass_kernel");
  if (rc != FL_OK) return rc;
  const int64_t total = (int64_t)B * H * n_ent;
  prune_sum_kernel<<<(unsigned)((total + 255) / 256), 256, 0, st>>>(part, n_chunks, n_ent, (int64_t)B * H, col_key);
  rc = check_launch("prune_sum_kernel");
  if (rc != FL_OK) return rc;
  return launch_topk(B * H, col_key, n_ent, n_ent, t_next, cols + ns, c_list, 0, cols_next, ns + t_next, ns,
                     nullptr, 0, st);
  FL_API_END
}
