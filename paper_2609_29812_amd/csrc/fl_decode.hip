// Decode step of one loop for the newest position (Appendix D.2, Eqs. (6) and (7) for one query row).
//
// For each (batch, head) the query of position t = T-1 attends over the column set S that the previous
// loop selected (or over every column 0..T-1 for a dense source loop), with the cached mass m:
//   p_j = m * exp(l_j - L), l_j = sm_scale * q . K_j, L = logsumexp over S,
//   o <- o - sub + sum_j p_j V_j          (dense: o = sum_j p_j V_j, m = 1),
// then selects the next loop's S' (sinks and window forced, then the largest p, ties to the lower
// column) and forms its mass m' = sum_{S'} p_j and subtract term sub' = sum_{S'} p_j V_j.  Within a row
// p_j grows with l_j, so the ranking key is fp32(l_j), available before L is known.
//
// One row per (b, h) is a GEMV: HBM-bound, split over columns.
//   decode_partial  chunks of 128 positions: fp64 logits (exact bf16 products, fp64 sums) and their fp32
//                   ranking keys (forced columns +inf), the chunk's max and exp-sum, and the
//                   exp-weighted sum of its V rows (fp32); K and V rows are each read once, 16 bytes per
//                   lane, D/8 lanes per row.
//   decode_combine  one workgroup per (b, h): merges the chunks into L and the output.
//   topk_select     the radix top-k of fl_select.hip over the keys (positions, ascending).
//   decode_select  workgroups of 256 selected positions: the selected columns and their parts of the
//                   mass and subtract term; then one workgroup per (b, h) adds the parts in order.
#include "fl_common.h"

#include <mutex>

namespace fl {

constexpr int kDecChunk = 128;           // positions per partial workgroup
constexpr int kSelChunk = 256;           // selected positions per selection workgroup

// 16-byte load marked non-temporal: the K and V rows of a step are streamed once
typedef uint32_t u32x4d __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 stream16(const uint16_t* p) {
  const u32x4d w = __builtin_nontemporal_load(reinterpret_cast<const u32x4d*>(p));
  return make_uint4(w[0], w[1], w[2], w[3]);
}

struct DecodeArgs {
  const uint16_t* q;         // [B, H, D]
  const uint16_t* k;         // [B, T, H, D]
  const uint16_t* v;
  const int32_t* cols;       // [B, H, c] or NULL (dense)
  const float* mass;         // [B, H]
  const float* sub;          // [B, H, D]
  float* o;                  // [B, H, D]
  float* lse;                // [B, H] optional
  double* logit;             // ws [B*H, n]
  double* pmax;              // ws [B*H, nch] chunk max
  double* psum;              // ws [B*H, nch] chunk exp-sum
  float* pacc;               // ws [B*H, nch, D]
  double* ltot;              // ws [B*H] log-normaliser
  float* key;                // ws [B*H, n]
  const int32_t* sel;        // ws [B*H, c_next] selected positions
  double* fmass;             // ws [B*H, nfc] parts of the next mass
  float* fsub;               // ws [B*H, nfc, D] parts of the next subtract term
  int32_t* cols_next;        // [B, H, c_next]
  float* mass_next;          // [B, H]
  float* sub_next;           // [B, H, D]
  int B, T, H, n, nch, c_next, nfc, n_sink, window;
  double scale;
};

__device__ __forceinline__ int dec_col(const DecodeArgs& a, int bh, int p) {
  return a.cols ? a.cols[(int64_t)bh * a.n + p] : p;
}

__device__ __forceinline__ double wave_max_f64(double x) {
  for (int off = 32; off > 0; off >>= 1) x = fmax(x, __shfl_xor(x, off, 64));
  return x;
}
__device__ __forceinline__ double wave_sum_f64_dec(double x) {
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// ---- partial: one chunk of positions of one (b, h) -------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void decode_partial_kernel(DecodeArgs a) {
  constexpr int LPC = D / 8;                 // lanes per row (16 bytes each)
  constexpr int CPW = 64 / LPC;              // rows per wave instruction
  constexpr int PER_WAVE = kDecChunk / 4;    // positions per wave
  constexpr int IT = PER_WAVE / CPW;
  __shared__ double s_red[4];
  __shared__ float s_acc[4][D];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sl = lane % LPC, grp = lane / LPC;
  const int chunk = blockIdx.x, bh = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int64_t HD = (int64_t)a.H * D;
  double qd[8];
  {
    const uint4 w = *reinterpret_cast<const uint4*>(a.q + (int64_t)bh * D + 8 * sl);
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      qd[2 * t] = (double)bf16_to_f32(ws[t] & 0xFFFFu);
      qd[2 * t + 1] = (double)bf16_to_f32(ws[t] >> 16);
    }
  }
  // pass 1: logits (every lane of a row group ends with the row's full dot product).  All column ids,
  // then all K and V loads, are issued before any use, so a chunk costs two load latencies.
  double lg[IT];
  int colv[IT];
  uint4 kw[IT], vw[IT];
  double mx = -INFINITY;
  const int p0 = chunk * kDecChunk + wave * PER_WAVE + grp;
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int p = p0 + it * CPW;
    colv[it] = p < a.n ? dec_col(a, bh, p) : 0;
  }
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int64_t off = ((int64_t)b * a.T + colv[it]) * HD + (int64_t)h * D + 8 * sl;
    kw[it] = stream16(a.k + off);
    vw[it] = stream16(a.v + off);
  }
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int p = p0 + it * CPW;
    const bool ok = p < a.n;
    const int col = colv[it];
    const uint4 w = kw[it];
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
    double acc = 0.0;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      acc = fma((double)bf16_to_f32(ws[t] & 0xFFFFu), qd[2 * t], acc);
      acc = fma((double)bf16_to_f32(ws[t] >> 16), qd[2 * t + 1], acc);
    }
#pragma unroll
    for (int off = 1; off < LPC; off <<= 1) acc += __shfl_xor(acc, off, 64);
    const double l = ok ? a.scale * acc : -INFINITY;
    lg[it] = l;
    mx = fmax(mx, l);
    if (ok && sl == 0) {
      a.logit[(int64_t)bh * a.n + p] = l;
      if (a.c_next > 0) {
        const bool forced = col < a.n_sink || (a.window > 0 && col >= a.T - a.window);
        a.key[(int64_t)bh * a.n + p] = forced ? INFINITY : (float)l;
      }
    }
  }
  mx = wave_max_f64(mx);
  if (lane == 0) s_red[wave] = mx;
  __syncthreads();
  mx = fmax(fmax(s_red[0], s_red[1]), fmax(s_red[2], s_red[3]));
  __syncthreads();
  // pass 2: exp-weights against the chunk max, exp-sum and the weighted V rows
  // (every lane of a row group holds the same logits: lane sl of the group takes the exponential of the
  // group's position sl and the group shares them by shuffles, one fp64 exp per lane instead of IT)
  static_assert(IT <= LPC, "one position per lane of a row group");
  double mine = 0.0;
#pragma unroll
  for (int it = 0; it < IT; ++it) mine = sl % IT == it ? lg[it] : mine;
  mine = exp(mine - mx);                        // 0 for positions past the end
  double es = 0.0;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const double e = __shfl(mine, grp * LPC + it, 64);
    if (sl == 0) es += e;
    const float wf = (float)e;
    const uint4 w = vw[it];
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      acc[2 * t] = fmaf(wf, bf16_to_f32(ws[t] & 0xFFFFu), acc[2 * t]);
      acc[2 * t + 1] = fmaf(wf, bf16_to_f32(ws[t] >> 16), acc[2 * t + 1]);
    }
  }
  es = wave_sum_f64_dec(es);
  // rows of a wave -> lanes 0..LPC-1, then the four waves through LDS
#pragma unroll
  for (int t = 0; t < 8; ++t)
    for (int off = LPC; off < 64; off <<= 1) acc[t] += __shfl_xor(acc[t], off, 64);
  if (lane < LPC) {
#pragma unroll
    for (int t = 0; t < 8; ++t) s_acc[wave][8 * sl + t] = acc[t];
  }
  if (lane == 0) s_red[wave] = es;
  __syncthreads();
  const int64_t slot = (int64_t)bh * a.nch + chunk;
  if (threadIdx.x < D) {
    const int dd = threadIdx.x;
    a.pacc[slot * D + dd] = s_acc[0][dd] + s_acc[1][dd] + s_acc[2][dd] + s_acc[3][dd];
  }
  if (threadIdx.x == 0) {
    a.pmax[slot] = mx;
    a.psum[slot] = s_red[0] + s_red[1] + s_red[2] + s_red[3];
  }
}

// ---- combine: the output of one (b, h) from its chunks (nch <= 512) -------------------------------------
template <int D>
__global__ __launch_bounds__(256) void decode_combine_kernel(DecodeArgs a) {
  __shared__ double s_m[4];
  __shared__ double s_l;
  __shared__ float s_f[512];
  const int bh = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool dense = a.cols == nullptr;
  const double m = dense ? 1.0 : (double)a.mass[bh];
  double mx = -INFINITY;
  for (int c = tid; c < a.nch; c += 256) mx = fmax(mx, a.pmax[(int64_t)bh * a.nch + c]);
  mx = wave_max_f64(mx);
  if (lane == 0) s_m[wave] = mx;
  __syncthreads();
  const double M = fmax(fmax(s_m[0], s_m[1]), fmax(s_m[2], s_m[3]));
  __syncthreads();
  double es = 0.0;
  for (int c = tid; c < a.nch; c += 256) {
    const int64_t sidx = (int64_t)bh * a.nch + c;
    es += a.psum[sidx] * exp(a.pmax[sidx] - M);
  }
  es = wave_sum_f64_dec(es);
  if (lane == 0) s_m[wave] = es;
  __syncthreads();
  if (tid == 0) s_l = s_m[0] + s_m[1] + s_m[2] + s_m[3];
  __syncthreads();
  const double S = s_l;
  const double L = M + log(S);
  for (int c = tid; c < a.nch; c += 256) s_f[c] = (float)(m * exp(a.pmax[(int64_t)bh * a.nch + c] - M) / S);
  __syncthreads();
  if (tid < D) {
    float add = 0.0f;
    for (int c = 0; c < a.nch; ++c) add = fmaf(s_f[c], a.pacc[((int64_t)bh * a.nch + c) * D + tid], add);
    const int64_t od = (int64_t)bh * D + tid;
    a.o[od] = dense ? add : a.o[od] - a.sub[od] + add;
  }
  if (tid == 0) {
    a.ltot[bh] = L;
    if (a.lse) a.lse[bh] = (float)L;
  }
}

// ---- finalize: the next loop's columns, mass and subtract term ---------------------------------------
// decode_select_partial: a workgroup takes 256 selected positions of one (b, h) (ids, probabilities and
// weighted V rows, every load of a stage issued before any use); decode_select_reduce adds the
// workgroups' parts in order (deterministic) into the mass and subtract term.
template <int D>
__global__ __launch_bounds__(256) void decode_select_partial_kernel(DecodeArgs a) {
  constexpr int LPC = D / 8;
  constexpr int CPW = 64 / LPC;
  constexpr int IT = (kSelChunk / 4) / CPW;
  __shared__ double s_red[4];
  __shared__ float s_acc[4][D];
  const int chunk = blockIdx.x, bh = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sl = lane % LPC, grp = lane / LPC;
  const int64_t HD = (int64_t)a.H * D;
  const double m = a.cols == nullptr ? 1.0 : (double)a.mass[bh];
  const double L = a.ltot[bh];
  const int i0 = chunk * kSelChunk + wave * (kSelChunk / 4) + grp;
  int p[IT], col[IT];
  double l[IT];
  uint4 w[IT];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int i = i0 + it * CPW;
    p[it] = i < a.c_next ? a.sel[(int64_t)bh * a.c_next + i] : 0;
  }
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    col[it] = dec_col(a, bh, p[it]);
    l[it] = a.logit[(int64_t)bh * a.n + p[it]];
  }
#pragma unroll
  for (int it = 0; it < IT; ++it)
    w[it] = *reinterpret_cast<const uint4*>(a.v + ((int64_t)b * a.T + col[it]) * HD + (int64_t)h * D + 8 * sl);
  double ms = 0.0;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int i = i0 + it * CPW;
    const bool ok = i < a.c_next;
    const double pr = ok ? m * exp(l[it] - L) : 0.0;
    if (ok && sl == 0) {
      a.cols_next[(int64_t)bh * a.c_next + i] = col[it];
      ms += pr;
    }
    const float wf = (float)pr;
    const uint32_t ws[4] = {w[it].x, w[it].y, w[it].z, w[it].w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      acc[2 * t] = fmaf(wf, bf16_to_f32(ws[t] & 0xFFFFu), acc[2 * t]);
      acc[2 * t + 1] = fmaf(wf, bf16_to_f32(ws[t] >> 16), acc[2 * t + 1]);
    }
  }
  ms = wave_sum_f64_dec(ms);
#pragma unroll
  for (int t = 0; t < 8; ++t)
    for (int off = LPC; off < 64; off <<= 1) acc[t] += __shfl_xor(acc[t], off, 64);
  if (lane < LPC) {
#pragma unroll
    for (int t = 0; t < 8; ++t) s_acc[wave][8 * sl + t] = acc[t];
  }
  if (lane == 0) s_red[wave] = ms;
  __syncthreads();
  const int64_t slot = (int64_t)bh * a.nfc + chunk;
  if (threadIdx.x < D) {
    const int dd = threadIdx.x;
    a.fsub[slot * D + dd] = s_acc[0][dd] + s_acc[1][dd] + s_acc[2][dd] + s_acc[3][dd];
  }
  if (threadIdx.x == 0) a.fmass[slot] = s_red[0] + s_red[1] + s_red[2] + s_red[3];
}

template <int D>
__global__ __launch_bounds__(256) void decode_select_reduce_kernel(DecodeArgs a) {
  const int bh = blockIdx.x;
  if (threadIdx.x < D) {
    float sacc = 0.0f;
    for (int c = 0; c < a.nfc; ++c) sacc += a.fsub[((int64_t)bh * a.nfc + c) * D + threadIdx.x];
    a.sub_next[(int64_t)bh * D + threadIdx.x] = sacc;
  }
  if (threadIdx.x == 0) {
    double ms = 0.0;
    for (int c = 0; c < a.nfc; ++c) ms += a.fmass[(int64_t)bh * a.nfc + c];
    a.mass_next[bh] = (float)ms;
  }
}

// workspace regions, each 256-byte aligned
struct DecodeWs {
  size_t logit, pmax, psum, pacc, ltot, key, sel, fmass, fsub, total;
};
static DecodeWs decode_ws(int B, int H, int d, int n, int c_next) {
  auto al = [](size_t x) { return (x + 255) / 256 * 256; };
  const size_t bh = (size_t)B * H;
  const size_t nch = ((size_t)n + kDecChunk - 1) / kDecChunk;
  DecodeWs w;
  size_t off = 0;
  w.logit = off; off += al(bh * n * sizeof(double));
  w.pmax = off; off += al(bh * nch * sizeof(double));
  w.psum = off; off += al(bh * nch * sizeof(double));
  w.pacc = off; off += al(bh * nch * d * sizeof(float));
  w.ltot = off; off += al(bh * sizeof(double));
  w.key = off; off += al(bh * n * sizeof(float));
  w.sel = off; off += al(bh * (size_t)c_next * sizeof(int32_t));
  const size_t nfc = ((size_t)c_next + kSelChunk - 1) / kSelChunk;
  w.fmass = off; off += al(bh * nfc * sizeof(double));
  w.fsub = off; off += al(bh * nfc * d * sizeof(float));
  w.total = off;
  return w;
}

}  // namespace fl

using namespace fl;

extern "C" size_t fl_decode_step_ws(int B, int T, int H, int d, int c, int c_next) {
  if (B < 1 || T < 1 || H < 1 || (d != 64 && d != 128) || c < 0 || c_next < 0) return 0;
  const int n = c > 0 ? c : T;
  return decode_ws(B, H, d, n, c_next).total;
}

static int decode_scratch(void** out);

// ws == nullptr with use_scratch: the library's own scratch array, looked up after the arguments pass
static int decode_step(const char* fn, bool use_scratch, const uint16_t* q, const uint16_t* k_cache,
                       const uint16_t* v_cache, const int32_t* cols, int c, const float* mass, const float* sub,
                       int B, int T, int H, int d, float sm_scale, float* o, float* lse, int n_sink, int window, int c_next,
                       int32_t* cols_next, float* mass_next, float* sub_next, void* ws, size_t ws_bytes,
                       void* stream) {
  FL_REQUIRE(q && k_cache && v_cache && o, FL_E_NULL, "%s: q, k_cache, v_cache and o are required", fn);
  FL_REQUIRE(B >= 1 && T >= 1 && H >= 1, FL_E_SHAPE, "%s: need B, T, H >= 1", fn);
  FL_REQUIRE(d == 64 || d == 128, FL_E_SHAPE, "%s: head dim %d not in {64, 128}", fn, d);
  FL_REQUIRE((int64_t)T * H * d < ((int64_t)1 << 31), FL_E_SHAPE, "%s: T * H * d too large", fn);
  FL_REQUIRE(sm_scale > 0.0f && std::isfinite(sm_scale), FL_E_RANGE, "%s: sm_scale must be > 0", fn);
  const bool dense = cols == nullptr;
  if (dense) {
    FL_REQUIRE(c == 0 || c == T, FL_E_SHAPE, "%s: without cols, c must be 0 or T", fn);
  } else {
    FL_REQUIRE(c >= 1 && c <= T, FL_E_RANGE, "%s: c=%d outside [1, T]", fn, c);
    FL_REQUIRE(mass && sub, FL_E_NULL, "%s: a sparse loop needs its cached mass and subtract term", fn);
  }
  const int n = dense ? T : c;
  FL_REQUIRE(n <= 65536, FL_E_SHAPE, "%s: %d columns exceed the 65536 the selection supports", fn, n);
  FL_REQUIRE(c_next >= 0 && c_next <= n, FL_E_RANGE, "%s: c_next=%d outside [0, %d]", fn, c_next, n);
  FL_REQUIRE(c_next == 0 || (cols_next && mass_next && sub_next), FL_E_NULL,
             "%s: cols_next, mass_next and sub_next are required when c_next > 0", fn);
  FL_REQUIRE(n_sink >= 0 && window >= 0, FL_E_RANGE, "%s: n_sink and window must be >= 0", fn);
  const DecodeWs L = decode_ws(B, H, d, n, c_next);
  if (use_scratch) {
    FL_REQUIRE(L.total <= (size_t)FL_DECODE_SCRATCH_BYTES, FL_E_RANGE,
               "%s: the step needs %zu bytes of scratch, above the %zu available (use fl_decode_step with a "
               "workspace)", fn, L.total, (size_t)FL_DECODE_SCRATCH_BYTES);
    const int rc = decode_scratch(&ws);
    if (rc != FL_OK) return rc;
    ws_bytes = (size_t)FL_DECODE_SCRATCH_BYTES;
  }
  FL_REQUIRE(ws && ws_bytes >= L.total, FL_E_WORKSPACE, "%s: workspace of %zu bytes required", fn, L.total);
  hipStream_t st = as_stream(stream);
  FL_CHECK_LIST(fn, "cols", cols, (int64_t)B * H, c, 0, T, st);
  char* base = static_cast<char*>(ws);
  DecodeArgs a{};
  a.q = q; a.k = k_cache; a.v = v_cache; a.cols = cols; a.mass = mass; a.sub = sub; a.o = o; a.lse = lse;
  a.logit = reinterpret_cast<double*>(base + L.logit);
  a.pmax = reinterpret_cast<double*>(base + L.pmax);
  a.psum = reinterpret_cast<double*>(base + L.psum);
  a.pacc = reinterpret_cast<float*>(base + L.pacc);
  a.ltot = reinterpret_cast<double*>(base + L.ltot);
  a.key = reinterpret_cast<float*>(base + L.key);
  a.sel = reinterpret_cast<const int32_t*>(base + L.sel);
  a.fmass = reinterpret_cast<double*>(base + L.fmass);
  a.fsub = reinterpret_cast<float*>(base + L.fsub);
  a.cols_next = cols_next; a.mass_next = mass_next; a.sub_next = sub_next;
  a.B = B; a.T = T; a.H = H; a.n = n; a.nch = (n + kDecChunk - 1) / kDecChunk; a.c_next = c_next;
  a.nfc = (c_next + kSelChunk - 1) / kSelChunk;
  a.n_sink = n_sink; a.window = window; a.scale = (double)sm_scale;
  const int BH = B * H;
  dim3 gp(a.nch, BH);
  if (d == 128) decode_partial_kernel<128><<<gp, 256, 0, st>>>(a);
  else decode_partial_kernel<64><<<gp, 256, 0, st>>>(a);
  int rc = check_launch("decode_partial_kernel");
  if (rc != FL_OK) return rc;
  if (d == 128) decode_combine_kernel<128><<<BH, 256, 0, st>>>(a);
  else decode_combine_kernel<64><<<BH, 256, 0, st>>>(a);
  rc = check_launch("decode_combine_kernel");
  if (rc != FL_OK || c_next == 0) return rc;
  rc = launch_topk(BH, a.key, n, n, c_next, nullptr, 0, 0, const_cast<int32_t*>(a.sel), c_next, 0, nullptr, 0, st);
  if (rc != FL_OK) return rc;
  dim3 gf(a.nfc, BH);
  if (d == 128) decode_select_partial_kernel<128><<<gf, 256, 0, st>>>(a);
  else decode_select_partial_kernel<64><<<gf, 256, 0, st>>>(a);
  rc = check_launch("decode_select_partial_kernel");
  if (rc != FL_OK) return rc;
  if (d == 128) decode_select_reduce_kernel<128><<<BH, 256, 0, st>>>(a);
  else decode_select_reduce_kernel<64><<<BH, 256, 0, st>>>(a);
  return check_launch("decode_select_reduce_kernel");
}

extern "C" int fl_decode_step(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                              const int32_t* cols, int c, const float* mass, const float* sub, int B, int T,
                              int H, int d, float sm_scale, float* o, float* lse, int n_sink, int window,
                              int c_next, int32_t* cols_next, float* mass_next, float* sub_next, void* ws,
                              size_t ws_bytes, void* stream) {
  FL_API_BEGIN
  return decode_step("fl_decode_step", false, q, k_cache, v_cache, cols, c, mass, sub, B, T, H, d, sm_scale, o, lse,
                     n_sink, window, c_next, cols_next, mass_next, sub_next, ws, ws_bytes, stream);
  FL_API_END
}

// ---- the decode step without a caller workspace ----------------------------------------------------------
// The workspace lives in a file-scope device array of FL_DECODE_SCRATCH_BYTES, one copy per GPU, held
// until the process ends.  Host code never passes the array's name to a kernel (on the host it is only a
// stand-in for the symbol): the device address of each GPU's copy is looked up once with
// hipGetSymbolAddress, with that GPU current, and that address is what the kernels receive.  Every region
// of the workspace is written before it is read within one call, so nothing needs clearing between calls.
static __device__ __align__(256) unsigned char scratch[FL_DECODE_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];
}  // namespace

static int decode_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  FL_REQUIRE(e == hipSuccess && dev >= 0 && dev < kMaxDevices, FL_E_HIP,
             "fl_decode_step_noalloc: no current device (%s)", hipGetErrorString(e));
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    FL_REQUIRE(e == hipSuccess && p != nullptr, FL_E_HIP,
               "fl_decode_step_noalloc: hipGetSymbolAddress failed on device %d (%s)", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FL_OK;
}

extern "C" int fl_decode_step_noalloc(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                                      const int32_t* cols, int c, const float* mass, const float* sub, int B,
                                      int T, int H, int d, float sm_scale, float* o, float* lse, int n_sink,
                                      int window, int c_next, int32_t* cols_next, float* mass_next,
                                      float* sub_next, void* stream) {
  FL_API_BEGIN
  return decode_step("fl_decode_step_noalloc", true, q, k_cache, v_cache, cols, c, mass, sub, B, T, H, d, sm_scale,
                     o, lse, n_sink, window, c_next, cols_next, mass_next, sub_next, nullptr, 0, stream);
  FL_API_END
}
