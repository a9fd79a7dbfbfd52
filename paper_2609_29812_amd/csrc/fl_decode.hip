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
// One row per (b, h) is a GEMV: HBM-bound, split over columns.  Two launches:
//   decode_partial   chunks of 128 positions: fp64 logits (exact bf16 products, fp64 sums) and their fp32
//                    ranking keys (forced columns +inf), the chunk's max and exp-sum, and the
//                    exp-weighted sum of its V rows (fp32); K and V rows are each read once, 16 bytes per
//                    lane, D/8 lanes per row.
//   decode_finalize  one 1024-thread workgroup per (b, h): merges the chunks into L and the output, and
//                    forms the next loop's columns, mass and subtract term: directly when every column
//                    is kept, else by the radix top-k of fl_topk.h over the keys and a gather of the
//                    selected V rows (read once more).
#include "fl_common.h"
#include "fl_topk.h"

#include <mutex>

namespace fl {

constexpr int kDecChunk = 128;           // positions per partial workgroup
constexpr int kSelWin = 1024;            // selected positions gathered per round of the finalize

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
  float* key;                // ws [B*H, n]
  const int32_t* sel;        // ws [B*H, c_next] selected positions
  int32_t* cols_next;        // [B, H, c_next]
  float* mass_next;          // [B, H]
  float* sub_next;           // [B, H, D]
  int B, T, H, n, nch, c_next, n_sink, window;
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

// ---- finalize: one 1024-thread workgroup per (b, h) ----------------------------------------------------
// (1) merges the chunks into L and the output; (2) with c_next > 0, the next loop's columns, mass m' =
// sum_{S'} p_j and subtract term sub' = sum_{S'} p_j V_j.  When the next loop keeps every column
// (c_next = n) these are the columns themselves, m' = m (the probabilities over S sum to m) and sub' = the
// add term just formed.  Otherwise the radix top-k of fl_topk.h writes the selected positions (ascending)
// to the workspace, and windows of kSelWin of them are gathered: ids, logits and weights into LDS, then
// their V rows (every load of a window issued before any use); the waves' sums are added in order
// (deterministic).
template <int D, int M>
__global__ __launch_bounds__(kTopkThreads) void decode_finalize_kernel(DecodeArgs a) {
  constexpr int NW = kTopkThreads / 64;      // waves
  constexpr int PARTS = kTopkThreads / D;    // threads per output dimension in the merge
  constexpr int LPC = D / 8;                 // lanes per V row (16 bytes each)
  constexpr int CPW = 64 / LPC;              // rows per wave instruction
  constexpr int IT = kSelWin / (NW * CPW);   // window rows per lane
  static_assert(IT * NW * CPW == kSelWin && kSelWin == kTopkThreads, "one id per thread, IT rows per lane");
  constexpr int BUF = NW * D > 2 * kSelWin ? NW * D : 2 * kSelWin;
  __shared__ double s_m[NW];
  __shared__ double s_l;
  __shared__ float s_f[512];                 // chunk weights (nch <= 512)
  __shared__ __attribute__((aligned(16))) float s_buf[BUF];   // partial sums; a window's ids and weights
  float (*s_acc)[D] = reinterpret_cast<float (*)[D]>(s_buf);
  int32_t* s_col = reinterpret_cast<int32_t*>(s_buf);
  float* s_w = s_buf + kSelWin;
  const int bh = blockIdx.x;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool dense = a.cols == nullptr;
  const double m = dense ? 1.0 : (double)a.mass[bh];
  // (1) L = M + log S over the chunks' maxima and exp-sums; the add term and the output
  double mx = -INFINITY;
  for (int c = tid; c < a.nch; c += kTopkThreads) mx = fmax(mx, a.pmax[(int64_t)bh * a.nch + c]);
  mx = wave_max_f64(mx);
  if (lane == 0) s_m[wave] = mx;
  __syncthreads();
  double Mx = s_m[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) Mx = fmax(Mx, s_m[w]);
  __syncthreads();
  double es = 0.0;
  for (int c = tid; c < a.nch; c += kTopkThreads) {
    const int64_t sidx = (int64_t)bh * a.nch + c;
    es += a.psum[sidx] * exp(a.pmax[sidx] - Mx);
  }
  es = wave_sum_f64_dec(es);
  if (lane == 0) s_m[wave] = es;
  __syncthreads();
  if (tid == 0) {
    double S = 0.0;
    for (int w = 0; w < NW; ++w) S += s_m[w];
    s_l = S;
  }
  __syncthreads();
  const double S = s_l;
  const double L = Mx + log(S);
  for (int c = tid; c < a.nch; c += kTopkThreads) s_f[c] = (float)(m * exp(a.pmax[(int64_t)bh * a.nch + c] - Mx) / S);
  __syncthreads();
  {
    // thread (part, dd) adds the chunks part, part + PARTS, ...; the parts are then added in order
    const int dd = tid % D, part = tid / D;
    float add = 0.0f;
    for (int c = part; c < a.nch; c += PARTS) add = fmaf(s_f[c], a.pacc[((int64_t)bh * a.nch + c) * D + dd], add);
    s_acc[part][dd] = add;
  }
  __syncthreads();
  float o_add = 0.0f;
  if (tid < D) {
#pragma unroll
    for (int q = 0; q < PARTS; ++q) o_add += s_acc[q][tid];
    const int64_t od = (int64_t)bh * D + tid;
    a.o[od] = dense ? o_add : a.o[od] - a.sub[od] + o_add;
  }
  if (tid == 0 && a.lse) a.lse[bh] = (float)L;
  if (a.c_next == 0) return;               // uniform
  if (a.c_next == a.n) {                   // every column kept
    for (int i = tid; i < a.n; i += kTopkThreads) a.cols_next[(int64_t)bh * a.n + i] = dec_col(a, bh, i);
    if (tid < D) a.sub_next[(int64_t)bh * D + tid] = o_add;
    if (tid == 0) a.mass_next[bh] = (float)m;
    return;
  }
  // (2) the selected positions, ascending, into the workspace; this workgroup's writes are visible to
  // its own threads after a workgroup-scope release and acquire around the barrier
  int32_t* sel = const_cast<int32_t*>(a.sel) + (int64_t)bh * a.c_next;
  topk_block<M>(a.key + (int64_t)bh * a.n, a.n, a.c_next, nullptr, 0, sel, 0, nullptr, 0);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  const int sl = lane % LPC, grp = lane / LPC;
  const int64_t HD = (int64_t)a.H * D;
  double ms = 0.0;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int lo = 0; lo < a.c_next; lo += kSelWin) {
    // ids, weights p_j = m exp(l_j - L) and the next loop's columns of the window (thread t: entry t)
    {
      const int i = lo + tid;
      const bool ok = i < a.c_next;
      const int p = ok ? sel[i] : 0;
      const int col = dec_col(a, bh, p);
      const double pr = ok ? m * exp(a.logit[(int64_t)bh * a.n + p] - L) : 0.0;
      if (ok) a.cols_next[(int64_t)bh * a.c_next + i] = col;
      ms += pr;
      s_col[tid] = col;
      s_w[tid] = (float)pr;
    }
    __syncthreads();
    // their V rows: wave w, row group g takes window entries (w * CPW + g) + it * NW * CPW
    uint4 vw[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int e = wave * CPW + grp + it * NW * CPW;
      vw[it] = *reinterpret_cast<const uint4*>(a.v + ((int64_t)b * a.T + s_col[e]) * HD + (int64_t)h * D + 8 * sl);
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int e = wave * CPW + grp + it * NW * CPW;
      const float wf = s_w[e];             // 0 past the end of the selection
      const uint32_t ws[4] = {vw[it].x, vw[it].y, vw[it].z, vw[it].w};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        acc[2 * t] = fmaf(wf, bf16_to_f32(ws[t] & 0xFFFFu), acc[2 * t]);
        acc[2 * t + 1] = fmaf(wf, bf16_to_f32(ws[t] >> 16), acc[2 * t + 1]);
      }
    }
    __syncthreads();                       // the window's ids and weights are no longer read
  }
  ms = wave_sum_f64_dec(ms);
#pragma unroll
  for (int t = 0; t < 8; ++t)
    for (int off = LPC; off < 64; off <<= 1) acc[t] += __shfl_xor(acc[t], off, 64);
  if (lane < LPC) {
#pragma unroll
    for (int t = 0; t < 8; ++t) s_acc[wave][8 * sl + t] = acc[t];
  }
  if (lane == 0) s_m[wave] = ms;
  __syncthreads();
  if (tid < D) {
    float sacc = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) sacc += s_acc[w][tid];
    a.sub_next[(int64_t)bh * D + tid] = sacc;
  }
  if (tid == 0) {
    double mt = 0.0;
    for (int w = 0; w < NW; ++w) mt += s_m[w];
    a.mass_next[bh] = (float)mt;
  }
}

// workspace regions, each 256-byte aligned
struct DecodeWs {
  size_t logit, pmax, psum, pacc, key, sel, total;
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
  w.key = off; off += al(bh * n * sizeof(float));
  w.sel = off; off += al(bh * (size_t)c_next * sizeof(int32_t));
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
  a.key = reinterpret_cast<float*>(base + L.key);
  a.sel = reinterpret_cast<const int32_t*>(base + L.sel);
  a.cols_next = cols_next; a.mass_next = mass_next; a.sub_next = sub_next;
  a.B = B; a.T = T; a.H = H; a.n = n; a.nch = (n + kDecChunk - 1) / kDecChunk; a.c_next = c_next;
  a.n_sink = n_sink; a.window = window; a.scale = (double)sm_scale;
  const int BH = B * H;
  dim3 gp(a.nch, BH);
  if (d == 128) decode_partial_kernel<128><<<gp, 256, 0, st>>>(a);
  else decode_partial_kernel<64><<<gp, 256, 0, st>>>(a);
  int rc = check_launch("decode_partial_kernel");
  if (rc != FL_OK) return rc;
  // finalize: the top-k's register depth follows the number of keys (as in the selection kernels)
  const int per = (n + kTopkThreads - 1) / kTopkThreads;
  const dim3 gf(BH);
#define FL_FIN(MM)                                                                        \
  do {                                                                                    \
    if (d == 128) decode_finalize_kernel<128, MM><<<gf, kTopkThreads, 0, st>>>(a);        \
    else decode_finalize_kernel<64, MM><<<gf, kTopkThreads, 0, st>>>(a);                  \
  } while (0)
  if (per <= 1) FL_FIN(1);
  else if (per <= 2) FL_FIN(2);
  else if (per <= 4) FL_FIN(4);
  else if (per <= 8) FL_FIN(8);
  else if (per <= 16) FL_FIN(16);
  else if (per <= 32) FL_FIN(32);
  else FL_FIN(64);
#undef FL_FIN
  return check_launch("decode_finalize_kernel");
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
