// Mass-corrected sparse attention update (Sections 3.2 and 4.2, Eq. 3; Appendix D.2, Eq. 7) and the
// dense source loop (Eq. 2, causal).
//
// A wave owns 32 updated rows of one (batch, head).  Columns are visited in tiles of 32:
//   list phase : entries of the per-(batch, head) column list with j + window <= i (columns inside the
//                row's band are left to the band phase, so a column in both is counted once);
//   band phase : the contiguous range covering every row's band (i - window, i], masked per row;
//                the dense loop is the band phase with an unbounded window.
// Per tile the gathered K rows are staged in LDS row-major (bf16) and the V rows transposed (fp16), for
// the loop r-1 state (cache) and the loop r state (new rows via the slot map, cache otherwise).
// Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16 so that each lane holds
// 16 columns of a single row; the probabilities then feed O^T += V^T P^T (v_mfma_f32_32x32x16_f16)
// straight from registers, and every accumulator of a lane belongs to that lane's row.
//   subtract pass : pp = exp(a - lse_ref), no running max needed (lse_ref bounds the logits);
//   add pass      : online softmax with a running max shared by the two half-waves of a row.
#include "fl_common.h"

namespace fl {

constexpr int kBM = 32;      // rows per wave
constexpr int kBN = 32;      // columns per tile
constexpr int kKPad = 8;     // bf16 elements of padding per LDS K row
constexpr int kVPad = 4;     // fp16 elements of padding per LDS V^T row

struct AttnArgs {
  const uint16_t* q_cur;
  const uint16_t* q_prev;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const uint16_t* k_new;
  const uint16_t* v_new;
  const int32_t* slot;
  const int32_t* rows;
  const int32_t* cols;
  float* lse_ref;
  float* o;
  int k, c_list, window, N, H;
  float scale_log2;   // sm_scale * log2(e)
  int dense;
};

template <int D>
struct AttnSmem {
  uint16_t k[2][kBN][D + kKPad];     // [0] loop r-1 (cache), [1] loop r
  _Float16 vt[2][D][kBN + kVPad];
  int cid[kBN];
  int nslot[kBN];
};

__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  _Float16 ha = (_Float16)a, hb = (_Float16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, ha) | ((uint32_t)__builtin_bit_cast(uint16_t, hb) << 16);
}

// bf16 pair (packed in a uint32) -> fp16 pair, exact for normal-range values.
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w) {
  return pack_f16x2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
}

// Stage one tile of gathered K (row-major) and V (transposed, fp16) for both states into LDS.
template <int D>
__device__ __forceinline__ void stage_tile(const AttnArgs& a, AttnSmem<D>& sm, int b, int h,
                                           bool need_old) {
  const int lane = threadIdx.x;
  constexpr int CH = D / 8;                   // 16-byte chunks per row
  const int64_t HD = (int64_t)a.H * D;
  // K: 32 columns x CH chunks
#pragma unroll
  for (int q = lane; q < kBN * CH; q += 64) {
    const int c = q / CH, ch = q % CH;
    const int cid = sm.cid[c], ns = sm.nslot[c];
    uint4 old = make_uint4(0, 0, 0, 0), nw;
    if (cid >= 0)
      old = *reinterpret_cast<const uint4*>(a.k_cache + ((int64_t)b * a.N + cid) * HD + (int64_t)h * D + ch * 8);
    nw = old;
    if (ns >= 0)
      nw = *reinterpret_cast<const uint4*>(a.k_new + ((int64_t)b * a.k + ns) * HD + (int64_t)h * D + ch * 8);
    if (need_old) *reinterpret_cast<uint4*>(&sm.k[0][c][ch * 8]) = old;
    *reinterpret_cast<uint4*>(&sm.k[1][c][ch * 8]) = nw;
  }
  // V: groups of 4 columns x CH chunks, written transposed (dims x columns)
#pragma unroll
  for (int q = lane; q < (kBN / 4) * CH; q += 64) {
    const int cg = q / CH, ch = q % CH;
    uint4 vo[4], vn[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = cg * 4 + u;
      const int cid = sm.cid[c], ns = sm.nslot[c];
      vo[u] = make_uint4(0, 0, 0, 0);
      if (cid >= 0)
        vo[u] = *reinterpret_cast<const uint4*>(a.v_cache + ((int64_t)b * a.N + cid) * HD + (int64_t)h * D + ch * 8);
      vn[u] = vo[u];
      if (ns >= 0)
        vn[u] = *reinterpret_cast<const uint4*>(a.v_new + ((int64_t)b * a.k + ns) * HD + (int64_t)h * D + ch * 8);
    }
#pragma unroll
    for (int which = 0; which < 2; ++which) {
      if (which == 0 && !need_old) continue;
      const uint4* src = which ? vn : vo;
      // element e of chunk: word e/2, half e&1
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        uint32_t hv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t wsel = (e >> 1) == 0 ? src[u].x : (e >> 1) == 1 ? src[u].y : (e >> 1) == 2 ? src[u].z : src[u].w;
          const uint32_t bits = (e & 1) ? (wsel >> 16) : (wsel & 0xFFFFu);
          hv[u] = bits;
        }
        const uint32_t lo = pack_f16x2(bf16_to_f32(hv[0]), bf16_to_f32(hv[1]));
        const uint32_t hi = pack_f16x2(bf16_to_f32(hv[2]), bf16_to_f32(hv[3]));
        *reinterpret_cast<uint2*>(&sm.vt[which][ch * 8 + e][cg * 4]) = make_uint2(lo, hi);
      }
    }
  }
}

template <int D>
__global__ __launch_bounds__(64) void loop_attn_kernel(AttnArgs a) {
  __shared__ AttnSmem<D> sm;
  constexpr int KS = D / 16;    // k-steps of the QK^T contraction
  constexpr int DB = D / 32;    // 32-dim blocks of the output
  const int lane = threadIdx.x;
  const int hw = lane >> 5;     // half-wave
  const int r32 = lane & 31;    // this lane's row within the tile
  const int p0 = blockIdx.x * kBM;
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t HD = (int64_t)a.H * D;

  const int p = p0 + r32;
  const bool row_ok = p < a.k;
  const int row_i = row_ok ? (a.rows ? a.rows[(int64_t)b * a.k + p] : p) : -1;
  const int last_p = min(p0 + kBM, a.k) - 1;
  const int min_row = a.rows ? a.rows[(int64_t)b * a.k + p0] : p0;
  const int max_row = a.rows ? a.rows[(int64_t)b * a.k + last_p] : last_p;

  // Q fragments (B operand of S^T = K Q^T): row r32, dims 16*ks + 8*hw .. +7
  bf16x8 qc[KS], qp[KS];
  {
    const int64_t qoff = ((int64_t)b * a.N + (row_ok ? row_i : 0)) * HD + (int64_t)h * D + hw * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint4 w = row_ok ? *reinterpret_cast<const uint4*>(a.q_cur + qoff + ks * 16) : make_uint4(0, 0, 0, 0);
      qc[ks] = __builtin_bit_cast(bf16x8, w);
      uint4 wp = make_uint4(0, 0, 0, 0);
      if (!a.dense && row_ok) wp = *reinterpret_cast<const uint4*>(a.q_prev + qoff + ks * 16);
      qp[ks] = __builtin_bit_cast(bf16x8, wp);
    }
  }
  float lse2 = 0.0f;
  if (!a.dense && row_ok) lse2 = a.lse_ref[((int64_t)b * a.N + row_i) * a.H + h] * 1.4426950408889634f;

  f32x16 acc_add[DB], acc_sub[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    acc_add[db] = f32x16{};
    acc_sub[db] = f32x16{};
  }
  float run_max = -INFINITY, lsum = 0.0f, msub = 0.0f;

  // phase extents
  const int32_t* colp = a.cols ? a.cols + ((int64_t)b * a.H + h) * a.c_list : nullptr;
  int n_list = 0;
  if (!a.dense && colp && a.c_list > 0) {
    const int lim = max_row - a.window;    // list columns need j + window <= i
    int lo = 0, hi = a.c_list;             // first index with cols[idx] > lim
    while (lo < hi) {
      int mid = (lo + hi) >> 1;
      if (colp[mid] <= lim) lo = mid + 1; else hi = mid;
    }
    n_list = lo;
  }
  int band_lo = 0, band_hi = -1;
  if (a.dense) {
    band_lo = 0;
    band_hi = max_row;
  } else if (a.window > 0) {
    band_lo = max(0, min_row - a.window + 1);
    band_hi = max_row;
  }
  const int n_list_tiles = (n_list + kBN - 1) / kBN;
  const int n_band_tiles = band_hi >= band_lo ? (band_hi - band_lo + 1 + kBN - 1) / kBN : 0;
  const bool need_old = !a.dense;

  for (int tile = 0; tile < n_list_tiles + n_band_tiles; ++tile) {
    const bool in_list = tile < n_list_tiles;
    if (lane < kBN) {
      int cid;
      if (in_list) {
        const int pos = tile * kBN + lane;
        cid = pos < n_list ? colp[pos] : -1;
      } else {
        const int j = band_lo + (tile - n_list_tiles) * kBN + lane;
        cid = j <= band_hi ? j : -1;
      }
      sm.cid[lane] = cid;
      sm.nslot[lane] = (cid >= 0 && a.slot) ? a.slot[(int64_t)b * a.N + cid] : -1;
    }
    __syncthreads();
    stage_tile<D>(a, sm, b, h, need_old);
    __syncthreads();

    // validity of this lane's 16 (column, row) pairs: column 8j + 4hw + i
    bool valid[16];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int cid = sm.cid[8 * j + 4 * hw + i];
        bool v;
        if (in_list) v = cid >= 0 && cid + a.window <= row_i;
        else v = cid >= 0 && cid <= row_i && (a.dense || cid > row_i - a.window);
        valid[4 * j + i] = v;
      }
    }

#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      if (pass == 0 && !need_old) continue;
      const int which = pass;   // 0 = subtract (loop r-1), 1 = add (loop r)
      f32x16 s = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const uint4 kw = *reinterpret_cast<const uint4*>(&sm.k[which][r32][ks * 16 + hw * 8]);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kw),
                                                    which ? qc[ks] : qp[ks], s, 0, 0, 0);
      }
      float pr[16];
      if (which == 0) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          pr[v] = valid[v] ? __builtin_amdgcn_exp2f(s[v] * a.scale_log2 - lse2) : 0.0f;
          msub += pr[v];
        }
      } else {
        float tmax = -INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          s[v] = valid[v] ? s[v] * a.scale_log2 : -INFINITY;
          tmax = fmaxf(tmax, s[v]);
        }
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
        const float new_max = fmaxf(run_max, tmax);
        float alpha = 1.0f;
        if (new_max != -INFINITY) {
          alpha = __builtin_amdgcn_exp2f(run_max - new_max);
#pragma unroll
          for (int v = 0; v < 16; ++v) pr[v] = valid[v] ? __builtin_amdgcn_exp2f(s[v] - new_max) : 0.0f;
        } else {
#pragma unroll
          for (int v = 0; v < 16; ++v) pr[v] = 0.0f;
        }
        run_max = new_max;
        float ts = 0.0f;
#pragma unroll
        for (int v = 0; v < 16; ++v) ts += pr[v];
        lsum = lsum * alpha + ts;
        if (alpha != 1.0f) {
#pragma unroll
          for (int db = 0; db < DB; ++db) acc_add[db] *= alpha;
        }
      }
      // O^T += V^T P^T over two 16-column k-blocks
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const uint32_t b0 = pack_f16x2(pr[8 * kb + 0], pr[8 * kb + 1]);
        const uint32_t b1 = pack_f16x2(pr[8 * kb + 2], pr[8 * kb + 3]);
        const uint32_t b2 = pack_f16x2(pr[8 * kb + 4], pr[8 * kb + 5]);
        const uint32_t b3 = pack_f16x2(pr[8 * kb + 6], pr[8 * kb + 7]);
        const f16x8 pf = __builtin_bit_cast(f16x8, make_uint4(b0, b1, b2, b3));
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const uint2 lo = *reinterpret_cast<const uint2*>(&sm.vt[which][db * 32 + r32][16 * kb + 4 * hw]);
          const uint2 hi = *reinterpret_cast<const uint2*>(&sm.vt[which][db * 32 + r32][16 * kb + 8 + 4 * hw]);
          const f16x8 vf = __builtin_bit_cast(f16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
          if (which) acc_add[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, pf, acc_add[db], 0, 0, 0);
          else acc_sub[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, pf, acc_sub[db], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }

  // the two half-waves hold disjoint columns of the same row
  lsum += __shfl_xor(lsum, 32, 64);
  msub += __shfl_xor(msub, 32, 64);
  if (!row_ok) return;
  const int64_t orow = ((int64_t)b * a.N + row_i) * HD + (int64_t)h * D;
  const int64_t lrow = ((int64_t)b * a.N + row_i) * a.H + h;
  if (a.dense) {
    if (!(lsum > 0.0f)) return;    // unreachable: column 0 is always causal
    const float inv = 1.0f / lsum;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int dim = db * 32 + 8 * j + 4 * hw;
        float4 out = make_float4(acc_add[db][4 * j] * inv, acc_add[db][4 * j + 1] * inv,
                                 acc_add[db][4 * j + 2] * inv, acc_add[db][4 * j + 3] * inv);
        *reinterpret_cast<float4*>(a.o + orow + dim) = out;
      }
    if (hw == 0) a.lse_ref[lrow] = (run_max + log2f(lsum)) * 0.6931471805599453f;
    return;
  }
  if (!(msub > 0.0f) || !(lsum > 0.0f)) return;     // empty column set or vanished mass: unchanged
  const float f = msub / lsum;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int dim = db * 32 + 8 * j + 4 * hw;
      float4 prev = *reinterpret_cast<const float4*>(a.o + orow + dim);
      prev.x = prev.x - acc_sub[db][4 * j + 0] + acc_add[db][4 * j + 0] * f;
      prev.y = prev.y - acc_sub[db][4 * j + 1] + acc_add[db][4 * j + 1] * f;
      prev.z = prev.z - acc_sub[db][4 * j + 2] + acc_add[db][4 * j + 2] * f;
      prev.w = prev.w - acc_sub[db][4 * j + 3] + acc_add[db][4 * j + 3] * f;
      *reinterpret_cast<float4*>(a.o + orow + dim) = prev;
    }
  if (hw == 0) a.lse_ref[lrow] = (run_max + log2f(lsum)) * 0.6931471805599453f - logf(msub);
}

}  // namespace fl

using namespace fl;

extern "C" size_t fl_loop_sparse_attn_ws(int B, int N, int H, int d, int k, int c_list, int window,
                                         int flags) {
  (void)B; (void)N; (void)H; (void)d; (void)k; (void)c_list; (void)window; (void)flags;
  return 0;
}

extern "C" int fl_loop_sparse_attn(const uint16_t* q_cur, const uint16_t* q_prev,
                                   const uint16_t* k_cache, const uint16_t* v_cache,
                                   const uint16_t* k_new, const uint16_t* v_new,
                                   const int32_t* slot, const int32_t* rows, int k,
                                   const int32_t* cols, int c_list, int window, int B, int N, int H,
                                   int d, float sm_scale, int flags, float* lse_ref, float* o,
                                   void* ws, size_t ws_bytes, void* stream) {
  FL_API_BEGIN
  (void)ws;
  const bool dense = (flags & FL_ATTN_DENSE) != 0;
  FL_REQUIRE((flags & ~FL_ATTN_DENSE) == 0, FL_E_UNSUPPORTED, "fl_loop_sparse_attn: unknown flags 0x%x", flags);
  FL_REQUIRE(q_cur && k_cache && v_cache && lse_ref && o, FL_E_NULL,
             "fl_loop_sparse_attn: q_cur, k_cache, v_cache, lse_ref and o are required");
  FL_REQUIRE(B >= 1 && N >= 1 && H >= 1, FL_E_SHAPE, "fl_loop_sparse_attn: need B, N, H >= 1");
  FL_REQUIRE(d == 64 || d == 128, FL_E_SHAPE, "fl_loop_sparse_attn: head dim %d not in {64, 128}", d);
  FL_REQUIRE((int64_t)N * H * d < ((int64_t)1 << 31), FL_E_SHAPE, "fl_loop_sparse_attn: N * H * d too large");
  FL_REQUIRE(sm_scale > 0.0f && std::isfinite(sm_scale), FL_E_RANGE, "fl_loop_sparse_attn: sm_scale must be > 0");
  FL_REQUIRE(ws_bytes >= fl_loop_sparse_attn_ws(B, N, H, d, k, c_list, window, flags), FL_E_WORKSPACE,
             "fl_loop_sparse_attn: workspace too small");
  if (dense) {
    FL_REQUIRE(rows == nullptr && k == N, FL_E_SHAPE, "fl_loop_sparse_attn: DENSE needs rows == NULL and k == N");
  } else {
    FL_REQUIRE(q_prev && k_new && v_new && slot && rows, FL_E_NULL,
               "fl_loop_sparse_attn: q_prev, k_new, v_new, slot and rows are required");
    FL_REQUIRE(k >= 0 && k <= N, FL_E_RANGE, "fl_loop_sparse_attn: k=%d outside [0, N]", k);
    FL_REQUIRE(c_list >= 0 && c_list <= N, FL_E_RANGE, "fl_loop_sparse_attn: c_list=%d outside [0, N]", c_list);
    FL_REQUIRE(c_list == 0 || cols, FL_E_NULL, "fl_loop_sparse_attn: cols is required when c_list > 0");
    FL_REQUIRE(window >= 0, FL_E_RANGE, "fl_loop_sparse_attn: window must be >= 0");
  }
  if (k == 0) return FL_OK;
  AttnArgs a{q_cur, q_prev, k_cache, v_cache, k_new, v_new, slot, dense ? nullptr : rows,
             dense ? nullptr : cols, lse_ref, o, k, dense ? 0 : c_list, dense ? 0 : window, N, H,
             sm_scale * 1.4426950408889634f, dense ? 1 : 0};
  if (dense) { a.slot = nullptr; a.q_prev = nullptr; a.k_new = nullptr; a.v_new = nullptr; }
  dim3 grid((k + kBM - 1) / kBM, H, B);
  hipStream_t st = as_stream(stream);
  if (d == 128) loop_attn_kernel<128><<<grid, 64, 0, st>>>(a);
  else loop_attn_kernel<64><<<grid, 64, 0, st>>>(a);
  return check_launch("loop_attn_kernel");
  FL_API_END
}
