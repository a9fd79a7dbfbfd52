// Token selection (Section 4.1; Appendix D.1, Eq. 5) and column-list selection (Appendix D.2, Eq. 6).
//
// score_rows: one wave per candidate row streams the four bf16 rows (K and V, current and previous)
//   with non-temporal 16-byte loads, forms fp32 differences, accumulates squared norms in fp64,
//   reduces across the wave and writes the fp32 key.  HBM-bound: 4 * D * 2 bytes per candidate.
//   When the budget keeps every candidate (k = n_cand, nested loops with a constant budget), extra
//   workgroups of the same launch write the selection itself: the candidates and their slot map.
// topk_select: one 1024-thread workgroup per segment.  Keys are mapped to order-preserving uint32 and
//   held in registers (M per thread).  The k-th largest key is found in two stages: an LDS histogram
//   of the top 12 bits and a block scan over its 4096 bins give the bin that holds it; the keys of
//   that bin are compacted into LDS and the remaining 20 bits are resolved with digit histograms of
//   8, 8 and 4 bits over that (small) set (bit by bit over the registers if the bin overflows the LDS
//   buffer).  The selected positions are then compacted in candidate order with two block scans, which
//   emits rows ascending and breaks ties by the lower index.
#include "fl_common.h"

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

// ---- block-wide helpers for a 1024-thread workgroup (16 waves) -----------------------------------
constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;

__device__ __forceinline__ int block_sum(int v, int* red /* [2][16] */, int parity) {
  v = wave_sum_i32(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[parity * kTopkWaves + w] = v;
  __syncthreads();
  int total = 0;
#pragma unroll
  for (int i = 0; i < kTopkWaves; ++i) total += red[parity * kTopkWaves + i];
  return total;   // callers alternate parity, so the next write never races this read
}

// Exclusive prefix sum over threads in thread order; returns the prefix and sets *total.
__device__ __forceinline__ int block_exclusive_scan(int v, int* scratch /* [16] */, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  __syncthreads();                                   // previous users of scratch are done
  if (lane == 63) scratch[w] = incl;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < kTopkWaves; ++i) {
    int s = scratch[i];
    before += (i < w) ? s : 0;
    all += s;
  }
  *total = all;
  return before + incl - v;
}

// Histogram of one digit per lane and round, for keys that crowd into few bins: the bin of the wave's
// first key of the first round is counted in a register with ballots (one LDS atomic at the end), the
// other keys add with LDS atomics.  Same-address LDS atomics from many waves serialize; this keeps them
// to one per wave for the crowded bin.
struct WaveHist {
  uint32_t lead = 0;
  int count = 0;
  bool started = false;
  __device__ __forceinline__ void add(int* hist, uint32_t bin, bool want) {
    if (!started) {                                        // uniform
      lead = __builtin_amdgcn_readfirstlane(bin);
      started = true;
    }
    const bool same = want && bin == lead;
    count += (int)__builtin_popcountll(__builtin_amdgcn_ballot_w64(same));
    if (want && !same) atomicAdd(&hist[bin], 1);
  }
  __device__ __forceinline__ void flush(int* hist) {
    if ((threadIdx.x & 63) == 0 && count > 0) atomicAdd(&hist[lead], count);
  }
};

// The bin, scanning bins from the highest, where the running count of keys first reaches krem.
// hist holds nbins counts (nbins <= 4 * kTopkThreads); result in meta[0..2] = (bin, krem left in it,
// its count).  Block-wide; ends with a barrier.
__device__ __forceinline__ void find_bin(const int* hist, int nbins, int krem, int* scratch, int* meta) {
  const int t = threadIdx.x;
  const int per = nbins > kTopkThreads ? nbins / kTopkThreads : 1;   // 4 or 1
  int hb[4] = {0, 0, 0, 0}, local = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int bin = nbins - 1 - per * t - q;
    if (q < per && bin >= 0) {
      hb[q] = hist[bin];
      local += hb[q];
    }
  }
  int total;
  const int above = block_exclusive_scan(local, scratch, &total);
  if (above < krem && above + local >= krem) {
    int acc = above;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (q < per && acc < krem && acc + hb[q] >= krem) {
        meta[0] = nbins - 1 - per * t - q;
        meta[1] = krem - acc;
        meta[2] = hb[q];
      }
      acc += hb[q];
    }
  }
  __syncthreads();
}

__device__ __forceinline__ uint32_t orderable(float f) {
  uint32_t u = __float_as_uint(f + 0.0f);   // -0 and +0 are the same key
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Segment s selects the top k of n keys.  Position p has id cand[p] (cand != NULL) or id_base + p.
// Selected ids are written ascending at out[s * out_stride + n_prefix + pos]; ids 0..n_prefix-1 are
// written first (column sinks).  Optional slot map: slot[s * slot_n + id] = pos (or -1).
// Thread t holds the keys of positions t + 1024 j (coalesced loads; the threshold search does not care
// about order); the ascending output comes from bitmaps of the selected positions.
template <int M>
__global__ __launch_bounds__(kTopkThreads) void topk_select_kernel(
    const float* __restrict__ keys, int64_t key_stride, int n, int k,
    const int32_t* __restrict__ cand, int64_t cand_stride, int id_base,
    int32_t* __restrict__ out, int64_t out_stride, int n_prefix,
    int32_t* __restrict__ slot, int slot_n) {
  constexpr int kHistBits = 12, kBins = 1 << kHistBits;
  static_assert(kBins == 4 * kTopkThreads, "each thread owns four histogram bins");
  constexpr int kCap = M * kTopkThreads < 32768 ? M * kTopkThreads : 32768;
  constexpr int kWords = M * kTopkThreads / 32;            // bitmap words over all positions
  constexpr int kWordsPerThread = (kWords + kTopkThreads - 1) / kTopkThreads;
  static_assert(2 * kWords <= kCap, "the bitmaps reuse the compaction buffer");
  __shared__ int red[2 * kTopkWaves];
  __shared__ int scan_scratch[kTopkWaves];
  __shared__ int hist[kBins];
  __shared__ uint32_t cbuf[kCap];          // keys of the threshold's bin, later the two bitmaps
  __shared__ int meta[3];                  // that bin, keys still to take from it, its size
  const int s = blockIdx.x;
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const float* kp = keys + (int64_t)s * key_stride;
  const int32_t* cp = cand ? cand + (int64_t)s * cand_stride : nullptr;
  int32_t* op = out + (int64_t)s * out_stride;

  if (slot) {
    int32_t* sp = slot + (int64_t)s * slot_n;
    for (int i = t; i < slot_n; i += kTopkThreads) sp[i] = -1;
  }
  for (int i = t; i < n_prefix; i += kTopkThreads) op[i] = i;

  // (buffer loads: out-of-range positions read 0 without a branch, so all M loads are in flight at once;
  // a bounds-checked pointer load puts each one behind its own branch and wait)
  uint32_t u[M];
  {
    const __amdgpu_buffer_rsrc_t kr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(kp), (short)0, n * 4, 0x00020000);
#pragma unroll
    for (int j = 0; j < M; ++j) {
      const int p = t + kTopkThreads * j;
      const float x = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(kr, (uint32_t)p * 4u, 0, 0));
      u[j] = orderable(x) & (0u - (uint32_t)(p < n));    // padding: 0 (as a mask, not a branch)
    }
  }

  // k-th largest key: (1) histogram of the top kHistBits bits and the bin that holds it.  With k == n
  // every position is taken and no threshold is needed.
  const bool take_all = k == n;
  uint32_t prefix = 0, mask = 0;
  int krem = take_all ? 0 : k;
  if (k > 0 && !take_all) {                               // uniform
    for (int i = t; i < kBins; i += kTopkThreads) hist[i] = 0;
    __syncthreads();
    WaveHist wh;
#pragma unroll
    for (int j = 0; j < M; ++j) wh.add(hist, u[j] >> (32 - kHistBits), t + kTopkThreads * j < n);
    wh.flush(hist);
    __syncthreads();
    find_bin(hist, kBins, k, scan_scratch, meta);
    const uint32_t bin = (uint32_t)meta[0];
    const int cnt = meta[2];
    krem = meta[1];
    prefix = bin << (32 - kHistBits);
    mask = ~0u << (32 - kHistBits);
    if (cnt <= kCap) {
      // (2) compact that bin's keys into LDS (any order), then resolve the low 20 bits with digit
      // histograms of 8, 8 and 4 bits over them
      int n_in = 0;
#pragma unroll
      for (int j = 0; j < M; ++j) n_in += (t + kTopkThreads * j < n && (u[j] >> (32 - kHistBits)) == bin) ? 1 : 0;
      int tot;
      int off = block_exclusive_scan(n_in, scan_scratch, &tot);
#pragma unroll
      for (int j = 0; j < M; ++j)
        if (t + kTopkThreads * j < n && (u[j] >> (32 - kHistBits)) == bin) cbuf[off++] = u[j];
      int shift = 32 - kHistBits;
      for (int pass = 0; pass < 3; ++pass) {
        const int nb = pass < 2 ? 8 : 4;
        shift -= nb;
        for (int i = t; i < (1 << nb); i += kTopkThreads) hist[i] = 0;
        __syncthreads();                                  // also orders the compaction writes
        WaveHist dh;
        for (int i0 = 0; i0 < cnt; i0 += kTopkThreads) {
          const int i = i0 + t;
          const uint32_t v = i < cnt ? cbuf[i] : 0u;
          dh.add(hist, (v >> shift) & ((1u << nb) - 1), i < cnt && (v & mask) == prefix);
        }
        dh.flush(hist);
        __syncthreads();
        find_bin(hist, 1 << nb, krem, scan_scratch, meta);
        prefix |= (uint32_t)meta[0] << shift;
        mask |= ((1u << nb) - 1) << shift;
        krem = meta[1];
      }
    } else {
      // (2b) too many keys in one bin for the LDS buffer: resolve the low bits over the registers
      for (int bit = 31 - kHistBits; bit >= 0; --bit) {
        const uint32_t want = prefix | (1u << bit), m2 = mask | (1u << bit);
        int c = 0;
#pragma unroll
        for (int j = 0; j < M; ++j) c += ((t + kTopkThreads * j) < n && (u[j] & m2) == want) ? 1 : 0;
        c = block_sum(c, red, bit & 1);
        if (c >= krem) prefix = want; else krem -= c;
        mask = m2;
      }
    }
  }
  // (3) bitmaps of the positions with a key above the threshold and equal to it (bit p % 32 of word
  // p / 32): positions t + 1024 j of a wave's lanes 0-31 and 32-63 form words 32 j + 2 wave and
  // 32 j + 2 wave + 1, taken by ballot.  The wave gathers its 2 M words per map into lanes (word
  // 2 j + h in lane (2 j + h) % 64 of register (2 j + h) / 64) and stores them without branches.
  uint32_t* bm_gt = cbuf;
  uint32_t* bm_eq = cbuf + kWords;
  constexpr int kRegs = (2 * M + 63) / 64;
  uint32_t gv[kRegs], ev[kRegs];
#pragma unroll
  for (int r = 0; r < kRegs; ++r) gv[r] = ev[r] = 0u;
#pragma unroll
  for (int j = 0; j < M; ++j) {
    const bool valid = k > 0 && t + kTopkThreads * j < n;
    const uint64_t g = __builtin_amdgcn_ballot_w64(valid && (take_all || u[j] > prefix));
    const uint64_t e = __builtin_amdgcn_ballot_w64(valid && !take_all && u[j] == prefix);
    const int r = (2 * j) / 64, l0 = (2 * j) % 64;
    gv[r] = lane == l0 ? (uint32_t)g : lane == l0 + 1 ? (uint32_t)(g >> 32) : gv[r];
    ev[r] = lane == l0 ? (uint32_t)e : lane == l0 + 1 ? (uint32_t)(e >> 32) : ev[r];
  }
  __syncthreads();                                        // cbuf is no longer read
#pragma unroll
  for (int r = 0; r < kRegs; ++r) {
    const int wj = 64 * r + lane;                         // word 2 j + h of this wave
    if (wj < 2 * M) {
      const int wd = 32 * (wj >> 1) + 2 * wave + (wj & 1);
      bm_gt[wd] = gv[r];
      bm_eq[wd] = ev[r];
    }
  }
  __syncthreads();
  // thread t owns words t * kWordsPerThread ..; the equal keys taken are the krem lowest positions
  uint32_t gw[kWordsPerThread], ew[kWordsPerThread];
  int n_eq = 0;
#pragma unroll
  for (int q = 0; q < kWordsPerThread; ++q) {
    const int wd = t * kWordsPerThread + q;
    gw[q] = wd < kWords ? bm_gt[wd] : 0u;
    ew[q] = wd < kWords ? bm_eq[wd] : 0u;
    n_eq += __builtin_popcount(ew[q]);
  }
  int total;
  const int eq_before = block_exclusive_scan(n_eq, scan_scratch, &total);
  int take = krem - eq_before;                          // equal keys this thread still takes
  int n_sel = 0;
#pragma unroll
  for (int q = 0; q < kWordsPerThread; ++q) {
    uint32_t e = ew[q], keep = 0;
    while (e != 0 && take > 0) {
      const uint32_t low = e & (0u - e);
      keep |= low;
      e ^= low;
      --take;
    }
    gw[q] |= keep;
    n_sel += __builtin_popcount(gw[q]);
  }
  int pos = block_exclusive_scan(n_sel, scan_scratch, &total);
  if constexpr (M <= 4) {
    // few keys per thread: record each word's selected bits and first output position, then every thread
    // writes the selected positions among its own (t + 1024 j: coalesced id loads)
    uint32_t* sel_w = cbuf;                               // reuses the bitmaps' space (read above)
    int* pos_w = reinterpret_cast<int*>(cbuf + kWords);
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kWordsPerThread; ++q) {
      const int wd = t * kWordsPerThread + q;
      if (wd < kWords) {
        sel_w[wd] = gw[q];
        pos_w[wd] = pos;
      }
      pos += __builtin_popcount(gw[q]);
    }
    // the -1 fill above is complete before positions are written (same workgroup: a workgroup-scope
    // release suffices; a device-scope fence would also write back the L2)
    if (slot) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __syncthreads();
#pragma unroll
    for (int j = 0; j < M; ++j) {
      const int p = t + kTopkThreads * j;
      if (p >= n) continue;
      const uint32_t sw = sel_w[p >> 5];
      if ((sw >> (p & 31)) & 1u) {
        const int o = pos_w[p >> 5] + __builtin_popcount(sw & ((1u << (p & 31)) - 1u));
        if (o < k) {                // exactly k positions are selected; the bound is a safety net
          const int id = cp ? cp[p] : id_base + p;
          op[n_prefix + o] = id;
          if (slot) slot[(int64_t)s * slot_n + id] = o;
        }
      }
    }
  } else {
    // many keys per thread, few selected per word: thread t writes the selected positions of its own
    // words in order
    if (slot) {   // the -1 fill above is complete before positions are written (workgroup scope suffices)
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      __syncthreads();
    }
#pragma unroll
    for (int q = 0; q < kWordsPerThread; ++q) {
      uint32_t g = gw[q];
      while (g != 0) {
        const int p = 32 * (t * kWordsPerThread + q) + __builtin_ctz(g);
        g &= g - 1;
        if (pos < k) {              // exactly k positions are selected; the bound is a safety net
          const int id = cp ? cp[p] : id_base + p;
          op[n_prefix + pos] = id;
          if (slot) slot[(int64_t)s * slot_n + id] = pos;
        }
        ++pos;
      }
    }
  }
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
