// Radix top-k of one segment by one 1024-thread workgroup, shared by the selection kernels and the
// decode step (Appendix D.1, Eq. 5; Appendix D.2, Eq. 6: the largest keys, ties to the lower position,
// emitted in ascending position order).
//
// Keys are mapped to order-preserving uint32 and held in registers (M per thread).  The k-th largest
// key is found in two stages: an LDS histogram of the top 12 bits and a block scan over its 4096 bins
// give the bin that holds it; the keys of that bin are compacted into LDS and the remaining 20 bits are
// resolved with digit histograms of 8, 8 and 4 bits over that (small) set (bit by bit over the
// registers if the bin overflows the LDS buffer).  The selected positions are then compacted in
// position order with two block scans, which emits them ascending and breaks ties by the lower index.
#pragma once
#include "fl_common.h"

#include <climits>

namespace fl {

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

// One workgroup (kTopkThreads threads) selects the top k of n keys kp[0..n).  Position p has id cp[p]
// (cp != NULL) or id_base + p.  Selected ids are written ascending at op[n_prefix + pos]; ids
// 0..n_prefix-1 are written first (column sinks).  Optional slot map: sp[id] = pos (or -1), sp holding
// slot_n entries.  Only output positions pos in [out_lo, out_hi) are written, at op[n_prefix + pos -
// out_lo] (the sink ids only when out_lo == 0): a workgroup that needs one window of the selection keeps
// it in LDS.  Thread t holds the keys of positions t + 1024 j (coalesced loads; the threshold search does
// not care about order); the ascending output comes from bitmaps of the selected positions.  Ends with
// the ids written by this workgroup's threads (no trailing barrier).
template <int M>
__device__ __forceinline__ void topk_block(const float* __restrict__ kp, int n, int k,
                                           const int32_t* __restrict__ cp, int id_base,
                                           int32_t* __restrict__ op, int n_prefix,
                                           int32_t* __restrict__ sp, int slot_n, int out_lo = 0,
                                           int out_hi = INT_MAX) {
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
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  int32_t* slot = sp;
  if (slot) {
    for (int i = t; i < slot_n; i += kTopkThreads) sp[i] = -1;
  }
  if (out_lo == 0)
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

  // k-th largest key.  (1) The keys' range [lo, hi]: the codes become offsets v = u - lo (order kept), and
  // the first histogram takes the kHistBits bits of v from the highest bit the range needs (shift0 up),
  // so the bins cover the keys' actual range and the bin that holds the k-th largest is small.  With
  // k == n every position is taken and no threshold is needed.
  const bool take_all = k == n;
  uint32_t prefix = 0, mask = 0;
  int krem = take_all ? 0 : k;
  // (the range is taken on every path, so the keys have one form, offsets, in registers: with the raw keys
  // kept for the paths without a search, the 32K-key kernel ran out of registers)
  uint32_t lo = 0xFFFFFFFFu, hi = 0u;
#pragma unroll
  for (int j = 0; j < M; ++j) {
    const bool valid = t + kTopkThreads * j < n;
    lo = valid ? min(lo, u[j]) : lo;
    hi = valid ? max(hi, u[j]) : hi;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    lo = min(lo, (uint32_t)__shfl_xor((int)lo, off, 64));
    hi = max(hi, (uint32_t)__shfl_xor((int)hi, off, 64));
  }
  if (lane == 0) {
    red[wave] = (int)lo;
    red[kTopkWaves + wave] = (int)hi;
  }
  for (int i = t; i < kBins; i += kTopkThreads) hist[i] = 0;
  __syncthreads();
#pragma unroll
  for (int w2 = 0; w2 < kTopkWaves; ++w2) {
    lo = min(lo, (uint32_t)red[w2]);
    hi = max(hi, (uint32_t)red[kTopkWaves + w2]);
  }
  const uint32_t span = hi - lo;
  const int shift0 = span >> kHistBits ? 32 - __builtin_clz(span) - kHistBits : 0;   // span >> shift0 < kBins
#pragma unroll
  for (int j = 0; j < M; ++j) u[j] = (t + kTopkThreads * j < n) ? u[j] - lo : 0u;
  if (k > 0 && !take_all) {                               // uniform
    WaveHist wh;
#pragma unroll
    for (int j = 0; j < M; ++j) wh.add(hist, u[j] >> shift0, t + kTopkThreads * j < n);
    wh.flush(hist);
    __syncthreads();                                      // (also: every wave has read red)
    find_bin(hist, kBins, k, scan_scratch, meta);
    const uint32_t bin = (uint32_t)meta[0];
    const int cnt = meta[2];
    krem = meta[1];
    prefix = bin << shift0;
    mask = shift0 < 32 ? ~0u << shift0 : 0u;
    if (shift0 == 0) {
      // every offset is its own bin: the threshold is known
    } else if (cnt <= kCap) {
      // (2) compact that bin's keys into LDS (any order), then resolve the low shift0 bits with digit
      // histograms of up to 8 bits over them
      int n_in = 0;
#pragma unroll
      for (int j = 0; j < M; ++j) n_in += (t + kTopkThreads * j < n && (u[j] & mask) == prefix) ? 1 : 0;
      int tot;
      int off = block_exclusive_scan(n_in, scan_scratch, &tot);
#pragma unroll
      for (int j = 0; j < M; ++j)
        if (t + kTopkThreads * j < n && (u[j] & mask) == prefix) cbuf[off++] = u[j];
      int shift = shift0;
      while (shift > 0) {                                 // uniform
        const int nb = shift < 8 ? shift : 8;
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
      for (int bit = shift0 - 1; bit >= 0; --bit) {
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
          if (o >= out_lo && o < out_hi) op[n_prefix + o - out_lo] = id;
          if (slot) sp[id] = o;
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
          if (pos >= out_lo && pos < out_hi) op[n_prefix + pos - out_lo] = id;
          if (slot) sp[id] = pos;
        }
        ++pos;
      }
    }
  }
}

}  // namespace fl
