// Mass-corrected sparse attention update (Sections 3.2 and 4.2, Eq. 3; Appendix D.2, Eq. 7) and the
// dense source loop (Eq. 2, causal).
//
// Column sets.  For updated row i the columns are S_i = (list U band(i)) restricted to j <= i; a column
// in both is counted once by giving list columns the condition j + window <= i and band columns
// i - window < j <= i.  The subtract pass needs the loop r-1 state of every column of S_i; the add pass
// needs the loop r state, which differs from the cache only for columns updated in this loop (those in
// the active set).  So every tile is staged from ONE state:
//   phase A  list columns, cache state      subtract: all; add: columns not updated this loop
//   phase B  band columns, cache state      subtract: all; add: columns not updated this loop
//   phase C  updated list columns, new rows add only (compacted per (batch, head) by a prep kernel)
//   phase D  updated band columns, new rows add only (a contiguous range of the active rows)
// The dense loop is phase B alone with an unbounded band.
//
// Work decomposition.  A workgroup of 4 waves takes consecutive updated rows of one (batch, head): 64
// rows in the sparse update, where waves 0-1 run the subtract pass and waves 2-3 the add pass for the
// same two groups of 32 rows, and 128 rows in the dense loop, where every wave runs the softmax pass.
// When the subtract term is the previous loop's stored add term (loops >= 3), reuse_attn_kernel runs the
// add pass alone with one 16-row group per wave.  The row tiles of one (batch, head) map to one XCD so
// its list columns stay in that XCD's L2.
//
// Data movement.  Column tiles of 32 are gathered straight from HBM into a ring of 4 LDS slots with
// buffer_load ... lds (no registers), three tiles ahead of the one being computed; out-of-range offsets
// return zeros, which masks padding without branches.  K rows are stored with their 16-byte chunks
// XOR-swizzled by the row and read as the A operand of S^T = K Q^T (v_mfma_f32_32x32x16_bf16), so each
// lane holds 16 columns of one row.  V rows are converted in place to fp16 (exact for |v| in
// [2^-14, 65504]) by the wave whose DMA wrote them, and read transposed with ds_read_b64_tr_b16 as the A
// operand of O^T += V^T P^T (v_mfma_f32_32x32x16_f16, P in fp16).
//   subtract pass : pp = exp(a - lse_ref), no running max needed (lse_ref bounds the logits);
//   add pass      : online softmax with a running max shared by the two half-waves of a row.
#include "fl_attn_util.h"

#include <algorithm>

#include <type_traits>

namespace fl {

constexpr int kRing = 4;           // LDS ring slots

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
  const int2* rec;           // tile records written by the prep kernel (see attn_prep_kernel)
  const int32_t* n_upd;      // [B, H] updated list entries per (batch, head)
  int off_upd, off_band, off_rows, off_sent;   // record offsets of the regions and the sentinel
  uint32_t rec_bytes;        // bytes of the record array, sentinel included
  float* lse_ref;
  float* o;
  const float* term_prev;    // reuse: [B, k_prev, H, d] add term of the previous loop, by its row position
  const float* mass_prev;    // reuse: [B, k_prev, H] cached mass of the previous loop
  const int32_t* slot_prev;  // reuse: [B, N] position of each row in the previous loop's rows
  float* term_out;           // optional [B, k, H, d]: this loop's add term (the next loop's subtract term)
  float* mass_out;           // optional [B, k, H]: the cached mass m of each updated row
  int k, k_prev, c_list, window, B, N, H;
  float scale_log2;          // sm_scale * log2(e)
  int cache_current;         // reuse: the caches already hold X_hat^(r) of the updated rows (no new rows)
  float pinf;                // +inf
};

// MODE: kDense (loop 1, every row over all causal columns) or kFull (a sparse loop with both passes).
constexpr int kDense = 0, kFull = 1;

template <int D, int MODE>
__global__ __launch_bounds__(256, 2) void loop_attn_kernel(AttnArgs a) {
  constexpr bool DENSE = MODE == kDense;
  constexpr int GROUPS = DENSE ? 4 : 2;
  constexpr int BM = 32 * GROUPS;
  constexpr int KS = D / 16;              // k-steps of QK^T
  constexpr int DB = D / 32;              // 32-dim output blocks
  constexpr int CH = D / 8;               // 16-byte chunks per row
  constexpr int COLS_PER_INST = 64 / CH;  // rows covered by one 1 KB LDS-DMA instruction
  constexpr int INST_PER_TILE = kBN / COLS_PER_INST;
  constexpr int INST_PER_WAVE = INST_PER_TILE / 4;   // per tensor (K and V each)
  __shared__ Slot<D> s0, s1, s2, s3;
  // tables of tile v in entry v % 8, written by two 64-lane stores with no branch:
  //   [0, kBN)        column ids, plain (dense loop, subtract pass; kPad = padding)
  //   [kBN, 2 kBN)    column ids for the add pass, where the columns updated this loop are padding
  //   [2 kBN, 3 kBN)  byte offset of each column's row in its source (kOOB: none)
  //   [3 kBN, 4 kBN)  whether some column of the tile was updated this loop (every entry the same)
  __shared__ uint32_t tab[8][4 * kBN];
  __shared__ float xm[2][64];             // end-of-loop hand-off per group: the subtract pass's mass
  __shared__ int s_meta[2];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int hw = lane >> 5;
  const int r32 = lane & 31;
  const int group = wave % GROUPS;
  const bool add_pass = MODE != kFull || wave >= 2;

  // work item -> (batch*head, row tile); the row tiles of one (batch, head) stay on one XCD
  const int n_rt = (a.k + BM - 1) / BM;
  const int n_bh = a.B * a.H;
  int bh, rt;
  if ((n_bh & 7) == 0) {
    const int g = blockIdx.x & 7, s = blockIdx.x >> 3;
    bh = g + 8 * (s / n_rt);
    rt = n_rt - 1 - (s % n_rt);
  } else {
    bh = blockIdx.x / n_rt;
    rt = n_rt - 1 - (blockIdx.x % n_rt);
  }
  const int b = bh / a.H, h = bh % a.H;
  const int64_t HD = (int64_t)a.H * D;
  const int32_t* rowp = DENSE ? nullptr : a.rows + (int64_t)b * a.k;
  auto row_of = [&](int p) { return DENSE ? p : rowp[p]; };

  const int p0 = rt * BM;
  const int last_p = min(p0 + BM, a.k) - 1;
  const int min_row = row_of(p0), max_row = row_of(last_p);
  const int gp0 = p0 + 32 * group;
  const bool group_has_rows = gp0 < a.k;
  const int gmin = group_has_rows ? row_of(gp0) : 0;
  const int gmax = group_has_rows ? row_of(min(gp0 + 32, a.k) - 1) : -1;
  const int p = gp0 + r32;
  const bool row_ok = p < a.k;
  const int row_i = row_ok ? row_of(p) : -1;

  // query fragments (B operand of S^T = K Q^T): row r32, dims 16*ks + 8*hw .. +7
  bf16x8 qf[KS];
  {
    const uint16_t* qsrc = add_pass ? a.q_cur : a.q_prev;
    const int64_t qoff = ((int64_t)b * a.N + (row_ok ? row_i : 0)) * HD + (int64_t)h * D + hw * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint4 w = row_ok ? *reinterpret_cast<const uint4*>(qsrc + qoff + ks * 16) : make_uint4(0, 0, 0, 0);
      qf[ks] = __builtin_bit_cast(bf16x8, w);
    }
  }
  float lse2 = 0.0f;
  if (!DENSE && !add_pass && row_ok) lse2 = a.lse_ref[((int64_t)b * a.N + row_i) * a.H + h] * 1.4426950408889634f;

  // ---- phase extents (uniform) ----------------------------------------------------------------------
  const int recA = bh * a.c_list;                  // record offsets of the four phases
  const int recC = a.off_upd + bh * a.c_list;
  const int recB = a.off_band + b * a.N;
  const int recD = a.off_rows + b * a.k;
  const int2* descp = DENSE ? nullptr : a.rec + recA;
  const int2* updp = DENSE ? nullptr : a.rec + recC;
  if (tid < 2) {
    int n = 0;
    if (!DENSE && a.c_list > 0) {
      // tid 0: list entries with j + window <= max_row; tid 1: the same among the updated entries
      const int2* lp = tid == 0 ? descp : updp;
      const int len = tid == 0 ? a.c_list : a.n_upd[(int64_t)b * a.H + h];
      const int lim = max_row - a.window;
      int lo = 0, hi = len;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (lp[mid].x <= lim) lo = mid + 1; else hi = mid;
      }
      n = lo;
    }
    s_meta[tid] = n;
  }
  // band extent of the workgroup's rows
  const int bandLo = DENSE ? 0 : (a.window > 0 ? max(0, min_row - a.window + 1) : 0);
  const int bandHi = DENSE ? max_row : (a.window > 0 ? max_row : -1);
  // phase D: the active rows inside [bandLo, bandHi] are a contiguous range of the sorted row list,
  // ending with this tile's last row
  int pa = 0, pb = 0;
  if (!DENSE && a.window > 0) {
    int lo = 0, hi = a.k;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (rowp[mid] < bandLo) lo = mid + 1; else hi = mid;
    }
    pa = lo;
    pb = last_p + 1;
  }
  __syncthreads();
  const int nA = __builtin_amdgcn_readfirstlane(s_meta[0]);   // (uniform: scalar tests and branches below)
  const int nC = __builtin_amdgcn_readfirstlane(s_meta[1]);
  const int tA = (nA + kBN - 1) / kBN;
  const int tB = bandHi >= bandLo ? (bandHi - bandLo + kBN) / kBN : 0;
  const int tC = (nC + kBN - 1) / kBN;
  const int tD = (pb - pa + kBN - 1) / kBN;
  const int n_old = tA + tB;             // tiles staged from the cache state
  const int n_tiles = n_old + tC + tD;
  // band tiles run upward in even row tiles and downward in odd ones, so two neighbouring row tiles
  // (dispatched together on one XCD) read the band columns they share at about the same time
  const bool band_down = (rt & 1) != 0;

  // ---- tile descriptors ----------------------------------------------------------------------------
  // Every tile is described by 32 records (column, aux): list entries (column, slot), band columns
  // (j, slot[j]), updated list entries (column, slot) and updated band rows (rows[p], p), all in one
  // array so that one 8-byte load per lane fetches them for any phase; entries past a phase's end read
  // a sentinel (kPad, -1).  Records are loaded eight tiles ahead and four steps later turned into the LDS
  // tables of entry v % 8: column ids for the masks and the byte offset of the row the DMA reads.
  const int c32 = lane & 31;
  const rsrc_t recR = make_rsrc(DENSE ? (const void*)a.k_cache : (const void*)a.rec, DENSE ? 0u : a.rec_bytes);
  const uint32_t sentinel = (uint32_t)a.off_sent * 8u;
  auto load_desc = [=](int v) -> u32x2 {
    if constexpr (DENSE) return u32x2{0u, 0u};
    const bool inA = v < tA, inB = v < n_old, inC = v < n_old + tC;   // uniform
    const int start = inA ? 0 : inB ? tA : inC ? n_old : n_old + tC;
    const int base = inA ? recA : inB ? recB + bandLo : inC ? recC : recD + pa;
    const int cnt = inA ? nA : inB ? bandHi - bandLo + 1 : inC ? nC : pb - pa;
    const int t = (band_down && inB && !inA) ? tB - 1 - (v - start) : v - start;
    const int i = t * kBN + c32;
    const uint32_t off = lane >= kBN ? kOOB : i < cnt ? (uint32_t)(base + i) * 8u : sentinel;
    return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(recR, off, 0, 0));
  };
  // buffer descriptors of the K/V tensors of this batch element
  const uint32_t rb = (uint32_t)(HD * 2);
  const uint32_t head_off = (uint32_t)(h * D * 2);
  const rsrc_t kcR = make_rsrc(a.k_cache + (int64_t)b * a.N * HD, (uint32_t)a.N * rb);
  const rsrc_t vcR = make_rsrc(a.v_cache + (int64_t)b * a.N * HD, (uint32_t)a.N * rb);

  auto store_desc = [=](int v, u32x2 w) {
    int cid, row;
    bool upd;
    if constexpr (DENSE) {
      cid = v * kBN + c32;                 // the band from column 0
      if (cid > bandHi) cid = kPad;
      row = cid;
      upd = false;
    } else {
      const bool newer = v >= n_old;
      cid = (int)w[0];
      const int aux = (int)w[1];
      upd = !newer && aux >= 0;            // updated this loop but staged from the cache
      row = newer ? aux : cid;
    }
    const bool valid = cid != kPad;
    // lanes 0-31 hold the records; lanes 32-63 take their add-view ids across the half-swap
    const uint32_t cid_add = upd ? (uint32_t)kPad : (uint32_t)cid;
    const auto sw = __builtin_amdgcn_permlane32_swap(cid_add, cid_add, false, false);
    const uint32_t off = valid ? (uint32_t)row * rb + head_off : kOOB;
    const uint64_t any = __builtin_amdgcn_ballot_w64(lane < kBN && valid && upd);
    tab[v & 7][lane] = lane < kBN ? (uint32_t)cid : (uint32_t)sw[0];
    tab[v & 7][2 * kBN + lane] = lane < kBN ? off : (uint32_t)(any != 0);
  };

  // LDS-DMA of tile u into slot sl: each wave issues INST_PER_WAVE K and INST_PER_WAVE V instructions,
  // always (padding and tiles past the end load nothing: their offsets are out of range)
  // DMA plan: every wave issues NI = 2 * INST_PER_WAVE one-kilobyte instructions per tile.  In the
  // sparse update the subtract waves (0-1) load all of V and convert it, the add waves (2-3) load all
  // of K; in the dense loop every wave loads its share of both.  inst_of(t) is the instruction (row
  // block of the tile) of the wave's t-th op, is_v_op(t) whether it targets V.
  constexpr int NI = 2 * INST_PER_WAVE;
  constexpr bool SPLIT_KV = MODE == kFull;
  const bool v_wave = SPLIT_KV && __builtin_amdgcn_readfirstlane(wave) < 2;
  // the sparse update's per-wave source tensors (cache state and new rows)
  const rsrc_t srcC = make_rsrc((v_wave ? a.v_cache : a.k_cache) + (int64_t)b * a.N * HD, (uint32_t)a.N * rb);
  const rsrc_t srcN = make_rsrc(DENSE ? a.k_cache : (v_wave ? a.v_new : a.k_new) + (int64_t)b * a.k * HD,
                                DENSE ? 0u : (uint32_t)a.k * rb);
  const rsrc_t knR = make_rsrc(DENSE ? a.k_cache : a.k_new + (int64_t)b * a.k * HD, DENSE ? 0u : (uint32_t)a.k * rb);
  const rsrc_t vnR = make_rsrc(DENSE ? a.v_cache : a.v_new + (int64_t)b * a.k * HD, DENSE ? 0u : (uint32_t)a.k * rb);
  auto inst_of = [=](int t) { return SPLIT_KV ? (wave & 1) * NI + t : wave * INST_PER_WAVE + (t % INST_PER_WAVE); };
  auto is_v_op = [=](int t) { return SPLIT_KV ? v_wave : t >= INST_PER_WAVE; };
  // source byte offsets of this lane's chunks of tile u (read from the tables ahead of the barrier)
  struct Offs { uint32_t o[NI]; };
  auto tile_offs = [=](int u) {
    Offs r;
#pragma unroll
    for (int t = 0; t < NI; ++t) {
      const int c = inst_of(t) * COLS_PER_INST + lane / CH;
      r.o[t] = tab[u & 7][2 * kBN + c] + (uint32_t)((lane % CH) ^ swz32_f<D>(c)) * 16;   // kOOB + 240: still out of range
    }
    return r;
  };
  // (each offset goes through a local: handing the struct member straight to the builtin makes the
  // host compilation drop the kernel's launch stub)
  auto issue = [=](int u, Slot<D>& sl, const Offs& of) {
    if constexpr (!SPLIT_KV) {
      const bool newer = !DENSE && u >= n_old;   // uniform: one of two scalar branches, same op count
      if (newer) {
#pragma unroll
        for (int t = 0; t < NI; ++t) {
          const int inst = inst_of(t);
          const uint32_t off = of.o[t];
          if (t < INST_PER_WAVE)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(knR, FL_LDS(sl.k + inst * 512), 16, off, 0, 0, kDmaPolicy);
          else
            __builtin_amdgcn_raw_ptr_buffer_load_lds(vnR, FL_LDS(sl.v + inst * 512), 16, off, 0, 0, kDmaPolicy);
        }
      } else {
#pragma unroll
        for (int t = 0; t < NI; ++t) {
          const int inst = inst_of(t);
          const uint32_t off = of.o[t];
          if (t < INST_PER_WAVE)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(kcR, FL_LDS(sl.k + inst * 512), 16, off, 0, 0, kDmaPolicy);
          else
            __builtin_amdgcn_raw_ptr_buffer_load_lds(vcR, FL_LDS(sl.v + inst * 512), 16, off, 0, 0, kDmaPolicy);
        }
      }
    } else {
      uint16_t* dst = v_wave ? sl.v : sl.k;
      if (u >= n_old) {                   // uniform: one of two scalar branches, same op count
#pragma unroll
        for (int t = 0; t < NI; ++t) {
          const uint32_t off = of.o[t];
          __builtin_amdgcn_raw_ptr_buffer_load_lds(srcN, FL_LDS(dst + inst_of(t) * 512), 16, off, 0, 0, kDmaPolicy);
        }
      } else {
#pragma unroll
        for (int t = 0; t < NI; ++t) {
          const uint32_t off = of.o[t];
          __builtin_amdgcn_raw_ptr_buffer_load_lds(srcC, FL_LDS(dst + inst_of(t) * 512), 16, off, 0, 0, kDmaPolicy);
        }
      }
    }
  };

  f32x16 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x16{};
  float run_max = -INFINITY, lsum = 0.0f;   // add pass: running max (log2 units) and row sum
  float msub = 0.0f;                        // subtract pass: mass of the columns seen

  // wave w converts, in place, the V rows its own LDS-DMA wrote (bf16 -> fp16, exact for |v| in
  // [2^-14, 65504]); the barrier that follows publishes them to the other waves
  auto convert_v = [=](Slot<D>& sl) {
    u32x4 w[NI];
#pragma unroll
    for (int t = 0; t < NI; ++t)           // all reads first: one LDS round trip for the batch
      if (is_v_op(t)) w[t] = *reinterpret_cast<const u32x4*>(sl.v + inst_of(t) * 512 + lane * 8);
#pragma unroll
    for (int t = 0; t < NI; ++t) {
      if (!is_v_op(t)) continue;
      u32x4 h;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        h[e] = pack_f16x2(__uint_as_float(w[t][e] << 16), __uint_as_float(w[t][e] & 0xFFFF0000u));
      *reinterpret_cast<u32x4*>(sl.v + inst_of(t) * 512 + lane * 8) = h;
    }
  };

  // LDS read offsets (elements) that depend on the lane; the rest of each read address is a constant.
  // K (A operand of S^T = K Q^T): row r32, data chunk 2ks + hw.  V (transposed reads for O^T += V^T P^T):
  // lane (16g + 4t + q) points at V[col][dim0 + 4q] of column 16kb + 4(g >> 1) + t (and the same + 8),
  // dims 32db + 16(g & 1) + 4q (data chunk 4db + 2(g & 1) + (q >> 1)), so the transpose read hands lane m
  // of the group V[col_t][dim0 + m]; the swizzle of those columns is the same for every kb (voff), and
  // the + 8 columns have their own (voff8).
  int koff[KS], voff[DB], voff8[DB];
  {
    const int g16 = lane >> 4, m16 = lane & 15;
    const int tq = m16 >> 2, q = m16 & 3;
    const int col0 = 4 * (g16 >> 1) + tq;
    const int c_lo = 2 * (g16 & 1) + (q >> 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) koff[ks] = r32 * D + ((2 * ks + hw) ^ swz32_f<D>(r32)) * 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      voff[db] = col0 * D + ((4 * db + c_lo) ^ swz32_f<D>(col0)) * 8 + 4 * (q & 1);
      voff8[db] = (col0 + 8) * D + ((4 * db + c_lo) ^ swz32_f<D>(col0 + 8)) * 8 + 4 * (q & 1);
    }
  }

  // first and last column id of tile u and whether it holds an updated column (uniform; read ahead of
  // the barrier, the entries were written four steps earlier)
  struct TileHead { int c0, clast, any; };
  auto tile_head = [=](int u) {
    return TileHead{__builtin_amdgcn_readfirstlane((int)tab[u & 7][0]),
                    __builtin_amdgcn_readfirstlane((int)tab[u & 7][kBN - 1]),
                    __builtin_amdgcn_readfirstlane((int)tab[u & 7][3 * kBN])};
  };

  auto compute = [=, &acc, &run_max, &lsum, &msub](int u, const Slot<D>& sl, const TileHead& th) {
    const int ri = u & 7;
    const bool newer = u >= n_old;
    const bool is_list = u < tA || (newer && u < n_old + tC);
    if (newer && !add_pass) return;
    // does any row of this wave's group see any column of this tile, and do all rows see all of it?
    // (column ids ascend within a tile and padding, kPad, sits at the end)
    const int c0 = th.c0;
    const int clast = th.clast;
    bool active, full;
    if (is_list) {
      active = group_has_rows && c0 <= gmax - a.window;
      full = clast <= gmin - a.window;
    } else {
      const int t_hi = clast != kPad ? clast : bandHi;
      active = group_has_rows && c0 <= gmax && (DENSE || t_hi > gmin - a.window);
      full = clast <= gmin && (DENSE || c0 > gmax - a.window);
    }
    if (!active) return;
    if (!DENSE && add_pass && !newer && th.any) full = false;   // updated columns drop out
    // S^T = K Q^T: lane holds columns 8j + 4hw + i of row r32
    f32x16 s = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const u32x4 kw = *reinterpret_cast<const u32x4*>(&sl.k[koff[ks]]);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kw), qf[ks], s, 0, 0, 0);
    }
    // masks, softmax and O^T += V^T P^T over the lane's 16 elements, fp16 operands
    constexpr int NE = 16;
    if (!full) {
      // column masks: list columns need j + window <= i, band columns i - window < j <= i (any j <= i in
      // the dense loop); padding and, for the add pass, the columns updated this loop carry kPad
      const int view = (!DENSE && add_pass) ? 1 : 0;
      int cc[16];
#pragma unroll
      for (int j = 0; j < NE / 4; ++j) {
        const int4 c4 = *reinterpret_cast<const int4*>(&tab[ri][kBN * view + 8 * j + 4 * hw]);
        cc[4 * j] = c4.x; cc[4 * j + 1] = c4.y; cc[4 * j + 2] = c4.z; cc[4 * j + 3] = c4.w;
      }
      if (is_list) {
        const int lim = row_i - a.window;
#pragma unroll
        for (int v = 0; v < NE; ++v) s[v] = cc[v] <= lim ? s[v] : -INFINITY;
      } else if (DENSE) {
#pragma unroll
        for (int v = 0; v < NE; ++v) s[v] = cc[v] <= row_i ? s[v] : -INFINITY;
      } else {
        const uint32_t w = (uint32_t)a.window;
#pragma unroll
        for (int v = 0; v < NE; ++v) s[v] = (uint32_t)row_i - (uint32_t)cc[v] < w ? s[v] : -INFINITY;
      }
    }
    float pr[16];
    if (!add_pass) {
#pragma unroll
      for (int v = 0; v < NE; ++v) {
        pr[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], a.scale_log2, -lse2));   // masked: exp2(-inf) = 0
        msub += pr[v];
      }
    } else {
      // online softmax with a lazily raised reference: the reference (run_max, log2 units) only moves
      // when a score exceeds it by more than 8, so probabilities stay <= 256 and the accumulators are
      // rescaled rarely; the final normaliser uses the same reference
      float tmax = s[0];
#pragma unroll
      for (int v = 1; v < NE; ++v) tmax = fmaxf(tmax, s[v]);
      tmax = xor32_max(tmax) * a.scale_log2;
      const bool raise = tmax > run_max + 8.0f;          // false while both are -inf
      if (__builtin_amdgcn_ballot_w64(raise) != 0) {      // uniform: rescale the rows that need it
        const float nm = raise ? tmax : run_max;
        const float alpha = raise ? __builtin_amdgcn_exp2f(run_max - nm) : 1.0f;   // exp2(-inf) = 0
        lsum *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) acc[db] *= alpha;
        run_max = nm;
      }
      const float ref = run_max == -INFINITY ? 0.0f : run_max;
      float ts = 0.0f;
#pragma unroll
      for (int v = 0; v < NE; ++v) {
        pr[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[v], a.scale_log2, -ref));
        ts += pr[v];
      }
      lsum += ts;
    }
#pragma unroll
    for (int kb = 0; kb < NE / 8; ++kb) {
      const u32x4 pw = {pack_f16x2(pr[8 * kb + 0], pr[8 * kb + 1]), pack_f16x2(pr[8 * kb + 2], pr[8 * kb + 3]),
                        pack_f16x2(pr[8 * kb + 4], pr[8 * kb + 5]), pack_f16x2(pr[8 * kb + 6], pr[8 * kb + 7])};
      const f16x8 pf = __builtin_bit_cast(f16x8, pw);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const i16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(FL_LDS4(&sl.v[voff[db] + 16 * kb * D]));
        const i16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(FL_LDS4(&sl.v[voff8[db] + 16 * kb * D]));
        const i16x8 v8 = __builtin_shufflevector(va, vb, 0, 1, 2, 3, 4, 5, 6, 7);
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, v8), pf, acc[db], 0, 0, 0);
      }
    }
  };

  // ---- pipeline --------------------------------------------------------------------------------------
  // step s: read the table entries of tiles s+3 and s; wait for tile s; convert this wave's V rows of
  // it; finalize the records of tile s+4; barrier; load the records of tile s+8; LDS-DMA tile s+3 into
  // the slot tile s-1 used; compute tile s.  Every step issues the same number of VMEM ops (one record
  // load in the sparse update and 2 * INST_PER_WAVE DMA), so "tile s has landed" is exactly
  // vmcnt(2 * OPS_PER_STEP) on every path.
  // Every wave loads the records (equal op counts keep every wait exact); one wave writes the tables:
  // an add wave when the subtract waves convert all of V.
  const bool rec_wave = __builtin_amdgcn_readfirstlane(wave) == (SPLIT_KV ? 2 : 0);
  constexpr int OPS_PER_STEP = (DENSE ? 0 : 1) + NI;
  // Records are loaded four steps before they are turned into tables (step s loads tile s + 8 and
  // describes tile s + 4), so the wave that writes the tables never waits for them: a record load is
  // always older than the tile load the step waits for.
  u32x2 dA, dB, dC, dD;                   // records in flight, by tile mod 4
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const u32x2 r = load_desc(v);
    if (rec_wave) store_desc(v, r);
  }
  FL_WAIT_VM(0);                          // query fragments have arrived
  lds_barrier();
  // the scheduling barriers keep this order, which the wait counts of the first steps assume
  dA = load_desc(4);                      // as step -4
  __builtin_amdgcn_sched_barrier(0);
  dB = load_desc(5);                      // as step -3
  __builtin_amdgcn_sched_barrier(0);
  issue(0, s0, tile_offs(0));
  __builtin_amdgcn_sched_barrier(0);
  dC = load_desc(6);                      // as step -2
  __builtin_amdgcn_sched_barrier(0);
  issue(1, s1, tile_offs(1));
  __builtin_amdgcn_sched_barrier(0);
  dD = load_desc(7);                      // as step -1
  __builtin_amdgcn_sched_barrier(0);
  issue(2, s2, tile_offs(2));

  auto step = [&](int u, Slot<D>& cur, Slot<D>& nxt, u32x2& w) {
    const Offs of = tile_offs(u + 3);     // tables of tiles u+3 and u were published by earlier barriers
    const TileHead th = tile_head(u);
    FL_WAIT_VM(2 * OPS_PER_STEP);
    convert_v(cur);
    if (rec_wave) store_desc(u + 4, w);
    lds_barrier();
    w = load_desc(u + 8);
    __builtin_amdgcn_sched_barrier(0);    // keep the record load ahead of the DMA (the waits count on it)
    issue(u + 3, nxt, of);
    if (u < n_tiles) compute(u, cur, th);
  };
  const int n_steps = (n_tiles + kRing - 1) / kRing * kRing;
  for (int u = 0; u < n_steps; u += kRing) {
    step(u, s0, s3, dA);
    step(u + 1, s1, s0, dB);
    step(u + 2, s2, s1, dC);
    step(u + 3, s3, s2, dD);
  }
  FL_WAIT_VM(0);
  lds_barrier();

  // the two half-waves hold disjoint columns of the same row
  lsum = xor32_add(lsum);
  msub = xor32_add(msub);
  // hand-off through the idle ring: group g uses slot g (D * 128 bytes >= 32 rows x D floats); the
  // subtract waves hand their term and mass to the add waves of the same rows
  float4* xacc = reinterpret_cast<float4*>(group == 0 ? &s0 : &s1);
  if constexpr (!DENSE) {
    if (!add_pass) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          xacc[(db * 4 + j) * 64 + lane] =
              make_float4(acc[db][4 * j], acc[db][4 * j + 1], acc[db][4 * j + 2], acc[db][4 * j + 3]);
      xm[group][lane] = msub;
    }
    lds_barrier();
    if (!add_pass) return;
    msub = xm[group][lane];
  }
  if (!row_ok) return;
  const int64_t orow = ((int64_t)b * a.N + row_i) * HD + (int64_t)h * D;
  const int64_t lrow = ((int64_t)b * a.N + row_i) * a.H + h;
  if constexpr (DENSE) {
    if (!(lsum > 0.0f)) return;    // unreachable: column 0 is always causal
    const float inv = 1.0f / lsum;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int dim = db * 32 + 8 * j + 4 * hw;
        float4 out = make_float4(acc[db][4 * j] * inv, acc[db][4 * j + 1] * inv,
                                 acc[db][4 * j + 2] * inv, acc[db][4 * j + 3] * inv);
        *reinterpret_cast<float4*>(a.o + orow + dim) = out;
      }
    if (hw == 0) a.lse_ref[lrow] = (run_max + log2f(lsum)) * 0.6931471805599453f;
  } else {
    const int64_t trow = ((int64_t)b * a.k + p) * a.H + h;
    const bool keep = a.term_out != nullptr;
    if (!(msub > 0.0f) || !(lsum > 0.0f)) {     // empty column set or vanished mass: unchanged
      if (keep) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            *reinterpret_cast<float4*>(a.term_out + trow * D + db * 32 + 8 * j + 4 * hw) = make_float4(0, 0, 0, 0);
        if (hw == 0) a.mass_out[trow] = 0.0f;
      }
      return;
    }
    const float f = msub / lsum;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int dim = db * 32 + 8 * j + 4 * hw;
        const float4 sub = xacc[(db * 4 + j) * 64 + lane];
        const float4 add = make_float4(acc[db][4 * j + 0] * f, acc[db][4 * j + 1] * f,
                                       acc[db][4 * j + 2] * f, acc[db][4 * j + 3] * f);
        float4 prev = *reinterpret_cast<const float4*>(a.o + orow + dim);
        prev.x = prev.x - sub.x + add.x;
        prev.y = prev.y - sub.y + add.y;
        prev.z = prev.z - sub.z + add.z;
        prev.w = prev.w - sub.w + add.w;
        *reinterpret_cast<float4*>(a.o + orow + dim) = prev;
        if (keep) *reinterpret_cast<float4*>(a.term_out + trow * D + dim) = add;
      }
    if (hw == 0) {
      a.lse_ref[lrow] = (run_max + log2f(lsum)) * 0.6931471805599453f - logf(msub);
      if (keep) a.mass_out[trow] = msub;
    }
  }
}

// ---- sparse update with the previous loop's add term as the subtract term (loops >= 3) -----------------
// Only the add pass remains.  A workgroup of 4 waves takes 64 consecutive updated rows of one (batch,
// head) and wave w owns rows 16w .. 16w+15, so every wave does the same kind of work and a wave's band is
// that of 16 rows (the 32-row groups of loop_attn_kernel would need two waves per group here and compute
// S twice).  The tiles, records and LDS pipeline are those of loop_attn_kernel.  The contractions use
// v_mfma_f32_16x16x32: S^T = K Q^T per 16-column block leaves lane (j, g) = (lane % 16,
// lane / 16) with columns 16c + 4g .. +3 of row j, which is exactly the B-operand layout of
// O^T += V^T P^T when the k order of a 32-column tile is (4g .. 4g+3, 16+4g .. 16+4g+3) for lane group
// g; the transposed V reads follow that order.  The accumulators of a lane belong to the same row j,
// so the softmax state never leaves the lane (row reductions are two cross-row swaps).  V stays bf16 as
// the LDS-DMA wrote it (no conversion step in the pipeline): P goes in as two bf16 parts, hi = bf16(p)
// and lo = bf16(p - hi), so p.v takes two bf16 MFMAs and P keeps about 16 significant bits.
typedef float f32x4 __attribute__((ext_vector_type(4)));


// CUR: the caches already hold this loop's rows (no new-row tiles and no updated columns), so tiles are
// described straight from the column list and the band range, without the prep kernel's records.
template <int D, bool CUR>
__global__ __launch_bounds__(256, 2) void reuse_attn_kernel(AttnArgs a) {
  constexpr int BM = 64;                  // rows per workgroup (4 waves x 16)
  constexpr int KS = D / 32;              // k-steps of QK^T (32 dims each)
  constexpr int DB = D / 16;              // 16-dim output blocks
  constexpr int CH = D / 8;               // 16-byte chunks per row
  constexpr int COLS_PER_INST = 64 / CH;  // rows covered by one 1 KB LDS-DMA instruction
  constexpr int INST_PER_TILE = kBN / COLS_PER_INST;
  constexpr int INST_PER_WAVE = INST_PER_TILE / 4;   // per tensor (K and V each)
  constexpr int NI = 2 * INST_PER_WAVE;
  __shared__ Slot<D> s0, s1, s2, s3;
  // tables of tile v in entry v % 8: [0, kBN) column ids for the add pass (kPad = padding; in phases A/B
  // the columns updated this loop are padding too), [kBN, 2 kBN) byte offset of each column's row in its
  // source (kOOB: none), so with current caches one 64-lane LDS write stores both halves
  __shared__ uint32_t tab[8][2 * kBN];
  __shared__ int thd[8][4];               // tile v: first and last column id, any column updated
  __shared__ int s_meta[2];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j16 = lane & 15, g4 = lane >> 4;

  // work item -> (batch*head, row tile); the row tiles of one (batch, head) stay on one XCD
  const int n_rt = (a.k + BM - 1) / BM;
  const int n_bh = a.B * a.H;
  int bh, rt;
  if ((n_bh & 7) == 0) {
    const int g = blockIdx.x & 7, s = blockIdx.x >> 3;
    bh = g + 8 * (s / n_rt);
    rt = n_rt - 1 - (s % n_rt);
  } else {
    bh = blockIdx.x / n_rt;
    rt = n_rt - 1 - (blockIdx.x % n_rt);
  }
  const int b = bh / a.H, h = bh % a.H;
  const int64_t HD = (int64_t)a.H * D;
  const int32_t* rowp = a.rows + (int64_t)b * a.k;

  const int p0 = rt * BM;
  const int last_p = min(p0 + BM, a.k) - 1;
  const int min_row = rowp[p0], max_row = rowp[last_p];
  const int gp0 = p0 + 16 * wave;
  const bool group_has_rows = gp0 < a.k;
  const int gmin = group_has_rows ? rowp[gp0] : 0;
  const int gmax = group_has_rows ? rowp[min(gp0 + 16, a.k) - 1] : -1;
  const int p = gp0 + j16;
  const bool row_ok = p < a.k;
  const int row_i = row_ok ? rowp[p] : -1;

  // query fragments (B operand of S^T = K Q^T): row j16, dims 32 ks + 8 g4 .. +7
  bf16x8 qa[KS];
  {
    const int64_t qoff = ((int64_t)b * a.N + (row_ok ? row_i : 0)) * HD + (int64_t)h * D + g4 * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint4 w = row_ok ? *reinterpret_cast<const uint4*>(a.q_cur + qoff + ks * 32) : make_uint4(0, 0, 0, 0);
      qa[ks] = __builtin_bit_cast(bf16x8, w);
    }
  }

  // ---- phase extents (uniform) ----------------------------------------------------------------------
  const int recA = bh * a.c_list;
  const int recC = a.off_upd + bh * a.c_list;
  const int recB = a.off_band + b * a.N;
  const int recD = a.off_rows + b * a.k;
  const int2* descp = CUR ? nullptr : a.rec + recA;
  const int2* updp = CUR ? nullptr : a.rec + recC;
  if (tid < 2) {
    int n = 0;
    if (a.c_list > 0 && !(CUR && tid == 1)) {
      // tid 0: list entries with j + window <= max_row; tid 1: the same among the updated entries
      const int lim = max_row - a.window;
      int lo = 0, hi = tid == 0 ? a.c_list : a.n_upd[(int64_t)b * a.H + h];
      if constexpr (CUR) {
        const int32_t* cp = a.cols + (int64_t)bh * a.c_list;
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (cp[mid] <= lim) lo = mid + 1; else hi = mid;
        }
      } else {
        const int2* lp = tid == 0 ? descp : updp;
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (lp[mid].x <= lim) lo = mid + 1; else hi = mid;
        }
      }
      n = lo;
    }
    s_meta[tid] = n;                      // (current caches: no new-row tiles)
  }
  const int bandLo = a.window > 0 ? max(0, min_row - a.window + 1) : 0;
  const int bandHi = a.window > 0 ? max_row : -1;
  int pa = 0, pb = 0;
  if (a.window > 0) {
    int lo = 0, hi = a.k;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (rowp[mid] < bandLo) lo = mid + 1; else hi = mid;
    }
    pa = lo;
    pb = CUR ? lo : last_p + 1;
  }
  __syncthreads();
  const int nA = __builtin_amdgcn_readfirstlane(s_meta[0]);   // (uniform: scalar tests and branches below)
  const int nC = __builtin_amdgcn_readfirstlane(s_meta[1]);
  const int tA = (nA + kBN - 1) / kBN;
  const int tB = bandHi >= bandLo ? (bandHi - bandLo + kBN) / kBN : 0;
  const int tC = (nC + kBN - 1) / kBN;
  const int tD = (pb - pa + kBN - 1) / kBN;
  const int n_old = tA + tB;
  const int n_tiles = n_old + tC + tD;
  const bool band_down = (rt & 1) != 0;   // band tile order as in loop_attn_kernel

  // ---- tile descriptors (records as in the four-phase layout; see attn_prep_kernel) -----------------
  const int c32 = lane & 31;
  const rsrc_t recR = make_rsrc(a.rec, a.rec_bytes);
  const uint32_t sentinel = (uint32_t)a.off_sent * 8u;
  // CUR: entry i of tile v is list entry i of (b, h) or band column bandLo + i (kPad past the end); the
  // list entry is loaded here and the id formed when the tile is described, so the load stays in flight
  const rsrc_t colR = make_rsrc(a.cols, CUR ? (uint32_t)a.B * a.H * a.c_list * 4u : 0u);
  auto cur_entry = [=](int v, int& i, bool& list, bool& ok) {
    list = v < tA;
    const int t = list ? v : band_down ? tB - 1 - (v - tA) : v - tA;
    i = t * kBN + c32;
    ok = lane < kBN && v < n_old && i < (list ? nA : bandHi - bandLo + 1);
  };
  auto load_desc = [=](int v) -> u32x2 {
    if constexpr (CUR) {
      int i;
      bool list, ok;
      cur_entry(v, i, list, ok);
      const uint32_t off = ok && list ? (uint32_t)(recA + i) * 4u : kOOB;
      return u32x2{(uint32_t)__builtin_amdgcn_raw_buffer_load_b32(colR, off, 0, 0), 0u};
    }
    const bool inA = v < tA, inB = v < n_old, inC = v < n_old + tC;   // uniform
    const int start = inA ? 0 : inB ? tA : inC ? n_old : n_old + tC;
    const int base = inA ? recA : inB ? recB + bandLo : inC ? recC : recD + pa;
    const int cnt = inA ? nA : inB ? bandHi - bandLo + 1 : inC ? nC : pb - pa;
    const int t = (band_down && inB && !inA) ? tB - 1 - (v - start) : v - start;
    const int i = t * kBN + c32;
    const uint32_t off = lane >= kBN ? kOOB : i < cnt ? (uint32_t)(base + i) * 8u : sentinel;
    return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(recR, off, 0, 0));
  };
  const uint32_t rb = (uint32_t)(HD * 2);
  const uint32_t head_off = (uint32_t)(h * D * 2);
  const rsrc_t kcR = make_rsrc(a.k_cache + (int64_t)b * a.N * HD, (uint32_t)a.N * rb);
  const rsrc_t vcR = make_rsrc(a.v_cache + (int64_t)b * a.N * HD, (uint32_t)a.N * rb);
  // (with current caches there are no new rows: an empty range makes every access to them read zero)
  const uint32_t new_bytes = CUR ? 0u : (uint32_t)a.k * rb;
  const rsrc_t knR = make_rsrc(CUR ? a.k_cache : a.k_new + (int64_t)b * a.k * HD, new_bytes);
  const rsrc_t vnR = make_rsrc(CUR ? a.v_cache : a.v_new + (int64_t)b * a.k * HD, new_bytes);

  auto store_desc = [=](int v, u32x2 w) {
    if constexpr (CUR) {
      // lanes 0-31 form the column ids and offsets; lanes 32-63 take the offsets across the half-swap and
      // store them beside the ids, in one write with no branch (the tile's head comes from the ids)
      int i;
      bool list, ok;
      cur_entry(v, i, list, ok);
      const int cid = !ok ? kPad : list ? (int)w[0] : bandLo + i;
      const uint32_t off = ok ? (uint32_t)cid * rb + head_off : kOOB;
      const auto sw = __builtin_amdgcn_permlane32_swap(off, off, false, false);
      tab[v & 7][lane] = lane < kBN ? (uint32_t)cid : (uint32_t)sw[0];
      return;
    }
    const bool newer = v >= n_old;
    const int cid = (int)w[0];
    const int aux = (int)w[1];
    const bool upd = !newer && aux >= 0;  // updated this loop, staged from the cache
    const int row = newer ? aux : cid;
    const bool valid = cid != kPad;
    if (lane < kBN) {
      tab[v & 7][c32] = (uint32_t)(upd ? kPad : cid);
      if (c32 == 0) thd[v & 7][0] = cid;
      if (c32 == kBN - 1) thd[v & 7][1] = cid;
      tab[v & 7][kBN + c32] = valid ? (uint32_t)row * rb + head_off : kOOB;
    }
    const uint64_t any = __builtin_amdgcn_ballot_w64(lane < kBN && valid && upd);
    if (lane == 0) thd[v & 7][2] = any != 0;
  };

  // LDS-DMA plan: every wave issues INST_PER_WAVE K and INST_PER_WAVE V one-kilobyte instructions per
  // tile (row block inst_of(t) of the tile), always; padding and tiles past the end load nothing
  auto inst_of = [=](int t) { return wave * INST_PER_WAVE + (t % INST_PER_WAVE); };
  struct Offs { uint32_t o[NI]; };
  auto tile_offs = [=](int u) {
    Offs r;
#pragma unroll
    for (int t = 0; t < NI; ++t) {
      const int c = inst_of(t) * COLS_PER_INST + lane / CH;
      r.o[t] = tab[u & 7][kBN + c] + (uint32_t)((lane % CH) ^ swz16_f<D>(c)) * 16;   // kOOB + 240: still out of range
    }
    return r;
  };
  // (each offset goes through a local: handing the struct member straight to the builtin makes the
  // host compilation drop the kernel's launch stub)
  auto issue = [=](int u, Slot<D>& sl, const Offs& of) {
    if (u >= n_old) {                     // uniform: one of two scalar branches, same op count
#pragma unroll
      for (int t = 0; t < NI; ++t) {
        const int inst = inst_of(t);
        const uint32_t off = of.o[t];
        if (t < INST_PER_WAVE)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(knR, FL_LDS(sl.k + inst * 512), 16, off, 0, 0, kDmaPolicy);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(vnR, FL_LDS(sl.v + inst * 512), 16, off, 0, 0, kDmaPolicy);
      }
    } else {
#pragma unroll
      for (int t = 0; t < NI; ++t) {
        const int inst = inst_of(t);
        const uint32_t off = of.o[t];
        if (t < INST_PER_WAVE)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(kcR, FL_LDS(sl.k + inst * 512), 16, off, 0, 0, kDmaPolicy);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(vcR, FL_LDS(sl.v + inst * 512), 16, off, 0, 0, kDmaPolicy);
      }
    }
  };
  // LDS read offsets (elements) that depend on the lane.  K (A operand): row j16 (+16 for the second
  // column block), data chunk 4 ks + g4.  V (transposed reads): lane (g4, t, q) points at dims
  // 16 db + 4q of column 4 g4 + t (+16 for the second half of the k order), data chunk 2 db + (q >> 1).
  int koff[KS], voff[DB];
  {
    const int t4 = j16 >> 2, q = lane & 3;
    const int colv = 4 * g4 + t4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) koff[ks] = j16 * D + ((4 * ks + g4) ^ swz16_f<D>(j16)) * 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) voff[db] = colv * D + ((2 * db + (q >> 1)) ^ swz16_f<D>(colv)) * 8 + 4 * (q & 1);
  }

  f32x4 acc[DB];                          // add term, O^T blocks
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x4{};
  float run_max = -INFINITY, lsum = 0.0f;   // add pass: running reference (log2 units) and row sum

  struct TileHead { int c0, clast, any; };
  auto tile_head = [=](int u) {
    if constexpr (CUR)
      return TileHead{__builtin_amdgcn_readfirstlane((int)tab[u & 7][0]),
                      __builtin_amdgcn_readfirstlane((int)tab[u & 7][kBN - 1]), 0};
    return TileHead{__builtin_amdgcn_readfirstlane(thd[u & 7][0]), __builtin_amdgcn_readfirstlane(thd[u & 7][1]),
                    __builtin_amdgcn_readfirstlane(thd[u & 7][2])};
  };

  // column mask of the lane's 8 entries (ids cc, columns 16c + 4 g4 + v): list columns need
  // j + window <= i, band columns i - window < j <= i; padding and the columns updated this loop (in the
  // cache tiles) carry kPad
  auto apply_mask = [=](f32x4 (&s)[2], const int4 (&cc)[2], bool is_list) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int ci[4] = {cc[c].x, cc[c].y, cc[c].z, cc[c].w};
      if (is_list) {
        const int lim = row_i - a.window;
#pragma unroll
        for (int v = 0; v < 4; ++v) s[c][v] = ci[v] <= lim ? s[c][v] : -INFINITY;
      } else {
        const uint32_t w = (uint32_t)a.window;
#pragma unroll
        for (int v = 0; v < 4; ++v) s[c][v] = (uint32_t)row_i - (uint32_t)ci[v] < w ? s[c][v] : -INFINITY;
      }
    }
  };

  auto compute = [=, &acc, &run_max, &lsum](int u, const Slot<D>& sl, const TileHead& th) {
    const int ri = u & 7;
    const bool newer = u >= n_old;
    const bool is_list = u < tA || (newer && u < n_old + tC);
    // does any row of this wave's group see any column of this tile, and do all rows see all of it?
    // (column ids ascend within a tile and padding, kPad, sits at the end)
    const int c0 = th.c0, clast = th.clast;
    bool active, full;
    if (is_list) {
      active = group_has_rows && c0 <= gmax - a.window;
      full = clast <= gmin - a.window;
    } else {
      const int t_hi = clast != kPad ? clast : bandHi;
      active = group_has_rows && c0 <= gmax && t_hi > gmin - a.window;
      full = clast <= gmin && c0 > gmax - a.window;
    }
    if (!active) return;
    if (!newer && th.any) full = false;    // updated columns drop out of the cache tiles
    // every LDS read of the tile first, unconditionally (column ids, K and V fragments): a read under a
    // branch can lose the information that tells it apart from the pending LDS-DMA writes
    int4 ca_[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) ca_[c] = *reinterpret_cast<const int4*>(&tab[ri][16 * c + 4 * g4]);
    u32x4 kw[KS][2];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        kw[ks][c] = *reinterpret_cast<const u32x4*>(&sl.k[koff[ks] + 16 * c * D]);
    i16x4 vr[DB][2];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int o = voff[db];
      vr[db][0] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(FL_LDS4(&sl.v[o]));
      vr[db][1] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(FL_LDS4(&sl.v[o + 16 * D]));
    }
    // S^T = K Q^T per 16-column block c: lane holds columns 16c + 4 g4 + v of row j16
    f32x4 sa[2] = {f32x4{}, f32x4{}};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        sa[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kw[ks][c]), qa[ks], sa[c], 0, 0, 0);
    // online softmax with a lazily raised reference (it moves only when a score exceeds it by more than 8
    // in log2 units, so probabilities stay <= 256 and rescaling is rare)
    if (!full) apply_mask(sa, ca_, is_list);
    float tmax = fmaxf(fmaxf(fmaxf(sa[0][0], sa[0][1]), fmaxf(sa[0][2], sa[0][3])),
                       fmaxf(fmaxf(sa[1][0], sa[1][1]), fmaxf(sa[1][2], sa[1][3])));
    tmax = row4_max(tmax) * a.scale_log2;
    const bool raise = tmax > run_max + 8.0f;            // false while both are -inf
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {        // uniform: rescale the rows that need it
      const float nm = raise ? tmax : run_max;
      const float alpha = raise ? __builtin_amdgcn_exp2f(run_max - nm) : 1.0f;   // exp2(-inf) = 0
      lsum *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) acc[db] *= alpha;
      run_max = nm;
    }
    const float ref = run_max == -INFINITY ? 0.0f : run_max;
    float pr[8];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        pr[4 * c + v] = __builtin_amdgcn_exp2f(__builtin_fmaf(sa[c][v], a.scale_log2, -ref));
        lsum += pr[4 * c + v];
      }
    // P as two bf16 parts, p = hi + lo with hi = bf16(p) and lo = bf16(p - hi) (p - hi is exact in fp32), so
    // V stays bf16 as loaded (no conversion pass) and P keeps about 16 significant bits
    u32x4 ph, pl;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ph[e] = pack_bf16x2(pr[2 * e], pr[2 * e + 1]);
      pl[e] = pack_bf16x2(pr[2 * e] - __uint_as_float(ph[e] << 16), pr[2 * e + 1] - __uint_as_float(ph[e] & 0xFFFF0000u));
    }
    // O^T += V^T P^T, 16 dims per block, k = the tile's 32 columns in the lane-group order above
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(vr[db][0], vr[db][1], 0, 1, 2, 3, 4, 5, 6, 7));
      acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, __builtin_bit_cast(bf16x8, ph), acc[db], 0, 0, 0);
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(vr[db][0], vr[db][1], 0, 1, 2, 3, 4, 5, 6, 7));
      acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, __builtin_bit_cast(bf16x8, pl), acc[db], 0, 0, 0);
    }
  };

  // ---- pipeline (as in loop_attn_kernel, without the V conversion): step s reads the table entries of
  // tiles s+3 and s, waits for tile s, finalizes the records of tile s+4, passes the barrier,
  // loads the records of tile s+8, LDS-DMAs tile s+3 into the slot tile s-1 used and computes tile s.
  // Every step issues the same number of VMEM ops (one record load + NI DMA), so "tile s has landed" is
  // exactly vmcnt(2 * OPS_PER_STEP) on every path.
  const bool rec_wave = wave == 0;
  constexpr int OPS_PER_STEP = 1 + NI;
  u32x2 dA, dB, dC, dD;                   // records loaded four steps ahead, as in loop_attn_kernel
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const u32x2 r = load_desc(v);
    if (rec_wave) store_desc(v, r);
  }
  FL_WAIT_VM(0);                          // query fragments have arrived
  lds_barrier();
  dA = load_desc(4);
  __builtin_amdgcn_sched_barrier(0);
  dB = load_desc(5);
  __builtin_amdgcn_sched_barrier(0);
  issue(0, s0, tile_offs(0));
  __builtin_amdgcn_sched_barrier(0);
  dC = load_desc(6);
  __builtin_amdgcn_sched_barrier(0);
  issue(1, s1, tile_offs(1));
  __builtin_amdgcn_sched_barrier(0);
  dD = load_desc(7);
  __builtin_amdgcn_sched_barrier(0);
  issue(2, s2, tile_offs(2));

  auto step = [&](int u, Slot<D>& cur, Slot<D>& nxt, u32x2& w) {
    const Offs of = tile_offs(u + 3);
    const TileHead th = tile_head(u);
    FL_WAIT_VM(2 * OPS_PER_STEP);
    if (rec_wave) store_desc(u + 4, w);
    lds_barrier();
    w = load_desc(u + 8);
    __builtin_amdgcn_sched_barrier(0);
    issue(u + 3, nxt, of);
    if (u < n_tiles) compute(u, cur, th);
  };
  const int n_steps = (n_tiles + kRing - 1) / kRing * kRing;
  for (int u = 0; u < n_steps; u += kRing) {
    step(u, s0, s3, dA);
    step(u + 1, s1, s0, dB);
    step(u + 2, s2, s1, dC);
    step(u + 3, s3, s2, dD);
  }
  FL_WAIT_VM(0);
  lds_barrier();

  // ---- epilogue: lane (j16, g4) holds dims 16 db + 4 g4 .. +3 of row j16 ----------------------------
  lsum = row4_add(lsum);
  if (!row_ok) return;
  const int64_t orow = ((int64_t)b * a.N + row_i) * HD + (int64_t)h * D;
  const int64_t lrow = ((int64_t)b * a.N + row_i) * a.H + h;
  // the subtract term and mass are the previous loop's add term and mass of this row
  const int pp = a.slot_prev[(int64_t)b * a.N + row_i];
  const int64_t tp = ((int64_t)b * a.k_prev + pp) * a.H + h;
  const float msub = pp >= 0 ? a.mass_prev[tp] : 0.0f;
  const float* subp = a.term_prev + tp * D;
  const int64_t trow = ((int64_t)b * a.k + p) * a.H + h;
  const bool keep = a.term_out != nullptr;
  if (!(msub > 0.0f) || !(lsum > 0.0f)) {     // empty column set or vanished mass: unchanged
    if (keep) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<float4*>(a.term_out + trow * D + db * 16 + 4 * g4) = make_float4(0, 0, 0, 0);
      if (g4 == 0) a.mass_out[trow] = 0.0f;
    }
    return;
  }
  const float f = msub / lsum;
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const int dim = db * 16 + 4 * g4;
    const float4 sub = *reinterpret_cast<const float4*>(subp + dim);
    const float4 add = make_float4(acc[db][0] * f, acc[db][1] * f, acc[db][2] * f, acc[db][3] * f);
    float4 prev = *reinterpret_cast<const float4*>(a.o + orow + dim);
    prev.x = prev.x - sub.x + add.x;
    prev.y = prev.y - sub.y + add.y;
    prev.z = prev.z - sub.z + add.z;
    prev.w = prev.w - sub.w + add.w;
    *reinterpret_cast<float4*>(a.o + orow + dim) = prev;
    if (keep) *reinterpret_cast<float4*>(a.term_out + trow * D + dim) = add;
  }
  if (g4 == 0) {
    a.lse_ref[lrow] = (run_max + log2f(lsum)) * 0.6931471805599453f - logf(msub);
    if (keep) a.mass_out[trow] = msub;
  }
}

// ---- one pass over caches that hold a single loop's state, the column list in LDS -----------------------
// A tile is either 32 consecutive entries of the (b, h) column list or 32 consecutive band columns.  A
// workgroup copies the list entries into LDS once (up to kListCap of them), so every wave forms its own DMA
// offsets, column ids and tile bounds from that copy or from the band range: the pipeline has no record
// loads and no per-step table writes, and each step is one wait, one barrier, the DMA of tile s+3 and the
// math of tile s.  Rows, tiles and masks are those of reuse_attn_kernel.  Two kernels share the body:
//   cur_attn_kernel (SUB false): the add pass of loop r over the caches after the commit, with the online
//     softmax and the epilogue of reuse_attn_kernel (o_i <- o_i - term_prev_i + m_i add_i);
//   cur_sub_kernel (SUB true): the subtract pass over loop r-1's queries, caches and lse_ref (Section 4.2,
//     the removed part of the correction): probabilities against the fixed reference lse_ref (at most 1,
//     it normalizes a superset of S_i), so no running maximum; the epilogue writes the term
//     sum_{j in S_i} p_ij v_j and the mass sum_{j in S_i} p_ij at the row's position in rows.
constexpr int kListCap = 3072;


template <int D, bool SUB>
__device__ __forceinline__ void cur_body(const AttnArgs& a) {
  constexpr int BM = 64;                  // rows per workgroup (4 waves x 16)
  constexpr int KS = D / 32;              // k-steps of QK^T (32 dims each)
  constexpr int DB = D / 16;              // 16-dim output blocks
  constexpr int CH = D / 8;               // 16-byte chunks per row
  constexpr int COLS_PER_INST = 64 / CH;  // rows covered by one 1 KB LDS-DMA instruction
  constexpr int INST_PER_TILE = kBN / COLS_PER_INST;
  constexpr int INST_PER_WAVE = INST_PER_TILE / 4;   // per tensor (K and V each)
  constexpr int NI = 2 * INST_PER_WAVE;
  __shared__ Slot<D> s0, s1, s2, s3;
  __shared__ __attribute__((aligned(16))) int lst[kListCap + kBN];   // list entries of (b, h), kPad-padded to whole tiles
  __shared__ int s_meta[1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j16 = lane & 15, g4 = lane >> 4;

  // work item -> (batch*head, row tile); the row tiles of one (batch, head) stay on one XCD
  const int n_rt = (a.k + BM - 1) / BM;
  const int n_bh = a.B * a.H;
  int bh, rt;
  if ((n_bh & 7) == 0) {
    const int g = blockIdx.x & 7, s = blockIdx.x >> 3;
    bh = g + 8 * (s / n_rt);
    rt = n_rt - 1 - (s % n_rt);
  } else {
    bh = blockIdx.x / n_rt;
    rt = n_rt - 1 - (blockIdx.x % n_rt);
  }
  const int b = bh / a.H, h = bh % a.H;
  const int64_t HD = (int64_t)a.H * D;
  const int32_t* rowp = a.rows + (int64_t)b * a.k;

  const int p0 = rt * BM;
  const int last_p = min(p0 + BM, a.k) - 1;
  const int min_row = rowp[p0], max_row = rowp[last_p];
  const int gp0 = p0 + 16 * wave;
  const bool group_has_rows = gp0 < a.k;
  const int gmin = group_has_rows ? rowp[gp0] : 0;
  const int gmax = group_has_rows ? rowp[min(gp0 + 16, a.k) - 1] : -1;
  const int p = gp0 + j16;
  const bool row_ok = p < a.k;
  const int row_i = row_ok ? rowp[p] : -1;

  // query fragments (B operand of S^T = K Q^T): row j16, dims 32 ks + 8 g4 .. +7
  bf16x8 qa[KS];
  {
    const int64_t qoff = ((int64_t)b * a.N + (row_ok ? row_i : 0)) * HD + (int64_t)h * D + g4 * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint4 w = row_ok ? *reinterpret_cast<const uint4*>((SUB ? a.q_prev : a.q_cur) + qoff + ks * 32)
                             : make_uint4(0, 0, 0, 0);
      qa[ks] = __builtin_bit_cast(bf16x8, w);
    }
  }

  // ---- the list in LDS and the phase extents (uniform) --------------------------------------------------
  // nA = list entries j with j + window <= max_row (the only ones a row of this workgroup can see); the
  // list ascends, so thread i finds the boundary between entries i and i + 1
  const int32_t* cp = a.cols + (int64_t)bh * a.c_list;
  const int lim = max_row - a.window;
  if (tid == 0) s_meta[0] = 0;
  for (int i = tid; i < a.c_list; i += 256) lst[i] = cp[i];
  __syncthreads();
  for (int i = tid; i < a.c_list; i += 256)
    if (lst[i] <= lim && (i + 1 == a.c_list || lst[i + 1] > lim)) s_meta[0] = i + 1;
  __syncthreads();
  const int nA = __builtin_amdgcn_readfirstlane(s_meta[0]);
  if (tid < kBN) lst[nA + tid] = kPad;    // the last list tile's padding (entries nA .. are not read before)
  const int bandLo = a.window > 0 ? max(0, min_row - a.window + 1) : 0;
  const int bandHi = a.window > 0 ? max_row : -1;
  const int tA = (nA + kBN - 1) / kBN;
  const int tB = bandHi >= bandLo ? (bandHi - bandLo + kBN) / kBN : 0;
  const int n_tiles = tA + tB;
  const bool band_down = (rt & 1) != 0;   // neighbouring row tiles meet in the band columns they share
  // tile v: list entries [kBN v, kBN v + kBN) or band columns [first, first + kBN) (ascending columns in
  // both); returns the first entry index (list) or first column (band)
  auto tile_first = [=](int v) {
    const int tb = band_down ? tA + tB - 1 - v : v - tA;
    return v < tA ? v * kBN : bandLo + tb * kBN;
  };

  // ---- LDS-DMA offsets: lane column c of instruction t (same for K and V) -------------------------------
  const uint32_t rb = (uint32_t)(HD * 2);
  const uint32_t head_off = (uint32_t)(h * D * 2);
  const rsrc_t kcR = make_rsrc(a.k_cache + (int64_t)b * a.N * HD, (uint32_t)a.N * rb);
  const rsrc_t vcR = make_rsrc(a.v_cache + (int64_t)b * a.N * HD, (uint32_t)a.N * rb);
  auto inst_of = [=](int t) { return wave * INST_PER_WAVE + (t % INST_PER_WAVE); };
  int lcol[INST_PER_WAVE];                // tile column of this lane in instruction t
  uint32_t lsw[INST_PER_WAVE];            // its swizzled chunk offset
#pragma unroll
  for (int t = 0; t < INST_PER_WAVE; ++t) {
    lcol[t] = inst_of(t) * COLS_PER_INST + lane / CH;
    lsw[t] = (uint32_t)((lane % CH) ^ swz16_f<D>(lcol[t])) * 16 + head_off;
  }
  struct Offs { uint32_t o[INST_PER_WAVE]; };
  // (no branches: the list copy is read at a valid index for band tiles too, and the choice is a select)
  auto tile_offs = [=](int v) {
    Offs r;
    const int f = tile_first(v);
    const bool in_list = v < tA;
    const int fl = in_list ? f : 0;
    const int hi = in_list ? kBN - 1 : v < n_tiles ? bandHi - f : -1;   // tile columns c <= hi exist
#pragma unroll
    for (int t = 0; t < INST_PER_WAVE; ++t) {
      const int idl = lst[fl + lcol[t]];
      const int id = in_list ? idl : f + lcol[t];
      r.o[t] = ((id != kPad) & (lcol[t] <= hi)) ? (uint32_t)id * rb + lsw[t] : kOOB;
    }
    return r;
  };
  // (each offset goes through a local: handing the struct member straight to the builtin makes the
  // host compilation drop the kernel's launch stub)
  auto issue = [=](Slot<D>& sl, const Offs& of) {
#pragma unroll
    for (int t = 0; t < NI; ++t) {
      const int inst = inst_of(t);
      const uint32_t off = of.o[t % INST_PER_WAVE];
      if (t < INST_PER_WAVE)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(kcR, FL_LDS(sl.k + inst * 512), 16, off, 0, 0, kDmaPolicy);
      else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(vcR, FL_LDS(sl.v + inst * 512), 16, off, 0, 0, kDmaPolicy);
    }
  };
  // LDS read offsets (elements) of the fragments.  K (A operand): row j16 (+16 for the second column
  // block), data chunk 4 ks + g4.  V (transposed reads): lane (g4, t, q) reads dims 16 db + 4q of column
  // 4 g4 + t (+16 for the second half of the k order), data chunk 2 db + (q >> 1).
  int koff[KS], voff[DB];
  {
    const int t4 = j16 >> 2, q = lane & 3;
    const int colv = 4 * g4 + t4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) koff[ks] = j16 * D + ((4 * ks + g4) ^ swz16_f<D>(j16)) * 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) voff[db] = colv * D + ((2 * db + (q >> 1)) ^ swz16_f<D>(colv)) * 8 + 4 * (q & 1);
  }

  f32x4 acc[DB];                          // add (or subtract) term, O^T blocks
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x4{};
  float run_max = -INFINITY, lsum = 0.0f;   // running reference (log2 units) and row sum
  // subtract pass: the row's loop r-1 log-normaliser in log2 units, the fixed reference
  float lse2 = 0.0f;
  if (SUB && row_ok) lse2 = a.lse_ref[((int64_t)b * a.N + row_i) * a.H + h] * 1.4426950408889634f;

  // the lane's 8 column ids (16c + 4 g4 + v) come from the list copy or the band range
  auto compute = [=, &acc, &run_max, &lsum](int u, const Slot<D>& sl) {
    const bool is_list = u < tA;          // uniform
    const int f = tile_first(u);
    const int fl = is_list ? f : 0;
    // first and last column of the tile (kPad past the list's end; the band's last tile ends at bandHi)
    const int l0 = __builtin_amdgcn_readfirstlane(lst[fl]);
    const int l1 = __builtin_amdgcn_readfirstlane(lst[fl + kBN - 1]);
    const int c0 = is_list ? l0 : f;
    const int clast = is_list ? l1 : min(f + kBN - 1, bandHi);
    // (bitwise, so the tests stay scalar arithmetic without branches)
    const bool active = group_has_rows & (c0 <= (is_list ? gmax - a.window : gmax)) &
                        (is_list | (clast > gmin - a.window));
    const bool full = is_list ? clast <= gmin - a.window
                              : (f + kBN - 1 <= bandHi) & (clast <= gmin) & (c0 > gmax - a.window);
    if (!active) return;
    // every LDS read of the tile first, unconditionally (a read under a branch can lose the information
    // that tells it apart from the pending LDS-DMA writes)
    int4 ca_[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) ca_[c] = *reinterpret_cast<const int4*>(&lst[fl + 16 * c + 4 * g4]);
    u32x4 kw[KS][2];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        kw[ks][c] = *reinterpret_cast<const u32x4*>(&sl.k[koff[ks] + 16 * c * D]);
    i16x4 vr[DB][2];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int o = voff[db];
      vr[db][0] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(FL_LDS4(&sl.v[o]));
      vr[db][1] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(FL_LDS4(&sl.v[o + 16 * D]));
    }
    f32x4 sa[2] = {f32x4{}, f32x4{}};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        sa[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kw[ks][c]), qa[ks], sa[c], 0, 0, 0);
    // scores in log2 units first (the products are canonical, so the maximum needs no quieting step)
#pragma unroll
    for (int c = 0; c < 2; ++c) sa[c] *= a.scale_log2;
    if (!full) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        if (is_list) {                    // list columns: j + window <= i
          const int ci[4] = {ca_[c].x, ca_[c].y, ca_[c].z, ca_[c].w};
          const int lim_i = row_i - a.window;
#pragma unroll
          for (int v = 0; v < 4; ++v) sa[c][v] = ci[v] <= lim_i ? sa[c][v] : -INFINITY;
        } else {                          // band columns f + 16c + 4 g4 + v: i - window < j <= i
          const uint32_t w = (uint32_t)a.window;
          const uint32_t d0 = (uint32_t)(row_i - f - 16 * c - 4 * g4);
#pragma unroll
          for (int v = 0; v < 4; ++v) sa[c][v] = d0 - (uint32_t)v < w ? sa[c][v] : -INFINITY;
        }
      }
    }
    float ref = lse2;
    if constexpr (!SUB) {
      const float pinf = a.pinf;
      float tmax = fmax_nn(fmax_nn(fmax_nn(sa[0][0], sa[0][1], pinf), fmax_nn(sa[0][2], sa[0][3], pinf), pinf),
                           fmax_nn(fmax_nn(sa[1][0], sa[1][1], pinf), fmax_nn(sa[1][2], sa[1][3], pinf), pinf), pinf);
      {
        auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(tmax), __float_as_uint(tmax), false, false);
        tmax = fmax_nn(__uint_as_float(r[0]), __uint_as_float(r[1]), pinf);
        r = __builtin_amdgcn_permlane32_swap(__float_as_uint(tmax), __float_as_uint(tmax), false, false);
        tmax = fmax_nn(__uint_as_float(r[0]), __uint_as_float(r[1]), pinf);
      }
      // online softmax with a lazily raised reference (it moves only when a score exceeds it by more than
      // 8 in log2 units, so probabilities stay <= 256 and rescaling is rare)
      const bool raise = tmax > run_max + 8.0f;            // false while both are -inf
      if (__builtin_amdgcn_ballot_w64(raise) != 0) {        // uniform: rescale the rows that need it
        const float nm = raise ? tmax : run_max;
        const float alpha = raise ? __builtin_amdgcn_exp2f(run_max - nm) : 1.0f;   // exp2(-inf) = 0
        lsum *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) acc[db] *= alpha;
        run_max = nm;
      }
      ref = run_max == -INFINITY ? 0.0f : run_max;
    }
    float pr[8];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        pr[4 * c + v] = __builtin_amdgcn_exp2f(sa[c][v] - ref);
        lsum += pr[4 * c + v];
      }
    // P as two bf16 parts, p = hi + lo with hi = bf16(p) and lo = bf16(p - hi) (p - hi is exact in fp32)
    u32x4 ph, pl;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ph[e] = pack_bf16x2(pr[2 * e], pr[2 * e + 1]);
      pl[e] = pack_bf16x2(pr[2 * e] - __uint_as_float(ph[e] << 16), pr[2 * e + 1] - __uint_as_float(ph[e] & 0xFFFF0000u));
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(vr[db][0], vr[db][1], 0, 1, 2, 3, 4, 5, 6, 7));
      acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, __builtin_bit_cast(bf16x8, ph), acc[db], 0, 0, 0);
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(vr[db][0], vr[db][1], 0, 1, 2, 3, 4, 5, 6, 7));
      acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, __builtin_bit_cast(bf16x8, pl), acc[db], 0, 0, 0);
    }
  };

  // ---- pipeline: step s waits for tile s (issued three steps earlier: tiles s+1 and s+2 may still be in
  // flight, 2 NI operations), passes the barrier (every wave is done with tile s-1), LDS-DMAs tile s+3
  // into the slot tile s-1 used and computes tile s.  Every step issues exactly NI VMEM operations.
  __syncthreads();                        // the padding entries
  FL_WAIT_VM(0);                          // query fragments have arrived
  issue(s0, tile_offs(0));
  __builtin_amdgcn_sched_barrier(0);
  issue(s1, tile_offs(1));
  __builtin_amdgcn_sched_barrier(0);
  issue(s2, tile_offs(2));
  auto step = [&](int u, Slot<D>& cur, Slot<D>& nxt) {
    const Offs of = tile_offs(u + 3);
    FL_WAIT_VM(2 * NI);
    lds_barrier();
    issue(nxt, of);
    if (u < n_tiles) compute(u, cur);
  };
  const int n_steps = (n_tiles + kRing - 1) / kRing * kRing;
  for (int u = 0; u < n_steps; u += kRing) {
    step(u, s0, s3);
    step(u + 1, s1, s0);
    step(u + 2, s2, s1);
    step(u + 3, s3, s2);
  }
  FL_WAIT_VM(0);
  lds_barrier();

  // ---- epilogue: lane (j16, g4) holds dims 16 db + 4 g4 .. +3 of row j16 ----------------------------
  lsum = row4_add(lsum);
  if (!row_ok) return;
  if constexpr (SUB) {                    // the subtract term and the mass, at the row's position in rows
    const int64_t srow = ((int64_t)b * a.k + p) * a.H + h;
#pragma unroll
    for (int db = 0; db < DB; ++db)
      *reinterpret_cast<float4*>(a.term_out + srow * D + db * 16 + 4 * g4) =
          make_float4(acc[db][0], acc[db][1], acc[db][2], acc[db][3]);
    if (g4 == 0) a.mass_out[srow] = lsum;
    return;
  }
  const int64_t orow = ((int64_t)b * a.N + row_i) * HD + (int64_t)h * D;
  const int64_t lrow = ((int64_t)b * a.N + row_i) * a.H + h;
  // the subtract term and mass are the previous loop's add term and mass of this row
  const int pp = a.slot_prev[(int64_t)b * a.N + row_i];
  const int64_t tp = ((int64_t)b * a.k_prev + pp) * a.H + h;
  const float msub = pp >= 0 ? a.mass_prev[tp] : 0.0f;
  const float* subp = a.term_prev + tp * D;
  const int64_t trow = ((int64_t)b * a.k + p) * a.H + h;
  const bool keep = a.term_out != nullptr;
  if (!(msub > 0.0f) || !(lsum > 0.0f)) {     // empty column set or vanished mass: unchanged
    if (keep) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<float4*>(a.term_out + trow * D + db * 16 + 4 * g4) = make_float4(0, 0, 0, 0);
      if (g4 == 0) a.mass_out[trow] = 0.0f;
    }
    return;
  }
  const float fm = msub / lsum;
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const int dim = db * 16 + 4 * g4;
    const float4 sub = *reinterpret_cast<const float4*>(subp + dim);
    const float4 add = make_float4(acc[db][0] * fm, acc[db][1] * fm, acc[db][2] * fm, acc[db][3] * fm);
    float4 prev = *reinterpret_cast<const float4*>(a.o + orow + dim);
    prev.x = prev.x - sub.x + add.x;
    prev.y = prev.y - sub.y + add.y;
    prev.z = prev.z - sub.z + add.z;
    prev.w = prev.w - sub.w + add.w;
    *reinterpret_cast<float4*>(a.o + orow + dim) = prev;
    if (keep) *reinterpret_cast<float4*>(a.term_out + trow * D + dim) = add;
  }
  if (g4 == 0) {
    a.lse_ref[lrow] = (run_max + log2f(lsum)) * 0.6931471805599453f - logf(msub);
    if (keep) a.mass_out[trow] = msub;
  }
}

template <int D>
__global__ __launch_bounds__(256, 2) void cur_attn_kernel(AttnArgs a) {
  cur_body<D, false>(a);
}
template <int D>
__global__ __launch_bounds__(256, 2) void cur_sub_kernel(AttnArgs a) {
  cur_body<D, true>(a);
}

// Tile records of the sparse update, each an int2 (column, aux):
//   [0, BH*c)                         list of (b, h): (column, slot of the column)
//   [off_upd + bh*c, ...)             its entries updated this loop, compacted in order: (column, slot)
//   [off_band + b*N, ... + N)         every column j of batch b: (j, slot[j])
//   [off_rows + b*k, ... + k)         the updated rows of batch b: (rows[p], p)
//   off_sent                          sentinel (kPad, -1)
// followed by n_upd[B*H].  Blocks [0, B*H) build the lists, the remaining ones the per-batch regions.
constexpr int kPrepThreads = 1024;
__global__ __launch_bounds__(kPrepThreads) void attn_prep_kernel(const int32_t* __restrict__ cols,
                                                        const int32_t* __restrict__ slot,
                                                        const int32_t* __restrict__ rows, int c_list,
                                                        int N, int H, int B, int k, int per_batch,
                                                        int off_upd, int off_band, int off_rows, int off_sent,
                                                        int2* __restrict__ rec, int32_t* __restrict__ n_upd) {
  constexpr int kWaves = kPrepThreads / 64;
  __shared__ int wsum[kWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if ((int)blockIdx.x >= B * H) {
    const int e = blockIdx.x - B * H;
    const int b = e / per_batch, part = e % per_batch;
    for (int j = part * kPrepThreads + tid; j < N; j += per_batch * kPrepThreads)
      rec[off_band + (int64_t)b * N + j] = make_int2(j, slot[(int64_t)b * N + j]);
    for (int p = part * kPrepThreads + tid; p < k; p += per_batch * kPrepThreads)
      rec[off_rows + (int64_t)b * k + p] = make_int2(rows[(int64_t)b * k + p], p);
    if (e == 0 && tid == 0) rec[off_sent] = make_int2(kPad, -1);
    return;
  }
  const int bh = blockIdx.x, b = bh / H;
  const int32_t* cp = cols + (int64_t)bh * c_list;
  int2* dp = rec + (int64_t)bh * c_list;
  int2* up = rec + off_upd + (int64_t)bh * c_list;
  int base = 0;
  for (int p0 = 0; p0 < c_list; p0 += kPrepThreads) {
    const int pos = p0 + tid;
    int cid = -1, s = -1;
    if (pos < c_list) {
      cid = cp[pos];
      s = slot[(int64_t)b * N + cid];
      dp[pos] = make_int2(cid, s);
    }
    const int flag = (pos < c_list && s >= 0) ? 1 : 0;
    int incl = flag;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int t = __shfl_up(incl, off, 64);
      if (lane >= off) incl += t;
    }
    __syncthreads();
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      before += (w < wave) ? wsum[w] : 0;
      total += wsum[w];
    }
    if (flag) up[base + before + incl - 1] = make_int2(cid, s);
    base += total;
  }
  if (tid == 0) n_upd[bh] = base;
}

}  // namespace fl

using namespace fl;

// record counts of the workspace regions (see attn_prep_kernel)
struct RecLayout {
  size_t off_upd, off_band, off_rows, off_sent, n_rec;
};
static RecLayout rec_layout(int B, int N, int H, int k, int c_list) {
  RecLayout L;
  const size_t list = (size_t)B * H * (size_t)c_list;
  L.off_upd = list;
  L.off_band = 2 * list;
  L.off_rows = L.off_band + (size_t)B * N;
  L.off_sent = L.off_rows + (size_t)B * k;
  L.n_rec = L.off_sent + 1;
  return L;
}

static size_t attn_ws_bytes(int B, int N, int H, int k, int c_list, bool dense) {
  if (dense || B < 1 || N < 1 || H < 1 || k < 0 || c_list < 0) return 0;
  const RecLayout L = rec_layout(B, N, H, k, c_list);
  return L.n_rec * sizeof(int2) + (size_t)B * H * sizeof(int32_t);
}

extern "C" size_t fl_loop_sparse_attn_ws(int B, int N, int H, int d, int k, int c_list, int window,
                                         int flags) {
  (void)d; (void)window;
  return attn_ws_bytes(B, N, H, k, c_list, (flags & FL_ATTN_DENSE) != 0);
}

static int loop_sparse_attn(const uint16_t* q_cur, const uint16_t* q_prev, const uint16_t* k_cache,
                            const uint16_t* v_cache, const uint16_t* v16, const uint16_t* k_new, const uint16_t* v_new,
                            const int32_t* slot, const int32_t* rows, int k, const int32_t* cols, int c_list,
                            int window, int B, int N, int H, int d, float sm_scale, int flags, float* lse_ref,
                            float* o, const float* term_prev, const float* mass_prev, const int32_t* slot_prev,
                            int k_prev, float* term_out, float* mass_out, void* ws, size_t ws_bytes,
                            void* stream) {
  const bool dense = (flags & FL_ATTN_DENSE) != 0;
  const bool reuse = term_prev != nullptr;
  FL_REQUIRE((flags & ~FL_ATTN_DENSE) == 0, FL_E_UNSUPPORTED, "fl_loop_sparse_attn: unknown flags 0x%x", flags);
  FL_REQUIRE(q_cur && k_cache && v_cache && lse_ref && o, FL_E_NULL,
             "fl_loop_sparse_attn: q_cur, k_cache, v_cache, lse_ref and o are required");
  FL_REQUIRE(B >= 1 && N >= 1 && H >= 1, FL_E_SHAPE, "fl_loop_sparse_attn: need B, N, H >= 1");
  FL_REQUIRE(d == 64 || d == 128, FL_E_SHAPE, "fl_loop_sparse_attn: head dim %d not in {64, 128}", d);
  FL_REQUIRE((int64_t)N * H * d <= ((int64_t)1 << 30), FL_E_SHAPE,
             "fl_loop_sparse_attn: N * H * d above 2^30 (byte offsets must stay below 2^31)");
  FL_REQUIRE(sm_scale > 0.0f && std::isfinite(sm_scale), FL_E_RANGE, "fl_loop_sparse_attn: sm_scale must be > 0");
  FL_REQUIRE((term_out == nullptr) == (mass_out == nullptr), FL_E_NULL,
             "fl_loop_sparse_attn: term_out and mass_out go together");
  if (dense) {
    FL_REQUIRE(rows == nullptr && k == N, FL_E_SHAPE, "fl_loop_sparse_attn: DENSE needs rows == NULL and k == N");
    FL_REQUIRE(!reuse && term_out == nullptr, FL_E_UNSUPPORTED, "fl_loop_sparse_attn: DENSE keeps no terms");
  } else {
    // (with given terms over current caches the tiles come straight from cols and the band: no slot map)
    FL_REQUIRE(rows && (reuse || q_prev) && (slot || (reuse && k_new == nullptr)), FL_E_NULL,
               "fl_loop_sparse_attn: q_prev (unless reusing terms), slot and rows are required");
    FL_REQUIRE((k_new == nullptr) == (v_new == nullptr), FL_E_NULL,
               "fl_loop_sparse_attn: k_new and v_new go together");
    FL_REQUIRE(reuse || k_new, FL_E_NULL,
               "fl_loop_sparse_attn: k_new and v_new are required unless reusing terms with current caches");
    FL_REQUIRE(k >= 0 && k <= N, FL_E_RANGE, "fl_loop_sparse_attn: k=%d outside [0, N]", k);
    FL_REQUIRE(c_list >= 0 && c_list <= N, FL_E_RANGE, "fl_loop_sparse_attn: c_list=%d outside [0, N]", c_list);
    FL_REQUIRE(c_list == 0 || cols, FL_E_NULL, "fl_loop_sparse_attn: cols is required when c_list > 0");
    FL_REQUIRE(window >= 0, FL_E_RANGE, "fl_loop_sparse_attn: window must be >= 0");
    if (reuse) {
      FL_REQUIRE(mass_prev && slot_prev, FL_E_NULL, "fl_loop_sparse_attn: term_prev needs mass_prev and slot_prev");
      FL_REQUIRE(k_prev >= k && k_prev <= N, FL_E_RANGE, "fl_loop_sparse_attn: k_prev=%d outside [k, N]", k_prev);
    }
  }
  // (given terms over current caches build no tile records: no workspace)
  const bool current = !dense && reuse && k_new == nullptr;
  const size_t need = current ? 0 : attn_ws_bytes(B, N, H, k, c_list, dense);
  FL_REQUIRE(dense || current || rec_layout(B, N, H, k, c_list).n_rec * sizeof(int2) <= ((size_t)1 << 31) - 8, FL_E_SHAPE,
             "fl_loop_sparse_attn: tile records above 2^31 bytes (reduce B * H * c_list + B * (N + k))");
  FL_REQUIRE(need == 0 || (ws && ws_bytes >= need), FL_E_WORKSPACE,
             "fl_loop_sparse_attn: workspace of %zu bytes required", need);
  if (k == 0) return FL_OK;
  hipStream_t st = as_stream(stream);
  if (!dense) {
    FL_CHECK_LIST("fl_loop_sparse_attn", "rows", rows, B, k, 0, N, st);
    FL_CHECK_LIST("fl_loop_sparse_attn", "cols", cols, (int64_t)B * H, c_list, 0, N, st);
  }
  {
    // the products with V run in fp16 on the dense, two-pass and band add-pass paths
    int rc = check_f16_range("fl_loop_sparse_attn", "v_cache", v_cache, (int64_t)B * N * H * d, st);
    if (rc == FL_OK && !dense && v_new) rc = check_f16_range("fl_loop_sparse_attn", "v_new", v_new, (int64_t)B * k * H * d, st);
    if (rc != FL_OK) return rc;
  }
  AttnArgs a{};
  a.q_cur = q_cur;
  a.q_prev = (dense || reuse) ? nullptr : q_prev;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.k_new = dense ? nullptr : k_new;
  a.v_new = dense ? nullptr : v_new;
  a.slot = dense ? nullptr : slot;
  a.rows = dense ? nullptr : rows;
  a.cols = dense ? nullptr : cols;
  a.lse_ref = lse_ref;
  a.o = o;
  a.term_prev = term_prev;
  a.mass_prev = mass_prev;
  a.slot_prev = slot_prev;
  a.term_out = term_out;
  a.mass_out = mass_out;
  a.k = k;
  a.k_prev = reuse ? k_prev : 0;
  a.c_list = dense ? 0 : c_list;
  a.window = dense ? 0 : window;
  a.B = B;
  a.N = N;
  a.H = H;
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  a.cache_current = (!dense && reuse && k_new == nullptr) ? 1 : 0;
  a.pinf = INFINITY;
  if (!dense && !a.cache_current) {       // (current caches: tiles come straight from cols and the band)
    const RecLayout L = rec_layout(B, N, H, k, c_list);
    int2* rec = static_cast<int2*>(ws);
    int32_t* n_upd = reinterpret_cast<int32_t*>(rec + L.n_rec);
    a.rec = rec;
    a.n_upd = n_upd;
    a.off_upd = (int)L.off_upd;
    a.off_band = (int)L.off_band;
    a.off_rows = (int)L.off_rows;
    a.off_sent = (int)L.off_sent;
    a.rec_bytes = (uint32_t)(L.n_rec * sizeof(int2));
    const int per_batch = std::min(64, (N + k + 4 * kPrepThreads - 1) / (4 * kPrepThreads));
    attn_prep_kernel<<<B * H + B * per_batch, kPrepThreads, 0, st>>>(cols, slot, rows, c_list, N, H, B, k, per_batch,
                                                          a.off_upd, a.off_band, a.off_rows, a.off_sent, rec,
                                                          n_upd);
    int rc = check_launch("attn_prep_kernel");
    if (rc != FL_OK) return rc;
  }
  const int bm = dense ? 128 : 64;          // rows per workgroup
  dim3 grid(((k + bm - 1) / bm) * B * H);
  if (dense) {
    if (d == 128) loop_attn_kernel<128, kDense><<<grid, 256, 0, st>>>(a);
    else loop_attn_kernel<64, kDense><<<grid, 256, 0, st>>>(a);
    return check_launch("loop_attn_kernel");
  }
  if (!reuse) {
    if (d == 128) loop_attn_kernel<128, kFull><<<grid, 256, 0, st>>>(a);
    else loop_attn_kernel<64, kFull><<<grid, 256, 0, st>>>(a);
    return check_launch("loop_attn_kernel");
  }
#define FL_REUSE(DD, CC) reuse_attn_kernel<DD, CC><<<grid, 256, 0, st>>>(a)
  if (a.cache_current) {
    const int rc = launch_seg_cur(q_cur, k_cache, v_cache, v16, rows, k, cols, c_list, window, B, N, H, d, sm_scale, lse_ref,
                                  o, term_prev, mass_prev, slot_prev, k_prev, term_out, mass_out, st);
    if (rc != FL_E_UNSUPPORTED) return rc;
  }
  if (a.cache_current && c_list <= kListCap) {
    if (d == 128) cur_attn_kernel<128><<<grid, 256, 0, st>>>(a);
    else cur_attn_kernel<64><<<grid, 256, 0, st>>>(a);
    return check_launch("cur_attn_kernel");
  }
  if (a.cache_current) {
    if (d == 128) FL_REUSE(128, true); else FL_REUSE(64, true);
  } else {
    if (d == 128) FL_REUSE(128, false); else FL_REUSE(64, false);
  }
#undef FL_REUSE
  return check_launch("reuse_attn_kernel");
}

extern "C" int fl_loop_sparse_attn(const uint16_t* q_cur, const uint16_t* q_prev,
                                   const uint16_t* k_cache, const uint16_t* v_cache,
                                   const uint16_t* k_new, const uint16_t* v_new,
                                   const int32_t* slot, const int32_t* rows, int k,
                                   const int32_t* cols, int c_list, int window, int B, int N, int H,
                                   int d, float sm_scale, int flags, float* lse_ref, float* o,
                                   void* ws, size_t ws_bytes, void* stream) {
  FL_API_BEGIN
  return loop_sparse_attn(q_cur, q_prev, k_cache, v_cache, nullptr, k_new, v_new, slot, rows, k, cols, c_list,
                          window, B, N, H, d, sm_scale, flags, lse_ref, o, nullptr, nullptr, nullptr, 0, nullptr,
                          nullptr, ws, ws_bytes, stream);
  FL_API_END
}

extern "C" int fl_loop_sparse_attn_terms(const uint16_t* q_cur, const uint16_t* q_prev,
                                         const uint16_t* k_cache, const uint16_t* v_cache,
                                         const uint16_t* k_new, const uint16_t* v_new,
                                         const int32_t* slot, const int32_t* rows, int k,
                                         const int32_t* cols, int c_list, int window, int B, int N, int H,
                                         int d, float sm_scale, float* lse_ref, float* o,
                                         const float* term_prev, const float* mass_prev,
                                         const int32_t* slot_prev, int k_prev, float* term_out,
                                         float* mass_out, void* ws, size_t ws_bytes, void* stream) {
  FL_API_BEGIN
  return loop_sparse_attn(q_cur, q_prev, k_cache, v_cache, nullptr, k_new, v_new, slot, rows, k, cols, c_list,
                          window, B, N, H, d, sm_scale, 0, lse_ref, o, term_prev, mass_prev, slot_prev, k_prev,
                          term_out, mass_out, ws, ws_bytes, stream);
  FL_API_END
}

extern "C" int fl_loop_sparse_attn_terms_v16(const uint16_t* q_cur, const uint16_t* k_cache, const uint16_t* v_cache,
                                             const uint16_t* v_cache_f16, const int32_t* rows, int k,
                                             const int32_t* cols, int c_list, int window, int B, int N, int H,
                                             int d, float sm_scale, float* lse_ref, float* o,
                                             const float* term_prev, const float* mass_prev,
                                             const int32_t* slot_prev, int k_prev, float* term_out,
                                             float* mass_out, void* stream) {
  FL_API_BEGIN
  FL_REQUIRE(v_cache_f16 != nullptr, FL_E_NULL, "fl_loop_sparse_attn_terms_v16: v_cache_f16 is required");
  FL_REQUIRE(term_prev != nullptr, FL_E_NULL, "fl_loop_sparse_attn_terms_v16: term_prev is required");
  // (current caches and given terms: no record workspace)
  return loop_sparse_attn(q_cur, nullptr, k_cache, v_cache, v_cache_f16, nullptr, nullptr, nullptr, rows, k, cols,
                          c_list, window, B, N, H, d, sm_scale, 0, lse_ref, o, term_prev, mass_prev, slot_prev,
                          k_prev, term_out, mass_out, nullptr, 0, stream);
  FL_API_END
}

// Shapes the subtract pass covers: the segment kernels (a list of at most 2048 entries and, with a band,
// their descriptor table), else the 64-row kernel with the list in LDS (a list of at most kListCap entries).
static bool subtract_supported(int k, int c_list, int window, int N, int d) {
  return seg_supported(k, c_list, window, N, d) ||
         ((d == 64 || d == 128) && window >= 0 && c_list >= 0 && c_list <= kListCap);
}

extern "C" const char* fl_attn_kernel_name(int pass, int k, int c_list, int window, int B, int N, int H, int d) {
  if (k < 1 || k > N || B < 1 || H < 1 || c_list < 0 || c_list > N || window < 0 || (d != 64 && d != 128))
    return nullptr;
  const int teams = seg_teams(k, c_list, window, N, d, B * H);
  switch (pass) {
    case FL_PASS_ADD:
      return teams == 1 ? "seg1_cur_kernel" : teams == 2 ? "seg_cur_kernel"
             : c_list <= kListCap ? "cur_attn_kernel" : "reuse_attn_kernel";
    case FL_PASS_SUBTRACT:
      return teams == 1 ? "seg1_sub_kernel" : teams == 2 ? "seg_sub_kernel"
             : c_list <= kListCap ? "cur_sub_kernel" : nullptr;
    case FL_PASS_BOTH:
      return "loop_attn_kernel";
    default:
      return nullptr;
  }
}

extern "C" int fl_loop_subtract_terms_supported(int k, int c_list, int window, int N, int d) {
  return subtract_supported(k, c_list, window, N, d) ? 1 : 0;
}

// The subtract pass (fl_loop_subtract_terms, and with v16 an fp16 copy of v_cache for the segment kernels).
static int subtract_terms(const char* fn, const uint16_t* q_prev, const uint16_t* k_cache, const uint16_t* v_cache,
                          const uint16_t* v16, const int32_t* rows, int k, const int32_t* cols, int c_list,
                          int window, int B, int N, int H, int d, float sm_scale, const float* lse_ref,
                          float* term_out, float* mass_out, void* stream) {
  FL_REQUIRE(q_prev && k_cache && v_cache && lse_ref, FL_E_NULL, "%s: q_prev, k_cache, v_cache and lse_ref are required",
             fn);
  FL_REQUIRE(k == 0 || (rows && term_out && mass_out), FL_E_NULL, "%s: rows, term_out and mass_out are required", fn);
  FL_REQUIRE(B >= 1 && N >= 1 && H >= 1 && k >= 0 && k <= N, FL_E_SHAPE, "%s: need B, N, H >= 1 and 0 <= k <= N", fn);
  FL_REQUIRE(d == 64 || d == 128, FL_E_SHAPE, "%s: head dim %d not in {64, 128}", fn, d);
  FL_REQUIRE((int64_t)N * H * d <= ((int64_t)1 << 30), FL_E_SHAPE,
             "%s: N * H * d above 2^30 (byte offsets must stay below 2^31)", fn);
  FL_REQUIRE(c_list >= 0 && c_list <= N && (c_list == 0 || cols), FL_E_SHAPE, "%s: bad column list", fn);
  FL_REQUIRE(window >= 0, FL_E_SHAPE, "%s: window must be >= 0", fn);
  FL_REQUIRE(sm_scale > 0.0f && std::isfinite(sm_scale), FL_E_RANGE, "%s: sm_scale must be > 0", fn);
  if (k == 0) return FL_OK;
  FL_REQUIRE(subtract_supported(k, c_list, window, N, d), FL_E_UNSUPPORTED,
             "%s: column list of %d entries above %d (fl_loop_sparse_attn runs both passes for every shape)", fn,
             c_list, kListCap);
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FL_CHECK_LIST(fn, "rows", rows, B, k, 0, N, st);
  FL_CHECK_LIST(fn, "cols", cols, (int64_t)B * H, c_list, 0, N, st);
  if (seg_supported(k, c_list, window, N, d)) {
    // (the segment kernel's products with V run in fp16)
    const int rc = check_f16_range(fn, "v_cache", v_cache, (int64_t)B * N * H * d, st);
    if (rc != FL_OK) return rc;
    return launch_seg_sub(q_prev, k_cache, v_cache, v16, rows, k, cols, c_list, window, B, N, H, d, sm_scale, lse_ref,
                          term_out, mass_out, st);
  }
  AttnArgs a{};
  a.q_prev = q_prev;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.rows = rows;
  a.cols = cols;
  a.lse_ref = const_cast<float*>(lse_ref);   // (read only in this pass)
  a.term_out = term_out;
  a.mass_out = mass_out;
  a.k = k;
  a.c_list = c_list;
  a.window = window;
  a.B = B;
  a.N = N;
  a.H = H;
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  a.cache_current = 1;
  a.pinf = INFINITY;
  dim3 grid((unsigned)(((k + 63) / 64) * B * H));
  if (d == 128) cur_sub_kernel<128><<<grid, 256, 0, st>>>(a);
  else cur_sub_kernel<64><<<grid, 256, 0, st>>>(a);
  return check_launch("cur_sub_kernel");
}

extern "C" int fl_loop_subtract_terms(const uint16_t* q_prev, const uint16_t* k_cache, const uint16_t* v_cache,
                                      const int32_t* rows, int k, const int32_t* cols, int c_list, int window,
                                      int B, int N, int H, int d, float sm_scale, const float* lse_ref,
                                      float* term_out, float* mass_out, void* stream) {
  FL_API_BEGIN
  return subtract_terms("fl_loop_subtract_terms", q_prev, k_cache, v_cache, nullptr, rows, k, cols, c_list, window,
                        B, N, H, d, sm_scale, lse_ref, term_out, mass_out, stream);
  FL_API_END
}

extern "C" int fl_loop_subtract_terms_v16(const uint16_t* q_prev, const uint16_t* k_cache, const uint16_t* v_cache,
                                          const uint16_t* v_cache_f16, const int32_t* rows, int k,
                                          const int32_t* cols, int c_list, int window, int B, int N, int H, int d,
                                          float sm_scale, const float* lse_ref, float* term_out, float* mass_out,
                                          void* stream) {
  FL_API_BEGIN
  FL_REQUIRE(v_cache_f16 != nullptr, FL_E_NULL, "fl_loop_subtract_terms_v16: v_cache_f16 is required");
  return subtract_terms("fl_loop_subtract_terms_v16", q_prev, k_cache, v_cache, v_cache_f16, rows, k, cols, c_list,
                        window, B, N, H, d, sm_scale, lse_ref, term_out, mass_out, stream);
  FL_API_END
}
