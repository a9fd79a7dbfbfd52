// Mass-corrected sparse attention update over row segments (Appendix D.2, Eq. 7; Sections 3.2, 4.2): two
// passes, each in a two-team and a one-team layout, all from one body.
//   seg_cur_kernel, the add pass, for a loop whose subtract term and mass are given (the previous loop's
//   stored add term, or the subtract pass below) and whose caches already hold this loop's state:
//     L_i = log sum_{j in S_i} exp(l_ij),  add_i = sum_j exp(l_ij - L_i) v_j,  l_ij = sigma q_i . k_j,
//     o_i <- o_i - term_prev_i + m_i add_i,   lse_ref_i <- L_i - log m_i;
//   seg_sub_kernel, the subtract pass over the previous loop's queries, caches and lse_ref:
//     sub_i = sum_{j in S_i} exp(l_ij - lse_ref_i) v_j,  m_i = sum_{j in S_i} exp(l_ij - lse_ref_i)
//     (a fixed reference: no running maximum, and the two teams' sums simply add);
// over S_i = (list U {j : i - w < j <= i}) restricted to j <= i, list columns taking the condition
// j + w <= i so that a column in both is counted once.
//
// Work decomposition.  One workgroup of 8 waves takes a segment of up to 128 consecutive updated rows of
// one (batch, head).  The rows form four 32-row groups, each held by one wave of each team (query
// fragments, running maximum, sum and output blocks).  The column tiles of the segment -- the
// list entries the segment's last row can see, and the band columns from its first row's band start to
// its last row -- form one sequence in which list and band tiles are interleaved evenly (the band tiles
// stream from HBM while the list tiles, shared by every segment of the head and kept in L2, keep the
// matrix cores busy).  Step s gives tile 2s to team 0 and tile 2s + 1 to team 1; each team keeps its own
// softmax state, and the two are merged per row at the end.  Without a band and with enough rows, the
// one-team kernels (seg1_*: four waves, step s takes tile s, no merge) run two workgroups per CU that step
// independently instead of eight waves in lockstep.
//
// L2 sharing of the band.  Neighbouring segments of a head need the same band columns around their
// boundary (about w columns).  Each segment walks the band tiles it shares with a neighbour before the
// rest: even segments the lower shared range first, odd segments the upper one first, so both segments of
// every boundary reach the shared columns at about the same time.  The segments of one (batch, head) run
// on one XCD, which holds its L2.
//
// Data movement: tiles of 32 columns are gathered by LDS-DMA (buffer_load ... lds) into a ring of four
// steps (two tiles each) three steps ahead; out-of-range offsets read zeros.  Each wave converts the value
// rows its own DMA wrote from bf16 to fp16 in place (exact for 2^-14 <= |v| <= 65504; smaller magnitudes
// round to a multiple of 2^-24; larger ones overflow) one step before they are used, after its own math.
// Contractions: S^T = K Q^T
// on v_mfma_f32_32x32x16_bf16 (lane (r, h) holds columns 8j + 4h .. +3, j = 0..3, of row r of the group),
// O^T += V^T P^T on v_mfma_f32_32x32x16_f16 with V read transposed and P rounded to fp16; the transposed V
// reads take the columns in the order the lane already holds them, so P needs no shuffle.
#include "fl_attn_util.h"

#include <algorithm>
#include <type_traits>

namespace fl {

constexpr int kSegRows = 128;        // rows per segment at most (4 groups of 32)
constexpr int kSegListCap = 2048;    // list entries kept in LDS
constexpr int kSegTileCap = 2048;    // tile descriptors kept in LDS (list tiles + band tiles of a segment)
constexpr int kSeg1TileCap = 128;    // the same for the one-team kernels (list tiles only: no band)
static_assert((kSegListCap + kBN - 1) / kBN + 1 <= kSeg1TileCap, "the one-team table holds every list tile");
constexpr int kSegSteps = 4;         // ring depth in steps

struct SegArgs {
  const uint16_t* q;          // [B, N, H, d] queries of this loop
  const uint16_t* k_cache;    // [B, N, H, d] this loop's K_hat, V_hat
  const uint16_t* v_cache;
  const uint16_t* v16;        // optional fp16 copy of v_cache (same layout): the tiles' values need no conversion
  const int32_t* rows;        // [B, k] ascending updated rows
  const int32_t* cols;        // [B, H, c_list] ascending column list
  float* lse_ref;             // [B, N, H]
  float* o;                   // [B, N, H, d]
  const float* term_prev;     // [B, k_prev, H, d]
  const float* mass_prev;     // [B, k_prev, H]
  const int32_t* slot_prev;   // [B, N]
  float* term_out;            // optional [B, k, H, d]
  float* mass_out;            // optional [B, k, H]
  int k, k_prev, c_list, window, B, N, H;
  int n_seg, seg_rows;        // segments per (batch, head) and rows per segment (<= kSegRows)
  float scale_log2;           // sm_scale * log2(e)
  float pinf;                 // +inf (a kernel argument, so the median below is not folded into a max)
};

template <int D, bool SUB, int TEAMS, bool V16>
__device__ __forceinline__ void seg_body(const SegArgs& a) {
  static_assert(TEAMS == 1 || TEAMS == 2, "one or two teams of four waves");
  constexpr int NT = 256 * TEAMS;         // threads
  constexpr int kTileCap = TEAMS == 2 ? kSegTileCap : kSeg1TileCap;
  constexpr int KS = D / 16;              // k-steps of QK^T (16 dims each)
  constexpr int DB = D / 32;              // 32-dim output blocks
  constexpr int CH = D / 8;               // 16-byte chunks per row
  constexpr int CPI = 64 / CH;            // tile columns covered by one 1 KB LDS-DMA instruction
  constexpr int IPT = kBN / CPI;          // instructions per tensor and tile
  constexpr int NIK = IPT / 4;            // K (and V) instructions per wave: a team's 4 waves load its tile
  constexpr int NI = 2 * NIK;             // VMEM operations per wave and step
  // The four ring slots and the list are separate LDS objects (a slot holds both teams' tiles): the compiler
  // then tells every LDS read apart from the LDS-DMA writes still in flight into the other slots (one
  // object would make it wait for all of them before each read).
  __shared__ Slot<D> ring0[TEAMS], ring1[TEAMS], ring2[TEAMS], ring3[TEAMS];   // step slot s, team t: ring<s>[t]
  __shared__ __attribute__((aligned(16))) int lst[kSegListCap + kBN];   // the (b, h) list, kPad-padded
  __shared__ int2 tdesc[kTileCap];        // per sequence position: first column or entry, kind, group bits
  __shared__ int s_grp[8];                // first and last row of each of the 4 groups
  __shared__ int s_meta[1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int team = TEAMS == 2 ? wave >> 2 : 0, w4 = wave & 3;
  // the wave's row group: team 0 wave w takes group w, team 1 wave w group w + 2 (mod 4), so the two waves
  // of one group sit on different SIMDs when waves w and w + 4 share one (a band tile is often seen by one
  // or two neighbouring groups only)
  const int grp = team ? (w4 + 2) & 3 : w4;
  const int r32 = lane & 31, hw = lane >> 5;

  // ---- work item -> (batch*head, segment); the segments of one (batch, head) stay on one XCD ----------
  const int n_bh = a.B * a.H;
  int bh, seg;
  if ((n_bh & 7) == 0) {
    const int x = blockIdx.x & 7, s = blockIdx.x >> 3;
    bh = x + 8 * (s / a.n_seg);
    seg = s % a.n_seg;
  } else {
    bh = blockIdx.x / a.n_seg;
    seg = blockIdx.x % a.n_seg;
  }
  const int b = bh / a.H, h = bh % a.H;
  const int64_t HD = (int64_t)a.H * D;
  const int32_t* rowp = a.rows + (int64_t)b * a.k;
  const int P0 = seg * a.seg_rows;
  const int P1 = min(P0 + a.seg_rows, a.k);
  const int min_row = rowp[P0], max_row = rowp[P1 - 1];

  // ---- the wave's group: rows 32 grp .. +31 of the segment --------------------------------------------
  const int pos = P0 + 32 * grp + r32;
  const bool row_ok = pos < P1;
  const int row_i = row_ok ? rowp[pos] : -1;
  bf16x8 qf[KS];                          // B operand of S^T = K Q^T: row r32, dims 16 ks + 8 hw .. +7
  {
    const int64_t qoff = ((int64_t)b * a.N + (row_ok ? row_i : 0)) * HD + (int64_t)h * D + hw * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint4 w = row_ok ? *reinterpret_cast<const uint4*>(a.q + qoff + ks * 16) : make_uint4(0, 0, 0, 0);
      qf[ks] = __builtin_bit_cast(bf16x8, w);
    }
  }
  // add pass: the row's slot in the previous loop's terms, looked up with the queries (the epilogue's other
  // loads depend on it)
  int pp = -1;
  if constexpr (!SUB) {
    if (row_ok && team == 0) pp = a.slot_prev[(int64_t)b * a.N + row_i];
  }

  // ---- the list in LDS; nA = entries j with j + window <= max_row (the ones a row here can see) -------
  const int32_t* cp = a.cols + (int64_t)bh * a.c_list;
  const int w = a.window;
  const int lim = max_row - w;
  if (tid == 0) s_meta[0] = 0;
  if (tid < 4) {                          // group bounds (a group without rows gets last row -1)
    const int gp0 = P0 + 32 * tid;
    const bool has = gp0 < P1;
    s_grp[2 * tid] = has ? rowp[gp0] : 0;
    s_grp[2 * tid + 1] = has ? rowp[min(gp0 + 32, P1) - 1] : -1;
  }
  for (int i = tid; i < a.c_list; i += NT) lst[i] = cp[i];
  __syncthreads();
  for (int i = tid; i < a.c_list; i += NT)
    if (lst[i] <= lim && (i + 1 == a.c_list || lst[i + 1] > lim)) s_meta[0] = i + 1;
  __syncthreads();
  const int nA = __builtin_amdgcn_readfirstlane(s_meta[0]);
  if (tid < kBN) lst[nA + tid] = kPad;   // padding of the last list tile (entries from nA on are unread)

  // ---- tile sequence: nL list tiles and nB band tiles, interleaved evenly -----------------------------
  const int bandLo = w > 0 ? max(0, min_row - w + 1) : 0;
  const int bandHi = w > 0 ? max_row : -1;
  const int nL = (nA + kBN - 1) / kBN;
  const int nB = bandHi >= bandLo ? (bandHi - bandLo + kBN) / kBN : 0;
  // positions are handed out in pairs (position 2p to team 0, 2p + 1 to team 1), and both positions of a
  // pair hold the same kind of tile, so the two teams do similar work between two barriers
  const int nLP = (nL + 1) / 2, nBP = (nB + 1) / 2, nP = nLP + nBP;
  const int n_tiles = min(2 * nP, kTileCap);   // (the host keeps 2 nP within the table)
  // band tiles shared with the previous segment ([bandLo, its last row]) and with the next one
  // ([its first row - w + 1, bandHi]); the rest in the middle
  int nBot = 0, nTop = 0;
  if (w > 0 && nB > 0) {
    if (P0 > 0) {
      const int prev_last = rowp[P0 - 1];
      nBot = prev_last >= bandLo ? min(nB, (prev_last - bandLo) / kBN + 1) : 0;
    }
    if (P1 < a.k) {
      const int from = rowp[P1] - w + 1;
      const int t0 = from > bandLo ? (from - bandLo) / kBN : 0;
      nTop = nB - max(t0, nBot);
      nTop = nTop > 0 ? nTop : 0;
    }
  }
  const bool top_first = (seg & 1) != 0;
  __syncthreads();                        // list padding and group bounds
  // Descriptor of sequence position u = 2p + t: pair p holds list tiles when floor((p + 1) nLP / nP) >
  // floor(p nLP / nP) (list pairs spread evenly through the band pairs); a position past the last tile of
  // its kind is empty (no group bits, no columns).
  //   x: first list entry (list tile) or first column (band tile), bit 31 set for a band tile;
  //   y: bit g: group g (rows 32 g .. +31) sees some column of the tile; bit 8 + g: it sees every column;
  //      bits 16-20: the last existing column of the tile (band tiles end at the last row); bit 21: empty.
  for (int u = tid; u < n_tiles; u += NT) {
    const int pr = u >> 1, t = u & 1;
    const int before = (pr * nLP) / nP, after = ((pr + 1) * nLP) / nP;
    const bool is_list = after > before;
    int f = 0, c0 = 0, clast = -1, hi = 0;
    bool empty;
    if (is_list) {
      const int lt = 2 * before + t;
      empty = lt >= nL;
      f = lt * kBN;
      if (!empty) {
        c0 = lst[f];
        clast = lst[f + kBN - 1];
        hi = kBN - 1;
      }
    } else {
      const int q = 2 * (pr - before) + t;  // band order position
      empty = q >= nB;
      int bt;
      if (!top_first) bt = q < nBot ? q : q < nBot + nTop ? nB - nTop + (q - nBot) : q - nTop;
      else bt = q < nTop ? nB - nTop + q : q - nTop;
      f = bandLo + bt * kBN;
      if (!empty) {
        c0 = f;
        clast = min(f + kBN - 1, bandHi);
        hi = clast - f;
      }
    }
    uint32_t bits = ((uint32_t)hi << 16) | ((uint32_t)empty << 21);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int gmin = s_grp[2 * g], gmax = s_grp[2 * g + 1];
      const bool act = !empty & (gmax >= 0) & (c0 <= (is_list ? gmax - w : gmax)) & (is_list | (clast > gmin - w));
      const bool full = is_list ? clast <= gmin - w : (hi == kBN - 1) & (clast <= gmin) & (c0 > gmax - w);
      bits |= ((uint32_t)act << g) | ((uint32_t)(act & full) << (8 + g));
    }
    tdesc[u] = make_int2(is_list ? f : (int)(0x80000000u | (uint32_t)f), (int)bits);
  }

  // (a slot holds team 0's tile, then team 1's: the team's part is an offset from the slot's first tile, so
  // every address keeps the slot's own constant base)
  const int tofs = team * (int)(sizeof(Slot<D>) / sizeof(uint16_t));
  // ---- LDS-DMA offsets of this wave's instructions (its team's tile) -----------------------------------
  const uint32_t rb = (uint32_t)(HD * 2);
  const uint32_t head_off = (uint32_t)(h * D * 2);
  const rsrc_t kcR = make_rsrc(a.k_cache + (int64_t)b * a.N * HD, (uint32_t)a.N * rb);
  const rsrc_t vcR = make_rsrc((V16 ? a.v16 : a.v_cache) + (int64_t)b * a.N * HD, (uint32_t)a.N * rb);
  int lcol[NIK];
  uint32_t lsw[NIK];
#pragma unroll
  for (int t = 0; t < NIK; ++t) {
    const int inst = w4 * NIK + t;
    lcol[t] = inst * CPI + lane / CH;
    lsw[t] = (uint32_t)((lane % CH) ^ swz32_f<D>(lcol[t])) * 16 + head_off;
  }
  struct Offs { uint32_t o[NIK]; };
  // (the descriptor of position u is passed in: the step reads the next DMA tile's a step ahead)
  auto tile_offs_d = [&](int u, int2 dsc) __attribute__((always_inline)) {
    Offs r;
    const bool have = u < n_tiles;
    const int dx = __builtin_amdgcn_readfirstlane(dsc.x), dy = __builtin_amdgcn_readfirstlane(dsc.y);
    const bool in_list = dx >= 0;
    const int f = dx & 0x7FFFFFFF;
    const int hi = (have & !((dy >> 21) & 1)) ? (dy >> 16) & 31 : -1;   // tile columns c <= hi exist
    const int fl = (in_list & (hi >= 0)) ? f : 0;
#pragma unroll
    for (int t = 0; t < NIK; ++t) {
      const int idl = lst[fl + lcol[t]];
      const int id = in_list ? idl : f + lcol[t];
      r.o[t] = ((id != kPad) & (lcol[t] <= hi)) ? (uint32_t)id * rb + lsw[t] : kOOB;
    }
    return r;
  };
  auto tile_offs = [&](int u) __attribute__((always_inline)) {
    return tile_offs_d(u, tdesc[u < n_tiles ? u : 0]);
  };
  auto issue = [&](Slot<D>& sl, const Offs& of) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < NI; ++t) {
      const int inst = w4 * NIK + (t % NIK);
      const uint32_t off = of.o[t % NIK];
      if (t < NIK)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(kcR, FL_LDS(sl.k + tofs + inst * 512), 16, off, 0, 0, kDmaPolicy);
      else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(vcR, FL_LDS(sl.v + tofs + inst * 512), 16, off, 0, 0, kDmaPolicy);
    }
  };

  // LDS read offsets (elements).  K (A operand of S^T = K Q^T): row r32, data chunk 2 ks + hw.  V
  // (transposed reads for O^T += V^T P^T): lane (16 g + 4 t + q) points at V[col][dim0 + 4 q] of column
  // 16 kb + 4 (g >> 1) + t (and the same + 8), dims 32 db + 16 (g & 1) + 4 q, so the transpose hands lane
  // m of the group V[col_t][dim0 + m] and P^T needs no shuffle.
  int koff[KS], voff[DB], voff8[DB];
  {
    const int g16 = lane >> 4, m16 = lane & 15;
    const int tq = m16 >> 2, q = m16 & 3;
    const int col0 = 4 * (g16 >> 1) + tq;
    const int c_lo = 2 * (g16 & 1) + (q >> 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) koff[ks] = tofs + r32 * D + ((2 * ks + hw) ^ swz32_f<D>(r32)) * 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      voff[db] = tofs + col0 * D + ((4 * db + c_lo) ^ swz32_f<D>(col0)) * 8 + 4 * (q & 1);
      voff8[db] = tofs + (col0 + 8) * D + ((4 * db + c_lo) ^ swz32_f<D>(col0 + 8)) * 8 + 4 * (q & 1);
    }
  }

  f32x16 acc[DB];                         // O^T blocks: lane (r32, hw) holds dims 32 db + 8 j + 4 hw + i
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x16{};
  float run_max = -INFINITY, lsum = 0.0f; // log2 units; the lane's part of the row sum
  const int rband = row_i - 4 * hw;       // the row less the lane's column offset within a block of 8

  // ---- this wave's value rows of a tile, bf16 -> fp16 in place (the 16 bytes per lane its DMA wrote) ---
  auto convert = [&](Slot<D>& sl) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < NIK; ++t) {
      u32x4* pv = reinterpret_cast<u32x4*>(sl.v + tofs + (w4 * NIK + t) * 512 + lane * 8);
      const u32x4 x = *pv;
      u32x4 y;
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = pack_f16x2(__uint_as_float(x[e] << 16), __uint_as_float(x[e] & 0xFFFF0000u));
      *pv = y;
    }
  };

  // ---- one tile (list or band) for the wave's group: one code path for both kinds, so the accumulators
  // keep their registers across tiles; only the mask differs, and a tile every row of the group sees in
  // full skips it
  const float pinf = a.pinf;
  const float sc = a.scale_log2;
  // subtract pass: the previous loop's log-normaliser (log2 units) is the fixed reference
  float lse2 = 0.0f;
  if (SUB && row_ok) lse2 = a.lse_ref[((int64_t)b * a.N + row_i) * a.H + h] * 1.4426950408889634f;
  auto compute = [&](int dx, int dy, const Slot<D>& sl) __attribute__((always_inline)) {
    if (((dy >> grp) & 1) == 0) return;   // no row of the group sees a column of the tile
    const bool full = ((dy >> (8 + grp)) & 1) != 0;
    const bool is_list = dx >= 0;         // uniform
    const int f = dx & 0x7FFFFFFF;
    constexpr int NE = 16;                // scores per lane: columns 8 j + 4 hw + i of row r32
    // K fragments: the first half read before the products start, each later one issued with the product
    // KS/2 before it, so that a product waits on one LDS latency at most (the compiler's own order waits
    // between every pair: 1.5 % slower on both 32K passes; all KS reads ahead measured no faster)
    f32x16 sv = f32x16{};
    u32x4 kw[KS];
#pragma unroll
    for (int ks = 0; ks < KS / 2; ++ks) kw[ks] = *reinterpret_cast<const u32x4*>(&sl.k[koff[ks]]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + KS / 2 < KS) kw[ks + KS / 2] = *reinterpret_cast<const u32x4*>(&sl.k[koff[ks + KS / 2]]);
      sv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kw[ks]), qf[ks], sv, 0, 0, 0);
    }
    if (!full) {
      if (is_list) {                      // list columns: j + w <= i
        const int lim = row_i - w;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int4 c4 = *reinterpret_cast<const int4*>(&lst[f + 8 * j + 4 * hw]);
          sv[4 * j + 0] = c4.x <= lim ? sv[4 * j + 0] : -INFINITY;
          sv[4 * j + 1] = c4.y <= lim ? sv[4 * j + 1] : -INFINITY;
          sv[4 * j + 2] = c4.z <= lim ? sv[4 * j + 2] : -INFINITY;
          sv[4 * j + 3] = c4.w <= lim ? sv[4 * j + 3] : -INFINITY;
        }
      } else {                            // band columns f + 8 j + 4 hw + i: i - w < j <= i
        const uint32_t d0 = (uint32_t)(rband - f);
#pragma unroll
        for (int v = 0; v < NE; ++v) {
          const uint32_t off = (uint32_t)(8 * (v >> 2) + (v & 3));
          sv[v] = d0 - off < (uint32_t)w ? sv[v] : -INFINITY;
        }
      }
    }
    // subtract pass: probabilities against the fixed reference (they are at most 1: the reference is the
    // log-normaliser over a superset of the columns); add pass: the online softmax below
    float ref = lse2;
    if constexpr (!SUB) {
      // row maximum and (below) row sum as trees: the tile's chain of dependent instructions is its latency
      float m8[8];
#pragma unroll
      for (int v = 0; v < 8; ++v) m8[v] = fmax_nn(sv[v], sv[v + 8], pinf);
#pragma unroll
      for (int v = 0; v < 4; ++v) m8[v] = fmax_nn(m8[v], m8[v + 4], pinf);
      m8[0] = fmax_nn(m8[0], m8[2], pinf);
      m8[1] = fmax_nn(m8[1], m8[3], pinf);
      float t = fmax_nn(m8[0], m8[1], pinf);
      {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(t), __float_as_uint(t), false, false);
        t = fmax_nn(__uint_as_float(r[0]), __uint_as_float(r[1]), pinf);
      }
      const float tmax = t * sc;            // log2 units (sc > 0 keeps the order; -inf stays -inf)
      // online softmax with a lazily raised reference (moved only when a score exceeds it by more than 8 in
      // log2 units: probabilities stay <= 256 and rescaling is rare)
      const bool raise = tmax > run_max + 8.0f;
      if (__builtin_amdgcn_ballot_w64(raise) != 0) {
        const float nm = raise ? tmax : run_max;
        const float alpha = raise ? __builtin_amdgcn_exp2f(run_max - nm) : 1.0f;   // exp2(-inf) = 0
        lsum *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) acc[db] *= alpha;
        run_max = nm;
      }
      ref = run_max == -INFINITY ? 0.0f : run_max;
    }
    float pr[NE];
#pragma unroll
    for (int v = 0; v < NE; ++v) pr[v] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[v], sc, -ref));
    {
      float a4[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) a4[v] = (pr[v] + pr[v + 4]) + (pr[v + 8] + pr[v + 12]);
      lsum += (a4[0] + a4[1]) + (a4[2] + a4[3]);
    }
    // O^T += V^T P^T, P rounded to fp16, two 16-column halves of the tile
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

  // ---- pipeline: step s passes the barrier (every wave is done with step s-1, and every value row of step s
  // was converted to fp16 by the wave whose DMA wrote it), computes its tile of step s, has each team DMA
  // its tile of step s+3 into the slot step s-1 used (after the math, which the barrier releases first),
  // then waits for its own rows of step s+1 (issued two steps earlier; s+2 and s+3 may still be in flight,
  // 2 NI operations per wave) and converts their values, while slower waves still compute.  Every step
  // issues exactly NI VMEM operations per wave.
  __syncthreads();                        // the descriptors
  FL_WAIT_VM(0);                          // query fragments have arrived
  const int n_steps = (n_tiles + TEAMS - 1) / TEAMS;
  const int n_loop = (n_steps + kSegSteps - 1) / kSegSteps * kSegSteps;
  issue(ring0[0], tile_offs(team));
  __builtin_amdgcn_sched_barrier(0);
  issue(ring1[0], tile_offs(TEAMS + team));
  __builtin_amdgcn_sched_barrier(0);
  issue(ring2[0], tile_offs(2 * TEAMS + team));
  int u = team;                           // this team's position at the current step
  int2 dsc = tdesc[u < n_tiles ? u : 0];  // its descriptor, read one step ahead
  // the descriptor of the tile the step DMAs, also read a step ahead, so the offsets at the top of a step
  // wait on the list reads alone (1-2 % on both 32K passes)
  int2 dsc_dma = tdesc[u + 3 * TEAMS < n_tiles ? u + 3 * TEAMS : 0];
  if constexpr (!V16) {                   // (an fp16 copy of the values lands ready)
    FL_WAIT_VM(2 * NI);                   // step 0 has landed
    convert(ring0[0]);
  }
  auto step = [&](Slot<D>& cur, Slot<D>& nxt, Slot<D>& nx1) __attribute__((always_inline)) {   // (the slots' first tiles; the team's is at tofs)
    const Offs of = tile_offs_d(u + 3 * TEAMS, dsc_dma);
    dsc_dma = tdesc[u + 4 * TEAMS < n_tiles ? u + 4 * TEAMS : 0];
    const int dx = __builtin_amdgcn_readfirstlane(dsc.x), dy = __builtin_amdgcn_readfirstlane(dsc.y);
    const bool have = u < n_tiles;
    dsc = tdesc[u + TEAMS < n_tiles ? u + TEAMS : 0];
    FL_WAIT_VM(2 * NI);                   // (step s: converted at the end of step s-1, so already landed)
    lds_barrier();
    if (have) compute(dx, dy, cur);
    issue(nxt, of);                       // (after the math: the step's critical path starts at the barrier)
    if constexpr (!V16) {
      FL_WAIT_VM(2 * NI);                 // step s+1 has landed (s+2 and s+3 may be in flight)
      convert(nx1);                       // its value rows to fp16, in the shadow of the other waves' math
    }
    u += TEAMS;
  };
  for (int s = 0; s < n_loop; s += kSegSteps) {
    step(ring0[0], ring3[0], ring1[0]);
    step(ring1[0], ring0[0], ring2[0]);
    step(ring2[0], ring1[0], ring3[0]);
    step(ring3[0], ring2[0], ring0[0]);
  }
  FL_WAIT_VM(0);
  lds_barrier();

  // ---- merge the two teams' states per row; team 0 finishes the group -------------------------------
  // Team 1's partial goes through the (now idle) ring: per wave 32 rows x D fp32 output values (DB x 16 x
  // 64 lanes) in slot grp of team 1's half, and the reference and sum of each lane's row (64 x 2) in slot
  // 3 of team 0's half.
  lsum = xor32_add(lsum);                 // the two half-waves hold disjoint columns of the same row
  if constexpr (TEAMS == 2) {
    float* xs = reinterpret_cast<float*>(ring3[0].k) + grp * 128;
    float* xo = reinterpret_cast<float*>(grp == 0 ? ring0[1].k : grp == 1 ? ring1[1].k : grp == 2 ? ring2[1].k
                                                                                         : ring3[1].k);
    if (team) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<f32x4*>(&xo[((db * 4 + j) * 64 + lane) * 4]) =
              f32x4{acc[db][4 * j], acc[db][4 * j + 1], acc[db][4 * j + 2], acc[db][4 * j + 3]};
      xs[lane * 2] = run_max;
      xs[lane * 2 + 1] = lsum;
    }
    lds_barrier();
    if (team) return;
    const float m_o = xs[lane * 2], l_o = xs[lane * 2 + 1];
    // combine (run_max, lsum, acc) with (m_o, l_o, team 1's acc); an empty state has sum 0 and reference
    // -inf, and contributes nothing (its factor is exp2(-inf) = 0)
    // (the subtract pass has one fixed reference: plain sums)
    const float mm = fmaxf(run_max, m_o);
    const float fs = SUB ? 1.0f : mm == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(run_max - mm);
    const float fo = SUB ? 1.0f : mm == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(m_o - mm);
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 ao = *reinterpret_cast<const f32x4*>(&xo[((db * 4 + j) * 64 + lane) * 4]);
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[db][4 * j + i] = acc[db][4 * j + i] * fs + ao[i] * fo;
      }
    lsum = lsum * fs + l_o * fo;
    run_max = mm;
    // (the combine stays here: sunk into the epilogue, team 1's partial would be live beside the
    // epilogue's loads)
#pragma unroll
    for (int db = 0; db < DB; ++db) asm volatile("" : "+v"(acc[db]));
  }
  // ---- epilogue ----------------------------------------------------------------------------------------
  // The wave's 32 x D results (lane (r32, hw) holds dims 32 db + 8 j + 4 hw .. +3 of row r32) go through LDS
  // and back, so that every global access covers whole rows: 256 / D rows per instruction, each lane 16
  // contiguous bytes (in the MFMA layout an instruction touches 32 rows, 32 bytes of each).  The wave's
  // LDS block is its own: ring slot grp of the last team (two teams: the slot team 1's partial came
  // through, already read; one team: the ring is idle after the last barrier).  Chunk c (16 bytes) of row
  // rr sits at chunk position c ^ (rr & 7) of the row.
  constexpr int CPR = D / 4;              // 16-byte chunks per row
  constexpr int NR = 64 / CPR;            // rows per instruction
  constexpr int NIE = 32 / NR;            // instructions per 32 rows
  float* es = reinterpret_cast<float*>(grp == 0 ? ring0[TEAMS - 1].k : grp == 1 ? ring1[TEAMS - 1].k
                                       : grp == 2 ? ring2[TEAMS - 1].k : ring3[TEAMS - 1].k);
  auto es_at = [&](int rr, int c) __attribute__((always_inline)) { return es + (rr * CPR + (c ^ (rr & 7))) * 4; };
  const int rsub = lane / CPR, cc = lane % CPR;   // this lane's row (within an instruction's rows) and chunk
  const int g0 = P0 + 32 * grp;           // position in rows of the group's first row
  const int nrow = min(32, P1 - g0);      // rows of the group (<= 0: none)
  if constexpr (SUB) {                    // the subtract term and the mass, at the row's position in rows
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<f32x4*>(es_at(r32, 8 * db + 2 * j + hw)) =
            f32x4{acc[db][4 * j], acc[db][4 * j + 1], acc[db][4 * j + 2], acc[db][4 * j + 3]};
#pragma unroll
    for (int i = 0; i < NIE; ++i) {
      const int rr = NR * i + rsub;
      const f32x4 t = *reinterpret_cast<const f32x4*>(es_at(rr, cc));
      if (rr < nrow)
        *reinterpret_cast<f32x4*>(a.term_out + (((int64_t)b * a.k + g0 + rr) * a.H + h) * D + 4 * cc) = t;
    }
    if (row_ok && hw == 0) a.mass_out[((int64_t)b * a.k + pos) * a.H + h] = lsum;
    return;
  }
  // add pass: rows whose previous term has mass and whose new columns have some are updated; the others
  // keep their output and get a zero term and mass
  const int64_t tp = ((int64_t)b * a.k_prev + (pp >= 0 ? pp : 0)) * a.H + h;
  const float msub = pp >= 0 ? a.mass_prev[tp] : 0.0f;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<f32x4*>(es_at(r32, 8 * db + 2 * j + hw)) =
          f32x4{acc[db][4 * j], acc[db][4 * j + 1], acc[db][4 * j + 2], acc[db][4 * j + 3]};
  __builtin_amdgcn_sched_barrier(0);      // (the accumulators' registers are free from here)
  // the output rows and the previous terms in the row-contiguous layout (each row's slot was looked up
  // with the queries); every load goes out before the first use
  f32x4 po[NIE], ps[NIE];
#pragma unroll
  for (int i = 0; i < NIE; ++i) {
    const int rr = NR * i + rsub;
    const int ri = __shfl(row_i, rr, 64), pr = __shfl(pp, rr, 64);
    const bool ld = rr < nrow && pr >= 0;
    const int64_t orr = ((int64_t)b * a.N + (ld ? ri : 0)) * HD + (int64_t)h * D + 4 * cc;
    const int64_t tpr = (((int64_t)b * a.k_prev + (ld ? pr : 0)) * a.H + h) * D + 4 * cc;
    po[i] = ld ? *reinterpret_cast<const f32x4*>(a.o + orr) : f32x4{};
    ps[i] = ld ? *reinterpret_cast<const f32x4*>(a.term_prev + tpr) : f32x4{};
  }
  const bool upd = row_ok && msub > 0.0f && lsum > 0.0f;
  const float fsh = upd ? msub / lsum : -1.0f;    // the row's factor m / sum; negative: not updated
  const bool keep_terms = a.term_out != nullptr;
#pragma unroll
  for (int i = 0; i < NIE; ++i) {
    const int rr = NR * i + rsub;
    // (both permutes before the branch: a permute reads 0 from a source lane that is switched off, and
    // lane rr's own row in this instruction may be past the group's last)
    const float f = __shfl(fsh, rr, 64);            // (negative for a row past the group's last)
    const int ri = __shfl(row_i, rr, 64);
    const f32x4 t = *reinterpret_cast<const f32x4*>(es_at(rr, cc));
    const f32x4 add = f >= 0.0f ? f32x4{t[0] * f, t[1] * f, t[2] * f, t[3] * f} : f32x4{};
    if (f >= 0.0f) {
      *reinterpret_cast<f32x4*>(a.o + ((int64_t)b * a.N + ri) * HD + (int64_t)h * D + 4 * cc) =
          (po[i] - ps[i]) + add;
    }
    if (keep_terms && rr < nrow)
      *reinterpret_cast<f32x4*>(a.term_out + (((int64_t)b * a.k + g0 + rr) * a.H + h) * D + 4 * cc) = add;
  }
  if (row_ok && hw == 0) {
    const int64_t trow = ((int64_t)b * a.k + pos) * a.H + h;
    if (upd) a.lse_ref[((int64_t)b * a.N + row_i) * a.H + h] =
        (run_max + log2f(lsum)) * 0.6931471805599453f - logf(msub);
    if (keep_terms) a.mass_out[trow] = upd ? msub : 0.0f;
  }
}

// V16: the values come from the fp16 copy (a.v16) instead of being converted in LDS.
template <int D, bool V16>
__global__ __launch_bounds__(512, 2) void seg_cur_kernel(SegArgs a) {
  seg_body<D, false, 2, V16>(a);
}
template <int D, bool V16>
__global__ __launch_bounds__(512, 2) void seg_sub_kernel(SegArgs a) {
  seg_body<D, true, 2, V16>(a);
}
// One team of four waves (no band): two workgroups per CU instead of one lockstep workgroup of eight waves.
template <int D, bool V16>
__global__ __launch_bounds__(256, 2) void seg1_cur_kernel(SegArgs a) {
  seg_body<D, false, 1, V16>(a);
}
template <int D, bool V16>
__global__ __launch_bounds__(256, 2) void seg1_sub_kernel(SegArgs a) {
  seg_body<D, true, 1, V16>(a);
}

// The launch of one of the four kernels for head dim d and an optional fp16 value copy.
#define FL_SEG_LAUNCH(KERNEL, THREADS)                                                      \
  do {                                                                                        \
    if (d == 128) {                                                                           \
      if (a.v16) KERNEL<128, true><<<grid, THREADS, 0, st>>>(a);                              \
      else KERNEL<128, false><<<grid, THREADS, 0, st>>>(a);                                   \
    } else {                                                                                  \
      if (a.v16) KERNEL<64, true><<<grid, THREADS, 0, st>>>(a);                               \
      else KERNEL<64, false><<<grid, THREADS, 0, st>>>(a);                                    \
    }                                                                                         \
  } while (0)

// Whether the segment kernels cover a shape: a list that fits in LDS and, with a band, the descriptor table
// (without one, the table holds at most ceil(c_list / 32) + 1 positions, within either kernel's).
bool seg_supported(int k, int c_list, int window, int N, int d) {
  if (window < 0 || c_list > kSegListCap || (d != 64 && d != 128) || k < 1) return false;
  if (window == 0) return true;
  // the descriptor table holds every position: at most ceil(c_list / 32) list tiles and ceil(N / 32) + 1 band
  // tiles, plus one empty position per kind when the counts are odd
  return (c_list + kBN - 1) / kBN + (N + kBN - 1) / kBN + 3 <= kSegTileCap;
}

// One team or two.  Without a band, the one-team kernel runs two independent workgroups per CU, each
// stepping at its own pace, where the two-team workgroup steps eight waves in lockstep; it pays off once
// there are about 1.5 full 128-row segments per CU (measured on the 16K batch-4 loops: 12-22 % faster
// from 706 rows per (b, h) up, 12-14 % slower at 328).  With a band the two teams share the band tiles.
static bool seg_one_team(int k, int window, int bh) {
  return window == 0 && (int64_t)((k + kSegRows - 1) / kSegRows) * bh >= 384;
}

int seg_teams(int k, int c_list, int window, int N, int d, int bh) {
  if (!seg_supported(k, c_list, window, N, d)) return 0;
  return seg_one_team(k, window, bh) ? 1 : 2;
}

// Segments per (batch, head): at least one per 128 rows; more (down to 64 rows) while the grid is below
// `per_cu` workgroups per CU.  Sets a.n_seg and a.seg_rows.
static void seg_grid(SegArgs& a, int k, int bh, int per_cu) {
  constexpr int kCUs = 256;
  int n_seg = (k + kSegRows - 1) / kSegRows;
  const int fill = (per_cu * kCUs + bh - 1) / bh;
  const int n_max = (k + 63) / 64;
  if (n_seg < fill) n_seg = std::min(fill, n_max);
  if (n_seg < 1) n_seg = 1;
  const int seg_rows = (k + n_seg - 1) / n_seg;
  a.n_seg = (k + seg_rows - 1) / seg_rows;
  a.seg_rows = seg_rows;
}

// Subtract pass over the previous loop's state (queries q of loop r-1, caches X_hat^(r-1), lse_ref of loop
// r-1): per updated row the term sum_j exp(sigma q . k_j - lse_ref) v_j and its mass, written at the row's
// position in rows.  FL_E_UNSUPPORTED (nothing launched) outside seg_supported.
int launch_seg_sub(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, const uint16_t* v16,
                   const int32_t* rows, int k,
                   const int32_t* cols, int c_list, int window, int B, int N, int H, int d, float sm_scale,
                   const float* lse_ref, float* term_out, float* mass_out, hipStream_t st) {
  const int teams = seg_teams(k, c_list, window, N, d, B * H);
  if (teams == 0) return FL_E_UNSUPPORTED;
  SegArgs a{};
  a.q = q; a.k_cache = k_cache; a.v_cache = v_cache; a.v16 = v16; a.rows = rows; a.cols = cols;
  a.lse_ref = const_cast<float*>(lse_ref);   // (read only in this pass)
  a.term_out = term_out; a.mass_out = mass_out;
  a.k = k; a.c_list = c_list; a.window = window; a.B = B; a.N = N; a.H = H;
  const bool one = teams == 1;
  seg_grid(a, k, B * H, one ? 2 : 1);
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  a.pinf = INFINITY;
  dim3 grid((unsigned)(a.n_seg * B * H));
  if (one) {
    FL_SEG_LAUNCH(seg1_sub_kernel, 256);
    return check_launch("seg1_sub_kernel");
  }
  FL_SEG_LAUNCH(seg_sub_kernel, 512);
  return check_launch("seg_sub_kernel");
}

// Launch of the segment kernel for a reuse loop over current caches; returns FL_E_UNSUPPORTED (nothing
// launched) when the shape is outside what it covers, so the caller can take another kernel.
int launch_seg_cur(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, const uint16_t* v16,
                   const int32_t* rows, int k,
                   const int32_t* cols, int c_list, int window, int B, int N, int H, int d, float sm_scale,
                   float* lse_ref, float* o, const float* term_prev, const float* mass_prev,
                   const int32_t* slot_prev, int k_prev, float* term_out, float* mass_out, hipStream_t st) {
  const int teams = seg_teams(k, c_list, window, N, d, B * H);
  if (teams == 0) return FL_E_UNSUPPORTED;
  SegArgs a{};
  a.q = q; a.k_cache = k_cache; a.v_cache = v_cache; a.v16 = v16; a.rows = rows; a.cols = cols;
  a.lse_ref = lse_ref; a.o = o; a.term_prev = term_prev; a.mass_prev = mass_prev; a.slot_prev = slot_prev;
  a.term_out = term_out; a.mass_out = mass_out;
  a.k = k; a.k_prev = k_prev; a.c_list = c_list; a.window = window; a.B = B; a.N = N; a.H = H;
  const bool one = teams == 1;
  seg_grid(a, k, B * H, one ? 2 : 1);
  a.scale_log2 = sm_scale * 1.4426950408889634f;
  a.pinf = INFINITY;
  dim3 grid((unsigned)(a.n_seg * B * H));
  if (one) {
    FL_SEG_LAUNCH(seg1_cur_kernel, 256);
    return check_launch("seg1_cur_kernel");
  }
  FL_SEG_LAUNCH(seg_cur_kernel, 512);
  return check_launch("seg_cur_kernel");
}

}  // namespace fl
