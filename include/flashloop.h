/*
 * flashloop.h -- C ABI of the FlashLoop per-loop attention step for MI355X (gfx950).
 *
 * The step updates one layer of a looped Transformer block at sparse loop r >= 2 (the method of
 * "FlashLoop: Fast and Memory-Efficient Looped Transformers via Lazy Updates"):
 *   1. fl_select_tokens       pick the rows whose state moved most since loop r-1
 *                             (Section 4.1; Appendix D.1, Eq. 5);
 *   2. fl_kv_residual_quant   store K/V of those rows as group-wise low-bit residuals against the
 *                             previous reconstruction (Section 4.3, Eq. 4; Appendix D.3, Eq. 8);
 *   3. fl_kv_residual_dequant rebuild X_hat^(r) rows from the residual (Eq. 8);
 *   4. fl_loop_sparse_attn    update the attention output of those rows from the previous loop's output
 *                             with a mass-corrected correction over predicted key columns
 *                             (Sections 3.2, 4.2, Eq. 3; Appendix D.2, Eq. 7).
 * plus two set-up helpers for a dense source loop (Appendix D.2, Eq. 6 with all causal keys):
 *   fl_column_scores, fl_select_columns; the decode step (fl_decode_step), the list pruning for a
 *   shrinking budget (fl_prune_columns) and the recent-token bf16 tail (fl_kv_keep_recent).
 *
 * Conventions shared by every call
 *   - Every data pointer is a DEVICE pointer (HIP device memory).  The caller allocates and owns all
 *     memory and keeps it alive until the enqueued work has completed.  The library never allocates,
 *     frees or synchronizes, and keeps no pointer after the call returns.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).  All work is enqueued
 *     asynchronously on it; nothing is read back to the host.
 *   - bf16 and fp16 values are passed as their raw 16-bit patterns (uint16_t).
 *   - Layouts are dense and row-major as written: [B, N, H, d] means element (b, i, h, e) lives at
 *     ((b * N + i) * H + h) * d + e.  Index lists are int32 and strictly ascending.
 *   - Return value: FL_OK, or an FL_E_* status.  Arguments are validated on the host before anything
 *     is enqueued; on a non-OK return nothing was launched and no output was written.  FL_E_HIP means
 *     a launch was rejected by the runtime; faults inside kernels surface at the caller's next
 *     synchronization.  fl_last_error() returns a thread-local message for the last non-OK return.
 *   - Results are deterministic: the same inputs give bitwise-identical outputs (no float atomics).
 *   - Supported sizes: head dim d in {64, 128}; B, N, H >= 1; N < 2^31 / (H * d), and for
 *     fl_loop_sparse_attn N * H * d <= 2^30 (byte offsets of one batch element stay below 2^31).
 */
#ifndef FLASHLOOP_H
#define FLASHLOOP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FL_ABI_VERSION 1

enum fl_status {
  FL_OK = 0,
  FL_E_NULL = 1,        /* a required pointer is NULL */
  FL_E_SHAPE = 2,       /* inconsistent or unsupported sizes */
  FL_E_RANGE = 3,       /* a count is out of its range (e.g. k > n_cand) */
  FL_E_UNSUPPORTED = 4, /* unsupported bit width, axis, mode or flag */
  FL_E_WORKSPACE = 5,   /* workspace missing or too small */
  FL_E_HIP = 6,         /* the HIP runtime rejected a launch */
  FL_E_INTERNAL = 7
};

const char* fl_status_str(int status);
const char* fl_last_error(void);
int fl_abi_version(void);

/* Debugging aid: with on != 0 (or the environment variable FL_CHECK_INDICES set to a non-zero value when the
 * library is first used), every call that takes index lists first synchronizes its stream, copies the lists
 * to the host and returns FL_E_RANGE (launching nothing) if one is not strictly ascending or holds an entry
 * outside its range (rows and columns in [0, N), or [0, T) for decode).  The same switch has
 * fl_loop_sparse_attn check that every V value it reads (v_cache, and v_new when given) has magnitude
 * <= 65504, since its products with V run in fp16 (a small reduction launch, then FL_E_RANGE).  Off by
 * default; not usable under stream capture.  Process-wide. */
void fl_set_index_checks(int on);

/* ------------------------------------------------------------------------------------------------
 * (1) Token selection -- Section 4.1; Appendix D.1, Eq. 5.
 *
 * For every candidate row i of batch b the score is
 *     s_i = ||delta_i||_2 / (||cur_i||_2 + eps)        (normalize != 0)
 *     s_i = ||delta_i||_2                              (normalize == 0)
 * over the concatenation of the (k_cur, k_prev) and (v_cur, v_prev) rows, with
 * delta = fp32(cur) - fp32(prev) (fp32, round to nearest even) and both squared norms accumulated in
 * fp64; the selection key is fp32(s_i) (round to nearest even).  The active set is the k candidates
 * with the largest keys, ties broken by the lower row index, emitted in ascending row order.
 *
 *   k_cur, k_prev, v_cur, v_prev : bf16 [B, N, D] (D = H * d; rows of all heads).  v_cur and v_prev may
 *                                  both be NULL to score one pair only.  Row starts 16-byte aligned.
 *   cand     : int32 [B, n_cand] ascending candidate rows (the previous active set), or NULL for all N
 *              rows (then n_cand must equal N).
 *   k        : 0 <= k <= n_cand, else FL_E_RANGE.  n_cand <= 65536.
 *   out_key  : fp32 [B, n_cand] selection keys, in candidate order (required).
 *   out_idx  : int32 [B, k] the active rows, ascending (required when k > 0).
 *   out_slot : int32 [B, N] position of each row in out_idx, -1 for rows not selected (NULL = skip).
 *   D must be a multiple of 8.
 * ---------------------------------------------------------------------------------------------- */
int fl_select_tokens(const uint16_t* k_cur, const uint16_t* k_prev,
                     const uint16_t* v_cur, const uint16_t* v_prev,
                     int B, int N, int D,
                     const int32_t* cand, int n_cand, int k, int normalize, double eps,
                     float* out_key, int32_t* out_idx, int32_t* out_slot, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (2a) Residual quantization -- Section 4.3, Eq. 4; Appendix D.3, Eq. 8; Appendix E (asymmetric
 * group-wise quantization with scale and offset from the group min/max; keys per channel, values per
 * token).
 *
 * For packed row p < k with token i = idx[b, p]:  delta = fp32(x_cur[b,i]) - fp32(x_ref[b,i]).
 *   axis FL_AXIS_TOKEN   (keys):   a group is G consecutive packed rows x one (head, channel); the last
 *                                  group may be partial.  scale/zero: fp16 [B, ceil(k/G), H, d].
 *   axis FL_AXIS_CHANNEL (values): a group is one (row, head) x G consecutive channels (G | d).
 *                                  scale/zero: fp16 [B, k, H, d/G].
 * Per group: z = largest fp16 <= min, s = smallest fp16 >= (max - z) / (2^bits - 1) (fp64), and codes
 * q = clamp(rint(fp32(delta - z) / fp32(s)), 0, 2^bits - 1) (IEEE fp32 division, ties to even;
 * q = 0 when s == 0).  Signed zeros in z and s are stored as +0.
 * Codes: uint8 [B, k, H, d * bits / 8], packed LSB-first along channels (channel e at byte
 * e*bits/8, bit (e mod 8/bits)*bits); bits = 8 is one byte per code; bits = 16 stores the raw bf16
 * state (no quantization; scale/zero untouched and may be NULL).
 *
 *   x_cur    : bf16 [B, N, H, d] the loop-r state X^(r).
 *   x_ref    : bf16 [B, N, H, d] the previous reconstruction X_hat^(r-1), or NULL for zeros (the base).
 *   idx      : int32 [B, k] ascending active rows, or NULL for all rows (then k must equal N).
 *   bits     : 2, 4, 8 or 16.  group: 8 <= G <= 128, a multiple of 8 (and G | d on the CHANNEL axis).
 *   out_rows : optional bf16 [B, k, H, d]: also write the reconstructed rows
 *              bf16(fp32(x_ref[b,i]) + fp32(z + q*s)) (what fl_kv_residual_dequant COMPACT returns).
 *              May alias x_ref only when idx is NULL (in-place base reconstruction).
 * With k = 0 nothing is read or written, and codes, scale and zero may be NULL.
 * ---------------------------------------------------------------------------------------------- */
enum fl_axis { FL_AXIS_TOKEN = 0, FL_AXIS_CHANNEL = 1 };

int fl_kv_residual_quant(const uint16_t* x_cur, const uint16_t* x_ref, const int32_t* idx, int k,
                         int B, int N, int H, int d, int bits, int group, int axis,
                         uint8_t* codes, uint16_t* scale, uint16_t* zero, uint16_t* out_rows,
                         void* stream);

/* (2a') The same quantization with the reconstruction committed in place -- Eq. 4 and Appendix D.3,
 * Eq. 8: x_hat holds X_hat^(r-1) and is the reference; codes, scale and zero are written as by
 * fl_kv_residual_quant(x_cur, x_hat, idx, ...), and rows idx of x_hat become X_hat^(r) (what
 * fl_kv_residual_dequant FL_DQ_COMMIT would write from those codes).  One pass instead of two, for a
 * loop whose attention update reads the new state from the cache (fl_loop_sparse_attn_terms with
 * k_new = v_new = NULL).  x_hat must not be NULL; other arguments as fl_kv_residual_quant. */
int fl_kv_residual_quant_commit(const uint16_t* x_cur, uint16_t* x_hat, const int32_t* idx, int k,
                                int B, int N, int H, int d, int bits, int group, int axis,
                                uint8_t* codes, uint16_t* scale, uint16_t* zero, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (2b) Residual dequantization and reconstruction -- Eq. 4 and Appendix D.3, Eq. 8:
 *     X_hat^(r)[i] = bf16(fp32(X_hat^(r-1)[i]) + fp32(z + q * s))   for i = idx[b, p], p < k;
 * other rows keep X_hat^(r-1).  q * s is exact in fp32, so the sum is rounded once.
 *   mode FL_DQ_COMPACT : read x_hat rows, write out_rows bf16 [B, k, H, d]; x_hat is not modified.
 *   mode FL_DQ_COMMIT  : update rows idx of x_hat in place (out_rows must be NULL).
 * codes/scale/zero/bits/group/axis as produced by fl_kv_residual_quant.  idx NULL = all rows (k = N).
 * ---------------------------------------------------------------------------------------------- */
enum fl_dq_mode { FL_DQ_COMPACT = 0, FL_DQ_COMMIT = 1 };

int fl_kv_residual_dequant(const uint8_t* codes, const uint16_t* scale, const uint16_t* zero,
                           const int32_t* idx, int k, int B, int N, int H, int d,
                           int bits, int group, int axis, int mode,
                           uint16_t* x_hat, uint16_t* out_rows, void* stream);

/* (2c) Keys and values of one loop in one call -- Eq. 4 and Appendix D.3, Eq. 8 with the Appendix E
 * axes: keys on FL_AXIS_TOKEN, values on FL_AXIS_CHANNEL, one bits and group for both.  The outputs
 * are bitwise those of two fl_kv_residual_quant calls (mode FL_DQ_COMPACT) or of two
 * fl_kv_residual_quant_commit calls (mode FL_DQ_COMMIT); the two tensors share one kernel launch.
 *   k_cur, v_cur     : bf16 [B, N, H, d] loop-r keys and values.
 *   k_ref, v_ref     : bf16 [B, N, H, d] previous reconstructions (NULL for zeros in COMPACT mode);
 *                      in COMMIT mode both are required, distinct, and rows idx are updated in place.
 *   k_codes, k_scale, k_zero / v_codes, v_scale, v_zero : as fl_kv_residual_quant for each axis
 *                      (distinct code buffers).
 *   k_rows, v_rows   : COMPACT: optional bf16 [B, k, H, d] reconstructed rows (may alias the reference
 *                      only when idx is NULL).  COMMIT: must be NULL.
 * Other arguments as fl_kv_residual_quant. */
int fl_kv_residual_quant_kv(const uint16_t* k_cur, uint16_t* k_ref, const uint16_t* v_cur, uint16_t* v_ref,
                            const int32_t* idx, int k, int B, int N, int H, int d, int bits, int group,
                            uint8_t* k_codes, uint16_t* k_scale, uint16_t* k_zero,
                            uint8_t* v_codes, uint16_t* v_scale, uint16_t* v_zero,
                            uint16_t* k_rows, uint16_t* v_rows, int mode, void* stream);

/* (2c') The same with an fp16 copy of the value cache kept current -- for the attention calls of (3e).
 * COMMIT mode of (2c) (no compact rows): rows idx of k_ref and v_ref are updated in place, and rows idx of
 * v_f16 (fp16 [B, N, H, d], the value cache's copy) receive fp16(v_ref) of the updated rows, each value
 * rounded to nearest even from its bf16 value (exact for 2^-14 <= |v| <= 65504; smaller magnitudes round
 * to a multiple of 2^-24, larger ones overflow).  k_ref, v_ref and v_f16 are required and distinct.
 * Other arguments and outputs as fl_kv_residual_quant_kv with mode FL_DQ_COMMIT. */
int fl_kv_residual_quant_kv_v16(const uint16_t* k_cur, uint16_t* k_ref, const uint16_t* v_cur, uint16_t* v_ref,
                                uint16_t* v_f16, const int32_t* idx, int k, int B, int N, int H, int d, int bits,
                                int group, uint8_t* k_codes, uint16_t* k_scale, uint16_t* k_zero,
                                uint8_t* v_codes, uint16_t* v_scale, uint16_t* v_zero, void* stream);

/* (2c'') fp16 copy of rows of a bf16 tensor -- the value cache's copy for the attention calls of (3e).
 *   x     : bf16 [B, N, H, d] (d a multiple of 8);  x_f16 : fp16 [B, N, H, d], distinct from x.
 *   idx   : int32 [B, k] rows to copy (ascending, in [0, N)), or NULL with k = N for every row; k = 0
 *           copies nothing (idx may then be NULL).
 * x_f16[b, i] = fp16(x[b, i]) for the rows named, rounding as in (2c'); other rows are left unchanged.
 * Used after the calls that write the value cache without the copy (the base codec of the set-up, the
 * bf16 tail of (6), the COMMIT of (2d)). */
int fl_kv_f16_rows(const uint16_t* x, const int32_t* idx, int k, int B, int N, int H, int d, uint16_t* x_f16,
                   void* stream);

/* (2d) Reconstruction of keys and values in one call -- Eq. 4 and Appendix D.3, Eq. 8 with the axes of
 * (2c).  Bitwise the results of fl_kv_residual_dequant for the keys (FL_AXIS_TOKEN) and the values
 * (FL_AXIS_CHANNEL) with the same bits, group and mode; one kernel launch.
 *   mode FL_DQ_COMPACT : k_rows and v_rows (bf16 [B, k, H, d]) are required; k_hat, v_hat are read only.
 *   mode FL_DQ_COMMIT  : rows idx of k_hat and v_hat (distinct) are updated in place; k_rows = v_rows = NULL.
 * Other arguments as fl_kv_residual_dequant. */
int fl_kv_residual_dequant_kv(const uint8_t* k_codes, const uint16_t* k_scale, const uint16_t* k_zero,
                              const uint8_t* v_codes, const uint16_t* v_scale, const uint16_t* v_zero,
                              const int32_t* idx, int k, int B, int N, int H, int d, int bits, int group,
                              int mode, uint16_t* k_hat, uint16_t* v_hat, uint16_t* k_rows,
                              uint16_t* v_rows, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (3) Mass-corrected sparse attention update -- Sections 3.2 and 4.2, Eq. 3; Appendix D.2, Eq. 7.
 *
 * For every updated row i = rows[b, p] (p < k) and head h, over the column set
 *     S_i = ({cols[b, h, :]} U {j : i - window < j <= i}) restricted to j <= i   (a set)
 * with sigma = sm_scale:
 *   subtract (loop r-1):  pp_j = exp(sigma q_prev_i . k_cache_j - lse_ref_i),  m_i = sum pp_j,
 *                         sub = sum pp_j v_cache_j
 *   add      (loop r):    L = logsumexp_j (sigma q_cur_i . knew_j),  pc_j = m_i exp(sigma q_cur_i.knew_j - L),
 *                         add = sum pc_j vnew_j
 *   o_i <- o_i - sub + add,   lse_ref_i <- L - log(m_i)
 * where knew_j/vnew_j is row slot[b, j] of k_new/v_new when slot[b, j] >= 0 (a row updated this loop)
 * and the cache row otherwise.  Rows with an empty S_i or m_i == 0 are left unchanged; rows not in
 * `rows` are never touched.  lse_ref carries the cached column mass: exp(logit - lse_ref) reproduces
 * the cached probabilities of the previous loop.
 *
 * flags FL_ATTN_DENSE (the dense source loop): rows is NULL (every row, k = N), cols/slot/q_prev/
 *   k_new/v_new are unused, window is ignored (S_i = [0, i]); writes o_i = softmax(sigma q_i K^T) V
 *   over j <= i and lse_ref_i = its log-normaliser (inputs o/lse_ref are overwritten, not read).
 *
 *   q_cur, q_prev     : bf16 [B, N, H, d]  (queries of loop r and r-1)
 *   k_cache, v_cache  : bf16 [B, N, H, d]  X_hat^(r-1)
 *   k_new, v_new      : bf16 [B, k, H, d]  X_hat^(r) of the rows, in `rows` order (both or neither;
 *                                          neither only with term_prev, see (3b))
 *   slot              : int32 [B, N]       position in rows, or -1
 *   rows              : int32 [B, k]       ascending updated rows
 *   cols              : int32 [B, H, c_list] ascending column list (0 <= c_list <= N)
 *   window            : band width w >= 0
 *   lse_ref           : fp32 [B, N, H]     in/out
 *   o                 : fp32 [B, N, H, d]  in/out
 *   ws, ws_bytes      : workspace of at least fl_loop_sparse_attn_ws(...) bytes (may be NULL if 0).
 *                       Scratch: a prep kernel fills it with the column records of every tile on each
 *                       call (about 8 * (2 B H c_list + B (N + k)) bytes; FL_E_SHAPE above 2^31).
 * Precision.  q.k is a bf16 MFMA product with fp32 accumulation; softmax and the update are fp32.  p.v
 * depends on the path: the dense loop, the two-pass loop and the add pass over current caches in the
 * segment kernels (c_list <= 2048, with or without a band) convert the value rows to fp16 (or read them from
 * v_cache_f16) and multiply fp16 probabilities (exact conversion for
 * 2^-14 <= |v| <= 65504; smaller magnitudes round to a multiple of 2^-24; values beyond 65504 in magnitude
 * overflow to infinity and are outside the supported input range); the other add-pass paths keep values
 * in bf16 and split each probability into two bf16 parts (about 16 significant bits).
 * ---------------------------------------------------------------------------------------------- */
enum fl_attn_flags { FL_ATTN_DENSE = 1 };

size_t fl_loop_sparse_attn_ws(int B, int N, int H, int d, int k, int c_list, int window, int flags);

int fl_loop_sparse_attn(const uint16_t* q_cur, const uint16_t* q_prev,
                        const uint16_t* k_cache, const uint16_t* v_cache,
                        const uint16_t* k_new, const uint16_t* v_new,
                        const int32_t* slot, const int32_t* rows, int k,
                        const int32_t* cols, int c_list, int window,
                        int B, int N, int H, int d, float sm_scale, int flags,
                        float* lse_ref, float* o, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (3b) The same update keeping the add term for the next loop -- Appendix D.2, Eq. 7.
 *
 * After the update of loop r, lse_ref_i = L - log m_i, so the next loop's subtract term over the same
 * S_i and the same (q^(r), X_hat^(r)) is sum_j exp(sigma q^(r)_i . k_j - lse_ref_i) v_j = add, with mass
 * m_i: it equals this loop's add term in exact arithmetic, as long as the column sets stay fixed and
 * every row of loop r+1 was updated in loop r (nested selection).  This call
 *   - with term_out/mass_out: also writes add (fp32 [B, k, H, d], row p of `rows`) and m_i
 *     (fp32 [B, k, H]); rows left unchanged get 0 and 0;
 *   - with term_prev (mass_prev, slot_prev, k_prev): takes the subtract term and m_i of row i from row
 *     slot_prev[b, i] of the previous loop's term_out/mass_out (k_prev rows) instead of recomputing the
 *     subtract pass, so q_prev is unused (may be NULL).  Every row of `rows` must have
 *     slot_prev[b, i] >= 0; a row without one is left unchanged.  The kernel then runs the add pass
 *     only, with one 16-row group per wave;
 *   - with term_prev and k_new = v_new = NULL: k_cache and v_cache already hold X_hat^(r) of the updated
 *     rows (committed before this call, e.g. by fl_kv_residual_quant_commit), and every column is read
 *     from them; slot may then be NULL and no workspace is needed (no tile records are built).
 * term_prev and term_out may not alias.  Other arguments as fl_loop_sparse_attn (never DENSE).
 * ---------------------------------------------------------------------------------------------- */
int fl_loop_sparse_attn_terms(const uint16_t* q_cur, const uint16_t* q_prev,
                              const uint16_t* k_cache, const uint16_t* v_cache,
                              const uint16_t* k_new, const uint16_t* v_new,
                              const int32_t* slot, const int32_t* rows, int k,
                              const int32_t* cols, int c_list, int window,
                              int B, int N, int H, int d, float sm_scale,
                              float* lse_ref, float* o,
                              const float* term_prev, const float* mass_prev,
                              const int32_t* slot_prev, int k_prev,
                              float* term_out, float* mass_out,
                              void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (3c) The subtract pass alone -- Appendix D.2, Eq. 7 (the cached loop r-1 probabilities over S_i).
 *
 * For every updated row i = rows[b, p] and head h, over S_i as in (3):
 *   term_out[b, p, h, :] = sum_{j in S_i} exp(sigma q_prev_i . k_cache_j - lse_ref_i) v_cache_j,
 *   mass_out[b, p, h]    = sum_{j in S_i} exp(sigma q_prev_i . k_cache_j - lse_ref_i)   (m_i)
 * with the loop r-1 queries, caches and lse_ref (read only).  A loop without stored add terms can then
 * commit its new rows into the caches (fl_kv_residual_quant_commit) and run the add pass alone with
 * fl_loop_sparse_attn_terms(term_prev = term_out, mass_prev = mass_out, slot_prev = this loop's slot map,
 * k_prev = k, k_new = v_new = NULL): the same update as the two-pass fl_loop_sparse_attn, in exact
 * arithmetic.  Covers c_list <= 3072, with or without a band (fl_loop_subtract_terms_supported returns 1):
 * c_list <= 2048 (and, with a band, the segment kernel's tile table) runs the segment kernels, the others the
 * 64-row kernel with the list in LDS.  FL_E_UNSUPPORTED otherwise, with nothing launched.
 * Arrays as in (3): q_prev bf16 [B, N, H, d]; k_cache, v_cache bf16 [B, N, H, d]; rows int32 [B, k]
 * ascending; cols int32 [B, H, c_list] ascending; lse_ref fp32 [B, N, H]; term_out fp32 [B, k, H, d];
 * mass_out fp32 [B, k, H] (rows, term_out and mass_out may be NULL when k = 0: nothing to do).
 * Precision: q.k bf16 MFMA with fp32 accumulation; p.v with fp16 probabilities and values in the segment
 * kernel (the value rows are converted to fp16 as in (3), and v_cache must fit fp16), with bf16 values and
 * each probability split into two bf16 parts in the 64-row kernel.
 * ---------------------------------------------------------------------------------------------- */
int fl_loop_subtract_terms_supported(int k, int c_list, int window, int N, int d);

int fl_loop_subtract_terms(const uint16_t* q_prev, const uint16_t* k_cache, const uint16_t* v_cache,
                           const int32_t* rows, int k, const int32_t* cols, int c_list, int window,
                           int B, int N, int H, int d, float sm_scale, const float* lse_ref,
                           float* term_out, float* mass_out, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (3e) The add pass over current caches and the subtract pass, reading the values from an fp16 copy.
 * v_cache_f16 (fp16 [B, N, H, d]) must equal fp16(v_cache) row for row (kept by (2c') and (2c'')); the
 * segment kernels then load value tiles as they are instead of converting them in LDS (the same
 * rounding, so the results are bitwise those of the calls without the copy), and the other kernels
 * ignore it.  fl_loop_sparse_attn_terms_v16: fl_loop_sparse_attn_terms with q_prev, k_new, v_new and
 * slot NULL, term_prev required and no workspace (given terms over current caches build no tile
 * records).  fl_loop_subtract_terms_v16: fl_loop_subtract_terms.  Arguments otherwise as there.
 * ---------------------------------------------------------------------------------------------- */
int fl_loop_sparse_attn_terms_v16(const uint16_t* q_cur, const uint16_t* k_cache, const uint16_t* v_cache,
                                  const uint16_t* v_cache_f16, const int32_t* rows, int k, const int32_t* cols,
                                  int c_list, int window, int B, int N, int H, int d, float sm_scale,
                                  float* lse_ref, float* o, const float* term_prev, const float* mass_prev,
                                  const int32_t* slot_prev, int k_prev, float* term_out, float* mass_out,
                                  void* stream);

int fl_loop_subtract_terms_v16(const uint16_t* q_prev, const uint16_t* k_cache, const uint16_t* v_cache,
                               const uint16_t* v_cache_f16, const int32_t* rows, int k, const int32_t* cols,
                               int c_list, int window, int B, int N, int H, int d, float sm_scale,
                               const float* lse_ref, float* term_out, float* mass_out, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (3d) Which kernel an attention call launches -- for profilers that look the launch up in a trace.
 * Host-only: no device call, no argument is dereferenced.  pass: FL_PASS_ADD, the add pass over caches
 * that hold the loop's state (fl_loop_sparse_attn_terms with k_new = v_new = NULL); FL_PASS_SUBTRACT,
 * fl_loop_subtract_terms; FL_PASS_BOTH, both passes (fl_loop_sparse_attn, and loop 2 without terms).
 * Returns a static string naming the __global__ function (e.g. "seg_cur_kernel"), or NULL for a shape the
 * pass does not cover or arguments outside 1 <= k <= N, 0 <= c_list <= N, window >= 0, d in {64, 128},
 * B, H >= 1.
 * ---------------------------------------------------------------------------------------------- */
enum fl_attn_pass { FL_PASS_ADD = 0, FL_PASS_SUBTRACT = 1, FL_PASS_BOTH = 2 };

const char* fl_attn_kernel_name(int pass, int k, int c_list, int window, int B, int N, int H, int d);

/* ------------------------------------------------------------------------------------------------
 * (4) Column statistic of a dense source loop -- Appendix D.2, Eq. 6 with all causal keys and cached
 * mass 1, summed over all rows of a prefill:
 *     col_key[b, h, j] = fp32( sum_{i >= j} exp(l_ij - lse_i) ),  l_ij = sigma * sum_e q_ie k_je,
 *     lse_i = log sum_{j <= i} exp(l_ij),   sigma = 1 / sqrt(d),
 * all in fp64 (products of bf16 values are exact in fp64).
 *   q, k_cache : bf16 [B, N, H, d];  col_key : fp32 [B, H, N].
 *   ws         : at least fl_column_scores_ws(B, N, H) bytes (the fp64 row log-normalisers).
 * ---------------------------------------------------------------------------------------------- */
size_t fl_column_scores_ws(int B, int N, int H);

int fl_column_scores(const uint16_t* q, const uint16_t* k_cache, int B, int N, int H, int d,
                     float* col_key, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (5) Column list -- Appendix D.2, Eq. 6: S = {0 .. n_sink-1} U TopK_t(col_key over j >= n_sink),
 * ties broken by the lower column index, emitted ascending.
 *   col_key : fp32 [B, H, N];  cols : int32 [B, H, ns + t] with ns = min(n_sink, N);
 *   0 <= t <= N - ns, else FL_E_RANGE;  N - ns <= 65536.  An empty list (ns + t = 0) writes nothing and
 *   takes NULL pointers.
 * ---------------------------------------------------------------------------------------------- */
int fl_select_columns(const float* col_key, int B, int H, int N, int n_sink, int t,
                      int32_t* cols, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (6) Decode step of one loop for the newest position -- Appendix D.2, Eqs. 6 and 7 for one query row.
 * For each (b, h), the query of position t = T - 1 attends over the columns S selected by the previous
 * loop with their cached mass m, or over every column 0 .. T-1 with m = 1 (a dense source loop):
 *     p_j = m * exp(l_j - L),  l_j = sm_scale * q . K_j (fp64),  L = log sum_{j in S} exp(l_j),
 *     o <- o - sub + sum_{j in S} p_j V_j          (dense: o = sum_j p_j V_j),
 * then selects the next loop's S' of c_next columns: columns j < n_sink and j >= T - window first
 * (lower columns first if they alone exceed c_next), then fp32(l_j) descending, ties to the lower column,
 * emitted ascending; m' = sum_{j in S'} p_j and sub' = sum_{j in S'} p_j V_j (the next loop's subtract
 * term p_S'^(r) V_S'^(r)).
 *   q                 : bf16 [B, H, d] the query of position T - 1 at this loop.
 *   k_cache, v_cache  : bf16 [B, T, H, d] this loop's K_hat, V_hat of positions 0 .. T-1.
 *   cols, c           : int32 [B, H, c] ascending S (1 <= c <= T), with mass fp32 [B, H] and sub fp32
 *                       [B, H, d] from the loop that selected it; or cols = NULL (dense, c = 0 or T;
 *                       mass and sub unused and may be NULL).
 *   o                 : fp32 [B, H, d] the previous loop's output in (unused when dense), this loop's out.
 *   lse               : optional fp32 [B, H]: L.
 *   c_next            : 0 <= c_next <= |S| (0: no selection; the outputs below may then be NULL).
 *   cols_next         : int32 [B, H, c_next];  mass_next : fp32 [B, H];  sub_next : fp32 [B, H, d].
 *   ws                : at least fl_decode_step_ws(B, T, H, d, c, c_next) bytes (|S| <= 65536).
 * Two launches: chunked logits (with their fp32 ranking keys) and weighted V rows; then one workgroup
 * per (b, h) merges them into L and the output and forms S', m' and sub' (c_next = |S| keeps every
 * column: S' = S, m' = m and sub' is the add term just formed; otherwise a top-k and a gather of the
 * selected V rows).  Within a row p_j grows with l_j, so S' is ranked by fp32(l_j) (fp64 logits keep
 * the selection exact).
 * ---------------------------------------------------------------------------------------------- */
size_t fl_decode_step_ws(int B, int T, int H, int d, int c, int c_next);

int fl_decode_step(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                   const int32_t* cols, int c, const float* mass, const float* sub, int B, int T, int H,
                   int d, float sm_scale, float* o, float* lse, int n_sink, int window, int c_next,
                   int32_t* cols_next, float* mass_next, float* sub_next, void* ws, size_t ws_bytes,
                   void* stream);

/* (6b) The decode step without a workspace argument, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  Arguments and
 * results are those of fl_decode_step; the workspace is a library-owned device array of
 * FL_DECODE_SCRATCH_BYTES per GPU (allocated with the code object when the library is loaded on that
 * GPU, held until the process ends).  The call itself allocates and frees nothing.
 *   - FL_E_RANGE when fl_decode_step_ws(B, T, H, d, c, c_next) exceeds FL_DECODE_SCRATCH_BYTES (32 MiB:
 *     about 1.9 million (batch, head, position) entries in a dense loop, e.g. B = 1, H = 16, T = 64K).
 *   - Every call on one GPU shares that GPU's array: calls that overlap on one GPU (two streams, two
 *     threads) race on it and must be ordered by the caller.  Nothing in the array needs clearing between
 *     calls; the last call's contents stay there.
 *   - The first call on a device looks up that device's copy of the array (hipGetSymbolAddress); the
 *     current device must be the one `stream` belongs to. */
#define FL_DECODE_SCRATCH_BYTES (32u << 20)

int fl_decode_step_noalloc(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                           const int32_t* cols, int c, const float* mass, const float* sub, int B, int T, int H,
                           int d, float sm_scale, float* o, float* lse, int n_sink, int window, int c_next,
                           int32_t* cols_next, float* mass_next, float* sub_next, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (7) Pruning the column list for a smaller budget -- Section 4.2 (later loops with smaller budgets
 * prune the selected set by the preceding sparse loop's attention statistics) and Appendix D.2, Eq. 6
 * with a sparse source.  After loop r has updated the rows A, for each (b, h) and each list entry
 * j = cols[b, h, e], e >= ns (ns = min(n_sink, c_list)):
 *     col_key[b, h, e - ns] = fp32( sum_{i in A, i >= j} exp(sm_scale * q_i . k_j - lse_ref_i) )   (fp64)
 * the probability mass loop r gives column j, summed over the updated rows that attend to it, each row's
 * probabilities recovered from its reference log-normaliser (the cached mass is folded into lse_ref).
 * cols_next keeps the ns sinks and the t_next entries with the largest keys (ties to the lower column),
 * ascending: a subset of cols.  The band is not pruned.  A following two-pass loop over cols_next
 * subtracts the kept probabilities with the same lse_ref, so their mass m' needs no separate output.
 *   q, k_cache : bf16 [B, N, H, d] loop r's queries and K_hat (rows A and the list columns are read).
 *   rows, k    : int32 [B, k] ascending updated rows of loop r (NULL allowed when k = 0).
 *   cols       : int32 [B, H, c_list] ascending, 1 <= c_list <= N, whose first ns entries are the sinks
 *                0 .. ns-1 (as fl_select_columns and this call emit them).
 *   lse_ref    : fp32 [B, N, H] after loop r (read at the rows A).
 *   col_key    : fp32 [B, H, c_list - ns] out (may be NULL when c_list == ns);  c_list - ns <= 65536.
 *   cols_next  : int32 [B, H, ns + t_next] out, 0 <= t_next <= c_list - ns.
 *   ws         : at least fl_prune_columns_ws(B, H, k, c_list, n_sink) bytes (fp64 partial sums of
 *                256-row chunks; H * ceil(k / 256) <= 65535).
 * Three launches: the fp64 statistic per 256-row chunk of updated rows (dot products on fp64 matrix
 * instructions, 16 list entries per wave against query rows staged in LDS), the ordered sum of the chunks,
 * and the top-k.
 * ---------------------------------------------------------------------------------------------- */
size_t fl_prune_columns_ws(int B, int H, int k, int c_list, int n_sink);

int fl_prune_columns(const uint16_t* q, const uint16_t* k_cache, const int32_t* rows, int k,
                     const int32_t* cols, int c_list, const float* lse_ref, int B, int N, int H, int d,
                     double sm_scale, int n_sink, int t_next, float* col_key, int32_t* cols_next,
                     void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------------------------------
 * (8) Recent tokens kept in bf16 -- Appendix E (the most recent 64 tokens stay in BF16).  For every active
 * row i = idx[b, p] (or every row when idx == NULL) with i >= N - tail, the stored row becomes the exact
 * input row:  cache[b, i] = x_cur[b, i]  and/or  rows[b, p] = x_cur[b, i].  The rows are still encoded
 * with the others by the codec calls; this call replaces what the state stores for them, after those calls.
 *   x_cur       : bf16 [B, N, H, d], d a positive multiple of 8 (16-byte aligned rows).
 *   idx, k      : int32 [B, k] ascending active rows (NULL: every row, k = N).
 *   cache       : bf16 [B, N, H, d] or NULL;  rows : bf16 [B, k, H, d] compact rows or NULL (not both NULL).
 *   tail = 0 does nothing.  One launch over the last min(k, tail) entries of idx.
 * ---------------------------------------------------------------------------------------------- */
int fl_kv_keep_recent(const uint16_t* x_cur, const int32_t* idx, int k, int B, int N, int H, int d, int tail,
                      uint16_t* cache, uint16_t* rows, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FLASHLOOP_H */
