/*
 * fold.h - C ABI of the FoldAttention decode hot path for MI355X (gfx950).
 *
 * Declared-reference softmax attention over a BF16 KV cache (FoldAttention,
 * arXiv 2609.33410).  For query row i a finite reference Z_i is fixed before
 * any key is read (Section 3, Eq. fold).  Every weight 2^(s_ij - Z_i) is then
 * final when computed, so a scan over any key subset yields an FP32 pair
 *     A_i = sum_{live j} 2^(s_ij - Z_i) v_j,   L_i = sum_{j} 2^(s_ij - Z_i)
 * and pairs from disjoint key ranges (split-KV slots, cascade levels) are
 * combined by plain addition, o_i = sum A_i / sum L_i (Proposition 1; Section
 * 4; Algorithm 1).  A per-call depth T cuts keys with s_ij - Z_i < -T from A
 * while their weight stays in L (Section 4, "Depth as a dial").
 *
 * Scores are base 2: s_ij = log2(e) * sm_scale * (q_i . k_j) (Section 2),
 * with sm_scale in natural-log units (1/sqrt(D) for standard attention).
 *
 * Conventions shared by every call:
 *   - Every pointer except the view structs themselves and fold_debug is a
 *     DEVICE pointer owned by the caller.  The library keeps no pointer after
 *     a call returns, allocates nothing, and never synchronises: work is
 *     enqueued on `stream` (a hipStream_t; NULL = the default stream).
 *   - Arguments are validated on the host before anything is launched.  A
 *     failed check returns FOLD_E_INVAL (or FOLD_E_UNSUPPORTED) and launches
 *     nothing; fold_last_error() then returns a thread-local message.  A launch
 *     failure returns FOLD_E_HIP.  No C++ exception crosses this boundary.
 *   - BF16 arrays hold raw bfloat16 bit patterns; q, k and v must be 16-byte
 *     aligned.
 *   - Device-side bounds: a kv sequence's length is clamped to what its view
 *     can address (max_seq_len, or max_pages_per_seq * page_size); a page id
 *     outside [0, num_pages) and a row request outside [0, batch) are skipped
 *     (they contribute nothing and are never dereferenced).
 *   - Results are deterministic: every sum has a fixed order.  The
 *     three-call path uses no atomics; the one-launch decodes count split
 *     arrivals with one atomic add per workgroup, and the split that counts
 *     last adds the slots in slot order, so arrival order never changes a
 *     bit of the result.
 */
#ifndef FOLD_H
#define FOLD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FOLD_ABI_VERSION 2

typedef enum fold_status {
  FOLD_OK = 0,
  FOLD_E_INVAL = 1,       /* an argument failed validation; nothing launched */
  FOLD_E_UNSUPPORTED = 2, /* a valid request this build does not implement */
  FOLD_E_HIP = 3          /* the HIP runtime reported a launch error */
} fold_status;

typedef enum fold_dtype { FOLD_DTYPE_F32 = 0, FOLD_DTYPE_BF16 = 1 } fold_dtype;

/*
 * One scan level's view of the KV cache (Section 4: paged cache with a
 * per-request block table; value-product paragraph: a shared prefix is one
 * kv sequence attended by the stacked query rows of every request holding it).
 *
 * Paged (block_table != NULL): k and v are [num_pages][num_kv_heads]
 *   [page_size][head_dim] bf16; key j of kv sequence s, head g, lives at page
 *   block_table[s * max_pages_per_seq + j / page_size], slot j % page_size.
 *   page_size must be a positive multiple of 16.
 * Contiguous (block_table == NULL): k and v are [num_seqs][num_kv_heads]
 *   [max_seq_len][head_dim] bf16.
 * seq_lens [num_seqs] int32 (device): keys per kv sequence.
 * Rows: with row_indptr == row_req == NULL, kv sequence s is attended by
 *   request s (num_seqs <= batch).  Otherwise kv sequence s is attended by the
 *   requests row_req[row_indptr[s] .. row_indptr[s+1]) (CSR, device arrays),
 *   and max_reqs_per_seq bounds row_indptr[s+1] - row_indptr[s] on the host.
 * Query head h reads kv head h / (num_heads / num_kv_heads).
 */
typedef struct fold_kv_view {
  const void* k;
  const void* v;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const int32_t* row_indptr;
  const int32_t* row_req;
  int32_t num_seqs;
  int32_t num_kv_heads;
  int32_t head_dim;          /* 64 or 128 */
  int32_t page_size;         /* ignored when contiguous */
  int32_t max_pages_per_seq; /* row stride of block_table */
  int32_t num_pages;         /* pages in k / v (paged) */
  int32_t max_seq_len;       /* host bound on seq_lens; contiguous row stride */
  int32_t max_reqs_per_seq;  /* host bound for CSR rows; ignored otherwise */
} fold_kv_view;

/* Query rows: q is [batch][num_heads][head_dim] bf16; row i = r * num_heads + h. */
typedef struct fold_q_view {
  const void* q;
  int32_t batch;
  int32_t num_heads;
} fold_q_view;

/* Estimator constants (Section 3, "Choosing the reference"): the first `sink`
 * keys and the last `recent` keys are scored exactly; the keys in between are
 * cut into `strata` contiguous strata represented by their centres, whose
 * weights are sorted and trimmed by `trim_lo` / `trim_hi` before their mean
 * stands for the whole middle range.  Rows of at most sink+recent+strata keys
 * get their exact log-sum-exp.  NULL selects {1, 63, 128, 8, 8}. */
typedef struct fold_est_params {
  int32_t sink;
  int32_t recent;
  int32_t strata;
  int32_t trim_lo;
  int32_t trim_hi;
} fold_est_params;

/* Optional exports of exactly the values the scan compared (not timed).
 * x_out [batch][num_heads][max_seq_len] fp32: x_ij = s_ij - Z_i.
 * key_gate_out [num_seqs][num_kv_heads][row_groups][max_seq_len] u8: 1 if the
 *   value row was read (some row of the read group is live on key j).
 * page_gate_out [num_seqs][num_kv_heads][row_groups][ceil(max_seq_len/16)] u8:
 *   1 if any key of the 16-key page was read.
 * A call with exports reads exactly these value rows.  Without exports, the
 * scan of read groups of 64 rows (more than 32 rows on one kv sequence, a
 * latency-bound contraction) fetches every value row with its key and applies
 * the same verdicts to the weights: the results are the same bits.
 * row_groups = fold_decode_row_groups(kv, q).  The rows attending one
 * (kv sequence s, kv head g) are numbered rho = c * G + (h mod G), where c is
 * the position of the row's request in the sequence's row list (0 without CSR
 * rows) and G = num_heads / num_kv_heads; read group u holds the rows
 * rho in [u * R, (u + 1) * R) with R = fold_decode_rows_per_group(kv, q).
 * Entries of read groups that hold no row are left unwritten.  Any pointer
 * may be NULL. */
typedef struct fold_debug {
  float* x_out;
  uint8_t* key_gate_out;
  uint8_t* page_gate_out;
} fold_debug;

/* Cut-key value model (Section 4, "Depth as a dial"): at a finite depth the
 * keys cut from row i's A are modelled by the mean value row of row i's
 * request and kv head.  Their summed weight, the cut mass (an extra output
 * of the scans, one FP32 per slot and row), multiplies that mean in
 * fold_combine: a virtual row whose weight is the cut mass.  The term is
 * linear in the cut mass, so it is the same added per slot or after the slot
 * sum, and pairs stay additive.
 *   part_Lcut [num_slots][num_rows] fp32: the scans' cut masses
 *   mean      [batch][num_kv_heads][head_dim] fp32: request means
 *             (fold_value_mean, fold_value_mean_append)
 *   rows are [batch][num_heads]; row r * num_heads + h uses
 *   mean[r][h / (num_heads / num_kv_heads)]. */
typedef struct fold_value_model {
  const float* part_Lcut;
  const float* mean;
  int32_t num_heads;
  int32_t num_kv_heads;
} fold_value_model;

/* FOLD_ABI_VERSION of the built library. */
int fold_abi_version(void);

/* Static text for a status code. */
const char* fold_status_string(fold_status s);

/* Thread-local message describing the last failed call on this thread. */
const char* fold_last_error(void);

/* Rows per read group and number of read groups per (kv sequence, kv head)
 * that fold_decode_split uses for this view (the group over which read
 * verdicts are ORed, Section 4 "Weight-gated reads"): 1 when one row attends
 * a (kv sequence, kv head), 16 for up to 16 rows, 32 for up to 32, and 64 above
 * that (stacked rows, Appendix E).  Returns -1 on an invalid view. */
int32_t fold_decode_rows_per_group(const fold_kv_view* kv, const fold_q_view* q);
int32_t fold_decode_row_groups(const fold_kv_view* kv, const fold_q_view* q);

/*
 * fold_ref_estimate - per-row finite reference Z_i (Section 3, "Choosing the
 * reference"): a base-2 log-sum-exp estimate from the sink, the most recent
 * keys and trimmed stratified centres, with no state carried between calls.
 *   kv      per-request view (row_indptr must be NULL; a cascade passes its
 *           flat prefix ++ suffix tables)
 *   q       query rows
 *   z_out   [batch][num_heads] fp32 (device).  Requests r >= num_seqs and
 *           rows of empty sequences get Z = 0.
 */
fold_status fold_ref_estimate(const fold_kv_view* kv, const fold_q_view* q, float sm_scale,
                              const fold_est_params* params, float* z_out, void* stream);

/*
 * fold_decode_split - gated split-KV scan of one level (Section 4; Algorithm 1).
 * Split s of num_splits walks the 64-key tiles t with t mod num_splits == s,
 * reads every key row, scores it against the fixed Z_i, ORs the live verdicts
 * over the read group, reads only live value rows, and writes its FP32 pair to
 * slot slot_offset + s:
 *   part_A [num_slots][batch][num_heads][head_dim] fp32,
 *   part_L [num_slots][batch][num_heads] fp32.
 * A split with no keys writes zeros.  Only the rows this view covers are
 * written.
 *   z        [batch][num_heads] fp32, the declared references
 *   depth_T  +INFINITY for dense decode, else a finite T >= 0 (NaN or negative
 *            is FOLD_E_INVAL); a key is live for row i iff x_ij >= -T
 *   part_Lcut [num_slots][batch][num_heads] fp32 or NULL: the cut mass of
 *            each written slot and row (the summed weights of keys with
 *            x_ij < -T; 0 at T = inf), for the cut-key value model
 *   dbg      NULL, or the optional exports above
 */
fold_status fold_decode_split(const fold_kv_view* kv, const fold_q_view* q, float sm_scale,
                              const float* z, float depth_T, int32_t num_splits,
                              int32_t slot_offset, int32_t num_slots, float* part_A,
                              float* part_L, float* part_Lcut, const fold_debug* dbg,
                              void* stream);

/*
 * fold_decode_cascade - both levels of a shared-prefix cascade in one scan
 * launch (Section 4, "Value product": pairs add, so a prefix decoded once with
 * the rows of its requests stacked and each request's own suffix may share a
 * slot; Appendix E).
 *   prefix   CSR view whose kv sequences carry more than 32 stacked rows each
 *            (fold_decode_rows_per_group == 64)
 *   suffix   per-request view (row_indptr NULL, num_seqs == q->batch) of the
 *            requests' own keys in the same k / v pages: same k, v,
 *            num_kv_heads, head_dim, page_size and num_pages, both paged
 * Split s walks the prefix tiles t with t mod num_splits == s, as
 * fold_decode_split does, and then the suffix tiles that fall to it.  For a
 * read group of 64 stacked rows (rows 64 g .. 64 g + 63 of a prefix kv
 * sequence and kv head), the requests those rows belong to take positions
 * p = 0, 1, ... in row order; suffix tile u (keys 64 u .. 64 u + 63) of the
 * request at position p is pair p * U + u, U = ceil(suffix->max_seq_len / 64),
 * and goes to split (p * U + u) mod num_splits, weighed for that request's
 * rows only.  Slot slot_offset + s holds the prefix split's pair plus the
 * pairs of those suffix tiles, so fold_combine over the num_splits slots
 * finishes the decode.  A split with no keys writes zeros.
 *   z ... part_Lcut  as fold_decode_split (no debug exports)
 * FOLD_E_UNSUPPORTED when the prefix is not a stacked level, the two views do
 * not share their cache arrays and layout, or one workgroup would own more
 * than 64 tiles (prefix tiles of its split plus its suffix tiles: raise
 * num_splits).
 */
fold_status fold_decode_cascade(const fold_kv_view* prefix, const fold_kv_view* suffix,
                                const fold_q_view* q, float sm_scale, const float* z,
                                float depth_T, int32_t num_splits, int32_t slot_offset,
                                int32_t num_slots, float* part_A, float* part_L,
                                float* part_Lcut, void* stream);

/*
 * fold_combine - additive combine (Algorithm 1, last step; Section 4): for
 * each row, sum the slots in increasing slot order and take the quotient
 * o = sum A / sum L.  No maximum is compared and nothing is rescaled.
 *   part_A [num_slots][num_rows][head_dim], part_L [num_slots][num_rows] fp32
 *   out     [num_rows][head_dim], fp32 or bf16 (round to nearest even)
 *   z       [num_rows] fp32; needed only when lse_out is requested
 *   lse_out [num_rows] fp32 or NULL: base-2 log-sum-exp Z + log2(sum L)
 *   cert_out [num_rows] u8 or NULL: range certificate of Section 3,
 *            bit0 sum L < 2^-1, bit1 sum L > 2^100, bit2 a non-finite output
 *   model    NULL, or the cut-key value model: o = (sum A + (sum Lcut) mean) / sum L
 *            (num_rows must equal batch * num_heads of the model's rows)
 */
fold_status fold_combine(const float* part_A, const float* part_L, int32_t num_slots,
                         int32_t num_rows, int32_t head_dim, const float* z, void* out,
                         fold_dtype out_dtype, float* lse_out, uint8_t* cert_out,
                         const fold_value_model* model, void* stream);

/*
 * fold_decode_fused - the whole decode of a single level in one launch:
 * fold_ref_estimate, fold_decode_split over splits [0, num_splits) and
 * fold_combine, with the same bits in z_out, out, lse_out and cert_out
 * (Section 3, "Choosing the reference"; Section 4; Algorithm 1).  Every
 * (request, kv head, split) workgroup computes its group's references Z_i
 * while its first keys load, scans its tiles, writes its slot, and the split
 * that finishes last adds the slots in increasing order into the output.
 *   kv, q, sm_scale, params  as fold_ref_estimate: a per-request view
 *           (row_indptr NULL, num_seqs == batch) whose kv heads each serve
 *           2 to 8 query rows (GQA); other group sizes are FOLD_E_UNSUPPORTED
 *           (use the three calls)
 *   depth_T, num_splits      as fold_decode_split
 *   part_A  [num_splits][batch][num_heads][head_dim] fp32 (under 2 GiB),
 *           part_L [num_splits][batch][num_heads] fp32: workspace for the
 *           slots (their contents after the call are those of fold_decode_split)
 *   arrivals [num_seqs][num_kv_heads] int32 (device): must be zero before the
 *           first call; every call leaves it zero.  Calls that share it or
 *           the slots must not run concurrently.
 *   z_out   [batch][num_heads] fp32: the references, as fold_ref_estimate
 *   out, out_dtype, lse_out, cert_out  as fold_combine (no value model);
 *           part_A and out must be 16-byte aligned.
 */
fold_status fold_decode_fused(const fold_kv_view* kv, const fold_q_view* q, float sm_scale,
                              const fold_est_params* params, float depth_T, int32_t num_splits,
                              float* part_A, float* part_L, int32_t* arrivals, float* z_out,
                              void* out, fold_dtype out_dtype, float* lse_out,
                              uint8_t* cert_out, void* stream);

/*
 * fold_decode_fused_noalloc - fold_decode_fused for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  The slots and arrival counts live in a
 * fixed scratch array inside the library (8 MiB per GPU, held from the first
 * call on that GPU until the process ends); the call allocates nothing and
 * takes no workspace argument.
 *   kv, q, sm_scale, params, depth_T, num_splits, z_out, out, out_dtype,
 *   lse_out, cert_out  as fold_decode_fused (same validation, same results,
 *           bit for bit: the same kernel).
 *   Scratch: num_splits*batch*num_heads*(head_dim + 1)*4 bytes of slots plus
 *           num_seqs*num_kv_heads*4 bytes of counts (each rounded up to 256
 *           bytes) must fit in 8 MiB, else FOLD_E_INVAL and nothing is
 *           launched (e.g. 16 splits x 8 requests x 32 heads at head_dim 128
 *           use 2.1 MB).  The counts are cleared by a small fill kernel on
 *           `stream` before the decode, so each call starts from zero.
 *   Concurrency: every call on one GPU uses that GPU's one scratch array, and
 *           it keeps the last call's contents; calls that overlap on one GPU
 *           (other streams, other host threads) race and must be serialised
 *           by the caller.
 *   The first call on a GPU looks up the scratch address (no allocation, no
 *           synchronisation); FOLD_E_HIP if that lookup fails.
 */
fold_status fold_decode_fused_noalloc(const fold_kv_view* kv, const fold_q_view* q,
                                      float sm_scale, const fold_est_params* params,
                                      float depth_T, int32_t num_splits, float* z_out, void* out,
                                      fold_dtype out_dtype, float* lse_out, uint8_t* cert_out,
                                      void* stream);

/*
 * fold_value_mean - request mean value rows (the running mean of Section 4's
 * value model): mean_out[s][g] = mean of value rows 0..n_s-1 of kv sequence
 * s, head g (0 for an empty sequence), FP32 sums in a fixed order.
 *   kv        per-request view (kv->v read; kv->k not read; no CSR rows)
 *   mean_out  [num_seqs][num_kv_heads][head_dim] fp32
 */
fold_status fold_value_mean(const fold_kv_view* kv, float* mean_out, void* stream);

/*
 * fold_value_mean_append - running update of the request means for appended
 * tokens: mean[s][g] += (v - mean[s][g]) / (pos + 1) for a token of kv
 * sequence s at position pos (its new length is pos + 1).
 *   kv        layout of the means (num_seqs, num_kv_heads, head_dim)
 *   v_src     [n_tok][num_kv_heads][head_dim] bf16, the tokens' value rows
 *   tok_seq, tok_pos [n_tok] int32; a token with an unknown sequence or a
 *             negative position is skipped.  At most one token per sequence
 *             per call (two would race).
 */
fold_status fold_value_mean_append(const fold_kv_view* kv, const void* v_src,
                                   const int32_t* tok_seq, const int32_t* tok_pos,
                                   int32_t n_tok, float* mean, void* stream);

/*
 * fold_value_block_mean - block means of the block model of BF16 values
 * (Section 4, "Depth as a dial"): mean_out[s][g][t] = mean of value rows
 * 64 t .. min(64 t + 64, n_s) - 1 of kv sequence s, head g, FP32 sums in key
 * order; blocks t >= ceil(n_s / 64) get zeros.  A key on a page id outside
 * [0, num_pages) adds zeros to its block's sum.
 *   kv          any view (kv->v read; kv->k and the row lists not read)
 *   max_blocks  row stride of mean_out in blocks, >= ceil(max_seq_len / 64)
 *   mean_out    [num_seqs][num_kv_heads][max_blocks][head_dim] fp32, 16-byte
 *               aligned
 */
fold_status fold_value_block_mean(const fold_kv_view* kv, int32_t max_blocks, float* mean_out,
                                  void* stream);

/*
 * fold_value_block_mean_append - running update of the block means for
 * appended tokens: for a token of kv sequence s at position pos,
 * mean[s][g][pos / 64] += (v - mean[s][g][pos / 64]) / (pos mod 64 + 1), so a
 * block's mean stays the mean of the keys it holds.
 *   kv, max_blocks, mean  as fold_value_block_mean (kv gives the layout)
 *   v_src, tok_seq, tok_pos, n_tok  as fold_value_mean_append; a token with
 *               pos / 64 >= max_blocks is skipped.  At most one token per
 *               sequence per call.
 */
fold_status fold_value_block_mean_append(const fold_kv_view* kv, int32_t max_blocks,
                                         const void* v_src, const int32_t* tok_seq,
                                         const int32_t* tok_pos, int32_t n_tok, float* mean,
                                         void* stream);

/* Block model of BF16 values for fold_decode_split_blocks.
 *   block_mean  [num_seqs][num_kv_heads][max_blocks][head_dim] fp32 block means
 *               of the view's kv sequences (fold_value_block_mean), 16-byte
 *               aligned
 *   max_blocks  >= ceil(max_seq_len / 64)
 *   chunk_cut   [batch][num_heads][ceil(max_seq_len / 16)] fp32 workspace: the
 *               scan writes each row's cut mass of every 16-key chunk of its
 *               kv sequence there (finite depth; not read at T = inf, may be
 *               NULL then).  Entries of chunks past a sequence's end and of
 *               rows the view does not cover are left unwritten. */
typedef struct fold_block_model {
  const float* block_mean;
  int32_t max_blocks;
  float* chunk_cut;
} fold_block_model;

/*
 * fold_decode_split_blocks - fold_decode_split with the block model of BF16
 * values (Section 4, "Depth as a dial"; Algorithm 1, the tile's virtual row):
 * the cut keys of 64-key block t of (kv sequence s, kv head g) are modelled
 * by the block's mean value row mu_t.  One virtual row per tile, whose weight
 * is row i's summed weight of the tile's cut keys c_it, adds c_it mu_t to the
 * A of the split that owns the tile:
 *     A_i^s = sum_{live j in split s} w_ij v_j + sum_{tiles t of split s} c_it mu_t.
 * L is fold_decode_split's (it holds every weight), so pairs stay additive
 * and fold_combine (without its request-mean model) finishes the decode.
 * At T = inf no key is cut and the call is fold_decode_split.  The scan
 * writes the cut masses per 16-key chunk, then a second kernel adds the
 * virtual rows into the slots (both on `stream`).
 *   kv ... num_slots, part_A, part_L  as fold_decode_split
 *   model    the block means and the chunk workspace (required)
 *   dbg      NULL, or the optional exports of fold_decode_split
 */
fold_status fold_decode_split_blocks(const fold_kv_view* kv, const fold_q_view* q,
                                     float sm_scale, const float* z, float depth_T,
                                     int32_t num_splits, int32_t slot_offset, int32_t num_slots,
                                     float* part_A, float* part_L,
                                     const fold_block_model* model, const fold_debug* dbg,
                                     void* stream);

/*
 * fold_append_kv - cache append (Section 4, "Weight-gated reads": the front
 * appends each step's new token): token t's key and value rows are stored at
 * position tok_pos[t] of kv sequence tok_seq[t].
 *   kv       layout of the destination cache (block table, page size, sizes;
 *            kv->k, kv->v, seq_lens and the row lists are not read)
 *   k_src, v_src [n_tok][num_kv_heads][head_dim] bf16, 16-byte aligned
 *   tok_seq, tok_pos [n_tok] int32 (device).  A token whose sequence or
 *            position the view cannot address, or whose page id is outside
 *            [0, num_pages), is skipped.
 *   k_cache, v_cache  the arrays written, in the view's element layout
 *            (16-byte aligned); either may be NULL (that side is not written)
 * Two tokens with the same destination race.  The caller extends seq_lens.
 */
fold_status fold_append_kv(const fold_kv_view* kv, const void* k_src, const void* v_src,
                           const int32_t* tok_seq, const int32_t* tok_pos, int32_t n_tok,
                           void* k_cache, void* v_cache, void* stream);

/*
 * fold_cert_update - references of the certificate's rerun (Section 3,
 * certificate paragraph: a row outside the window is decoded again with Z
 * set to its base-2 log-sum-exp).  For every row with nonzero cert bits
 * (fold_combine's cert_out): z = lse where lse is finite; z - 64 where
 * lse = -inf (sum L was 0); z + 64 where lse = +inf; a NaN lse keeps z.
 *   cert [num_rows] u8, lse [num_rows] fp32 (fold_combine's outputs, the
 *            latter computed with the same z)
 *   z        [num_rows] fp32, updated in place
 *   reruns   [num_rows] int32 or NULL: incremented for flagged rows
 *   count_out [1] int32 (device): the number of flagged rows
 * One workgroup.  The caller reads count_out (a synchronisation of its own)
 * and, if it is nonzero, decodes and combines again with the updated z;
 * rows that were not flagged keep their z and reproduce their output bit
 * for bit.
 */
fold_status fold_cert_update(const uint8_t* cert, const float* lse, float* z, int32_t num_rows,
                             int32_t* reruns, int32_t* count_out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FOLD_H */
