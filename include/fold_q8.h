/*
 * fold_q8.h - two-plane INT8 key cache for the FoldAttention decode path on
 * MI355X (gfx950): the cache writer, the per-step query split, the reference
 * estimate from coarse logits, and the gated scan (Section 4, "Cache format",
 * "Weight-gated reads", "Value product"; Algorithm 1 with BF16 values).
 *
 * Rotation.  Keys and queries are multiplied by the Sylvester Hadamard matrix
 * H_D (entries +-1, H H^T = D I).  The paper rotates by the orthonormal
 * H_D / sqrt(D); the factor 1/D that this leaves on a rotated dot product is
 * folded into the query scale, so scores are unchanged.
 *
 * Codes.  A rotated key k'' = e (a + b/256): INT8 planes a, b and one BF16
 * scale e per key, e the smallest BF16 value >= max|k''| / 127 (rounded up,
 * so plane A never saturates); a = rint(k''/e) and b = rint(256 (k''/e - a))
 * clamped to [-128, 127] (rint rounds half to even).  A key whose scale would
 * fall below 2^-126 is stored as zero.  A key's code depends on that key
 * alone.  A rotated query q'' = f (qa + qb/256) the same way with
 * f = max|q''| / 127 (FP64), and the row's base-2 score scale
 * eta = log2(e) sm_scale f / D rounded once to FP32.  The rotation and the
 * codes are computed in FP64; the rotated values are exact for inputs whose
 * nonzero magnitudes span at most 38 binades, so the codes are reproducible.
 *
 * Scan (per call depth T, per request refine threshold tau_r):
 *   coarse  xc_ij = eta_i e_j (a_j . qa_i + (a_j . qb_i) / 256) - Z_i   (FP32)
 *   gates   per GQA group (the rows of one request that share a kv head):
 *           live_j = OR_i [xc_ij >= -T] (T = inf: every key),
 *           refine_j = live_j AND OR_i [xc_ij >= -tau_r]
 *   refine  x_ij = xc_ij + [refine_j] eta_i e_j (b_j . qa_i + (b_j . qb_i) / 256) / 256
 *   fold    w = 2^x_ij; A_i += w v_j for keys with x_ij >= -T; L_i += w for
 *           every key (cut keys keep their mass)
 * Plane B is read only for keys refined by some group of the read group and
 * value rows only for live keys.  Bytes per key at D = 128: 128 (plane A) +
 * 2 (scale) + 128 r_K (plane B, refined fraction r_K) + 256 lambda (values,
 * live fraction lambda).  The partial pairs are those of fold_decode_split
 * (same slot layout); fold_combine adds them.
 *
 * Layouts.  plane_a and plane_b use the element layout of a BF16 key cache
 * (include/fold.h, fold_kv_view) with one byte per element; scale uses it
 * with one BF16 element per key ([num_pages][Hkv][page_size], or
 * [num_seqs][Hkv][max_seq_len] for a contiguous view).  Query planes are
 * [batch][num_heads][2][head_dim] int8 (qa then qb); eta [batch][num_heads]
 * fp32; tau [batch] fp32.  All pointers are device pointers owned by the
 * caller.  The conventions of include/fold.h hold for every call here (no
 * allocation, no synchronisation, host-side validation, status codes).
 */
#ifndef FOLD_Q8_H
#define FOLD_Q8_H

#include "fold.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct fold_q8_keys {
  const int8_t* plane_a;  /* 16-byte aligned */
  const int8_t* plane_b;  /* 16-byte aligned */
  const uint16_t* scale;  /* BF16 bits, 16-byte aligned */
} fold_q8_keys;

typedef struct fold_q8_query {
  const int8_t* planes;  /* [batch][num_heads][2][head_dim], 16-byte aligned */
  const float* eta;      /* [batch][num_heads] */
  const float* tau;      /* [batch]; read by fold_q8_decode_split only */
  int32_t batch;
  int32_t num_heads;
  const float* tau_v;    /* [batch] refine-V thresholds; read with 8-bit values only */
} fold_q8_query;

/* 8-bit values (Section 4, "Cache format"): two E4M3 planes under one
 * power-of-two scale 2^scale_exp for the cache.  E4M3 is the OCP E4M3FN
 * format (bias 7, largest finite 448).  Value row v is stored as
 * p = E4M3(v 2^-e) and r = E4M3(16 (v 2^-e - p)), both rounded to nearest
 * even and saturating at 448, and stands for 2^e (p + r/16); for BF16 values
 * with 2^-6 <= |v 2^-e| <= 448 that is v exactly.  Layout: the element layout
 * of the BF16 value cache, one byte per element, 16-byte aligned.  The scan
 * reads p for live keys and r only for keys whose refine-V verdict is set:
 * refine_v_j = live_j AND OR over the GQA group of [xc_ij >= -tau_v_r]
 * (Algorithm 1's third verdict bit), tau_v_r = kappa_v + ceil(log2 n_r). */
typedef struct fold_v8_values {
  const uint8_t* plane_p;
  const uint8_t* plane_r;
  int32_t scale_exp;
} fold_v8_values;

/* Optional exports of exactly the values the scan compared (not timed); the
 * shapes and the read-group numbering are those of fold_debug.
 * x_out, xc_out [batch][num_heads][max_seq_len] fp32: refined and coarse x.
 * key_gate_out / page_gate_out: value rows / 16-key pages read.
 * refine_gate_out [num_seqs][num_kv_heads][row_groups][max_seq_len] u8:
 *   plane-B rows read.  refine_v_gate_out, same shape: second value plane
 *   rows read (8-bit values). */
typedef struct fold_q8_debug {
  float* x_out;
  float* xc_out;
  uint8_t* key_gate_out;
  uint8_t* page_gate_out;
  uint8_t* refine_gate_out;
  uint8_t* refine_v_gate_out;
} fold_q8_debug;

/*
 * fold_q8_write_keys - cache writer (Section 4, "Cache format"; Appendix E,
 * cache construction): rotates and splits n_tok BF16 keys and stores their
 * codes.  Used for a prompt (every position) and for the per-step append.
 *   kv       layout of the destination cache (block table, page size, sizes;
 *            kv->k, kv->v, seq_lens and the row lists are not read)
 *   k_src    [n_tok][num_kv_heads][head_dim] bf16, in the model's basis
 *   tok_seq, tok_pos [n_tok] int32: kv sequence and position of each token.
 *            A token whose sequence or position the view cannot address, or
 *            whose page id is outside [0, num_pages), is skipped.
 *   plane_a, plane_b, scale: the cache arrays written.
 * Two tokens with the same destination race (the last write is unspecified).
 */
fold_status fold_q8_write_keys(const fold_kv_view* kv, const void* k_src, const int32_t* tok_seq,
                               const int32_t* tok_pos, int32_t n_tok, int8_t* plane_a,
                               int8_t* plane_b, uint16_t* scale, void* stream);

/*
 * fold_q8_split_query - per-step query split (Section 4, "Cache format": the
 * query is split the same way each step) and the refine thresholds
 * (Section 4, "Weight-gated reads": the refine thresholds follow each
 * request's own length).
 *   q          bf16 query rows in the model's basis; head_dim 64 or 128
 *   planes_out [batch][num_heads][2][head_dim] int8; eta_out [batch][num_heads]
 *   req_lens   [batch] int32 (device): each request's total key count (all
 *              levels of a cascade); tau_out [batch] fp32 receives
 *              tau_r = kappa + ceil(log2 n_r) (ceil(log2 n) = 0 for n <= 1).
 *              Both NULL: no thresholds are written.
 *   kappa      any value but NaN; +INFINITY refines every live key,
 *              -INFINITY none.  0 refines the keys whose coarse weight
 *              2^xc is at least 2^-ceil(log2 n_r), about their mean share;
 *              -4 (16 times that share) is the Python binding's default.
 *   kappa_v, tau_v_out: the same for the second value plane of 8-bit values
 *              (tau_v_out may be NULL; written only with req_lens).
 */
fold_status fold_q8_split_query(const fold_q_view* q, int32_t head_dim, float sm_scale,
                                const int32_t* req_lens, float kappa, float kappa_v,
                                int8_t* planes_out, float* eta_out, float* tau_out,
                                float* tau_v_out, void* stream);

/*
 * fold_v8_write_values - writer of 8-bit values (Section 4, "Cache format"):
 * the two E4M3 planes of n_tok BF16 value rows, stored like
 * fold_q8_write_keys stores key codes (same token list, view and skipping).
 *   v_src      [n_tok][num_kv_heads][head_dim] bf16
 *   scale_exp  e of the cache's scale 2^e (choose e >= log2(max|v| / 448))
 *   plane_p, plane_r: the value planes written
 */
fold_status fold_v8_write_values(const fold_kv_view* kv, const void* v_src,
                                 const int32_t* tok_seq, const int32_t* tok_pos, int32_t n_tok,
                                 int32_t scale_exp, uint8_t* plane_p, uint8_t* plane_r,
                                 void* stream);

/*
 * fold_q8_ref_estimate - fold_ref_estimate on the coarse logits
 * eta_i e_j (a_j . qa_i + (a_j . qb_i) / 256) (Section 3, "Choosing the
 * reference": the estimate is scored with the kernel's own coarse logits).
 * Same sample, trim, output and restrictions as fold_ref_estimate; kv->k is
 * not read.
 */
fold_status fold_q8_ref_estimate(const fold_kv_view* kv, const fold_q8_keys* keys,
                                 const fold_q8_query* q, const fold_est_params* params,
                                 float* z_out, void* stream);

/*
 * fold_q8_front - the per-step front of a two-plane key cache in one launch
 * (the paper fuses the query quantisation and the reference estimate into
 * one front kernel; Section 4, "Cache format"; Section 3, "Choosing the
 * reference"): the result of fold_q8_split_query(q, kv->head_dim, sm_scale,
 * req_lens, kappa, kappa_v, planes_out, eta_out, tau_out, tau_v_out)
 * followed by fold_q8_ref_estimate(kv, keys, {planes_out, eta_out, tau_out,
 * q->batch, q->num_heads, tau_v_out}, params, z_out), bit for bit.
 *   kv, keys   the per-request view of the cache (no CSR rows) and its planes
 *   q          bf16 query rows [batch][num_heads][kv->head_dim], 16-byte aligned
 *   other arguments and outputs: as those two calls.  Errors: as those two
 *   calls; the GQA group must be at most 16 rows.
 */
fold_status fold_q8_front(const fold_kv_view* kv, const fold_q8_keys* keys, const fold_q_view* q,
                          float sm_scale, const int32_t* req_lens, float kappa, float kappa_v,
                          int8_t* planes_out, float* eta_out, float* tau_out, float* tau_v_out,
                          const fold_est_params* params, float* z_out, void* stream);

/* Rows per read group (1 when one row attends each kv sequence and head, else
 * 16 or 32) and read groups per (kv sequence, kv head) of
 * fold_q8_decode_split; -1 on an invalid view.  The GQA group size
 * num_heads / num_kv_heads must be 1, 2, 4, 8, 16 or 32, so that every read
 * group holds whole GQA groups. */
int32_t fold_q8_decode_rows_per_group(const fold_kv_view* kv, const fold_q8_query* q);
int32_t fold_q8_decode_row_groups(const fold_kv_view* kv, const fold_q8_query* q);

/*
 * fold_q8_decode_split - gated split-KV scan of one level over a two-plane
 * key cache (Algorithm 1): the split layout, slots, depth rule and outputs
 * of fold_decode_split, with the coarse/refine scores above.
 *   kv       view of the level (kv->k is not read; kv->v holds BF16 values)
 *   keys     the cache's planes and scales
 *   q        query codes, eta and tau (fold_q8_split_query)
 *   z        [batch][num_heads] fp32 references
 *   depth_T  +INFINITY (dense) or a finite T >= 0
 *   values   NULL (BF16 values from kv->v), or 8-bit values (then q->tau_v
 *            is required and kv->v is not read)
 *   part_Lcut NULL, or the cut masses for the value model (fold_decode_split)
 *   dbg      NULL, or the optional exports above
 */
fold_status fold_q8_decode_split(const fold_kv_view* kv, const fold_q8_keys* keys,
                                 const fold_q8_query* q, const fold_v8_values* values,
                                 const float* z, float depth_T, int32_t num_splits,
                                 int32_t slot_offset, int32_t num_slots, float* part_A,
                                 float* part_L, float* part_Lcut, const fold_q8_debug* dbg,
                                 void* stream);

/*
 * Stacked levels over a two-plane key cache (Appendix E, tile layouts: past
 * 64 stacked query rows a level runs laid out as prefill is, and its logit is
 * one FP16 product of each key's code, rounded once per prefix, against the
 * rows' queries).  A level that more than 32 rows attend per kv sequence (a
 * shared prefix, a wide draft level) is decoded from FP16 keys written once:
 *
 * fold_q8_stack_keys - k_f16 = fp16(e (a + b/256)) for every key of the
 * view's kv sequences, rounded to nearest even (a + b/256 and its product with
 * the BF16 scale are exact in FP32; the scale is folded in before the one
 * rounding).
 *   kv     the level's view (sequences, lengths, block table; kv->k and kv->v
 *          are not read)
 *   keys   the cache's planes and scales
 *   k_f16  FP16 bits in the element layout of the planes (2 bytes per
 *          element), 16-byte aligned; elements of keys past a sequence's
 *          length or on a page id outside [0, num_pages) are not written
 */
fold_status fold_q8_stack_keys(const fold_kv_view* kv, const fold_q8_keys* keys,
                               uint16_t* k_f16, void* stream);

/*
 * fold_q8_decode_stacked - the split scan of a stacked level over the FP16
 * keys: s_ij = eta_i (k^_j . q^_i), k^ from fold_q8_stack_keys, q^ =
 * fp16(qa + qb/256) from the query codes, the product accumulated in FP32;
 * then the depth rule, slots and outputs of fold_decode_split (read groups of
 * 64 rows, as fold_decode_rows_per_group gives them).  There is no coarse
 * pass and no refine gate: the product holds both planes (q->tau is not read).
 *   kv       the level's view with kv->k = the FP16 keys and kv->v the BF16
 *            values; more than 32 rows must attend each kv sequence, else
 *            FOLD_E_UNSUPPORTED (fold_q8_decode_split serves such levels)
 *   q        query codes and eta (fold_q8_split_query)
 *   z, depth_T, num_splits, slot_offset, num_slots, part_A, part_L,
 *   part_Lcut, dbg   as fold_decode_split
 */
fold_status fold_q8_decode_stacked(const fold_kv_view* kv, const fold_q8_query* q, const float* z,
                                   float depth_T, int32_t num_splits, int32_t slot_offset,
                                   int32_t num_slots, float* part_A, float* part_L,
                                   float* part_Lcut, const fold_debug* dbg, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FOLD_Q8_H */
