/*
 * fold_draft.h - draft columns for speculative verification (Section 4,
 * "Value product": speculative drafts and verification trees are extra query
 * columns masked to their ancestors).
 *
 * Request r of a paged view holds n_r keys; its last m_r keys belong to its
 * m_r draft tokens, in column order, and it owns m_r query columns.  Column c
 * (draft c of r, 0 <= c < m_r) has a parent column parent[c] in [-1, c)
 * (-1: the committed cache) and sees the committed keys [0, n_r - m_r) plus
 * the draft keys of c and of all its ancestors.
 *
 * The columns are decoded as two levels whose pairs add (Proposition 1(i)):
 *   - committed level: the requests' own view with seq_lens = the committed
 *     lengths and the columns of request r as its stacked rows
 *     (row_indptr = col_indptr, row_req = 0 .. num_cols - 1), so every
 *     committed key is read once for all of a request's columns;
 *   - ancestor level: one kv sequence per column holding the keys of its
 *     ancestors (itself included) in position order, copied by
 *     fold_draft_gather into spare pages of the same pool (block table =
 *     the column's spare pages, seq_lens = anc_lens).
 * References come from the estimate on a per-column view of the committed
 * keys (block table = the request's, written by fold_draft_gather; lengths
 * = the committed lengths).  The combine adds the two levels' slots.
 */
#ifndef FOLD_DRAFT_H
#define FOLD_DRAFT_H

#include "fold.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * fold_draft_plan - host-side plan (no GPU work; every pointer is a host
 * pointer).
 *   num_seqs      requests
 *   seq_lens      [num_seqs] keys of each request, its drafts included
 *   col_indptr    [num_seqs + 1] the columns of request r are
 *                 [col_indptr[r], col_indptr[r + 1]); col_indptr[0] = 0
 *   parent        [num_cols] parent column relative to the request's first
 *                 column, in [-1, c)
 *   page_size, pages_per_col: spare pages per column; a column's ancestor
 *                 count must fit pages_per_col * page_size
 * Outputs (host arrays the caller then copies to the device):
 *   committed_lens [num_seqs]  n_r - m_r
 *   col_req        [num_cols]  request of each column
 *   col_lens       [num_cols]  committed length of the column's request
 *   anc_lens       [num_cols]  number of keys of the ancestor level
 *   anc_pos        [num_cols][pages_per_col * page_size] positions (within
 *                  the request) of those keys in increasing order; -1 after
 * FOLD_E_INVAL on any violation above (nothing written then).
 */
fold_status fold_draft_plan(int32_t num_seqs, const int32_t* seq_lens, const int32_t* col_indptr,
                            const int32_t* parent, int32_t page_size, int32_t pages_per_col,
                            int32_t* committed_lens, int32_t* col_req, int32_t* col_lens,
                            int32_t* anc_lens, int32_t* anc_pos);

/*
 * fold_draft_gather - copy every column's ancestor rows of one cache array
 * into its spare pages (device work).
 *   kv            the requests' paged view (block table, page size, pool
 *                 size; kv->k, kv->v and seq_lens are not read)
 *   col_req, anc_lens, anc_pos: the plan's arrays, on the device
 *   spare_pages   [num_cols][pages_per_col] int32 page ids of the pool; the
 *                 caller keeps them apart from every request's pages
 *   row_bytes     bytes of one (page, kv head, slot) row of the array: 2 D
 *                 for BF16 keys or values, D for INT8 / E4M3 planes, 2 for
 *                 key scales; 1 .. 4096
 *   src, dst      the array read and written (the same pool array, or two
 *                 with one layout); both NULL copies nothing.  16-byte
 *                 aligned when row_bytes is a multiple of 16, else 2-byte
 *                 aligned when it is even.
 *   col_block_table [num_cols][kv->max_pages_per_seq] int32 or NULL:
 *                 receives each column's request's block-table row (the
 *                 estimate's per-column view)
 * Positions or spare pages the view cannot address are skipped.
 */
fold_status fold_draft_gather(const fold_kv_view* kv, const int32_t* col_req,
                              const int32_t* anc_lens, const int32_t* anc_pos,
                              const int32_t* spare_pages, int32_t num_cols,
                              int32_t pages_per_col, int32_t row_bytes, const void* src,
                              void* dst, int32_t* col_block_table, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FOLD_DRAFT_H */
