// Host side of the C ABI declared in include/fold.h and include/fold_q8.h:
// argument validation and kernel launches.  Nothing here allocates,
// synchronises or keeps a pointer.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdint.h>

#include <algorithm>
#include <string>
#include <vector>

#include "fold.h"
#include "fold_q8.h"
#include "fold_draft.h"
#include "fold_internal.h"

namespace {

thread_local std::string g_last_error;

fold_status fail(fold_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

fold_status ok() {
  g_last_error.clear();
  return FOLD_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

const float kLog2e = 1.4426950408889634f;

// Size and layout checks of a view read by query rows [batch][num_heads];
// fills the geometry.  Pointer checks are the caller's.
fold_status check_layout(const fold_kv_view* kv, int32_t batch, int32_t num_heads,
                         fold::ScanGeometry* g) {
  if (kv->head_dim != 64 && kv->head_dim != 128)
    return fail(FOLD_E_INVAL, "head_dim %d: must be 64 or 128", kv->head_dim);
  if (kv->num_kv_heads < 1 || num_heads < 1 || num_heads % kv->num_kv_heads != 0)
    return fail(FOLD_E_INVAL, "num_heads %d must be a positive multiple of num_kv_heads %d",
                num_heads, kv->num_kv_heads);
  if (kv->num_seqs < 0 || batch < 0 || kv->max_seq_len < 0)
    return fail(FOLD_E_INVAL, "negative size");
  if (kv->block_table) {
    if (kv->page_size <= 0 || kv->page_size % fold::kChunk != 0)
      return fail(FOLD_E_INVAL, "page_size %d: must be a positive multiple of 16", kv->page_size);
    if (kv->max_pages_per_seq < 1 || kv->num_pages < 1)
      return fail(FOLD_E_INVAL, "max_pages_per_seq and num_pages must be positive");
  }
  if ((kv->row_indptr == nullptr) != (kv->row_req == nullptr))
    return fail(FOLD_E_INVAL, "row_indptr and row_req must both be set or both be NULL");
  if (kv->row_indptr && kv->max_reqs_per_seq < 1)
    return fail(FOLD_E_INVAL, "max_reqs_per_seq must be positive with CSR rows");
  if (!kv->row_indptr && kv->num_seqs > batch)
    return fail(FOLD_E_INVAL, "num_seqs %d exceeds batch %d (request s attends kv sequence s)",
                kv->num_seqs, batch);
  g->k = static_cast<const uint16_t*>(kv->k);
  g->v = static_cast<const uint16_t*>(kv->v);
  g->block_table = kv->block_table;
  g->seq_lens = kv->seq_lens;
  g->row_indptr = kv->row_indptr;
  g->row_req = kv->row_req;
  g->num_seqs = kv->num_seqs;
  g->hkv = kv->num_kv_heads;
  g->page_size = kv->block_table ? kv->page_size : 0;
  g->max_pages = kv->block_table ? kv->max_pages_per_seq : 0;
  g->num_pages = kv->block_table ? kv->num_pages : 0;
  g->max_seq_len = kv->max_seq_len;
  g->batch = batch;
  g->heads = num_heads;
  g->group = num_heads / kv->num_kv_heads;
  return FOLD_OK;
}

// Checks shared by the calls that read a BF16 cache; fills the geometry.
fold_status check_view(const fold_kv_view* kv, const fold_q_view* q, fold::ScanGeometry* g,
                       bool need_v) {
  if (!kv || !q) return fail(FOLD_E_INVAL, "kv view and q view are required");
  if (!kv->k || (need_v && !kv->v) || !kv->seq_lens || !q->q)
    return fail(FOLD_E_INVAL, "k%s, seq_lens and q pointers are required", need_v ? ", v" : "");
  if (!aligned16(kv->k) || (need_v && !aligned16(kv->v)) || !aligned16(q->q))
    return fail(FOLD_E_INVAL, "q, k and v must be 16-byte aligned");
  return check_layout(kv, q->batch, q->num_heads, g);
}

// Checks shared by the calls that read a two-plane key cache.
fold_status check_q8_view(const fold_kv_view* kv, const fold_q8_keys* keys, const fold_q8_query* q,
                          fold::ScanGeometry* g, bool need_v) {
  if (!kv || !keys || !q) return fail(FOLD_E_INVAL, "kv view, keys and q are required");
  if ((need_v && !kv->v) || !kv->seq_lens || !keys->plane_a || !keys->plane_b || !keys->scale ||
      !q->planes || !q->eta)
    return fail(FOLD_E_INVAL, "%splane_a, plane_b, scale, seq_lens, query planes and eta are "
                "required", need_v ? "v, " : "");
  if ((need_v && !aligned16(kv->v)) || !aligned16(keys->plane_a) || !aligned16(keys->plane_b) ||
      !aligned16(keys->scale) || !aligned16(q->planes))
    return fail(FOLD_E_INVAL, "v, planes and scales must be 16-byte aligned");
  fold_status st = check_layout(kv, q->batch, q->num_heads, g);
  if (st != FOLD_OK) return st;
  const int G = g->group;
  if (G > 32 || (G & (G - 1)) != 0)
    return fail(FOLD_E_UNSUPPORTED, "GQA group %d: the two-plane scan needs 1, 2, 4, 8, 16 or 32", G);
  return FOLD_OK;
}

int q8_rows_per_group(int rows) { return rows <= 1 ? 1 : (rows <= 16 ? 16 : 32); }

int rows_per_seq_of(const fold_kv_view* kv, int num_heads) {
  const int group = num_heads / kv->num_kv_heads;
  const long long reqs = kv->row_indptr ? kv->max_reqs_per_seq : 1;
  const long long rows = reqs * group;
  return rows > (1 << 30) ? (1 << 30) : static_cast<int>(rows);
}

int rows_per_seq(const fold_kv_view* kv, const fold_q_view* q) {
  return rows_per_seq_of(kv, q->num_heads);
}

fold_status check_depth(float depth_T) {
  if (isnan(depth_T) || depth_T < 0.0f)
    return fail(FOLD_E_INVAL, "depth_T must be +INFINITY or a finite value >= 0");
  return FOLD_OK;
}

fold_status check_est_params(const fold_est_params* params, fold_est_params* p) {
  *p = {1, 63, 128, 8, 8};
  if (params) *p = *params;
  if (p->sink < 0 || p->recent < 0 || p->strata < 1 || p->trim_lo < 0 || p->trim_hi < 0 ||
      p->trim_lo + p->trim_hi >= p->strata ||
      static_cast<long long>(p->sink) + p->recent + p->strata > fold::kMaxEstSamples)
    return fail(FOLD_E_INVAL, "estimator parameters out of range");
  return FOLD_OK;
}

}  // namespace

extern "C" {

int fold_abi_version(void) { return FOLD_ABI_VERSION; }

const char* fold_status_string(fold_status s) {
  switch (s) {
    case FOLD_OK: return "FOLD_OK";
    case FOLD_E_INVAL: return "FOLD_E_INVAL: invalid argument";
    case FOLD_E_UNSUPPORTED: return "FOLD_E_UNSUPPORTED: not supported by this build";
    case FOLD_E_HIP: return "FOLD_E_HIP: HIP launch error";
  }
  return "unknown fold_status";
}

const char* fold_last_error(void) { return g_last_error.c_str(); }

int32_t fold_decode_rows_per_group(const fold_kv_view* kv, const fold_q_view* q) {
  fold::ScanGeometry g;
  if (check_view(kv, q, &g, false) != FOLD_OK) return -1;
  return fold::decode_rows_per_group(rows_per_seq(kv, q));
}

int32_t fold_decode_row_groups(const fold_kv_view* kv, const fold_q_view* q) {
  fold::ScanGeometry g;
  if (check_view(kv, q, &g, false) != FOLD_OK) return -1;
  const int rows = rows_per_seq(kv, q);
  const int gr = fold::decode_rows_per_group(rows);
  return (rows + gr - 1) / gr;
}

fold_status fold_ref_estimate(const fold_kv_view* kv, const fold_q_view* q, float sm_scale,
                              const fold_est_params* params, float* z_out, void* stream) {
  fold::EstimateArgs a;
  fold_status st = check_view(kv, q, &a.geo, false);
  if (st != FOLD_OK) return st;
  if (!z_out) return fail(FOLD_E_INVAL, "z_out is required");
  if (kv->row_indptr) return fail(FOLD_E_INVAL, "the estimate needs a per-request view (no CSR rows)");
  if (!isfinite(sm_scale)) return fail(FOLD_E_INVAL, "sm_scale must be finite");
  if (a.geo.group > fold::kMaxEstRows)
    return fail(FOLD_E_UNSUPPORTED, "GQA group %d exceeds %d", a.geo.group, fold::kMaxEstRows);
  fold_est_params p;
  st = check_est_params(params, &p);
  if (st != FOLD_OK) return st;
  a.q = static_cast<const uint16_t*>(q->q);
  a.z_out = z_out;
  a.score_scale = kLog2e * sm_scale;
  a.sink = p.sink;
  a.recent = p.recent;
  a.strata = p.strata;
  a.trim_lo = p.trim_lo;
  a.trim_hi = p.trim_hi;
  if (static_cast<long long>(q->batch) * kv->num_kv_heads > 0x7fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  hipError_t e = fold::launch_estimate(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "estimate launch: %s", hipGetErrorString(e));
  return ok();
}

// Validation and arguments of one level's split scan (shared by
// fold_decode_split and fold_decode_split_blocks); launches nothing.
static fold_status split_args(const fold_kv_view* kv, const fold_q_view* q, float sm_scale,
                              const float* z, float depth_T, int32_t num_splits,
                              int32_t slot_offset, int32_t num_slots, float* part_A,
                              float* part_L, float* part_Lcut, const fold_debug* dbg,
                              fold::DecodeArgs* out) {
  fold::DecodeArgs& a = *out;
  a = fold::DecodeArgs{};
  fold_status st = check_view(kv, q, &a.geo, true);
  if (st != FOLD_OK) return st;
  if (!z || !part_A || !part_L) return fail(FOLD_E_INVAL, "z, part_A and part_L are required");
  st = check_depth(depth_T);
  if (st != FOLD_OK) return st;
  if (!isfinite(sm_scale)) return fail(FOLD_E_INVAL, "sm_scale must be finite");
  if (num_splits < 1) return fail(FOLD_E_INVAL, "num_splits must be >= 1");
  if (slot_offset < 0 || static_cast<long long>(slot_offset) + num_splits > num_slots)
    return fail(FOLD_E_INVAL, "slots [%d, %d) exceed num_slots %d", slot_offset,
                slot_offset + num_splits, num_slots);
  const int rows = rows_per_seq(kv, q);
  const int gr = fold::decode_rows_per_group(rows);
  const int groups = (rows + gr - 1) / gr;
  const long long blocks = static_cast<long long>(kv->num_seqs) * kv->num_kv_heads * num_splits * groups;
  if (blocks > 0x7fffffffLL) return fail(FOLD_E_INVAL, "grid too large");
  a.q = static_cast<const uint16_t*>(q->q);
  a.z = z;
  a.part_A = part_A;
  a.part_L = part_L;
  a.part_Lcut = part_Lcut;
  a.x_out = dbg ? dbg->x_out : nullptr;
  a.key_gate_out = dbg ? dbg->key_gate_out : nullptr;
  a.page_gate_out = dbg ? dbg->page_gate_out : nullptr;
  a.score_scale = kLog2e * sm_scale;
  a.dense = isinf(depth_T) ? 1 : 0;
  a.neg_T = a.dense ? 0.0f : -depth_T;
  a.num_splits = num_splits;
  a.slot_offset = slot_offset;
  a.rows_per_seq = rows;
  a.rows_per_group = gr;
  a.row_groups = groups;
  a.by_length = (!kv->row_indptr && kv->num_seqs >= 2 && kv->num_seqs <= fold::kOrderMax) ? 1 : 0;
  return FOLD_OK;
}

fold_status fold_decode_split(const fold_kv_view* kv, const fold_q_view* q, float sm_scale,
                              const float* z, float depth_T, int32_t num_splits,
                              int32_t slot_offset, int32_t num_slots, float* part_A,
                              float* part_L, float* part_Lcut, const fold_debug* dbg,
                              void* stream) {
  fold::DecodeArgs a;
  fold_status st = split_args(kv, q, sm_scale, z, depth_T, num_splits, slot_offset, num_slots,
                              part_A, part_L, part_Lcut, dbg, &a);
  if (st != FOLD_OK) return st;
  hipError_t e = fold::launch_decode(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "decode launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_decode_cascade(const fold_kv_view* prefix, const fold_kv_view* suffix,
                                const fold_q_view* q, float sm_scale, const float* z,
                                float depth_T, int32_t num_splits, int32_t slot_offset,
                                int32_t num_slots, float* part_A, float* part_L,
                                float* part_Lcut, void* stream) {
  fold::DecodeArgs a;
  fold_status st = split_args(prefix, q, sm_scale, z, depth_T, num_splits, slot_offset, num_slots,
                              part_A, part_L, part_Lcut, nullptr, &a);
  if (st != FOLD_OK) return st;
  if (!suffix) return fail(FOLD_E_INVAL, "suffix view is required");
  fold::ScanGeometry sg;
  st = check_view(suffix, q, &sg, true);
  if (st != FOLD_OK) return st;
  if (!prefix->row_indptr || a.rows_per_group != 64)
    return fail(FOLD_E_UNSUPPORTED, "the prefix must be a CSR level of more than 32 stacked rows "
                "per kv sequence");
  if (suffix->row_indptr || suffix->num_seqs != q->batch)
    return fail(FOLD_E_UNSUPPORTED, "the suffix must be a per-request view of q->batch sequences");
  if (suffix->k != prefix->k || suffix->v != prefix->v ||
      suffix->num_kv_heads != prefix->num_kv_heads || suffix->head_dim != prefix->head_dim ||
      !suffix->block_table || !prefix->block_table || sg.page_size <= 0 ||
      sg.page_size != a.geo.page_size || sg.num_pages != a.geo.num_pages)
    return fail(FOLD_E_UNSUPPORTED, "prefix and suffix must share k, v and one paged layout");
  const long long U = (static_cast<long long>(suffix->max_seq_len) + fold::kTile - 1) / fold::kTile;
  if (U < 1) return fail(FOLD_E_INVAL, "suffix max_seq_len must be >= 1");
  const long long G = a.geo.group;
  const long long positions = std::min<long long>(63 / G + 2, prefix->max_reqs_per_seq);
  const long long pre_tiles = (static_cast<long long>(prefix->max_seq_len) + fold::kTile - 1) / fold::kTile;
  const long long per_wg = (pre_tiles + num_splits - 1) / num_splits +
                           (positions * U + num_splits - 1) / num_splits;
  if (per_wg > 64)
    return fail(FOLD_E_UNSUPPORTED, "a workgroup would own up to %lld tiles (at most 64): raise "
                "num_splits", per_wg);
  a.sfx_block_table = suffix->block_table;
  a.sfx_seq_lens = suffix->seq_lens;
  a.sfx_max_pages = suffix->max_pages_per_seq;
  a.sfx_cap = fold::view_capacity(sg);
  a.sfx_tiles = static_cast<int>(U);
  hipError_t e = fold::launch_decode_cascade(a, prefix->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "cascade launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_decode_split_blocks(const fold_kv_view* kv, const fold_q_view* q,
                                     float sm_scale, const float* z, float depth_T,
                                     int32_t num_splits, int32_t slot_offset, int32_t num_slots,
                                     float* part_A, float* part_L,
                                     const fold_block_model* model, const fold_debug* dbg,
                                     void* stream) {
  fold::DecodeArgs a;
  fold_status st = split_args(kv, q, sm_scale, z, depth_T, num_splits, slot_offset, num_slots,
                              part_A, part_L, nullptr, dbg, &a);
  if (st != FOLD_OK) return st;
  if (!model || !model->block_mean) return fail(FOLD_E_INVAL, "the block model is required");
  const long long need_blocks = (static_cast<long long>(kv->max_seq_len) + fold::kTile - 1) / fold::kTile;
  if (model->max_blocks < need_blocks)
    return fail(FOLD_E_INVAL, "max_blocks %d < ceil(max_seq_len / 64) = %lld", model->max_blocks,
                need_blocks);
  if (!aligned16(model->block_mean)) return fail(FOLD_E_INVAL, "block_mean must be 16-byte aligned");
  if (!a.dense && !model->chunk_cut)
    return fail(FOLD_E_INVAL, "chunk_cut is required at a finite depth");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (a.dense) {  // no key is cut: the plain scan
    hipError_t e = fold::launch_decode(a, kv->head_dim, s);
    if (e != hipSuccess) return fail(FOLD_E_HIP, "decode launch: %s", hipGetErrorString(e));
    return ok();
  }
  a.chunk_cut = model->chunk_cut;
  a.chunk_stride = static_cast<int>((static_cast<long long>(kv->max_seq_len) + fold::kChunk - 1) /
                                    fold::kChunk);
  fold::BlockModelArgs b;
  b.geo = a.geo;
  b.part_A = part_A;
  b.chunk_cut = model->chunk_cut;
  b.block_mean = model->block_mean;
  b.chunk_stride = a.chunk_stride;
  b.max_blocks = model->max_blocks;
  b.num_splits = num_splits;
  b.slot_offset = slot_offset;
  b.rows_per_seq = a.rows_per_seq;
  const int rb = fold::block_model_rows(a.rows_per_seq);
  b.row_tiles = (a.rows_per_seq + rb - 1) / rb;
  const long long blocks = static_cast<long long>(kv->num_seqs) * kv->num_kv_heads * num_splits *
                           b.row_tiles;
  if (blocks > 0x7fffffffLL) return fail(FOLD_E_INVAL, "grid too large");
  hipError_t e = fold::launch_decode(a, kv->head_dim, s);
  if (e != hipSuccess) return fail(FOLD_E_HIP, "decode launch: %s", hipGetErrorString(e));
  e = fold::launch_block_model(b, kv->head_dim, s);
  if (e != hipSuccess) return fail(FOLD_E_HIP, "block model launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_combine(const float* part_A, const float* part_L, int32_t num_slots,
                         int32_t num_rows, int32_t head_dim, const float* z, void* out,
                         fold_dtype out_dtype, float* lse_out, uint8_t* cert_out,
                         const fold_value_model* model, void* stream) {
  if (!part_A || !part_L || !out) return fail(FOLD_E_INVAL, "part_A, part_L and out are required");
  if (num_slots < 1 || num_rows < 0) return fail(FOLD_E_INVAL, "num_slots >= 1, num_rows >= 0");
  if (head_dim != 64 && head_dim != 128)
    return fail(FOLD_E_INVAL, "head_dim %d: must be 64 or 128", head_dim);
  if (out_dtype != FOLD_DTYPE_F32 && out_dtype != FOLD_DTYPE_BF16)
    return fail(FOLD_E_INVAL, "unknown out_dtype");
  if (lse_out && !z) return fail(FOLD_E_INVAL, "lse_out needs z");
  fold::CombineArgs a;
  a.part_Lcut = nullptr;
  a.mean = nullptr;
  a.heads = a.hkv = 1;
  if (model) {
    if (!model->part_Lcut || !model->mean)
      return fail(FOLD_E_INVAL, "the value model needs part_Lcut and mean");
    if (model->num_kv_heads < 1 || model->num_heads < 1 ||
        model->num_heads % model->num_kv_heads != 0 || num_rows % model->num_heads != 0)
      return fail(FOLD_E_INVAL, "value model: num_heads %d must be a multiple of num_kv_heads %d "
                  "and divide num_rows %d", model->num_heads, model->num_kv_heads, num_rows);
    a.part_Lcut = model->part_Lcut;
    a.mean = model->mean;
    a.heads = model->num_heads;
    a.hkv = model->num_kv_heads;
  }
  a.part_A = part_A;
  a.part_L = part_L;
  a.z = z;
  a.out = out;
  a.lse_out = lse_out;
  a.cert_out = cert_out;
  a.num_slots = num_slots;
  a.num_rows = num_rows;
  a.head_dim = head_dim;
  a.out_bf16 = out_dtype == FOLD_DTYPE_BF16 ? 1 : 0;
  hipError_t e = fold::launch_combine(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "combine launch: %s", hipGetErrorString(e));
  return ok();
}

// Validation and arguments of the one-launch decode (shared by
// fold_decode_fused and fold_decode_fused_noalloc); launches nothing.
static fold_status fused_args(const fold_kv_view* kv, const fold_q_view* q, float sm_scale,
                              const fold_est_params* params, float depth_T, int32_t num_splits,
                              float* part_A, float* part_L, int32_t* arrivals, float* z_out,
                              void* out, fold_dtype out_dtype, float* lse_out,
                              uint8_t* cert_out, fold::FusedArgs* fa) {
  fold::FusedArgs& f = *fa;
  f = fold::FusedArgs{};
  fold::DecodeArgs& a = f.d;
  fold_status st = check_view(kv, q, &a.geo, true);
  if (st != FOLD_OK) return st;
  if (!part_A || !part_L || !arrivals || !z_out || !out)
    return fail(FOLD_E_INVAL, "part_A, part_L, arrivals, z_out and out are required");
  if (kv->row_indptr) return fail(FOLD_E_INVAL, "the fused decode needs a per-request view (no CSR rows)");
  if (kv->num_seqs != q->batch)
    return fail(FOLD_E_INVAL, "the fused decode needs num_seqs %d == batch %d", kv->num_seqs, q->batch);
  st = check_depth(depth_T);
  if (st != FOLD_OK) return st;
  if (!isfinite(sm_scale)) return fail(FOLD_E_INVAL, "sm_scale must be finite");
  if (num_splits < 1) return fail(FOLD_E_INVAL, "num_splits must be >= 1");
  if (out_dtype != FOLD_DTYPE_F32 && out_dtype != FOLD_DTYPE_BF16)
    return fail(FOLD_E_INVAL, "unknown out_dtype");
  if ((reinterpret_cast<uintptr_t>(part_A) & 15u) != 0 || (reinterpret_cast<uintptr_t>(out) & 15u) != 0)
    return fail(FOLD_E_INVAL, "part_A and out must be 16-byte aligned");
  const int rows = rows_per_seq(kv, q);
  if (rows < 2 || rows > 8)
    return fail(FOLD_E_UNSUPPORTED, "the fused decode serves 2 to 8 rows per kv head (got %d)", rows);
  fold_est_params p;
  st = check_est_params(params, &p);
  if (st != FOLD_OK) return st;
  const long long blocks = static_cast<long long>(kv->num_seqs) * kv->num_kv_heads * num_splits;
  if (blocks > 0x7fffffffLL) return fail(FOLD_E_INVAL, "grid too large");
  if (static_cast<long long>(num_splits) * q->batch * q->num_heads * kv->head_dim * 4 >= (1LL << 31))
    return fail(FOLD_E_UNSUPPORTED, "the fused decode's slots must stay under 2 GiB");
  a.q = static_cast<const uint16_t*>(q->q);
  a.z = nullptr;
  a.part_A = part_A;
  a.part_L = part_L;
  a.part_Lcut = nullptr;
  a.score_scale = kLog2e * sm_scale;
  a.dense = isinf(depth_T) ? 1 : 0;
  a.neg_T = a.dense ? 0.0f : -depth_T;
  a.num_splits = num_splits;
  a.slot_offset = 0;
  a.rows_per_seq = rows;
  a.rows_per_group = fold::decode_rows_per_group(rows);
  a.row_groups = 1;
  fold::EstimateArgs& e = f.x.est.e;
  e.geo = a.geo;
  e.q = a.q;
  e.z_out = z_out;
  e.score_scale = a.score_scale;
  e.sink = p.sink;
  e.recent = p.recent;
  e.strata = p.strata;
  e.trim_lo = p.trim_lo;
  e.trim_hi = p.trim_hi;
  f.x.arrivals = arrivals;
  f.x.out = out;
  f.x.lse_out = lse_out;
  f.x.cert_out = cert_out;
  f.x.out_bf16 = out_dtype == FOLD_DTYPE_BF16 ? 1 : 0;
  return FOLD_OK;
}

fold_status fold_decode_fused(const fold_kv_view* kv, const fold_q_view* q, float sm_scale,
                              const fold_est_params* params, float depth_T, int32_t num_splits,
                              float* part_A, float* part_L, int32_t* arrivals, float* z_out,
                              void* out, fold_dtype out_dtype, float* lse_out,
                              uint8_t* cert_out, void* stream) {
  fold::FusedArgs f;
  fold_status st = fused_args(kv, q, sm_scale, params, depth_T, num_splits, part_A, part_L,
                              arrivals, z_out, out, out_dtype, lse_out, cert_out, &f);
  if (st != FOLD_OK) return st;
  hipError_t err = fold::launch_decode_fused(f, kv->head_dim, static_cast<hipStream_t>(stream));
  if (err != hipSuccess) return fail(FOLD_E_HIP, "fused decode launch: %s", hipGetErrorString(err));
  return ok();
}

fold_status fold_decode_fused_noalloc(const fold_kv_view* kv, const fold_q_view* q,
                                      float sm_scale, const fold_est_params* params,
                                      float depth_T, int32_t num_splits, float* z_out, void* out,
                                      fold_dtype out_dtype, float* lse_out, uint8_t* cert_out,
                                      void* stream) {
  if (!kv || !q) return fail(FOLD_E_INVAL, "kv and q views are required");
  if (num_splits < 1) return fail(FOLD_E_INVAL, "num_splits must be >= 1");
  if (q->batch < 0 || q->num_heads < 0 || kv->num_seqs < 0 || kv->num_kv_heads < 0 ||
      (kv->head_dim != 64 && kv->head_dim != 128))
    return fail(FOLD_E_INVAL, "bad view sizes");
  // scratch layout: slots A, slots L, arrival counts, each from a 256-byte boundary
  auto up = [](long long b) { return (b + 255) / 256 * 256; };
  const long long rows = static_cast<long long>(q->batch) * q->num_heads;
  if (num_splits > (1 << 20) || rows > (1LL << 31) ||
      static_cast<long long>(kv->num_seqs) * kv->num_kv_heads > (1LL << 31))
    return fail(FOLD_E_INVAL, "the call is far larger than the fixed scratch");
  const long long bytes_a = up(static_cast<long long>(num_splits) * rows * kv->head_dim * 4);
  const long long bytes_l = up(static_cast<long long>(num_splits) * rows * 4);
  const long long bytes_c = up(static_cast<long long>(kv->num_seqs) * kv->num_kv_heads * 4);
  const long long need = bytes_a + bytes_l + bytes_c;
  if (need > static_cast<long long>(fold::scratch_capacity()))
    return fail(FOLD_E_INVAL,
                "the call needs %lld bytes of scratch (slots and arrival counts); the fixed "
                "scratch holds %lld: use fold_decode_fused with caller workspace",
                need, static_cast<long long>(fold::scratch_capacity()));
  // validate every argument first (placeholder workspace addresses with the
  // scratch's alignment), so a refused call touches no HIP state
  char* base = reinterpret_cast<char*>(uintptr_t{256});
  fold::FusedArgs f;
  fold_status st = fused_args(kv, q, sm_scale, params, depth_T, num_splits,
                              reinterpret_cast<float*>(base), reinterpret_cast<float*>(base + bytes_a),
                              reinterpret_cast<int32_t*>(base + bytes_a + bytes_l), z_out, out,
                              out_dtype, lse_out, cert_out, &f);
  if (st != FOLD_OK) return st;
  hipError_t err = fold::scratch_device_ptr(reinterpret_cast<void**>(&base));
  if (err != hipSuccess) return fail(FOLD_E_HIP, "scratch address: %s", hipGetErrorString(err));
  float* part_A = reinterpret_cast<float*>(base);
  float* part_L = reinterpret_cast<float*>(base + bytes_a);
  int32_t* arrivals = reinterpret_cast<int32_t*>(base + bytes_a + bytes_l);
  f.d.part_A = part_A;
  f.d.part_L = part_L;
  f.x.arrivals = arrivals;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  err = fold::launch_clear_i32(arrivals, kv->num_seqs * kv->num_kv_heads, s);
  if (err != hipSuccess) return fail(FOLD_E_HIP, "scratch clear launch: %s", hipGetErrorString(err));
  err = fold::launch_decode_fused(f, kv->head_dim, s);
  if (err != hipSuccess) return fail(FOLD_E_HIP, "fused decode launch: %s", hipGetErrorString(err));
  return ok();
}

fold_status fold_value_mean(const fold_kv_view* kv, float* mean_out, void* stream) {
  if (!kv) return fail(FOLD_E_INVAL, "kv view is required");
  fold::MeanArgs a{};
  fold_status st = check_layout(kv, kv->num_seqs, kv->num_kv_heads, &a.geo);
  if (st != FOLD_OK) return st;
  if (kv->row_indptr) return fail(FOLD_E_INVAL, "the means need a per-request view (no CSR rows)");
  if (kv->num_seqs > 0 && (!kv->v || !kv->seq_lens || !mean_out))
    return fail(FOLD_E_INVAL, "v, seq_lens and mean_out are required");
  a.mean = mean_out;
  hipError_t e = fold::launch_value_mean(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "value mean launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_value_mean_append(const fold_kv_view* kv, const void* v_src,
                                   const int32_t* tok_seq, const int32_t* tok_pos,
                                   int32_t n_tok, float* mean, void* stream) {
  if (!kv) return fail(FOLD_E_INVAL, "kv view is required");
  if (n_tok < 0) return fail(FOLD_E_INVAL, "n_tok must be >= 0");
  fold::MeanArgs a{};
  fold_status st = check_layout(kv, kv->num_seqs, kv->num_kv_heads, &a.geo);
  if (st != FOLD_OK) return st;
  if (n_tok > 0 && (!v_src || !tok_seq || !tok_pos || !mean))
    return fail(FOLD_E_INVAL, "v_src, tok_seq, tok_pos and mean are required");
  if (static_cast<long long>(n_tok) * kv->num_kv_heads > 0x1fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  a.mean = mean;
  a.v_src = static_cast<const uint16_t*>(v_src);
  a.tok_seq = tok_seq;
  a.tok_pos = tok_pos;
  a.n_tok = n_tok;
  hipError_t e = fold::launch_value_mean_append(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "value mean append launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_value_block_mean(const fold_kv_view* kv, int32_t max_blocks, float* mean_out,
                                  void* stream) {
  if (!kv) return fail(FOLD_E_INVAL, "kv view is required");
  fold::MeanArgs a{};
  fold_status st = check_layout(kv, kv->num_seqs, kv->num_kv_heads, &a.geo);
  if (st != FOLD_OK) return st;
  const long long need = (static_cast<long long>(kv->max_seq_len) + fold::kTile - 1) / fold::kTile;
  if (max_blocks < need)
    return fail(FOLD_E_INVAL, "max_blocks %d < ceil(max_seq_len / 64) = %lld", max_blocks, need);
  if (kv->num_seqs > 0 && (!kv->v || !kv->seq_lens || !mean_out))
    return fail(FOLD_E_INVAL, "v, seq_lens and mean_out are required");
  if (kv->num_seqs > 0 && (!aligned16(kv->v) || !aligned16(mean_out)))
    return fail(FOLD_E_INVAL, "v and mean_out must be 16-byte aligned");
  if (static_cast<long long>(kv->num_seqs) * kv->num_kv_heads * max_blocks > 0x1fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  a.mean = mean_out;
  a.max_blocks = max_blocks;
  hipError_t e = fold::launch_block_mean(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "block mean launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_value_block_mean_append(const fold_kv_view* kv, int32_t max_blocks,
                                         const void* v_src, const int32_t* tok_seq,
                                         const int32_t* tok_pos, int32_t n_tok, float* mean,
                                         void* stream) {
  if (!kv) return fail(FOLD_E_INVAL, "kv view is required");
  if (n_tok < 0) return fail(FOLD_E_INVAL, "n_tok must be >= 0");
  if (max_blocks < 1) return fail(FOLD_E_INVAL, "max_blocks must be >= 1");
  fold::MeanArgs a{};
  fold_status st = check_layout(kv, kv->num_seqs, kv->num_kv_heads, &a.geo);
  if (st != FOLD_OK) return st;
  if (n_tok > 0 && (!v_src || !tok_seq || !tok_pos || !mean))
    return fail(FOLD_E_INVAL, "v_src, tok_seq, tok_pos and mean are required");
  if (static_cast<long long>(n_tok) * kv->num_kv_heads > 0x1fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  a.mean = mean;
  a.v_src = static_cast<const uint16_t*>(v_src);
  a.tok_seq = tok_seq;
  a.tok_pos = tok_pos;
  a.n_tok = n_tok;
  a.max_blocks = max_blocks;
  hipError_t e = fold::launch_block_mean_append(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "block mean append launch: %s", hipGetErrorString(e));
  return ok();
}

int32_t fold_q8_decode_rows_per_group(const fold_kv_view* kv, const fold_q8_query* q) {
  if (!kv || !q) return -1;
  fold::ScanGeometry g;
  if (check_layout(kv, q->batch, q->num_heads, &g) != FOLD_OK) return -1;
  return q8_rows_per_group(rows_per_seq_of(kv, q->num_heads));
}

int32_t fold_q8_decode_row_groups(const fold_kv_view* kv, const fold_q8_query* q) {
  if (!kv || !q) return -1;
  fold::ScanGeometry g;
  if (check_layout(kv, q->batch, q->num_heads, &g) != FOLD_OK) return -1;
  const int rows = rows_per_seq_of(kv, q->num_heads);
  const int gr = q8_rows_per_group(rows);
  return (rows + gr - 1) / gr;
}

fold_status fold_q8_write_keys(const fold_kv_view* kv, const void* k_src, const int32_t* tok_seq,
                               const int32_t* tok_pos, int32_t n_tok, int8_t* plane_a,
                               int8_t* plane_b, uint16_t* scale, void* stream) {
  if (!kv) return fail(FOLD_E_INVAL, "kv view is required");
  if (n_tok < 0) return fail(FOLD_E_INVAL, "n_tok must be >= 0");
  fold::Q8WriteArgs a;
  fold_status st = check_layout(kv, kv->num_seqs, kv->num_kv_heads, &a.geo);
  if (st != FOLD_OK) return st;
  if (n_tok > 0 && (!k_src || !tok_seq || !tok_pos || !plane_a || !plane_b || !scale))
    return fail(FOLD_E_INVAL, "k_src, tok_seq, tok_pos, plane_a, plane_b and scale are required");
  if (static_cast<long long>(n_tok) * kv->num_kv_heads > 0x1fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  a.k_src = static_cast<const uint16_t*>(k_src);
  a.tok_seq = tok_seq;
  a.tok_pos = tok_pos;
  a.n_tok = n_tok;
  a.ka = plane_a;
  a.kb = plane_b;
  a.ks = scale;
  hipError_t e = fold::launch_q8_write(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "q8 write launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_v8_write_values(const fold_kv_view* kv, const void* v_src,
                                 const int32_t* tok_seq, const int32_t* tok_pos, int32_t n_tok,
                                 int32_t scale_exp, uint8_t* plane_p, uint8_t* plane_r,
                                 void* stream) {
  if (!kv) return fail(FOLD_E_INVAL, "kv view is required");
  if (n_tok < 0) return fail(FOLD_E_INVAL, "n_tok must be >= 0");
  if (scale_exp < -100 || scale_exp > 100)
    return fail(FOLD_E_INVAL, "scale_exp %d out of range", scale_exp);
  fold::V8WriteArgs a;
  fold_status st = check_layout(kv, kv->num_seqs, kv->num_kv_heads, &a.geo);
  if (st != FOLD_OK) return st;
  if (n_tok > 0 && (!v_src || !tok_seq || !tok_pos || !plane_p || !plane_r))
    return fail(FOLD_E_INVAL, "v_src, tok_seq, tok_pos, plane_p and plane_r are required");
  if (static_cast<long long>(n_tok) * kv->num_kv_heads > 0x1fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  a.v_src = static_cast<const uint16_t*>(v_src);
  a.tok_seq = tok_seq;
  a.tok_pos = tok_pos;
  a.n_tok = n_tok;
  a.scale_exp = scale_exp;
  a.vp = plane_p;
  a.vr = plane_r;
  hipError_t e = fold::launch_v8_write(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "v8 write launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_q8_split_query(const fold_q_view* q, int32_t head_dim, float sm_scale,
                                const int32_t* req_lens, float kappa, float kappa_v,
                                int8_t* planes_out, float* eta_out, float* tau_out,
                                float* tau_v_out, void* stream) {
  if (!q) return fail(FOLD_E_INVAL, "q view is required");
  if (head_dim != 64 && head_dim != 128)
    return fail(FOLD_E_INVAL, "head_dim %d: must be 64 or 128", head_dim);
  if (q->batch < 0 || q->num_heads < 1) return fail(FOLD_E_INVAL, "batch >= 0, num_heads >= 1");
  const long long rows = static_cast<long long>(q->batch) * q->num_heads;
  if (rows > 0x1fffffffLL) return fail(FOLD_E_INVAL, "grid too large");
  if (rows > 0 && (!q->q || !planes_out || !eta_out))
    return fail(FOLD_E_INVAL, "q, planes_out and eta_out are required");
  if ((req_lens == nullptr) != (tau_out == nullptr))
    return fail(FOLD_E_INVAL, "req_lens and tau_out must both be set or both be NULL");
  if (!isfinite(sm_scale)) return fail(FOLD_E_INVAL, "sm_scale must be finite");
  if (isnan(kappa) || isnan(kappa_v)) return fail(FOLD_E_INVAL, "kappa and kappa_v must not be NaN");
  if (tau_v_out && !req_lens) return fail(FOLD_E_INVAL, "tau_v_out needs req_lens");
  fold::Q8SplitArgs a;
  a.q = static_cast<const uint16_t*>(q->q);
  a.qp = planes_out;
  a.eta = eta_out;
  a.rows = static_cast<int>(rows);
  a.sm_scale = sm_scale;
  a.req_lens = req_lens;
  a.tau = tau_out;
  a.tau_v = tau_v_out;
  a.batch = q->batch;
  a.kappa = kappa;
  a.kappa_v = kappa_v;
  hipError_t e = fold::launch_q8_split(a, head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "q8 split launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_q8_ref_estimate(const fold_kv_view* kv, const fold_q8_keys* keys,
                                 const fold_q8_query* q, const fold_est_params* params,
                                 float* z_out, void* stream) {
  fold::Q8EstimateArgs a;
  fold_status st = check_q8_view(kv, keys, q, &a.e.geo, false);
  if (st != FOLD_OK) return st;
  if (!z_out) return fail(FOLD_E_INVAL, "z_out is required");
  if (kv->row_indptr) return fail(FOLD_E_INVAL, "the estimate needs a per-request view (no CSR rows)");
  if (a.e.geo.group > fold::kMaxEstRows)
    return fail(FOLD_E_UNSUPPORTED, "GQA group %d exceeds %d", a.e.geo.group, fold::kMaxEstRows);
  fold_est_params p;
  st = check_est_params(params, &p);
  if (st != FOLD_OK) return st;
  if (static_cast<long long>(q->batch) * kv->num_kv_heads > 0x7fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  a.e.q = nullptr;
  a.e.z_out = z_out;
  a.e.score_scale = 0.0f;
  a.e.sink = p.sink;
  a.e.recent = p.recent;
  a.e.strata = p.strata;
  a.e.trim_lo = p.trim_lo;
  a.e.trim_hi = p.trim_hi;
  a.keys = {keys->plane_a, keys->plane_b, keys->scale};
  a.qp = q->planes;
  a.eta = q->eta;
  hipError_t e = fold::launch_q8_estimate(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "q8 estimate launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_q8_front(const fold_kv_view* kv, const fold_q8_keys* keys, const fold_q_view* q,
                          float sm_scale, const int32_t* req_lens, float kappa, float kappa_v,
                          int8_t* planes_out, float* eta_out, float* tau_out, float* tau_v_out,
                          const fold_est_params* params, float* z_out, void* stream) {
  if (!q || !q->q) return fail(FOLD_E_INVAL, "q view with query rows is required");
  if (!planes_out || !eta_out) return fail(FOLD_E_INVAL, "planes_out and eta_out are required");
  if ((req_lens == nullptr) != (tau_out == nullptr))
    return fail(FOLD_E_INVAL, "req_lens and tau_out must both be set or both be NULL");
  if (tau_v_out && !req_lens) return fail(FOLD_E_INVAL, "tau_v_out needs req_lens");
  if (!isfinite(sm_scale)) return fail(FOLD_E_INVAL, "sm_scale must be finite");
  if (isnan(kappa) || isnan(kappa_v)) return fail(FOLD_E_INVAL, "kappa and kappa_v must not be NaN");
  if (!aligned16(q->q)) return fail(FOLD_E_INVAL, "q must be 16-byte aligned");
  const fold_q8_query codes{planes_out, eta_out, tau_out, q->batch, q->num_heads, tau_v_out};
  fold::Q8EstimateArgs a{};
  fold_status st = check_q8_view(kv, keys, &codes, &a.e.geo, false);
  if (st != FOLD_OK) return st;
  if (!z_out) return fail(FOLD_E_INVAL, "z_out is required");
  if (kv->row_indptr) return fail(FOLD_E_INVAL, "the estimate needs a per-request view (no CSR rows)");
  if (a.e.geo.group > fold::kMaxEstRows)
    return fail(FOLD_E_UNSUPPORTED, "GQA group %d exceeds %d", a.e.geo.group, fold::kMaxEstRows);
  fold_est_params p;
  st = check_est_params(params, &p);
  if (st != FOLD_OK) return st;
  if (static_cast<long long>(q->batch) * kv->num_kv_heads > 0x7fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  a.e.q = nullptr;
  a.e.z_out = z_out;
  a.e.score_scale = 0.0f;
  a.e.sink = p.sink;
  a.e.recent = p.recent;
  a.e.strata = p.strata;
  a.e.trim_lo = p.trim_lo;
  a.e.trim_hi = p.trim_hi;
  a.keys = {keys->plane_a, keys->plane_b, keys->scale};
  a.qp = planes_out;
  a.eta = eta_out;
  a.q_src = static_cast<const uint16_t*>(q->q);
  a.qp_out = planes_out;
  a.eta_out = eta_out;
  a.sm_scale = sm_scale;
  a.req_lens = req_lens;
  a.tau = tau_out;
  a.tau_v = tau_v_out;
  a.kappa = kappa;
  a.kappa_v = kappa_v;
  hipError_t e = fold::launch_q8_front(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "q8 front launch: %s", hipGetErrorString(e));
  return ok();
}


fold_status fold_q8_decode_split(const fold_kv_view* kv, const fold_q8_keys* keys,
                                 const fold_q8_query* q, const fold_v8_values* values,
                                 const float* z, float depth_T, int32_t num_splits,
                                 int32_t slot_offset, int32_t num_slots, float* part_A,
                                 float* part_L, float* part_Lcut, const fold_q8_debug* dbg,
                                 void* stream) {
  fold::Q8DecodeArgs a;
  fold_status st = check_q8_view(kv, keys, q, &a.d.geo, values == nullptr);
  if (st != FOLD_OK) return st;
  if (!q->tau) return fail(FOLD_E_INVAL, "tau is required");
  a.vp = nullptr;
  a.vr = nullptr;
  a.v_scale = 1.0f;
  a.tau_v = nullptr;
  if (values) {
    if (!values->plane_p || !values->plane_r || !q->tau_v)
      return fail(FOLD_E_INVAL, "8-bit values need plane_p, plane_r and q->tau_v");
    if (!aligned16(values->plane_p) || !aligned16(values->plane_r))
      return fail(FOLD_E_INVAL, "value planes must be 16-byte aligned");
    if (values->scale_exp < -100 || values->scale_exp > 100)
      return fail(FOLD_E_INVAL, "scale_exp %d out of range", values->scale_exp);
    a.vp = values->plane_p;
    a.vr = values->plane_r;
    a.v_scale = ldexpf(1.0f, values->scale_exp);
    a.tau_v = q->tau_v;
  }
  if (!z || !part_A || !part_L) return fail(FOLD_E_INVAL, "z, part_A and part_L are required");
  st = check_depth(depth_T);
  if (st != FOLD_OK) return st;
  if (num_splits < 1) return fail(FOLD_E_INVAL, "num_splits must be >= 1");
  if (slot_offset < 0 || static_cast<long long>(slot_offset) + num_splits > num_slots)
    return fail(FOLD_E_INVAL, "slots [%d, %d) exceed num_slots %d", slot_offset,
                slot_offset + num_splits, num_slots);
  const int rows = rows_per_seq_of(kv, q->num_heads);
  const int gr = q8_rows_per_group(rows);
  const int groups = (rows + gr - 1) / gr;
  const long long blocks = static_cast<long long>(kv->num_seqs) * kv->num_kv_heads * num_splits * groups;
  if (blocks > 0x7fffffffLL) return fail(FOLD_E_INVAL, "grid too large");
  a.d.q = nullptr;
  a.d.z = z;
  a.d.part_A = part_A;
  a.d.part_L = part_L;
  a.d.part_Lcut = part_Lcut;
  a.d.x_out = dbg ? dbg->x_out : nullptr;
  a.d.key_gate_out = dbg ? dbg->key_gate_out : nullptr;
  a.d.page_gate_out = dbg ? dbg->page_gate_out : nullptr;
  a.d.score_scale = 0.0f;
  a.d.dense = isinf(depth_T) ? 1 : 0;
  a.d.neg_T = a.d.dense ? 0.0f : -depth_T;
  a.d.num_splits = num_splits;
  a.d.slot_offset = slot_offset;
  a.d.rows_per_seq = rows;
  a.d.rows_per_group = gr;
  a.d.row_groups = groups;
  a.d.by_length = (gr == 1 && !kv->row_indptr && kv->num_seqs >= 2 &&
                   kv->num_seqs <= fold::kOrderMax) ? 1 : 0;
  a.keys = {keys->plane_a, keys->plane_b, keys->scale};
  a.qp = q->planes;
  a.eta = q->eta;
  a.tau = q->tau;
  a.xc_out = dbg ? dbg->xc_out : nullptr;
  a.refine_gate_out = dbg ? dbg->refine_gate_out : nullptr;
  a.refine_v_gate_out = dbg ? dbg->refine_v_gate_out : nullptr;
  hipError_t e = fold::launch_q8_decode(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "q8 decode launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_q8_stack_keys(const fold_kv_view* kv, const fold_q8_keys* keys, uint16_t* k_f16,
                               void* stream) {
  if (!kv || !keys) return fail(FOLD_E_INVAL, "kv view and keys are required");
  fold::Q8StackArgs a;
  fold_status st = check_layout(kv, kv->num_seqs, kv->num_kv_heads, &a.geo);
  if (st != FOLD_OK) return st;
  if (kv->num_seqs == 0) return ok();
  if (!kv->seq_lens || !keys->plane_a || !keys->plane_b || !keys->scale || !k_f16)
    return fail(FOLD_E_INVAL, "seq_lens, plane_a, plane_b, scale and k_f16 are required");
  if (!aligned16(keys->plane_a) || !aligned16(keys->plane_b) || !aligned16(k_f16))
    return fail(FOLD_E_INVAL, "planes and k_f16 must be 16-byte aligned");
  const long long per = (static_cast<long long>(fold::view_capacity(a.geo)) + 31) / 16;
  if (static_cast<long long>(kv->num_seqs) * kv->num_kv_heads * per > 0x7fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  a.ka = keys->plane_a;
  a.kb = keys->plane_b;
  a.ks = keys->scale;
  a.out = k_f16;
  hipError_t e = fold::launch_q8_stack_keys(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "stack keys launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_q8_decode_stacked(const fold_kv_view* kv, const fold_q8_query* q, const float* z,
                                   float depth_T, int32_t num_splits, int32_t slot_offset,
                                   int32_t num_slots, float* part_A, float* part_L,
                                   float* part_Lcut, const fold_debug* dbg, void* stream) {
  if (!kv || !q) return fail(FOLD_E_INVAL, "kv view and q are required");
  fold::DecodeArgs a;
  fold_status st = check_layout(kv, q->batch, q->num_heads, &a.geo);
  if (st != FOLD_OK) return st;
  if (!kv->k || !kv->v || !kv->seq_lens || !q->planes || !q->eta)
    return fail(FOLD_E_INVAL, "k (the FP16 keys), v, seq_lens, query planes and eta are required");
  if (!aligned16(kv->k) || !aligned16(kv->v) || !aligned16(q->planes))
    return fail(FOLD_E_INVAL, "k, v and the query planes must be 16-byte aligned");
  if (!z || !part_A || !part_L) return fail(FOLD_E_INVAL, "z, part_A and part_L are required");
  st = check_depth(depth_T);
  if (st != FOLD_OK) return st;
  if (num_splits < 1) return fail(FOLD_E_INVAL, "num_splits must be >= 1");
  if (slot_offset < 0 || static_cast<long long>(slot_offset) + num_splits > num_slots)
    return fail(FOLD_E_INVAL, "slots [%d, %d) exceed num_slots %d", slot_offset,
                slot_offset + num_splits, num_slots);
  const int rows = rows_per_seq_of(kv, q->num_heads);
  const int gr = fold::decode_rows_per_group(rows);
  if (gr != 64)
    return fail(FOLD_E_UNSUPPORTED, "%d rows per kv sequence: the stacked level needs more than "
                "32 (use fold_q8_decode_split)", rows);
  const int groups = (rows + gr - 1) / gr;
  const long long blocks = static_cast<long long>(kv->num_seqs) * kv->num_kv_heads * num_splits * groups;
  if (blocks > 0x7fffffffLL) return fail(FOLD_E_INVAL, "grid too large");
  a.q = nullptr;
  a.z = z;
  a.part_A = part_A;
  a.part_L = part_L;
  a.part_Lcut = part_Lcut;
  a.x_out = dbg ? dbg->x_out : nullptr;
  a.key_gate_out = dbg ? dbg->key_gate_out : nullptr;
  a.page_gate_out = dbg ? dbg->page_gate_out : nullptr;
  a.score_scale = 0.0f;
  a.dense = isinf(depth_T) ? 1 : 0;
  a.neg_T = a.dense ? 0.0f : -depth_T;
  a.num_splits = num_splits;
  a.slot_offset = slot_offset;
  a.rows_per_seq = rows;
  a.rows_per_group = gr;
  a.row_groups = groups;
  a.qplanes = q->planes;
  a.qeta = q->eta;
  hipError_t e = fold::launch_decode(a, kv->head_dim, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "stacked decode launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_append_kv(const fold_kv_view* kv, const void* k_src, const void* v_src,
                           const int32_t* tok_seq, const int32_t* tok_pos, int32_t n_tok,
                           void* k_cache, void* v_cache, void* stream) {
  if (!kv) return fail(FOLD_E_INVAL, "kv view is required");
  if (n_tok < 0) return fail(FOLD_E_INVAL, "n_tok must be >= 0");
  fold::AppendArgs a;
  fold_status st = check_layout(kv, kv->num_seqs, kv->num_kv_heads, &a.geo);
  if (st != FOLD_OK) return st;
  if (n_tok > 0) {
    if (!tok_seq || !tok_pos) return fail(FOLD_E_INVAL, "tok_seq and tok_pos are required");
    if ((k_cache && !k_src) || (v_cache && !v_src))
      return fail(FOLD_E_INVAL, "a written cache needs its source rows");
    if ((k_cache && (!aligned16(k_cache) || !aligned16(k_src))) ||
        (v_cache && (!aligned16(v_cache) || !aligned16(v_src))))
      return fail(FOLD_E_INVAL, "caches and source rows must be 16-byte aligned");
  }
  if (static_cast<long long>(n_tok) * kv->num_kv_heads > 0x1fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  a.k_src = static_cast<const uint8_t*>(k_src);
  a.v_src = static_cast<const uint8_t*>(v_src);
  a.k_dst = static_cast<uint8_t*>(k_cache);
  a.v_dst = static_cast<uint8_t*>(v_cache);
  a.tok_seq = tok_seq;
  a.tok_pos = tok_pos;
  a.n_tok = (k_cache || v_cache) ? n_tok : 0;
  a.row_bytes = 2 * kv->head_dim;
  hipError_t e = fold::launch_append_rows(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "append launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_cert_update(const uint8_t* cert, const float* lse, float* z, int32_t num_rows,
                             int32_t* reruns, int32_t* count_out, void* stream) {
  if (num_rows < 0) return fail(FOLD_E_INVAL, "num_rows must be >= 0");
  if (!count_out) return fail(FOLD_E_INVAL, "count_out is required");
  if (num_rows > 0 && (!cert || !lse || !z))
    return fail(FOLD_E_INVAL, "cert, lse and z are required");
  fold::CertArgs a{cert, lse, z, reruns, count_out, num_rows};
  hipError_t e = fold::launch_cert_update(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "certificate update launch: %s", hipGetErrorString(e));
  return ok();
}

fold_status fold_draft_plan(int32_t num_seqs, const int32_t* seq_lens, const int32_t* col_indptr,
                            const int32_t* parent, int32_t page_size, int32_t pages_per_col,
                            int32_t* committed_lens, int32_t* col_req, int32_t* col_lens,
                            int32_t* anc_lens, int32_t* anc_pos) {
  if (num_seqs < 0) return fail(FOLD_E_INVAL, "num_seqs must be >= 0");
  if (page_size < 1 || pages_per_col < 1)
    return fail(FOLD_E_INVAL, "page_size and pages_per_col must be positive");
  if (static_cast<long long>(page_size) * pages_per_col > (1 << 20))
    return fail(FOLD_E_INVAL, "pages_per_col * page_size too large");
  if (!col_indptr || (num_seqs > 0 && (!seq_lens || !committed_lens)))
    return fail(FOLD_E_INVAL, "seq_lens, col_indptr and committed_lens are required");
  if (col_indptr[0] != 0) return fail(FOLD_E_INVAL, "col_indptr[0] must be 0");
  for (int r = 0; r < num_seqs; ++r) {
    const int m = col_indptr[r + 1] - col_indptr[r];
    if (m < 0) return fail(FOLD_E_INVAL, "col_indptr decreases at request %d", r);
    if (seq_lens[r] < m)
      return fail(FOLD_E_INVAL, "request %d holds %d keys but has %d drafts", r, seq_lens[r], m);
  }
  const int cols = num_seqs > 0 ? col_indptr[num_seqs] : 0;
  if (cols > 0 && (!parent || !col_req || !col_lens || !anc_lens || !anc_pos))
    return fail(FOLD_E_INVAL, "parent, col_req, col_lens, anc_lens and anc_pos are required");
  const int cap = page_size * pages_per_col;
  for (int r = 0; r < num_seqs; ++r) {
    const int c0 = col_indptr[r];
    const int m = col_indptr[r + 1] - c0;
    for (int c = 0; c < m; ++c) {
      const int p = parent[c0 + c];
      if (p < -1 || p >= c)
        return fail(FOLD_E_INVAL, "parent[%d] = %d: must be in [-1, %d)", c0 + c, p, c);
    }
    for (int c = 0; c < m; ++c) {  // parents precede their children: every walk ends
      int depth = 0;
      for (int t = c; t >= 0; t = parent[c0 + t]) ++depth;
      if (depth > cap)
        return fail(FOLD_E_INVAL, "column %d has %d ancestors: more than the %d spare slots",
                    c0 + c, depth, cap);
    }
  }
  // every check passed: write the plan
  std::vector<int> path;
  for (int r = 0; r < num_seqs; ++r) {
    const int c0 = col_indptr[r];
    const int m = col_indptr[r + 1] - c0;
    const int n0 = seq_lens[r] - m;
    committed_lens[r] = n0;
    for (int c = 0; c < m; ++c) {
      path.clear();
      for (int t = c; t >= 0; t = parent[c0 + t]) path.push_back(t);
      std::sort(path.begin(), path.end());
      const int col = c0 + c;
      col_req[col] = r;
      col_lens[col] = n0;
      anc_lens[col] = static_cast<int32_t>(path.size());
      int32_t* out = anc_pos + static_cast<size_t>(col) * cap;
      for (int i = 0; i < cap; ++i)
        out[i] = i < static_cast<int>(path.size()) ? n0 + path[i] : -1;
    }
  }
  return ok();
}

fold_status fold_draft_gather(const fold_kv_view* kv, const int32_t* col_req,
                              const int32_t* anc_lens, const int32_t* anc_pos,
                              const int32_t* spare_pages, int32_t num_cols,
                              int32_t pages_per_col, int32_t row_bytes, const void* src,
                              void* dst, int32_t* col_block_table, void* stream) {
  if (!kv) return fail(FOLD_E_INVAL, "kv view is required");
  if (num_cols < 0) return fail(FOLD_E_INVAL, "num_cols must be >= 0");
  fold::DraftGatherArgs a;
  fold_status st = check_layout(kv, kv->num_seqs, kv->num_kv_heads, &a.geo);
  if (st != FOLD_OK) return st;
  if (!kv->block_table) return fail(FOLD_E_INVAL, "drafts need a paged view");
  if (pages_per_col < 1) return fail(FOLD_E_INVAL, "pages_per_col must be positive");
  if (static_cast<long long>(pages_per_col) * kv->page_size > (1 << 20))
    return fail(FOLD_E_INVAL, "pages_per_col * page_size too large");
  if (row_bytes < 1 || row_bytes > 4096)
    return fail(FOLD_E_INVAL, "row_bytes %d: must be in [1, 4096]", row_bytes);
  if ((src == nullptr) != (dst == nullptr))
    return fail(FOLD_E_INVAL, "src and dst must both be set or both be NULL");
  if (num_cols > 0 && (!col_req || !anc_lens || !anc_pos || !spare_pages))
    return fail(FOLD_E_INVAL, "col_req, anc_lens, anc_pos and spare_pages are required");
  const uintptr_t align = (row_bytes % 16 == 0) ? 16 : (row_bytes % 2 == 0 ? 2 : 1);
  if (src && ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % align))
    return fail(FOLD_E_INVAL, "src and dst must be %zu-byte aligned", static_cast<size_t>(align));
  if (static_cast<long long>(num_cols) * kv->num_kv_heads > 0x1fffffffLL)
    return fail(FOLD_E_INVAL, "grid too large");
  a.col_req = col_req;
  a.anc_lens = anc_lens;
  a.anc_pos = anc_pos;
  a.spare_pages = spare_pages;
  a.col_block_table = col_block_table;
  a.src = static_cast<const uint8_t*>(src);
  a.dst = static_cast<uint8_t*>(dst);
  a.num_cols = (src || col_block_table) ? num_cols : 0;
  a.pages_per_col = pages_per_col;
  a.row_bytes = row_bytes;
  hipError_t e = fold::launch_draft_gather(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FOLD_E_HIP, "draft gather launch: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"
