// Internal launch interface between the C ABI (fold_api.cpp) and the HIP
// kernels.  Not installed; the public contract is include/fold.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fold {

// Keys per split-interleave tile and per page-gate bit (Section 4: splits
// interleave by 64-key tiles; pages are 16 keys).
constexpr int kTile = 64;
constexpr int kChunk = 16;
// Largest per-request view whose scan dispatches its sequences by decreasing
// length (each workgroup ranks the lengths itself).
constexpr int kOrderMax = 64;

struct ScanGeometry {
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const int32_t* row_indptr;
  const int32_t* row_req;
  int num_seqs;
  int hkv;
  int page_size;   // 0 => contiguous
  int max_pages;
  int num_pages;
  int max_seq_len;
  int batch;
  int heads;
  int group;       // heads / hkv
};

struct DecodeArgs {
  ScanGeometry geo;
  const uint16_t* q;
  const float* z;
  float* part_A;
  float* part_L;
  float* part_Lcut;   // cut keys' summed weights per slot and row, or NULL
  float* x_out;
  uint8_t* key_gate_out;
  uint8_t* page_gate_out;
  float score_scale;  // log2(e) * sm_scale
  float neg_T;        // -T (finite depth) ; unused when dense
  int dense;          // T == +inf
  int num_splits;
  int slot_offset;
  int rows_per_seq;   // bound on rows attending one (kv seq, kv head)
  int rows_per_group; // rows one workgroup serves (template GR)
  int row_groups;
  int by_length = 0;  // block order over sequences by decreasing length (per-request views)
  // Block model of BF16 values: the scan also writes each row's cut mass of
  // every 16-key chunk, chunk_cut[row * chunk_stride + chunk] (finite depth).
  float* chunk_cut = nullptr;
  int chunk_stride = 0;  // ceil(max_seq_len / 16)
  // Stacked level of a two-plane key cache: geo.k holds the FP16 keys
  // fp16(e (a + b/256)); the query operand is fp16(qa + qb/256) from the
  // query codes and the score scale is eta per row (q is not read).
  const int8_t* qplanes = nullptr;  // [batch][heads][2][D]
  const float* qeta = nullptr;      // [batch][heads]
  // Cascade in one scan (stacked prefix level only): the 64-key tiles of the
  // suffixes of a read group's requests ride in the prefix workgroups, after
  // the prefix tiles.  The suffixes are a per-request view over the same
  // pages (request r's suffix: sfx_seq_lens[r] keys, block-table row r).
  const int32_t* sfx_block_table = nullptr;  // [batch][sfx_max_pages]
  const int32_t* sfx_seq_lens = nullptr;     // [batch]
  int sfx_max_pages = 0;
  int sfx_cap = 0;    // keys a suffix can hold
  int sfx_tiles = 0;  // 64-key tiles of the longest suffix (0: no suffix)
};

struct EstimateArgs {
  ScanGeometry geo;
  const uint16_t* q;
  float* z_out;
  float score_scale;
  int sink, recent, strata, trim_lo, trim_hi;
};

struct CombineArgs {
  const float* part_A;
  const float* part_L;
  const float* part_Lcut;  // value model: cut masses per slot and row, or NULL
  const float* mean;       // value model: [batch][hkv][D] request means
  int heads, hkv;          // value model: rows are [batch][heads]
  const float* z;
  void* out;
  float* lse_out;
  uint8_t* cert_out;
  int num_slots;
  int num_rows;
  int head_dim;
  int out_bf16;
};

// Request mean value rows (the cut-key value model).
struct MeanArgs {
  ScanGeometry geo;       // per-request view (geo.k unused)
  float* mean;            // [num_seqs][hkv][D], or block means [num_seqs][hkv][max_blocks][D]
  const uint16_t* v_src;  // append: [n_tok][hkv][D] bf16
  const int32_t* tok_seq;
  const int32_t* tok_pos;
  int n_tok;
  int max_blocks;         // block means: row stride in blocks
};

// Virtual rows of the block model: adds sum over the split's tiles t of
// c_it * mu_t to the split's slot of every row of the level (after the scan).
struct BlockModelArgs {
  ScanGeometry geo;
  float* part_A;              // the scan's slots
  const float* chunk_cut;     // [batch * heads][chunk_stride] cut masses per 16-key chunk
  const float* block_mean;    // [num_seqs][hkv][max_blocks][D]
  int chunk_stride;
  int max_blocks;
  int num_splits;
  int slot_offset;
  int rows_per_seq;           // host bound on rows attending one (kv seq, kv head)
  int row_tiles;              // row blocks of RB rows per (kv seq, kv head)
};

// Two-plane INT8 key cache (Section 4, "Cache format"): the planes use the
// element layout of a BF16 key cache with one byte per element; the BF16
// scales one element per key.
struct Q8Keys {
  const int8_t* ka;
  const int8_t* kb;
  const uint16_t* ks;
};

struct Q8DecodeArgs {
  DecodeArgs d;           // d.geo.k and d.q are not read; d.x_out holds the refined x
  Q8Keys keys;
  const int8_t* qp;       // [batch][heads][2][D]: qa then qb
  const float* eta;       // [batch][heads]
  const float* tau;       // [batch] refine thresholds
  float* xc_out;          // coarse x (debug)
  uint8_t* refine_gate_out;
  // 8-bit values (NULL vp: BF16 values from d.geo.v)
  const uint8_t* vp;      // plane 1, one byte per element
  const uint8_t* vr;      // plane 2 (residual x 16)
  float v_scale;          // 2^scale_exp
  const float* tau_v;     // [batch] refine-V thresholds
  uint8_t* refine_v_gate_out;
};

struct Q8WriteArgs {
  ScanGeometry geo;       // layout of the destination cache (geo.k, geo.v unused)
  const uint16_t* k_src;  // [n_tok][hkv][D] bf16
  const int32_t* tok_seq;
  const int32_t* tok_pos;
  int n_tok;
  int8_t* ka;
  int8_t* kb;
  uint16_t* ks;
};

struct V8WriteArgs {
  ScanGeometry geo;       // layout of the destination cache
  const uint16_t* v_src;  // [n_tok][hkv][D] bf16
  const int32_t* tok_seq;
  const int32_t* tok_pos;
  int n_tok;
  int scale_exp;          // values are stored as 2^scale_exp (p + r/16)
  uint8_t* vp;
  uint8_t* vr;
};

struct AppendArgs {
  ScanGeometry geo;       // layout of the destination cache (geo.k, geo.v unused)
  const uint8_t* k_src;   // [n_tok][hkv][row_bytes]
  const uint8_t* v_src;
  uint8_t* k_dst;         // cache arrays written (either may be null)
  uint8_t* v_dst;
  const int32_t* tok_seq;
  const int32_t* tok_pos;
  int n_tok;
  int row_bytes;          // bytes of one (token, kv head) row
};

struct CertArgs {
  const uint8_t* cert;    // [n] certificate bits of the last decode
  const float* lse;       // [n] base-2 log-sum-exp of the last decode
  float* z;               // [n] references, updated in place for flagged rows
  int32_t* reruns;        // [n] or null: incremented for flagged rows
  int32_t* count;         // [1] number of flagged rows
  int n;
};

struct DraftGatherArgs {
  ScanGeometry geo;       // the requests' paged view (source layout; pool size)
  const int32_t* col_req;      // [num_cols] request of each column
  const int32_t* anc_lens;     // [num_cols]
  const int32_t* anc_pos;      // [num_cols][pages_per_col * page_size] positions
  const int32_t* spare_pages;  // [num_cols][pages_per_col]
  int32_t* col_block_table;    // [num_cols][max_pages] or null
  const uint8_t* src;          // pool array read (may alias dst), or null
  uint8_t* dst;
  int num_cols;
  int pages_per_col;
  int row_bytes;
};

struct Q8SplitArgs {
  const uint16_t* q;      // [rows][D] bf16
  int8_t* qp;             // [rows][2][D]
  float* eta;             // [rows]
  int rows;
  float sm_scale;
  const int32_t* req_lens;  // [batch] or NULL
  float* tau;               // [batch] or NULL: refine-K thresholds
  float* tau_v;             // [batch] or NULL: refine-V thresholds
  int batch;
  float kappa;
  float kappa_v;
};

struct Q8EstimateArgs {
  EstimateArgs e;         // e.geo.k and e.q are not read
  Q8Keys keys;
  const int8_t* qp;
  const float* eta;
  // Fused front (the query split in the same launch; q_src non-NULL): the
  // codes of each (request, kv head)'s rows are computed from q_src, written
  // to qp_out / eta_out and scored from LDS; the thresholds as Q8SplitArgs.
  const uint16_t* q_src;  // [batch][heads][D] bf16
  int8_t* qp_out;         // [batch][heads][2][D]
  float* eta_out;         // [batch][heads]
  float sm_scale;
  const int32_t* req_lens;
  float* tau;
  float* tau_v;
  float kappa;
  float kappa_v;
};

// The one-launch decode of a single level over a per-request view: every
// split's workgroup computes its (request, kv head)'s reference in its
// prologue (the estimate routine, the same bits as the estimate kernel), and
// the last split to finish adds the slots (the combine's order and bits).
struct FusedExtra {
  Q8EstimateArgs est;   // the estimate of the scan's view (est.e.z_out: Z)
  int32_t* arrivals;    // [num_seqs][hkv]: zero before a call, zero after it
  void* out;            // [batch][heads][D] fp32 or bf16
  float* lse_out;       // [batch][heads] or NULL
  uint8_t* cert_out;    // [batch][heads] or NULL
  int out_bf16;
};

struct FusedArgs {
  DecodeArgs d;         // the scan (d.z is not read; d.part_Lcut is NULL)
  FusedExtra x;
};

// Keys a kv sequence of this view can hold: max_seq_len, and for a paged view
// also max_pages * page_size.  Device-supplied lengths are clamped to it.
__host__ __device__ inline int view_capacity(const ScanGeometry& g) {
  if (g.page_size > 0) {
    const long long paged = static_cast<long long>(g.max_pages) * g.page_size;
    return paged < g.max_seq_len ? static_cast<int>(paged) : g.max_seq_len;
  }
  return g.max_seq_len;
}

// Each returns hipSuccess or the launch error.
hipError_t launch_decode(const DecodeArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_estimate(const EstimateArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_combine(const CombineArgs& a, hipStream_t stream);
hipError_t launch_q8_decode(const Q8DecodeArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_q8_front(const Q8EstimateArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_decode_fused(const FusedArgs& a, int head_dim, hipStream_t stream);
// Prefix and suffix levels of a shared-prefix cascade in one stacked scan
// (decode_stacked.hip); every workgroup's tiles must fit one 64-tile window.
hipError_t launch_decode_cascade(const DecodeArgs& a, int head_dim, hipStream_t stream);
// The library's fixed device scratch (noalloc.hip): its capacity in bytes, its
// address on the current device (looked up once per device), and a fill
// kernel that zeroes n int32 values of it.
size_t scratch_capacity();
hipError_t scratch_device_ptr(void** out);
hipError_t launch_clear_i32(int32_t* p, int n, hipStream_t stream);
hipError_t launch_value_mean(const MeanArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_value_mean_append(const MeanArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_block_mean(const MeanArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_block_mean_append(const MeanArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_block_model(const BlockModelArgs& a, int head_dim, hipStream_t stream);
// The stacked level's FP16 keys of a two-plane cache (q8_front.hip).
struct Q8StackArgs {
  ScanGeometry geo;       // the level's view (its sequences' keys are converted)
  const int8_t* ka;
  const int8_t* kb;
  const uint16_t* ks;
  uint16_t* out;          // FP16 bits, the element layout of the planes
};
hipError_t launch_q8_stack_keys(const Q8StackArgs& a, int head_dim, hipStream_t stream);
// Rows per workgroup of the block model's virtual-row kernel for a bound on
// the rows attending one (kv sequence, kv head).
int block_model_rows(int rows_per_seq);
hipError_t launch_q8_write(const Q8WriteArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_q8_split(const Q8SplitArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_v8_write(const V8WriteArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_q8_estimate(const Q8EstimateArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_append_rows(const AppendArgs& a, hipStream_t stream);
hipError_t launch_cert_update(const CertArgs& a, hipStream_t stream);
hipError_t launch_draft_gather(const DraftGatherArgs& a, hipStream_t stream);

// Rows per read group the decode kernel is instantiated for, given the rows
// that attend one (kv sequence, kv head).
int decode_rows_per_group(int rows_per_seq);

// Largest estimator sample the kernel's LDS holds.
constexpr int kMaxEstSamples = 512;
constexpr int kMaxEstRows = 16;

}  // namespace fold
