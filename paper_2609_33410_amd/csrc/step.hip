// The decode step around the scan: BF16 token append, the certificate's
// reference update, and the row gather that lays out draft columns.
//
// * append: the front writes each step's new token into the paged cache
//   (Section 4, "Weight-gated reads").
// * certificate update (Section 3, certificate paragraph): a flagged row is
//   decoded again with Z = its base-2 log-sum-exp; where that is not finite
//   (L formed as 0 or infinity) Z moves 64 binades towards it.
// * draft gather (Section 4, "Value product": drafts are query columns masked
//   to their ancestors): each column's ancestor keys are copied into spare
//   pages, so that the column's visible keys are the committed keys (shared
//   by every column of the request) plus a private level of its own.
//
// All three are latency-bound: a wave per (item, kv head) moving one row of
// at most 256 bytes, or one block for the update.

#include "fold_internal.h"
#include "fold_device.h"

namespace fold {
namespace {

constexpr int kStepThreads = 256;
constexpr int kStepWaves = kStepThreads / 64;
constexpr float kCertStep = 64.0f;

// Copy one row with the widest unit its size allows; both rows start at a
// multiple of row_bytes from a 16-byte aligned base.
__device__ __forceinline__ void copy_row(uint8_t* dst, const uint8_t* src, int row_bytes,
                                         int lane) {
  if ((row_bytes & 15) == 0) {
    for (int i = lane; i < (row_bytes >> 4); i += 64)
      reinterpret_cast<uint4*>(dst)[i] = reinterpret_cast<const uint4*>(src)[i];
  } else if ((row_bytes & 1) == 0) {
    for (int i = lane; i < (row_bytes >> 1); i += 64)
      reinterpret_cast<uint16_t*>(dst)[i] = reinterpret_cast<const uint16_t*>(src)[i];
  } else {
    for (int i = lane; i < row_bytes; i += 64) dst[i] = src[i];
  }
}

// Element-row index of (sequence, position, kv head) in the view's layout,
// or -1 when the view cannot address it.
__device__ __forceinline__ long long row_of(const ScanGeometry& g, int seq, int pos, int kvh) {
  if (seq < 0 || seq >= g.num_seqs || pos < 0 || pos >= view_capacity(g)) return -1;
  if (g.page_size > 0) {
    const int phys =
        ld_uniform(g.block_table, static_cast<size_t>(seq) * g.max_pages + pos / g.page_size);
    if (phys < 0 || phys >= g.num_pages) return -1;
    return (static_cast<long long>(phys) * g.hkv + kvh) * g.page_size + pos % g.page_size;
  }
  return (static_cast<long long>(seq) * g.hkv + kvh) * g.max_seq_len + pos;
}

__global__ __launch_bounds__(kStepThreads) void append_rows_kernel(const AppendArgs a) {
  const int lane = threadIdx.x & 63;
  const long long item = static_cast<long long>(blockIdx.x) * kStepWaves +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (item >= static_cast<long long>(a.n_tok) * a.geo.hkv) return;  // uniform per wave
  const int tok = static_cast<int>(item / a.geo.hkv);
  const int kvh = static_cast<int>(item % a.geo.hkv);
  const long long row = row_of(a.geo, ld_uniform(a.tok_seq, tok), ld_uniform(a.tok_pos, tok), kvh);
  if (row < 0) return;
  const size_t src = static_cast<size_t>(item) * a.row_bytes;
  const size_t dst = static_cast<size_t>(row) * a.row_bytes;
  if (a.k_dst) copy_row(a.k_dst + dst, a.k_src + src, a.row_bytes, lane);
  if (a.v_dst) copy_row(a.v_dst + dst, a.v_src + src, a.row_bytes, lane);
}

__global__ __launch_bounds__(kStepThreads) void cert_update_kernel(const CertArgs a) {
  __shared__ int partial[kStepWaves];
  int flagged = 0;
  for (int i = threadIdx.x; i < a.n; i += kStepThreads) {
    if (a.cert[i] == 0) continue;
    const float l = a.lse[i];
    const float z = a.z[i];
    float nz = z;  // NaN: no better reference is known
    if (isfinite(l))
      nz = l;
    else if (l < 0.0f)
      nz = z - kCertStep;
    else if (l > 0.0f)
      nz = z + kCertStep;
    a.z[i] = nz;
    if (a.reruns) a.reruns[i] += 1;
    ++flagged;
  }
  for (int off = 32; off > 0; off >>= 1) flagged += __shfl_xor(flagged, off);
  if ((threadIdx.x & 63) == 0) partial[threadIdx.x >> 6] = flagged;
  __syncthreads();
  if (threadIdx.x == 0) {
    int total = 0;
    for (int w = 0; w < kStepWaves; ++w) total += partial[w];
    a.count[0] = total;
  }
}

// One wave per (column, kv head): copy the column's ancestor rows into its
// spare pages; the kv head 0 wave also copies the request's block-table row
// into the column's table when one is requested.
__global__ __launch_bounds__(kStepThreads) void draft_gather_kernel(const DraftGatherArgs a) {
  const int lane = threadIdx.x & 63;
  const long long item = static_cast<long long>(blockIdx.x) * kStepWaves +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (item >= static_cast<long long>(a.num_cols) * a.geo.hkv) return;  // uniform per wave
  const int col = static_cast<int>(item / a.geo.hkv);
  const int kvh = static_cast<int>(item % a.geo.hkv);
  const int req = ld_uniform(a.col_req, col);
  const int cap = a.pages_per_col * a.geo.page_size;
  int n = ld_uniform(a.anc_lens, col);
  n = n < 0 ? 0 : (n > cap ? cap : n);
  if (a.col_block_table && kvh == 0 && req >= 0 && req < a.geo.num_seqs) {
    for (int p = lane; p < a.geo.max_pages; p += 64)
      a.col_block_table[static_cast<size_t>(col) * a.geo.max_pages + p] =
          a.geo.block_table[static_cast<size_t>(req) * a.geo.max_pages + p];
  }
  if (!a.src || !a.dst) return;
  for (int i = 0; i < n; ++i) {
    const int pos = ld_uniform(a.anc_pos, static_cast<size_t>(col) * cap + i);
    const long long src = row_of(a.geo, req, pos, kvh);
    const int spare =
        ld_uniform(a.spare_pages, static_cast<size_t>(col) * a.pages_per_col + i / a.geo.page_size);
    if (src < 0 || spare < 0 || spare >= a.geo.num_pages) continue;
    const long long dst =
        (static_cast<long long>(spare) * a.geo.hkv + kvh) * a.geo.page_size + i % a.geo.page_size;
    copy_row(a.dst + static_cast<size_t>(dst) * a.row_bytes,
             a.src + static_cast<size_t>(src) * a.row_bytes, a.row_bytes, lane);
  }
}

}  // namespace

hipError_t launch_append_rows(const AppendArgs& a, hipStream_t stream) {
  const long long items = static_cast<long long>(a.n_tok) * a.geo.hkv;
  if (items == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((items + kStepWaves - 1) / kStepWaves);
  hipLaunchKernelGGL(append_rows_kernel, dim3(blocks), dim3(kStepThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_cert_update(const CertArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(cert_update_kernel, dim3(1), dim3(kStepThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_draft_gather(const DraftGatherArgs& a, hipStream_t stream) {
  const long long items = static_cast<long long>(a.num_cols) * a.geo.hkv;
  if (items == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((items + kStepWaves - 1) / kStepWaves);
  hipLaunchKernelGGL(draft_gather_kernel, dim3(blocks), dim3(kStepThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace fold
