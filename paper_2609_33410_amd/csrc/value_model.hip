// Request mean value rows for the cut-key value model (Section 4, "Depth as a
// dial": cut keys are modelled by the request's running mean, which needs no
// fit).
//
// value_mean_kernel: one workgroup of 16 wave64s per (kv sequence, kv head) of
// a per-request view.  Wave w adds the value rows of keys w, w + 16, ...; lane l
// owns channels [l D/64, (l + 1) D/64), so a key row is one coalesced read.  The
// waves' sums are added in wave order through LDS and divided by the length.
// Bound by HBM bandwidth over the request's values (a prompt-time call).
//
// value_mean_append_kernel: one wave64 per (token, kv head): the running
// update mu += (v - mu) / (pos + 1) for a token appended at position pos.
#include "fold_device.h"
#include "fold_internal.h"

namespace fold {
namespace {

constexpr int kMeanWaves = 16;
constexpr int kMeanThreads = 64 * kMeanWaves;

template <int D>
__global__ __launch_bounds__(kMeanThreads) void value_mean_kernel(const MeanArgs a) {
  constexpr int CPL = D / 64;  // channels per lane
  const ScanGeometry& g = a.geo;
  const int seq = blockIdx.x / g.hkv;
  const int kvh = blockIdx.x % g.hkv;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n = clamp_len(ld_uniform(g.seq_lens, seq), view_capacity(g));
  float sum[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) sum[c] = 0.0f;
  for (int j = wave; j < n; j += kMeanWaves) {
    size_t row;
    bool ok = true;
    if (g.page_size > 0) {
      const int phys = g.block_table[static_cast<size_t>(seq) * g.max_pages + j / g.page_size];
      ok = phys >= 0 && phys < g.num_pages;
      row = (static_cast<size_t>(ok ? phys : 0) * g.hkv + kvh) * g.page_size + j % g.page_size;
    } else {
      row = (static_cast<size_t>(seq) * g.hkv + kvh) * g.max_seq_len + j;
    }
    if (!ok) continue;  // uniform: the page id is outside the pool
    const uint16_t* v = g.v + row * D + CPL * lane;
#pragma unroll
    for (int c = 0; c < CPL; ++c) sum[c] += bf16_lo(v[c]);
  }
  __shared__ float red[kMeanWaves][D];
#pragma unroll
  for (int c = 0; c < CPL; ++c) red[wave][CPL * lane + c] = sum[c];
  __syncthreads();
  for (int d = threadIdx.x; d < D; d += kMeanThreads) {
    float t = 0.0f;
    for (int w = 0; w < kMeanWaves; ++w) t += red[w][d];
    a.mean[(static_cast<size_t>(seq) * g.hkv + kvh) * D + d] = n > 0 ? t / static_cast<float>(n) : 0.0f;
  }
}

template <int D>
__global__ __launch_bounds__(256) void value_mean_append_kernel(const MeanArgs a) {
  constexpr int CPL = D / 64;
  const ScanGeometry& g = a.geo;
  const long long item = static_cast<long long>(blockIdx.x) * 4 +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (item >= static_cast<long long>(a.n_tok) * g.hkv) return;  // uniform per wave
  const int tok = static_cast<int>(item / g.hkv);
  const int kvh = static_cast<int>(item % g.hkv);
  const int seq = ld_uniform(a.tok_seq, tok);
  const int pos = ld_uniform(a.tok_pos, tok);
  if (seq < 0 || seq >= g.num_seqs || pos < 0) return;
  const int lane = threadIdx.x & 63;
  const uint16_t* v = a.v_src + (static_cast<size_t>(tok) * g.hkv + kvh) * D + CPL * lane;
  float* mu = a.mean + (static_cast<size_t>(seq) * g.hkv + kvh) * D + CPL * lane;
  const float inv = 1.0f / static_cast<float>(pos + 1);
#pragma unroll
  for (int c = 0; c < CPL; ++c) mu[c] = __builtin_fmaf(bf16_lo(v[c]) - mu[c], inv, mu[c]);
}

}  // namespace

hipError_t launch_value_mean(const MeanArgs& a, int head_dim, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv;
  if (blocks == 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(value_mean_kernel<128>, dim3(static_cast<unsigned>(blocks)),
                       dim3(kMeanThreads), 0, stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(value_mean_kernel<64>, dim3(static_cast<unsigned>(blocks)),
                       dim3(kMeanThreads), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_value_mean_append(const MeanArgs& a, int head_dim, hipStream_t stream) {
  const long long items = static_cast<long long>(a.n_tok) * a.geo.hkv;
  if (items == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((items + 3) / 4);
  if (head_dim == 128)
    hipLaunchKernelGGL(value_mean_append_kernel<128>, dim3(blocks), dim3(256), 0, stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(value_mean_append_kernel<64>, dim3(blocks), dim3(256), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace fold
