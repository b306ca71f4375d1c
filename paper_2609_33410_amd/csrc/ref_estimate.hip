// Reference estimate Z_i for gfx950 (Section 3, "Choosing the reference").
//
// One workgroup = one (request, kv head); four wave64s run the estimate
// routine of estimate_device.h (sampling, MFMA scoring, trimmed stratified
// sum).  The fused front (FRONT, two-plane INT8 keys) first splits the
// workgroup's own query rows into the scan's codes, with the query split's
// transform and rounding, writes them for the scan and scores them from LDS:
// one launch instead of two, the same bits.
#include "estimate_device.h"
#include "q8_split.h"

namespace fold {
namespace {

using est::kThreads;

template <int D, bool Q8, bool FRONT = false, int NT = kThreads>
__global__ __launch_bounds__(NT) void estimate_kernel(const Q8EstimateArgs qa8) {
  const ScanGeometry& g = qa8.e.geo;
  const int req = blockIdx.x / g.hkv;
  const int kvh = blockIdx.x % g.hkv;

  __shared__ float sc[kMaxEstRows][kMaxEstSamples];

  // Fused front: split the query rows of this (request, kv head) first (the
  // query split's own transform and rounding, so the codes are the same bits);
  // the codes go out for the scan and into LDS for the scoring below.
  __shared__ __attribute__((aligned(16))) int8_t qs[FRONT ? kMaxEstRows : 1][2 * D];
  __shared__ float etas[FRONT ? kMaxEstRows : 1];
  if constexpr (FRONT) {
    est::front_split_rows<D, NT>(qa8, req, kvh, qs, etas, true);
    __syncthreads();
  }

  est::estimate_rows<D, Q8, FRONT, NT>(qa8, req, kvh, sc, qs, etas, true, nullptr, [] {});
}

template <bool Q8>
hipError_t launch_est(const Q8EstimateArgs& a, int head_dim, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.e.geo.batch) * a.e.geo.hkv;
  if (blocks == 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL((estimate_kernel<128, Q8>), dim3(static_cast<unsigned>(blocks)),
                       dim3(kThreads), 0, stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL((estimate_kernel<64, Q8>), dim3(static_cast<unsigned>(blocks)),
                       dim3(kThreads), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_estimate(const EstimateArgs& a, int head_dim, hipStream_t stream) {
  Q8EstimateArgs q{};
  q.e = a;
  return launch_est<false>(q, head_dim, stream);
}

hipError_t launch_q8_estimate(const Q8EstimateArgs& a, int head_dim, hipStream_t stream) {
  return launch_est<true>(a, head_dim, stream);
}

// The fused front: eight waves for groups of more than four rows, so that
// each wave splits (and later reduces) one row.
template <int D>
void launch_front_d(const Q8EstimateArgs& a, unsigned blocks, hipStream_t stream) {
  if (a.e.geo.group > 4)
    hipLaunchKernelGGL((estimate_kernel<D, true, true, 2 * kThreads>), dim3(blocks),
                       dim3(2 * kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((estimate_kernel<D, true, true>), dim3(blocks), dim3(kThreads), 0, stream,
                       a);
}

hipError_t launch_q8_front(const Q8EstimateArgs& a, int head_dim, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.e.geo.batch) * a.e.geo.hkv;
  if (blocks == 0) return hipSuccess;
  if (head_dim == 128)
    launch_front_d<128>(a, static_cast<unsigned>(blocks), stream);
  else if (head_dim == 64)
    launch_front_d<64>(a, static_cast<unsigned>(blocks), stream);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace fold
