// Additive combine for gfx950 (Algorithm 1, last step; Section 4; the range
// certificate of Section 3).
//
// One workgroup of head_dim threads per query row.  Thread d adds the slots'
// A[d] in increasing slot order; every thread forms the same L sum in the same
// order.  o = A / L with no maximum and no rescale.  Optional outputs: the
// base-2 log-sum-exp Z + log2 L and the certificate bits.  With the cut-key
// value model (Section 4, depth paragraph) the slots' cut masses, summed in
// slot order, multiply the request's mean value row and join A: a virtual row
// standing in for every cut key.
#include "fold_device.h"
#include "fold_internal.h"

namespace fold {
namespace {

__global__ __launch_bounds__(128) void combine_kernel(const CombineArgs a) {
  const int row = blockIdx.x;
  const int d = threadIdx.x;
  const int D = a.head_dim;
  float acc = 0.0f;
  float l = 0.0f;
  // Slots are added in increasing order; loads are batched eight at a time so
  // they are in flight together.
  int s = 0;
  for (; s + 8 <= a.num_slots; s += 8) {
    float av[8], lv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const size_t sr = static_cast<size_t>(s + u) * a.num_rows + row;
      av[u] = a.part_A[sr * D + d];
      lv[u] = a.part_L[sr];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      acc += av[u];
      l += lv[u];
    }
  }
  for (; s < a.num_slots; ++s) {
    const size_t sr = static_cast<size_t>(s) * a.num_rows + row;
    acc += a.part_A[sr * D + d];
    l += a.part_L[sr];
  }
  if (a.part_Lcut) {
    float c = 0.0f;
    for (int t = 0; t < a.num_slots; ++t) c += a.part_Lcut[static_cast<size_t>(t) * a.num_rows + row];
    const int req = row / a.heads;
    const int kvh = (row - req * a.heads) / (a.heads / a.hkv);
    acc = __builtin_fmaf(c, a.mean[(static_cast<size_t>(req) * a.hkv + kvh) * D + d], acc);
  }
  const float o = acc / l;
  const size_t oi = static_cast<size_t>(row) * D + d;
  if (a.out_bf16)
    static_cast<uint16_t*>(a.out)[oi] = f32_to_bf16_rne(o);
  else
    static_cast<float*>(a.out)[oi] = o;
  const int bad = __syncthreads_or(!isfinite(o) ? 1 : 0);
  if (d == 0) {
    if (a.lse_out) a.lse_out[row] = a.z[row] + log2f(l);
    if (a.cert_out) {
      uint8_t c = 0;
      if (l < 0.5f) c |= 1;
      if (l > 0x1p100f) c |= 2;
      if (bad) c |= 4;
      a.cert_out[row] = c;
    }
  }
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, hipStream_t stream) {
  if (a.num_rows == 0) return hipSuccess;
  hipLaunchKernelGGL(combine_kernel, dim3(a.num_rows), dim3(a.head_dim), 0, stream, a);
  return hipGetLastError();
}

}  // namespace fold
