// Reference estimate Z_i for gfx950 (Section 3, "Choosing the reference").
//
// One workgroup = one (request, kv head); four wave64s.  The sampled keys are
// the first `sink` keys, the last `recent` keys and the centre of each of
// `strata` contiguous strata of the keys in between (every key when the row is
// short).  They are scored against all query rows of the GQA group with the
// same BF16 dot products as the decode scan, kept in LDS, and then one wave
// per row forms
//     Z = M + log2( sum_exact 2^(s - M) + (r / kept) * sum_kept 2^(s_c - M) )
// where M is the largest sampled score and the kept centres are those whose
// rank (by score, ties broken by stratum index) lies in
// [trim_lo, strata - trim_hi).  Ranking by score equals ranking by weight
// because 2^x is monotone.  All sums use fixed-order wave reductions.
#include "fold_device.h"
#include "fold_internal.h"

namespace fold {
namespace {

constexpr int kThreads = 256;

template <int D>
__global__ __launch_bounds__(kThreads) void estimate_kernel(const EstimateArgs a) {
  constexpr int LPK = D / 8;
  constexpr int KPI = 64 / LPK;
  const ScanGeometry& g = a.geo;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int part = lane % LPK;
  const int kslot = lane / LPK;
  const int req = blockIdx.x / g.hkv;
  const int kvh = blockIdx.x % g.hkv;
  const int G = g.group;

  __shared__ u32x4 qs[kMaxEstRows][D / 8];
  __shared__ float sc[kMaxEstRows][kMaxEstSamples];
  __shared__ int sidx[kMaxEstSamples];

  int n = 0;
  if (req < g.num_seqs) {
    n = clamp_len(g.seq_lens[req], view_capacity(g));
  }
  if (n == 0) {
    for (int r = threadIdx.x; r < G; r += kThreads)
      a.z_out[static_cast<size_t>(req) * g.heads + kvh * G + r] = 0.0f;
    return;
  }
  const int full = a.sink + a.recent + a.strata;
  const bool stratified = n > full;
  const int m = stratified ? full : n;
  const int n_exact = stratified ? a.sink + a.recent : n;
  const long long rmid = static_cast<long long>(n) - a.sink - a.recent;

  for (int t = threadIdx.x; t < m; t += kThreads) {
    int j;
    if (!stratified) {
      j = t;
    } else if (t < a.sink) {
      j = t;
    } else if (t < a.sink + a.recent) {
      j = n - a.recent + (t - a.sink);
    } else {
      const long long b = t - a.sink - a.recent;
      const long long lo = a.sink + (b * rmid) / a.strata;
      const long long hi = a.sink + ((b + 1) * rmid) / a.strata;
      j = static_cast<int>((lo + hi - 1) / 2);
    }
    sidx[t] = j;
  }
  for (int t = threadIdx.x; t < G * (D / 8); t += kThreads) {
    const int r = t / (D / 8);
    const int c = t - r * (D / 8);
    const size_t row = static_cast<size_t>(req) * g.heads + kvh * G + r;
    qs[r][c] = *reinterpret_cast<const u32x4*>(a.q + row * D + 8 * c);
  }
  __syncthreads();

  // Score every sampled key against every row.  Each lane scores up to
  // kBatch keys per pass; their block-table entries and key bytes are each
  // requested together (branch-free, always in-bounds indices), so a pass
  // costs two memory round trips.
  constexpr int kBatch = 12;
  constexpr int kKeysPerPass = kThreads / LPK;
  for (int t0 = 0; t0 < m; t0 += kKeysPerPass * kBatch) {
    int jb[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int t = t0 + b * kKeysPerPass + wave * KPI + kslot;
      jb[b] = sidx[t < m ? t : m - 1];
    }
    int phys[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b)
      phys[b] = g.page_size > 0
                    ? g.block_table[static_cast<size_t>(req) * g.max_pages + jb[b] / g.page_size]
                    : 0;
    u32x4 kv[kBatch];
#pragma unroll
    for (int b = 0; b < kBatch; ++b) {
      const int t = t0 + b * kKeysPerPass + wave * KPI + kslot;
      const int j = jb[b];
      size_t off;
      bool ok = t < m;
      if (g.page_size > 0) {
        ok = ok && phys[b] >= 0 && phys[b] < g.num_pages;
        off = ((static_cast<size_t>(ok ? phys[b] : 0) * g.hkv + kvh) * g.page_size +
               (j % g.page_size)) * D;
      } else {
        off = ((static_cast<size_t>(req) * g.hkv + kvh) * g.max_seq_len + j) * D;
      }
      const u32x4 v = *reinterpret_cast<const u32x4*>(g.k + (ok ? off : 0) + 8 * part);
      kv[b] = ok ? v : u32x4{0, 0, 0, 0};
    }
    for (int r = 0; r < G; ++r) {
      const u32x4 qf = qs[r][part];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int t = t0 + b * kKeysPerPass + wave * KPI + kslot;
        if (t0 + b * kKeysPerPass >= m) break;  // uniform
        const float dot = group_sum<LPK>(dot8_bf16(kv[b], qf, 0.0f));
        if (t < m && part == 0) sc[r][t] = dot * a.score_scale;
      }
    }
  }
  __syncthreads();

  for (int r = wave; r < G; r += kThreads / 64) {
    float mx = -INFINITY;
    for (int t = lane; t < m; t += 64) mx = fmaxf(mx, sc[r][t]);
    mx = wave_max(mx);
    float ex = 0.0f;
    for (int t = lane; t < n_exact; t += 64) ex += exp2_fast(sc[r][t] - mx);
    ex = wave_sum(ex);
    float mass = 0.0f;
    if (stratified) {
      const float* cs = &sc[r][a.sink + a.recent];
      float kept = 0.0f;
      // Trim: remove the trim_hi largest and the trim_lo smallest centre scores
      // one at a time (wave-wide max / min; among equal scores the lowest
      // stratum index goes first), then add the weights of the rest.  Ranking
      // by score equals ranking by weight because 2^x is monotone.
      constexpr int kPerLane = kMaxEstSamples / 64;
      const int nu = (a.strata + 63) / 64;
      float sv[kPerLane];
      bool keep[kPerLane];
#pragma unroll
      for (int u = 0; u < kPerLane; ++u) {
        const int b = lane + 64 * u;
        keep[u] = u < nu && b < a.strata;
        sv[u] = keep[u] ? cs[b] : 0.0f;
      }
      for (int k = 0; k < a.trim_hi + a.trim_lo; ++k) {
        const bool top = k < a.trim_hi;
        float ext = top ? -INFINITY : INFINITY;
#pragma unroll
        for (int u = 0; u < kPerLane; ++u)
          if (u < nu && keep[u]) ext = top ? fmaxf(ext, sv[u]) : fminf(ext, sv[u]);
        ext = top ? wave_max(ext) : -wave_max(-ext);
        bool removed = false;  // uniform
#pragma unroll
        for (int u = 0; u < kPerLane; ++u) {
          if (u >= nu || removed) break;
          const uint64_t hit = __ballot(keep[u] && sv[u] == ext);
          if (hit) {
            if (lane == __builtin_ctzll(hit)) keep[u] = false;
            removed = true;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < kPerLane; ++u)
        if (u < nu && keep[u]) kept += exp2_fast(sv[u] - mx);
      kept = wave_sum(kept);
      const int nkept = a.strata - a.trim_lo - a.trim_hi;
      mass = (static_cast<float>(rmid) / static_cast<float>(nkept)) * kept;
    }
    if (lane == 0)
      a.z_out[static_cast<size_t>(req) * g.heads + kvh * G + r] = mx + log2_fast(ex + mass);
  }
}

}  // namespace

hipError_t launch_estimate(const EstimateArgs& a, int head_dim, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.geo.batch) * a.geo.hkv;
  if (blocks == 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(estimate_kernel<128>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0,
                       stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(estimate_kernel<64>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0,
                       stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace fold
