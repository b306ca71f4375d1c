// The reference estimate of one (request, kv head) (Section 3, "Choosing the
// reference"), as a device routine of NT / 64 wave64s (four by default; the
// fused front takes eight for groups of more than four rows): the estimate
// kernel runs it once per workgroup, the fused decode as the prologue of
// every split's workgroup.  Each row is reduced by one wave and each 16-sample
// tile scored by one MFMA chain, whatever the wave count, so all give Z the
// same bits.
//
// The sampled keys are the first `sink` keys, the last `recent` keys and the
// centre of each of `strata` contiguous strata of the keys in between (every
// key when the row is short).  They are scored against all query rows of the
// GQA group with the same BF16 dot products as the decode scan and kept in
// LDS; then one wave per row forms
//     Z = M + log2( sum_exact 2^(s - M) + (r / kept) * sum_kept 2^(s_c - M) )
// where M is the largest sampled score and the kept centres are those left
// after removing the trim_hi largest and the trim_lo smallest centre scores
// (ranking by score equals ranking by weight because 2^x is monotone).
//
// Over a two-plane INT8 key cache the samples are scored with the scan's own
// coarse logits, eta_i e_j (a_j . qa_i + a_j . qb_i / 256), from plane A and
// the scales (v_mfma_i32_16x16x64_i8, the same operand layout); with FRONT the
// query codes come from the workgroup's LDS (the fused query split).
//
// Latency, not bandwidth, bounds it (48 KiB per (request, kv head) at
// D = 128).  Scores come from the matrix cores, 16 samples x 16 rows per
// v_mfma_f32_16x16x32_bf16 (the decode scan's layout); every lane computes its
// samples' key indices, issues their block-table reads at once and then all
// their key loads, so scoring costs two memory round trips (the query load
// overlaps the first).  The trim sorts the centre scores with a bitonic
// network across the wave whose exchanges are DPP moves within rows of 16
// lanes; wave reductions use DPP and v_readlane.  Every sum has a fixed order,
// so the result is deterministic.
#pragma once

#include <type_traits>

#include "fold_device.h"
#include "fold_internal.h"
#include "q8_split.h"

namespace fold {
namespace est {

constexpr int kThreads = 256;

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Lane-xor exchange: the partner lane's value.  XOR 1, 2, 3, 7 and 15 are one
// DPP move (quad permutations, row half-mirror, row mirror), 4 and 8 two;
// partners in another row of 16 lanes go through the LDS crossbar.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}

template <int L>
__device__ __forceinline__ float lane_xor(float v) {
  if constexpr (L == 1) return dpp_f<0xB1>(v);
  else if constexpr (L == 2) return dpp_f<0x4E>(v);
  else if constexpr (L == 3) return dpp_f<0x1B>(v);
  else if constexpr (L == 4) return dpp_f<0x1B>(dpp_f<0x141>(v));
  else if constexpr (L == 7) return dpp_f<0x141>(v);
  else if constexpr (L == 8) return dpp_f<0x141>(dpp_f<0x140>(v));
  else if constexpr (L == 15) return dpp_f<0x140>(v);
  else return __shfl_xor(v, L, 64);
}

__device__ __forceinline__ void sort_pair(float& v0, float& v1) {
  const float lo = fminf(v0, v1), hi = fmaxf(v0, v1);
  v0 = lo;
  v1 = hi;
}

// One compare-exchange stage of the sorting network on elements e = 2 lane + u:
// element e meets e ^ (2L + 1) (FLIP: the mirror image within a block) or
// e ^ 2L; the lower element keeps the minimum.
template <int L, bool FLIP>
__device__ __forceinline__ void net_stage(float& v0, float& v1, int lane) {
  const float p0 = lane_xor<L>(v0), p1 = lane_xor<L>(v1);
  const float a0 = FLIP ? p1 : p0;
  const float a1 = FLIP ? p0 : p1;
  constexpr int hb = FLIP ? (L + 1) / 2 : L;  // highest bit where lane and partner differ
  const bool keep_min = (lane & hb) == 0;
  v0 = keep_min ? fminf(v0, a0) : fmaxf(v0, a0);
  v1 = keep_min ? fminf(v1, a1) : fmaxf(v1, a1);
}

// Ascending sort of 128 values held two per lane (element 2 lane + u): a
// bitonic network in its mirror form, so that every comparator keeps the
// minimum at the lower index and each block merge starts with a flip.  K
// independent rows go through each stage side by side, so that a wave
// sorting two rows overlaps their dependency chains.
template <int K, int L, bool FLIP>
__device__ __forceinline__ void net_stage_k(float (&v0)[K], float (&v1)[K], int lane) {
#pragma unroll
  for (int k = 0; k < K; ++k) net_stage<L, FLIP>(v0[k], v1[k], lane);
}

template <int K>
__device__ __forceinline__ void sort_pair_k(float (&v0)[K], float (&v1)[K]) {
#pragma unroll
  for (int k = 0; k < K; ++k) sort_pair(v0[k], v1[k]);
}

template <int K>
__device__ __forceinline__ void sort128(float (&v0)[K], float (&v1)[K], int lane) {
  sort_pair_k<K>(v0, v1);
  net_stage_k<K, 1, true>(v0, v1, lane);
  sort_pair_k<K>(v0, v1);
  net_stage_k<K, 3, true>(v0, v1, lane);
  net_stage_k<K, 1, false>(v0, v1, lane);
  sort_pair_k<K>(v0, v1);
  net_stage_k<K, 7, true>(v0, v1, lane);
  net_stage_k<K, 2, false>(v0, v1, lane);
  net_stage_k<K, 1, false>(v0, v1, lane);
  sort_pair_k<K>(v0, v1);
  net_stage_k<K, 15, true>(v0, v1, lane);
  net_stage_k<K, 4, false>(v0, v1, lane);
  net_stage_k<K, 2, false>(v0, v1, lane);
  net_stage_k<K, 1, false>(v0, v1, lane);
  sort_pair_k<K>(v0, v1);
  net_stage_k<K, 31, true>(v0, v1, lane);
  net_stage_k<K, 8, false>(v0, v1, lane);
  net_stage_k<K, 4, false>(v0, v1, lane);
  net_stage_k<K, 2, false>(v0, v1, lane);
  net_stage_k<K, 1, false>(v0, v1, lane);
  sort_pair_k<K>(v0, v1);
  net_stage_k<K, 63, true>(v0, v1, lane);
  net_stage_k<K, 16, false>(v0, v1, lane);
  net_stage_k<K, 8, false>(v0, v1, lane);
  net_stage_k<K, 4, false>(v0, v1, lane);
  net_stage_k<K, 2, false>(v0, v1, lane);
  net_stage_k<K, 1, false>(v0, v1, lane);
  sort_pair_k<K>(v0, v1);
}

// Key index of sample t of a row of n keys (the sink, the recent keys, then
// the stratum centres; every key when the row is short).
__device__ __forceinline__ int sample_index(int t, int n, bool stratified, int sink, int recent,
                                            int strata, long long rmid) {
  if (!stratified || t < sink) return t;
  if (t < sink + recent) return n - recent + (t - sink);
  // floor(b r / strata) in double: b r < 2^53 is exact, and a quotient that is
  // not an integer sits at least 1/strata above its floor, far more than the
  // division's rounding error.
  const int b = t - sink - recent;
  const int lo = sink + static_cast<int>(floor(static_cast<double>(b) * rmid / strata));
  const int hi = sink + static_cast<int>(floor(static_cast<double>(b + 1) * rmid / strata));
  return (lo + hi - 1) / 2;
}

// Refine threshold of a request of nr query rows: kappa + ceil(log2 nr)
// (the query split's rule).
__device__ __forceinline__ float refine_threshold(float kappa, int nr) {
  const int c = nr > 1 ? 32 - __builtin_clz(static_cast<unsigned>(nr - 1)) : 0;
  return kappa + static_cast<float>(c);
}

// The fused front's query split of the GQA rows of (req, kvh), wave w taking
// rows w, w+4, ...: the query split's own transform and rounding (so the
// codes are the same bits), into qs / etas in LDS and, when write_out, to
// qa8.qp_out / eta_out and the request's thresholds.  The caller puts a
// barrier before reading qs / etas.
template <int D, int NT = kThreads>
__device__ __forceinline__ void front_split_rows(const Q8EstimateArgs& qa8, int req, int kvh,
                                                 int8_t (*qs)[2 * D], float* etas,
                                                 bool write_out) {
  const ScanGeometry& g = qa8.e.geo;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int G = g.group;
  for (int r = wave; r < G; r += NT / 64) {
    const size_t row = static_cast<size_t>(req) * g.heads + kvh * G + r;
    double x[D / 64];
#pragma unroll
    for (int i = 0; i < D / 64; ++i)
      x[i] = static_cast<double>(bf16_lo(qa8.q_src[row * D + 64 * i + lane]));
    hadamard_wave<D>(x, lane);
    const double f = wave_absmax_f64<D>(x) / 127.0;
#pragma unroll
    for (int i = 0; i < D / 64; ++i) {
      int8_t ca, cb;
      split_value(x[i], f, &ca, &cb);
      if (write_out) {
        qa8.qp_out[row * 2 * D + 64 * i + lane] = ca;
        qa8.qp_out[row * 2 * D + D + 64 * i + lane] = cb;
      }
      qs[r][64 * i + lane] = ca;
      qs[r][D + 64 * i + lane] = cb;
    }
    if (lane == 0) {
      const float eta = static_cast<float>(((kLog2eF64 * static_cast<double>(qa8.sm_scale)) * f) / D);
      if (write_out) qa8.eta_out[row] = eta;
      etas[r] = eta;
    }
  }
  if (write_out && kvh == 0 && qa8.tau && threadIdx.x == 0) {
    const int nr = qa8.req_lens[req];
    qa8.tau[req] = refine_threshold(qa8.kappa, nr);
    if (qa8.tau_v) qa8.tau_v[req] = refine_threshold(qa8.kappa_v, nr);
  }
}

// Z of the GQA rows of (req, kvh), computed by all NT / 64 waves of the
// workgroup (it contains barriers).  sc: the workgroup's LDS score buffer.
// qs / etas: the LDS query codes and scales of the fused front (FRONT only).
// Z goes to a.z_out when write_z and to z_lds[r] when z_lds is not null.
// issued() runs once per wave of a non-empty row, right after the wave's
// first sample loads are issued: a caller's loads issued there fly while the
// estimate waits for its keys.
template <int D, bool Q8, bool FRONT, int NT = kThreads, typename Issued>
__device__ __forceinline__ void estimate_rows(const Q8EstimateArgs& qa8, int req, int kvh,
                                              float (*sc)[kMaxEstSamples],
                                              const int8_t (*qs)[2 * D], const float* etas,
                                              bool write_z, float* z_lds, Issued&& issued) {
  const EstimateArgs& a = qa8.e;
  constexpr int NK = Q8 ? D / 64 : D / 32;  // 16-byte key loads per lane per sample tile
  constexpr int kTilesPerPass = 4;      // sample tiles per wave whose loads fly together
  constexpr int kScanWavesEst = NT / 64;
  const ScanGeometry& g = a.geo;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int G = g.group;
  constexpr bool kHook = !std::is_empty_v<std::decay_t<Issued>>;

  int n = 0;
  if (req < g.num_seqs) n = clamp_len(ld_uniform(g.seq_lens, req), view_capacity(g));
  if (n == 0) {
    for (int r = threadIdx.x; r < G; r += NT) {
      if (write_z) a.z_out[static_cast<size_t>(req) * g.heads + kvh * G + r] = 0.0f;
      if (z_lds) z_lds[r] = 0.0f;
    }
    return;
  }
  const int full = a.sink + a.recent + a.strata;
  const bool stratified = n > full;
  const int m = stratified ? full : n;
  const int n_exact = stratified ? a.sink + a.recent : n;
  const long long rmid = static_cast<long long>(n) - a.sink - a.recent;

  // Q^T operand of the score product: lane l holds channels 32c + 8(l/16) .. +8
  // of query row l%16 (rows past the group are zero).
  const int n16 = lane & 15;
  const int grp = lane >> 4;
  // Q8: the same lanes hold 16 bytes of qa (and of qb) per product instead.
  u32x4 qb[NK], qb2[NK];
  float eta_r = 0.0f;
#pragma unroll
  for (int c = 0; c < NK; ++c) {
    qb[c] = u32x4{0, 0, 0, 0};
    qb2[c] = u32x4{0, 0, 0, 0};
    if (n16 < G) {
      const size_t row = static_cast<size_t>(req) * g.heads + kvh * G + n16;
      if constexpr (FRONT) {
        qb[c] = *reinterpret_cast<const u32x4*>(&qs[n16][64 * c + 16 * grp]);
        qb2[c] = *reinterpret_cast<const u32x4*>(&qs[n16][D + 64 * c + 16 * grp]);
      } else if constexpr (Q8) {
        qb[c] = *reinterpret_cast<const u32x4*>(qa8.qp + row * 2 * D + 64 * c + 16 * grp);
        qb2[c] = *reinterpret_cast<const u32x4*>(qa8.qp + row * 2 * D + D + 64 * c + 16 * grp);
      } else {
        qb[c] = *reinterpret_cast<const u32x4*>(a.q + row * D + 32 * c + 8 * grp);
      }
    }
  }
  if constexpr (Q8) {
    if (n16 < G) eta_r = FRONT ? etas[n16] : qa8.eta[static_cast<size_t>(req) * g.heads + kvh * G + n16];
  }

  // Tiles of 16 samples; wave w scores tiles w, w+4, ...; lane l loads sample l%16.
  const int ntiles = (m + 15) / 16;
  // One pass: the loads of tiles tau0, tau0 + 4, ... (clamped samples for
  // tiles past the end), then hook(), then the scores of every tile loaded
  // (those past the end are not stored), so that no load is left in flight
  // unread: a later wait would count it.
  auto pass = [&](int tau0, auto&& hook) {
    int jb[kTilesPerPass];
#pragma unroll
    for (int u = 0; u < kTilesPerPass; ++u) {
      const int t = 16 * (tau0 + kScanWavesEst * u) + n16;
      jb[u] = sample_index(t < m ? t : m - 1, n, stratified, a.sink, a.recent, a.strata, rmid);
    }
    int phys[kTilesPerPass];
#pragma unroll
    for (int u = 0; u < kTilesPerPass; ++u)
      phys[u] = g.page_size > 0
                    ? g.block_table[static_cast<size_t>(req) * g.max_pages + jb[u] / g.page_size]
                    : 0;
    // Raw loads; a lane whose sample is past the end or on a page outside
    // the pool (okl false) contributes zeros, applied after hook() so that no
    // wait for a load precedes the caller's loads.
    u32x4 kv[kTilesPerPass][NK];
    uint16_t ksr[kTilesPerPass];  // Q8: the scale of this lane's sample
    bool okl[kTilesPerPass];
#pragma unroll
    for (int u = 0; u < kTilesPerPass; ++u) {
      const int t = 16 * (tau0 + kScanWavesEst * u) + n16;
      const int j = jb[u];
      size_t krow;  // key row in the cache's element layout
      bool ok = t < m;
      if (g.page_size > 0) {
        ok = ok && phys[u] >= 0 && phys[u] < g.num_pages;
        krow = (static_cast<size_t>(ok ? phys[u] : 0) * g.hkv + kvh) * g.page_size +
               (j % g.page_size);
      } else {
        krow = (static_cast<size_t>(req) * g.hkv + kvh) * g.max_seq_len + j;
      }
      if (!ok) krow = 0;
#pragma unroll
      for (int c = 0; c < NK; ++c) {
        u32x4 v;
        if constexpr (Q8)
          v = *reinterpret_cast<const u32x4*>(qa8.keys.ka + krow * D + 64 * c + 16 * grp);
        else
          v = *reinterpret_cast<const u32x4*>(g.k + krow * D + 32 * c + 8 * grp);
        kv[u][c] = v;
      }
      okl[u] = ok;
      ksr[u] = 0;
      if constexpr (Q8) ksr[u] = qa8.keys.ks[krow];
    }
    hook();
#pragma unroll
    for (int u = 0; u < kTilesPerPass; ++u) {
      const int tau = tau0 + kScanWavesEst * u;
      float sv[4];
      if constexpr (Q8) {
        i32x4 caa = {0, 0, 0, 0}, cab = {0, 0, 0, 0};
#pragma unroll
        for (int c = 0; c < NK; ++c) {
          const u32x4 ka = okl[u] ? kv[u][c] : u32x4{0, 0, 0, 0};
          caa = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, ka),
                                                     __builtin_bit_cast(i32x4, qb[c]), caa, 0, 0, 0);
          cab = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, ka),
                                                     __builtin_bit_cast(i32x4, qb2[c]), cab, 0, 0, 0);
        }
        const float ks = okl[u] ? bf16_lo(ksr[u]) : 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // the scale of sample 4(l/16)+i sits in lane 4(l/16)+i
          const float e = __shfl(ks, 4 * grp + i, 64);
          const float t = static_cast<float>(caa[i]) + static_cast<float>(cab[i]) * (1.0f / 256.0f);
          sv[i] = (eta_r * e) * t;
        }
      } else {
        f32x4 s = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < NK; ++c)
          s = mfma_16x16x32(okl[u] ? kv[u][c] : u32x4{0, 0, 0, 0}, qb[c], s);
#pragma unroll
        for (int i = 0; i < 4; ++i) sv[i] = s[i] * a.score_scale;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = 16 * tau + 4 * grp + i;
        if (n16 < G && t < m) sc[n16][t] = sv[i];
      }
    }
  };
  // The first pass runs on every wave (one without a tile scores none), with
  // issued() at one fixed point of straight-line code: the caller's loads go
  // after this pass's sample loads, not before the block-table reads those
  // wait on (loads retire in issue order), and every wait for a sample counts
  // the caller's loads as issued after it.
  pass(wave, [&] {
    if constexpr (kHook) __builtin_amdgcn_sched_barrier(0);
    issued();
    if constexpr (kHook) __builtin_amdgcn_sched_barrier(0);
  });
  for (int tau0 = wave + kScanWavesEst * kTilesPerPass; tau0 < ntiles;
       tau0 += kScanWavesEst * kTilesPerPass)
    pass(tau0, [] {});
  __syncthreads();

  constexpr int kPerLane = kMaxEstSamples / 64;
  const int nu_all = (m + 63) / 64;
  const int nu = (a.strata + 63) / 64;
  const int nkept = a.strata - a.trim_lo - a.trim_hi;
  // Z of K rows of this wave.  With K = 2 the two rows' independent chains
  // run side by side; each row's operations and their order are those of a
  // row alone, so Z has the same bits either way.  Stratified rows sort their
  // (at most 128) centre scores across the wave, two per lane (element
  // e = 2 * lane + u), padded with +inf; sorted positions
  // [trim_lo, strata - trim_hi) are kept.  A fixed network: the kept
  // multiset, hence the sum, does not depend on tie order.
  auto rows_z = [&](auto kk, const int* rs) {
    constexpr int K = decltype(kk)::value;
    float mx[K], ex[K], mass[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      mx[k] = -INFINITY;
#pragma unroll
      for (int u = 0; u < kPerLane; ++u) {
        const int t = lane + 64 * u;
        if (u < nu_all && t < m) mx[k] = fmaxf(mx[k], sc[rs[k]][t]);
      }
    }
#pragma unroll
    for (int k = 0; k < K; ++k) mx[k] = wave_max_dpp(mx[k]);
#pragma unroll
    for (int k = 0; k < K; ++k) {
      ex[k] = 0.0f;
#pragma unroll
      for (int u = 0; u < kPerLane; ++u) {
        const int t = lane + 64 * u;
        if (u < nu_all && t < n_exact) ex[k] += exp2_fast(sc[rs[k]][t] - mx[k]);
      }
    }
#pragma unroll
    for (int k = 0; k < K; ++k) ex[k] = wave_sum_dpp(ex[k]);
#pragma unroll
    for (int k = 0; k < K; ++k) mass[k] = 0.0f;
    if (stratified) {
      float v0[K], v1[K], kept[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const float* cs = &sc[rs[k]][a.sink + a.recent];
        v0[k] = 2 * lane < a.strata ? cs[2 * lane] : INFINITY;
        v1[k] = 2 * lane + 1 < a.strata ? cs[2 * lane + 1] : INFINITY;
      }
      sort128<K>(v0, v1, lane);
      const int hi_pos = a.strata - a.trim_hi;
      const int e0 = 2 * lane, e1 = 2 * lane + 1;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        kept[k] = 0.0f;
        if (e0 >= a.trim_lo && e0 < hi_pos) kept[k] += exp2_fast(v0[k] - mx[k]);
        if (e1 >= a.trim_lo && e1 < hi_pos) kept[k] += exp2_fast(v1[k] - mx[k]);
      }
#pragma unroll
      for (int k = 0; k < K; ++k) {
        kept[k] = wave_sum_dpp(kept[k]);
        mass[k] = (static_cast<float>(rmid) / static_cast<float>(nkept)) * kept[k];
      }
    }
    if (lane == 0) {
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const float z = mx[k] + log2_fast(ex[k] + mass[k]);
        if (write_z) a.z_out[static_cast<size_t>(req) * g.heads + kvh * G + rs[k]] = z;
        if (z_lds) z_lds[rs[k]] = z;
      }
    }
  };
  constexpr int NW = NT / 64;
  if (!stratified || a.strata <= 128) {
    int r = wave;
    for (; r + NW < G; r += 2 * NW) {
      const int rs[2] = {r, r + NW};
      rows_z(std::integral_constant<int, 2>{}, rs);
    }
    if (r < G) {
      const int rs[1] = {r};
      rows_z(std::integral_constant<int, 1>{}, rs);
    }
    return;
  }
  // Larger stratifications: remove the trim_hi largest and the trim_lo
  // smallest centre scores one at a time (among equal scores the lowest
  // stratum index goes first), then add what is left.
  for (int r = wave; r < G; r += NW) {
    float mx = -INFINITY;
#pragma unroll
    for (int u = 0; u < kPerLane; ++u) {
      const int t = lane + 64 * u;
      if (u < nu_all && t < m) mx = fmaxf(mx, sc[r][t]);
    }
    mx = wave_max_dpp(mx);
    float ex = 0.0f;
#pragma unroll
    for (int u = 0; u < kPerLane; ++u) {
      const int t = lane + 64 * u;
      if (u < nu_all && t < n_exact) ex += exp2_fast(sc[r][t] - mx);
    }
    ex = wave_sum_dpp(ex);
    const float* cs = &sc[r][a.sink + a.recent];
    float kept = 0.0f;
    float sv[kPerLane];
    bool keep[kPerLane];
#pragma unroll
    for (int u = 0; u < kPerLane; ++u) {
      const int b = lane + 64 * u;
      keep[u] = u < nu && b < a.strata;
      sv[u] = keep[u] ? cs[b] : 0.0f;
    }
    for (int k = 0; k < a.trim_hi + a.trim_lo; ++k) {
      const bool top = k < a.trim_hi;  // uniform
      float ext = -INFINITY;
#pragma unroll
      for (int u = 0; u < kPerLane; ++u)
        if (u < nu && keep[u]) ext = fmaxf(ext, top ? sv[u] : -sv[u]);
      ext = wave_max_dpp(ext);
      if (!top) ext = -ext;
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
    kept = wave_sum_dpp(kept);
    const float mass = (static_cast<float>(rmid) / static_cast<float>(nkept)) * kept;
    if (lane == 0) {
      const float z = mx + log2_fast(ex + mass);
      if (write_z) a.z_out[static_cast<size_t>(req) * g.heads + kvh * G + r] = z;
      if (z_lds) z_lds[r] = z;
    }
  }
}


}  // namespace est
}  // namespace fold
