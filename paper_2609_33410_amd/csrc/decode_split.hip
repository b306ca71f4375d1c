// Gated split-KV decode scan for gfx950 (Section 4 "Weight-gated reads",
// "Value product", "Depth as a dial"; Algorithm 1).
//
// One workgroup = one (kv sequence, kv head, split, read group of GR query
// rows); W wave64s (4 or 8).  The split walks the 64-key tiles
// t == split (mod S); a tile holds four 16-key chunks, each a contiguous
// [16][D] bf16 slab in both cache layouts (pages hold a multiple of 16 keys).
// Wave w owns chunk (w mod 4) of the split's tiles k == w / 4 (mod W / 4), so
// the W waves share the split's tiles and a workgroup finishes its split W/4
// times sooner than four waves would: with the split count fixed by the
// caller, a long batch then drains in shorter workgroups (the last ones to be
// dispatched leave less of the call to a half-empty chip).  D/8 lanes hold
// one key row (8 channels each), so one wave-wide 128-bit load covers
// 64/(D/8) keys and 1 KiB of contiguous bytes.
//
// Loads go through buffer resources whose size is the chunk's valid bytes:
// keys past the sequence end and value rows of cut keys are given an offset
// outside the resource, so the hardware returns zero without touching memory.
// No load sits under a branch, which keeps the memory counters exact.
//
// Gated scan (finite T), software-pipelined three chunks deep per wave:
//   iteration t: issue K loads of chunk t+2;
//                score chunk t+1 (v_dot2_f32_bf16 + DPP row sums, x = s - Z in
//                FP32, live = x >= -T, ORed over the read group's rows) and
//                issue the value loads of its live keys only;
//                accumulate chunk t: A += [live] 2^x v, L += 2^x (FP32).
// Dense scan (T = inf): every key is live, so K and V of chunk t+1 are issued
// together before chunk t is scored and accumulated.
// At the end the lanes of a wave and then the W waves are reduced in a fixed
// order and the pair (A, L) of every row is written to its split's slot.
// CX (block model of BF16 values, finite T): each scored chunk's cut mass per
// row, the summed weights of its cut keys, is also written to chunk_cut.
#include "decode_common.h"

namespace fold {
namespace {

template <int D, int GR, bool DENSE, bool DBG, bool CX>
struct Scan {
  static constexpr int LPK = D / 8;        // lanes per key row
  static constexpr int KPI = 64 / LPK;     // keys per wave-wide 128-bit load
  static constexpr int NI = kChunk / KPI;  // loads per lane per 16-key chunk

  const DecodeArgs& a;
  const ScanGeometry& g;
  int seq, kvh, rg, nrows, req0, n, nchunks, lane, part, kslot;
  size_t gate_row;
  int gate_pages;
  u32x4 qv[GR];
  float zr[GR];
  bool rok[GR];
  size_t xrow[GR];  // query row index req * heads + head (debug export)
  float acc[GR][8];
  float lsum[GR];
  float lcut[GR];  // weights of cut keys (finite depth)

  __device__ Scan(const DecodeArgs& a_) : a(a_), g(a_.geo) {}

  __device__ __forceinline__ void load(rsrc_t r, u32x4 (&dst)[NI]) const {
#pragma unroll
    for (int i = 0; i < NI; ++i) dst[i] = buf_load(r, 1024u * i + 16u * lane);
  }

  __device__ __forceinline__ void load_gated(rsrc_t r, const bool (&live)[NI], u32x4 (&dst)[NI]) const {
#pragma unroll
    for (int i = 0; i < NI; ++i) dst[i] = buf_load(r, live[i] ? 1024u * i + 16u * lane : kOutOfRange);
  }

  // Scores, verdicts, L; the A-weights of live keys go to p.  Returns whether
  // any key of the chunk is read (wave-uniform).
  __device__ __forceinline__ bool score(int c, const u32x4 (&kv)[NI], float (&p)[NI][GR],
                                        bool (&anyl)[NI]) {
    float cc[GR];  // cut weights of this lane's keys of the chunk
#pragma unroll
    for (int r = 0; r < GR; ++r) cc[r] = 0.0f;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int j = c * kChunk + KPI * i + kslot;
      const bool kok = c < nchunks && j < n;
      anyl[i] = false;
#pragma unroll
      for (int r = 0; r < GR; ++r) {
        const float dot = group_sum<LPK>(dot8_bf16(kv[i], qv[r], 0.0f));
        const float x = __builtin_fmaf(dot, a.score_scale, -zr[r]);
        const bool ok = kok && rok[r];
        const bool live = ok && (DENSE || x >= a.neg_T);
        const float w = ok ? exp2_fast(x) : 0.0f;
        lsum[r] += w;
        if (!DENSE) lcut[r] += live ? 0.0f : w;
        if (!DENSE && (CX || DBG)) cc[r] += live ? 0.0f : w;
        p[i][r] = live ? w : 0.0f;
        anyl[i] = anyl[i] || live;
        if (DBG && a.x_out && ok && part == 0) a.x_out[xrow[r] * g.max_seq_len + j] = x;
      }
      if (DBG && a.key_gate_out && kok && part == 0)
        a.key_gate_out[gate_row * g.max_seq_len + j] = anyl[i] ? 1 : 0;
    }
    if constexpr (!DENSE && (CX || DBG)) {
      if (a.chunk_cut) {
        // the chunk's keys sit in the lanes of equal `part`
#pragma unroll
        for (int r = 0; r < GR; ++r) {
          float t = cc[r];
#pragma unroll
          for (int off = LPK; off < 64; off <<= 1) t += __shfl_xor(t, off, 64);
          if (lane == 0 && rok[r] && c < nchunks)
            a.chunk_cut[xrow[r] * a.chunk_stride + c] = t;
        }
      }
    }
    bool lane_any = false;
#pragma unroll
    for (int i = 0; i < NI; ++i) lane_any = lane_any || anyl[i];
    const bool chunk_any = __ballot(lane_any) != 0;
    if (DBG && a.page_gate_out && lane == 0 && c < nchunks)
      a.page_gate_out[gate_row * gate_pages + c] = chunk_any ? 1 : 0;
    return chunk_any;
  }

  __device__ __forceinline__ void accumulate(const u32x4 (&vv)[NI], const float (&p)[NI][GR]) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const float v0 = bf16_lo(vv[i].x), v1 = bf16_hi(vv[i].x);
      const float v2 = bf16_lo(vv[i].y), v3 = bf16_hi(vv[i].y);
      const float v4 = bf16_lo(vv[i].z), v5 = bf16_hi(vv[i].z);
      const float v6 = bf16_lo(vv[i].w), v7 = bf16_hi(vv[i].w);
#pragma unroll
      for (int r = 0; r < GR; ++r) {
        const float pr = p[i][r];
        acc[r][0] += pr * v0;
        acc[r][1] += pr * v1;
        acc[r][2] += pr * v2;
        acc[r][3] += pr * v3;
        acc[r][4] += pr * v4;
        acc[r][5] += pr * v5;
        acc[r][6] += pr * v6;
        acc[r][7] += pr * v7;
      }
    }
  }
};

template <int D, int GR, bool DENSE, bool DBG, int W, bool CX = false>
__global__ __launch_bounds__(64 * W) void decode_split_kernel(const DecodeArgs a) {
  constexpr int kWaves = W;
  constexpr int kThreads = 64 * W;
  using S = Scan<D, GR, DENSE, DBG, CX>;
  constexpr int NI = S::NI;
  const ScanGeometry& g = a.geo;
  S sc(a);
  sc.lane = threadIdx.x & 63;
  // wave-uniform (an SGPR), so chunk indices and buffer resources are scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  sc.part = sc.lane % S::LPK;
  sc.kslot = sc.lane / S::LPK;

  __shared__ int order[kOrderMax];
  const ScanPlace pl = a.by_length ? scan_place_by_length(a, order) : scan_place(a);
  sc.seq = pl.seq;
  sc.kvh = pl.kvh;
  const int split = pl.split;
  sc.rg = pl.rg;
  sc.req0 = pl.req0;
  sc.nrows = pl.nrows;
  if (sc.rg * GR >= sc.nrows) return;  // uniform: this read group has no rows
  sc.n = pl.n;
  sc.nchunks = pl.nchunks;
  sc.gate_row = (static_cast<size_t>(sc.seq) * g.hkv + sc.kvh) * a.row_groups + sc.rg;
  sc.gate_pages = (g.max_seq_len + kChunk - 1) / kChunk;

#pragma unroll
  for (int r = 0; r < GR; ++r) {
    const RowInfo ri = row_info(g, sc.seq, sc.kvh, sc.rg * GR + r, sc.nrows, sc.req0);
    sc.rok[r] = ri.ok;
    const size_t row = static_cast<size_t>(ri.req) * g.heads + ri.head;
    sc.qv[r] = ri.ok ? *reinterpret_cast<const u32x4*>(a.q + row * D + 8 * sc.part)
                     : u32x4{0, 0, 0, 0};
    sc.zr[r] = ri.ok ? a.z[row] : 0.0f;
    sc.xrow[r] = row;
    sc.lsum[r] = 0.0f;
    sc.lcut[r] = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) sc.acc[r][e] = 0.0f;
  }

  // Chunks of this wave: c_t = c0 + t * cstride, t < m (chunk w mod 4 of the
  // split's tiles k == w / 4 (mod W / 4)).
  const int cstride = kWaves * a.num_splits;
  const int c0 = 4 * split + 4 * a.num_splits * (wave >> 2) + (wave & 3);
  const int m = sc.nchunks > c0 ? (sc.nchunks - c0 + cstride - 1) / cstride : 0;

  if (DENSE) {
    u32x4 kA[NI], vA[NI], kB[NI], vB[NI];
    float p[NI][GR];
    bool anyl[NI];
    rsrc_t rk, rv;
    chunk_rsrc<D>(g, pl, c0, &rk, &rv);
    sc.load(rk, kA);
    sc.load(rv, vA);
    for (int t = 0; t < m; t += 2) {
      chunk_rsrc<D>(g, pl, c0 + (t + 1) * cstride, &rk, &rv);
      sc.load(rk, kB);
      sc.load(rv, vB);
      sc.score(c0 + t * cstride, kA, p, anyl);
      sc.accumulate(vA, p);
      if (t + 1 >= m) break;
      chunk_rsrc<D>(g, pl, c0 + (t + 2) * cstride, &rk, &rv);
      sc.load(rk, kA);
      sc.load(rv, vA);
      sc.score(c0 + (t + 1) * cstride, kB, p, anyl);
      sc.accumulate(vB, p);
    }
  } else {
    // kX: keys of chunk t+1 (scored this iteration); kY: keys of chunk t+2
    u32x4 kA[NI], kB[NI], vA[NI], vB[NI];
    float pA[NI][GR], pB[NI][GR];
    bool lA[NI], lB[NI];
    bool anyA = false, anyB = false;
    rsrc_t rk, rv;
    if (m > 0) {
      chunk_rsrc<D>(g, pl, c0, &rk, &rv);
      sc.load(rk, kA);
      rsrc_t rk1, rv1;
      chunk_rsrc<D>(g, pl, c0 + cstride, &rk1, &rv1);
      sc.load(rk1, kB);
      anyA = sc.score(c0, kA, pA, lA);
      sc.load_gated(rv, lA, vA);
    }
    for (int t = 0; t < m; t += 2) {
      // chunk t: V in vA / weights in pA; chunk t+1: K in kB
      rsrc_t rv1;
      chunk_rsrc<D>(g, pl, c0 + (t + 2) * cstride, &rk, &rv);
      sc.load(rk, kA);
      {
        rsrc_t rk1;
        chunk_rsrc<D>(g, pl, c0 + (t + 1) * cstride, &rk1, &rv1);
      }
      anyB = sc.score(c0 + (t + 1) * cstride, kB, pB, lB);
      sc.load_gated(rv1, lB, vB);
      if (anyA) sc.accumulate(vA, pA);
      if (t + 1 >= m) break;
      // chunk t+1: V in vB / weights in pB; chunk t+2: K in kA
      chunk_rsrc<D>(g, pl, c0 + (t + 3) * cstride, &rk, &rv1);
      sc.load(rk, kB);
      anyA = sc.score(c0 + (t + 2) * cstride, kA, pA, lA);
      sc.load_gated(rv, lA, vA);
      if (anyB) sc.accumulate(vB, pB);
    }
  }

  // Reduce over the key slots of the wave (lanes with equal `part`).
#pragma unroll
  for (int off = S::LPK; off < 64; off <<= 1) {
#pragma unroll
    for (int r = 0; r < GR; ++r) {
      sc.lsum[r] += __shfl_xor(sc.lsum[r], off, 64);
      if (!DENSE) sc.lcut[r] += __shfl_xor(sc.lcut[r], off, 64);
#pragma unroll
      for (int e = 0; e < 8; ++e) sc.acc[r][e] += __shfl_xor(sc.acc[r][e], off, 64);
    }
  }

  __shared__ float red_a[kWaves][GR][D];
  __shared__ float red_l[kWaves][GR];
  __shared__ float red_c[kWaves][GR];
  if (sc.kslot == 0) {
#pragma unroll
    for (int r = 0; r < GR; ++r)
#pragma unroll
      for (int e = 0; e < 8; ++e) red_a[wave][r][8 * sc.part + e] = sc.acc[r][e];
  }
  if (sc.lane == 0) {
#pragma unroll
    for (int r = 0; r < GR; ++r) {
      red_l[wave][r] = sc.lsum[r];
      red_c[wave][r] = sc.lcut[r];
    }
  }
  __syncthreads();

  const size_t slot = static_cast<size_t>(a.slot_offset) + split;
  for (int idx = threadIdx.x; idx < GR * D; idx += kThreads) {
    const int r = idx / D;
    const int d = idx - r * D;
    const RowInfo ri = row_info(g, sc.seq, sc.kvh, sc.rg * GR + r, sc.nrows, sc.req0);
    if (!ri.ok) continue;
    const size_t row = (slot * g.batch + ri.req) * g.heads + ri.head;
    float s = red_a[0][r][d];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) s += red_a[w][r][d];
    a.part_A[row * D + d] = s;
    if (d == 0) {
      float l = red_l[0][r];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) l += red_l[w][r];
      a.part_L[row] = l;
      if (a.part_Lcut) {
        float c = red_c[0][r];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) c += red_c[w][r];
        a.part_Lcut[row] = c;
      }
    }
  }
}

template <int D, bool DENSE, bool DBG, bool CX = false>
hipError_t launch_valu_w(const DecodeArgs& a, unsigned blocks, int waves, hipStream_t stream) {
  if (waves == 8)
    hipLaunchKernelGGL((decode_split_kernel<D, 1, DENSE, DBG, 8, CX>), dim3(blocks), dim3(64 * 8),
                       0, stream, a);
  else
    hipLaunchKernelGGL((decode_split_kernel<D, 1, DENSE, DBG, 4, CX>), dim3(blocks), dim3(64 * 4),
                       0, stream, a);
  return hipGetLastError();
}

// Waves per workgroup: 8 when every wave still gets at least 4 chunks of the
// longest sequence the view can hold, else 4 (so that no wave idles).
// Measured on the MHA 4 x 64K-128K decode (32 splits, longest sequences
// first): 8 waves 965 us dense / 563 us at T = 16, 4 waves 964 / 569, 16
// waves (one 1024-thread workgroup per CU) 966 / 576.
int mha_waves(const DecodeArgs& a) {
  const long long chunks = (static_cast<long long>(a.geo.max_seq_len) + kChunk - 1) / kChunk;
  return chunks / a.num_splits >= 8LL * 4 ? 8 : 4;
}

template <int D>
hipError_t launch_valu(const DecodeArgs& a, unsigned blocks, hipStream_t stream) {
  const bool dbg = a.x_out || a.key_gate_out || a.page_gate_out;
  const int w = mha_waves(a);
  if (a.dense)
    return dbg ? launch_valu_w<D, true, true>(a, blocks, w, stream)
               : launch_valu_w<D, true, false>(a, blocks, w, stream);
  if (dbg) return launch_valu_w<D, false, true>(a, blocks, w, stream);
  return a.chunk_cut ? launch_valu_w<D, false, false, true>(a, blocks, w, stream)
                     : launch_valu_w<D, false, false>(a, blocks, w, stream);
}

}  // namespace

// Rows per read group: one row (MHA, VALU scan), 16 / 32 rows (matrix-core
// scan for GQA groups and small stacks), or 64 rows (the stacked-row scan for
// more than 32 rows on one kv sequence).
int decode_rows_per_group(int rows_per_seq) {
  if (rows_per_seq <= 1) return 1;
  if (rows_per_seq <= 16) return 16;
  if (rows_per_seq <= 32) return 32;
  return 64;
}

hipError_t launch_decode_mfma(const DecodeArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_decode_stacked(const DecodeArgs& a, int head_dim, hipStream_t stream);

hipError_t launch_decode(const DecodeArgs& a, int head_dim, hipStream_t stream) {
  if (a.rows_per_group == 64) return launch_decode_stacked(a, head_dim, stream);
  if (a.rows_per_group > 1) return launch_decode_mfma(a, head_dim, stream);
  const long long blocks = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv * a.num_splits *
                           a.row_groups;
  if (blocks == 0) return hipSuccess;
  if (head_dim == 128) return launch_valu<128>(a, static_cast<unsigned>(blocks), stream);
  if (head_dim == 64) return launch_valu<64>(a, static_cast<unsigned>(blocks), stream);
  return hipErrorInvalidValue;
}

}  // namespace fold
