// Gated split-KV decode scan on the matrix cores, for GQA groups and for the
// stacked query rows of a shared-prefix cascade level (Section 4 "Weight-gated
// reads", "Value product", "Depth as a dial"; Appendix E, cascade levels;
// Algorithm 1).
//
// Workgroup = (kv sequence, kv head, split, read group of 16*RB query rows);
// four wave64s.  The split walks the 64-key tiles t == split (mod S); wave w
// owns the 16-key chunk 4t + w of each tile.  Per chunk and 16-row block:
//
//   scores   S^T[key][row] = K . Q^T with v_mfma_f32_16x16x32_bf16: keys on M
//            (lane l loads 16 bytes of key l%16 straight into the A operand),
//            query rows on N (a constant B operand), channels on K.  Lane l
//            ends up holding keys 4(l/16)+i, i < 4, of row l%16.
//   verdict  x = s - Z_i in FP32 (explicit FMA); live = x >= -T; the live bits
//            are ORed over the read group's rows with wave ballots, giving a
//            16-bit read mask of the chunk.
//   values   only live value rows are requested (the others get an offset past
//            the chunk's buffer resource, so no bytes move).
//   product  A^T[d][row] += V^T[d][key] . P^T[key][row] with
//            v_mfma_f32_16x16x16_bf16: channels on M, rows on N, the chunk's 16
//            keys on K.  The B operand P^T is the score output's own register
//            layout, so the weights never leave their lanes; the weight enters
//            as bf16(hi) + bf16(residual) (two products), while L adds the FP32
//            weight of every key, live or cut.  The A operand V^T is read from
//            the wave's value tile in LDS, transposed by 16-bit reads.
//
// CX (block model of BF16 values, finite T): each scored chunk's cut mass per
// row, the summed weights of its cut keys, is also written to chunk_cut.
//
// The scan is software-pipelined per wave exactly as the VALU scan: gated
// (finite T) issues the keys of chunk t+2, scores chunk t+1 and issues its live
// value rows, then forms the product of chunk t; dense (T = inf) issues keys
// and values of chunk t+1 together before working on chunk t.
#include "decode_common.h"

namespace fold {
namespace {

__device__ __forceinline__ f32x4 mfma_qk(u32x4 a, u32x4 b, f32x4 c) { return mfma_16x16x32(a, b, c); }
__device__ __forceinline__ f32x4 mfma_pv(u32x2 a, u32x2 b, f32x4 c) { return mfma_16x16x16(a, b, c); }

template <int D, int RB, bool DENSE, bool DBG, bool CX>
struct MfmaScan {
  static constexpr int NK = D / 32;           // 128-bit loads per lane per chunk (K, and V)
  static constexpr int NB = D / 16;           // 16-channel blocks of the value product
  static constexpr int VSTRIDE = 2 * D + 16;  // bytes per key row of the LDS value tile
  static constexpr int R = 16 * RB;           // rows per read group

  const DecodeArgs& a;
  const ScanGeometry& g;
  ScanPlace p;
  int lane, n16, grp;
  size_t gate_row;
  unsigned char* vt;  // this wave's value tile [16][VSTRIDE]

  u32x4 qb[RB][NK];
  float zr[RB];
  bool rok[RB];
  size_t xrow[RB];
  f32x4 acc[RB][NB];
  float lsum[RB];
  float lcut[RB];  // weights of cut keys (finite depth)

  __device__ MfmaScan(const DecodeArgs& a_) : a(a_), g(a_.geo) {}

  // Keys load as whole lines: lane l, load c takes the 16 bytes at
  // 1024 c + 16 l of the chunk (key (1024 c + 16 l) / 2D).  kstage() turns
  // them into the QK A operand through the wave's LDS tile.
  __device__ __forceinline__ void kload(rsrc_t r, u32x4 (&kv)[NK]) const {
#pragma unroll
    for (int c = 0; c < NK; ++c) kv[c] = buf_load(r, 1024u * c + 16u * lane);
  }

  // The QK A operand (lane l: key l%16, channels 32c + 8(l/16) .. +8) from a
  // chunk loaded by kload(), through the wave's tile (rows padded to VSTRIDE
  // bytes, so the 16 rows of one read fall in distinct banks).
  __device__ __forceinline__ void kstage(const u32x4 (&kv)[NK], u32x4 (&ka)[NK]) const {
#pragma unroll
    for (int c = 0; c < NK; ++c) {
      const uint32_t off = 1024u * c + 16u * lane;
      const uint32_t key = off / (2 * D);
      *reinterpret_cast<u32x4*>(vt + key * VSTRIDE + (off - key * 2 * D)) = kv[c];
    }
#pragma unroll
    for (int c = 0; c < NK; ++c)
      ka[c] = *reinterpret_cast<const u32x4*>(vt + n16 * VSTRIDE + 64 * c + 16 * grp);
  }

  __device__ __forceinline__ void vload(rsrc_t r, uint32_t mask, u32x4 (&vv)[NK]) const {
    // lane l, load i: the 16 bytes at 1024 i + 16 l of the chunk (key (1024 i + 16 l) / 2D)
#pragma unroll
    for (int i = 0; i < NK; ++i) {
      const uint32_t off = 1024u * i + 16u * lane;
      const uint32_t key = off / (2 * D);
      vv[i] = buf_load(r, DENSE || ((mask >> key) & 1u) ? off : kOutOfRange);
    }
  }

  // Scores, verdicts and L for chunk c; weights of live keys as bf16 hi/lo
  // pairs in the P^T operand layout.  Returns the chunk's 16-bit read mask.
  __device__ __forceinline__ uint32_t score(int c, const u32x4 (&kv)[NK], u32x2 (&phi)[RB],
                                            u32x2 (&plo)[RB]) {
    const int key0 = c * kChunk;
    const int nk = c < p.nchunks ? min(kChunk, p.n - key0) : 0;
    uint64_t any[4] = {0, 0, 0, 0};
    u32x4 ka[NK];
    kstage(kv, ka);
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      f32x4 s = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int c2 = 0; c2 < NK; ++c2) s = mfma_qk(ka[c2], qb[b][c2], s);
      uint32_t hi[4], lo[4];
      float cc = 0.0f;  // cut weights of this lane's keys of the chunk
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kk = 4 * grp + i;
        const bool ok = rok[b] && kk < nk;
        const float x = __builtin_fmaf(s[i], a.score_scale, -zr[b]);
        const bool live = ok && (DENSE || x >= a.neg_T);
        const float w = ok ? exp2_fast(x) : 0.0f;
        lsum[b] += w;
        if (!DENSE) lcut[b] += live ? 0.0f : w;
        if (!DENSE && (CX || DBG)) cc += live ? 0.0f : w;
        const float pw = live ? w : 0.0f;
        hi[i] = __float_as_uint(pw) & 0xffff0000u;
        lo[i] = f32_to_bf16_rne(pw - __uint_as_float(hi[i]));
        any[i] |= __ballot(live);
        if (DBG && a.x_out && ok) a.x_out[xrow[b] * g.max_seq_len + key0 + kk] = x;
      }
      if constexpr (!DENSE && (CX || DBG)) {
        if (a.chunk_cut) {
          // the four key groups of row n16 hold the chunk's 16 keys
          cc += __shfl_xor(cc, 16, 64);
          cc += __shfl_xor(cc, 32, 64);
          if (grp == 0 && rok[b] && c < p.nchunks) a.chunk_cut[xrow[b] * a.chunk_stride + c] = cc;
        }
      }
      phi[b] = u32x2{(hi[0] >> 16) | hi[1], (hi[2] >> 16) | hi[3]};
      plo[b] = u32x2{lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16)};
    }
    uint32_t mask = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if ((any[i] >> (16 * q)) & 0xffffull) mask |= 1u << (4 * q + i);
    if (DBG) {
      if (a.key_gate_out && lane < nk)
        a.key_gate_out[gate_row * g.max_seq_len + key0 + lane] = (mask >> lane) & 1u;
      if (a.page_gate_out && lane == 0 && c < p.nchunks)
        a.page_gate_out[gate_row * ((g.max_seq_len + kChunk - 1) / kChunk) + c] = mask ? 1 : 0;
    }
    return mask;
  }

  __device__ __forceinline__ void product(uint32_t mask, const u32x4 (&vv)[NK],
                                          const u32x2 (&phi)[RB], const u32x2 (&plo)[RB]) {
    if (mask == 0) return;  // wave-uniform: no live key in the chunk
#pragma unroll
    for (int i = 0; i < NK; ++i) {
      const uint32_t off = 1024u * i + 16u * lane;
      const uint32_t key = off / (2 * D);
      *reinterpret_cast<u32x4*>(vt + key * VSTRIDE + (off - key * 2 * D)) = vv[i];
    }
    const unsigned char* col = vt + (4 * grp) * VSTRIDE + 2 * n16;
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
      const unsigned char* e = col + 32 * blk;
      const uint32_t v0 = *reinterpret_cast<const uint16_t*>(e);
      const uint32_t v1 = *reinterpret_cast<const uint16_t*>(e + VSTRIDE);
      const uint32_t v2 = *reinterpret_cast<const uint16_t*>(e + 2 * VSTRIDE);
      const uint32_t v3 = *reinterpret_cast<const uint16_t*>(e + 3 * VSTRIDE);
      const u32x2 va = {v0 | (v1 << 16), v2 | (v3 << 16)};
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        acc[b][blk] = mfma_pv(va, phi[b], acc[b][blk]);
        acc[b][blk] = mfma_pv(va, plo[b], acc[b][blk]);
      }
    }
  }
};

template <int D, int RB, bool DENSE, bool DBG, bool CX = false>
__global__ __launch_bounds__(kScanThreads) void decode_mfma_kernel(const DecodeArgs a) {
  using S = MfmaScan<D, RB, DENSE, DBG, CX>;
  constexpr int NK = S::NK;
  constexpr int R = S::R;
  constexpr int kTileBytes = kScanWaves * 16 * S::VSTRIDE;
  constexpr int kRedBytes = (R * D + RB * 64) * 4;
  __shared__ __attribute__((aligned(16))) unsigned char smem[kTileBytes > kRedBytes ? kTileBytes : kRedBytes];

  const ScanGeometry& g = a.geo;
  S sc(a);
  sc.p = scan_place(a);
  if (sc.p.rg * R >= sc.p.nrows) return;  // uniform: this read group has no rows
  sc.lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  sc.n16 = sc.lane & 15;
  sc.grp = sc.lane >> 4;
  sc.vt = smem + wave * 16 * S::VSTRIDE;
  sc.gate_row = (static_cast<size_t>(sc.p.seq) * g.hkv + sc.p.kvh) * a.row_groups + sc.p.rg;

#pragma unroll
  for (int b = 0; b < RB; ++b) {
    const RowInfo ri = row_info(g, sc.p.seq, sc.p.kvh, sc.p.rg * R + 16 * b + sc.n16,
                                sc.p.nrows, sc.p.req0);
    sc.rok[b] = ri.ok;
    const size_t row = static_cast<size_t>(ri.req) * g.heads + ri.head;
    sc.xrow[b] = row;
    sc.zr[b] = ri.ok ? a.z[row] : 0.0f;
#pragma unroll
    for (int c = 0; c < NK; ++c)
      sc.qb[b][c] = ri.ok ? *reinterpret_cast<const u32x4*>(a.q + row * D + 32 * c + 8 * sc.grp)
                          : u32x4{0, 0, 0, 0};
    sc.lsum[b] = 0.0f;
    sc.lcut[b] = 0.0f;
#pragma unroll
    for (int blk = 0; blk < S::NB; ++blk) sc.acc[b][blk] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  }

  const int cstride = kScanWaves * a.num_splits;
  const int c0 = kScanWaves * sc.p.split + wave;
  const int m = sc.p.nchunks > c0 ? (sc.p.nchunks - c0 + cstride - 1) / cstride : 0;

  if (DENSE) {
    // three chunks in flight per wave: keys and values of t+1 and t+2 load
    // while chunk t is scored and multiplied
    u32x4 kA[NK], vA[NK], kB[NK], vB[NK], kC[NK], vC[NK];
    u32x2 phi[RB], plo[RB];
    rsrc_t rk, rv;
    chunk_rsrc<D>(g, sc.p, c0, &rk, &rv);
    sc.kload(rk, kA);
    sc.vload(rv, 0xffffu, vA);
    chunk_rsrc<D>(g, sc.p, c0 + cstride, &rk, &rv);
    sc.kload(rk, kB);
    sc.vload(rv, 0xffffu, vB);
    for (int t = 0; t < m; t += 3) {
      chunk_rsrc<D>(g, sc.p, c0 + (t + 2) * cstride, &rk, &rv);
      sc.kload(rk, kC);
      sc.vload(rv, 0xffffu, vC);
      uint32_t mk = sc.score(c0 + t * cstride, kA, phi, plo);
      sc.product(mk, vA, phi, plo);
      if (t + 1 >= m) break;
      chunk_rsrc<D>(g, sc.p, c0 + (t + 3) * cstride, &rk, &rv);
      sc.kload(rk, kA);
      sc.vload(rv, 0xffffu, vA);
      mk = sc.score(c0 + (t + 1) * cstride, kB, phi, plo);
      sc.product(mk, vB, phi, plo);
      if (t + 2 >= m) break;
      chunk_rsrc<D>(g, sc.p, c0 + (t + 4) * cstride, &rk, &rv);
      sc.kload(rk, kB);
      sc.vload(rv, 0xffffu, vB);
      mk = sc.score(c0 + (t + 2) * cstride, kC, phi, plo);
      sc.product(mk, vC, phi, plo);
    }
  } else if (m > 0) {
    u32x4 kA[NK], kB[NK], vA[NK], vB[NK];
    u32x2 hA[RB], lA[RB], hB[RB], lB[RB];
    rsrc_t rk, rv, rk1, rv1;
    chunk_rsrc<D>(g, sc.p, c0, &rk, &rv);
    sc.kload(rk, kA);
    chunk_rsrc<D>(g, sc.p, c0 + cstride, &rk1, &rv1);
    sc.kload(rk1, kB);
    uint32_t mA = sc.score(c0, kA, hA, lA);
    sc.vload(rv, mA, vA);
    uint32_t mB = 0;
    for (int t = 0; t < m; t += 2) {
      // chunk t: values in vA, weights hA/lA; chunk t+1: keys in kB (resources rk1/rv1)
      chunk_rsrc<D>(g, sc.p, c0 + (t + 2) * cstride, &rk, &rv);
      sc.kload(rk, kA);
      mB = sc.score(c0 + (t + 1) * cstride, kB, hB, lB);
      sc.vload(rv1, mB, vB);
      sc.product(mA, vA, hA, lA);
      if (t + 1 >= m) break;
      // chunk t+1: values in vB; chunk t+2: keys in kA (resources rk/rv)
      chunk_rsrc<D>(g, sc.p, c0 + (t + 3) * cstride, &rk1, &rv1);
      sc.kload(rk1, kB);
      mA = sc.score(c0 + (t + 2) * cstride, kA, hA, lA);
      sc.vload(rv, mA, vA);
      sc.product(mB, vB, hB, lB);
    }
  }

  // L partials: lanes of one row (l%16) hold different keys; add them.
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    sc.lsum[b] += __shfl_xor(sc.lsum[b], 16, 64);
    sc.lsum[b] += __shfl_xor(sc.lsum[b], 32, 64);
    if (!DENSE) {
      sc.lcut[b] += __shfl_xor(sc.lcut[b], 16, 64);
      sc.lcut[b] += __shfl_xor(sc.lcut[b], 32, 64);
    }
  }

  // Add the four waves in order through LDS (the value tiles are dead now),
  // in the accumulators' own lane order so that no two lanes share a bank.
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);  // [RB][NB][4][64]
  float* redl = red + RB * S::NB * 4 * 64;      // [RB][64]
  for (int w = 0; w < kScanWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int b = 0; b < RB; ++b) {
#pragma unroll
        for (int blk = 0; blk < S::NB; ++blk)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float* r = red + ((b * S::NB + blk) * 4 + i) * 64 + sc.lane;
            *r = (w == 0 ? 0.0f : *r) + sc.acc[b][blk][i];
          }
        // lanes 0-15 add the row's L, lanes 16-31 its cut mass
        if (sc.lane < 32) {
          float* d = redl + b * 64 + sc.lane;
          *d = (w == 0 ? 0.0f : *d) + (sc.lane < 16 ? sc.lsum[b] : sc.lcut[b]);
        }
      }
    }
    __syncthreads();
  }

  // The LDS sums sit at ((b * NB + blk) * 4 + i) * 64 + l for row 16 b + l%16
  // and channel 16 blk + 4 (l/16) + i.  Wave i, lane l writes those entries of
  // every (b, blk): the rows its lane held during the scan, whose query-row
  // indices are already known.  No load is issued here: on gfx9 a wait for one
  // would also wait for the partial stores already in flight.
  const size_t slot_rows = (static_cast<size_t>(a.slot_offset) + sc.p.split) * g.batch * g.heads;
  const int wl = threadIdx.x & 63;
  const int wi = threadIdx.x >> 6;
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    if (!sc.rok[b]) continue;
    const size_t row = slot_rows + sc.xrow[b];
#pragma unroll
    for (int blk = 0; blk < S::NB; ++blk)
      a.part_A[row * D + 16 * blk + 4 * (wl >> 4) + wi] = red[((b * S::NB + blk) * 4 + wi) * 64 + wl];
    if (wi == 0 && wl < 16) a.part_L[row] = redl[b * 64 + wl];
    if (a.part_Lcut && wi == 1 && wl < 16) a.part_Lcut[row] = redl[b * 64 + 16 + wl];
  }
}

template <int D, int RB, bool DENSE>
hipError_t launch_rb(const DecodeArgs& a, bool dbg, unsigned blocks, hipStream_t stream) {
  bool cx = false;
  if constexpr (!DENSE) cx = !dbg && a.chunk_cut;
  if (dbg) {
    hipLaunchKernelGGL((decode_mfma_kernel<D, RB, DENSE, true>), dim3(blocks), dim3(kScanThreads),
                       0, stream, a);
  } else if (cx) {
    if constexpr (!DENSE)
      hipLaunchKernelGGL((decode_mfma_kernel<D, RB, DENSE, false, true>), dim3(blocks),
                         dim3(kScanThreads), 0, stream, a);
  } else
    hipLaunchKernelGGL((decode_mfma_kernel<D, RB, DENSE, false>), dim3(blocks), dim3(kScanThreads),
                       0, stream, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_mfma_d(const DecodeArgs& a, unsigned blocks, hipStream_t stream) {
  const bool dbg = a.x_out || a.key_gate_out || a.page_gate_out;
  const int rb = a.rows_per_group / 16;
  if (rb == 1) return a.dense ? launch_rb<D, 1, true>(a, dbg, blocks, stream)
                              : launch_rb<D, 1, false>(a, dbg, blocks, stream);
  if (rb == 2) return a.dense ? launch_rb<D, 2, true>(a, dbg, blocks, stream)
                              : launch_rb<D, 2, false>(a, dbg, blocks, stream);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_decode_packed(const DecodeArgs& a, int head_dim, hipStream_t stream);

hipError_t launch_decode_mfma(const DecodeArgs& a, int head_dim, hipStream_t stream) {
  // at most eight rows per kv sequence: several chunks per score pass
  if (a.rows_per_seq <= 8) return launch_decode_packed(a, head_dim, stream);
  const long long blocks = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv * a.num_splits *
                           a.row_groups;
  if (blocks == 0) return hipSuccess;
  if (head_dim == 128) return launch_mfma_d<128>(a, static_cast<unsigned>(blocks), stream);
  if (head_dim == 64) return launch_mfma_d<64>(a, static_cast<unsigned>(blocks), stream);
  return hipErrorInvalidValue;
}

}  // namespace fold
