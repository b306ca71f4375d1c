// Split-KV decode scan for read groups of at most eight query rows, at any
// depth: the GQA groups of 2, 4 or 8 rows that attend one kv sequence
// (Section 4 "Weight-gated reads", "Value product", "Depth as a dial";
// Algorithm 1).  At T = inf (DENSE) every key is live and a step's value rows
// are all requested once its keys are scored.
//
// Workgroup = (kv sequence, kv head, split); four wave64s; wave w owns the
// 16-key chunks 4t + w of its split's 64-key tiles, as in the other scans.  A
// step takes PK of the wave's chunks, PK = 16 / BW, where BW (4 or 8) bounds
// the group's rows:
//
//   keys      whole 128-byte lines per load (lane l: bytes 1024 c + 16 l of
//             the chunk), non-temporal, turned into the QK operand layout
//             through the wave's LDS tile.
//   scores    one v_mfma_f32_16x16x32_bf16 chain per chunk: keys on M, rows on
//             N.  Only the first BW lanes of each 16-lane row carry a row.
//   packing   DPP row shifts with bank masks move chunk p's row lanes to lanes
//             [BW p, BW p + BW) of every 16-lane row, so that one register set
//             holds the scores of the step's PK chunks with every lane on a
//             real (row, key) pair.  x = s - Z, the verdict x >= -T, the
//             weight 2^x and the cut mass take one pass per step instead of
//             one per chunk.  L adds the weights in the dense scan's order, so
//             that it has the same bits at every depth (mass kept exactly).
//   read mask the live bits of a lane's four keys, ORed over the rows of its
//             chunk (quad DPP) and over the four key groups (lane exchanges),
//             give every chunk's 16-bit value-read mask at once.
//   values    issued only for steps with a live key; cut keys of such a chunk
//             get offsets past its buffer resource, so no bytes move for them.
//   product   at the start of the next step: the packed x of a chunk with a
//             live key go back to the MFMA operand layout (DPP row shifts),
//             the live weights enter as bf16 hi + bf16 residual, and
//             A^T += V^T P^T runs on v_mfma_f32_16x16x16_bf16 with V^T read
//             transposed from the wave's value tile in LDS.
//
// CX (block model of BF16 values, finite T): each scored chunk's cut mass per
// row, the summed weights of its cut keys, is also written to chunk_cut.
//
// Two register sets of PK chunks alternate: the keys of step j+1 load while
// step j is scored, and a step's value rows reuse its key registers.  A step
// without a live key issues no value load, so at small depths the key stream
// of the next step is the only load a wave waits for.
#include "decode_common.h"
#include "estimate_device.h"
#include "fused_combine.h"

namespace fold {
namespace {

typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Lanes selected by BANKS (4-lane banks of each 16-lane row) receive src moved
// by the DPP control CTRL; the others keep old.
template <int CTRL, int BANKS>
__device__ __forceinline__ float dpp_move(float old, float src) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(src),
                                                    CTRL, 0xF, BANKS, false));
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_or(uint32_t v) {
  return v | static_cast<uint32_t>(
                 __builtin_amdgcn_update_dpp(0, static_cast<int>(v), CTRL, 0xF, 0xF, false));
}

constexpr int kDppRowShl = 0x100;    // row_shl:n = 0x100 + n (lane i reads lane i + n)
constexpr int kDppRowShr = 0x110;    // row_shr:n = 0x110 + n (lane i reads lane i - n)
constexpr int kDppIdentity = 0xE4;   // quad_perm [0, 1, 2, 3]

template <int D, int PK, bool DENSE, bool DBG, bool CX>
struct PackedScan {
  static constexpr int NK = D / 32;           // 128-bit loads per lane per chunk
  static constexpr int NB = D / 16;           // 16-channel blocks of the value product
  static constexpr int BW = 16 / PK;          // lanes (rows) per chunk in the packed layout
  static constexpr int VSTRIDE = 2 * D + 16;  // bytes per key row of the LDS value tile

  // Banks (4 lanes each) of chunk slot q in the packed layout.
  template <int Q>
  static constexpr int banks() { return ((1 << (BW / 4)) - 1) << (Q * BW / 4); }

  const DecodeArgs& a;
  const ScanGeometry& g;
  ScanPlace p;
  int lane, n16, grp;
  int cstride, c0;
  int slot;          // chunk slot of this lane's bank in the packed layout (n16 / BW)
  size_t gate_row;
  unsigned char* vt; // this wave's value tile [16][VSTRIDE]

  u32x4 qb[NK];      // Q^T operand of row n16
  bool rok;          // row n16 exists
  size_t xrow;       // its query row index
  bool pok;          // packed row n16 % BW exists
  size_t prow;       // its query row index
  float zp;          // its reference
  f32x4 acc[NB];
  float lsum, lcut;
  float xs[4];       // packed weights of the last scored step entering A (0: cut or no key)
  uint32_t ms[PK];   // value-read masks of its chunks

  __device__ PackedScan(const DecodeArgs& a_) : a(a_), g(a_.geo) {}

  __device__ __forceinline__ int chunk_of(int step, int q) const {
    return c0 + (step * PK + q) * cstride;
  }

  __device__ __forceinline__ void issue_keys(int step, u32x4 (&X)[PK][NK], rsrc_t (&rv)[PK]) {
#pragma unroll
    for (int q = 0; q < PK; ++q) {
      rsrc_t rk;
      chunk_rsrc<D>(g, p, chunk_of(step, q), &rk, &rv[q]);
      // whole lines: lane l, load c takes the 16 bytes at 1024 c + 16 l
#pragma unroll
      for (int c = 0; c < NK; ++c) X[q][c] = buf_load(rk, 1024u * c + 16u * lane);
    }
  }

  __device__ __forceinline__ void issue_values(u32x4 (&X)[PK][NK], const rsrc_t (&rv)[PK]) const {
#pragma unroll
    for (int q = 0; q < PK; ++q) {
      // lane l, load i: the 16 bytes at 1024 i + 16 l of the chunk (key (1024 i + 16 l) / 2D)
#pragma unroll
      for (int i = 0; i < NK; ++i) {
        const uint32_t off = 1024u * i + 16u * lane;
        const uint32_t key = off / (2 * D);
        X[q][i] = buf_load(rv[q], DENSE || ((ms[q] >> key) & 1u) ? off : kOutOfRange);
      }
    }
  }

  template <int Q>
  __device__ __forceinline__ void add_in_chunk_order(const float (&w)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      lsum += Q == 0 ? w[i] : dpp_move<kDppRowShl + Q * BW, 0xF>(0.0f, w[i]);
  }

  // Scores of the step's chunks, packed; verdicts, weights, L and cut mass;
  // the chunks' read masks.  Returns their union (wave-uniform).
  __device__ __forceinline__ uint32_t score(int step, const u32x4 (&X)[PK][NK]) {
    f32x4 s[PK];
#pragma unroll
    for (int q = 0; q < PK; ++q) {
      // the QK A operand (lane l: key l%16, channels 32c + 8(l/16) .. +8)
      // through the wave's tile, rows padded to VSTRIDE bytes
#pragma unroll
      for (int c = 0; c < NK; ++c) {
        const uint32_t off = 1024u * c + 16u * lane;
        const uint32_t key = off / (2 * D);
        *reinterpret_cast<u32x4*>(vt + key * VSTRIDE + (off - key * 2 * D)) = X[q][c];
      }
      u32x4 ka[NK];
#pragma unroll
      for (int c = 0; c < NK; ++c)
        ka[c] = *reinterpret_cast<const u32x4*>(vt + n16 * VSTRIDE + 64 * c + 16 * grp);
      s[q] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int c = 0; c < NK; ++c) s[q] = mfma_16x16x32(ka[c], qb[c], s[q]);
    }
    float sv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sv[i] = s[0][i];
      if constexpr (PK >= 2) sv[i] = dpp_move<kDppRowShr + BW, banks<1>()>(sv[i], s[1][i]);
      if constexpr (PK == 4) {
        sv[i] = dpp_move<kDppRowShr + 2 * BW, banks<2>()>(sv[i], s[2][i]);
        sv[i] = dpp_move<kDppRowShr + 3 * BW, banks<3>()>(sv[i], s[3][i]);
      }
    }
    // this lane's chunk and its valid keys
    const int cl = chunk_of(step, slot);
    const int nkl = cl < p.nchunks ? min(kChunk, p.n - cl * kChunk) : 0;
    uint32_t bits = 0;
    float w[4];
    float cc = 0.0f;  // cut weights of this lane's keys of chunk cl
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int kk = 4 * grp + i;
      const bool ok = pok && kk < nkl;
      const float x = ok ? __builtin_fmaf(sv[i], a.score_scale, -zp) : -INFINITY;
      const bool live = DENSE ? ok : x >= a.neg_T;
      w[i] = exp2_fast(x);
      if (!DENSE) lcut += live ? 0.0f : w[i];
      if (!DENSE && (CX || DBG)) cc += live ? 0.0f : w[i];
      xs[i] = live ? w[i] : 0.0f;  // the product takes these weights as they are
      bits |= live ? (1u << i) : 0u;
      if (DBG && a.x_out && ok) a.x_out[prow * g.max_seq_len + cl * kChunk + kk] = x;
    }
    if constexpr (!DENSE && (CX || DBG)) {
      if (a.chunk_cut) {
        // the four key groups of a packed (row, chunk) lane hold its 16 keys
        cc += __shfl_xor(cc, 16, 64);
        cc += __shfl_xor(cc, 32, 64);
        if (grp == 0 && pok && cl < p.nchunks) a.chunk_cut[prow * a.chunk_stride + cl] = cc;
      }
    }
    // L adds the weights in the dense scan's order (chunk by chunk, then key
    // 4 grp + i), in the lanes of chunk slot 0, so that L has the same bits at
    // every depth: each chunk's weights are moved back to those lanes.
    add_in_chunk_order<0>(w);
    if constexpr (PK >= 2) add_in_chunk_order<1>(w);
    if constexpr (PK == 4) {
      add_in_chunk_order<2>(w);
      add_in_chunk_order<3>(w);
    }
    // OR over the rows of the chunk (the lanes of its bank or banks) ...
    bits = dpp_or<0xB1>(bits);                      // quad_perm [1, 0, 3, 2]
    bits = dpp_or<0x4E>(bits);                      // quad_perm [2, 3, 0, 1]
    if constexpr (BW == 8) bits = dpp_or<0x141>(bits);  // row_half_mirror
    // ... and over the key groups: bit 4 grp + i is key 4 grp + i of the chunk
    bits <<= 4 * grp;
    bits |= static_cast<uint32_t>(__shfl_xor(static_cast<int>(bits), 16, 64));
    bits |= static_cast<uint32_t>(__shfl_xor(static_cast<int>(bits), 32, 64));
    uint32_t any = 0;
#pragma unroll
    for (int q = 0; q < PK; ++q) {
      ms[q] = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(bits), BW * q));
      any |= ms[q];
    }
    if (DBG) {
#pragma unroll
      for (int q = 0; q < PK; ++q) {
        const int c = chunk_of(step, q);
        const int nk = c < p.nchunks ? min(kChunk, p.n - c * kChunk) : 0;
        if (a.key_gate_out && lane < nk)
          a.key_gate_out[gate_row * g.max_seq_len + c * kChunk + lane] = (ms[q] >> lane) & 1u;
        if (a.page_gate_out && lane == 0 && c < p.nchunks)
          a.page_gate_out[gate_row * ((g.max_seq_len + kChunk - 1) / kChunk) + c] = ms[q] ? 1 : 0;
      }
    }
    return any;
  }

  // Value product of chunk slot Q of the last scored step (values in V).
  template <int Q>
  __device__ __forceinline__ void product_chunk(const u32x4 (&V)[NK]) {
    if (ms[Q] == 0) return;  // wave-uniform
#pragma unroll
    for (int i = 0; i < NK; ++i) {
      const uint32_t off = 1024u * i + 16u * lane;
      const uint32_t key = off / (2 * D);
      *reinterpret_cast<u32x4*>(vt + key * VSTRIDE + (off - key * 2 * D)) = V[i];
    }
    // x of the chunk in the operand layout (lane l: keys 4(l/16)+i of row l%16)
    uint32_t hi[4], lo[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float pw =
          dpp_move<Q == 0 ? kDppIdentity : kDppRowShl + Q * BW, banks<0>()>(0.0f, xs[i]);
      hi[i] = __float_as_uint(pw) & 0xffff0000u;
      lo[i] = f32_to_bf16_rne(pw - __uint_as_float(hi[i]));
    }
    const u32x2 phi = {(hi[0] >> 16) | hi[1], (hi[2] >> 16) | hi[3]};
    const u32x2 plo = {lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16)};
    // V^T: lane 4i + a of each 16-lane group points at channels 16 blk + 4a .. +4
    // of key 4(l/16) + i; lane l receives channel 16 blk + l%16 of those keys.
    const unsigned char* src = vt + (4 * grp + (n16 >> 2)) * VSTRIDE + 8 * (n16 & 3);
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
      const u32x2 va = __builtin_bit_cast(
          u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(src + 32 * blk)));
      acc[blk] = mfma_16x16x16(va, phi, acc[blk]);
      acc[blk] = mfma_16x16x16(va, plo, acc[blk]);
    }
  }

  __device__ __forceinline__ void product(const u32x4 (&X)[PK][NK]) {
    product_chunk<0>(X[0]);
    if constexpr (PK >= 2) product_chunk<1>(X[1]);
    if constexpr (PK == 4) {
      product_chunk<2>(X[2]);
      product_chunk<3>(X[3]);
    }
  }
};

// The scan of one (kv sequence, kv head, split) workgroup.  FUSED (the
// one-launch decode of a single level, per-request view): the prologue
// computes the group's references with the estimate routine while the first
// keys load, and the last split to finish adds the slots into the output.
template <int D, int PK, bool DENSE, bool DBG, bool FUSED, bool CX = false>
__device__ __forceinline__ void packed_scan(const DecodeArgs& a, const FusedExtra* fx) {
  using S = PackedScan<D, PK, DENSE, DBG, CX>;
  constexpr int NK = S::NK;
  constexpr int kTileBytes = kScanWaves * 16 * S::VSTRIDE;
  constexpr int kWaveFloats = S::NB * 4 * 64 + 64;  // one wave's accumulators, L and cut mass
  constexpr int kRedBytes = kScanWaves * kWaveFloats * 4;
  constexpr int kEstBytes = FUSED ? kMaxEstRows * kMaxEstSamples * 4 : 0;  // the estimate's scores
  constexpr int kSmemBytes = kTileBytes > kRedBytes ? (kTileBytes > kEstBytes ? kTileBytes : kEstBytes)
                                                    : (kRedBytes > kEstBytes ? kRedBytes : kEstBytes);
  __shared__ __attribute__((aligned(16))) unsigned char smem[kSmemBytes];

  const ScanGeometry& g = a.geo;
  S sc(a);
  sc.p = scan_place(a);
  if (sc.p.rg > 0) return;  // one read group holds every row
  sc.lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  sc.n16 = sc.lane & 15;
  sc.grp = sc.lane >> 4;
  sc.slot = sc.n16 / S::BW;
  sc.vt = smem + wave * 16 * S::VSTRIDE;
  sc.gate_row = static_cast<size_t>(sc.p.seq) * g.hkv + sc.p.kvh;

  {
    const RowInfo ri = row_info(g, sc.p.seq, sc.p.kvh, sc.n16, sc.p.nrows, sc.p.req0);
    sc.rok = ri.ok;
    const size_t row = static_cast<size_t>(ri.req) * g.heads + ri.head;
    sc.xrow = row;
#pragma unroll
    for (int c = 0; c < NK; ++c)
      sc.qb[c] = ri.ok ? *reinterpret_cast<const u32x4*>(a.q + row * D + 32 * c + 8 * sc.grp)
                       : u32x4{0, 0, 0, 0};
    const RowInfo rp = row_info(g, sc.p.seq, sc.p.kvh, sc.n16 % S::BW, sc.p.nrows, sc.p.req0);
    sc.pok = rp.ok;
    sc.prow = static_cast<size_t>(rp.req) * g.heads + rp.head;
    if (!FUSED) sc.zp = rp.ok ? a.z[sc.prow] : 0.0f;
  }
  sc.lsum = 0.0f;
  sc.lcut = 0.0f;
#pragma unroll
  for (int blk = 0; blk < S::NB; ++blk) sc.acc[blk] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  sc.cstride = kScanWaves * a.num_splits;
  sc.c0 = kScanWaves * sc.p.split + wave;
  const int m = sc.p.nchunks > sc.c0 ? (sc.p.nchunks - sc.c0 + sc.cstride - 1) / sc.cstride : 0;
  const int steps = (m + PK - 1) / PK;

  u32x4 X0[PK][NK], X1[PK][NK];
  rsrc_t rv0[PK], rv1[PK];
  __shared__ float zs[16];  // FUSED: Z of row n16
  if constexpr (FUSED) {
    // Z of the group's rows (split 0 also writes them out); the wave's first
    // keys are issued as soon as the estimate's sample loads are, so they
    // fly during its second round trip.  The scores' LDS is free again after
    // the barrier.
    est::estimate_rows<D, false, false>(fx->est, sc.p.seq, sc.p.kvh,
                                        reinterpret_cast<float (*)[kMaxEstSamples]>(smem), nullptr,
                                        nullptr, sc.p.split == 0, zs,
                                        [&] { sc.issue_keys(0, X0, rv0); });
    __syncthreads();
    sc.zp = sc.pok ? zs[sc.n16 % S::BW] : 0.0f;
  } else {
    sc.issue_keys(0, X0, rv0);
  }
  bool pend = false;  // the last scored step has value rows in flight
  for (int j = 0; j < steps; j += 2) {
    if (pend) sc.product(X1);  // step j - 1
    sc.issue_keys(j + 1, X1, rv1);
    pend = sc.score(j, X0) != 0;
    if (pend) sc.issue_values(X0, rv0);
    if (j + 1 >= steps) break;
    if (pend) sc.product(X0);  // step j
    sc.issue_keys(j + 2, X0, rv0);
    pend = sc.score(j + 1, X1) != 0;
    if (pend) sc.issue_values(X1, rv1);
  }
  if (pend) {
    if ((steps - 1) & 1)
      sc.product(X1);
    else
      sc.product(X0);
  }

  // L: lane n16 < BW of each key group holds row n16's chunk-ordered sum; add
  // the key groups as the dense scan does.  Cut mass: the lanes of packed row
  // r (n16 % BW == r, every key group) hold different keys; add them.
#pragma unroll
  for (int sh = S::BW; sh < 16; sh <<= 1) sc.lcut += __shfl_xor(sc.lcut, sh, 64);
  sc.lsum += __shfl_xor(sc.lsum, 16, 64);
  sc.lsum += __shfl_xor(sc.lsum, 32, 64);
  sc.lcut += __shfl_xor(sc.lcut, 16, 64);
  sc.lcut += __shfl_xor(sc.lcut, 32, 64);

  // Add the four waves through LDS (the tiles are dead now): each wave stores
  // its accumulators in its own region (in their lane order, so that no two
  // lanes share a bank), one barrier, then every thread adds four channels of
  // one row over the waves in wave order and stores them as one 16-byte group.
  // Row n16's accumulator sits at (blk * 4 + i) * 64 + l with l % 16 = n16 and
  // channel 16 blk + 4 (l / 16) + i; lanes 0-15 of a region hold L, lanes
  // 16-31 the cut mass (lane n16 < BW holds packed row n16).
  __shared__ long long out_row[16];  // query row of row n16, or -1
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);
  {
    float* mine = red + wave * kWaveFloats;
#pragma unroll
    for (int blk = 0; blk < S::NB; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) mine[(blk * 4 + i) * 64 + sc.lane] = sc.acc[blk][i];
    if (sc.lane < 32) mine[S::NB * 4 * 64 + sc.lane] = sc.lane < 16 ? sc.lsum : sc.lcut;
    if (wave == 0 && sc.lane < 16) out_row[sc.lane] = sc.rok ? static_cast<long long>(sc.xrow) : -1;
  }
  __syncthreads();
  const size_t slot_rows = (static_cast<size_t>(a.slot_offset) + sc.p.split) * g.batch * g.heads;
  const bool vec_ok = (reinterpret_cast<uintptr_t>(a.part_A) & 15u) == 0;
  rsrc_t ra, rl;  // FUSED: the slot arrays
  if constexpr (FUSED) slot_rsrc<D>(a, &ra, &rl);
  for (int f = threadIdx.x; f < 16 * (D / 4); f += kScanThreads) {
    const int r = f / (D / 4);
    const int d = 4 * (f % (D / 4));
    const long long xr = out_row[r];
    if (xr < 0) continue;
    const int base = (d / 16) * 4 * 64 + 16 * ((d % 16) / 4) + r;
    float v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = base + i * 64;
      v[i] = ((red[e] + red[kWaveFloats + e]) + red[2 * kWaveFloats + e]) + red[3 * kWaveFloats + e];
    }
    float* dst = a.part_A + (slot_rows + static_cast<size_t>(xr)) * D + d;
    if constexpr (FUSED) {
      slot_store4(ra, static_cast<uint32_t>((slot_rows + static_cast<size_t>(xr)) * D + d) * 4u,
                  f32x4{v[0], v[1], v[2], v[3]});
    } else if (vec_ok) {
      *reinterpret_cast<f32x4*>(dst) = f32x4{v[0], v[1], v[2], v[3]};
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[i] = v[i];
    }
  }
  if (threadIdx.x < 32) {
    const int r = threadIdx.x & 15;
    const long long xr = out_row[r];
    const int e = S::NB * 4 * 64 + threadIdx.x;
    const float v = ((red[e] + red[kWaveFloats + e]) + red[2 * kWaveFloats + e]) + red[3 * kWaveFloats + e];
    if (xr >= 0) {
      if (FUSED && threadIdx.x < 16)
        slot_store1(rl, static_cast<uint32_t>(slot_rows + static_cast<size_t>(xr)) * 4u, v);
      else if (threadIdx.x < 16)
        a.part_L[slot_rows + static_cast<size_t>(xr)] = v;
      else if (a.part_Lcut)
        a.part_Lcut[slot_rows + static_cast<size_t>(xr)] = v;
    }
  }
  if constexpr (FUSED) fused_combine<D>(a, *fx, sc.p, out_row, zs);
}

template <int D, int PK, bool DENSE, bool DBG, bool CX = false>
__global__ __launch_bounds__(kScanThreads) __attribute__((amdgpu_waves_per_eu(2))) void decode_packed_kernel(const DecodeArgs a) {
  packed_scan<D, PK, DENSE, DBG, false, CX>(a, nullptr);
}

template <int D, int PK, bool DENSE>
__global__ __launch_bounds__(kScanThreads) __attribute__((amdgpu_waves_per_eu(2))) void decode_fused_kernel(const FusedArgs fa) {
  packed_scan<D, PK, DENSE, false, true>(fa.d, &fa.x);
}

template <int D, int PK, bool DENSE>
hipError_t launch_pkd(const DecodeArgs& a, bool dbg, unsigned blocks, hipStream_t stream) {
  bool cx = false;
  if constexpr (!DENSE) cx = !dbg && a.chunk_cut;
  if (dbg) {
    hipLaunchKernelGGL((decode_packed_kernel<D, PK, DENSE, true>), dim3(blocks),
                       dim3(kScanThreads), 0, stream, a);
  } else if (cx) {
    if constexpr (!DENSE)
      hipLaunchKernelGGL((decode_packed_kernel<D, PK, DENSE, false, true>), dim3(blocks),
                         dim3(kScanThreads), 0, stream, a);
  } else
    hipLaunchKernelGGL((decode_packed_kernel<D, PK, DENSE, false>), dim3(blocks),
                       dim3(kScanThreads), 0, stream, a);
  return hipGetLastError();
}

template <int D, int PK>
hipError_t launch_pk(const DecodeArgs& a, unsigned blocks, hipStream_t stream) {
  const bool dbg = a.x_out || a.key_gate_out || a.page_gate_out;
  return a.dense ? launch_pkd<D, PK, true>(a, dbg, blocks, stream)
                 : launch_pkd<D, PK, false>(a, dbg, blocks, stream);
}

template <int D, int PK>
hipError_t launch_fused_pk(const FusedArgs& a, unsigned blocks, hipStream_t stream) {
  if (a.d.dense)
    hipLaunchKernelGGL((decode_fused_kernel<D, PK, true>), dim3(blocks), dim3(kScanThreads), 0,
                       stream, a);
  else
    hipLaunchKernelGGL((decode_fused_kernel<D, PK, false>), dim3(blocks), dim3(kScanThreads), 0,
                       stream, a);
  return hipGetLastError();
}

}  // namespace

// One-launch decode of a single level: read groups of two to eight rows of a
// per-request view.
hipError_t launch_decode_fused(const FusedArgs& a, int head_dim, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.d.geo.num_seqs) * a.d.geo.hkv * a.d.num_splits;
  if (blocks == 0) return hipSuccess;
  const unsigned nb = static_cast<unsigned>(blocks);
  const bool four = a.d.rows_per_seq <= 4;
  if (head_dim == 128) return four ? launch_fused_pk<128, 4>(a, nb, stream) : launch_fused_pk<128, 2>(a, nb, stream);
  if (head_dim == 64) return four ? launch_fused_pk<64, 4>(a, nb, stream) : launch_fused_pk<64, 2>(a, nb, stream);
  return hipErrorInvalidValue;
}

// Scan of read groups of at most eight rows (one read group per kv sequence
// and head), at any depth.
hipError_t launch_decode_packed(const DecodeArgs& a, int head_dim, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv * a.num_splits;
  if (blocks == 0) return hipSuccess;
  const unsigned nb = static_cast<unsigned>(blocks);
  const bool four = a.rows_per_seq <= 4;
  if (head_dim == 128) return four ? launch_pk<128, 4>(a, nb, stream) : launch_pk<128, 2>(a, nb, stream);
  if (head_dim == 64) return four ? launch_pk<64, 4>(a, nb, stream) : launch_pk<64, 2>(a, nb, stream);
  return hipErrorInvalidValue;
}

}  // namespace fold
