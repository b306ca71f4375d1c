// Split-KV decode over a two-plane INT8 key cache for read groups of at most
// eight query rows, at any depth (Section 4, "Cache format", "Weight-gated reads",
// "Value product", "Depth as a dial"; Algorithm 1 with BF16 or 8-bit values).
//
// The arithmetic is the two-plane scan's (decode_q8.hip): coarse scores from
// plane A and the key scales, per-GQA-group live / refine-K / refine-V verdicts
// on them, plane B only for refined keys, value rows only for live keys, the
// weight 2^x with every key's weight in L.  What differs is the work layout,
// as in the packed BF16 scan:
//
//   loads     plane A (and B, and the values) as whole 128-byte lines: lane
//             l, load c takes bytes 1024 c + 16 l of the chunk; a plane chunk
//             reaches the i8 operand layout (lane l: 16 bytes of key l%16)
//             through the wave's LDS tile.
//   packing   a step takes PK = 2 of the wave's chunks, each on BW = 8 of the
//             16 row lanes (the rows are at most eight).  The integer coarse products of the PK chunks
//             are packed by DPP row shifts with bank masks, so every lane
//             holds a real (row, key) pair: the coarse score, the three
//             verdicts, the group ORs and the read masks cost one pass per
//             step; so do the refined score, the weight, L and the cut mass.
//   pipeline  plane A of steps j+1 and j+2 is in flight while step j is
//             scored; step j's plane-B rows and value rows are requested once
//             it is scored, before plane A of step j+2, and used in the same
//             step (refine, weights, products).  A step without a refined or
//             live key requests nothing beyond plane A and the scales and
//             waits for nothing but plane A.
#include "q8_common.h"

namespace fold {
namespace {

template <int CTRL, int BANKS>
__device__ __forceinline__ float dpp_movf(float old, float src) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(src),
                                                    CTRL, 0xF, BANKS, false));
}

template <int CTRL, int BANKS>
__device__ __forceinline__ int dpp_movi(int old, int src) {
  return __builtin_amdgcn_update_dpp(old, src, CTRL, 0xF, BANKS, false);
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_or(uint32_t v) {
  return v | static_cast<uint32_t>(
                 __builtin_amdgcn_update_dpp(0, static_cast<int>(v), CTRL, 0xF, 0xF, false));
}

constexpr int kDppRowShl = 0x100;   // row_shl:n = 0x100 + n (lane i reads lane i + n)
constexpr int kDppRowShr = 0x110;   // row_shr:n = 0x110 + n (lane i reads lane i - n)
constexpr int kDppIdentity = 0xE4;  // quad_perm [0, 1, 2, 3]

template <int D, int PK, bool DENSE, bool DBG, bool V8>
struct Q8Packed {
  static constexpr int NKI = D / 64;               // plane loads per lane per chunk
  static constexpr int NKV = V8 ? D / 64 : D / 32;  // value loads per lane per chunk
  static constexpr int NB = D / 16;                // 16-channel blocks of the value product
  static constexpr int BW = 16 / PK;               // lanes (rows) per chunk, packed
  static constexpr int VSTRIDE = 2 * D + 16;       // bytes per row of the LDS value tile
  static constexpr int PSTRIDE = D + 16;           // bytes per row of the LDS plane tile

  template <int Q>
  static constexpr int banks() { return ((1 << (BW / 4)) - 1) << (Q * BW / 4); }
  template <int Q>
  static constexpr int to_packed() { return Q == 0 ? kDppIdentity : kDppRowShr + Q * BW; }
  template <int Q>
  static constexpr int from_packed() { return Q == 0 ? kDppIdentity : kDppRowShl + Q * BW; }

  const Q8DecodeArgs& a;
  const ScanGeometry& g;
  ScanPlace p;
  int lane, n16, grp, slot, cstride, c0, pshift, gspan;
  size_t gate_row;
  unsigned char* vt;

  u32x4 qa[NKI], qb[NKI];  // query planes of row n16 (the operand layout)
  bool rok;
  size_t xrow;
  bool pok;                // packed row n16 % BW
  size_t prow;
  float zp, etap, ntaup, ntauvp;
  f32x4 acc[NB];
  float lsum, lcut;
  // the last scored step, packed: coarse x (-inf for no key), key scales,
  // 4-bit fields of the lane's keys (exists, group refine-K, group refine-V)
  float xc[4], e[4];
  uint32_t okl, refl, refvl;
  uint32_t vm[PK], bm[PK], rvm[PK];  // per-chunk read masks (wave-uniform)
  uint32_t anyb, anyv;

  __device__ Q8Packed(const Q8DecodeArgs& a_) : a(a_), g(a_.d.geo) {}

  __device__ __forceinline__ int chunk_of(int step, int q) const {
    return c0 + (step * PK + q) * cstride;
  }

  // Plane A and the scales of a step's chunks; lane l of chunk slot q's bank
  // fetches the scale of key 4(l/16) + l%4 of that chunk.
  __device__ __forceinline__ void issue_a(int step, u32x4 (&A)[PK][NKI], uint32_t& sc,
                                          Q8Loc (&loc)[PK]) const {
    sc = 0;
#pragma unroll
    for (int q = 0; q < PK; ++q) {
      const int c = chunk_of(step, q);
      loc[q] = q8_loc(g, p, c, q8_chunk_phys(g, p, c, pshift), pshift);
      const rsrc_t ra = make_rsrc(a.keys.ka + loc[q].row * D, loc[q].nk * D);
#pragma unroll
      for (int i = 0; i < NKI; ++i) A[q][i] = buf_load(ra, 1024u * i + 16u * lane);
      const rsrc_t rs = make_rsrc(a.keys.ks + loc[q].row, loc[q].nk * 2);
      sc |= buf_load2(rs, slot == q ? 2u * (4 * grp + (lane & 3)) : kOutOfRange);
    }
  }

  // Dense decode: every value row of a step's chunks (or the first E4M3
  // plane), requested together with its plane A.
  __device__ __forceinline__ void issue_v(const Q8Loc (&loc)[PK], u32x4 (&V)[PK][NKV]) const {
#pragma unroll
    for (int q = 0; q < PK; ++q) {
      const rsrc_t rv = V8 ? make_rsrc(a.vp + loc[q].row * D, loc[q].nk * D)
                           : make_rsrc(g.v + loc[q].row * D, loc[q].nk * D * 2);
#pragma unroll
      for (int i = 0; i < NKV; ++i) V[q][i] = buf_load(rv, 1024u * i + 16u * lane);
    }
  }

  // Plane-B rows of refined keys and value rows of live keys (and, 8-bit
  // values, second-plane rows of refine-V keys) of the scored step.
  __device__ __forceinline__ void issue_bv(const Q8Loc (&loc)[PK], u32x4 (&B)[PK][NKI],
                                           u32x4 (&V)[PK][NKV], u32x4 (&R)[PK][V8 ? D / 64 : 1]) const {
#pragma unroll
    for (int q = 0; q < PK; ++q) {
      if (bm[q]) {
        const rsrc_t rb = make_rsrc(a.keys.kb + loc[q].row * D, loc[q].nk * D);
#pragma unroll
        for (int i = 0; i < NKI; ++i) {
          const uint32_t off = 1024u * i + 16u * lane;
          B[q][i] = buf_load(rb, ((bm[q] >> (off / D)) & 1u) ? off : kOutOfRange);
        }
      }
      if (!DENSE && vm[q]) {  // dense decode: requested with plane A
        constexpr uint32_t kRowBytes = V8 ? D : 2 * D;
        const rsrc_t rv = V8 ? make_rsrc(a.vp + loc[q].row * D, loc[q].nk * D)
                             : make_rsrc(g.v + loc[q].row * D, loc[q].nk * D * 2);
#pragma unroll
        for (int i = 0; i < NKV; ++i) {
          const uint32_t off = 1024u * i + 16u * lane;
          V[q][i] = buf_load(rv, ((vm[q] >> (off / kRowBytes)) & 1u) ? off : kOutOfRange);
        }
      }
      if constexpr (V8) {
        if (rvm[q]) {
          const rsrc_t rr = make_rsrc(a.vr + loc[q].row * D, loc[q].nk * D);
#pragma unroll
          for (int i = 0; i < D / 64; ++i) {
            const uint32_t off = 1024u * i + 16u * lane;
            R[q][i] = buf_load(rr, ((rvm[q] >> (off / D)) & 1u) ? off : kOutOfRange);
          }
        }
      }
    }
  }

  // The i8 operand (lane l: key l%16, bytes 64c + 16(l/16) .. +16) of a plane
  // chunk from its whole-line loads, through the wave's tile.  The tile is
  // wave-private and used in program order.
  __device__ __forceinline__ void plane_operand(const u32x4 (&ld)[NKI], u32x4 (&op)[NKI]) const {
#pragma unroll
    for (int c = 0; c < NKI; ++c) {
      const uint32_t off = 1024u * c + 16u * lane;
      const uint32_t key = off / D;
      *reinterpret_cast<u32x4*>(vt + key * PSTRIDE + (off - key * D)) = ld[c];
    }
#pragma unroll
    for (int c = 0; c < NKI; ++c)
      op[c] = *reinterpret_cast<const u32x4*>(vt + n16 * PSTRIDE + 64 * c + 16 * grp);
  }

  template <int Q>
  __device__ __forceinline__ void coarse_chunk(const u32x4 (&A)[NKI], i32x4& caa, i32x4& cab) const {
    u32x4 ka[NKI];
    plane_operand(A, ka);
    i32x4 ta = {0, 0, 0, 0}, tb = {0, 0, 0, 0};
#pragma unroll
    for (int c = 0; c < NKI; ++c) {
      ta = mfma_i8(ka[c], qa[c], ta);
      tb = mfma_i8(ka[c], qb[c], tb);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      caa[i] = dpp_movi<to_packed<Q>(), banks<Q>()>(caa[i], ta[i]);
      cab[i] = dpp_movi<to_packed<Q>(), banks<Q>()>(cab[i], tb[i]);
    }
  }

  // Coarse scores, verdicts and read masks of a step (plane A in A, scales in sc).
  __device__ __forceinline__ void coarse(int step, const u32x4 (&A)[PK][NKI], uint32_t sc) {
    {  // scale of key 4(l/16)+i: lane i of the lane's quad fetched it
      const int v = static_cast<int>(sc);
      e[0] = bf16_lo(static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, v, 0x00, 0xF, 0xF, false)));
      e[1] = bf16_lo(static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, v, 0x55, 0xF, 0xF, false)));
      e[2] = bf16_lo(static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, v, 0xAA, 0xF, 0xF, false)));
      e[3] = bf16_lo(static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, v, 0xFF, 0xF, 0xF, false)));
    }
    i32x4 caa = {0, 0, 0, 0}, cab = {0, 0, 0, 0};
    coarse_chunk<0>(A[0], caa, cab);
    if constexpr (PK >= 2) coarse_chunk<1>(A[1], caa, cab);
    if constexpr (PK == 4) {
      coarse_chunk<2>(A[2], caa, cab);
      coarse_chunk<3>(A[3], caa, cab);
    }
    const int cl = chunk_of(step, slot);
    const int nkl = cl < p.nchunks ? min(kChunk, p.n - cl * kChunk) : 0;
    uint32_t lv = 0, rf = 0, rv = 0, okb = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool ok = pok && 4 * grp + i < nkl;
      const float t = static_cast<float>(caa[i]) + static_cast<float>(cab[i]) * (1.0f / 256.0f);
      const float x = __builtin_fmaf(etap * e[i], t, -zp);
      xc[i] = ok ? x : -INFINITY;
      if (ok) okb |= 1u << i;
      if (ok && (DENSE || x >= a.d.neg_T)) lv |= 1u << i;
      if (ok && x >= ntaup) rf |= 1u << i;
      if (V8 && ok && x >= ntauvp) rv |= 1u << i;
      if (DBG && a.xc_out && ok) a.xc_out[prow * g.max_seq_len + cl * kChunk + 4 * grp + i] = x;
    }
    okl = okb;
    // OR over the rows of one GQA group (aligned groups of G lanes of a bank);
    // refine only live keys
    uint32_t bits = lv | (rv << 8) | (rf << 16);
    if (gspan >= 1) bits = dpp_or<0xB1>(bits);   // quad_perm [1, 0, 3, 2]
    if (gspan >= 3) bits = dpp_or<0x4E>(bits);   // quad_perm [2, 3, 0, 1]
    if (gspan >= 7) bits = dpp_or<0x141>(bits);  // row_half_mirror
    bits &= ((bits & 0xFFu) << 16) | ((bits & 0xFFu) << 8) | 0xFFu;
    refl = (bits >> 16) & 0xFu;
    refvl = (bits >> 8) & 0xFu;
    // unions over the chunk's rows, then over the key groups: bit 4 grp + i
    // of each 16-bit field is key 4 grp + i of the chunk
    uint32_t u = dpp_or<0x4E>(dpp_or<0xB1>(bits));
    if constexpr (BW == 8) u = dpp_or<0x141>(u);
    uint32_t w1 = ((u & 0xFu) | (((u >> 16) & 0xFu) << 16)) << (4 * grp);
    w1 |= static_cast<uint32_t>(__shfl_xor(static_cast<int>(w1), 16, 64));
    w1 |= static_cast<uint32_t>(__shfl_xor(static_cast<int>(w1), 32, 64));
    uint32_t w2 = 0;
    if constexpr (V8) {
      w2 = ((u >> 8) & 0xFu) << (4 * grp);
      w2 |= static_cast<uint32_t>(__shfl_xor(static_cast<int>(w2), 16, 64));
      w2 |= static_cast<uint32_t>(__shfl_xor(static_cast<int>(w2), 32, 64));
    }
    anyb = anyv = 0;
#pragma unroll
    for (int q = 0; q < PK; ++q) {
      const uint32_t r = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(w1), BW * q));
      vm[q] = r & 0xFFFFu;
      bm[q] = r >> 16;
      rvm[q] = V8 ? static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(w2), BW * q)) : 0u;
      anyv |= vm[q];
      anyb |= bm[q];
    }
    if (DBG) {
#pragma unroll
      for (int q = 0; q < PK; ++q) {
        const int c = chunk_of(step, q);
        const int nk = c < p.nchunks ? min(kChunk, p.n - c * kChunk) : 0;
        const size_t kr = gate_row * g.max_seq_len + c * kChunk + lane;
        if (a.d.key_gate_out && lane < nk) a.d.key_gate_out[kr] = (vm[q] >> lane) & 1u;
        if (a.refine_gate_out && lane < nk) a.refine_gate_out[kr] = (bm[q] >> lane) & 1u;
        if (V8 && a.refine_v_gate_out && lane < nk) a.refine_v_gate_out[kr] = (rvm[q] >> lane) & 1u;
        if (a.d.page_gate_out && lane == 0 && c < p.nchunks)
          a.d.page_gate_out[gate_row * ((g.max_seq_len + kChunk - 1) / kChunk) + c] = vm[q] ? 1 : 0;
      }
    }
  }

  template <int Q>
  __device__ __forceinline__ void refine_chunk(const u32x4 (&B)[NKI], float (&tbp)[4]) const {
    if (bm[Q] == 0) return;  // wave-uniform
    u32x4 kb[NKI];
    plane_operand(B, kb);
    i32x4 cba = {0, 0, 0, 0}, cbb = {0, 0, 0, 0};
#pragma unroll
    for (int c = 0; c < NKI; ++c) {
      cba = mfma_i8(kb[c], qa[c], cba);
      cbb = mfma_i8(kb[c], qb[c], cbb);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float tb = static_cast<float>(cba[i]) + static_cast<float>(cbb[i]) * (1.0f / 256.0f);
      tbp[i] = dpp_movf<to_packed<Q>(), banks<Q>()>(tbp[i], tb);
    }
  }

  // The value tile of a chunk in LDS: [16 keys][VSTRIDE] BF16 rows (8-bit
  // values widened exactly by v_cvt_scalef32_pk_bf16_fp8; the second plane
  // with scale 1/16).
  template <int NL>
  __device__ __forceinline__ void stage(const u32x4 (&vv)[NL], float scale) const {
    if constexpr (V8) {
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const uint32_t off = 1024u * i + 16u * lane;  // 16 codes of key off / D
        const uint32_t key = off / D;
        uint32_t w[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          w[2 * j] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(
                                                      static_cast<int>(vv[i][j]), scale, false));
          w[2 * j + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(
                                                          static_cast<int>(vv[i][j]), scale, true));
        }
        unsigned char* dst = vt + key * VSTRIDE + 2 * (off - key * D);
        *reinterpret_cast<u32x4*>(dst) = u32x4{w[0], w[1], w[2], w[3]};
        *reinterpret_cast<u32x4*>(dst + 16) = u32x4{w[4], w[5], w[6], w[7]};
      }
    } else {
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const uint32_t off = 1024u * i + 16u * lane;
        const uint32_t key = off / (2 * D);
        *reinterpret_cast<u32x4*>(vt + key * VSTRIDE + (off - key * 2 * D)) = vv[i];
      }
    }
  }

  // acc += V^T P^T over the staged tile: one transposing LDS read per 16
  // channels (lane l receives channel 16 blk + l%16 of keys 4(l/16) .. +3).
  __device__ __forceinline__ void product(const u32x2& phi, const u32x2& plo) {
    const unsigned char* src = vt + (4 * grp + (n16 >> 2)) * VSTRIDE + 8 * (n16 & 3);
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
      const u32x2 va = __builtin_bit_cast(
          u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(src + 32 * blk)));
      acc[blk] = mfma_16x16x16(va, phi, acc[blk]);
      acc[blk] = mfma_16x16x16(va, plo, acc[blk]);
    }
  }

  template <int Q>
  __device__ __forceinline__ void product_chunk(const float (&xs)[4], const u32x4 (&V)[NKV],
                                                const u32x4 (&R)[V8 ? D / 64 : 1]) {
    if (vm[Q] == 0) return;  // wave-uniform
    // weights of chunk Q in the operand layout (lane l: keys 4(l/16)+i of row l%16)
    uint32_t hi[4];
    float res[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // the packed weights entering A (0 for a cut key or none)
      const float pw = dpp_movf<from_packed<Q>(), banks<0>()>(0.0f, xs[i]);
      hi[i] = __float_as_uint(pw) & 0xffff0000u;
      res[i] = pw - __uint_as_float(hi[i]);
    }
    const u32x2 phi = {(hi[0] >> 16) | hi[1], (hi[2] >> 16) | hi[3]};
    const u32x2 plo = {pack_bf16_rne(res[0], res[1]), pack_bf16_rne(res[2], res[3])};
    stage(V, 1.0f);
    product(phi, plo);
    if constexpr (V8) {
      if (rvm[Q]) {
        // the second plane counts only where this row's own group read it
        const uint32_t rv =
            static_cast<uint32_t>(dpp_movi<from_packed<Q>(), banks<0>()>(0, static_cast<int>(refvl)));
        const u32x2 m = {((rv & 1u) ? 0x0000FFFFu : 0u) | ((rv & 2u) ? 0xFFFF0000u : 0u),
                         ((rv & 4u) ? 0x0000FFFFu : 0u) | ((rv & 8u) ? 0xFFFF0000u : 0u)};
        stage(R, 0.0625f);
        product(u32x2{phi.x & m.x, phi.y & m.y}, u32x2{plo.x & m.x, plo.y & m.y});
      }
    }
  }

  // Refined scores, weights, L, cut mass and value products of a scored step.
  __device__ __forceinline__ void finish(int step, const u32x4 (&B)[PK][NKI],
                                         const u32x4 (&V)[PK][NKV],
                                         const u32x4 (&R)[PK][V8 ? D / 64 : 1]) {
    float x[4] = {xc[0], xc[1], xc[2], xc[3]};
    if (anyb) {  // wave-uniform: some key of the step is refined
      float tbp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      refine_chunk<0>(B[0], tbp);
      if constexpr (PK >= 2) refine_chunk<1>(B[1], tbp);
      if constexpr (PK == 4) {
        refine_chunk<2>(B[2], tbp);
        refine_chunk<3>(B[3], tbp);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if ((refl >> i) & 1u) x[i] = xc[i] + (etap * e[i]) * (tbp[i] * (1.0f / 256.0f));
    }
    const int cl = chunk_of(step, slot);
    float wv[4];  // the weights entering A (0 for a cut key): the products take them as they are
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float w = exp2_fast(x[i]);
      wv[i] = DENSE || x[i] >= a.d.neg_T ? w : 0.0f;
      lsum += w;
      if (!DENSE) lcut += x[i] >= a.d.neg_T ? 0.0f : w;
      if (DBG && a.d.x_out && ((okl >> i) & 1u))
        a.d.x_out[prow * g.max_seq_len + cl * kChunk + 4 * grp + i] = x[i];
    }
    if (anyv) {
      product_chunk<0>(wv, V[0], R[0]);
      if constexpr (PK >= 2) product_chunk<1>(wv, V[1], R[1]);
      if constexpr (PK == 4) {
        product_chunk<2>(wv, V[2], R[2]);
        product_chunk<3>(wv, V[3], R[3]);
      }
    }
  }
};

// The scan of one (kv sequence, kv head, split) workgroup.
template <int D, int PK, bool DENSE, bool DBG, bool V8>
__device__ __forceinline__ void q8_packed_scan(const Q8DecodeArgs& a) {
  using S = Q8Packed<D, PK, DENSE, DBG, V8>;
  constexpr int NKI = S::NKI;
  constexpr int NKV = S::NKV;
  constexpr int kTileBytes = kScanWaves * 16 * S::VSTRIDE;
  constexpr int kWaveFloats = S::NB * 4 * 64 + 64;  // one wave's accumulators, L and cut mass
  constexpr int kRedBytes = kScanWaves * kWaveFloats * 4;
  constexpr int kSmemBytes = kTileBytes > kRedBytes ? kTileBytes : kRedBytes;
  __shared__ __attribute__((aligned(16))) unsigned char smem[kSmemBytes];

  const ScanGeometry& g = a.d.geo;
  S sc(a);
  sc.p = scan_place(a.d);
  if (sc.p.rg > 0) return;  // one read group holds every row
  sc.lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  sc.n16 = sc.lane & 15;
  sc.grp = sc.lane >> 4;
  sc.slot = sc.n16 / S::BW;
  sc.vt = smem + wave * 16 * S::VSTRIDE;
  sc.gate_row = static_cast<size_t>(sc.p.seq) * g.hkv + sc.p.kvh;
  sc.gspan = (g.group < 16 ? g.group : 16) - 1;
  sc.pshift = q8_page_shift(g);

  {
    const RowInfo ri = row_info(g, sc.p.seq, sc.p.kvh, sc.n16, sc.p.nrows, sc.p.req0);
    sc.rok = ri.ok;
    const size_t row = static_cast<size_t>(ri.req) * g.heads + ri.head;
    sc.xrow = row;
#pragma unroll
    for (int c = 0; c < NKI; ++c) {
      sc.qa[c] = ri.ok ? *reinterpret_cast<const u32x4*>(a.qp + row * 2 * D + 64 * c + 16 * sc.grp)
                       : u32x4{0, 0, 0, 0};
      sc.qb[c] = ri.ok ? *reinterpret_cast<const u32x4*>(a.qp + row * 2 * D + D + 64 * c + 16 * sc.grp)
                       : u32x4{0, 0, 0, 0};
    }
    const RowInfo rp = row_info(g, sc.p.seq, sc.p.kvh, sc.n16 % S::BW, sc.p.nrows, sc.p.req0);
    sc.pok = rp.ok;
    sc.prow = static_cast<size_t>(rp.req) * g.heads + rp.head;
    sc.zp = rp.ok ? a.d.z[sc.prow] : 0.0f;
    sc.etap = rp.ok ? a.eta[sc.prow] : 0.0f;
    sc.ntaup = rp.ok ? -a.tau[rp.req] : 0.0f;
    sc.ntauvp = V8 && rp.ok ? -a.tau_v[rp.req] : 0.0f;
  }
  sc.lsum = 0.0f;
  sc.lcut = 0.0f;
#pragma unroll
  for (int blk = 0; blk < S::NB; ++blk) sc.acc[blk] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  sc.cstride = kScanWaves * a.d.num_splits;
  sc.c0 = kScanWaves * sc.p.split + wave;
  const int m = sc.p.nchunks > sc.c0 ? (sc.p.nchunks - sc.c0 + sc.cstride - 1) / sc.cstride : 0;
  const int steps = (m + PK - 1) / PK;

  u32x4 A0[PK][NKI], A1[PK][NKI];
  uint32_t sc0, sc1;
  Q8Loc l0[PK], l1[PK];
  if constexpr (DENSE) {
    // Step j: coarse pass (plane A of j), its plane-B (and refine-V) requests,
    // plane A of step j+2 into the freed set, refine and products of step j
    // (values of j, requested with its plane A two steps earlier), then the
    // values of step j+2 into the freed value set.
    u32x4 V0[PK][NKV], V1[PK][NKV];
    sc.issue_a(0, A0, sc0, l0);
    sc.issue_v(l0, V0);
    sc.issue_a(1, A1, sc1, l1);
    sc.issue_v(l1, V1);
    for (int j = 0; j < steps; j += 2) {
      {
        u32x4 B[PK][NKI], R[PK][V8 ? D / 64 : 1];
        sc.coarse(j, A0, sc0);
        sc.issue_bv(l0, B, V0, R);
        sc.issue_a(j + 2, A0, sc0, l0);
        sc.finish(j, B, V0, R);
        sc.issue_v(l0, V0);
      }
      if (j + 1 >= steps) break;
      {
        u32x4 B[PK][NKI], R[PK][V8 ? D / 64 : 1];
        sc.coarse(j + 1, A1, sc1);
        sc.issue_bv(l1, B, V1, R);
        sc.issue_a(j + 3, A1, sc1, l1);
        sc.finish(j + 1, B, V1, R);
        sc.issue_v(l1, V1);
      }
    }
  } else {
    sc.issue_a(0, A0, sc0, l0);
    sc.issue_a(1, A1, sc1, l1);
    // Step j: coarse pass (plane A of j), its plane-B and value requests,
    // plane A of step j+2 into the freed set, then refine and products of
    // step j.  The requests of step j precede plane A of step j+2, so waiting
    // for them leaves that load in flight.
    for (int j = 0; j < steps; j += 2) {
      {
        u32x4 B[PK][NKI], V[PK][NKV], R[PK][V8 ? D / 64 : 1];
        sc.coarse(j, A0, sc0);
        sc.issue_bv(l0, B, V, R);
        sc.issue_a(j + 2, A0, sc0, l0);
        sc.finish(j, B, V, R);
      }
      if (j + 1 >= steps) break;
      {
        u32x4 B[PK][NKI], V[PK][NKV], R[PK][V8 ? D / 64 : 1];
        sc.coarse(j + 1, A1, sc1);
        sc.issue_bv(l1, B, V, R);
        sc.issue_a(j + 3, A1, sc1, l1);
        sc.finish(j + 1, B, V, R);
      }
    }
  }

  // L and cut mass: the lanes of packed row r (n16 % BW == r, every key
  // group) hold different keys; add them.
#pragma unroll
  for (int sh = S::BW; sh < 64; sh <<= 1) {
    sc.lsum += __shfl_xor(sc.lsum, sh, 64);
    sc.lcut += __shfl_xor(sc.lcut, sh, 64);
  }

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
  const size_t slot_rows = (static_cast<size_t>(a.d.slot_offset) + sc.p.split) * g.batch * g.heads;
  const bool vec_ok = (reinterpret_cast<uintptr_t>(a.d.part_A) & 15u) == 0;
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
      if (V8) v[i] *= a.v_scale;  // 2^e: exact
    }
    float* dst = a.d.part_A + (slot_rows + static_cast<size_t>(xr)) * D + d;
    if (vec_ok) {
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
      if (threadIdx.x < 16)
        a.d.part_L[slot_rows + static_cast<size_t>(xr)] = v;
      else if (a.d.part_Lcut)
        a.d.part_Lcut[slot_rows + static_cast<size_t>(xr)] = v;
    }
  }
}

template <int D, int PK, bool DENSE, bool DBG, bool V8>
__global__ __launch_bounds__(kScanThreads) __attribute__((amdgpu_waves_per_eu(2)))
void decode_q8_packed_kernel(const Q8DecodeArgs a) {
  q8_packed_scan<D, PK, DENSE, DBG, V8>(a);
}

template <int D, int PK, bool DENSE, bool V8>
hipError_t launch_qp(const Q8DecodeArgs& a, bool dbg, unsigned blocks, hipStream_t stream) {
  if (dbg)
    hipLaunchKernelGGL((decode_q8_packed_kernel<D, PK, DENSE, true, V8>), dim3(blocks),
                       dim3(kScanThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((decode_q8_packed_kernel<D, PK, DENSE, false, V8>), dim3(blocks),
                       dim3(kScanThreads), 0, stream, a);
  return hipGetLastError();
}

template <int D, int PK>
hipError_t launch_qp_v(const Q8DecodeArgs& a, bool dbg, unsigned blocks, hipStream_t stream) {
  if (a.d.dense)
    return a.vp ? launch_qp<D, PK, true, true>(a, dbg, blocks, stream)
                : launch_qp<D, PK, true, false>(a, dbg, blocks, stream);
  return a.vp ? launch_qp<D, PK, false, true>(a, dbg, blocks, stream)
              : launch_qp<D, PK, false, false>(a, dbg, blocks, stream);
}

}  // namespace

// Two-plane scan of read groups of at most eight rows (one read group per kv
// sequence and head), at any depth.
hipError_t launch_q8_decode_packed(const Q8DecodeArgs& a, int head_dim, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.d.geo.num_seqs) * a.d.geo.hkv * a.d.num_splits;
  if (blocks == 0) return hipSuccess;
  const unsigned nb = static_cast<unsigned>(blocks);
  const bool dbg = a.d.x_out || a.d.key_gate_out || a.d.page_gate_out || a.xc_out ||
                   a.refine_gate_out || a.refine_v_gate_out;
  // two chunks per pass: four would need more than 256 registers per lane
  // (plane A of two steps in flight plus a step's plane-B and value rows)
  if (head_dim == 128) return launch_qp_v<128, 2>(a, dbg, nb, stream);
  if (head_dim == 64) return launch_qp_v<64, 2>(a, dbg, nb, stream);
  return hipErrorInvalidValue;
}

}  // namespace fold
