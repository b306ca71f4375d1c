// Gated split-KV decode over a two-plane INT8 key cache (Section 4, "Cache
// format", "Weight-gated reads", "Value product"; Algorithm 1 with BF16 values).
//
// Workgroup = (kv sequence, kv head, split, read group of 16*RB query rows);
// four wave64s; wave w owns 16-key chunk 4t + w of each 64-key tile t of its
// split, as in the BF16 scan.  Per chunk and 16-row block:
//
//   coarse   c_aa = A_keys . Qa^T and c_ab = A_keys . Qb^T with
//            v_mfma_i32_16x16x64_i8 (keys on M, rows on N, channels on K;
//            exact integer sums); xc = (eta_i e_j)(c_aa + c_ab/256) - Z_i in
//            FP32.  Lane l loads 16 bytes of plane A of key l%16 per product
//            and holds keys 4(l/16)+i of row l%16 afterwards.
//   gates    per GQA group (the rows of one request): live = OR [xc >= -T],
//            refine = live AND OR [xc >= -tau_r], ORed across the lanes that
//            hold the group's rows; the unions over the read group are the
//            chunk's 16-bit plane-B and value-row read masks.
//   refine   plane B of refined keys only (other keys get an offset past the
//            chunk's buffer resource, so no bytes move); c_ba, c_bb by the
//            same product; x = xc + [refine] (eta_i e_j)(c_ba + c_bb/256)/256.
//   values   value rows of live keys only; w = 2^x; a key counts for row i
//            iff x >= -T; L adds every w.  The value product is the BF16
//            scan's: channels on M, rows on N, the chunk's keys on K, the
//            weight as bf16 hi + bf16 residual.
//   8-bit    (values as two E4M3 planes under a scale 2^e for the cache)
//            the first plane is read for live keys and the second only for
//            keys whose refine-V verdict (coarse score >= -tau_v, ORed per GQA
//            group) is set; both widen exactly to BF16 (v_cvt_scalef32_pk_bf16_
//            fp8, scale 1 and 1/16) and enter two value products, the second
//            with weights kept only where the row's own group set the verdict.
//            A is multiplied by 2^e when written.
//
// Pipeline per wave: while chunk t is refined and multiplied, chunk t+1 has
// been scored and its plane-B and value rows requested, and plane A of the
// next chunks is in flight in a ring of four (at a finite depth chunks t+2 ..
// t+5; in dense decode, where every value row is requested with plane A,
// chunks t+1 .. t+3).
#include "q8_common.h"

namespace fold {
namespace {

// 16-byte value loads per lane and chunk: BF16 rows, or one E4M3 plane.
template <int D, bool V8>
constexpr int kValueLoads = V8 ? D / 64 : D / 32;

template <int D, bool DENSE, bool V8>
struct Q8AStage {
  Q8Loc loc;
  u32x4 ka[D / 64];
  uint32_t sc;                    // BF16 scale of key 4(l/16) + l%4 (2-byte loads: any row alignment)
  u32x4 vv[DENSE ? kValueLoads<D, V8> : 1];
};

// A chunk from its coarse pass to its product.
template <int D, int RB, bool DENSE, bool V8>
struct Q8BStage {
  Q8Loc loc;
  float e[4];       // BF16 scales of keys 4(l/16)+i
  u32x4 kb[D / 64];
  u32x4 vv[DENSE ? 1 : kValueLoads<D, V8>];
  u32x4 vr[V8 ? D / 64 : 1];  // second value plane (8-bit values)
  float xc[RB][4];
  uint32_t ref;     // bit 4b+i: key 4(l/16)+i refined for the group of row block b
  uint32_t refv;    // the same for the second value plane (8-bit values)
  uint32_t vmask;   // value rows to read (wave-uniform)
  uint32_t bmask;   // plane-B rows to read (wave-uniform)
  uint32_t rvmask;  // second-value-plane rows to read (wave-uniform)
};

template <int D, int RB, bool DENSE, bool DBG, bool V8>
struct Q8Scan {
  static constexpr int NKI = D / 64;          // 16-byte plane loads per lane per chunk
  static constexpr int NK = kValueLoads<D, V8>;  // 16-byte value loads per lane per chunk
  static constexpr int NB = D / 16;           // 16-channel blocks of the value product
  static constexpr int VSTRIDE = 2 * D + 16;  // bytes per key row of the LDS value tile
  static constexpr int R = 16 * RB;
  static constexpr int NA = 4;                 // plane-A ring depth (chunks)
  using AS = Q8AStage<D, DENSE, V8>;
  using BS = Q8BStage<D, RB, DENSE, V8>;

  const Q8DecodeArgs& a;
  const ScanGeometry& g;
  ScanPlace p;
  int lane, n16, grp;
  int gspan;     // lanes (within a 16-lane row) that share a GQA group, minus 1
  bool cross_b;  // the GQA group spans both 16-row blocks
  size_t gate_row;
  unsigned char* vt;

  u32x4 qa[RB][NKI], qb[RB][NKI];
  float eta[RB], zr[RB], ntau[RB], ntau_v[RB];
  bool rok[RB];
  size_t xrow[RB];
  f32x4 acc[RB][NB];
  float lsum[RB];
  float lcut[RB];  // weights of cut keys (finite depth)

  __device__ Q8Scan(const Q8DecodeArgs& a_) : a(a_), g(a_.d.geo) {}

  // Plane A and the scales (dense decode: and every value row) of a chunk.
  __device__ __forceinline__ void load_a(AS& s) const {
    const rsrc_t ra = make_rsrc(a.keys.ka + s.loc.row * D, s.loc.nk * D);
    const rsrc_t rs = make_rsrc(a.keys.ks + s.loc.row, s.loc.nk * 2);
#pragma unroll
    for (int c = 0; c < NKI; ++c) s.ka[c] = buf_load(ra, n16 * D + 64 * c + 16 * grp);
    s.sc = buf_load2(rs, 2 * (4 * grp + (lane & 3)));
    if constexpr (DENSE) load_v(s.loc, 0xFFFFu, s.vv);
  }

  // BF16 value rows, or the first E4M3 plane (8-bit values), of the chunk's
  // keys in mask.
  __device__ __forceinline__ void load_v(const Q8Loc& loc, uint32_t mask, u32x4 (&vv)[NK]) const {
    constexpr uint32_t kRowBytes = V8 ? D : 2 * D;
    const rsrc_t rv = V8 ? make_rsrc(a.vp + loc.row * D, loc.nk * D)
                         : make_rsrc(g.v + loc.row * D, loc.nk * D * 2);
    // lane l, load i: the 16 bytes at 1024 i + 16 l of the chunk (key (1024 i + 16 l) / row bytes)
#pragma unroll
    for (int i = 0; i < NK; ++i) {
      const uint32_t off = 1024u * i + 16u * lane;
      const uint32_t key = off / kRowBytes;
      vv[i] = buf_load(rv, DENSE || ((mask >> key) & 1u) ? off : kOutOfRange);
    }
  }

  // Second E4M3 value plane of the chunk's keys in mask.
  __device__ __forceinline__ void load_vr(const Q8Loc& loc, uint32_t mask, u32x4 (&vr)[D / 64]) const {
    const rsrc_t rr = make_rsrc(a.vr + loc.row * D, loc.nk * D);
#pragma unroll
    for (int i = 0; i < D / 64; ++i) {
      const uint32_t off = 1024u * i + 16u * lane;
      vr[i] = buf_load(rr, ((mask >> (off / D)) & 1u) ? off : kOutOfRange);
    }
  }

  // The gated requests of a scored chunk: plane B of refined keys (and, at a
  // finite depth, value rows of live keys).
  __device__ __forceinline__ void load_bv(BS& s) const {
    if (s.bmask) {  // wave-uniform: no request at all when no key is refined
      const rsrc_t rb = make_rsrc(a.keys.kb + s.loc.row * D, s.loc.nk * D);
      const bool want = (s.bmask >> n16) & 1u;
#pragma unroll
      for (int c = 0; c < NKI; ++c)
        s.kb[c] = buf_load(rb, want ? n16 * D + 64 * c + 16 * grp : kOutOfRange);
    }
    if constexpr (!DENSE) {
      if (s.vmask) load_v(s.loc, s.vmask, s.vv);
    }
    if constexpr (V8) {
      if (s.rvmask) load_vr(s.loc, s.rvmask, s.vr);
    }
  }

  // Scales of keys 4(l/16)+i, i < 4: lane l loaded key 4(l/16) + l%4, so key
  // 4(l/16)+i sits in lane i of the lane's own quad (DPP quad broadcast).
  __device__ __forceinline__ void scales(uint32_t sc16, float (&e)[4]) const {
    const int v = static_cast<int>(sc16);
    e[0] = bf16_lo(static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, v, 0x00, 0xF, 0xF, false)));
    e[1] = bf16_lo(static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, v, 0x55, 0xF, 0xF, false)));
    e[2] = bf16_lo(static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, v, 0xAA, 0xF, 0xF, false)));
    e[3] = bf16_lo(static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, v, 0xFF, 0xF, 0xF, false)));
  }

  // Coarse scores, group gates and read masks of chunk c (plane A in in.ka).
  __device__ __forceinline__ void coarse(int c, const AS& in, BS& s) const {
    const int key0 = c * kChunk;
    const int nk = c < p.nchunks ? min(kChunk, p.n - key0) : 0;
    s.loc = in.loc;
    float (&e)[4] = s.e;
    scales(in.sc, e);
    uint32_t lv = 0, rf = 0, rv = 0;
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      i32x4 caa = {0, 0, 0, 0}, cab = {0, 0, 0, 0};
#pragma unroll
      for (int c2 = 0; c2 < NKI; ++c2) {
        caa = mfma_i8(in.ka[c2], qa[b][c2], caa);
        cab = mfma_i8(in.ka[c2], qb[b][c2], cab);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ok = rok[b] && 4 * grp + i < nk;
        const float t = static_cast<float>(caa[i]) + static_cast<float>(cab[i]) * (1.0f / 256.0f);
        const float xc = __builtin_fmaf(eta[b] * e[i], t, -zr[b]);
        s.xc[b][i] = xc;
        if (ok && (DENSE || xc >= a.d.neg_T)) lv |= 1u << (4 * b + i);
        if (ok && xc >= ntau[b]) rf |= 1u << (4 * b + i);
        if (V8 && ok && xc >= ntau_v[b]) rv |= 1u << (4 * b + i);
        if (DBG && a.xc_out && ok) a.xc_out[xrow[b] * g.max_seq_len + key0 + 4 * grp + i] = xc;
      }
    }
    // OR over the lanes holding the rows of one GQA group: aligned groups of
    // 2, 4, 8 or 16 lanes (quad swaps, then half-row and row mirrors).
    uint32_t both = lv | (rv << 8) | (rf << 16);
    if (gspan >= 1) both |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(both), 0xB1, 0xF, 0xF, false));
    if (gspan >= 3) both |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(both), 0x4E, 0xF, 0xF, false));
    if (gspan >= 7) both |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(both), 0x141, 0xF, 0xF, false));
    if (gspan >= 15) both |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(both), 0x140, 0xF, 0xF, false));
    if (cross_b) both |= ((both >> 4) & 0x000F000Fu) | ((both & 0x000F000Fu) << 4);
    both &= ((both & 0xFFu) << 16) | ((both & 0xFFu) << 8) | 0xFFu;  // refine only live keys
    s.ref = both >> 16;
    s.refv = (both >> 8) & 0xFFu;
    // Unions over the read group: OR over each 16-lane row (row q holds keys
    // 4q..4q+3), then one row value per readlane; the row blocks fold together.
    const uint32_t u = group_or16(RB == 2 ? both | (both >> 4) : both);
    uint32_t vmask = 0, bmask = 0, rvmask = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t r = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(u), 16 * q));
      vmask |= (r & 0xFu) << (4 * q);
      rvmask |= ((r >> 8) & 0xFu) << (4 * q);
      bmask |= ((r >> 16) & 0xFu) << (4 * q);
    }
    s.vmask = vmask;
    s.bmask = bmask;
    s.rvmask = V8 ? rvmask : 0u;
    if (DBG) {
      if (a.d.key_gate_out && lane < nk)
        a.d.key_gate_out[gate_row * g.max_seq_len + key0 + lane] = (vmask >> lane) & 1u;
      if (a.refine_gate_out && lane < nk)
        a.refine_gate_out[gate_row * g.max_seq_len + key0 + lane] = (bmask >> lane) & 1u;
      if (V8 && a.refine_v_gate_out && lane < nk)
        a.refine_v_gate_out[gate_row * g.max_seq_len + key0 + lane] = (rvmask >> lane) & 1u;
      if (a.d.page_gate_out && lane == 0 && c < p.nchunks)
        a.d.page_gate_out[gate_row * ((g.max_seq_len + kChunk - 1) / kChunk) + c] = vmask ? 1 : 0;
    }
  }

  // The value tile of a chunk in LDS: [16 keys][VSTRIDE] BF16 rows.  8-bit
  // values are widened exactly by v_cvt_scalef32_pk_bf16_fp8 (2 codes per
  // instruction), the second plane with scale 1/16.
  __device__ __forceinline__ void stage(const u32x4 (&vv)[NK], float scale) const {
    if constexpr (V8) {
#pragma unroll
      for (int i = 0; i < NK; ++i) {
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
      for (int i = 0; i < NK; ++i) {
        const uint32_t off = 1024u * i + 16u * lane;
        const uint32_t key = off / (2 * D);
        *reinterpret_cast<u32x4*>(vt + key * VSTRIDE + (off - key * 2 * D)) = vv[i];
      }
    }
  }

  // acc += V^T P^T over the staged tile (hi and residual weights).  The V^T
  // operand is one transposing LDS read per 16 channels: lane 4i + a of each
  // 16-lane group points at channels 16 blk + 4a .. +4 of key 4(l/16) + i, and
  // lane l receives channel 16 blk + l%16 of those four keys.
  __device__ __forceinline__ void product(const u32x2 (&phi)[RB], const u32x2 (&plo)[RB]) {
    const unsigned char* src = vt + (4 * grp + (n16 >> 2)) * VSTRIDE + 8 * (n16 & 3);
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) {
      const u32x2 va = __builtin_bit_cast(
          u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(src + 32 * blk)));
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        acc[b][blk] = mfma_16x16x16(va, phi[b], acc[b][blk]);
        acc[b][blk] = mfma_16x16x16(va, plo[b], acc[b][blk]);
      }
    }
  }

  // Refined scores, weights, L and the value product of chunk c.
  __device__ __forceinline__ void finish(int c, const BS& s, const u32x4 (&vv)[NK]) {
    const int key0 = c * kChunk;
    const int nk = c < p.nchunks ? min(kChunk, p.n - key0) : 0;
    const float (&e)[4] = s.e;
    u32x2 phi[RB], plo[RB];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      i32x4 cba = {0, 0, 0, 0}, cbb = {0, 0, 0, 0};
      if (s.bmask) {  // wave-uniform: some key of the chunk is refined
#pragma unroll
        for (int c2 = 0; c2 < NKI; ++c2) {
          cba = mfma_i8(s.kb[c2], qa[b][c2], cba);
          cbb = mfma_i8(s.kb[c2], qb[b][c2], cbb);
        }
      }
      uint32_t hi[4];
      float res[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ok = rok[b] && 4 * grp + i < nk;
        float x = s.xc[b][i];
        if ((s.ref >> (4 * b + i)) & 1u) {
          const float tb = static_cast<float>(cba[i]) + static_cast<float>(cbb[i]) * (1.0f / 256.0f);
          x = x + (eta[b] * e[i]) * (tb * (1.0f / 256.0f));
        }
        const bool live = ok && (DENSE || x >= a.d.neg_T);
        const float w = ok ? exp2_fast(x) : 0.0f;
        lsum[b] += w;
        if (!DENSE) lcut[b] += live ? 0.0f : w;
        const float pw = live ? w : 0.0f;
        hi[i] = __float_as_uint(pw) & 0xffff0000u;
        res[i] = pw - __uint_as_float(hi[i]);
        if (DBG && a.d.x_out && ok) a.d.x_out[xrow[b] * g.max_seq_len + key0 + 4 * grp + i] = x;
      }
      phi[b] = u32x2{(hi[0] >> 16) | hi[1], (hi[2] >> 16) | hi[3]};
      plo[b] = u32x2{pack_bf16_rne(res[0], res[1]), pack_bf16_rne(res[2], res[3])};
    }
    if (s.vmask == 0) return;  // wave-uniform: no live key in the chunk
    stage(vv, 1.0f);
    product(phi, plo);
    if constexpr (V8) {
      // second plane (r / 16) of the keys some group of the read group refined;
      // the tile is wave-private and its reads above precede these writes
      if (s.rvmask) {
        // the second plane counts only where this row's own group read it:
        // keep the 16-bit weight halves of keys 4(l/16)+i with refv bit 4b+i
        u32x2 phi2[RB], plo2[RB];
#pragma unroll
        for (int b = 0; b < RB; ++b) {
          const uint32_t rv = s.refv >> (4 * b);
          const u32x2 m = {((rv & 1u) ? 0x0000FFFFu : 0u) | ((rv & 2u) ? 0xFFFF0000u : 0u),
                           ((rv & 4u) ? 0x0000FFFFu : 0u) | ((rv & 8u) ? 0xFFFF0000u : 0u)};
          phi2[b] = u32x2{phi[b].x & m.x, phi[b].y & m.y};
          plo2[b] = u32x2{plo[b].x & m.x, plo[b].y & m.y};
        }
        stage(s.vr, 0.0625f);
        product(phi2, plo2);
      }
    }
  }
};

template <int D, int RB, bool DENSE, bool DBG, bool V8>
__global__ __launch_bounds__(kScanThreads) void decode_q8_kernel(const Q8DecodeArgs a) {
  using S = Q8Scan<D, RB, DENSE, DBG, V8>;
  constexpr int NKI = S::NKI;
  constexpr int R = S::R;
  constexpr int kTileBytes = kScanWaves * 16 * S::VSTRIDE;
  constexpr int kRedBytes = (R * D + RB * 64) * 4;
  __shared__ __attribute__((aligned(16))) unsigned char smem[kTileBytes > kRedBytes ? kTileBytes : kRedBytes];

  const ScanGeometry& g = a.d.geo;
  S sc(a);
  sc.p = scan_place(a.d);
  if (sc.p.rg * R >= sc.p.nrows) return;  // uniform: this read group has no rows
  sc.lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  sc.n16 = sc.lane & 15;
  sc.grp = sc.lane >> 4;
  sc.vt = smem + wave * 16 * S::VSTRIDE;
  sc.gate_row = (static_cast<size_t>(sc.p.seq) * g.hkv + sc.p.kvh) * a.d.row_groups + sc.p.rg;
  sc.gspan = (g.group < 16 ? g.group : 16) - 1;
  sc.cross_b = RB == 2 && g.group > 16;

#pragma unroll
  for (int b = 0; b < RB; ++b) {
    const RowInfo ri = row_info(g, sc.p.seq, sc.p.kvh, sc.p.rg * R + 16 * b + sc.n16,
                                sc.p.nrows, sc.p.req0);
    sc.rok[b] = ri.ok;
    const size_t row = static_cast<size_t>(ri.req) * g.heads + ri.head;
    sc.xrow[b] = row;
    sc.zr[b] = ri.ok ? a.d.z[row] : 0.0f;
    sc.eta[b] = ri.ok ? a.eta[row] : 0.0f;
    sc.ntau[b] = ri.ok ? -a.tau[ri.req] : 0.0f;
    sc.ntau_v[b] = V8 && ri.ok ? -a.tau_v[ri.req] : 0.0f;
#pragma unroll
    for (int c = 0; c < NKI; ++c) {
      sc.qa[b][c] = ri.ok ? *reinterpret_cast<const u32x4*>(a.qp + row * 2 * D + 64 * c + 16 * sc.grp)
                          : u32x4{0, 0, 0, 0};
      sc.qb[b][c] = ri.ok ? *reinterpret_cast<const u32x4*>(a.qp + row * 2 * D + D + 64 * c + 16 * sc.grp)
                          : u32x4{0, 0, 0, 0};
    }
    sc.lsum[b] = 0.0f;
    sc.lcut[b] = 0.0f;
#pragma unroll
    for (int blk = 0; blk < S::NB; ++blk) sc.acc[b][blk] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  }

  int pshift = -1;
  if (g.page_size > 0) {
    const int cpp = g.page_size / kChunk;
    if ((cpp & (cpp - 1)) == 0) pshift = __builtin_ctz(static_cast<unsigned>(cpp));
  }
  const int cstride = kScanWaves * a.d.num_splits;
  const int c0 = kScanWaves * sc.p.split + wave;
  const int m = sc.p.nchunks > c0 ? (sc.p.nchunks - c0 + cstride - 1) / cstride : 0;

  if (m > 0) {
    // Chunk k's plane A lives in A[k % NA] from its request to its coarse pass
    // (dense: to its product); its gated requests and coarse scores in
    // B[k % 2] until its product.
    constexpr int NA = S::NA;
    typename S::AS A[NA];
    typename S::BS B[2];
    // Block-table entries of this wave's chunks c0 + k cstride, 64 local
    // chunks at a time: lane j holds local chunk pt_base + j.  One vector load
    // per window (one window covers a split of up to 64 chunks per wave), read
    // with v_readlane, instead of a scalar load and its wait per chunk.
    int pt = 0, pt_base = -64;
    auto page_window = [&](int base) {
      pt_base = base;
      const int c = c0 + (base + sc.lane) * cstride;
      pt = g.page_size > 0 && c < sc.p.nchunks
               ? g.block_table[static_cast<size_t>(sc.p.seq) * g.max_pages +
                               chunk_page_of(g, c, pshift)]
               : 0;
    };
    auto request_a = [&](typename S::AS& s, int k) {
      if (k >= pt_base + 64) page_window(k & ~63);  // uniform
      const int phys = __builtin_amdgcn_readlane(pt, k - pt_base);
      s.loc = q8_loc(g, sc.p, c0 + k * cstride, phys, pshift);
      sc.load_a(s);
    };
#pragma unroll
    for (int k = 0; k < NA; ++k)
      if (k < m) request_a(A[k], k);
    sc.coarse(c0, A[0], B[0]);
    if (!DENSE && NA < m) request_a(A[0], NA);
    sc.load_bv(B[0]);
    for (int t = 0; t < m; t += NA) {
#pragma unroll
      for (int u = 0; u < NA; ++u) {
        const int k = t + u;
        if (k >= m) break;  // uniform
        const int u1 = (u + 1) % NA;
        if (k + 1 < m) {
          sc.coarse(c0 + (k + 1) * cstride, A[u1], B[(u + 1) & 1]);
          if (!DENSE && k + 1 + NA < m) request_a(A[u1], k + 1 + NA);
          sc.load_bv(B[(u + 1) & 1]);
        }
        if constexpr (DENSE) {
          sc.finish(c0 + k * cstride, B[u & 1], A[u].vv);
          if (k + NA < m) request_a(A[u], k + NA);
        } else {
          sc.finish(c0 + k * cstride, B[u & 1], B[u & 1].vv);
        }
      }
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

  // Add the four waves in order through LDS (the value tiles are dead now).
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);  // [RB][NB][4][64]
  float* redl = red + RB * S::NB * 4 * 64;      // [RB][64]
  for (int w = 0; w < kScanWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int b = 0; b < RB; ++b) {
#pragma unroll
        for (int blk = 0; blk < S::NB; ++blk) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float* d = red + ((b * S::NB + blk) * 4 + i) * 64 + sc.lane;
            *d = (w == 0 ? 0.0f : *d) + sc.acc[b][blk][i];
          }
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
  const size_t slot_rows = (static_cast<size_t>(a.d.slot_offset) + sc.p.split) * g.batch * g.heads;
  const int wl = threadIdx.x & 63;
  const int wi = threadIdx.x >> 6;
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    if (!sc.rok[b]) continue;
    const size_t row = slot_rows + sc.xrow[b];
#pragma unroll
    for (int blk = 0; blk < S::NB; ++blk) {
      const float v = red[((b * S::NB + blk) * 4 + wi) * 64 + wl];
      a.d.part_A[row * D + 16 * blk + 4 * (wl >> 4) + wi] = V8 ? v * a.v_scale : v;  // 2^e: exact
    }
    if (wi == 0 && wl < 16) a.d.part_L[row] = redl[b * 64 + wl];
    if (a.d.part_Lcut && wi == 1 && wl < 16) a.d.part_Lcut[row] = redl[b * 64 + 16 + wl];
  }
}

template <int D, int RB, bool DENSE, bool V8>
hipError_t launch_q8_rb(const Q8DecodeArgs& a, bool dbg, unsigned blocks, hipStream_t stream) {
  if (dbg)
    hipLaunchKernelGGL((decode_q8_kernel<D, RB, DENSE, true, V8>), dim3(blocks), dim3(kScanThreads),
                       0, stream, a);
  else
    hipLaunchKernelGGL((decode_q8_kernel<D, RB, DENSE, false, V8>), dim3(blocks), dim3(kScanThreads),
                       0, stream, a);
  return hipGetLastError();
}

template <int D, int RB, bool V8>
hipError_t launch_q8_v(const Q8DecodeArgs& a, bool dbg, unsigned blocks, hipStream_t stream) {
  return a.d.dense ? launch_q8_rb<D, RB, true, V8>(a, dbg, blocks, stream)
                   : launch_q8_rb<D, RB, false, V8>(a, dbg, blocks, stream);
}

template <int D>
hipError_t launch_q8_d(const Q8DecodeArgs& a, unsigned blocks, hipStream_t stream) {
  const bool dbg = a.d.x_out || a.d.key_gate_out || a.d.page_gate_out || a.xc_out ||
                   a.refine_gate_out || a.refine_v_gate_out;
  const int rb = a.d.rows_per_group / 16;
  const bool v8 = a.vp != nullptr;
  if (rb == 1) return v8 ? launch_q8_v<D, 1, true>(a, dbg, blocks, stream)
                         : launch_q8_v<D, 1, false>(a, dbg, blocks, stream);
  if (rb == 2) return v8 ? launch_q8_v<D, 2, true>(a, dbg, blocks, stream)
                         : launch_q8_v<D, 2, false>(a, dbg, blocks, stream);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_q8_decode_packed(const Q8DecodeArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_q8_decode_valu(const Q8DecodeArgs& a, int head_dim, hipStream_t stream);

hipError_t launch_q8_decode(const Q8DecodeArgs& a, int head_dim, hipStream_t stream) {
  // one row per kv sequence and head: the VALU scan
  if (a.d.rows_per_group == 1) return launch_q8_decode_valu(a, head_dim, stream);
  // at most eight rows per kv sequence: several chunks per pass
  if (a.d.rows_per_seq <= 8) return launch_q8_decode_packed(a, head_dim, stream);
  const long long blocks = static_cast<long long>(a.d.geo.num_seqs) * a.d.geo.hkv *
                           a.d.num_splits * a.d.row_groups;
  if (blocks == 0) return hipSuccess;
  if (head_dim == 128) return launch_q8_d<128>(a, static_cast<unsigned>(blocks), stream);
  if (head_dim == 64) return launch_q8_d<64>(a, static_cast<unsigned>(blocks), stream);
  return hipErrorInvalidValue;
}

}  // namespace fold
