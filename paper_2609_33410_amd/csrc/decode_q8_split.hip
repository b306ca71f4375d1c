// Split-KV decode over a two-plane INT8 key cache for one query row per kv
// sequence and head (MHA), on VALU (Section 4, "Cache format", "Weight-gated
// reads", "Depth as a dial"; Algorithm 1 with BF16 or 8-bit values).
//
// The arithmetic is the two-plane scans' (decode_q8.hip): coarse scores from
// plane A and the key scales, the live / refine-K / refine-V verdicts on them,
// plane B only for refined keys, value rows only for live keys, the weight
// 2^x with every key's weight in L.  With one row the read group is the row,
// so the verdicts are also the read bits.  The layout is the BF16 MHA scan's
// (decode_split.hip): no matrix core would have more than one of its sixteen
// columns busy.
//
// Workgroup = (kv sequence, kv head, split), W wave64s sharing the split's
// 64-key tiles (wave w owns chunk w mod 4 of tiles k == w / 4 (mod W / 4);
// W = 4 is launched);
// for a per-request view of at most 64 sequences the longest are dispatched
// first.  LPK = D/16 lanes hold one key, lane part p owning channels
// 16p .. 16p+15 of the key planes and of the E4M3 value planes (16 bytes per
// lane) and, with BF16 values, channels 8p .. 8p+7 and D/2 + 8p .. +7 (one
// 16-byte load per half row, so that the key's lanes read contiguous bytes);
// one wave-wide load covers KPI = 64/LPK keys.  Sixteen channels per lane
// keep the lane-sum chains short: the scan is bound by instruction issue
// more than by bytes.
//
//   coarse   the lane's c_aa = a . qa and c_ab = a . qb by v_dot4_i32_i8,
//            its 256 c_aa + c_ab added over the key's LPK lanes in int32
//            (exact: below 2^30 in magnitude) and rounded to FP32 once, so
//            the coarse logit c_aa + c_ab/256 is the FP32 sum of the two
//            exact integer totals; xc = (eta e)(c_aa + c_ab/256) - Z in FP32.
//   refine   plane B of refined keys only (the others get an offset past the
//            chunk's buffer resource: no bytes move), c_ba and c_bb the same
//            way, x = xc + [refine] (eta e)((c_ba + c_bb/256)/256).
//   values   w = 2^x; a key counts iff x >= -T; L adds every w; A += w v in
//            FP32.  8-bit values are widened exactly to FP32
//            (v_cvt_scalef32_pk_f32_fp8), the second plane with scale 1/16,
//            and A, a sum over p + [refine-V] r/16, is multiplied by 2^e when
//            written.
//
// Pipeline per wave: plane A and the scales of chunk t+2 are requested while
// chunk t+1 is scored and its plane-B and value rows requested, and chunk t
// is refined and accumulated.  At T = inf every value row is requested once
// its chunk is scored (plane B still waits for the refine verdict).
#include "q8_common.h"

namespace fold {
namespace {

typedef float f32x2 __attribute__((ext_vector_type(2)));

// Signed INT8 dot product of two 16-byte groups, added to acc.
__device__ __forceinline__ int sdot16(u32x4 a, u32x4 b, int acc) {
  acc = __builtin_amdgcn_sdot4(static_cast<int>(a.x), static_cast<int>(b.x), acc, false);
  acc = __builtin_amdgcn_sdot4(static_cast<int>(a.y), static_cast<int>(b.y), acc, false);
  acc = __builtin_amdgcn_sdot4(static_cast<int>(a.z), static_cast<int>(b.z), acc, false);
  return __builtin_amdgcn_sdot4(static_cast<int>(a.w), static_cast<int>(b.w), acc, false);
}

// c_xa + c_xb / 256 for one key, from the lane's 16 channels of a plane and
// of the two query code vectors: 256 c_xa + c_xb is summed over the key's
// LANES lanes in int32 (|c_xa|, |c_xb| <= D * 128 * 128 <= 2^21, so the total
// stays below 2^30) and rounded to FP32 once.  Scaling by 256 is exact, so
// this is the FP32 sum of the exact totals c_xa and c_xb / 256.
template <int LANES>
__device__ __forceinline__ float coarse_logit(u32x4 k, u32x4 qa, u32x4 qb) {
  static_assert(LANES == 4 || LANES == 8, "a key on 4 or 8 lanes");
  int v = sdot16(k, qb, sdot16(k, qa, 0) * 256);
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
  if constexpr (LANES == 8) v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  return static_cast<float>(v) * (1.0f / 256.0f);
}

template <int D>
struct Q8VPlaneA {  // a chunk whose plane A and scales are requested
  static constexpr int NI = kChunk / (64 / (D / 16));
  Q8Loc loc;
  u32x4 ka[NI];        // plane A, the lane's 16 channels of key KPI i + kslot
  uint32_t sc[NI];     // its BF16 scale (low half)
};

template <int D, bool V8>
struct Q8VScored {  // a scored chunk whose plane-B and value rows are requested
  static constexpr int NI = kChunk / (64 / (D / 16));
  float xc[NI];        // coarse score
  float es[NI];        // the key's scale
  uint32_t bits;       // bit i: live, 8 + i: refine, 16 + i: refine-V, 24 + i: key exists
  bool anyref;         // some key of the chunk is refined (wave-uniform)
  bool anylive;        // some key of the chunk is live (wave-uniform)
  bool anyrv;          // some key of the chunk is refine-V (wave-uniform)
  u32x4 kb[NI];        // plane B of refined keys
  u32x4 vv[V8 ? 1 : NI][2];  // BF16 values of live keys (channels 8p .. +7, D/2 + 8p .. +7)
  u32x4 vp[V8 ? NI : 1];     // first E4M3 plane of live keys
  u32x4 vr[V8 ? NI : 1];     // second E4M3 plane of refine-V keys
};

template <int D, bool DENSE, bool DBG, bool V8>
struct Q8Valu {
  static constexpr int LPK = D / 16;       // lanes per key row
  static constexpr int KPI = 64 / LPK;     // keys per wave-wide load
  static constexpr int NI = kChunk / KPI;  // loads per lane per 16-key chunk
  using PA = Q8VPlaneA<D>;
  using SC = Q8VScored<D, V8>;

  const Q8DecodeArgs& a;
  const ScanGeometry& g;
  ScanPlace p;
  int lane, part, kslot, pshift;
  size_t gate_row;
  int gate_pages;
  u32x4 qa, qb;  // query codes of the lane's channels
  float eta, zr, ntau, ntau_v;
  bool rok;
  size_t xrow;
  // A over the lane's channels: 16p + e (8-bit values) or, with BF16 values,
  // 8p + e and D/2 + 8p + e (e < 8) for acc[e] and acc[8 + e]
  float acc[16];
  float lsum, lcut;

  __device__ Q8Valu(const Q8DecodeArgs& a_) : a(a_), g(a_.d.geo) {}

  // Plane A and the scales of chunk c.
  __device__ __forceinline__ void load_a(int c, PA& s) const {
    s.loc = q8_loc(g, p, c, q8_chunk_phys(g, p, c, pshift), pshift);
    const rsrc_t ra = make_rsrc(a.keys.ka + s.loc.row * D, s.loc.nk * D);
    const rsrc_t rs = make_rsrc(a.keys.ks + s.loc.row, s.loc.nk * 2);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const uint32_t key = KPI * i + kslot;
      s.ka[i] = buf_load(ra, key * D + 16 * part);
      s.sc[i] = buf_load2(rs, 2 * key);
    }
  }

  // Coarse scores and verdicts of chunk c (plane A in in), then the requests
  // its verdicts allow: plane B of refined keys, value rows of live keys.
  __device__ __forceinline__ void coarse(int c, const PA& in, SC& s) const {
    const int key0 = c * kChunk;
    const int nk = c < p.nchunks ? min(kChunk, p.n - key0) : 0;
    uint32_t bits = 0;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int kk = KPI * i + kslot;
      const bool ok = rok && kk < nk;
      const float t = coarse_logit<LPK>(in.ka[i], qa, qb);
      const float e = bf16_lo(in.sc[i]);
      s.es[i] = e;
      const float xc = __builtin_fmaf(eta * e, t, -zr);
      s.xc[i] = xc;
      const bool live = ok && (DENSE || xc >= a.d.neg_T);
      const bool ref = live && xc >= ntau;
      const bool rv = V8 && live && xc >= ntau_v;
      bits |= (live ? 1u : 0u) << i;
      bits |= (ref ? 1u : 0u) << (8 + i);
      bits |= (rv ? 1u : 0u) << (16 + i);
      bits |= (ok ? 1u : 0u) << (24 + i);
      if (DBG && ok && part == 0) {
        const size_t j = static_cast<size_t>(key0) + kk;
        if (a.xc_out) a.xc_out[xrow * g.max_seq_len + j] = xc;
        if (a.d.key_gate_out) a.d.key_gate_out[gate_row * g.max_seq_len + j] = live ? 1 : 0;
        if (a.refine_gate_out) a.refine_gate_out[gate_row * g.max_seq_len + j] = ref ? 1 : 0;
        if (V8 && a.refine_v_gate_out)
          a.refine_v_gate_out[gate_row * g.max_seq_len + j] = rv ? 1 : 0;
      }
    }
    s.bits = bits;
    s.anylive = __ballot((bits & 0xFFu) != 0) != 0;
    s.anyref = __ballot((bits & 0xFF00u) != 0) != 0;
    s.anyrv = V8 && __ballot((bits & 0xFF0000u) != 0) != 0;
    if (DBG && a.d.page_gate_out && lane == 0 && c < p.nchunks)
      a.d.page_gate_out[gate_row * gate_pages + c] = s.anylive ? 1 : 0;
    if (s.anyref) {  // wave-uniform: no request at all when no key is refined
      const rsrc_t rb = make_rsrc(a.keys.kb + in.loc.row * D, in.loc.nk * D);
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const uint32_t key = KPI * i + kslot;
        s.kb[i] = buf_load(rb, (bits >> (8 + i)) & 1u ? key * D + 16 * part : kOutOfRange);
      }
    }
    if (s.anylive) {
      if constexpr (V8) {
        const rsrc_t rp = make_rsrc(a.vp + in.loc.row * D, in.loc.nk * D);
#pragma unroll
        for (int i = 0; i < NI; ++i) {
          const uint32_t key = KPI * i + kslot;
          s.vp[i] = buf_load(rp, (bits >> i) & 1u ? key * D + 16 * part : kOutOfRange);
        }
        if (s.anyrv) {
          const rsrc_t rr = make_rsrc(a.vr + in.loc.row * D, in.loc.nk * D);
#pragma unroll
          for (int i = 0; i < NI; ++i) {
            const uint32_t key = KPI * i + kslot;
            s.vr[i] = buf_load(rr, (bits >> (16 + i)) & 1u ? key * D + 16 * part : kOutOfRange);
          }
        }
      } else {
        const rsrc_t rv = make_rsrc(g.v + in.loc.row * D, in.loc.nk * D * 2);
#pragma unroll
        for (int i = 0; i < NI; ++i) {
          const uint32_t key = KPI * i + kslot;
          // each load reads one half of the row, 16 bytes per lane, so
          // the key's lanes cover 8 * 16 contiguous bytes per instruction
          const uint32_t off = (bits >> i) & 1u ? key * 2 * D + 16 * part : kOutOfRange;
          s.vv[i][0] = buf_load(rv, off);
          s.vv[i][1] = buf_load(rv, off + static_cast<uint32_t>(D));
        }
      }
    }
  }

  // Refined scores, weights, L and the accumulation of chunk c.
  __device__ __forceinline__ void finish(int c, const SC& s) {
    const int key0 = c * kChunk;
    float pw[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      float x = s.xc[i];
      if (s.anyref) {
        const float tb = coarse_logit<LPK>(s.kb[i], qa, qb);
        if ((s.bits >> (8 + i)) & 1u) x = x + (eta * s.es[i]) * (tb * (1.0f / 256.0f));
      }
      const bool ok = (s.bits >> (24 + i)) & 1u;
      const bool counts = ok && (DENSE || x >= a.d.neg_T);
      const float w = ok ? exp2_fast(x) : 0.0f;
      lsum += w;
      if (!DENSE) lcut += counts ? 0.0f : w;
      pw[i] = counts ? w : 0.0f;
      if (DBG && a.d.x_out && ok && part == 0)
        a.d.x_out[xrow * g.max_seq_len + static_cast<size_t>(key0) + KPI * i + kslot] = x;
    }
    if (!s.anylive) return;  // wave-uniform: no value row was read
    if constexpr (V8) {
      accumulate_v8(s, pw);
    } else {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const u32x4 w = s.vv[i][h];
          float v[8];
          v[0] = bf16_lo(w.x), v[1] = bf16_hi(w.x);
          v[2] = bf16_lo(w.y), v[3] = bf16_hi(w.y);
          v[4] = bf16_lo(w.z), v[5] = bf16_hi(w.z);
          v[6] = bf16_lo(w.w), v[7] = bf16_hi(w.w);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[8 * h + e] += pw[i] * v[e];
        }
      }
    }
  }

  // A += w (p + [refine-V] r / 16) over the chunk's live keys.  The second
  // plane is widened only in chunks with a refine-V key; there a key without
  // the bit read its plane-R bytes at an offset past the buffer, so its r is
  // +0 and adding it changes nothing.
  __device__ __forceinline__ void accumulate_v8(const SC& s, const float (&pw)[NI]) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const int wp = static_cast<int>(s.vp[i][h]);
        const f32x2 p0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(wp, 1.0f, false);
        const f32x2 p1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(wp, 1.0f, true);
        float v[4] = {p0.x, p0.y, p1.x, p1.y};
        if (s.anyrv) {  // wave-uniform
          const int wr = static_cast<int>(s.vr[i][h]);
          const f32x2 r0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(wr, 0.0625f, false);
          const f32x2 r1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(wr, 0.0625f, true);
          v[0] += r0.x, v[1] += r0.y, v[2] += r1.x, v[3] += r1.y;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[4 * h + e] += pw[i] * v[e];
      }
    }
  }
};

// Occupancy: the two chunk stages fit in 128 registers (about 120 at D = 128),
// four waves per SIMD at every depth; with two waves per SIMD the key-plane
// stream lacked memory-level parallelism (517 against 420 us at T = 16 on the
// MHA 4 x 64K-128K decode, eight channels per lane).
template <int D, bool DENSE, bool DBG, bool V8, int W>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(DBG ? 2 : (DENSE ? 3 : 4))))
void decode_q8_split_kernel(const Q8DecodeArgs a) {
  using S = Q8Valu<D, DENSE, DBG, V8>;
  const ScanGeometry& g = a.d.geo;
  S sc(a);
  sc.lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  sc.part = sc.lane % S::LPK;
  sc.kslot = sc.lane / S::LPK;
  __shared__ int order[kOrderMax];
  sc.p = a.d.by_length ? scan_place_by_length(a.d, order) : scan_place(a.d);
  if (sc.p.rg >= sc.p.nrows) return;  // uniform: no row
  sc.pshift = q8_page_shift(g);
  sc.gate_row = (static_cast<size_t>(sc.p.seq) * g.hkv + sc.p.kvh) * a.d.row_groups + sc.p.rg;
  sc.gate_pages = (g.max_seq_len + kChunk - 1) / kChunk;
  {
    const RowInfo ri = row_info(g, sc.p.seq, sc.p.kvh, sc.p.rg, sc.p.nrows, sc.p.req0);
    sc.rok = ri.ok;
    const size_t row = static_cast<size_t>(ri.req) * g.heads + ri.head;
    sc.xrow = row;
    const int8_t* qp = a.qp + (ri.ok ? row : 0) * 2 * D + 16 * sc.part;
    sc.qa = *reinterpret_cast<const u32x4*>(qp);
    sc.qb = *reinterpret_cast<const u32x4*>(qp + D);
    // one row per workgroup: its scalars are wave-uniform
    auto uni = [](float v) {
      return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
    };
    sc.eta = uni(ri.ok ? a.eta[row] : 0.0f);
    sc.zr = uni(ri.ok ? a.d.z[row] : 0.0f);
    sc.ntau = uni(ri.ok ? -a.tau[ri.req] : 0.0f);
    sc.ntau_v = uni((V8 && ri.ok) ? -a.tau_v[ri.req] : 0.0f);
  }
  sc.lsum = 0.0f;
  sc.lcut = 0.0f;
#pragma unroll
  for (int e = 0; e < 16; ++e) sc.acc[e] = 0.0f;

  // chunks of this wave: c_t = c0 + t * cstride, t < m
  const int cstride = W * a.d.num_splits;
  const int c0 = 4 * sc.p.split + 4 * a.d.num_splits * (wave >> 2) + (wave & 3);
  const int m = sc.p.nchunks > c0 ? (sc.p.nchunks - c0 + cstride - 1) / cstride : 0;
  if (m > 0) {
    // A0 / A1: plane A of chunks t and t+1 (parity of t); S0 / S1: scored chunks
    typename S::PA A0, A1;
    typename S::SC S0, S1;
    sc.load_a(c0, A0);
    sc.load_a(c0 + cstride, A1);
    sc.coarse(c0, A0, S0);
    for (int t = 0; t < m; t += 2) {
      // S0: chunk t scored (plane B / values in flight); A1: plane A of t+1
      sc.load_a(c0 + (t + 2) * cstride, A0);
      sc.coarse(c0 + (t + 1) * cstride, A1, S1);
      sc.finish(c0 + t * cstride, S0);
      if (t + 1 >= m) break;
      // S1: chunk t+1 scored; A0: plane A of t+2
      sc.load_a(c0 + (t + 3) * cstride, A1);
      sc.coarse(c0 + (t + 2) * cstride, A0, S0);
      sc.finish(c0 + (t + 1) * cstride, S1);
    }
  }

  // Reduce over the key slots of the wave (lanes with equal `part`).
#pragma unroll
  for (int off = S::LPK; off < 64; off <<= 1) {
    sc.lsum += __shfl_xor(sc.lsum, off, 64);
    if (!DENSE) sc.lcut += __shfl_xor(sc.lcut, off, 64);
#pragma unroll
    for (int e = 0; e < 16; ++e) sc.acc[e] += __shfl_xor(sc.acc[e], off, 64);
  }
  __shared__ float red_a[W][D];
  __shared__ float red_l[W];
  __shared__ float red_c[W];
  if (sc.kslot == 0) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int ch = V8 ? 16 * sc.part + e : (e < 8 ? 8 * sc.part + e : D / 2 + 8 * sc.part + e - 8);
      red_a[wave][ch] = sc.acc[e];
    }
  }
  if (sc.lane == 0) {
    red_l[wave] = sc.lsum;
    red_c[wave] = sc.lcut;
  }
  __syncthreads();
  if (!sc.rok) return;
  const size_t slot = static_cast<size_t>(a.d.slot_offset) + sc.p.split;
  const size_t prow = slot * g.batch * g.heads + sc.xrow;
  for (int d = threadIdx.x; d < D; d += 64 * W) {
    float s = red_a[0][d];
#pragma unroll
    for (int w = 1; w < W; ++w) s += red_a[w][d];
    if (V8) s *= a.v_scale;  // 2^e: exact
    a.d.part_A[prow * D + d] = s;
    if (d == 0) {
      float l = red_l[0];
#pragma unroll
      for (int w = 1; w < W; ++w) l += red_l[w];
      a.d.part_L[prow] = l;
      if (a.d.part_Lcut) {
        float cm = red_c[0];
#pragma unroll
        for (int w = 1; w < W; ++w) cm += red_c[w];
        a.d.part_Lcut[prow] = cm;
      }
    }
  }
}

template <int D, bool DENSE, bool V8>
hipError_t launch_qs_dbg(const Q8DecodeArgs& a, bool dbg, unsigned blocks, hipStream_t stream) {
  // four waves per workgroup: a compute unit then holds four workgroups
  // (eight-wave workgroups at 135 registers left it one or two: 517 against
  // 417 us at T = 16 on the MHA 4 x 64K-128K decode)
  if (dbg)
    hipLaunchKernelGGL((decode_q8_split_kernel<D, DENSE, true, V8, 4>), dim3(blocks), dim3(256),
                       0, stream, a);
  else
    hipLaunchKernelGGL((decode_q8_split_kernel<D, DENSE, false, V8, 4>), dim3(blocks), dim3(256),
                       0, stream, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_qs(const Q8DecodeArgs& a, unsigned blocks, hipStream_t stream) {
  const bool dbg = a.d.x_out || a.d.key_gate_out || a.d.page_gate_out || a.xc_out ||
                   a.refine_gate_out || a.refine_v_gate_out;
  if (a.d.dense)
    return a.vp ? launch_qs_dbg<D, true, true>(a, dbg, blocks, stream)
                : launch_qs_dbg<D, true, false>(a, dbg, blocks, stream);
  return a.vp ? launch_qs_dbg<D, false, true>(a, dbg, blocks, stream)
              : launch_qs_dbg<D, false, false>(a, dbg, blocks, stream);
}

}  // namespace

// Two-plane scan of one row per kv sequence and head (read groups of one row).
hipError_t launch_q8_decode_valu(const Q8DecodeArgs& a, int head_dim, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.d.geo.num_seqs) * a.d.geo.hkv *
                           a.d.num_splits * a.d.row_groups;
  if (blocks == 0) return hipSuccess;
  if (head_dim == 128) return launch_qs<128>(a, static_cast<unsigned>(blocks), stream);
  if (head_dim == 64) return launch_qs<64>(a, static_cast<unsigned>(blocks), stream);
  return hipErrorInvalidValue;
}

}  // namespace fold
