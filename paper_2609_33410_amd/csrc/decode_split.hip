// Gated split-KV decode scan for gfx950 (Section 4 "Weight-gated reads",
// "Value product", "Depth as a dial"; Algorithm 1).
//
// One workgroup = one (kv sequence, kv head, split, read group of GR query
// rows); four wave64s.  The split walks the 64-key tiles t == split (mod S);
// wave w of the workgroup owns the 16-key chunk 4t + w of each tile, which is
// a contiguous [16][D] bf16 slab in both cache layouts (pages hold a multiple
// of 16 keys).  Per chunk a wave:
//   1. issues the 128-bit loads of the NEXT chunk's keys (prefetch),
//   2. scores this chunk's keys against the GR rows: D/8 lanes hold one key
//      row (8 channels each, v_dot2_f32_bf16), a DPP row reduction gives every
//      lane of the key the full dot product; x = s - Z_i in FP32,
//   3. takes the verdict live = (T infinite) or (x >= -T), ORs it over the
//      rows, and issues the value loads of live keys only (lanes of cut keys
//      are masked off, so their bytes are never requested; a chunk with no
//      live key issues none),
//   4. accumulates A += [live] 2^x v and L += 2^x in FP32 registers.
// Waves never synchronise inside the loop.  At the end the lanes of a wave
// and then the four waves are reduced in a fixed order and the pair (A, L) of
// every row is written to its split's slot.
#include "fold_device.h"
#include "fold_internal.h"

namespace fold {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

// First element of the 16-key chunk `c` of (seq, head), or nullptr when the
// chunk's page id is out of range.
__device__ __forceinline__ const uint16_t* chunk_base(const uint16_t* base, const ScanGeometry& g,
                                                      int seq, int head, int c, int D) {
  if (g.page_size > 0) {
    const int key0 = c * kChunk;
    const int page = key0 / g.page_size;
    const int off = key0 - page * g.page_size;
    const int phys = g.block_table[static_cast<size_t>(seq) * g.max_pages + page];
    if (phys < 0 || phys >= g.num_pages) return nullptr;
    return base + ((static_cast<size_t>(phys) * g.hkv + head) * g.page_size + off) * D;
  }
  return base + ((static_cast<size_t>(seq) * g.hkv + head) * g.max_seq_len +
                 static_cast<size_t>(c) * kChunk) * D;
}

struct RowInfo {
  int req;
  int head;
  bool ok;
};

__device__ __forceinline__ RowInfo row_info(const ScanGeometry& g, int seq, int kvh, int rho,
                                            int nrows, int req0) {
  RowInfo ri;
  ri.ok = rho < nrows;
  const int rr = ri.ok ? rho : 0;
  ri.req = g.row_indptr ? g.row_req[req0 + rr / g.group] : seq;
  ri.head = kvh * g.group + rr % g.group;
  ri.ok = ri.ok && ri.req >= 0 && ri.req < g.batch;
  return ri;
}

template <int D, int GR>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(const DecodeArgs a) {
  constexpr int LPK = D / 8;         // lanes per key row
  constexpr int KPI = 64 / LPK;      // keys per wave-wide 128-bit load
  constexpr int NI = kChunk / KPI;   // loads per lane per 16-key chunk
  const ScanGeometry& g = a.geo;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int part = lane % LPK;
  const int kslot = lane / LPK;

  int bid = blockIdx.x;
  const int seq = bid % g.num_seqs;
  bid /= g.num_seqs;
  const int kvh = bid % g.hkv;
  bid /= g.hkv;
  const int split = bid % a.num_splits;
  const int rg = bid / a.num_splits;

  int req0 = seq, nreq = 1;
  if (g.row_indptr) {
    req0 = g.row_indptr[seq];
    nreq = g.row_indptr[seq + 1] - req0;
  }
  const int nrows = nreq * g.group;
  if (rg * GR >= nrows) return;  // uniform: this read group has no rows

  const int n = clamp_len(g.seq_lens[seq], view_capacity(g));
  const int nchunks = (n + kChunk - 1) / kChunk;

  // Query rows of the read group: 8 BF16 channels per lane, and Z_i.
  u32x4 qv[GR];
  float zr[GR];
  bool rok[GR];
#pragma unroll
  for (int r = 0; r < GR; ++r) {
    const RowInfo ri = row_info(g, seq, kvh, rg * GR + r, nrows, req0);
    rok[r] = ri.ok;
    const size_t row = static_cast<size_t>(ri.req) * g.heads + ri.head;
    qv[r] = ri.ok ? *reinterpret_cast<const u32x4*>(a.q + row * D + 8 * part) : u32x4{0, 0, 0, 0};
    zr[r] = ri.ok ? a.z[row] : 0.0f;
  }

  float acc[GR][8];
  float lsum[GR];
#pragma unroll
  for (int r = 0; r < GR; ++r) {
    lsum[r] = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[r][e] = 0.0f;
  }

  const int cstride = kWaves * a.num_splits;
  int c = kWaves * split + wave;
  const size_t gate_row = (static_cast<size_t>(seq) * g.hkv + kvh) * a.row_groups + rg;
  const int gate_pages = (g.max_seq_len + kChunk - 1) / kChunk;

  u32x4 kcur[NI];
  const uint16_t* kbase = c < nchunks ? chunk_base(g.k, g, seq, kvh, c, D) : nullptr;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int j = c * kChunk + KPI * i + kslot;
    kcur[i] = (kbase && j < n) ? *reinterpret_cast<const u32x4*>(kbase + 512 * i + 8 * lane)
                               : u32x4{0, 0, 0, 0};
  }

  for (; c < nchunks; c += cstride) {
    const bool have_k = kbase != nullptr;
    // 1. prefetch the next chunk's keys
    const int cn = c + cstride;
    const uint16_t* kbase_n = cn < nchunks ? chunk_base(g.k, g, seq, kvh, cn, D) : nullptr;
    u32x4 knext[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int j = cn * kChunk + KPI * i + kslot;
      knext[i] = (kbase_n && j < n) ? *reinterpret_cast<const u32x4*>(kbase_n + 512 * i + 8 * lane)
                                    : u32x4{0, 0, 0, 0};
    }

    // 2-3. scores, verdicts and the read mask of this chunk
    float p[NI][GR];
    bool anyl[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int j = c * kChunk + KPI * i + kslot;
      const bool kok = have_k && j < n;
      anyl[i] = false;
#pragma unroll
      for (int r = 0; r < GR; ++r) {
        const float dot = group_sum<LPK>(dot8_bf16(kcur[i], qv[r], 0.0f));
        const float x = dot * a.score_scale - zr[r];
        const bool ok = kok && rok[r];
        const bool live = ok && (a.dense || x >= a.neg_T);
        const float w = ok ? exp2_fast(x) : 0.0f;
        lsum[r] += w;
        p[i][r] = live ? w : 0.0f;
        anyl[i] = anyl[i] || live;
        if (a.x_out && ok && part == 0) {
          const RowInfo ri = row_info(g, seq, kvh, rg * GR + r, nrows, req0);
          a.x_out[(static_cast<size_t>(ri.req) * g.heads + ri.head) * g.max_seq_len + j] = x;
        }
      }
      if (a.key_gate_out && kok && part == 0)
        a.key_gate_out[gate_row * g.max_seq_len + j] = anyl[i] ? 1 : 0;
    }
    bool lane_any = false;
#pragma unroll
    for (int i = 0; i < NI; ++i) lane_any = lane_any || anyl[i];
    const bool chunk_any = __ballot(lane_any) != 0;
    if (a.page_gate_out && lane == 0 && have_k)
      a.page_gate_out[gate_row * gate_pages + c] = chunk_any ? 1 : 0;

    // 4. gated value reads and accumulation
    if (chunk_any) {
      const uint16_t* vbase = chunk_base(g.v, g, seq, kvh, c, D);
      u32x4 vv[NI];
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        vv[i] = u32x4{0, 0, 0, 0};
        if (anyl[i]) vv[i] = *reinterpret_cast<const u32x4*>(vbase + 512 * i + 8 * lane);
      }
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
#pragma unroll
    for (int i = 0; i < NI; ++i) kcur[i] = knext[i];
    kbase = kbase_n;
  }

  // Reduce over the key slots of the wave (lanes with equal `part`).
#pragma unroll
  for (int off = LPK; off < 64; off <<= 1) {
#pragma unroll
    for (int r = 0; r < GR; ++r) {
      lsum[r] += __shfl_xor(lsum[r], off, 64);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[r][e] += __shfl_xor(acc[r][e], off, 64);
    }
  }

  __shared__ float red_a[kWaves][GR][D];
  __shared__ float red_l[kWaves][GR];
  if (kslot == 0) {
#pragma unroll
    for (int r = 0; r < GR; ++r)
#pragma unroll
      for (int e = 0; e < 8; ++e) red_a[wave][r][8 * part + e] = acc[r][e];
  }
  if (lane == 0) {
#pragma unroll
    for (int r = 0; r < GR; ++r) red_l[wave][r] = lsum[r];
  }
  __syncthreads();

  const size_t slot = static_cast<size_t>(a.slot_offset) + split;
  for (int idx = threadIdx.x; idx < GR * D; idx += kThreads) {
    const int r = idx / D;
    const int d = idx - r * D;
    const RowInfo ri = row_info(g, seq, kvh, rg * GR + r, nrows, req0);
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
    }
  }
}

template <int D, int GR>
hipError_t launch_dg(const DecodeArgs& a, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv * a.num_splits *
                           a.row_groups;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL((decode_split_kernel<D, GR>), dim3(static_cast<unsigned>(blocks)),
                     dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(const DecodeArgs& a, hipStream_t stream) {
  switch (a.rows_per_group) {
    case 1: return launch_dg<D, 1>(a, stream);
    case 2: return launch_dg<D, 2>(a, stream);
    case 4: return launch_dg<D, 4>(a, stream);
    case 8: return launch_dg<D, 8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int decode_rows_per_group(int rows_per_seq) {
  if (rows_per_seq <= 1) return 1;
  if (rows_per_seq <= 2) return 2;
  if (rows_per_seq <= 4) return 4;
  return 8;
}

hipError_t launch_decode(const DecodeArgs& a, int head_dim, hipStream_t stream) {
  if (head_dim == 128) return launch_d<128>(a, stream);
  if (head_dim == 64) return launch_d<64>(a, stream);
  return hipErrorInvalidValue;
}

}  // namespace fold
