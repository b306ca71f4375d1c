// Request mean value rows for the cut-key value model (Section 4, "Depth as a
// dial": cut keys are modelled by the request's running mean, which needs no
// fit).
//
// value_mean_kernel: one workgroup of 16 wave64s per (kv sequence, kv head) of
// a per-request view.  Wave w adds the value rows of keys w, w + 16, ...; lane l
// owns channels [l D/64, (l + 1) D/64), so a key row is one coalesced read.  The
// waves' sums are added in wave order through LDS and divided by the length.
// Bound by HBM bandwidth over the request's values (a prompt-time call).
//
// value_mean_append_kernel: one wave64 per (token, kv head): the running
// update mu += (v - mu) / (pos + 1) for a token appended at position pos.
//
// Block model of BF16 values (Section 4, "Depth as a dial"; Algorithm 1, the
// tile's virtual row): a cut key of 64-key block t is modelled by the block's
// mean value row mu_t, and one virtual row per tile, weighted by the row's
// summed weight of the tile's cut keys c_it, adds c_it mu_t to the A of the
// split that owns the tile.
//
// block_mean_kernel: one wave64 per (kv sequence, kv head, block); D/8 lanes
// hold a key row (8 channels each, one 16-byte load), the wave's key slots are
// added with a butterfly and divided by the keys the block holds.  A prompt-
// time call, bound by HBM bandwidth over the values.
//
// block_mean_append_kernel: one wave64 per (token, kv head): the running
// update of the token's block, mu_t += (v - mu_t) / (pos mod 64 + 1).
//
// block_model_kernel: after the scan has written every row's cut mass per
// 16-key chunk, one workgroup per (kv sequence, kv head, split, RB rows) adds
// sum_t c_it mu_t over the split's tiles to the split's slot.  Thread (u, r,
// cg) takes every U-th tile of the split for row r and channels 8 cg .. +8;
// the U partial sums are added in order through LDS.  Bound by HBM bandwidth
// over the block means (D FP32 per 64 keys: 1.6% of the BF16 K+V bytes at
// D = 128) and the cut masses (4 bytes per row per 16 keys).
#include "decode_common.h"

namespace fold {
namespace {

constexpr int kMeanWaves = 16;
constexpr int kMeanThreads = 64 * kMeanWaves;

template <int D>
__global__ __launch_bounds__(kMeanThreads) void value_mean_kernel(const MeanArgs a) {
  constexpr int CPL = D / 64;  // channels per lane
  const ScanGeometry& g = a.geo;
  const int seq = blockIdx.x / g.hkv;
  const int kvh = blockIdx.x % g.hkv;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n = clamp_len(ld_uniform(g.seq_lens, seq), view_capacity(g));
  float sum[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) sum[c] = 0.0f;
  for (int j = wave; j < n; j += kMeanWaves) {
    size_t row;
    bool ok = true;
    if (g.page_size > 0) {
      const int phys = g.block_table[static_cast<size_t>(seq) * g.max_pages + j / g.page_size];
      ok = phys >= 0 && phys < g.num_pages;
      row = (static_cast<size_t>(ok ? phys : 0) * g.hkv + kvh) * g.page_size + j % g.page_size;
    } else {
      row = (static_cast<size_t>(seq) * g.hkv + kvh) * g.max_seq_len + j;
    }
    if (!ok) continue;  // uniform: the page id is outside the pool
    const uint16_t* v = g.v + row * D + CPL * lane;
#pragma unroll
    for (int c = 0; c < CPL; ++c) sum[c] += bf16_lo(v[c]);
  }
  __shared__ float red[kMeanWaves][D];
#pragma unroll
  for (int c = 0; c < CPL; ++c) red[wave][CPL * lane + c] = sum[c];
  __syncthreads();
  for (int d = threadIdx.x; d < D; d += kMeanThreads) {
    float t = 0.0f;
    for (int w = 0; w < kMeanWaves; ++w) t += red[w][d];
    a.mean[(static_cast<size_t>(seq) * g.hkv + kvh) * D + d] = n > 0 ? t / static_cast<float>(n) : 0.0f;
  }
}

template <int D>
__global__ __launch_bounds__(256) void value_mean_append_kernel(const MeanArgs a) {
  constexpr int CPL = D / 64;
  const ScanGeometry& g = a.geo;
  const long long item = static_cast<long long>(blockIdx.x) * 4 +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (item >= static_cast<long long>(a.n_tok) * g.hkv) return;  // uniform per wave
  const int tok = static_cast<int>(item / g.hkv);
  const int kvh = static_cast<int>(item % g.hkv);
  const int seq = ld_uniform(a.tok_seq, tok);
  const int pos = ld_uniform(a.tok_pos, tok);
  if (seq < 0 || seq >= g.num_seqs || pos < 0) return;
  const int lane = threadIdx.x & 63;
  const uint16_t* v = a.v_src + (static_cast<size_t>(tok) * g.hkv + kvh) * D + CPL * lane;
  float* mu = a.mean + (static_cast<size_t>(seq) * g.hkv + kvh) * D + CPL * lane;
  const float inv = 1.0f / static_cast<float>(pos + 1);
#pragma unroll
  for (int c = 0; c < CPL; ++c) mu[c] = __builtin_fmaf(bf16_lo(v[c]) - mu[c], inv, mu[c]);
}

template <int D>
__global__ __launch_bounds__(256) void block_mean_kernel(const MeanArgs a) {
  constexpr int LPK = D / 8;      // lanes per key row
  constexpr int KPI = 64 / LPK;   // keys per wave-wide load
  const ScanGeometry& g = a.geo;
  const long long item = static_cast<long long>(blockIdx.x) * 4 +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const long long per_seq = static_cast<long long>(g.hkv) * a.max_blocks;
  if (item >= per_seq * g.num_seqs) return;  // uniform per wave
  const int seq = static_cast<int>(item / per_seq);
  const int kvh = static_cast<int>((item / a.max_blocks) % g.hkv);
  const int t = static_cast<int>(item % a.max_blocks);
  const int lane = threadIdx.x & 63;
  const int part = lane % LPK;
  const int kslot = lane / LPK;
  const int n = clamp_len(ld_uniform(g.seq_lens, seq), view_capacity(g));
  const int key0 = t * kTile;
  const int count = min(kTile, n - key0);  // keys the block holds (<= 0 past the end)
  float sum[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) sum[e] = 0.0f;
#pragma unroll 4
  for (int i = 0; i < kTile / KPI; ++i) {
    const int j = key0 + KPI * i + kslot;
    if (j >= n) break;  // keys run in order: none after this one either
    size_t row;
    bool ok = true;
    if (g.page_size > 0) {
      const int phys = g.block_table[static_cast<size_t>(seq) * g.max_pages + j / g.page_size];
      ok = phys >= 0 && phys < g.num_pages;
      row = (static_cast<size_t>(ok ? phys : 0) * g.hkv + kvh) * g.page_size + j % g.page_size;
    } else {
      row = (static_cast<size_t>(seq) * g.hkv + kvh) * g.max_seq_len + j;
    }
    if (!ok) continue;  // a page id outside the pool adds nothing
    const u32x4 v = *reinterpret_cast<const u32x4*>(g.v + row * D + 8 * part);
    sum[0] += bf16_lo(v.x);
    sum[1] += bf16_hi(v.x);
    sum[2] += bf16_lo(v.y);
    sum[3] += bf16_hi(v.y);
    sum[4] += bf16_lo(v.z);
    sum[5] += bf16_hi(v.z);
    sum[6] += bf16_lo(v.w);
    sum[7] += bf16_hi(v.w);
  }
#pragma unroll
  for (int off = LPK; off < 64; off <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) sum[e] += __shfl_xor(sum[e], off, 64);
  if (kslot == 0) {
    const float inv = count > 0 ? 1.0f / static_cast<float>(count) : 0.0f;
    float* dst = a.mean + (item * D + 8 * part);
    f32x4 lo4, hi4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo4[e] = count > 0 ? sum[e] * inv : 0.0f;
      hi4[e] = count > 0 ? sum[4 + e] * inv : 0.0f;
    }
    reinterpret_cast<f32x4*>(dst)[0] = lo4;
    reinterpret_cast<f32x4*>(dst)[1] = hi4;
  }
}

template <int D>
__global__ __launch_bounds__(256) void block_mean_append_kernel(const MeanArgs a) {
  constexpr int CPL = D / 64;
  const ScanGeometry& g = a.geo;
  const long long item = static_cast<long long>(blockIdx.x) * 4 +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (item >= static_cast<long long>(a.n_tok) * g.hkv) return;  // uniform per wave
  const int tok = static_cast<int>(item / g.hkv);
  const int kvh = static_cast<int>(item % g.hkv);
  const int seq = ld_uniform(a.tok_seq, tok);
  const int pos = ld_uniform(a.tok_pos, tok);
  if (seq < 0 || seq >= g.num_seqs || pos < 0 || pos / kTile >= a.max_blocks) return;
  const int lane = threadIdx.x & 63;
  const uint16_t* v = a.v_src + (static_cast<size_t>(tok) * g.hkv + kvh) * D + CPL * lane;
  float* mu = a.mean + ((static_cast<size_t>(seq) * g.hkv + kvh) * a.max_blocks + pos / kTile) * D +
              CPL * lane;
  const float inv = 1.0f / static_cast<float>(pos % kTile + 1);
#pragma unroll
  for (int c = 0; c < CPL; ++c) mu[c] = __builtin_fmaf(bf16_lo(v[c]) - mu[c], inv, mu[c]);
}

template <int D, int RB>
__global__ __launch_bounds__(256) void block_model_kernel(const BlockModelArgs a) {
  constexpr int CG = D / 8;              // channel groups of 8
  constexpr int U = 256 / (RB * CG);     // tile slices
  static_assert(U >= 1 && U * RB * CG == 256, "thread layout");
  const ScanGeometry& g = a.geo;
  int bid = blockIdx.x;
  const int seq = bid % g.num_seqs;
  bid /= g.num_seqs;
  const int kvh = bid % g.hkv;
  bid /= g.hkv;
  const int split = bid % a.num_splits;
  const int rt = bid / a.num_splits;
  int req0 = seq, nreq = 1;
  if (g.row_indptr) {
    req0 = ld_uniform(g.row_indptr, seq);
    nreq = ld_uniform(g.row_indptr, seq + 1) - req0;
  }
  const int nrows = nreq * g.group;
  if (rt * RB >= nrows) return;  // uniform: no row in this row block
  const int n = clamp_len(ld_uniform(g.seq_lens, seq), view_capacity(g));
  const int ntiles = (n + kTile - 1) / kTile;
  const int nchunks = (n + kChunk - 1) / kChunk;
  const int cg = threadIdx.x % CG;
  const int r = (threadIdx.x / CG) % RB;
  const int u = threadIdx.x / (CG * RB);
  const RowInfo ri = row_info(g, seq, kvh, rt * RB + r, nrows, req0);
  const size_t row = static_cast<size_t>(ri.req) * g.heads + ri.head;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
  if (ri.ok) {
    const float* cut = a.chunk_cut + row * a.chunk_stride;
    const float* mu = a.block_mean + (static_cast<size_t>(seq) * g.hkv + kvh) * a.max_blocks * D + 8 * cg;
    for (int t = split + a.num_splits * u; t < ntiles; t += a.num_splits * U) {
      const int c0 = kTile / kChunk * t;
      float c = cut[c0];
#pragma unroll
      for (int q = 1; q < kTile / kChunk; ++q) c += c0 + q < nchunks ? cut[c0 + q] : 0.0f;
      const f32x4 m0 = reinterpret_cast<const f32x4*>(mu + static_cast<size_t>(t) * D)[0];
      const f32x4 m1 = reinterpret_cast<const f32x4*>(mu + static_cast<size_t>(t) * D)[1];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[e] = __builtin_fmaf(c, m0[e], acc[e]);
        acc[4 + e] = __builtin_fmaf(c, m1[e], acc[4 + e]);
      }
    }
  }
  __shared__ f32x4 red[U][RB][CG][2];
  red[u][r][cg][0] = f32x4{acc[0], acc[1], acc[2], acc[3]};
  red[u][r][cg][1] = f32x4{acc[4], acc[5], acc[6], acc[7]};
  __syncthreads();
  if (u != 0 || !ri.ok) return;
  f32x4 s0 = red[0][r][cg][0], s1 = red[0][r][cg][1];
#pragma unroll
  for (int w = 1; w < U; ++w) {
    s0 += red[w][r][cg][0];
    s1 += red[w][r][cg][1];
  }
  const size_t slot = static_cast<size_t>(a.slot_offset) + split;
  float* dst = a.part_A + ((slot * g.batch + ri.req) * g.heads + ri.head) * D + 8 * cg;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    dst[e] += s0[e];
    dst[4 + e] += s1[e];
  }
}

template <int D, int RB>
hipError_t launch_bm(const BlockModelArgs& a, unsigned blocks, hipStream_t stream) {
  hipLaunchKernelGGL((block_model_kernel<D, RB>), dim3(blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_bm_d(const BlockModelArgs& a, int rb, unsigned blocks, hipStream_t stream) {
  switch (rb) {
    case 1: return launch_bm<D, 1>(a, blocks, stream);
    case 2: return launch_bm<D, 2>(a, blocks, stream);
    case 4: return launch_bm<D, 4>(a, blocks, stream);
    case 8: return launch_bm<D, 8>(a, blocks, stream);
    case 16: return launch_bm<D, 16>(a, blocks, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int block_model_rows(int rows_per_seq) {
  int rb = 1;
  while (rb < 16 && rb < rows_per_seq) rb <<= 1;
  return rb;
}

hipError_t launch_block_mean(const MeanArgs& a, int head_dim, hipStream_t stream) {
  const long long items = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv * a.max_blocks;
  if (items == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((items + 3) / 4);
  if (head_dim == 128)
    hipLaunchKernelGGL(block_mean_kernel<128>, dim3(blocks), dim3(256), 0, stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(block_mean_kernel<64>, dim3(blocks), dim3(256), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_block_mean_append(const MeanArgs& a, int head_dim, hipStream_t stream) {
  const long long items = static_cast<long long>(a.n_tok) * a.geo.hkv;
  if (items == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((items + 3) / 4);
  if (head_dim == 128)
    hipLaunchKernelGGL(block_mean_append_kernel<128>, dim3(blocks), dim3(256), 0, stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(block_mean_append_kernel<64>, dim3(blocks), dim3(256), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_block_model(const BlockModelArgs& a, int head_dim, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv * a.num_splits *
                           a.row_tiles;
  if (blocks == 0) return hipSuccess;
  const int rb = block_model_rows(a.rows_per_seq);
  if (head_dim == 128) return launch_bm_d<128>(a, rb, static_cast<unsigned>(blocks), stream);
  if (head_dim == 64) return launch_bm_d<64>(a, rb, static_cast<unsigned>(blocks), stream);
  return hipErrorInvalidValue;
}

hipError_t launch_value_mean(const MeanArgs& a, int head_dim, hipStream_t stream) {
  const long long blocks = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv;
  if (blocks == 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(value_mean_kernel<128>, dim3(static_cast<unsigned>(blocks)),
                       dim3(kMeanThreads), 0, stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(value_mean_kernel<64>, dim3(static_cast<unsigned>(blocks)),
                       dim3(kMeanThreads), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_value_mean_append(const MeanArgs& a, int head_dim, hipStream_t stream) {
  const long long items = static_cast<long long>(a.n_tok) * a.geo.hkv;
  if (items == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((items + 3) / 4);
  if (head_dim == 128)
    hipLaunchKernelGGL(value_mean_append_kernel<128>, dim3(blocks), dim3(256), 0, stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(value_mean_append_kernel<64>, dim3(blocks), dim3(256), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace fold
