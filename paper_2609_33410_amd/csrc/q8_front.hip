// Front of a two-plane INT8 key cache (Section 4, "Cache format"): the key
// writer, the per-step query split and the writer of 8-bit values; and the
// stacked level's FP16 keys (Appendix E, tile layouts: a level past 64
// stacked rows runs laid out as prefill is, with one FP16 product per logit
// of each key's code rounded once per prefix): q8_stack_kernel writes
// fp16(e (a + b/256)) per element, the product being exact in FP32 (a 16-bit
// code times an 8-bit scale) and rounded once, to nearest even.
//
// Both rotate a D-vector by the Sylvester Hadamard matrix H_D (entries +-1;
// the paper's orthonormal rotation is H_D / sqrt(D), and its 1/D on a dot
// product is folded into the query scale) and split the result into two INT8
// planes under one scale:
//   key   k'' = e (a + b/256), e = the smallest BF16 value >= max|k''| / 127
//         (rounded up: plane A never saturates); a key whose scale would fall
//         below 2^-126 is stored as zero;
//   query q'' = f (qa + qb/256), f = max|q''| / 127, with the base-2 score
//         scale eta = log2(e) sm_scale f / D rounded once to FP32;
//   a = rint(x / s), b = rint(256 (x / s - a)) clamped to [-128, 127].
// One wave64 handles one vector; lane l holds elements 64 i + l.  The
// transform is a radix-2 butterfly in FP64: every partial sum of +-BF16
// inputs is exact while the inputs of one vector span at most 38 binades, so
// the codes do not depend on the order of the butterflies.  Division, rint and
// the rounded-up scale are exact IEEE FP64 operations.
#include "fold_internal.h"
#include "q8_split.h"

namespace fold {
namespace {

constexpr int kFrontThreads = 256;
constexpr int kWavesPerBlock = kFrontThreads / 64;

// Smallest value with 8 significant bits (a BF16 significand) >= t, t > 0 normal.
__device__ __forceinline__ double ceil_to_bf16(double t) {
  constexpr unsigned long long kLow = (1ull << 45) - 1;
  const unsigned long long u = static_cast<unsigned long long>(__double_as_longlong(t));
  return __longlong_as_double(static_cast<long long>((u + kLow) & ~kLow));
}

template <int D>
__global__ __launch_bounds__(kFrontThreads) void q8_write_kernel(const Q8WriteArgs a) {
  const ScanGeometry& g = a.geo;
  const int lane = threadIdx.x & 63;
  const long long item = static_cast<long long>(blockIdx.x) * kWavesPerBlock +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (item >= static_cast<long long>(a.n_tok) * g.hkv) return;  // uniform per wave
  const int tok = static_cast<int>(item / g.hkv);
  const int kvh = static_cast<int>(item % g.hkv);
  const int seq = ld_uniform(a.tok_seq, tok);
  const int pos = ld_uniform(a.tok_pos, tok);
  if (seq < 0 || seq >= g.num_seqs || pos < 0 || pos >= view_capacity(g)) return;
  size_t row;
  if (g.page_size > 0) {
    const int phys = ld_uniform(a.geo.block_table,
                                static_cast<size_t>(seq) * g.max_pages + pos / g.page_size);
    if (phys < 0 || phys >= g.num_pages) return;
    row = (static_cast<size_t>(phys) * g.hkv + kvh) * g.page_size + pos % g.page_size;
  } else {
    row = (static_cast<size_t>(seq) * g.hkv + kvh) * g.max_seq_len + pos;
  }
  const uint16_t* src = a.k_src + (static_cast<size_t>(tok) * g.hkv + kvh) * D;
  double x[D / 64];
#pragma unroll
  for (int i = 0; i < D / 64; ++i) x[i] = static_cast<double>(bf16_lo(src[64 * i + lane]));
  hadamard_wave<D>(x, lane);
  const double m = wave_absmax_f64<D>(x);
  const double e = m >= 127.0 * 0x1p-126 ? ceil_to_bf16(m / 127.0) : 0.0;
#pragma unroll
  for (int i = 0; i < D / 64; ++i) {
    int8_t qa, qb;
    split_value(x[i], e, &qa, &qb);
    a.ka[row * D + 64 * i + lane] = qa;
    a.kb[row * D + 64 * i + lane] = qb;
  }
  if (lane == 0) a.ks[row] = static_cast<uint16_t>(__float_as_uint(static_cast<float>(e)) >> 16);
}

template <int D>
__global__ __launch_bounds__(kFrontThreads) void q8_split_kernel(const Q8SplitArgs a) {
  const int lane = threadIdx.x & 63;
  if (blockIdx.x == 0 && a.tau) {
    for (int r = threadIdx.x; r < a.batch; r += kFrontThreads) {
      const int n = a.req_lens[r];
      const int c = n > 1 ? 32 - __builtin_clz(static_cast<unsigned>(n - 1)) : 0;
      a.tau[r] = a.kappa + static_cast<float>(c);
      if (a.tau_v) a.tau_v[r] = a.kappa_v + static_cast<float>(c);
    }
  }
  const long long row = static_cast<long long>(blockIdx.x) * kWavesPerBlock +
                        __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (row >= a.rows) return;  // uniform per wave
  const uint16_t* src = a.q + row * D;
  double x[D / 64];
#pragma unroll
  for (int i = 0; i < D / 64; ++i) x[i] = static_cast<double>(bf16_lo(src[64 * i + lane]));
  hadamard_wave<D>(x, lane);
  const double f = wave_absmax_f64<D>(x) / 127.0;
  int8_t* dst = a.qp + row * 2 * D;
#pragma unroll
  for (int i = 0; i < D / 64; ++i) {
    int8_t qa, qb;
    split_value(x[i], f, &qa, &qb);
    dst[64 * i + lane] = qa;
    dst[D + 64 * i + lane] = qb;
  }
  if (lane == 0)
    a.eta[row] = static_cast<float>(((kLog2eF64 * static_cast<double>(a.sm_scale)) * f) / D);
}

// E4M3 (OCP E4M3FN: bias 7, subnormals m 2^-9, largest finite 448) code of
// y rounded to nearest even; magnitudes of 448 and above saturate to 448.  The
// mantissa is rounded with rintf on an exactly scaled copy, so the tie goes
// to the even code.  *val receives the code's value.
__device__ __forceinline__ uint32_t e4m3_rne_sat(float y, float* val) {
  const uint32_t sign = (__float_as_uint(y) >> 24) & 0x80u;
  const float a = fabsf(y);
  const float sg = sign ? -1.0f : 1.0f;
  if (!(a < 448.0f)) {
    *val = sg * 448.0f;
    return sign | 0x7Eu;
  }
  if (a < 0x1p-6f) {  // subnormal steps of 2^-9; 8 steps is the code of 2^-6
    const float q = rintf(a * 512.0f);
    *val = sg * q * 0x1p-9f;
    return q == 0.0f ? 0u : sign | static_cast<uint32_t>(q);
  }
  int e = ilogbf(a);
  float q = rintf(ldexpf(a, 3 - e));  // in [8, 16]
  if (q == 16.0f) {
    q = 8.0f;
    e += 1;
  }
  *val = sg * ldexpf(q, e - 3);
  return sign | static_cast<uint32_t>((e + 7) << 3) | static_cast<uint32_t>(q - 8.0f);
}

template <int D>
__global__ __launch_bounds__(kFrontThreads) void v8_write_kernel(const V8WriteArgs a) {
  const ScanGeometry& g = a.geo;
  const int lane = threadIdx.x & 63;
  const long long item = static_cast<long long>(blockIdx.x) * kWavesPerBlock +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (item >= static_cast<long long>(a.n_tok) * g.hkv) return;  // uniform per wave
  const int tok = static_cast<int>(item / g.hkv);
  const int kvh = static_cast<int>(item % g.hkv);
  const int seq = ld_uniform(a.tok_seq, tok);
  const int pos = ld_uniform(a.tok_pos, tok);
  if (seq < 0 || seq >= g.num_seqs || pos < 0 || pos >= view_capacity(g)) return;
  size_t row;
  if (g.page_size > 0) {
    const int phys = ld_uniform(a.geo.block_table,
                                static_cast<size_t>(seq) * g.max_pages + pos / g.page_size);
    if (phys < 0 || phys >= g.num_pages) return;
    row = (static_cast<size_t>(phys) * g.hkv + kvh) * g.page_size + pos % g.page_size;
  } else {
    row = (static_cast<size_t>(seq) * g.hkv + kvh) * g.max_seq_len + pos;
  }
  const uint16_t* src = a.v_src + (static_cast<size_t>(tok) * g.hkv + kvh) * D;
#pragma unroll
  for (int i = 0; i < D / 64; ++i) {
    const float y = ldexpf(bf16_lo(src[64 * i + lane]), -a.scale_exp);  // exact
    float pv, rv;
    const uint32_t p = e4m3_rne_sat(y, &pv);
    const uint32_t r = e4m3_rne_sat(16.0f * (y - pv), &rv);  // y - pv and the x16 are exact
    a.vp[row * D + 64 * i + lane] = static_cast<uint8_t>(p);
    a.vr[row * D + 64 * i + lane] = static_cast<uint8_t>(r);
  }
}

// One thread per 8 elements of a key: D/8 threads per key, 256/(D/8) keys per
// workgroup.  Grid: (kv sequence, kv head, key block).
template <int D>
__global__ __launch_bounds__(kFrontThreads) void q8_stack_kernel(const Q8StackArgs a, int blocks_per_seq) {
  constexpr int TPK = D / 8;
  constexpr int KPB = kFrontThreads / TPK;
  const ScanGeometry& g = a.geo;
  int bid = blockIdx.x;
  const int kb = bid % blocks_per_seq;
  bid /= blocks_per_seq;
  const int kvh = bid % g.hkv;
  const int seq = bid / g.hkv;
  const int j = kb * KPB + static_cast<int>(threadIdx.x) / TPK;
  const int part = threadIdx.x % TPK;
  const int n = clamp_len(ld_uniform(g.seq_lens, seq), view_capacity(g));
  if (j >= n) return;
  size_t row;
  if (g.page_size > 0) {
    const int phys = g.block_table[static_cast<size_t>(seq) * g.max_pages + j / g.page_size];
    if (phys < 0 || phys >= g.num_pages) return;
    row = (static_cast<size_t>(phys) * g.hkv + kvh) * g.page_size + j % g.page_size;
  } else {
    row = (static_cast<size_t>(seq) * g.hkv + kvh) * g.max_seq_len + j;
  }
  const size_t el = row * D + 8 * part;
  const uint2 pa = *reinterpret_cast<const uint2*>(a.ka + el);
  const uint2 pb = *reinterpret_cast<const uint2*>(a.kb + el);
  const float e = bf16_lo(a.ks[row]);
  uint32_t h[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t wa = i < 4 ? pa.x : pa.y;
    const uint32_t wb = i < 4 ? pb.x : pb.y;
    const int ca = static_cast<int8_t>((wa >> (8 * (i & 3))) & 0xffu);
    const int cb = static_cast<int8_t>((wb >> (8 * (i & 3))) & 0xffu);
    // a + b/256 is exact in FP32, and so is its product with an 8-bit scale
    const float code = static_cast<float>(ca) + static_cast<float>(cb) * (1.0f / 256.0f);
    h[i] = f32_to_f16_bits(e * code);
  }
  *reinterpret_cast<u32x4*>(a.out + el) =
      u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
}

}  // namespace

hipError_t launch_q8_stack_keys(const Q8StackArgs& a, int head_dim, hipStream_t stream) {
  const int cap = view_capacity(a.geo);
  const int kpb = kFrontThreads / (head_dim / 8);
  const int per_seq = (cap + kpb - 1) / kpb;
  const long long blocks = static_cast<long long>(a.geo.num_seqs) * a.geo.hkv * per_seq;
  if (blocks == 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(q8_stack_kernel<128>, dim3(static_cast<unsigned>(blocks)),
                       dim3(kFrontThreads), 0, stream, a, per_seq);
  else if (head_dim == 64)
    hipLaunchKernelGGL(q8_stack_kernel<64>, dim3(static_cast<unsigned>(blocks)),
                       dim3(kFrontThreads), 0, stream, a, per_seq);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_v8_write(const V8WriteArgs& a, int head_dim, hipStream_t stream) {
  const long long items = static_cast<long long>(a.n_tok) * a.geo.hkv;
  if (items == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((items + kWavesPerBlock - 1) / kWavesPerBlock);
  if (head_dim == 128)
    hipLaunchKernelGGL(v8_write_kernel<128>, dim3(blocks), dim3(kFrontThreads), 0, stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(v8_write_kernel<64>, dim3(blocks), dim3(kFrontThreads), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_q8_write(const Q8WriteArgs& a, int head_dim, hipStream_t stream) {
  const long long items = static_cast<long long>(a.n_tok) * a.geo.hkv;
  if (items == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((items + kWavesPerBlock - 1) / kWavesPerBlock);
  if (head_dim == 128)
    hipLaunchKernelGGL(q8_write_kernel<128>, dim3(blocks), dim3(kFrontThreads), 0, stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(q8_write_kernel<64>, dim3(blocks), dim3(kFrontThreads), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_q8_split(const Q8SplitArgs& a, int head_dim, hipStream_t stream) {
  const long long waves = a.rows > 0 ? a.rows : 1;  // block 0 also writes tau
  if (a.rows == 0 && !a.tau) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((waves + kWavesPerBlock - 1) / kWavesPerBlock);
  if (head_dim == 128)
    hipLaunchKernelGGL(q8_split_kernel<128>, dim3(blocks), dim3(kFrontThreads), 0, stream, a);
  else if (head_dim == 64)
    hipLaunchKernelGGL(q8_split_kernel<64>, dim3(blocks), dim3(kFrontThreads), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace fold
