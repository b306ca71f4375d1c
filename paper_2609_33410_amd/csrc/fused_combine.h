// The slot handoff and combine of the one-launch decode (fold_decode_fused,
// fold_decode_fused_noalloc): every split stores its slot, counts its arrival, and
// the split that counts last adds the slots into the output (Algorithm 1, last
// step; Section 3 certificate).
#pragma once

#include "decode_common.h"

namespace fold {

// Slot values of the one-launch decode are stored and read with the
// device-scope cache bit (SC1): the accesses are coherent at the chip's
// coherence point past the per-XCD L2s, as device-scope atomics are, so a
// split that finishes on one XCD and the split that combines on another need
// no L2 write-back or invalidation (each costs far more than the few kilobytes
// it would publish).  Offsets are bytes from the slot array's base (the host
// keeps the array under 2 GiB).
constexpr int kDeviceScope = 16;  // the SC1 bit of the gfx950 cache-policy field

__device__ __forceinline__ void slot_store4(rsrc_t r, uint32_t off, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, off, 0, kDeviceScope);
}
__device__ __forceinline__ void slot_store1(rsrc_t r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, off, 0, kDeviceScope);
}
__device__ __forceinline__ f32x4 slot_load4(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kDeviceScope));
}
__device__ __forceinline__ float slot_load1(rsrc_t r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kDeviceScope));
}

// Buffer resources over the slot arrays A and L of the call's slots.
template <int D>
__device__ __forceinline__ void slot_rsrc(const DecodeArgs& a, rsrc_t* ra, rsrc_t* rl) {
  const uint32_t rows = static_cast<uint32_t>(
      static_cast<size_t>(a.slot_offset + a.num_splits) * a.geo.batch * a.geo.heads);
  *ra = make_rsrc(a.part_A, rows * static_cast<uint32_t>(D) * 4u);
  *rl = make_rsrc(a.part_L, rows * 4u);
}

// The last of a (kv sequence, kv head)'s splits adds their slots for the
// group's rows, as the combine does: A and L summed in increasing slot order
// from zero, o = A / L, the base-2 log-sum-exp Z + log2 L and the range
// certificate.  Every split waits until its slot stores are complete, then
// counts its arrival; the split that counts last reads the slots (its loads
// are issued only after it has seen the count) and leaves the count at zero
// for the next call.
template <int D>
__device__ __forceinline__ void fused_combine(const DecodeArgs& a, const FusedExtra& x,
                                              const ScanPlace& p, const long long (&out_row)[16],
                                              const float (&zs)[16]) {
  const ScanGeometry& g = a.geo;
  __shared__ int last;
  __shared__ float lrow[16];
  __shared__ int bad[16];
  // Ordering of the handoff.  The slot stores and loads carry SC1, the
  // encoding the memory model gives device-scope atomic stores and loads on
  // this target, so each one is coherent across XCDs by itself and the
  // protocol needs no L2 write-back or invalidate (a device-scope release
  // fence per workgroup, which issues one, costs 15 us per call on the
  // Llama-3-8B-shaped decode).  What remains is ordering:
  //  * hardware: s_waitcnt vmcnt(0) returns only after every slot store of
  //    the wave is acknowledged, and the barrier makes all four waves wait
  //    before the one atomic add; the last arriver's slot loads are issued
  //    after it has read the count through LDS and a second barrier;
  //  * compiler: the signal fences are compiler barriers (no instruction),
  //    so no slot store sinks below the count and no slot load rises above
  //    it whatever code generation does around the barriers.
  __builtin_amdgcn_s_waitcnt(0);  // this wave's slot stores are complete
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __syncthreads();
  int32_t* ctr = x.arrivals + static_cast<size_t>(p.seq) * g.hkv + p.kvh;
  if (threadIdx.x == 0)
    last = __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                   a.num_splits - 1
               ? 1
               : 0;
  if (threadIdx.x < 16) bad[threadIdx.x] = 0;
  __syncthreads();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  if (!last) return;
  const size_t nrows = static_cast<size_t>(g.batch) * g.heads;
  rsrc_t ra, rl;
  slot_rsrc<D>(a, &ra, &rl);
  for (int f = threadIdx.x; f < 16 * (D / 4); f += kScanThreads) {
    const int r = f / (D / 4);
    const int d = 4 * (f % (D / 4));
    const long long xr = out_row[r];
    if (xr < 0) continue;
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    float l = 0.0f;
    int s = 0;
    for (; s + 8 <= a.num_splits; s += 8) {
      f32x4 av[8];
      float lv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t sr = static_cast<uint32_t>(static_cast<size_t>(a.slot_offset + s + u) * nrows + xr);
        av[u] = slot_load4(ra, (sr * D + d) * 4u);
        lv[u] = slot_load1(rl, sr * 4u);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        acc += av[u];
        l += lv[u];
      }
    }
    for (; s < a.num_splits; ++s) {
      const uint32_t sr = static_cast<uint32_t>(static_cast<size_t>(a.slot_offset + s) * nrows + xr);
      acc += slot_load4(ra, (sr * D + d) * 4u);
      l += slot_load1(rl, sr * 4u);
    }
    float o[4];
    bool nf = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[i] = acc[i] / l;
      nf = nf || !isfinite(o[i]);
    }
    const size_t oi = static_cast<size_t>(xr) * D + d;
    if (x.out_bf16) {
      uint32_t h[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) h[i] = f32_to_bf16_rne(o[i]);
      const u32x2 ob = {h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
      *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(x.out) + oi) = ob;
    } else {
      *reinterpret_cast<f32x4*>(static_cast<float*>(x.out) + oi) = f32x4{o[0], o[1], o[2], o[3]};
    }
    if (nf) bad[r] = 1;
    if (d == 0) lrow[r] = l;
  }
  __syncthreads();
  if (threadIdx.x < 16) {
    const int r = threadIdx.x;
    const long long xr = out_row[r];
    if (xr >= 0) {
      const float l = lrow[r];
      if (x.lse_out) x.lse_out[xr] = zs[r] + log2f(l);
      if (x.cert_out) {
        uint8_t c = 0;
        if (l < 0.5f) c |= 1;
        if (l > 0x1p100f) c |= 2;
        if (bad[r]) c |= 4;
        x.cert_out[xr] = c;
      }
    }
  }
  if (threadIdx.x == 0) __hip_atomic_store(ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace fold
