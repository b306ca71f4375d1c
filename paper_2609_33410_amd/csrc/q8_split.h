// The per-vector transform and split of the two-plane INT8 format (Section 4,
// "Cache format"), shared by the key writer, the query split and the fused
// front: a Sylvester Hadamard rotation in FP64 across one wave64 (lane l holds
// elements 64 i + l), the wave's largest magnitude, and the split of one
// element into two INT8 planes under a scale.
#pragma once

#include "fold_device.h"

namespace fold {

constexpr double kLog2eF64 = 0x1.71547652b82fep+0;

template <int D>
__device__ __forceinline__ void hadamard_wave(double (&x)[D / 64], int lane) {
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) {
#pragma unroll
    for (int i = 0; i < D / 64; ++i) {
      const double o = __shfl_xor(x[i], s, 64);
      x[i] = (lane & s) ? o - x[i] : x[i] + o;
    }
  }
  if constexpr (D == 128) {
    const double u = x[0], v = x[1];
    x[0] = u + v;
    x[1] = u - v;
  }
}

template <int D>
__device__ __forceinline__ double wave_absmax_f64(const double (&x)[D / 64]) {
  double m = 0.0;
#pragma unroll
  for (int i = 0; i < D / 64; ++i) m = fmax(m, fabs(x[i]));
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) m = fmax(m, __shfl_xor(m, s, 64));
  return m;
}

__device__ __forceinline__ void split_value(double x, double s, int8_t* a, int8_t* b) {
  if (s > 0.0) {
    const double y = x / s;
    const double ai = rint(y);
    const double bi = fmin(fmax(rint(256.0 * (y - ai)), -128.0), 127.0);
    *a = static_cast<int8_t>(ai);
    *b = static_cast<int8_t>(bi);
  } else {
    *a = 0;
    *b = 0;
  }
}

}  // namespace fold
