// Differential attention epilogue (section 7.3): the mixing weight and the
// per-row RMS normalisation applied to y = A1 - lambda * A2, shared by the
// single-pass attention kernel and the split-KV combine.
#pragma once

#include "ef_device.hpp"
#include "ef_kernels.hpp"

namespace ef {

// Sum of x over the 64 lanes of the wave, in every lane.
__device__ __forceinline__ float wave_sum(float x) {
  x += __shfl_xor(x, 32, 64);
  x += __shfl_xor(x, 16, 64);
  return group_sum<16>(x);
}

// lambda = exp(<lq1, lk1>) - exp(<lq2, lk2>) + lambda_init over D entries.
// Every lane of the wave must call it; every lane gets lambda.
__device__ __forceinline__ float diff_lambda(const DiffParams& p, int lane, int D) {
  float a = 0.f, b = 0.f;
  for (int i = lane; i < D; i += 64) {
    a = fmaf(p.lq1[i], p.lk1[i], a);
    b = fmaf(p.lq2[i], p.lk2[i], b);
  }
  a = wave_sum(a);
  b = wave_sum(b);
  return expf(a) - expf(b) + p.lambda_init;
}

// Factor (1 - lambda_init) / sqrt(mean(y^2) + eps) of a row whose y^2 sums to
// ss over D entries; 0 when the mean plus eps is not positive (a row of zeros
// with eps = 0).
__device__ __forceinline__ float diff_row_factor(const DiffParams& p, float ss, int D) {
  const float ms = ss / (float)D + p.eps;
  return ms > 0.f ? (1.f - p.lambda_init) / sqrtf(ms) : 0.f;
}

}  // namespace ef
