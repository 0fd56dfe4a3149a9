// Combine of stored split-KV partial states (section 4.2: the fused reducer
// with h(c, s, s') = c * exp(s - s'), applied to the states that the producer
// stored along the partition axis, section 3.3 "Collection").
//
// One workgroup of 4 waves per output row. Pass 1 takes M = max_p m_p over
// the row's P partitions. Pass 2 lets wave w visit partitions w, w+4, ...,
// weight each state by exp(m_p - M) (0 for the identity state m_p = -inf) and
// accumulate the weighted acc (each lane owns D/64 adjacent elements) and the
// weighted l; two accumulators per wave alternate over partitions to keep
// the summation chains short. The four waves meet in LDS, in a fixed order,
// so the result is deterministic.
#include "ef_device.hpp"
#include "ef_kernels.hpp"

namespace ef {

template <int D>
__global__ __launch_bounds__(256) void combine_kernel(CombineParams a) {
  constexpr int NW = 4;
  constexpr int EPL = D / 64;  // elements per lane
  const int row = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int P = a.P;
  const float* mrow = a.m + (size_t)row * P;
  const float* lrow = a.l + (size_t)row * P;
  const float* arow = a.acc + (size_t)row * P * D;

  __shared__ float red[NW];
  __shared__ float lsum[NW];
  __shared__ float asum[NW][D];

  float mx = kNegInf;
  for (int p = threadIdx.x; p < P; p += NW * 64) mx = fmaxf(mx, mrow[p]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, shfl_xor(mx, off));
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  float M = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) M = fmaxf(M, red[w]);
  const float Ms = (M == kNegInf) ? 0.f : M;

  float A0[EPL], A1[EPL];
  float L0 = 0.f, L1 = 0.f;
#pragma unroll
  for (int e = 0; e < EPL; ++e) A0[e] = A1[e] = 0.f;
  int p = wave;
  for (; p + NW < P; p += 2 * NW) {
    const float w0 = exp2_fast((mrow[p] - Ms) * kLog2e);
    const float w1 = exp2_fast((mrow[p + NW] - Ms) * kLog2e);
    L0 = fmaf(w0, lrow[p], L0);
    L1 = fmaf(w1, lrow[p + NW], L1);
    const float* x0 = arow + (size_t)p * D + lane * EPL;
    const float* x1 = arow + (size_t)(p + NW) * D + lane * EPL;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      A0[e] = fmaf(w0, x0[e], A0[e]);
      A1[e] = fmaf(w1, x1[e], A1[e]);
    }
  }
  if (p < P) {
    const float w0 = exp2_fast((mrow[p] - Ms) * kLog2e);
    L0 = fmaf(w0, lrow[p], L0);
    const float* x0 = arow + (size_t)p * D + lane * EPL;
#pragma unroll
    for (int e = 0; e < EPL; ++e) A0[e] = fmaf(w0, x0[e], A0[e]);
  }
#pragma unroll
  for (int e = 0; e < EPL; ++e) asum[wave][lane * EPL + e] = A0[e] + A1[e];
  if (lane == 0) lsum[wave] = L0 + L1;
  __syncthreads();
  if (threadIdx.x < D) {
    const int d = threadIdx.x;
    const float L = (lsum[0] + lsum[1]) + (lsum[2] + lsum[3]);
    const float S = (asum[0][d] + asum[1][d]) + (asum[2][d] + asum[3][d]);
    a.o[(size_t)row * D + d] = (M == kNegInf || L == 0.f) ? 0.f : S / L;
  }
}

hipError_t launch_combine(const CombineParams& a, hipStream_t stream) {
  if (a.rows == 0) return hipSuccess;
  if (a.D == 128) {
    hipLaunchKernelGGL(combine_kernel<128>, dim3(a.rows), dim3(256), 0, stream, a);
  } else {
    hipLaunchKernelGGL(combine_kernel<64>, dim3(a.rows), dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

__global__ void zero_fill_kernel(float4* p, size_t n4) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n4;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

hipError_t launch_zero_fill(float* p, size_t n, hipStream_t stream) {
  // n is a multiple of 64 here (D in {64, 128}) and p is 16-byte aligned.
  const size_t n4 = n / 4;
  if (n4 == 0) return hipSuccess;
  size_t blocks = (n4 + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(zero_fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                     reinterpret_cast<float4*>(p), n4);
  return hipGetLastError();
}

}  // namespace ef
