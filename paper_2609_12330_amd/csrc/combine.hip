// Combine of stored split-KV partial states (section 4.2: the fused reducer
// with h(c, s, s') = c * exp(s - s'), applied to the states that the producer
// stored along the partition axis, section 3.3 "Collection").
//
// Two layouts. With few partitions (P <= 32) one wave takes a whole row, each
// lane owning D/64 adjacent elements and folding the partitions in order. With
// many partitions, one wave takes a (row, 8-element slice of D): lane l takes partitions
// p = l/2, l/2 + 32, ... and one 4-float half of the slice, so each pass of the
// wave reads 32 partitions x 32 contiguous bytes and every lane keeps several
// independent loads in flight. Each lane folds its partitions into one state
// with the same reducer (reference moves up to the larger maximum, the other
// side is rescaled by exp of the difference; the identity state (-inf, 0, 0)
// contributes nothing), then the 32 partition lanes of each half merge
// pairwise in a fixed butterfly order, so the result is deterministic.
#include "diff_norm.hpp"
#include "ef_device.hpp"
#include "ef_kernels.hpp"

namespace ef {

namespace {

constexpr int kSlice = 8;              // floats of D per wave
constexpr int kLanesPerPart = kSlice / 4;  // lanes per partition (one float4 each)
constexpr int kPartsPerPass = 64 / kLanesPerPart;
constexpr int kRowsKernelMaxP = 32;  // up to this many partitions: one wave per row

struct Acc4 {
  float m, l, a0, a1, a2, a3;
};

// Fold state (mb, lb, xb) into (s.m, s.l, s.a): rolling reducer on two states.
__device__ __forceinline__ void fold(Acc4& s, float mb, float lb, float b0, float b1, float b2,
                                     float b3) {
  const float mn = fmaxf(s.m, mb);
  const float ref = (mn == kNegInf) ? 0.f : mn;
  const float wa = exp2_fast((s.m - ref) * kLog2e);  // 0 for the identity
  const float wb = exp2_fast((mb - ref) * kLog2e);
  s.l = s.l * wa + lb * wb;
  s.a0 = s.a0 * wa + b0 * wb;
  s.a1 = s.a1 * wa + b1 * wb;
  s.a2 = s.a2 * wa + b2 * wb;
  s.a3 = s.a3 * wa + b3 * wb;
  s.m = mn;
}

}  // namespace

// Many partitions: one wave per (row, 8-float slice).
__global__ __launch_bounds__(64) void combine_sliced_kernel(CombineParams a) {
  const int lane = threadIdx.x;
  const int slices = a.D / kSlice;
  const int row = blockIdx.x / slices;
  const int slice = blockIdx.x % slices;
  const int P = a.P;
  const int half = lane % kLanesPerPart;
  const int p0 = lane / kLanesPerPart;
  const float* mrow = a.m + (size_t)row * P;
  const float* lrow = a.l + (size_t)row * P;
  const float* arow = a.acc + (size_t)row * P * a.D + slice * kSlice + half * 4;

  Acc4 s{kNegInf, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int p = p0; p < P; p += kPartsPerPass) {
    const float mp = mrow[p];
    const float lp = lrow[p];
    const float4 x = *reinterpret_cast<const float4*>(arow + (size_t)p * a.D);
    fold(s, mp, lp, x.x, x.y, x.z, x.w);
  }
#pragma unroll
  for (int off = kLanesPerPart; off < 64; off <<= 1) {
    const float mb = shfl_xor(s.m, off), lb = shfl_xor(s.l, off);
    const float b0 = shfl_xor(s.a0, off), b1 = shfl_xor(s.a1, off);
    const float b2 = shfl_xor(s.a2, off), b3 = shfl_xor(s.a3, off);
    fold(s, mb, lb, b0, b1, b2, b3);
  }
  if (lane < kLanesPerPart) {
    const bool empty = s.m == kNegInf || s.l == 0.f;
    const float inv = empty ? 0.f : 1.f / s.l;
    float4 out = make_float4(s.a0 * inv, s.a1 * inv, s.a2 * inv, s.a3 * inv);
    *reinterpret_cast<float4*>(a.o + (size_t)row * a.D + slice * kSlice + half * 4) = out;
  }
}

// Few partitions: one wave per row, each lane owning D/64 adjacent elements and
// folding the row's partitions in order. With DIFF the states are the first
// branch of a differential attention layer: the wave also forms
// y = A1 - lambda * A2 against the second branch's output already in o and
// writes the RMS-normalised row (section 7.3).
template <int D, bool DIFF>
__global__ __launch_bounds__(256) void combine_rows_kernel(CombineParams a) {
  constexpr int EPL = D / 64;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  const int lane = threadIdx.x & 63;
  const int P = a.P;
  const float* mrow = a.m + (size_t)row * P;
  const float* lrow = a.l + (size_t)row * P;
  const float* arow = a.acc + (size_t)row * P * D + lane * EPL;
  float M = kNegInf, L = 0.f, A[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) A[e] = 0.f;
#pragma unroll 4
  for (int p = 0; p < P; ++p) {
    const float mp = mrow[p];
    const float lp = lrow[p];
    float x[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) x[e] = arow[(size_t)p * D + e];
    const float mn = fmaxf(M, mp);
    const float ref = (mn == kNegInf) ? 0.f : mn;
    const float wa = exp2_fast((M - ref) * kLog2e);
    const float wb = exp2_fast((mp - ref) * kLog2e);
    L = L * wa + lp * wb;
#pragma unroll
    for (int e = 0; e < EPL; ++e) A[e] = A[e] * wa + x[e] * wb;
    M = mn;
  }
  const float inv = (M == kNegInf || L == 0.f) ? 0.f : 1.f / L;
  float* orow = a.o + (size_t)row * D + lane * EPL;
  if constexpr (DIFF) {
    const float lam = diff_lambda(a.diff, lane, D);
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      A[e] = fmaf(-lam, orow[e], A[e] * inv);
      ss = fmaf(A[e], A[e], ss);
    }
    const float rn = diff_row_factor(a.diff, wave_sum(ss), D);
#pragma unroll
    for (int e = 0; e < EPL; ++e) orow[e] = rn * a.diff.gamma[lane * EPL + e] * A[e];
  } else {
#pragma unroll
    for (int e = 0; e < EPL; ++e) orow[e] = A[e] * inv;
  }
}

hipError_t launch_combine(const CombineParams& a, hipStream_t stream) {
  if (a.rows == 0) return hipSuccess;
  const bool diff = a.diff.gamma != nullptr;
  if (a.P <= kRowsKernelMaxP || diff) {
    // The differential epilogue normalises whole rows, so it always takes the
    // one-wave-per-row layout.
    const unsigned blocks = (unsigned)((a.rows + 3) / 4);
    auto kern = a.D == 128 ? (diff ? combine_rows_kernel<128, true> : combine_rows_kernel<128, false>)
                           : (diff ? combine_rows_kernel<64, true> : combine_rows_kernel<64, false>);
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, stream, a);
  } else {
    const size_t waves = (size_t)a.rows * (a.D / kSlice);
    hipLaunchKernelGGL(combine_sliced_kernel, dim3((unsigned)waves), dim3(64), 0, stream, a);
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
