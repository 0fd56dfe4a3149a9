// Combine of stored split-KV partial states (section 4.2: the fused reducer
// with h(c, s, s') = c * exp(s - s'), applied to the states that the producer
// stored along the partition axis, section 3.3 "Collection").
//
// Two layouts. With few partitions (P <= 32) one wave takes a whole row, each
// lane owning D/64 adjacent elements and folding the partitions in order. With
// many partitions, a workgroup takes a (row, 16-element slice of D) and
// requests up to 512 partitions' values at once; each lane folds its
// partitions into one state with the same reducer (reference moves up to the
// larger maximum, the other side is rescaled by exp of the difference; the
// identity state (-inf, 0, 0) contributes nothing), then the lanes merge in a
// fixed butterfly order and the waves in a fixed order, so the result is
// deterministic.
#include "diff_norm.hpp"
#include "ef_device.hpp"
#include "ef_kernels.hpp"

namespace ef {

namespace {

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

// Many partitions, in one round trip: one workgroup of four waves per (row,
// 16-float slice of D). Four adjacent lanes read a partition's 64 contiguous
// bytes of the slice, so a pass of the workgroup covers 64 partitions, and the
// eight passes of 512 partitions are all requested before any is folded. Each
// lane folds its partitions in order with the reducer; the 16 partition lanes
// of each quarter in a wave merge by butterfly, then the four waves' states in
// order through LDS, so the result is deterministic.
constexpr int kWideSlice = 16;                         // floats of D per workgroup
constexpr int kWideLanes = kWideSlice / 4;             // lanes per partition (a float4 each)
constexpr int kWideThreads = 256;
constexpr int kWideGroups = kWideThreads / kWideLanes;  // partitions per pass
constexpr int kWidePasses = 8;                         // passes in flight

__global__ __launch_bounds__(kWideThreads) void combine_wide_kernel(CombineParams a) {
  const int slices = a.D / kWideSlice;
  const int row = blockIdx.x / slices;
  const int slice = blockIdx.x % slices;
  const int P = a.P;
  const int t = threadIdx.x;
  const int quarter = t % kWideLanes;
  const int g = t / kWideLanes;
  const float* mrow = a.m + (size_t)row * P;
  const float* lrow = a.l + (size_t)row * P;
  const float* arow = a.acc + (size_t)row * P * a.D + slice * kWideSlice + quarter * 4;

  Acc4 s{kNegInf, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int p0 = 0; p0 < P; p0 += kWideGroups * kWidePasses) {
    float mv[kWidePasses], lv[kWidePasses];
    float4 x[kWidePasses];
    // Unconditional reads of a clamped partition (a guarded read compiles to a
    // branch); a partition past the last folds as the identity state.
#pragma unroll
    for (int i = 0; i < kWidePasses; ++i) {
      const int pc = min(p0 + g + kWideGroups * i, P - 1);
      mv[i] = mrow[pc];
      lv[i] = lrow[pc];
      x[i] = *reinterpret_cast<const float4*>(arow + (size_t)pc * a.D);
    }
#pragma unroll
    for (int i = 0; i < kWidePasses; ++i) {
      const bool in = p0 + g + kWideGroups * i < P;
      fold(s, in ? mv[i] : kNegInf, in ? lv[i] : 0.f, in ? x[i].x : 0.f, in ? x[i].y : 0.f,
           in ? x[i].z : 0.f, in ? x[i].w : 0.f);
    }
  }
#pragma unroll
  for (int off = kWideLanes; off < 64; off <<= 1) {
    const float mb = shfl_xor(s.m, off), lb = shfl_xor(s.l, off);
    const float b0 = shfl_xor(s.a0, off), b1 = shfl_xor(s.a1, off);
    const float b2 = shfl_xor(s.a2, off), b3 = shfl_xor(s.a3, off);
    fold(s, mb, lb, b0, b1, b2, b3);
  }
  constexpr int kWaves = kWideThreads / 64;
  __shared__ float st[kWaves][kWideLanes][6];
  const int wave = t / 64, lane = t % 64;
  if (lane < kWideLanes) {
    st[wave][lane][0] = s.m;
    st[wave][lane][1] = s.l;
    st[wave][lane][2] = s.a0;
    st[wave][lane][3] = s.a1;
    st[wave][lane][4] = s.a2;
    st[wave][lane][5] = s.a3;
  }
  __syncthreads();
  if (t < kWideLanes) {
    Acc4 r{st[0][t][0], st[0][t][1], st[0][t][2], st[0][t][3], st[0][t][4], st[0][t][5]};
#pragma unroll
    for (int w = 1; w < kWaves; ++w)
      fold(r, st[w][t][0], st[w][t][1], st[w][t][2], st[w][t][3], st[w][t][4], st[w][t][5]);
    const bool empty = r.m == kNegInf || r.l == 0.f;
    const float inv = empty ? 0.f : 1.f / r.l;
    *reinterpret_cast<float4*>(a.o + (size_t)row * a.D + slice * kWideSlice + t * 4) =
        make_float4(r.a0 * inv, r.a1 * inv, r.a2 * inv, r.a3 * inv);
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
    const size_t blocks = (size_t)a.rows * (a.D / kWideSlice);
    hipLaunchKernelGGL(combine_wide_kernel, dim3((unsigned)blocks), dim3(kWideThreads), 0,
                       stream, a);
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
