// Combine of one group's stored partial states by the workgroup that stores
// the group's last state (the combine of section 4.2 fused into the split
// producer of section 3.3): an arrival counter per group decides which
// workgroup is last; that workgroup reads every partition's state of the
// group's rows and writes the output.
//
// Visibility across workgroups (and across the chip's XCDs, whose L2 caches
// are not coherent with each other): the producer stores its state with
// device-scope stores (global_store ... sc1), which are written through to the
// device coherence point; before taking a ticket each thread waits for those
// stores to complete; the last workgroup reads the states with device-scope
// loads (sc1), which do not hit stale lines in its own L2. This orders the
// states before the ticket without the full L2 write-back/invalidate of a
// device-scope release/acquire fence, which costs more than the whole
// producer when every workgroup issues one.
#pragma once

#include "ef_device.hpp"

namespace ef {

// Device-scope (coherent across XCDs) store and load of one float.
__device__ __forceinline__ void store_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_dev(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Takes a ticket on the group's arrival counter once this workgroup's
// device-scope state stores have completed; true in every thread of the
// workgroup that arrives last.
__device__ __forceinline__ bool last_of_group(unsigned* counter, int arrivals) {
  __shared__ unsigned ticket;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");  // waits for the stores above
  __syncthreads();
  if (threadIdx.x == 0)
    ticket = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  return ticket == (unsigned)(arrivals - 1);
}

__device__ __forceinline__ void reset_counter(unsigned* counter) {
  __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// o[row0 + r][:] = sum_p exp(m_p - M) acc_p / sum_p exp(m_p - M) l_p over the
// P stored states of rows row0 .. row0 + nrows - 1 (0 for a row with no
// visible key), the states read with device-scope loads. cw, cl: LDS of at
// least nrows * P floats; cinv: nrows floats.
template <int D, int NT>
__device__ void combine_group(const float* ws_m, const float* ws_l, const float* ws_acc, float* o,
                              size_t row0, int nrows, int P, float* cw, float* cl, float* cinv) {
  const int n = nrows * P;
  for (int i = threadIdx.x; i < n; i += NT) {
    cw[i] = load_dev(ws_m + row0 * P + i);
    cl[i] = load_dev(ws_l + row0 * P + i);
  }
  __syncthreads();
  for (int r = threadIdx.x; r < nrows; r += NT) {
    float M = kNegInf;
    for (int p = 0; p < P; ++p) M = fmaxf(M, cw[r * P + p]);
    const float ref = (M == kNegInf) ? 0.f : M;
    float L = 0.f;
    for (int p = 0; p < P; ++p) {
      const float w = exp2_fast((cw[r * P + p] - ref) * kLog2e);  // 0 for the identity
      cw[r * P + p] = w;
      L = fmaf(w, cl[r * P + p], L);
    }
    cinv[r] = (M == kNegInf || L == 0.f) ? 0.f : 1.f / L;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nrows * D; i += NT) {
    const int r = i / D, d = i % D;
    const float* ap = ws_acc + (row0 + r) * (size_t)P * D + d;
    float s0 = 0.f, s1 = 0.f;
    int p = 0;
    for (; p + 1 < P; p += 2) {
      s0 = fmaf(cw[r * P + p], load_dev(ap + (size_t)p * D), s0);
      s1 = fmaf(cw[r * P + p + 1], load_dev(ap + (size_t)(p + 1) * D), s1);
    }
    if (p < P) s0 = fmaf(cw[r * P + p], load_dev(ap + (size_t)p * D), s0);
    o[(row0 + r) * D + d] = (s0 + s1) * cinv[r];
  }
}

}  // namespace ef
