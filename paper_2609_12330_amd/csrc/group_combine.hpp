// Combine of one group's stored partial states by the workgroup that stores
// the group's last state (the combine of section 4.2 fused into the split
// producer of section 3.3): an arrival counter per group decides which
// workgroup is last; that workgroup reads every partition's state of the
// group's rows and writes the output.
//
// Visibility across workgroups (and across the chip's XCDs, whose L2 caches
// are not coherent with each other): the producer stores its state with
// device-scope stores (sc1), which are written through to the device
// coherence point and count in the wave's vector-memory counter until that
// point acknowledges them. Before the workgroup barrier every wave waits for
// that counter to drain (s_waitcnt vmcnt(0)), so when the ticket is taken all
// of the workgroup's state stores are visible at device scope; the last
// workgroup then reads the states with device-scope loads (sc1), which do not
// hit stale lines in its own L2. This orders the states before the ticket
// without the full L2 write-back/invalidate of a device-scope release/acquire
// fence, which costs more than the whole producer when every workgroup issues
// one. (A workgroup-scope release fence alone is not enough on this chip: it
// only orders the stores for the workgroup's own L2 view and compiles to no
// wait at all.)
#pragma once

#include "ef_device.hpp"
#include "ef_kernels.hpp"

namespace ef {

// Device-scope (coherent across XCDs) store and load of one float.
__device__ __forceinline__ void store_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_dev(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Takes a ticket on the group's arrival counter once this workgroup's
// device-scope state stores have completed; returns the ticket (the same in
// every thread of the workgroup). Tickets run 0 .. arrivals - 1 from a
// counter that is zero when the launch begins; the workgroup holding
// arrivals - 1 arrives last.
__device__ __forceinline__ unsigned arrival_ticket(unsigned* counter) {
  __shared__ unsigned ticket;
  // Compiler ordering: no store above may sink below this point.
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  // Hardware ordering: this wave's device-scope state stores have been
  // acknowledged (vmcnt(0); expcnt and lgkmcnt left at their maximum).
  __builtin_amdgcn_s_waitcnt(0x0f70);
  __syncthreads();
  if (threadIdx.x == 0)
    ticket = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  return ticket;
}

// Output rows row0 .. row0 + nrows - 1, channels [d0, d0 + DW), set to NaN. A
// ticket at or past the arrival count means the counter was not zero when the
// launch began (a workspace whose counter region was never cleared), so the
// group's combine cannot be trusted: its rows are made visibly invalid rather
// than silently stale.
template <int D, int DW, int NT>
__device__ __forceinline__ void poison_group(float* o, size_t row0, int nrows, int d0) {
  for (int i = threadIdx.x; i < nrows * DW; i += NT)
    o[(row0 + i / DW) * D + d0 + i % DW] = __builtin_nanf("");
}

__device__ __forceinline__ void reset_counter(unsigned* counter) {
  __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Lanes that form one row of the weights pass, and the maximum over each such
// aligned group of 16 lanes (every lane gets it).
constexpr int kRowLanes = 16;
__device__ __forceinline__ float row_max(float x) {
  x = fmaxf(x, dpp_mov<kDppRowRor8>(x));
  x = fmaxf(x, dpp_mov<kDppRowRor4>(x));
  x = fmaxf(x, dpp_mov<kDppQuadXor2>(x));
  x = fmaxf(x, dpp_mov<kDppQuadXor1>(x));
  return x;
}

// 16 bytes from byte offset `off` of a buffer, read at device scope (coherent
// across XCDs: the read does not hit a stale line of this XCD's L2); 0 when
// `off` is past the buffer.
__device__ __forceinline__ u32x4_t load16_dev(__amdgpu_buffer_rsrc_t rs, int off) {
  constexpr int kDeviceScope = 16;  // sc1 cache policy
  return __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, kDeviceScope);
}

// o[row0 + r][d0 : d0 + DW] = sum_p exp(m_p - M) acc_p / sum_p exp(m_p - M) l_p
// over the P stored states of rows row0 .. row0 + nrows - 1 (0 for a row with
// no visible key), the states read with device-scope loads; DW = D unless the
// group covers one output-channel slice of the rows; nrows <= MAXROWS and
// P <= kFusedMaxP. cw, cl: LDS of at least nrows * P floats; cinv: nrows
// floats. The combine is the tail of the producer that arrives last, so it is
// arranged for few round trips: each thread owns two 4-element slices of the
// output rows and requests the value states of 16 partitions of both at once,
// the first 16 right behind the reference points and sums.
template <int D, int DW, int NT, int MAXROWS>
__device__ __forceinline__ void combine_group(const float* ws_m, const float* ws_l,
                                              const float* ws_acc, float* o, size_t row0,
                                              int nrows, int P, float* cw, float* cl,
                                              float* cinv, int d0) {
  static_assert(DW % 4 == 0 && D % DW == 0, "whole 4-element slices of a row");
  constexpr int D4 = DW / 4;  // 4-element slices of a row's channel range
  constexpr int BATCH = 16;  // partitions per slice in flight
  const int n = nrows * P;
  const int bytes = n * D * 4;  // at most 8 * 64 * 128 * 4
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(ws_acc + row0 * (size_t)P * D), (short)0, bytes, 0x00020000);
  const int nslices = nrows * D4;

  // Byte offset of slice c's value state in partition p; the buffer's end (a
  // zero read) past the row's partitions or past the slices.
  auto slice_off = [&](int c, int p) {
    return (c < nslices && p < P) ? ((c / D4) * P * D + p * D + d0 + (c % D4) * 4) * 4 : bytes;
  };
  auto load_batch = [&](int c0, int p0, u32x4_t (&x0)[BATCH], u32x4_t (&x1)[BATCH]) {
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      x0[j] = load16_dev(rs, slice_off(c0, p0 + j));
      x1[j] = load16_dev(rs, slice_off(c0 + NT, p0 + j));
    }
  };
  auto fold_batch = [&](int c0, int p0, const u32x4_t (&x0)[BATCH], const u32x4_t (&x1)[BATCH],
                        floatx4& s0, floatx4& s1) {
    const int r0 = min(c0, nslices - 1) / D4, r1 = min(c0 + NT, nslices - 1) / D4;
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int p = min(p0 + j, P - 1);
      // Unconditional reads of a clamped index (a guarded read compiles to a branch
      // per partition); a weight past the row's partitions counts zero times.
      const float in = p0 + j < P ? 1.f : 0.f;
      const float w0 = cw[r0 * P + p] * in;
      const float w1 = cw[r1 * P + p] * in;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s0[e] = fmaf(w0, __uint_as_float(x0[j][e]), s0[e]);
        s1[e] = fmaf(w1, __uint_as_float(x1[j][e]), s1[e]);
      }
    }
  };
  auto store_slice = [&](int c, const floatx4& sv) {
    if (c < nslices) {
      const float inv = cinv[c / D4];
      *reinterpret_cast<float4*>(o + (row0 + c / D4) * D + d0 + (c % D4) * 4) =
          make_float4(sv[0] * inv, sv[1] * inv, sv[2] * inv, sv[3] * inv);
    }
  };

  // The reference points and sums first, all requested before any is used, then
  // the first values: loads complete in order, so the barrier waits for the
  // small loads only and the values land while the weights are formed.
  // At most MAXROWS rows of at most kFusedMaxP partitions: KMAX states per thread.
  constexpr int KMAX = (MAXROWS * kFusedMaxP + NT - 1) / NT;
  float mv[KMAX], lv[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    if (k * NT < n) {
      const int i = min((int)threadIdx.x + k * NT, n - 1);
      mv[k] = load_dev(ws_m + row0 * P + i);
      lv[k] = load_dev(ws_l + row0 * P + i);
    }
  }
  u32x4_t x0[BATCH], x1[BATCH];
  load_batch(threadIdx.x, 0, x0, x1);
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    const int i = (int)threadIdx.x + k * NT;
    if (k * NT < n && i < n) {
      cw[i] = mv[k];
      cl[i] = lv[k];
    }
  }
  __syncthreads();
  // Row weights: 16 lanes per row, lane j over partitions j, j + 16, ...; the
  // row's maximum and sum are combined across its lanes with DPP moves, so no
  // lane walks a row's partitions one after the other through LDS.
  static_assert(NT % kRowLanes == 0, "whole rows of lanes");
  constexpr int PPL = (kFusedMaxP + kRowLanes - 1) / kRowLanes;  // partitions per lane
  const int j = (int)threadIdx.x % kRowLanes;
  for (int r = (int)threadIdx.x / kRowLanes; r < nrows; r += NT / kRowLanes) {
    float mloc[PPL];
    float M = kNegInf;
#pragma unroll
    for (int k = 0; k < PPL; ++k) {
      const int p = j + k * kRowLanes;
      const float x = cw[r * P + min(p, P - 1)];  // clamped read; lanes past P count -inf
      mloc[k] = p < P ? x : kNegInf;
      M = fmaxf(M, mloc[k]);
    }
    M = row_max(M);
    const float ref = (M == kNegInf) ? 0.f : M;
    float L = 0.f;
#pragma unroll
    for (int k = 0; k < PPL; ++k) {
      const int p = j + k * kRowLanes;
      const float w = exp2_fast((mloc[k] - ref) * kLog2e);  // 0 for the identity and past P
      if (p < P) cw[r * P + p] = w;
      L = fmaf(w, cl[r * P + min(p, P - 1)], L);
    }
    L = group_sum<kRowLanes>(L);
    if (j == 0) cinv[r] = (M == kNegInf || L == 0.f) ? 0.f : 1.f / L;
  }
  __syncthreads();
  for (int c0 = threadIdx.x; c0 < nslices; c0 += 2 * NT) {
    floatx4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
    if (c0 != (int)threadIdx.x) load_batch(c0, 0, x0, x1);
    fold_batch(c0, 0, x0, x1, s0, s1);
    for (int p0 = BATCH; p0 < P; p0 += BATCH) {
      load_batch(c0, p0, x0, x1);
      fold_batch(c0, p0, x0, x1, s0, s1);
    }
    store_slice(c0, s0);
    store_slice(c0 + NT, s1);
  }
}

}  // namespace ef
