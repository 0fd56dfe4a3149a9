// Device helpers shared by the gfx950 attention kernels: bf16 packing,
// wave64 DPP reductions, the exp2 used by the online softmax, and the
// partial-state workspace layout.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ef {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_inff();

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// 16-byte global load marked non-temporal (streamed once, not kept in cache).
__device__ __forceinline__ uint4 load_nt16(const uint4* p) {
  const u32x4_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(x[0], x[1], x[2], x[3]);
}

// 16-byte global load, non-temporal or regular.
template <bool NT>
__device__ __forceinline__ uint4 load16(const uint4* p) {
  if constexpr (NT) {
    return load_nt16(p);
  } else {
    const u32x4_t x = *reinterpret_cast<const u32x4_t*>(p);
    return make_uint4(x[0], x[1], x[2], x[3]);
  }
}

// bf16 (upper half of binary32) <-> fp32.
__device__ __forceinline__ float bf16lo_to_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi_to_f32(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two fp32 -> packed bf16 pair (round to nearest even), lo in bits 0..15.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2_t p;
  p[0] = static_cast<__bf16>(lo);
  p[1] = static_cast<__bf16>(hi);
  return __builtin_bit_cast(uint32_t, p);
}

// dot of two packed bf16 pairs accumulated into fp32: c + a0*b0 + a1*b1.
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

// 2^x on the transcendental unit; exact 0 for -inf.
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// DPP lane moves inside a row of 16 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int kDppRowRor8 = 0x128;
constexpr int kDppRowRor4 = 0x124;
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppQuadXor2 = 0x4e;  // quad_perm [2,3,0,1]
constexpr int kDppQuadXor1 = 0xb1;  // quad_perm [1,0,3,2]

// Sum over aligned groups of LANES lanes (16, 8 or 4); every lane gets the group's sum.
template <int LANES>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(LANES == 16 || LANES == 8 || LANES == 4, "group of 4, 8 or 16 lanes");
  if constexpr (LANES == 16) {
    x += dpp_mov<kDppRowRor8>(x);
    x += dpp_mov<kDppRowRor4>(x);
  } else if constexpr (LANES == 8) {
    x += dpp_mov<kDppHalfMirror>(x);
  }
  x += dpp_mov<kDppQuadXor2>(x);
  x += dpp_mov<kDppQuadXor1>(x);
  return x;
}

__device__ __forceinline__ float shfl_xor(float x, int mask) {
  return __shfl_xor(x, mask, 64);
}

// The values of x in this lane and in its partner lane at distance OFF, as a
// pair (a, b) whose order may differ between the two lanes. OFF = 16 and 32
// pair lane l with l ^ OFF (permlane swaps); OFF = 4 and 8 pair lane l with
// lane l + OFF of its 16-lane row (DPP rotation; for 8 that is l ^ 8). Taking
// OFF = 4, 8, 16, 32 in increasing order from some start combines every lane
// group, like a butterfly.
template <int OFF>
__device__ __forceinline__ void lane_pair(float x, float& a, float& b) {
  static_assert(OFF == 4 || OFF == 8 || OFF == 16 || OFF == 32, "lane distance");
  if constexpr (OFF == 4 || OFF == 8) {
    a = x;
    b = dpp_mov<OFF == 4 ? kDppRowRor4 : kDppRowRor8>(x);
  } else if constexpr (OFF == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
  }
}

// Partial-state workspace: m [rows][P], l [rows][P], acc [rows][P][D] fp32.
__host__ __device__ __forceinline__ size_t ws_align256(size_t n) { return (n + 255) & ~size_t(255); }

struct PartialState {
  float* m;
  float* l;
  float* acc;
};

}  // namespace ef
