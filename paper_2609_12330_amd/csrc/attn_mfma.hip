// Tiled rolling attention on bf16 MFMA (form M2 of figure
// "attention-rewrites", section 3; code-generation mapping of section 6.1:
// the query-row tile axis is the grid, the key-tile axis is the loop inside a
// workgroup, and the (max, sum, value) reducer state is loop-carried).
//
// A workgroup holds NW waves and 32*NW query rows of one kv head. Rows are
// packed as r = sq*G + g, so the Hq/Hkv query heads that read the same kv
// head share every K/V tile the workgroup stages (replication by index,
// section 3.1). Each wave owns 32 rows and works on transposed tiles:
//
//   S^T[key][query] = K_tile (A operand, from LDS) * Q^T (B operand, registers)
//   O^T[d][query]  += V^T_tile (A operand, from LDS) * P^T (B operand, registers)
//
// with v_mfma_f32_32x32x16_bf16. In both products lane l owns query l % 32,
// so the row max, the exponentials, the row sum and the rescale of the
// carried value are lane-local; the score accumulator, converted to bf16, is
// already in the B-operand layout of the second product. Two lanes (l and
// l ^ 32) share a query and exchange one value per tile for the max.
//
// K/V tiles of 64 keys go HBM -> registers -> LDS with a double buffer: the
// loads of tile j+1 are in flight while tile j is multiplied. K is stored
// row-major with a 16-byte-chunk XOR swizzle; V is stored transposed (V^T)
// with its keys permuted so that each lane's 8 keys of a P^T fragment are
// contiguous, also XOR-swizzled against bank conflicts.
//
// The maximum used as the exponent reference is only moved up when a tile's
// maximum exceeds it by more than 8 (base-2 units), so the carried sum and
// value are rescaled rarely; weights stay below 2^8 and the final
// value / sum is unchanged (the repair h(c, s, s') = c * 2^(s - s') is exact
// for any reference point).
//
// In split mode the workgroup covers one key partition and stores the
// partition's (reference, sum, value) state instead of value / sum.
#include "ef_device.hpp"
#include "ef_kernels.hpp"

namespace ef {

namespace {

constexpr int BN = 64;             // keys per tile
constexpr float kLazyThreshold = 8.f;  // base-2 headroom before the reference moves

template <int D>
struct TileGeom {
  static constexpr int KCH = D / 8;                  // 16-byte chunks per K row
  static constexpr int K_BYTES = BN * D * 2;         // K tile
  static constexpr int V_BYTES = D * BN * 2;         // V^T tile
  static constexpr int STAGE = K_BYTES + V_BYTES;
};

__device__ __forceinline__ int swz_k(int row, int kch) { return row & (kch - 1); }
__device__ __forceinline__ int swz_v(int d) { return (d ^ (d >> 3)) & 7; }

// Slot of key kappa (0..63) inside a V^T row: swap bits 2 and 3 of kappa.
__device__ __forceinline__ int vslot(int kappa) {
  return (kappa & ~12) | ((kappa & 4) << 1) | ((kappa & 8) >> 1);
}

template <int D, int NW>
struct Loader {
  using G = TileGeom<D>;
  static constexpr int NT = NW * 64;
  static constexpr int K_CHUNKS = BN * G::KCH;          // 16-byte chunks per K tile
  static constexpr int K_PER_T = K_CHUNKS / NT;         // per thread
  static constexpr int V_GROUPS = (BN / 4) * G::KCH;    // (4 keys x 8 d) groups per V tile
  static constexpr int V_PER_T = (V_GROUPS + NT - 1) / NT;
  static_assert(K_CHUNKS % NT == 0, "K tile split");
  static_assert(V_GROUPS % NT == 0 || NT % V_GROUPS == 0, "V tile split");

  u32x4_t kreg[K_PER_T];
  u32x4_t vreg[V_PER_T][4];

  // Keys past the end of the range are clamped to the last valid key: the loads
  // stay unconditional (no divergent branch, so the compiler does not have to wait
  // for them before the compute that follows), the duplicated K rows are masked
  // out of the scores and the duplicated V rows meet a weight of exactly 0.
  __device__ __forceinline__ void load(const uint16_t* kh, const uint16_t* vh, int kb, int kend) {
    const int t = threadIdx.x;
    const int klast = kend - 1;
#pragma unroll
    for (int i = 0; i < K_PER_T; ++i) {
      const int id = t + i * NT;
      const int row = id / G::KCH, ch = id % G::KCH;
      const int key = min(kb + row, klast);
      kreg[i] = *reinterpret_cast<const u32x4_t*>(kh + (size_t)key * D + ch * 8);
    }
#pragma unroll
    for (int i = 0; i < V_PER_T; ++i) {
      const int gid = t + i * NT;
      const int ch = gid % G::KCH, kq = gid / G::KCH;
      if constexpr (V_GROUPS % NT != 0) {
        if (gid >= V_GROUPS) break;
      }
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int key = min(kb + kq * 4 + x, klast);
        vreg[i][x] = *reinterpret_cast<const u32x4_t*>(vh + (size_t)key * D + ch * 8);
      }
    }
  }

  __device__ __forceinline__ void store(char* stage) const {
    const int t = threadIdx.x;
    char* ks = stage;
    char* vs = stage + G::K_BYTES;
#pragma unroll
    for (int i = 0; i < K_PER_T; ++i) {
      const int id = t + i * NT;
      const int row = id / G::KCH, ch = id % G::KCH;
      *reinterpret_cast<u32x4_t*>(ks + row * (2 * D) + ((ch ^ swz_k(row, G::KCH)) << 4)) = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < V_PER_T; ++i) {
      const int gid = t + i * NT;
      const int ch = gid % G::KCH, kq = gid / G::KCH;
      if constexpr (V_GROUPS % NT != 0) {
        if (gid >= V_GROUPS) break;
      }
      const int slot = vslot(kq * 4);
      const u32x4_t x0 = vreg[i][0], x1 = vreg[i][1], x2 = vreg[i][2], x3 = vreg[i][3];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const uint32_t sel = half ? 0x07060302u : 0x05040100u;
          u32x2_t val;
          val[0] = __builtin_amdgcn_perm(x1[w], x0[w], sel);  // keys 0,1 at d
          val[1] = __builtin_amdgcn_perm(x3[w], x2[w], sel);  // keys 2,3 at d
          const int d = ch * 8 + w * 2 + half;
          const int chunk = (slot >> 3) ^ swz_v(d);
          *reinterpret_cast<u32x2_t*>(vs + d * (2 * BN) + (chunk << 4) + ((slot & 7) << 1)) = val;
        }
      }
    }
  }
};

// Occupancy target: two waves per SIMD for 4-wave workgroups (two workgroups per
// CU overlap each other's barrier and memory stalls); the 2-wave variant keeps
// its larger per-thread staging registers at one wave per SIMD.
template <int NW>
constexpr int kWavesPerEu = NW == 4 ? 2 : 1;

template <int D, int NW, bool NEG>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(kWavesPerEu<NW>)))
void attn_mfma_kernel(MfmaParams a) {
  using Geo = TileGeom<D>;
  constexpr int KSTEPS = D / 16;  // MFMA k-steps over the head dimension
  constexpr int DT = D / 32;      // 32-wide output tiles along D
  constexpr int BM = 32 * NW;
  extern __shared__ __align__(16) char smem[];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int h = lane >> 5;   // k-group of the MFMA operands
  const int ql = lane & 31;  // this lane's query inside the wave's 32 rows

  // Workgroup -> (row tile, partition, b*Hkv). Row tiles are visited last-first so
  // causal tiles with the most keys start first.
  const int mt = a.mtiles - 1 - (int)blockIdx.x;
  const int p = blockIdx.y;
  const int bh = blockIdx.z;
  const int b = bh / a.Hkv, hkv = bh % a.Hkv;

  const size_t kvhead = ((size_t)b * a.Hkv + hkv) * (size_t)a.Skv * D;
  const uint16_t* kh = a.k + kvhead;
  const uint16_t* vh = a.v + kvhead;

  // This lane's query row.
  const int r = mt * BM + wave * 32 + ql;
  const bool rvalid = r < a.R;
  const int sq = rvalid ? r / a.G : 0;
  const int g = rvalid ? r % a.G : 0;
  const size_t orow = (((size_t)b * a.Hq + (size_t)hkv * a.G + g) * a.Sq + sq);
  const int off = a.Skv - a.Sq;
  const int lim = !rvalid ? -1 : (a.causal ? sq + off : 0x7fffffff);

  // Key range of this workgroup: the partition, cut at the last key any row can see.
  int kbeg = p * a.T;
  int kend = min(kbeg + a.T, a.Skv);
  int lim_lo = 0x7fffffff, lim_hi = 0x7fffffff;
  if (a.causal) {
    const int r_lo = mt * BM;
    const int r_hi = min(mt * BM + BM, a.R) - 1;
    lim_lo = r_lo / a.G + off;
    lim_hi = r_hi / a.G + off;
    kend = min(kend, lim_hi + 1);
  }
  const int ntiles = kend > kbeg ? (kend - kbeg + BN - 1) / BN : 0;

  // Q^T fragments (B operand): lane holds q[row][16*s + 8*h .. +8].
  bf16x8_t qf[KSTEPS];
  {
    const u32x4_t* qp = reinterpret_cast<const u32x4_t*>(a.q + orow * D);
    const u32x4_t zero = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      u32x4_t x = rvalid ? qp[2 * s + h] : zero;
      qf[s] = __builtin_bit_cast(bf16x8_t, x);
    }
  }

  floatx16 oacc[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int j = 0; j < 16; ++j) oacc[i][j] = 0.f;
  float mref = kNegInf;  // reference maximum, base-2 units
  float lsum = 0.f;      // this lane's half of the row sum
  const float c = a.c_abs;

  Loader<D, NW> ld;
  if (ntiles > 0) {
    ld.load(kh, vh, kbeg, kend);
    ld.store(smem);
  }
  __syncthreads();

  for (int j = 0; j < ntiles; ++j) {
    const int kb = kbeg + j * BN;
    char* stage = smem + (j & 1) * Geo::STAGE;
    const bool more = j + 1 < ntiles;
    ld.load(kh, vh, kb + BN, kend);  // past the end: every key clamps to the last one

    // S^T = K * Q^T for two 32-key halves of the tile.
    floatx16 sacc[2];
    const char* ks = stage;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
      for (int i = 0; i < 16; ++i) sacc[half][i] = 0.f;
      const int krow = half * 32 + ql;
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
        const int ch = 2 * s + h;
        const u32x4_t kx = *reinterpret_cast<const u32x4_t*>(
            ks + krow * (2 * D) + ((ch ^ swz_k(krow, Geo::KCH)) << 4));
        sacc[half] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, kx), qf[s], sacc[half], 0, 0, 0);
      }
    }

    // Mask: keys past the range or past this row's causal limit.
    const bool need_mask = (kb + BN > kend) || (a.causal && kb + BN - 1 > lim_lo);
    float x[32];
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int i = 0; i < 16; ++i) x[half * 16 + i] = NEG ? -sacc[half][i] : sacc[half][i];
    if (need_mask) {
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kb + half * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
          if (key >= kend || key > lim) x[half * 16 + i] = kNegInf;
        }
    }
    float tmax = x[0];
#pragma unroll
    for (int i = 1; i < 32; ++i) tmax = fmaxf(tmax, x[i]);
    tmax = fmaxf(tmax, shfl_xor(tmax, 32));
    const float cand = tmax * c;  // tile maximum in base-2 units (c > 0)
    // Move the reference only when the tile exceeds it by the threshold.
    const bool up = cand > mref + kLazyThreshold;
    if (__builtin_amdgcn_ballot_w64(up)) {
      const float mnew = up ? cand : mref;
      const float rs = up ? exp2_fast(mref - mnew) : 1.f;  // 0 when mref = -inf
      mref = mnew;
      lsum *= rs;
#pragma unroll
      for (int i = 0; i < DT; ++i)
#pragma unroll
        for (int jj = 0; jj < 16; ++jj) oacc[i][jj] *= rs;
    }
    const float mneg = (mref == kNegInf) ? 0.f : -mref;
    float psum = 0.f;
    uint32_t pk[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float p0 = exp2_fast(fmaf(x[2 * i], c, mneg));
      const float p1 = exp2_fast(fmaf(x[2 * i + 1], c, mneg));
      psum += p0 + p1;
      pk[i] = pack_bf16x2(p0, p1);
    }
    lsum += psum;

    // O^T += V^T * P^T over the four 16-key steps of the tile.
    const char* vs = stage + Geo::K_BYTES;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      // P^T fragment: registers 8*(s%2) .. +8 of score half s/2, i.e. pk[4*s .. 4*s+3].
      const u32x4_t pv = {pk[4 * s], pk[4 * s + 1], pk[4 * s + 2], pk[4 * s + 3]};
      const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, pv);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int d = dt * 32 + ql;
        const int chunk = (2 * s + h) ^ swz_v(d);
        const u32x4_t vx = *reinterpret_cast<const u32x4_t*>(vs + d * (2 * BN) + (chunk << 4));
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vx), pf,
                                                          oacc[dt], 0, 0, 0);
      }
    }

    if (more) ld.store(smem + ((j + 1) & 1) * Geo::STAGE);
    __syncthreads();
  }

  // Row sum over both lane halves.
  const float ltot = lsum + shfl_xor(lsum, 32);
  if (!rvalid) return;
  if (a.ws_m == nullptr) {
    const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
    float* orp = a.o + orow * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = dt * 32 + 8 * q4 + 4 * h;
        float4 val = make_float4(oacc[dt][4 * q4] * inv, oacc[dt][4 * q4 + 1] * inv,
                                 oacc[dt][4 * q4 + 2] * inv, oacc[dt][4 * q4 + 3] * inv);
        *reinterpret_cast<float4*>(orp + d) = val;
      }
  } else {
    const size_t slot = orow * (size_t)a.P + p;
    if (h == 0) {
      // Reference in natural-log units, in terms of scale * q.k (sign restored).
      a.ws_m[slot] = (mref == kNegInf) ? kNegInf : mref * kLn2;
      a.ws_l[slot] = ltot;
    }
    float* ap = a.ws_acc + slot * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = dt * 32 + 8 * q4 + 4 * h;
        *reinterpret_cast<float4*>(ap + d) =
            make_float4(oacc[dt][4 * q4], oacc[dt][4 * q4 + 1], oacc[dt][4 * q4 + 2],
                        oacc[dt][4 * q4 + 3]);
      }
  }
}

template <int D, int NW>
hipError_t launch_nw(const MfmaParams& a, bool neg, hipStream_t stream) {
  const size_t lds = 2 * TileGeom<D>::STAGE;
  dim3 grid(a.mtiles, a.P, a.B * a.Hkv);
  if (neg) {
    hipLaunchKernelGGL((attn_mfma_kernel<D, NW, true>), grid, dim3(NW * 64), lds, stream, a);
  } else {
    hipLaunchKernelGGL((attn_mfma_kernel<D, NW, false>), grid, dim3(NW * 64), lds, stream, a);
  }
  return hipGetLastError();
}

}  // namespace

int mfma_rows_per_block(int R) { return R <= 64 ? 64 : 128; }

hipError_t launch_mfma_attention(const MfmaParams& a, bool neg, hipStream_t stream) {
  const int bm = a.mtiles > 0 ? mfma_rows_per_block(a.R) : 128;
  if (a.D == 128) {
    if (bm == 64) return launch_nw<128, 2>(a, neg, stream);
    return launch_nw<128, 4>(a, neg, stream);
  }
  if (bm == 64) return launch_nw<64, 2>(a, neg, stream);
  return launch_nw<64, 4>(a, neg, stream);
}

}  // namespace ef
