// Split-KV decode producer for few query rows per kv head (G*Sq <= 8).
//
// One workgroup owns (partition p, kv head, batch): it streams the partition's
// K and V rows from HBM exactly once with 128-bit loads and evaluates every
// query row that reads this kv head (grouped-query replication by index,
// section 3.1 "Replicate"). The rolling (max, sum, value) reducer of form M2
// (section 3, figure "attention-rewrites"; section 4.2 repair fusion) runs in
// registers, and the reduced state of the partition is stored for a later
// combine (section 3.3 "Collection"; section 4.4 storage rule).
//
// Lane layout: a key row of D bf16 is read by D/8 adjacent lanes, 16 bytes
// each, so one wave-wide load covers 64*16 contiguous bytes (4 rows at
// D = 128). Every lane keeps its 8-element slice of each query row; q.k is a
// packed-bf16 dot product followed by a DPP sum over the row's lanes, so all
// lanes of a row group end up with the full score. Each row group carries its
// own rolling state; the groups of a wave and the waves of the workgroup are
// merged with the same reducer at the end.
#include "ef_device.hpp"
#include "ef_kernels.hpp"
#include "group_combine.hpp"

namespace ef {

template <int D, int RMAX, int NW, int U, bool PF, bool NT = true, bool FUSED = false,
          bool LOCAL = false>
__global__ __launch_bounds__(NW * 64) void decode_split_kernel(DecodeParams a) {
  constexpr int LPR = D / 8;     // lanes per key row
  constexpr int TPL = 64 / LPR;  // key rows per wave-wide load
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int tl = lane / LPR;  // row slot inside a wave-wide load
  const int dc = lane % LPR;  // which 8-element slice of D this lane holds
  const int p = blockIdx.x, hkv = blockIdx.y, b = blockIdx.z;
  // Partition p covers virtual keys [t0, t1); with a window the virtual axis
  // skips the keys between the sink run and the window run.
  const int t0 = p * a.T;
  const int t1 = min(t0 + a.T, LOCAL ? a.runs.lv : a.Skv);
  const int la = a.runs.la, rshift = a.runs.bs - a.runs.la;
  auto key_of = [&](int vk) { return LOCAL ? (vk < la ? vk : vk + rshift) : vk; };
  const size_t kvhead = ((size_t)b * a.Hkv + hkv) * (size_t)a.Skv;
  const uint4* kp = reinterpret_cast<const uint4*>(a.k + kvhead * D) + dc;
  const uint4* vp = reinterpret_cast<const uint4*>(a.v + kvhead * D) + dc;
  // Query rows of this kv head are contiguous: row r = g*Sq + sq.
  const size_t row0 = ((size_t)b * a.Hq + (size_t)hkv * a.G) * (size_t)a.Sq;

  uint32_t qv[RMAX][4];
  int lim[RMAX];
#pragma unroll
  for (int r = 0; r < RMAX; ++r) {
    if (r < a.R) {
      uint4 x = reinterpret_cast<const uint4*>(a.q + (row0 + r) * D)[dc];
      qv[r][0] = x.x; qv[r][1] = x.y; qv[r][2] = x.z; qv[r][3] = x.w;
      lim[r] = a.causal ? (r % a.Sq) + a.Skv - a.Sq : 0x7fffffff;
    } else {
      qv[r][0] = qv[r][1] = qv[r][2] = qv[r][3] = 0u;
      lim[r] = -1;  // padding row: every key masked
    }
  }

  float m[RMAX], l[RMAX], acc[RMAX][8];
#pragma unroll
  for (int r = 0; r < RMAX; ++r) {
    m[r] = kNegInf;
    l[r] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[r][e] = 0.f;
  }

  const float c = a.c;  // scale * log2(e): scores are kept in base-2 units
  constexpr int STEP = NW * TPL;  // key rows per workgroup-wide load
  // Rows past the partition are clamped to its last row: the loads stay
  // unconditional and the duplicates are masked out of the scores. The rows of
  // the next iteration are requested before the current ones are used.
  const int tlast = t1 - 1;
  uint4 kn[U], vn[U];
  if constexpr (PF) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = key_of(min(t0 + (u * NW + wave) * TPL + tl, tlast));
      kn[u] = load16<NT>(kp + (size_t)t * LPR);
      vn[u] = load16<NT>(vp + (size_t)t * LPR);
    }
  }
  for (int tb = t0; tb < t1; tb += U * STEP) {
    uint4 kr[U], vr[U];
    int tok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      tok[u] = tb + (u * NW + wave) * TPL + tl;
      if constexpr (PF) {
        kr[u] = kn[u];
        vr[u] = vn[u];
      } else {
        const int t = key_of(min(tok[u], tlast));
        kr[u] = load16<NT>(kp + (size_t)t * LPR);
        vr[u] = load16<NT>(vp + (size_t)t * LPR);
      }
    }
    if constexpr (PF) {
      // Unconditional: past the end every row clamps to the partition's last row.
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = key_of(min(tb + U * STEP + (u * NW + wave) * TPL + tl, tlast));
        kn[u] = load16<NT>(kp + (size_t)t * LPR);
        vn[u] = load16<NT>(vp + (size_t)t * LPR);
      }
    }
    // Scores in base-2 units, masked to -inf where the key is not visible.
    float s[U][RMAX];
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int r = 0; r < RMAX; ++r) {
        float d = dot2_bf16(qv[r][0], kr[u].x, 0.f);
        d = dot2_bf16(qv[r][1], kr[u].y, d);
        d = dot2_bf16(qv[r][2], kr[u].z, d);
        d = dot2_bf16(qv[r][3], kr[u].w, d);
        d = group_sum<LPR>(d) * c;
        const int key = key_of(tok[u]);
        bool vis = tok[u] < t1 && key <= lim[r];
        if constexpr (LOCAL) vis = vis && (key > lim[r] - a.runs.window || key < a.runs.sinks);
        s[u][r] = vis ? d : kNegInf;
      }
    }
    float vf[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      vf[u][0] = bf16lo_to_f32(vr[u].x); vf[u][1] = bf16hi_to_f32(vr[u].x);
      vf[u][2] = bf16lo_to_f32(vr[u].y); vf[u][3] = bf16hi_to_f32(vr[u].y);
      vf[u][4] = bf16lo_to_f32(vr[u].z); vf[u][5] = bf16hi_to_f32(vr[u].z);
      vf[u][6] = bf16lo_to_f32(vr[u].w); vf[u][7] = bf16hi_to_f32(vr[u].w);
    }
    // Rolling update: next_max, rescale of the carried state, new weights.
#pragma unroll
    for (int r = 0; r < RMAX; ++r) {
      float bm = s[0][r];
#pragma unroll
      for (int u = 1; u < U; ++u) bm = fmaxf(bm, s[u][r]);
      const float mn = fmaxf(m[r], bm);
      const float ms = (mn == kNegInf) ? 0.f : mn;
      const float rs = exp2_fast(m[r] - ms);
      float psum = 0.f;
      float pw[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        pw[u] = exp2_fast(s[u][r] - ms);
        psum += pw[u];
      }
      l[r] = l[r] * rs + psum;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float x = acc[r][e] * rs;
#pragma unroll
        for (int u = 0; u < U; ++u) x = fmaf(pw[u], vf[u][e], x);
        acc[r][e] = x;
      }
      m[r] = mn;
    }
  }

  // Merge the row groups of the wave (lanes l and l ^ LPR*k hold the same D slice).
#pragma unroll
  for (int off = LPR; off < 64; off <<= 1) {
#pragma unroll
    for (int r = 0; r < RMAX; ++r) {
      const float mo = shfl_xor(m[r], off);
      const float lo = shfl_xor(l[r], off);
      const float mn = fmaxf(m[r], mo);
      const float ms = (mn == kNegInf) ? 0.f : mn;
      const float wa = exp2_fast(m[r] - ms), wb = exp2_fast(mo - ms);
      l[r] = l[r] * wa + lo * wb;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float ao = shfl_xor(acc[r][e], off);
        acc[r][e] = acc[r][e] * wa + ao * wb;
      }
      m[r] = mn;
    }
  }

  // Merge the waves through LDS and store the partition's state.
  __shared__ float sm[NW][RMAX], sl[NW][RMAX];
  __shared__ float sacc[NW][RMAX][D];
  if (tl == 0) {
#pragma unroll
    for (int r = 0; r < RMAX; ++r) {
      if (dc == 0) {
        sm[wave][r] = m[r];
        sl[wave][r] = l[r];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) sacc[wave][r][dc * 8 + e] = acc[r][e];
    }
  }
  __syncthreads();
  const int P = a.P;
  for (int idx = threadIdx.x; idx < a.R * D; idx += NW * 64) {
    const int r = idx / D, d = idx % D;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm[w][r]);
    const float ms = (M == kNegInf) ? 0.f : M;
    float L = 0.f, A = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float wt = exp2_fast(sm[w][r] - ms);
      L = fmaf(wt, sl[w][r], L);
      A = fmaf(wt, sacc[w][r][d], A);
    }
    const size_t slot = (row0 + r) * (size_t)P + p;
    const float mnat = (M == kNegInf) ? kNegInf : M * kLn2;  // natural-log units
    if constexpr (FUSED) {
      store_dev(&a.ws_acc[slot * D + d], A);  // read by another workgroup in this launch
      if (d == 0) {
        store_dev(&a.ws_m[slot], mnat);
        store_dev(&a.ws_l[slot], L);
      }
    } else {
      a.ws_acc[slot * D + d] = A;
      if (d == 0) {
        a.ws_m[slot] = mnat;
        a.ws_l[slot] = L;
      }
    }
  }

  if constexpr (FUSED) {
    // The last workgroup of this (batch, kv head) to store its state combines the
    // group's rows; every other workgroup is done.
    __shared__ float cw[RMAX * kFusedMaxP];
    __shared__ float cl[RMAX * kFusedMaxP];
    __shared__ float cinv[RMAX];
    if (!last_of_group(a.counters + (size_t)b * a.Hkv + hkv, P)) return;
    combine_group<D, NW * 64>(a.ws_m, a.ws_l, a.ws_acc, a.o, row0, a.R, P, cw, cl, cinv);
    if (threadIdx.x == 0) reset_counter(a.counters + (size_t)b * a.Hkv + hkv);
  }
}

// Launch shape by grid size (measured on the GQA decode and 131072-key
// workloads); local attention (window > 0) selects the variant that maps
// virtual keys onto the sink and window runs: a grid that fits the chip in one round runs best with 2-wave
// workgroups that request their next rows before using the current ones; a
// grid several rounds deep runs best with 4-wave workgroups and no prefetch.
template <int D, int RMAX, bool LOCAL>
static hipError_t launch_decode_rl(const DecodeParams& a, hipStream_t stream) {
  constexpr int U = RMAX <= 2 ? 4 : 2;
  const long long blocks = (long long)a.P * a.Hkv * a.B;
  dim3 grid(a.P, a.Hkv, a.B);
  const bool fused = a.counters != nullptr;
  if (blocks <= 2048) {
    if (fused) {
      hipLaunchKernelGGL((decode_split_kernel<D, RMAX, 2, U, true, true, true, LOCAL>), grid,
                         dim3(2 * 64), 0, stream, a);
    } else {
      hipLaunchKernelGGL((decode_split_kernel<D, RMAX, 2, U, true, true, false, LOCAL>), grid,
                         dim3(2 * 64), 0, stream, a);
    }
  } else {
    if (fused) {
      hipLaunchKernelGGL((decode_split_kernel<D, RMAX, 4, U, false, true, true, LOCAL>), grid,
                         dim3(4 * 64), 0, stream, a);
    } else {
      hipLaunchKernelGGL((decode_split_kernel<D, RMAX, 4, U, false, true, false, LOCAL>), grid,
                         dim3(4 * 64), 0, stream, a);
    }
  }
  return hipGetLastError();
}

template <int D, int RMAX>
static hipError_t launch_decode_r(const DecodeParams& a, hipStream_t stream) {
  return a.runs.window > 0 ? launch_decode_rl<D, RMAX, true>(a, stream)
                           : launch_decode_rl<D, RMAX, false>(a, stream);
}

template <int D>
static hipError_t launch_decode_d(const DecodeParams& a, hipStream_t stream) {
  if (a.R <= 1) return launch_decode_r<D, 1>(a, stream);
  if (a.R <= 2) return launch_decode_r<D, 2>(a, stream);
  if (a.R <= 4) return launch_decode_r<D, 4>(a, stream);
  return launch_decode_r<D, 8>(a, stream);
}

hipError_t launch_decode_split(const DecodeParams& a, hipStream_t stream) {
  return a.D == 128 ? launch_decode_d<128>(a, stream) : launch_decode_d<64>(a, stream);
}

}  // namespace ef
