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
// Lane layout: a key row of D bf16 is spread over LPR = D / (8 CH) adjacent
// lanes, each holding CH 16-byte chunks of it (chunks dc, dc + LPR, ...), so
// the CH loads of a wave read 64/LPR whole rows, each load whole 128-byte
// lines when LPR = 8. Every lane keeps the same chunks of each query row; q.k
// is a packed-bf16 dot product over the lane's chunks followed by a DPP sum
// over the row's lanes, so all lanes of a row group end up with the score.
//
// Loads go through buffer descriptors over the partition's rows (rows past
// it read as zero), two register sets deep. The arithmetic per key is kept
// small, since with a handful of waves per SIMD it does not hide entirely
// behind the loads:
//  - a negative scale is moved into q (bf16 negation is exact), so the
//    scale c is positive and the running maximum can be taken on raw q.k;
//  - the exponent reference moves only when a key exceeds it by more than
//    8 in base-2 units (the carried sum and value are rescaled then, which
//    keeps every weight below 2^8 and is exact for any reference point);
//  - p.V runs as packed-bf16 dot products over pairs of keys (one
//    instruction per value element and pair), with the weights rounded to
//    bf16 as the matrix-core kernel does; the sum l uses the fp32 weights.
// Each row group carries its own rolling state; the groups of a wave and the
// waves of the workgroup are merged with the same reducer at the end.
//
// Output-channel split (DS > 1; the N parallel refinement of the p.V product,
// section 4.1 and table "rules", which the paper's evaluation selects for
// one-sequence decode, section 7.2): DS
// workgroups share a partition. Each reads the partition's whole K rows and
// evaluates the same scores and softmax, but loads and accumulates only its
// D/DS value channels and writes only those. The reference point and sum it
// stores are bit-identical to the other slices' (same keys, same order), so
// the combine of a slice needs only its own slice's workgroups. With one
// partition and no workspace the workgroup writes o directly: no merge at all.
#include "ef_device.hpp"
#include "ef_kernels.hpp"
#include "group_combine.hpp"

namespace ef {

namespace {

constexpr float kMoveThreshold = 8.f;  // base-2 headroom before the reference moves
constexpr uint32_t kBufferFlags = 0x00020000u;  // raw 32-bit buffer access
constexpr int kNonTemporal = 2;                 // cache policy of streamed loads
constexpr int kDeviceScopeStore = 16;           // cache policy sc1: device-coherent store

// Pairs (x of key a, x of key b) of the bf16 elements 2w (lo) and 2w+1 (hi) of
// two packed words, for a packed-bf16 dot product over the two keys.
__device__ __forceinline__ uint32_t pair_lo(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ __forceinline__ uint32_t pair_hi(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

}  // namespace

// One partition p of the keys of kv head hkv of batch b, value channels
// [ds * D/DS, (ds + 1) * D/DS), by the NW waves of the calling workgroup.
template <int D, int RMAX, int NW, int U, int CH, bool FUSED, bool LOCAL, int DS>
__device__ __forceinline__ void decode_partition(const DecodeParams& a, const int p, const int hkv,
                                                 const int b, const int ds) {
  constexpr int LPR = D / (8 * CH);  // lanes per key row
  constexpr int TPL = 64 / LPR;      // key rows per wave-wide load
  constexpr int DL = 8 * CH;         // value elements per lane and row
  constexpr int DW = D / DS;         // value channels of this workgroup
  static_assert(U % 2 == 0, "keys are paired across the U slots");
  static_assert(DW % 8 == 0, "a channel slice holds whole 16-byte chunks");
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int tl = lane / LPR;  // row slot inside a wave-wide load
  const int dc = lane % LPR;  // first 16-byte chunk of the row this lane holds
  // Partition p covers virtual keys [t0, t1); with a window the virtual axis
  // skips the keys between the sink run and the window run.
  const int t0 = p * a.T;
  const int t1 = min(t0 + a.T, LOCAL ? a.runs.lv : a.Skv);
  const int la = a.runs.la, rshift = a.runs.bs - a.runs.la;
  auto key_of = [&](int vk) { return LOCAL ? (vk < la ? vk : vk + rshift) : vk; };
  const size_t kvhead = ((size_t)b * a.Hkv + hkv) * (size_t)a.Skv;
  // Buffer descriptors over the partition's rows (the whole head with a window,
  // whose partitions map onto two runs of keys): a row past the range reads as
  // zero without touching memory, so the loads need no clamping.
  // Byte counts and offsets stay below 2^32: a head holds fewer than 2^31 elements.
  const int rbase = LOCAL ? 0 : t0;
  const unsigned rbytes = (unsigned)(LOCAL ? a.Skv : t1 - t0) * (2u * D);
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.k + (kvhead + rbase) * D), (short)0, (int)rbytes, kBufferFlags);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.v + (kvhead + rbase) * D), (short)0, (int)rbytes, kBufferFlags);
  // Query rows of this kv head are contiguous: row r = g*Sq + sq.
  const size_t row0 = ((size_t)b * a.Hq + (size_t)hkv * a.G) * (size_t)a.Sq;
  // Value chunks of this lane inside the workgroup's channel slice; the others
  // are read at the buffer's end (zero, no memory access).
  bool vin[CH];
#pragma unroll
  for (int i = 0; i < CH; ++i) vin[i] = DS == 1 || ((dc + i * LPR) * 8) / DW == ds;

  // Positive scale: a negative one is moved into q. The floor keeps a zero
  // scale well defined (every visible key gets weight 1).
  const float c = fmaxf(fabsf(a.c), 1e-30f);
  const uint32_t qflip = a.c < 0.f ? 0x80008000u : 0u;
  const float thr = kMoveThreshold / c;  // reference headroom in raw q.k units

  u32x4_t qv[RMAX][CH];
  int lim[RMAX];
#pragma unroll
  for (int r = 0; r < RMAX; ++r) {
    if (r < a.R) {
      const u32x4_t* qp = reinterpret_cast<const u32x4_t*>(a.q + (row0 + r) * D) + dc;
#pragma unroll
      for (int i = 0; i < CH; ++i) qv[r][i] = qp[i * LPR] ^ qflip;
      lim[r] = a.causal ? (r % a.Sq) + a.Skv - a.Sq : 0x7fffffff;
    } else {
#pragma unroll
      for (int i = 0; i < CH; ++i) qv[r][i] = u32x4_t{0u, 0u, 0u, 0u};
      lim[r] = -1;  // padding row: every key masked
    }
  }
  // Whether every key of the partition is visible to every row (then only the
  // ragged end of the partition needs the mask).
  bool all_visible = !a.causal || a.Skv - a.Sq >= key_of(t1 - 1);
  if constexpr (LOCAL) all_visible = all_visible && key_of(t0) >= a.Skv - a.runs.window;
  all_visible = all_visible && a.R == RMAX;

  float m[RMAX], nmc[RMAX], l[RMAX], acc[RMAX][DL];
#pragma unroll
  for (int r = 0; r < RMAX; ++r) {
    m[r] = kNegInf;  // reference, raw q.k units
    nmc[r] = 0.f;    // -m * c (0 while m = -inf)
    l[r] = 0.f;
#pragma unroll
    for (int e = 0; e < DL; ++e) acc[r][e] = 0.f;
  }

  constexpr int STEP = NW * TPL;  // key rows per workgroup-wide load
  // Rows past the partition read as zero (their scores are masked).
  auto load_set = [&](u32x4_t (&kr)[U][CH], u32x4_t (&vr)[U][CH], int tb) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int tok = tb + (u * NW + wave) * TPL + tl;
      const unsigned row = LOCAL ? (tok < t1 ? key_of(tok) : a.Skv) : tok - t0;
      const unsigned off = row * (2u * D) + dc * 16u;
#pragma unroll
      for (int i = 0; i < CH; ++i) {
        kr[u][i] = __builtin_amdgcn_raw_buffer_load_b128(krs, off + i * LPR * 16, 0, kNonTemporal);
        vr[u][i] = __builtin_amdgcn_raw_buffer_load_b128(vrs, vin[i] ? off + i * LPR * 16 : rbytes,
                                                         0, kNonTemporal);
      }
    }
  };

  auto consume = [&](const u32x4_t (&kr)[U][CH], const u32x4_t (&vr)[U][CH], int tb) {
    // Raw scores q.k of this lane's key slots.
    float s[U][RMAX];
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int r = 0; r < RMAX; ++r) {
        float d = 0.f;
#pragma unroll
        for (int i = 0; i < CH; ++i)
#pragma unroll
          for (int w = 0; w < 4; ++w) d = dot2_bf16(qv[r][i][w], kr[u][i][w], d);
        s[u][r] = group_sum<LPR>(d);
      }
    }
    if (!all_visible || tb + U * STEP > t1) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int tok = tb + (u * NW + wave) * TPL + tl;
        const int key = key_of(tok);
#pragma unroll
        for (int r = 0; r < RMAX; ++r) {
          bool vis = tok < t1 && key <= lim[r];
          if constexpr (LOCAL) vis = vis && (key > lim[r] - a.runs.window || key < a.runs.sinks);
          s[u][r] = vis ? s[u][r] : kNegInf;
        }
      }
    }
    // Reference update, only where a key exceeds the reference by the threshold.
    float bm[RMAX];
    bool up = false;
#pragma unroll
    for (int r = 0; r < RMAX; ++r) {
      bm[r] = s[0][r];
#pragma unroll
      for (int u = 1; u < U; ++u) bm[r] = fmaxf(bm[r], s[u][r]);
      up = up || bm[r] > m[r] + thr;
    }
    if (__builtin_amdgcn_ballot_w64(up)) {
#pragma unroll
      for (int r = 0; r < RMAX; ++r) {
        const bool mv = bm[r] > m[r] + thr;
        const float rs = mv ? exp2_fast((m[r] - bm[r]) * c) : 1.f;  // 0 when m = -inf
        m[r] = mv ? bm[r] : m[r];
        nmc[r] = (m[r] == kNegInf) ? 0.f : -m[r] * c;
        l[r] *= rs;
#pragma unroll
        for (int e = 0; e < DL; ++e) acc[r][e] *= rs;
      }
    }
    // Value elements of key pairs (u, u+1), shared by all rows.
    uint32_t vlo[U / 2][CH][4], vhi[U / 2][CH][4];
#pragma unroll
    for (int h = 0; h < U / 2; ++h)
#pragma unroll
      for (int i = 0; i < CH; ++i)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          vlo[h][i][w] = pair_lo(vr[2 * h][i][w], vr[2 * h + 1][i][w]);
          vhi[h][i][w] = pair_hi(vr[2 * h][i][w], vr[2 * h + 1][i][w]);
        }
#pragma unroll
    for (int r = 0; r < RMAX; ++r) {
#pragma unroll
      for (int h = 0; h < U / 2; ++h) {
        const float p0 = exp2_fast(fmaf(s[2 * h][r], c, nmc[r]));
        const float p1 = exp2_fast(fmaf(s[2 * h + 1][r], c, nmc[r]));
        l[r] += p0 + p1;
        const uint32_t pk = pack_bf16x2(p0, p1);
#pragma unroll
        for (int i = 0; i < CH; ++i)
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            acc[r][i * 8 + 2 * w] = dot2_bf16(pk, vlo[h][i][w], acc[r][i * 8 + 2 * w]);
            acc[r][i * 8 + 2 * w + 1] = dot2_bf16(pk, vhi[h][i][w], acc[r][i * 8 + 2 * w + 1]);
          }
      }
    }
  };

  u32x4_t ka[U][CH], va[U][CH], kb[U][CH], vb[U][CH];
  // Two sets of registers alternate: the rows of the next two steps are in
  // flight while a step is used, each set reloaded right after its use. The
  // scheduling barriers keep the first two sets in issue order, so the wait
  // counts the loop relies on (the older set lands first) hold on entry as on
  // every turn.
  load_set(ka, va, t0);
  __builtin_amdgcn_sched_barrier(0);
  load_set(kb, vb, t0 + U * STEP);
  __builtin_amdgcn_sched_barrier(0);
  for (int tb = t0; tb < t1; tb += 2 * U * STEP) {
    consume(ka, va, tb);
    if (tb + U * STEP >= t1) break;
    load_set(ka, va, tb + 2 * U * STEP);
    consume(kb, vb, tb + U * STEP);
    load_set(kb, vb, tb + 3 * U * STEP);
  }

  // Reference in base-2 units of the scaled score for the merges below.
#pragma unroll
  for (int r = 0; r < RMAX; ++r) m[r] = (m[r] == kNegInf) ? kNegInf : m[r] * c;

  // Merge the row groups of the wave (lanes LPR, 2 LPR, ... apart hold the same
  // value elements of other keys): the row's largest reference over the groups
  // first, each lane's state scaled to it once, then plain sums. Every group
  // ends with the same merged state (each exchange combines the pair in the same
  // order on both sides, or with a commutative operation).
  float mx[RMAX];
#pragma unroll
  for (int r = 0; r < RMAX; ++r) mx[r] = m[r];
  auto max_over = [&](auto off_tag) {
    constexpr int OFF = decltype(off_tag)::value;
    if constexpr (OFF < 64) {
#pragma unroll
      for (int r = 0; r < RMAX; ++r) {
        float xa, xb;
        lane_pair<OFF>(mx[r], xa, xb);
        mx[r] = fmaxf(xa, xb);
      }
    }
  };
  auto sum_over = [&](auto off_tag) {
    constexpr int OFF = decltype(off_tag)::value;
    if constexpr (OFF < 64) {
#pragma unroll
      for (int r = 0; r < RMAX; ++r) {
        float xa, xb;
        lane_pair<OFF>(l[r], xa, xb);
        l[r] = xa + xb;
#pragma unroll
        for (int e = 0; e < DL; ++e) {
          lane_pair<OFF>(acc[r][e], xa, xb);
          acc[r][e] = xa + xb;
        }
      }
    }
  };
  max_over(std::integral_constant<int, LPR>{});
  max_over(std::integral_constant<int, 2 * LPR>{});
  max_over(std::integral_constant<int, 4 * LPR>{});
  max_over(std::integral_constant<int, 8 * LPR>{});
#pragma unroll
  for (int r = 0; r < RMAX; ++r) {
    const float ms = (mx[r] == kNegInf) ? 0.f : mx[r];
    const float w = exp2_fast(m[r] - ms);  // 0 for a group that saw no key
    l[r] *= w;
#pragma unroll
    for (int e = 0; e < DL; ++e) acc[r][e] *= w;
    m[r] = mx[r];
  }
  sum_over(std::integral_constant<int, LPR>{});
  sum_over(std::integral_constant<int, 2 * LPR>{});
  sum_over(std::integral_constant<int, 4 * LPR>{});
  sum_over(std::integral_constant<int, 8 * LPR>{});

  const int P = a.P;
  if constexpr (NW == 1) {
    // One wave: the lanes of row group 0 hold the partition's merged state (the
    // merge across waves below would weight it by exactly 1), so they store it
    // straight from registers, 16 bytes at a time; no LDS round trip, no barrier.
    if (tl == 0) {
#pragma unroll
      for (int r = 0; r < RMAX; ++r) {
        if (r >= a.R) break;
        const float M = m[r], L = l[r];
        const size_t slot = (row0 + r) * (size_t)P + p;
#pragma unroll
        for (int i = 0; i < CH; ++i) {
          if (!vin[i]) continue;
          const int d = (dc + i * LPR) * 8;  // first of this lane's 8 value channels
          const float* x = &acc[r][i * 8];
          if (!FUSED && a.ws_acc == nullptr) {
            // One partition, no workspace: the state is the row's result.
            const bool none = M == kNegInf || L == 0.f;
            float* op = a.o + (row0 + r) * D + d;
            *reinterpret_cast<float4*>(op) =
                none ? make_float4(0.f, 0.f, 0.f, 0.f)
                     : make_float4(x[0] / L, x[1] / L, x[2] / L, x[3] / L);
            *reinterpret_cast<float4*>(op + 4) =
                none ? make_float4(0.f, 0.f, 0.f, 0.f)
                     : make_float4(x[4] / L, x[5] / L, x[6] / L, x[7] / L);
            continue;
          }
          const float mnat = (M == kNegInf) ? kNegInf : M * kLn2;  // natural-log units
          // Every channel slice stores the row's reference and sum (the same values):
          // the combine of a slice waits only for that slice's workgroups.
          const bool first = d == ds * DW;
          if constexpr (FUSED) {
            // Read by another workgroup in this launch: device-scope stores into
            // the group's block of value states (at most 8 rows x 64 partitions).
            const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
                a.ws_acc + row0 * (size_t)P * D, (short)0, a.R * P * D * 4, kBufferFlags);
            const int off = ((r * P + p) * D + d) * 4;
            __builtin_amdgcn_raw_buffer_store_b128(
                u32x4_t{__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]),
                        __float_as_uint(x[3])},
                wrs, off, 0, kDeviceScopeStore);
            __builtin_amdgcn_raw_buffer_store_b128(
                u32x4_t{__float_as_uint(x[4]), __float_as_uint(x[5]), __float_as_uint(x[6]),
                        __float_as_uint(x[7])},
                wrs, off + 16, 0, kDeviceScopeStore);
            if (first) {
              store_dev(&a.ws_m[slot], mnat);
              store_dev(&a.ws_l[slot], L);
            }
          } else {
            float* ap = a.ws_acc + slot * D + d;
            *reinterpret_cast<float4*>(ap) = make_float4(x[0], x[1], x[2], x[3]);
            *reinterpret_cast<float4*>(ap + 4) = make_float4(x[4], x[5], x[6], x[7]);
            if (first) {
              a.ws_m[slot] = mnat;
              a.ws_l[slot] = L;
            }
          }
        }
      }
    }
  } else {
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
        for (int i = 0; i < CH; ++i)
#pragma unroll
          for (int e = 0; e < 8; ++e) sacc[wave][r][(dc + i * LPR) * 8 + e] = acc[r][i * 8 + e];
      }
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < a.R * DW; idx += NW * 64) {
      const int r = idx / DW, d = ds * DW + idx % DW;
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
      // Every channel slice stores the row's reference and sum (the same values):
      // the combine of a slice waits only for that slice's workgroups.
      const bool first = idx % DW == 0;
      if (!FUSED && a.ws_acc == nullptr) {
        // One partition, no workspace: the state is the row's result.
        a.o[(row0 + r) * D + d] = (M == kNegInf || L == 0.f) ? 0.f : A / L;
      } else if constexpr (FUSED) {
        store_dev(&a.ws_acc[slot * D + d], A);  // read by another workgroup in this launch
        if (first) {
          store_dev(&a.ws_m[slot], mnat);
          store_dev(&a.ws_l[slot], L);
        }
      } else {
        a.ws_acc[slot * D + d] = A;
        if (first) {
          a.ws_m[slot] = mnat;
          a.ws_l[slot] = L;
        }
      }
    }
  }

  if constexpr (FUSED) {
    // The last workgroup of this (batch, kv head) to store its state combines the
    // group's rows; every other workgroup is done.
    __shared__ float cw[RMAX * kFusedMaxP];
    __shared__ float cl[RMAX * kFusedMaxP];
    __shared__ float cinv[RMAX];
    unsigned* counter = a.counters + (((size_t)b * a.Hkv + hkv) * DS + ds) * kCounterStride;
    const unsigned ticket = arrival_ticket(counter);
    if (ticket >= (unsigned)P) {
      poison_group<D, DW, NW * 64>(a.o, row0, a.R, ds * DW);
      return;
    }
    if (ticket != (unsigned)(P - 1)) return;
    combine_group<D, DW, NW * 64, RMAX>(a.ws_m, a.ws_l, a.ws_acc, a.o, row0, a.R, P, cw, cl,
                                        cinv, ds * DW);
    if (threadIdx.x == 0) reset_counter(counter);
  }
}

// Grid: x = partition * DS + channel slice, y = kv head, z = batch.
template <int D, int RMAX, int NW, int U, int CH, bool FUSED, bool LOCAL, int DS>
__global__ __launch_bounds__(NW * 64) void decode_split_kernel(DecodeParams a) {
  decode_partition<D, RMAX, NW, U, CH, FUSED, LOCAL, DS>(a, blockIdx.x / DS, blockIdx.y,
                                                          blockIdx.z, blockIdx.x % DS);
}

// Launch shape per row count, measured on one-token decode with 1024
// workgroups of 256-key partitions (G = 1, 2, 4, 8) and on the 131072-key
// decode: one 16-byte chunk per lane and key row (16 lanes per row at
// D = 128; two chunks per lane cost more than the shorter reductions save),
// and the waves per workgroup and key slots per lane that ran fastest.
template <int RMAX>
constexpr int kWaves = (RMAX == 1 || RMAX == 4) ? 1 : 2;
template <int RMAX>
constexpr int kSlots = RMAX <= 2 ? 4 : 2;

template <int D, int RMAX, bool LOCAL, int DS>
static hipError_t launch_decode_rl(const DecodeParams& a, hipStream_t stream) {
  constexpr int NW = kWaves<RMAX>;
  constexpr int U = kSlots<RMAX>;
  dim3 grid(a.P * DS, a.Hkv, a.B);
  if (a.counters != nullptr) {
    hipLaunchKernelGGL((decode_split_kernel<D, RMAX, NW, U, 1, true, LOCAL, DS>), grid,
                       dim3(NW * 64), 0, stream, a);
  } else {
    hipLaunchKernelGGL((decode_split_kernel<D, RMAX, NW, U, 1, false, LOCAL, DS>), grid,
                       dim3(NW * 64), 0, stream, a);
  }
  return hipGetLastError();
}

template <int D, int RMAX>
static hipError_t launch_decode_r(const DecodeParams& a, hipStream_t stream) {
  if (a.runs.window > 0) return launch_decode_rl<D, RMAX, true, 1>(a, stream);
  switch (a.d_splits) {
    case 2: return launch_decode_rl<D, RMAX, false, 2>(a, stream);
    case 4: return launch_decode_rl<D, RMAX, false, 4>(a, stream);
    default: return launch_decode_rl<D, RMAX, false, 1>(a, stream);
  }
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
