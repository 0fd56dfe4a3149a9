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
// carried value are lane-local, and the score accumulator, converted to bf16,
// is already in the B-operand layout of the second product. Two lanes
// (l and l ^ 32) share a query and exchange one value per tile for the max.
//
// Software pipeline over tiles of BN keys (64, or 32 for the split producer
// of decode shapes, whose smaller stages let four workgroups share a compute
// unit): while the vector ALU turns tile j's
// scores into weights, the matrix core already computes tile j+1's scores,
// then tile j's values are multiplied. K is therefore staged one tile ahead
// of V: during step j, K stage (j+1)%2 holds K of tile j+1 and V stage j%2
// holds V of tile j, and the step loads K of tile j+2 and V of tile j+1 into
// the two stages nobody reads during it, so one workgroup barrier per tile
// suffices. Tiles go from HBM straight into LDS (direct loads, no staging
// registers), row-major with their 16-byte chunks permuted per row so that
// the fragment reads are free of bank conflicts. The V^T operand of the
// second product comes from transposing LDS reads (ds_read_b64_tr_b16) of the
// row-major V tile, in the key order of the P^T fragments.
//
// The maximum used as the exponent reference is only moved up when a tile's
// maximum exceeds it by more than 8 (base-2 units), so the carried sum and
// value are rescaled rarely; weights stay below 2^8 and the final
// value / sum is unchanged (the repair h(c, s, s') = c * 2^(s - s') is exact
// for any reference point).
//
// In split mode the workgroup covers one key partition and stores the
// partition's (reference, sum, value) state instead of value / sum.
//
// Local attention (a causal sliding window of W keys plus S sink keys; the
// sliding-window GQA and attention-sink layers of section 7.3) visits only
// the tiles some row of the workgroup can see: the tiles of the sink run
// [0, S) and those from the window start of the workgroup's first row to its
// causal end. Both runs feed the same rolling reducer, so the sink and window
// keys share one softmax normalisation; the keys in between are never read.
//
// Differential attention (section 7.3), single pass: the launch for the first
// branch finds the second branch's output in o, and its epilogue forms
// y = A1 - lambda * A2 from the carried value, mixes in lambda from the four
// learned vectors, RMS-normalises the row over D (the two lanes of a query
// hold its two halves) and writes the result, so A1 never reaches HBM.
#include <atomic>

#include "diff_norm.hpp"
#include "ef_device.hpp"
#include "ef_kernels.hpp"

namespace ef {

namespace {

constexpr float kLazyThreshold = 8.f;  // base-2 headroom before the reference moves
constexpr unsigned kXcds = 8;                   // accelerator dies of the chip

// Geometry of a BN-key tile (BN = 64, or 32 for the decode-shaped split
// producer, whose smaller stages let four workgroups share a compute unit).
template <int D, int BN>
struct TileGeom {
  static constexpr int KCH = D / 8;        // 16-byte chunks per row
  static constexpr int ROW = 2 * D;        // bytes per K or V row (no padding: swizzled)
  static constexpr int RPI = 64 / KCH;     // rows one wave-wide direct load fills
  static constexpr int TILE_BYTES = BN * ROW;
  // LDS: V stage 0, V stage 1, K stage 0, K stage 1 (all immediates < 64 KiB).
  static constexpr int V_OFF0 = 0;
  static constexpr int V_OFF1 = TILE_BYTES;
  static constexpr int K_OFF0 = 2 * TILE_BYTES;
  static constexpr int K_OFF1 = 3 * TILE_BYTES;
  static constexpr int LDS_BYTES = 4 * TILE_BYTES;
  template <int S>
  static constexpr int v_off() { return S == 0 ? V_OFF0 : V_OFF1; }
  template <int S>
  static constexpr int k_off() { return S == 0 ? K_OFF0 : K_OFF1; }
  // Tiles sit row-major in LDS with their 16-byte chunks permuted per row
  // (chunk c of row r at slot c ^ swz(r)), so the fragment reads below hit
  // distinct banks: K rows are read 16 rows at a time at one chunk, V rows four
  // rows at a time at 32 consecutive bytes (transposing reads).
  static __device__ __forceinline__ int swz_k(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
  static __device__ __forceinline__ int swz_v(int r) {
    return D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1);
  }
};

// Cross-half exchange: max of x over lanes l and l ^ 32.
__device__ __forceinline__ float max_with_other_half(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Key tiles of one workgroup, in visiting order: `na` tiles of the sink run
// starting at key a0 (keys below aend), then the tiles of the window run
// starting at b0 (keys below bend). Without a window the sink run is empty and
// the window run is the whole key range. Tiles past the last one cover no key.
template <int BN>
struct TileList {
  int a0, aend, na, b0, bend, n;
  int full_lo;  // a tile whose last key is at most this is below every row's causal limit
  int win_lo;   // a tile starting at or above this key lies in every row's window
  int sinks;    // keys below this are visible whatever the window
  __device__ __forceinline__ int base(int j) const {
    return j < na ? a0 + j * BN : b0 + (j - na) * BN;
  }
  __device__ __forceinline__ int end(int j) const { return j < na ? aend : bend; }
  // Whether some key of tile j is hidden from some row of the workgroup.
  __device__ __forceinline__ bool masked(int j) const {
    const int kb = base(j);
    return kb + BN > end(j) || kb + BN - 1 > full_lo || (kb < win_lo && kb + BN > sinks);
  }
};

// Tiles go straight from HBM to LDS (one 16-byte chunk per lane and load,
// each wave-wide load filling RPI whole rows): no staging registers and no
// LDS stores. Rows past the tile's run repeat its last row (their keys are
// masked, their values finite); a tile past the last one loads nothing.
//
// Cache policy: the split producer of decode shapes (32-key tiles, one row
// tile per kv head) reads every key exactly once, so its loads are
// non-temporal and stream past the caches, which lifts its read rate by
// about a sixth; the other launches keep the default policy, under which
// the row tiles of one kv head share its K/V tiles through the XCD's L2.
template <bool STREAM>
__device__ __forceinline__ void load_chunk(const uint16_t* g, char* l) {
  if constexpr (STREAM)
    __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)l, 16, 0,
                                     2 /* non-temporal */);
  else
    __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)l, 16, 0, 0);
}

template <int D, int NW, int BN>
struct Loader {
  using G = TileGeom<D, BN>;
  static constexpr int INSTS = BN / G::RPI / NW;  // direct loads per wave and tile
  static_assert(INSTS * G::RPI * NW == BN, "tile split over the waves");
  int row[INSTS];       // tile row whose chunk this lane loads
  int kchunk[INSTS];    // element offset of that chunk in a K row
  int vchunk[INSTS];    // element offset of that chunk in a V row
  unsigned koff[INSTS];  // byte offset of this lane's K chunk from the tile's first row
  unsigned voff[INSTS];  // the same for V
  int wave;              // wave index, uniform (scalar)

  __device__ __forceinline__ void init() {
    const int lane = threadIdx.x & 63;
    wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int i = 0; i < INSTS; ++i) {
      const int blk = wave + NW * i;
      row[i] = blk * G::RPI + lane / G::KCH;
      const int slot = lane % G::KCH;
      kchunk[i] = (slot ^ G::swz_k(row[i])) * 8;
      vchunk[i] = (slot ^ G::swz_v(row[i])) * 8;
      koff[i] = (unsigned)(row[i] * D + kchunk[i]) * 2u;
      voff[i] = (unsigned)(row[i] * D + vchunk[i]) * 2u;
    }
  }

  // The address is a uniform base (the tile's first row) plus a 32-bit lane
  // offset, so the vector ALU only clamps rows of a ragged tile.
  template <bool ISK>
  __device__ __forceinline__ void load(char* stage, const uint16_t* head, int kb, int kend) const {
    const int nrows = kend - kb;
    if (nrows <= 0) return;
    const char* base = reinterpret_cast<const char*>(head + (size_t)kb * D);
    if (nrows >= BN) {
#pragma unroll
      for (int i = 0; i < INSTS; ++i) {
        char* l = stage + (wave + NW * i) * 1024;
        const uint16_t* g = reinterpret_cast<const uint16_t*>(base + (ISK ? koff[i] : voff[i]));
        load_chunk<BN == 32>(g, l);
      }
    } else {
#pragma unroll
      for (int i = 0; i < INSTS; ++i) {
        const int r = min(row[i], nrows - 1);
        const unsigned off = (unsigned)(r * D + (ISK ? kchunk[i] : vchunk[i])) * 2u;
        char* l = stage + (wave + NW * i) * 1024;
        const uint16_t* g = reinterpret_cast<const uint16_t*>(base + off);
        load_chunk<BN == 32>(g, l);
      }
    }
  }
  template <int S>
  __device__ __forceinline__ void load_k(char* smem, const uint16_t* kh, int kb, int kend) const {
    load<true>(smem + G::template k_off<S>(), kh, kb, kend);
  }
  template <int S>
  __device__ __forceinline__ void load_v(char* smem, const uint16_t* vh, int kb, int kend) const {
    load<false>(smem + G::template v_off<S>(), vh, kb, kend);
  }
};

// Waits for this wave's direct-to-LDS loads (they count as vector memory loads).
__device__ __forceinline__ void wait_tile_loads() { __builtin_amdgcn_s_waitcnt(0x0f70); }

// Occupancy target: two waves per SIMD for 4-wave workgroups (two workgroups per
// CU overlap each other's barrier and latency stalls) and for 2-wave workgroups
// of 32-key tiles (four per CU); the 2-wave variant with 64-key tiles keeps its
// larger per-thread staging registers at one wave per SIMD.
template <int NW, int BN>
constexpr int kWavesPerEu = (NW == 4 || BN == 32) ? 2 : 1;

template <int D, bool NEG, int BN>
struct Tile {
  using Geo = TileGeom<D, BN>;
  static constexpr int KSTEPS = D / 16;  // MFMA k-steps over the head dimension
  static constexpr int DT = D / 32;      // 32-wide output tiles along D
  static constexpr int HALVES = BN / 32;  // 32-key halves of a tile
  static constexpr int PK = BN / 4;       // packed bf16 weight pairs per lane

  // S^T of the key tile in K stage S: 32-key halves, 16-deep MFMA k-steps.
  template <int S>
  static __device__ __forceinline__ void scores(const char* smem, const int* kread,
                                                const bf16x8_t* qf, floatx16* sacc) {
#pragma unroll
    for (int half = 0; half < HALVES; ++half)
#pragma unroll
      for (int i = 0; i < 16; ++i) sacc[half][i] = 0.f;
    if constexpr (HALVES == 1) {
      // One 32-key half: each K fragment has registers of its own, so the reads
      // can run several products ahead (the compiler issues them in two
      // batches) rather than one product ahead.
      u32x4_t kx[KSTEPS];
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s)
        kx[s] = *reinterpret_cast<const u32x4_t*>(smem + Geo::template k_off<S>() + kread[s]);
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s)
        sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kx[s]),
                                                         qf[s], sacc[0], 0, 0, 0);
    } else {
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
#pragma unroll
        for (int half = 0; half < HALVES; ++half) {
          const u32x4_t kx = *reinterpret_cast<const u32x4_t*>(
              smem + Geo::template k_off<S>() + kread[s] + half * 32 * Geo::ROW);
          sacc[half] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, kx), qf[s], sacc[half], 0, 0, 0);
        }
      }
    }
  }

  // Scores in exponent-ready form (sign applied, hidden keys at -inf) and the
  // rolling reference update; returns -reference (0 while nothing is visible).
  // A key is hidden from this lane's row when it is past the tile's run, past
  // the causal limit `lim`, or at most `lo` (left of the window) and not a sink.
  // The scores are rewritten in place.
  static __device__ __forceinline__ float prepare(floatx16* x, floatx16* oacc, float& lsum,
                                                  float& mref, float c, int kb, int kend,
                                                  bool masked, int lim, int lo, int sinks,
                                                  int h) {
    if constexpr (NEG) {
#pragma unroll
      for (int half = 0; half < HALVES; ++half)
#pragma unroll
        for (int i = 0; i < 16; ++i) x[half][i] = -x[half][i];
    }
    if (masked) {
      // Element i of half `half` holds key base + o(i) with a compile-time offset o.
      // The hidden keys become per-lane offset thresholds, clamped to the tile so the
      // arithmetic cannot overflow: past `vis` (the run's end or the causal limit), and
      // inside [wlo, whi] (left of the window, not a sink). Selects, not branches.
      const int base = kb + 4 * h;
      const int vis = min(min(kend - 1, lim), kb + BN) - base;
      const int wlo = max(sinks, kb) - base;
      const int whi = min(max(lo, kb - 1), kb + BN) - base;
      if (__builtin_amdgcn_ballot_w64(whi >= wlo)) {
#pragma unroll
        for (int half = 0; half < HALVES; ++half)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int o = half * 32 + 8 * (i >> 2) + (i & 3);
            const bool hide = (o > vis) | ((o >= wlo) & (o <= whi));
            x[half][i] = hide ? kNegInf : x[half][i];
          }
      } else {
#pragma unroll
        for (int half = 0; half < HALVES; ++half)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int o = half * 32 + 8 * (i >> 2) + (i & 3);
            x[half][i] = o > vis ? kNegInf : x[half][i];
          }
      }
    }
    float tmax = fmaxf(x[0][0], x[0][1]);
#pragma unroll
    for (int i = 2; i < 16 * HALVES; ++i) tmax = fmaxf(tmax, x[i >> 4][i & 15]);
    tmax = max_with_other_half(tmax);
    const float cand = tmax * c;  // tile maximum in base-2 units (c > 0)
    // Move the reference only when the tile exceeds it by the threshold.
    const bool up = cand > mref + kLazyThreshold;
    if (__builtin_amdgcn_ballot_w64(up)) {
      const float rs = up ? exp2_fast(mref - cand) : 1.f;  // 0 when mref = -inf
      mref = up ? cand : mref;
      lsum *= rs;
#pragma unroll
      for (int i = 0; i < DT; ++i)
#pragma unroll
        for (int jj = 0; jj < 16; ++jj) oacc[i][jj] *= rs;
    }
    return (mref == kNegInf) ? 0.f : -mref;
  }

  // Weights 2^(x*c - reference) as bf16 pairs (P^T fragments) and their row
  // sum in fp32. (A packed bf16 dot product with (1, 1) per pair would sum the
  // rounded weights in half the instructions, but between matrix products it
  // costs about ten cycles each; the two sums differ by far less than the
  // rounding of the weights themselves.)
  static __device__ __forceinline__ void weights(const floatx16* x, float c, float mneg,
                                                 uint32_t* pk, float& lsum) {
    float ps[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < PK; ++i) {
      const float p0 = exp2_fast(fmaf(x[(2 * i) >> 4][(2 * i) & 15], c, mneg));
      const float p1 = exp2_fast(fmaf(x[(2 * i + 1) >> 4][(2 * i + 1) & 15], c, mneg));
      pk[i] = pack_bf16x2(p0, p1);
      ps[i & 3] += p0 + p1;
    }
    lsum += (ps[0] + ps[1]) + (ps[2] + ps[3]);
  }

  // O^T += V^T * P^T over the 16-key steps of the tile in V stage S. The
  // V^T operand (8 keys of one value column per lane) comes from two
  // transposing reads of 4 keys each out of the row-major V tile.
  template <int S>
  static __device__ __forceinline__ void values(const char* smem, const int* vread,
                                                const uint32_t* pk, floatx16* oacc) {
    if constexpr (BN == 32) {
      values_asm<S>(smem, vread, pk, oacc);
    } else {
      typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
#pragma unroll
      for (int s = 0; s < BN / 16; ++s) {
        // P^T fragment: registers 8*(s%2) .. +8 of score half s/2, i.e. pk[4*s .. 4*s+3].
        const u32x4_t pv = {pk[4 * s], pk[4 * s + 1], pk[4 * s + 2], pk[4 * s + 3]};
        const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, pv);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const char* p = smem + Geo::template v_off<S>() + vread[dt] + 16 * s * Geo::ROW;
          const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (__attribute__((address_space(3))) bf16x4_t*)(p));
          const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (__attribute__((address_space(3))) bf16x4_t*)(p + 8 * Geo::ROW));
          const bf16x8_t vx = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vx, pf, oacc[dt], 0, 0, 0);
        }
      }
    }
  }

  // values() of a 32-key tile with the transposing reads issued from assembly:
  // the compiler cannot tell them from the direct-to-LDS loads into the other
  // stages still in flight, and waits for every outstanding load before the
  // first of them, which leaves the step's loads only its first half to land.
  // The reads of 16-key step s + 1 are requested before the products of step
  // s; LDS operations complete in order, so before step s's products a wait
  // until at most step s + 1's reads are outstanding suffices (other
  // operations counted by the same counter only make it longer). An empty
  // statement that rewrites the operands after the wait keeps the products
  // below it. (With 64-key tiles the extra registers this holds would spill.)
  template <int S>
  static __device__ __forceinline__ void values_asm(const char* smem, const int* vread,
                                                    const uint32_t* pk, floatx16* oacc) {
    constexpr int STEPS = BN / 16;
    constexpr int READS = 2 * DT;  // reads per 16-key step
    static_assert(READS <= 15, "outstanding reads exceed the LDS counter");
    const unsigned base = (unsigned)(uintptr_t)(
        (const __attribute__((address_space(3))) char*)(smem + Geo::template v_off<S>()));
    u32x2_t lo[2][DT], hi[2][DT];
    auto read_step = [&](int s, u32x2_t(&l)[DT], u32x2_t(&h)[DT]) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const unsigned addr = base + vread[dt] + 16 * s * Geo::ROW;
        asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(l[dt]) : "v"(addr));
        asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2"
                     : "=v"(h[dt])
                     : "v"(addr), "i"(8 * Geo::ROW));
      }
    };
    read_step(0, lo[0], hi[0]);
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int b = s & 1;
      if (s + 1 < STEPS) {
        read_step(s + 1, lo[b ^ 1], hi[b ^ 1]);
        asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(READS) : "memory");
      } else {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) asm volatile("" : "+v"(lo[b][dt]), "+v"(hi[b][dt]));
      // P^T fragment: registers 8*(s%2) .. +8 of score half s/2, i.e. pk[4*s .. 4*s+3].
      const u32x4_t pv = {pk[4 * s], pk[4 * s + 1], pk[4 * s + 2], pk[4 * s + 3]};
      const bf16x8_t pf = __builtin_bit_cast(bf16x8_t, pv);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const u32x4_t vx = {lo[b][dt][0], lo[b][dt][1], hi[b][dt][0], hi[b][dt][1]};
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vx), pf,
                                                          oacc[dt], 0, 0, 0);
      }
    }
  }
};

// One pipelined step on tile j (stage parity S = j % 2). On entry sacc[S] holds
// S^T of tile j, K stage 1-S holds tile j+1 and V stage S holds tile j. The
// step requests K of tile j+2 (into K stage S, last read for tile j's scores)
// and V of tile j+1 (into V stage 1-S, last read for tile j-1's values)
// straight into LDS, computes tile j's weights while the matrix core computes
// tile j+1's scores, multiplies tile j's values, and waits for its loads
// before the workgroup barrier.
template <int D, int NW, bool NEG, int S, int BN>
__device__ __forceinline__ void pipelined_step(
    char* smem, const Loader<D, NW, BN>& ld, const uint16_t* kh, const uint16_t* vh,
    const TileList<BN>& tl, int j, int lim, int lo, int h, const int* kread, const int* vread,
    const bf16x8_t* qf, floatx16 (*sacc)[BN / 32], floatx16* oacc, float& lsum, float& mref,
    float c) {
  using TileT = Tile<D, NEG, BN>;
  ld.template load_k<S>(smem, kh, tl.base(j + 2), tl.end(j + 2));  // nothing past the last tile
  ld.template load_v<1 - S>(smem, vh, tl.base(j + 1), tl.end(j + 1));
  const float mneg = TileT::prepare(sacc[S], oacc, lsum, mref, c, tl.base(j), tl.end(j),
                                    tl.masked(j), lim, lo, tl.sinks, h);
  uint32_t pk[TileT::PK];
  TileT::weights(sacc[S], c, mneg, pk, lsum);
  // Tile j+1's scores go to the other accumulator pair, so tile j's stay in place.
  TileT::template scores<1 - S>(smem, kread, qf, sacc[1 - S]);
  TileT::template values<S>(smem, vread, pk, oacc);
  wait_tile_loads();
  __syncthreads();
}

template <int D, int NW, bool NEG, bool DIFF, int BN>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(kWavesPerEu<NW, BN>)))
void attn_mfma_kernel(MfmaParams a) {
  using Geo = TileGeom<D, BN>;
  using TileT = Tile<D, NEG, BN>;
  constexpr int KSTEPS = TileT::KSTEPS;
  constexpr int DT = TileT::DT;
  constexpr int BM = 32 * NW;
  extern __shared__ __align__(16) char smem[];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int h = lane >> 5;   // k-group of the MFMA operands
  const int ql = lane & 31;  // this lane's query inside the wave's 32 rows

  // Workgroup -> (row tile, partition, b*Hkv). Workgroups are dispatched to the
  // chip's 8 XCDs round-robin by linear id; the id is remapped so that each XCD
  // receives a contiguous run of kv heads, and all row tiles of a head, which
  // read the same K/V, share one XCD's L2. Row tiles are visited last-first so
  // causal tiles with the most keys start first.
  const unsigned nwg = gridDim.x * gridDim.y * gridDim.z;
  unsigned lin = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  if (nwg % kXcds == 0) lin = (lin % kXcds) * (nwg / kXcds) + lin / kXcds;
  const int mt = a.mtiles - 1 - (int)(lin % gridDim.x);
  const int p = (int)((lin / gridDim.x) % gridDim.y);
  const int bh = (int)(lin / (gridDim.x * gridDim.y));
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
  const int W = a.runs.window;
  const int lo = W > 0 ? lim - W : INT_MIN;  // keys at or left of lo are outside the window

  // Key tiles of this workgroup. The partition is a range [v0, v1) of the
  // virtual key axis (the sink run [0, la) followed by the window run from key
  // bs); its part in each run is cut at the last key any row can see and, in
  // the window run, at the first key of the earliest row's window.
  TileList<BN> tl;
  {
    const int la = a.runs.la, bs = a.runs.bs;
    const int v0 = p * a.T;
    const int v1 = min(v0 + a.T, a.runs.lv);
    int cend = 0x7fffffff, wbeg = 0;
    tl.full_lo = 0x7fffffff;
    tl.win_lo = INT_MIN;
    if (a.causal) {
      const int r_lo = mt * BM;
      const int r_hi = min(mt * BM + BM, a.R) - 1;
      tl.full_lo = r_lo / a.G + off;
      cend = r_hi / a.G + off + 1;
      if (W > 0) {
        wbeg = max(0, tl.full_lo - W + 1) / BN * BN;
        tl.win_lo = r_hi / a.G + off - W + 1;
      }
    }
    tl.a0 = v0;
    tl.aend = min(min(v1, la), cend);
    tl.na = tl.aend > tl.a0 ? (tl.aend - tl.a0 + BN - 1) / BN : 0;
    tl.b0 = max(bs + max(v0, la) - la, wbeg);
    tl.bend = min(bs + v1 - la, cend);
    tl.n = tl.na + (tl.bend > tl.b0 ? (tl.bend - tl.b0 + BN - 1) / BN : 0);
    tl.sinks = W > 0 ? a.runs.sinks : 0;
  }
  const int ntiles = tl.n;

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
  // The floor keeps a zero scale well defined: every visible key gets weight 1
  // (2^(x c) rounds to 1 for any finite score), while a hidden key's -inf stays
  // -inf instead of becoming -inf * 0 = NaN.
  const float c = fmaxf(a.c_abs, 1e-30f);
  // Per-lane LDS byte offsets of the fragment reads inside a stage: K row ql,
  // chunk 2s + h of k-step s; and, per 32-column tile dt of V^T, the
  // transposing-read pointer of this lane (row 4(lane/32) + (lane%16)/4 of a
  // 16-key step, 8 bytes at column 32 dt + 16 ((lane/16)%2) + 4 (lane%4)).
  int kread[KSTEPS];
#pragma unroll
  for (int s = 0; s < KSTEPS; ++s) kread[s] = ql * Geo::ROW + ((2 * s + h) ^ Geo::swz_k(ql)) * 16;
  int vread[DT];
  {
    const int j16 = lane & 15, grp = lane >> 4;
    const int vr = 4 * (grp >> 1) + (j16 >> 2);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int d_off = 32 * dt + 16 * (grp & 1) + 4 * (j16 & 3);
      vread[dt] = vr * Geo::ROW + (((d_off >> 3) ^ Geo::swz_v(vr)) * 16) + 2 * (d_off & 7);
    }
  }

  // Prologue: K and V of tile 0 into stage 0, K of tile 1 into K stage 1, then
  // tile 0's scores; the second barrier orders those K reads before stage 0 is
  // rewritten by the first pipelined step.
  Loader<D, NW, BN> ld;
  ld.init();
  floatx16 sacc[2][BN / 32];  // S^T of the current and the next tile
  if (ntiles > 0) {
    ld.template load_k<0>(smem, kh, tl.base(0), tl.end(0));
    ld.template load_v<0>(smem, vh, tl.base(0), tl.end(0));
    ld.template load_k<1>(smem, kh, tl.base(1), tl.end(1));
  }
  wait_tile_loads();
  __syncthreads();
  if (ntiles > 0) TileT::template scores<0>(smem, kread, qf, sacc[0]);
  __syncthreads();

  for (int j = 0; j < ntiles; j += 2) {
    pipelined_step<D, NW, NEG, 0, BN>(smem, ld, kh, vh, tl, j, lim, lo, h, kread, vread, qf,
                                      sacc, oacc, lsum, mref, c);
    if (j + 1 < ntiles)
      pipelined_step<D, NW, NEG, 1, BN>(smem, ld, kh, vh, tl, j + 1, lim, lo, h, kread, vread,
                                        qf, sacc, oacc, lsum, mref, c);
  }

  // Row sum over both lane halves.
  const float ltot = lsum + __shfl_xor(lsum, 32, 64);
  if constexpr (DIFF) {
    // Differential attention, first branch (section 7.3): mix with the second
    // branch's output already in o and normalise the row. Lanes l and l ^ 32
    // hold the two halves of a row.
    const float lam = diff_lambda(a.diff, lane, D);
    const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
    const float* prev = a.o + orow * D;
    float ss = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = dt * 32 + 8 * q4 + 4 * h;
        const float4 a2 = rvalid ? *reinterpret_cast<const float4*>(prev + d)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
        const float a2v[4] = {a2.x, a2.y, a2.z, a2.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float y = fmaf(-lam, a2v[e], oacc[dt][4 * q4 + e] * inv);
          oacc[dt][4 * q4 + e] = y;
          ss = fmaf(y, y, ss);
        }
      }
    const float rn = diff_row_factor(a.diff, ss + __shfl_xor(ss, 32, 64), D);
    if (!rvalid) return;
    float* orp = a.o + orow * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = dt * 32 + 8 * q4 + 4 * h;
        const float4 gw = *reinterpret_cast<const float4*>(a.diff.gamma + d);
        *reinterpret_cast<float4*>(orp + d) =
            make_float4(rn * gw.x * oacc[dt][4 * q4], rn * gw.y * oacc[dt][4 * q4 + 1],
                        rn * gw.z * oacc[dt][4 * q4 + 2], rn * gw.w * oacc[dt][4 * q4 + 3]);
      }
    return;
  }
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

template <int D, int NW, bool NEG, bool DIFF, int BN>
hipError_t launch_one(const MfmaParams& a, hipStream_t stream) {
  const size_t lds = TileGeom<D, BN>::LDS_BYTES;
  auto kern = attn_mfma_kernel<D, NW, NEG, DIFF, BN>;
  // More than 64 KiB of LDS per workgroup needs the attribute, which belongs to
  // the kernel on one device: set once per device (ids below 64 are
  // remembered, higher ones set it on every launch).
  static std::atomic<unsigned long long> lds_set{0};
  int dev = 0;
  const hipError_t de = hipGetDevice(&dev);
  if (de != hipSuccess) return de;
  const unsigned long long bit = (dev >= 0 && dev < 64) ? 1ull << dev : 0ull;
  if (bit == 0 || (lds_set.load(std::memory_order_acquire) & bit) == 0) {
    const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (attr != hipSuccess) return attr;
    lds_set.fetch_or(bit, std::memory_order_acq_rel);
  }
  dim3 grid(a.mtiles, a.P, a.B * a.Hkv);
  hipLaunchKernelGGL(kern, grid, dim3(NW * 64), lds, stream, a);
  return hipGetLastError();
}

template <int D, int NW, int BN>
hipError_t launch_nw(const MfmaParams& a, bool neg, hipStream_t stream) {
  if (a.diff.gamma != nullptr)
    return neg ? launch_one<D, NW, true, true, BN>(a, stream)
               : launch_one<D, NW, false, true, BN>(a, stream);
  return neg ? launch_one<D, NW, true, false, BN>(a, stream)
             : launch_one<D, NW, false, false, BN>(a, stream);
}

}  // namespace

hipError_t launch_mfma_attention(const MfmaParams& a, bool neg, hipStream_t stream) {
  const int bm = a.bm;
  if (bm != 64 && bm != 128) return hipErrorInvalidValue;
  // The split producer with one row tile per kv head (decode shapes) runs
  // 32-key tiles, whose non-temporal loads assume every key is read once.
  const bool small = bm == 64 && a.mtiles == 1 && a.ws_m != nullptr;
  if (a.D == 128) {
    if (small) return launch_nw<128, 2, 32>(a, neg, stream);
    if (bm == 64) return launch_nw<128, 2, 64>(a, neg, stream);
    return launch_nw<128, 4, 64>(a, neg, stream);
  }
  if (small) return launch_nw<64, 2, 32>(a, neg, stream);
  if (bm == 64) return launch_nw<64, 2, 64>(a, neg, stream);
  return launch_nw<64, 4, 64>(a, neg, stream);
}

}  // namespace ef
