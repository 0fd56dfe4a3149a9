// Host side of the C ABI declared in include/ef_attention.h: argument
// validation (synchronous, before anything is enqueued), kernel selection,
// grid and workspace arithmetic.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "ef_attention.h"
#include "ef_device.hpp"
#include "ef_kernels.hpp"

namespace {

constexpr int kTileKeys = 64;        // key tile of the kernels; partitions are multiples of it
constexpr int kDecodeMaxRows = 8;    // the VALU split producer handles G*Sq <= 8 ...
constexpr int kDecodeValuRows = 4;   // ... and the split-KV paths give it G*Sq <= 4 (the MFMA
                                     // producer streams faster with more rows)
constexpr int kMaxGridYZ = 65535;
static_assert(ef::kCounterRegionBytes == EF_COUNTER_REGION_BYTES,
              "the counter region of the header is the kernels' one");

struct Shape {
  int B, Hq, Hkv, Sq, Skv, D;
  long long rows() const { return (long long)B * Hq * Sq; }
};

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

ef_status check_shape(const Shape& s) {
  if (s.B < 0 || s.Sq < 0 || s.Skv < 0 || s.Hq < 1 || s.Hkv < 1) return EF_ERR_INVALID_SHAPE;
  if (s.Hq % s.Hkv != 0) return EF_ERR_GQA_RATIO;
  if (s.D != 64 && s.D != 128) return EF_ERR_UNSUPPORTED_HEAD_DIM;
  // Per-head extents stay below 2^31 elements; batch*heads fits the grid.
  if ((long long)s.Sq * s.D >= (1LL << 31) || (long long)s.Skv * s.D >= (1LL << 31))
    return EF_ERR_INVALID_SHAPE;
  if ((long long)s.B * s.Hkv > kMaxGridYZ || (long long)(s.Hq / s.Hkv) * s.Sq >= (1LL << 31))
    return EF_ERR_INVALID_SHAPE;
  return EF_OK;
}

ef_status check_io(const Shape& s, const void* q, const void* k, const void* v, const float* o,
                   float scale) {
  if (!std::isfinite(scale)) return EF_ERR_INVALID_SCALE;
  if (s.rows() == 0) return EF_OK;
  if (q == nullptr || o == nullptr) return EF_ERR_NULL_POINTER;
  if (s.Skv > 0 && (k == nullptr || v == nullptr)) return EF_ERR_NULL_POINTER;
  if (misaligned(q) || misaligned(o) || misaligned(k) || misaligned(v)) return EF_ERR_MISALIGNED;
  return EF_OK;
}

// Visible key runs of a (batch, kv head) for a causal window of `window` keys
// and `sinks` sink keys (section 7.3). Every key of every query row lies in
// the sink run [0, la) or the window run [bs, Skv): bs is the first key of the
// earliest row's window (row 0, diagonal Skv - Sq) rounded down to a tile, la
// the sink count rounded up to one. The split producers partition the
// concatenation of the two runs (lv keys). A window of at least Skv keys hides
// nothing beyond the causal mask and is dropped.
ef::KeyRuns key_runs(int Sq, int Skv, int window, int sinks) {
  ef::KeyRuns r{0, 0, Skv, 0, 0};
  if (window <= 0 || window >= Skv) return r;
  const int sk = sinks < Skv ? sinks : Skv;
  int la = (sk + kTileKeys - 1) / kTileKeys * kTileKeys;
  if (la > Skv) la = Skv;
  long long ws = (long long)Skv - Sq - window + 1;  // window start of row 0
  if (ws < 0) ws = 0;
  int bs = (int)(ws / kTileKeys * kTileKeys);
  if (bs < la) bs = la;
  r.la = la;
  r.bs = bs;
  r.lv = la + (Skv - bs);
  r.window = window;
  r.sinks = sk;
  return r;
}

// Roofline model of one split-KV call with T keys per partition (section 6.2,
// over the legal schedules, minimise the largest work/throughput ratio over
// the modelled resources). Resources: HBM (K/V, q, o and the partial states
// written and read back) and the streaming time of one workgroup (T keys of K
// and V, or the fewer keys its rows can see, at that workgroup's rate, times
// the rounds of workgroups the chip holds); the combine follows (inside the producer for up to 64 partitions,
// else a second kernel). The rates were fitted to partition-size sweeps of
// twelve decode shapes on MI355X (1 to 64 query rows per kv head, 1K to 128K
// keys): the VALU producer streams 6.5 TB/s over the chip and 27.6, 51.1 or
// 10.3 GB/s per workgroup for 1, 2 or 4 query rows per kv head (one, two and
// one waves), plus 5 us per round; the combine inside it costs 4.4 us per 16
// partitions, the combine kernel 8.9 us plus its reads. The MFMA producer
// streams 5.85 TB/s over the chip and 9.9 GB/s per wave, plus 1 us per round,
// and its combine kernel costs 13.4 us plus its reads. 2048 waves are resident.
// The chip's rate is reached only with enough waves streaming at once: under
// load a wave draws about 16 GB/s (VALU) or 8.5 GB/s (MFMA), counted over the
// waves weighted by their share of the keys (a short last partition adds
// little).
constexpr double kHbmValuBytesPerUs = 6.5e6;
constexpr double kHbmMfmaBytesPerUs = 5.85e6;
constexpr double kWgValuBytesPerUs[3] = {27.6e3, 51.1e3, 10.3e3};  // 1, 2, 4 rows
constexpr double kWaveMfmaBytesPerUs = 9.9e3;
constexpr double kLoadedWaveValuBytesPerUs = 16.0e3;
constexpr double kLoadedWaveMfmaBytesPerUs = 8.5e3;
constexpr double kResidentWaves = 2048.0;
constexpr double kRoundValuUs = 5.0;
constexpr double kRoundMfmaUs = 1.0;
constexpr double kFusedCombineUsPer16 = 4.4;
constexpr double kCombineValuUs = 8.9;
constexpr double kCombineMfmaUs = 13.4;

// Rows per workgroup of the matrix-core kernel (section 6.2). The legal
// schedules hold 64 or 128 query rows of one kv head (two or four waves of 32
// rows). Each is charged an optimistic time, the larger of its matrix work over
// the bf16 peak and its global-memory traffic over the HBM peak, and the
// fastest is taken; with equal times, the one with less matrix work. Matrix
// work counts the rows padded to whole workgroups; traffic counts the K/V that
// every row tile stages (each re-read in full: the L2 is not credited) plus q
// and o once. `keys`: the keys a row tile streams.
constexpr double kMfmaPeakFlopsPerUs = 2.5e9;
constexpr double kHbmPeakBytesPerUs = 8.0e6;

int rows_per_block(const Shape& s, double keys) {
  const double R = (double)(s.Hq / s.Hkv) * s.Sq;
  const double kv_heads = (double)s.B * s.Hkv;
  int best = 0;
  double best_us = 0.0, best_flops = 0.0;
  for (const int bm : {64, 128}) {
    const double tiles = std::ceil(R / bm);
    const double flops = kv_heads * tiles * bm * keys * 4.0 * s.D;
    const double bytes = kv_heads * tiles * keys * 4.0 * s.D + (double)s.rows() * s.D * 6.0;
    const double us = std::max(flops / kMfmaPeakFlopsPerUs, bytes / kHbmPeakBytesPerUs);
    if (best == 0 || us < best_us || (us == best_us && flops < best_flops)) {
      best = bm;
      best_us = us;
      best_flops = flops;
    }
  }
  return best;
}

double split_model_us(const Shape& s, int keys, int T, int visible) {
  const int G = s.Hq / s.Hkv;
  const int R = G * s.Sq;
  const double P = std::ceil((double)keys / T);
  const double Tk = std::min<double>(T, keys);
  // A workgroup streams at most the keys its rows can see, however long its partition.
  const double Twg = std::min<double>(Tk, visible);
  const bool valu = R <= kDecodeValuRows;
  double nw, wg_per_part, wg_rate;
  if (valu) {
    const int bucket = R <= 1 ? 0 : R <= 2 ? 1 : 2;
    nw = bucket == 1 ? 2 : 1;  // waves per workgroup of the VALU producer
    wg_per_part = 1;
    wg_rate = kWgValuBytesPerUs[bucket];
  } else {
    const int bm = rows_per_block(s, std::min<double>(T, visible));
    nw = bm / 32;
    wg_per_part = std::ceil((double)R / bm);
    wg_rate = kWaveMfmaBytesPerUs * nw;
  }
  const double kv_heads = (double)s.B * s.Hkv;
  const double rows = (double)s.B * s.Hq * s.Sq;
  const double kv_bytes = kv_heads * keys * s.D * 4.0;
  const double io_bytes = rows * s.D * 6.0;
  const double state_bytes = rows * P * (s.D + 2) * 4.0;
  const double hbm = valu ? kHbmValuBytesPerUs : kHbmMfmaBytesPerUs;
  const double waves = kv_heads * P * wg_per_part * nw;
  const double waves_eff = kv_heads * wg_per_part * nw * keys / Tk;
  const double hbm_eff =
      std::min(hbm, std::min(waves_eff, kResidentWaves) *
                        (valu ? kLoadedWaveValuBytesPerUs : kLoadedWaveMfmaBytesPerUs));
  const double r_hbm = (kv_bytes + io_bytes + 2.0 * state_bytes) / hbm_eff;
  const double rounds = std::ceil(waves / kResidentWaves);
  const double r_wg =
      rounds * (Twg * s.D * 4.0 / wg_rate + (valu ? kRoundValuUs : kRoundMfmaUs));
  const bool fused = valu && P <= ef::kFusedMaxP && kv_heads <= ef::kCounterSlots;
  const double combine = fused ? kFusedCombineUsPer16 * std::ceil(P / 16.0)
                               : state_bytes / hbm + (valu ? kCombineValuUs : kCombineMfmaUs);
  return std::max(r_hbm, r_wg) + combine;
}

// Candidate partition sizes for a key axis of `keys` keys: 64, 128, 192, 256,
// 384, 512, ... (powers of two times 64 and 1.5 times them), up to one
// partition holding every key; at most 65535 partitions.
std::vector<int> partition_candidates(int keys) {
  std::vector<int> out;
  const long long top = ((long long)std::max(keys, 1) + kTileKeys - 1) / kTileKeys * kTileKeys;
  // Powers of two times the tile: sizes in between leave a ragged last
  // partition on power-of-two contexts and measured slower than both neighbours.
  for (long long t = kTileKeys; t < top; t *= 2)
    if ((keys + t - 1) / t <= kMaxGridYZ) out.push_back((int)t);
  out.push_back((int)top);
  std::sort(out.begin(), out.end());
  out.erase(std::unique(out.begin(), out.end()), out.end());
  return out;
}

// The most keys of the virtual key axis the rows of one workgroup can see: the
// whole axis without a window; with one, the sink run plus the union of the
// rows' windows. A workgroup of the matrix-core producer holds the rows of
// ceil(BM / G) query positions (rows are packed r = sq*G + g), one of the vector
// producer all Sq of them. A window run cut into partitions leaves each row
// tile most of its keys in one partition, so splitting it shortens no
// workgroup's stream (attention-sink prefill: 1024 positions, a 5,123-key run,
// 4,228 keys per row tile).
int visible_keys(const Shape& s, const ef::KeyRuns& runs) {
  if (runs.window <= 0) return runs.lv;
  const int G = s.Hq / s.Hkv;
  const int R = G * s.Sq;
  const int pos = R <= kDecodeValuRows
                      ? s.Sq
                      : std::min(s.Sq, (rows_per_block(s, runs.lv) + G - 1) / G);
  const long long v = (long long)runs.window + runs.sinks + pos;
  return (int)std::min<long long>(runs.lv, v);
}

// Keys per partition of a key axis of `keys` keys (the visible runs' length):
// the caller's choice, else the candidate the model rates fastest.
int resolve_partition(const Shape& s, int keys, int partition_size, int visible) {
  if (partition_size > 0) return partition_size;
  if (keys <= 0) return kTileKeys;
  int best = kTileKeys;
  double best_us = 1e300;
  for (int t : partition_candidates(keys)) {
    const double us = split_model_us(s, keys, t, visible);
    if (us < best_us) {
      best_us = us;
      best = t;
    }
  }
  return best;
}

ef_status check_mask(int window, int sinks) {
  return (window < 1 || sinks < 0) ? EF_ERR_INVALID_MASK : EF_OK;
}

struct WsLayout {
  size_t m_off, l_off, acc_off, cnt_off, bytes;
};

// Counters first (a region of fixed size, see kCounterRegionBytes), then the
// partial states.
WsLayout ws_layout(long long rows, long long P, int D) {
  WsLayout w;
  const size_t a = ef::ws_align256((size_t)(rows * P) * sizeof(float));
  w.cnt_off = 0;
  w.m_off = ef::kCounterRegionBytes;
  w.l_off = w.m_off + a;
  w.acc_off = w.m_off + 2 * a;
  w.bytes = w.acc_off + ef::ws_align256((size_t)(rows * P) * (size_t)D * sizeof(float));
  return w;
}

// Whether the producer combines the states itself: few query rows per kv head
// (the vector producer), few partitions, and a counter slot for every group.
bool fused_combine(const Shape& s, long long P, int d_splits) {
  return ((long long)(s.Hq / s.Hkv) * s.Sq <= kDecodeValuRows || d_splits > 0) &&
         P <= ef::kFusedMaxP &&
         (long long)s.B * s.Hkv * std::max(d_splits, 1) <= ef::kCounterSlots;
}

ef_status from_hip(hipError_t e) { return e == hipSuccess ? EF_OK : EF_ERR_HIP; }

ef_status launch_mfma(const Shape& s, const void* q, const void* k, const void* v, float* o,
                      float* ws_m, float* ws_l, float* ws_acc, int T, int P, float scale,
                      int causal, const ef::KeyRuns& runs, hipStream_t stream,
                      const ef::DiffParams* diff = nullptr) {
  ef::MfmaParams a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.o = o;
  a.ws_m = ws_m;
  a.ws_l = ws_l;
  a.ws_acc = ws_acc;
  a.B = s.B; a.Hq = s.Hq; a.Hkv = s.Hkv; a.Sq = s.Sq; a.Skv = s.Skv; a.D = s.D;
  a.G = s.Hq / s.Hkv;
  a.R = a.G * s.Sq;
  a.T = T;
  a.P = P;
  a.bm = rows_per_block(s, std::min(T, runs.lv));
  a.mtiles = (a.R + a.bm - 1) / a.bm;
  a.c_abs = std::fabs(scale) * ef::kLog2e;
  a.causal = causal ? 1 : 0;
  a.runs = runs;
  if (diff != nullptr) a.diff = *diff;
  return from_hip(ef::launch_mfma_attention(a, scale < 0.f, stream));
}

}  // namespace

extern "C" {

int ef_abi_version(void) { return EF_ABI_VERSION; }

const char* ef_status_string(int status) {
  switch (status) {
    case EF_OK: return "ok";
    case EF_ERR_NULL_POINTER: return "a required pointer is NULL";
    case EF_ERR_INVALID_SHAPE: return "invalid shape (negative size, Hq or Hkv < 1, or too large)";
    case EF_ERR_GQA_RATIO: return "Hq is not a multiple of Hkv";
    case EF_ERR_UNSUPPORTED_HEAD_DIM: return "head dimension must be 64 or 128";
    case EF_ERR_MISALIGNED: return "a pointer is not 16-byte aligned";
    case EF_ERR_INVALID_PARTITION:
      return "partition_size must be 0 or a positive multiple of 64 giving at most 65535 "
             "partitions";
    case EF_ERR_WORKSPACE_TOO_SMALL: return "workspace is NULL or too small";
    case EF_ERR_INVALID_SCALE: return "scale is not finite";
    case EF_ERR_HIP: return "HIP error while enqueueing work";
    case EF_ERR_INVALID_MASK: return "window must be >= 1 and sinks >= 0";
    case EF_ERR_INVALID_DIFF: return "lambda_init and eps must be finite and eps >= 0";
    case EF_ERR_INVALID_SPLIT:
      return "d_splits must be 1, 2 or 4, with at most 8 query rows per kv head";
    case EF_ERR_SCRATCH_TOO_SMALL:
      return "the problem needs more workspace than the library's static scratch holds";
    default: return "unknown status";
  }
}

}  // extern "C"

namespace {

ef_status fwd_impl(const Shape& s, const void* q, const void* k, const void* v, float* o,
                   float scale, int causal, const ef::KeyRuns& runs, void* stream) {
  ef_status st = check_shape(s);
  if (st != EF_OK) return st;
  st = check_io(s, q, k, v, o, scale);
  if (st != EF_OK) return st;
  if (s.rows() == 0) return EF_OK;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (s.Skv == 0) return from_hip(ef::launch_zero_fill(o, (size_t)s.rows() * s.D, hs));
  return launch_mfma(s, q, k, v, o, nullptr, nullptr, nullptr, runs.lv, 1, scale, causal, runs,
                     hs);
}

// The split-KV entry points reject more partitions than the grid takes; the
// size queries report such arguments as invalid (0) too.
int partition_size_impl(const Shape& s, const ef::KeyRuns& runs, int partition_size) {
  if (check_shape(s) != EF_OK) return 0;
  if (partition_size < 0 || partition_size % kTileKeys != 0) return 0;
  const int T = resolve_partition(s, runs.lv, partition_size, visible_keys(s, runs));
  if ((runs.lv + (long long)T - 1) / T > kMaxGridYZ) return 0;
  return T;
}

size_t workspace_size_impl(const Shape& s, const ef::KeyRuns& runs, int partition_size) {
  if (check_shape(s) != EF_OK) return 0;
  if (partition_size < 0 || partition_size % kTileKeys != 0) return 0;
  if (s.rows() == 0 || s.Skv == 0) return 0;
  const int T = resolve_partition(s, runs.lv, partition_size, visible_keys(s, runs));
  const long long P = (runs.lv + (long long)T - 1) / T;
  if (P > kMaxGridYZ) return 0;
  return ws_layout(s.rows(), P, s.D).bytes;
}

}  // namespace

extern "C" {

ef_status ef_attention_fwd(const void* q, const void* k, const void* v, float* o, int B, int Hq,
                           int Hkv, int Sq, int Skv, int D, float scale, int causal,
                           void* stream) {
  return fwd_impl(Shape{B, Hq, Hkv, Sq, Skv, D}, q, k, v, o, scale, causal,
                  key_runs(Sq, Skv, 0, 0), stream);
}

ef_status ef_attention_fwd_local(const void* q, const void* k, const void* v, float* o, int B,
                                 int Hq, int Hkv, int Sq, int Skv, int D, float scale, int window,
                                 int sinks, void* stream) {
  const Shape s{B, Hq, Hkv, Sq, Skv, D};
  ef_status st = check_shape(s);
  if (st != EF_OK) return st;
  st = check_mask(window, sinks);
  if (st != EF_OK) return st;
  return fwd_impl(s, q, k, v, o, scale, 1, key_runs(Sq, Skv, window, sinks), stream);
}

int ef_attention_splitkv_partition_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                        int partition_size) {
  return partition_size_impl(Shape{B, Hq, Hkv, Sq, Skv, D}, key_runs(Sq, Skv, 0, 0),
                             partition_size);
}

size_t ef_attention_splitkv_workspace_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                           int partition_size) {
  return workspace_size_impl(Shape{B, Hq, Hkv, Sq, Skv, D}, key_runs(Sq, Skv, 0, 0),
                             partition_size);
}

int ef_attention_splitkv_local_partition_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                              int window, int sinks, int partition_size) {
  if (check_mask(window, sinks) != EF_OK) return 0;
  return partition_size_impl(Shape{B, Hq, Hkv, Sq, Skv, D}, key_runs(Sq, Skv, window, sinks),
                             partition_size);
}

size_t ef_attention_splitkv_local_workspace_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                                 int window, int sinks, int partition_size) {
  if (check_mask(window, sinks) != EF_OK) return 0;
  return workspace_size_impl(Shape{B, Hq, Hkv, Sq, Skv, D}, key_runs(Sq, Skv, window, sinks),
                             partition_size);
}

}  // extern "C"

namespace {

// Validation shared by the split-KV entry points; on success fills the
// partition count and the workspace pointers.
ef_status split_prepare(const Shape& s, const void* q, const void* k, const void* v,
                        const float* o, float scale, const ef::KeyRuns& runs,
                        int partition_size, void* workspace, size_t workspace_bytes, int* T_out,
                        int* P_out, float** ws_m, float** ws_l, float** ws_acc,
                        unsigned** counters) {
  ef_status st = check_shape(s);
  if (st != EF_OK) return st;
  if (partition_size < 0 || partition_size % kTileKeys != 0) return EF_ERR_INVALID_PARTITION;
  st = check_io(s, q, k, v, o, scale);
  if (st != EF_OK) return st;
  *T_out = 0;
  *P_out = 0;
  if (s.rows() == 0 || s.Skv == 0) return EF_OK;
  const int T = resolve_partition(s, runs.lv, partition_size, visible_keys(s, runs));
  const long long P = (runs.lv + (long long)T - 1) / T;
  if (P > kMaxGridYZ) return EF_ERR_INVALID_PARTITION;
  const WsLayout w = ws_layout(s.rows(), P, s.D);
  if (workspace == nullptr || workspace_bytes < w.bytes) return EF_ERR_WORKSPACE_TOO_SMALL;
  if (misaligned(workspace)) return EF_ERR_MISALIGNED;
  char* ws = static_cast<char*>(workspace);
  *ws_m = reinterpret_cast<float*>(ws + w.m_off);
  *ws_l = reinterpret_cast<float*>(ws + w.l_off);
  *ws_acc = reinterpret_cast<float*>(ws + w.acc_off);
  *counters = reinterpret_cast<unsigned*>(ws + w.cnt_off);
  *T_out = T;
  *P_out = (int)P;
  return EF_OK;
}

// Stores the partition states; with `counters` and `o` given (decode path only),
// the last workgroup of each (batch, kv head) also combines them into o.
// d_splits = 0 lets the row count choose the producer; d_splits >= 1 asks for
// the VALU producer with that many output-channel slices.
ef_status split_produce(const Shape& s, const void* q, const void* k, const void* v, float scale,
                        int causal, const ef::KeyRuns& runs, int T, int P, float* ws_m,
                        float* ws_l, float* ws_acc, unsigned* counters, float* o,
                        hipStream_t hs, int d_splits = 0) {
  const int G = s.Hq / s.Hkv;
  const int R = G * s.Sq;
  if (d_splits > 0 || R <= kDecodeValuRows) {
    ef::DecodeParams a{};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.ws_m = ws_m;
    a.ws_l = ws_l;
    a.ws_acc = ws_acc;
    a.B = s.B; a.Hq = s.Hq; a.Hkv = s.Hkv; a.Sq = s.Sq; a.Skv = s.Skv; a.D = s.D;
    a.G = G;
    a.R = R;
    a.T = T;
    a.P = P;
    a.c = scale * ef::kLog2e;
    a.causal = causal ? 1 : 0;
    a.counters = counters;
    a.o = o;
    a.runs = runs;
    a.d_splits = d_splits > 0 ? d_splits : 1;
    return from_hip(ef::launch_decode_split(a, hs));
  }
  return launch_mfma(s, q, k, v, nullptr, ws_m, ws_l, ws_acc, T, P, scale, causal, runs, hs);
}

ef_status splitkv_impl(const Shape& s, const void* q, const void* k, const void* v, float* o,
                       float scale, int causal, const ef::KeyRuns& runs, int partition_size,
                       void* workspace, size_t workspace_bytes, void* stream) {
  int T = 0, P = 0;
  float *ws_m = nullptr, *ws_l = nullptr, *ws_acc = nullptr;
  unsigned* counters = nullptr;
  ef_status st = split_prepare(s, q, k, v, o, scale, runs, partition_size, workspace,
                               workspace_bytes, &T, &P, &ws_m, &ws_l, &ws_acc, &counters);
  if (st != EF_OK || s.rows() == 0) return st;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (s.Skv == 0) return from_hip(ef::launch_zero_fill(o, (size_t)s.rows() * s.D, hs));
  if (fused_combine(s, P, 0))
    return split_produce(s, q, k, v, scale, causal, runs, T, P, ws_m, ws_l, ws_acc, counters, o,
                         hs);
  st = split_produce(s, q, k, v, scale, causal, runs, T, P, ws_m, ws_l, ws_acc, nullptr, nullptr,
                     hs);
  if (st != EF_OK) return st;
  ef::CombineParams c{};
  c.m = ws_m;
  c.l = ws_l;
  c.acc = ws_acc;
  c.o = o;
  c.rows = (int)s.rows();
  c.P = P;
  c.D = s.D;
  return from_hip(ef::launch_combine(c, hs));
}

}  // namespace

namespace ef {

// ef_attention_splitkv over a caller-chosen workspace, for the library's other
// entry points (the allocation-free variant passes its static scratch).
ef_status splitkv_into(const void* q, const void* k, const void* v, float* o, int B, int Hq,
                       int Hkv, int Sq, int Skv, int D, float scale, int causal,
                       int partition_size, void* workspace, size_t workspace_bytes,
                       void* stream) {
  return splitkv_impl(Shape{B, Hq, Hkv, Sq, Skv, D}, q, k, v, o, scale, causal,
                      key_runs(Sq, Skv, 0, 0), partition_size, workspace, workspace_bytes,
                      stream);
}

}  // namespace ef

extern "C" {

ef_status ef_attention_splitkv_partials(const void* q, const void* k, const void* v, int B,
                                        int Hq, int Hkv, int Sq, int Skv, int D, float scale,
                                        int causal, int partition_size, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  const Shape s{B, Hq, Hkv, Sq, Skv, D};
  int T = 0, P = 0;
  float *ws_m = nullptr, *ws_l = nullptr, *ws_acc = nullptr;
  unsigned* counters = nullptr;
  // The output pointer is not used here; pass q so the shared check sees a non-null pointer.
  const ef::KeyRuns runs = key_runs(Sq, Skv, 0, 0);
  ef_status st = split_prepare(s, q, k, v, static_cast<const float*>(q), scale, runs,
                               partition_size, workspace, workspace_bytes, &T, &P, &ws_m, &ws_l,
                               &ws_acc, &counters);
  if (st != EF_OK || P == 0) return st;
  return split_produce(s, q, k, v, scale, causal, runs, T, P, ws_m, ws_l, ws_acc, nullptr,
                       nullptr, static_cast<hipStream_t>(stream));
}

ef_status ef_attention_splitkv(const void* q, const void* k, const void* v, float* o, int B,
                               int Hq, int Hkv, int Sq, int Skv, int D, float scale, int causal,
                               int partition_size, void* workspace, size_t workspace_bytes,
                               void* stream) {
  return splitkv_impl(Shape{B, Hq, Hkv, Sq, Skv, D}, q, k, v, o, scale, causal,
                      key_runs(Sq, Skv, 0, 0), partition_size, workspace, workspace_bytes,
                      stream);
}

ef_status ef_attention_splitkv_local(const void* q, const void* k, const void* v, float* o,
                                     int B, int Hq, int Hkv, int Sq, int Skv, int D, float scale,
                                     int window, int sinks, int partition_size, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  const Shape s{B, Hq, Hkv, Sq, Skv, D};
  ef_status st = check_shape(s);
  if (st != EF_OK) return st;
  st = check_mask(window, sinks);
  if (st != EF_OK) return st;
  return splitkv_impl(s, q, k, v, o, scale, 1, key_runs(Sq, Skv, window, sinks), partition_size,
                      workspace, workspace_bytes, stream);
}

ef_status ef_attention_combine(const float* m, const float* l, const float* acc, float* o,
                               int rows, int num_partitions, int D, void* stream) {
  if (rows < 0 || num_partitions < 1) return EF_ERR_INVALID_SHAPE;
  if (D != 64 && D != 128) return EF_ERR_UNSUPPORTED_HEAD_DIM;
  if (rows == 0) return EF_OK;
  if (m == nullptr || l == nullptr || acc == nullptr || o == nullptr) return EF_ERR_NULL_POINTER;
  if (misaligned(m) || misaligned(l) || misaligned(acc) || misaligned(o)) return EF_ERR_MISALIGNED;
  ef::CombineParams c{};
  c.m = m;
  c.l = l;
  c.acc = acc;
  c.o = o;
  c.rows = rows;
  c.P = num_partitions;
  c.D = D;
  return from_hip(ef::launch_combine(c, static_cast<hipStream_t>(stream)));
}

double ef_attention_splitkv_modeled_us(int B, int Hq, int Hkv, int Sq, int Skv, int D, int window,
                                        int sinks, int partition_size) {
  const Shape s{B, Hq, Hkv, Sq, Skv, D};
  if (check_shape(s) != EF_OK || window < 0 || sinks < 0) return -1.0;
  if (partition_size <= 0 || partition_size % kTileKeys != 0) return -1.0;
  const ef::KeyRuns runs = key_runs(Sq, Skv, window, sinks);
  if (s.rows() == 0 || runs.lv == 0) return 0.0;
  return split_model_us(s, runs.lv, partition_size, visible_keys(s, runs));
}

int ef_attention_rows_per_workgroup(int B, int Hq, int Hkv, int Sq, int Skv, int D, int keys) {
  const Shape s{B, Hq, Hkv, Sq, Skv, D};
  if (check_shape(s) != EF_OK || keys < 0) return 0;
  return rows_per_block(s, keys);
}

ef_status ef_attention_splitkv_tune(const void* q, const void* k, const void* v, float* o, int B,
                                    int Hq, int Hkv, int Sq, int Skv, int D, float scale,
                                    int causal, int window, int sinks, void* workspace,
                                    size_t workspace_bytes, void* stream, int* partition_size) {
  if (partition_size == nullptr) return EF_ERR_NULL_POINTER;
  const Shape s{B, Hq, Hkv, Sq, Skv, D};
  ef_status st = check_shape(s);
  if (st != EF_OK) return st;
  if (window < 0 || sinks < 0 || (window == 0 && sinks != 0)) return EF_ERR_INVALID_MASK;
  st = check_io(s, q, k, v, o, scale);
  if (st != EF_OK) return st;
  const bool local = window > 0;
  const ef::KeyRuns runs = key_runs(Sq, Skv, window, sinks);
  if (s.rows() == 0 || runs.lv == 0) {
    *partition_size = resolve_partition(s, runs.lv, 0, visible_keys(s, runs));
    return EF_OK;
  }
  // Candidates the model rates best, whose workspace fits.
  std::vector<std::pair<double, int>> ranked;
  for (int t : partition_candidates(runs.lv)) {
    if (workspace_size_impl(s, runs, t) <= workspace_bytes)
      ranked.push_back({split_model_us(s, runs.lv, t, visible_keys(s, runs)), t});
  }
  if (ranked.empty()) return EF_ERR_WORKSPACE_TOO_SMALL;
  std::sort(ranked.begin(), ranked.end());
  constexpr size_t kTried = 6;
  if (ranked.size() > kTried) ranked.resize(kTried);
  std::vector<int> cands;
  for (const auto& r : ranked) cands.push_back(r.second);

  hipStream_t hs = static_cast<hipStream_t>(stream);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    if (e0) (void)hipEventDestroy(e0);
    return EF_ERR_HIP;
  }
  auto call = [&](int t) {
    return splitkv_impl(s, q, k, v, o, scale, local ? 1 : causal, runs, t, workspace,
                        workspace_bytes, stream);
  };
  // Successive halving (section 6.3, progressive tuning): time every
  // remaining candidate, keep the faster half, double the repetitions.
  int reps = 2;
  while (cands.size() > 1 && st == EF_OK) {
    std::vector<std::pair<float, int>> timed;
    for (int t : cands) {
      st = call(t);  // warm-up
      if (st != EF_OK) break;
      if (hipEventRecord(e0, hs) != hipSuccess) { st = EF_ERR_HIP; break; }
      for (int r = 0; r < reps && st == EF_OK; ++r) st = call(t);
      if (st != EF_OK) break;
      float ms = 0.f;
      if (hipEventRecord(e1, hs) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
          hipEventElapsedTime(&ms, e0, e1) != hipSuccess) {
        st = EF_ERR_HIP;
        break;
      }
      timed.push_back({ms, t});
    }
    if (st != EF_OK) break;
    std::stable_sort(timed.begin(), timed.end());
    cands.clear();
    for (size_t i = 0; i < (timed.size() + 1) / 2; ++i) cands.push_back(timed[i].second);
    reps *= 2;
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (st == EF_OK) *partition_size = cands.front();
  return st;
}

}  // extern "C"

namespace {

// Number of partitions ef_diff_attention uses (1 = single pass), or 0 for an
// invalid shape or partition size.
long long diff_partitions(const Shape& s, int partition_size, int* T_out) {
  if (check_shape(s) != EF_OK) return 0;
  if (partition_size < 0 || partition_size % kTileKeys != 0) return 0;
  if (s.rows() == 0 || s.Skv == 0) return 1;
  const int T = resolve_partition(s, s.Skv, partition_size, s.Skv);
  *T_out = T;
  return (s.Skv + (long long)T - 1) / T;
}

// One branch through the split-KV producer and the combine; with `diff` the
// combine applies the differential epilogue against the A2 already in o.
ef_status diff_branch_split(const Shape& s, const void* q, const void* k, const void* v, float* o,
                            float scale, int causal, const ef::KeyRuns& runs, int T, int P,
                            const WsLayout& w, char* ws, const ef::DiffParams* diff,
                            hipStream_t hs) {
  float* ws_m = reinterpret_cast<float*>(ws + w.m_off);
  float* ws_l = reinterpret_cast<float*>(ws + w.l_off);
  float* ws_acc = reinterpret_cast<float*>(ws + w.acc_off);
  ef_status st = split_produce(s, q, k, v, scale, causal, runs, T, P, ws_m, ws_l, ws_acc, nullptr,
                               nullptr, hs);
  if (st != EF_OK) return st;
  ef::CombineParams c{};
  c.m = ws_m;
  c.l = ws_l;
  c.acc = ws_acc;
  c.o = o;
  c.rows = (int)s.rows();
  c.P = P;
  c.D = s.D;
  if (diff != nullptr) c.diff = *diff;
  return from_hip(ef::launch_combine(c, hs));
}

}  // namespace

extern "C" {

ef_status ef_diff_attention(const void* q1, const void* q2, const void* k1, const void* k2,
                            const void* v, float* o, const float* lambda_q1,
                            const float* lambda_k1, const float* lambda_q2,
                            const float* lambda_k2, const float* norm_weight, float lambda_init,
                            float eps, int B, int Hq, int Hkv, int Sq, int Skv, int D,
                            float scale, int causal, int partition_size, void* workspace,
                            size_t workspace_bytes, void* stream) {
  const Shape s{B, Hq, Hkv, Sq, Skv, D};
  ef_status st = check_shape(s);
  if (st != EF_OK) return st;
  if (partition_size < 0 || partition_size % kTileKeys != 0) return EF_ERR_INVALID_PARTITION;
  st = check_io(s, q1, k1, v, o, scale);
  if (st != EF_OK) return st;
  st = check_io(s, q2, k2, v, o, scale);
  if (st != EF_OK) return st;
  if (!std::isfinite(lambda_init) || !std::isfinite(eps) || eps < 0.f) return EF_ERR_INVALID_DIFF;
  if (s.rows() == 0) return EF_OK;
  if (lambda_q1 == nullptr || lambda_k1 == nullptr || lambda_q2 == nullptr ||
      lambda_k2 == nullptr || norm_weight == nullptr)
    return EF_ERR_NULL_POINTER;
  if (misaligned(norm_weight)) return EF_ERR_MISALIGNED;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  // No keys: A1 = A2 = 0, so y = 0 and every output row is 0.
  if (s.Skv == 0) return from_hip(ef::launch_zero_fill(o, (size_t)s.rows() * s.D, hs));
  int T = 0;
  const long long P = diff_partitions(s, partition_size, &T);
  if (P > kMaxGridYZ) return EF_ERR_INVALID_PARTITION;
  const ef::DiffParams diff{lambda_q1, lambda_k1, lambda_q2, lambda_k2, norm_weight, lambda_init,
                            eps};
  const ef::KeyRuns runs = key_runs(Sq, Skv, 0, 0);
  if (P == 1) {
    st = launch_mfma(s, q2, k2, v, o, nullptr, nullptr, nullptr, runs.lv, 1, scale, causal, runs,
                     hs);
    if (st != EF_OK) return st;
    return launch_mfma(s, q1, k1, v, o, nullptr, nullptr, nullptr, runs.lv, 1, scale, causal,
                       runs, hs, &diff);
  }
  const WsLayout w = ws_layout(s.rows(), P, s.D);
  if (workspace == nullptr || workspace_bytes < w.bytes) return EF_ERR_WORKSPACE_TOO_SMALL;
  if (misaligned(workspace)) return EF_ERR_MISALIGNED;
  char* ws = static_cast<char*>(workspace);
  st = diff_branch_split(s, q2, k2, v, o, scale, causal, runs, T, (int)P, w, ws, nullptr, hs);
  if (st != EF_OK) return st;
  return diff_branch_split(s, q1, k1, v, o, scale, causal, runs, T, (int)P, w, ws, &diff, hs);
}

size_t ef_diff_attention_workspace_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                        int partition_size) {
  const Shape s{B, Hq, Hkv, Sq, Skv, D};
  int T = 0;
  const long long P = diff_partitions(s, partition_size, &T);
  if (P <= 1 || P > kMaxGridYZ) return 0;
  return ws_layout(s.rows(), P, s.D).bytes;
}

}  // extern "C"

namespace {

// Partitions of the output-channel split decode (1: no workspace), or 0 for an
// invalid shape, partition size or split.
long long dsplit_partitions(const Shape& s, int d_splits, int partition_size, int* T_out) {
  if (check_shape(s) != EF_OK) return 0;
  if (d_splits != 1 && d_splits != 2 && d_splits != 4) return 0;
  if ((long long)(s.Hq / s.Hkv) * s.Sq > kDecodeMaxRows) return 0;
  if (partition_size < 0 || partition_size % kTileKeys != 0) return 0;
  if (s.rows() == 0 || s.Skv == 0) return 1;
  const int T = resolve_partition(s, s.Skv, partition_size, s.Skv);
  *T_out = T;
  return (s.Skv + (long long)T - 1) / T;
}

}  // namespace

extern "C" {

ef_status ef_attention_decode_dsplit(const void* q, const void* k, const void* v, float* o, int B,
                                     int Hq, int Hkv, int Sq, int Skv, int D, float scale,
                                     int causal, int d_splits, int partition_size,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  const Shape s{B, Hq, Hkv, Sq, Skv, D};
  ef_status st = check_shape(s);
  if (st != EF_OK) return st;
  if (d_splits != 1 && d_splits != 2 && d_splits != 4) return EF_ERR_INVALID_SPLIT;
  if ((long long)(Hq / Hkv) * Sq > kDecodeMaxRows) return EF_ERR_INVALID_SPLIT;
  if (partition_size < 0 || partition_size % kTileKeys != 0) return EF_ERR_INVALID_PARTITION;
  st = check_io(s, q, k, v, o, scale);
  if (st != EF_OK) return st;
  if (s.rows() == 0) return EF_OK;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (s.Skv == 0) return from_hip(ef::launch_zero_fill(o, (size_t)s.rows() * s.D, hs));
  int T = 0;
  const long long P = dsplit_partitions(s, d_splits, partition_size, &T);
  if (P < 1 || P * d_splits > 0x7fffffffLL) return EF_ERR_INVALID_PARTITION;
  const ef::KeyRuns runs = key_runs(Sq, Skv, 0, 0);
  if (P == 1)  // each workgroup writes its channels of o: no workspace, no merge
    return split_produce(s, q, k, v, scale, causal, runs, T, 1, nullptr, nullptr, nullptr,
                         nullptr, o, hs, d_splits);
  const WsLayout w = ws_layout(s.rows(), P, s.D);
  if (workspace == nullptr || workspace_bytes < w.bytes) return EF_ERR_WORKSPACE_TOO_SMALL;
  if (misaligned(workspace)) return EF_ERR_MISALIGNED;
  char* ws = static_cast<char*>(workspace);
  float* ws_m = reinterpret_cast<float*>(ws + w.m_off);
  float* ws_l = reinterpret_cast<float*>(ws + w.l_off);
  float* ws_acc = reinterpret_cast<float*>(ws + w.acc_off);
  unsigned* counters = reinterpret_cast<unsigned*>(ws + w.cnt_off);
  if (fused_combine(s, P, d_splits))
    return split_produce(s, q, k, v, scale, causal, runs, T, (int)P, ws_m, ws_l, ws_acc,
                         counters, o, hs, d_splits);
  st = split_produce(s, q, k, v, scale, causal, runs, T, (int)P, ws_m, ws_l, ws_acc, nullptr,
                     nullptr, hs, d_splits);
  if (st != EF_OK) return st;
  ef::CombineParams c{};
  c.m = ws_m;
  c.l = ws_l;
  c.acc = ws_acc;
  c.o = o;
  c.rows = (int)s.rows();
  c.P = (int)P;
  c.D = s.D;
  return from_hip(ef::launch_combine(c, hs));
}

size_t ef_attention_decode_dsplit_workspace_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                                 int d_splits, int partition_size) {
  const Shape s{B, Hq, Hkv, Sq, Skv, D};
  int T = 0;
  const long long P = dsplit_partitions(s, d_splits, partition_size, &T);
  if (P <= 1) return 0;
  return ws_layout(s.rows(), P, s.D).bytes;
}

}  // extern "C"
