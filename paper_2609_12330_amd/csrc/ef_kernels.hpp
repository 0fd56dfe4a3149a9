// Kernel parameter blocks and launchers of the gfx950 attention library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ef {

// Visible keys of one (batch, kv head) group as a virtual key axis of length lv:
// virtual keys [0, la) are keys [0, la) (the sink run) and virtual keys
// [la, lv) are keys [bs, bs + lv - la) (the window run). Without a window
// la = bs = 0 and lv = Skv. la and bs are multiples of 64, so 64-key tiles of
// the virtual axis are 64-key tiles of the real one.
struct KeyRuns {
  int la, bs, lv;
  int window, sinks;  // window > 0: key j visible to row i iff j > n_i - window or j < sinks
};

// Differential attention epilogue (section 7.3): the output row is
// (1 - lambda_init) * gamma * y / sqrt(mean(y^2) + eps) with y = A1 - lambda * A2
// and lambda = exp(<lq1, lk1>) - exp(<lq2, lk2>) + lambda_init. Unused while
// gamma is null.
struct DiffParams {
  const float* lq1;
  const float* lk1;
  const float* lq2;
  const float* lk2;
  const float* gamma;  // [D] fp32 each
  float lambda_init, eps;
};

// Split-KV decode producer (VALU path, G*Sq <= 8 query rows per kv head).
struct DecodeParams {
  const uint16_t* q;  // [B][Hq][Sq][D] bf16
  const uint16_t* k;  // [B][Hkv][Skv][D] bf16
  const uint16_t* v;
  float* ws_m;    // [rows][P]
  float* ws_l;    // [rows][P]
  float* ws_acc;  // [rows][P][D]
  int B, Hq, Hkv, Sq, Skv, D;
  int G;  // Hq / Hkv
  int R;  // G * Sq query rows per kv head
  int T;  // keys per partition
  int P;  // partitions
  float c;  // scale * log2(e)
  int causal;
  // Fused combine (optional): per-(batch, kv head, channel slice) arrival
  // counters, zero on entry and left zero on exit, and the output o
  // [B][Hq][Sq][D] fp32. With ws_acc null (one partition) o is written directly.
  unsigned* counters;
  float* o;
  KeyRuns runs;  // partitions cover the virtual key axis (T keys each)
  int d_splits;  // output-channel slices per partition: 1 (0 also means 1), 2 or 4
};

// Largest partition count for which the producer combines its group itself.
constexpr int kFusedMaxP = 64;

// Arrival counters sit 256 bytes apart (one counter per (batch, kv head),
// and channel slice): counters sharing a line serialise the workgroups'
// arrivals at the end. They occupy a region of fixed size at the start of
// every workspace, so a workspace reused for problems of other shapes keeps
// its counters in place (each completed call leaves the slots it used at
// zero, and no partial state is ever stored there). A launch with more
// groups than slots combines in a separate kernel instead.
constexpr int kCounterStride = 64;
constexpr int kCounterSlots = 512;
constexpr size_t kCounterRegionBytes = (size_t)kCounterSlots * kCounterStride * 4;

// MFMA attention (single pass, or split producer when ws_m != nullptr).
struct MfmaParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  float* o;       // [B][Hq][Sq][D] fp32, single-pass mode
  float* ws_m;    // split mode: partial states as in DecodeParams
  float* ws_l;
  float* ws_acc;
  int B, Hq, Hkv, Sq, Skv, D;
  int G, R;
  int T, P;      // keys per partition and partitions (T >= Skv, P = 1 in single-pass mode)
  int bm;        // query rows per workgroup: 64 (two waves) or 128 (four)
  int mtiles;    // query-row tiles per kv head
  float c_abs;   // |scale| * log2(e)
  int causal;
  KeyRuns runs;  // split mode: partitions cover the virtual key axis
  // Differential attention, single pass only: with diff.gamma set this launch
  // is the first branch and o already holds the second branch's output.
  DiffParams diff;
};

// Combine of stored partial states.
struct CombineParams {
  const float* m;
  const float* l;
  const float* acc;
  float* o;  // [rows][D]
  int rows, P, D;
  // Differential attention: with diff.gamma set the states are the first
  // branch's and o already holds the second branch's output.
  DiffParams diff;
};

// Fill of an fp32 buffer with zeros (output rows that see no key).
hipError_t launch_zero_fill(float* p, size_t n, hipStream_t stream);
hipError_t launch_decode_split(const DecodeParams& a, hipStream_t stream);
hipError_t launch_mfma_attention(const MfmaParams& a, bool negative_scale, hipStream_t stream);
hipError_t launch_combine(const CombineParams& a, hipStream_t stream);


}  // namespace ef
