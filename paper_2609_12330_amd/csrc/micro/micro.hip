// Achievable-ceiling microbenchmarks for the measurement script: a streaming
// read of device memory and a bare matrix-core loop. They bound what the
// attention kernels can reach on this chip at its running clock (the spec
// peaks stay the roofline targets). Not part of the attention library: built
// into a library of their own and loaded only by the benchmark.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr uint32_t kBufferFlags = 0x00020000u;  // raw 32-bit buffer access
constexpr int kNonTemporal = 2;

// Each workgroup streams one contiguous range of a slice of at most 2^31
// bytes through a buffer descriptor: per step its 256 threads read eight
// consecutive 4 KiB blocks, 16 bytes per thread and block (all eight loads in
// flight), and fold them with xor; one word per workgroup is written so the
// loads cannot be dropped.
__global__ __launch_bounds__(256) void stream_read_kernel(const unsigned char* buf,
                                                          unsigned bytes, uint32_t* sink) {
  constexpr int kInFlight = 8;
  constexpr unsigned kBlock = 256u * 16u;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<unsigned char*>(buf), (short)0, (int)bytes, kBufferFlags);
  const unsigned per = (bytes / gridDim.x + kBlock * kInFlight - 1) / (kBlock * kInFlight) *
                       (kBlock * kInFlight);
  const unsigned beg = blockIdx.x * per;
  const unsigned end = beg + per < bytes ? beg + per : bytes;
  u32x4_t acc = {0u, 0u, 0u, 0u};
  for (unsigned off = beg + threadIdx.x * 16u; off < end; off += kBlock * kInFlight) {
    u32x4_t x[kInFlight];
#pragma unroll
    for (int i = 0; i < kInFlight; ++i)
      x[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, off + i * kBlock, 0, kNonTemporal);
#pragma unroll
    for (int i = 0; i < kInFlight; ++i) acc ^= x[i];
  }
  uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o, 64);
  __shared__ uint32_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

// Each wave runs `iters` rounds of four independent chains of
// v_mfma_f32_32x32x16_bf16 on register operands (no memory traffic inside the
// loop) and writes one value, so the products cannot be dropped.
__global__ __launch_bounds__(256) void mfma_loop_kernel(float* out, int iters) {
  const int lane = threadIdx.x & 63;
  bf16x8_t a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (lane + i));
    b[i] = (__bf16)(0.002f * (lane - i));
  }
  floatx16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int it = 0; it < iters; ++it) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
  }
  float s = 0.f;
  for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  if (s == 12345.f) out[blockIdx.x] = s;  // practically never taken; keeps the loop
}

}  // namespace

extern "C" {

// Reads `bytes` (multiple of 16, below 2^31) of device memory at `buf` with
// `blocks` workgroups of 256 threads; `sink` holds `blocks` words. 0 on success.
int ef_micro_stream_read(const void* buf, size_t bytes, void* sink, int blocks, void* stream) {
  if (buf == nullptr || sink == nullptr || blocks < 1 || bytes == 0 || bytes >= (1ull << 31) ||
      bytes % 16 != 0)
    return 1;
  hipLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const unsigned char*>(buf),
                     (unsigned)bytes, static_cast<uint32_t*>(sink));
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

// `blocks` workgroups of 4 waves, each wave 4 * iters matrix products of
// 32 x 32 x 16 (32768 flops each). `out` holds `blocks` floats. 0 on success.
int ef_micro_mfma(void* out, int blocks, int iters, void* stream) {
  if (out == nullptr || blocks < 1 || iters < 1) return 1;
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(blocks), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<float*>(out), iters);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // extern "C"
