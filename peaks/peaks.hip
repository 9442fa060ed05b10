// On-device reference rates for the roofline peaks: a streaming read of a large
// buffer (the HBM rate this chip delivers to a plain coalesced read), a gather of
// random 16 KiB tiles (the rate reads that miss the L2 reach in that pattern), and a loop
// of dense bf16 32x32x16 matrix-core products held in registers (the matrix-core
// rate at the clock the chip runs).  Measurement aids only; not part of libgca.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

// Every thread reads 16-byte blocks in a grid-stride loop, four in flight, and
// folds them with XOR; the fold is stored only if it equals an impossible key, so
// the loads cannot be dropped and nothing is written.
__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4* __restrict__ p, int64_t n, uint32_t key,
                                                          uint32_t* __restrict__ sink) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  u32x4 acc = u32x4{0u, 0u, 0u, 0u};
  for (; i + 3 * stride < n; i += 4 * stride) {
    const u32x4 a = __builtin_nontemporal_load(p + i), b = __builtin_nontemporal_load(p + i + stride);
    const u32x4 c = __builtin_nontemporal_load(p + i + 2 * stride), d = __builtin_nontemporal_load(p + i + 3 * stride);
    acc ^= a ^ b ^ c ^ d;
  }
  for (; i < n; i += stride) acc ^= __builtin_nontemporal_load(p + i);
  const uint32_t f = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  if (f == key) sink[0] = f;
}

// Each workgroup reads whole 16 KiB tiles chosen by idx[] (tile t at p + idx[t] *
// 16 KiB), 64 bytes per thread per tile, T tiles in flight: the access pattern of
// the attention kernels' gathers of one retrieved chunk's K or V pair, without
// the compute.
template <int T>
__global__ __launch_bounds__(256) void tile_gather_kernel(const u32x4* __restrict__ p,
                                                          const int32_t* __restrict__ idx, int n, uint32_t key,
                                                          uint32_t* __restrict__ sink) {
  u32x4 acc = u32x4{0u, 0u, 0u, 0u};
  for (int t = blockIdx.x * T; t < n; t += gridDim.x * T) {
    u32x4 v[T][4];
#pragma unroll
    for (int u = 0; u < T; ++u) {
      const u32x4* tile = p + (int64_t)idx[t + u < n ? t + u : t] * 1024;
#pragma unroll
      for (int c = 0; c < 4; ++c) v[u][c] = tile[threadIdx.x + 256 * c];
    }
#pragma unroll
    for (int u = 0; u < T; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  const uint32_t f = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  if (f == key) sink[0] = f;
}

// Each wave runs `iters` rounds of 8 independent 32x32x16 bf16 products (8
// accumulators, so the matrix core never waits on a result).
__global__ __launch_bounds__(256) void mfma_loop_kernel(int iters, float key, float* __restrict__ sink) {
  bf16x8 a, b;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    a[m] = (__bf16)(0.001f * (float)(threadIdx.x + m));
    b[m] = (__bf16)(0.002f * (float)(threadIdx.x - m));
  }
  f32x16 c[8];
#pragma unroll
  for (int u = 0; u < 8; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) c[u][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int u = 0; u < 8; ++u) c[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[u], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < 8; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c[u][r];
  if (s == key) sink[0] = s;
}

}  // namespace

extern "C" {

// Launch the streaming read of n16 16-byte blocks at p on `stream`.
int peaks_stream_read(const void* p, int64_t n16, int blocks, void* sink, hipStream_t stream) {
  hipLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(256), 0, stream, (const u32x4*)p, n16, 0x9E3779B9u,
                     (uint32_t*)sink);
  return (int)hipGetLastError();
}

// Launch the gather of n 16 KiB tiles at p, tile t being p + idx[t] * 16 KiB
// (idx: n device int32 values, each below the number of whole tiles at p), with
// `in_flight` (1 or 2) tiles per workgroup at a time.
int peaks_tile_gather(const void* p, const void* idx, int n, int blocks, int in_flight, void* sink,
                      hipStream_t stream) {
  if (in_flight == 2)
    hipLaunchKernelGGL(tile_gather_kernel<2>, dim3(blocks), dim3(256), 0, stream, (const u32x4*)p,
                       (const int32_t*)idx, n, 0x9E3779B9u, (uint32_t*)sink);
  else
    hipLaunchKernelGGL(tile_gather_kernel<1>, dim3(blocks), dim3(256), 0, stream, (const u32x4*)p,
                       (const int32_t*)idx, n, 0x9E3779B9u, (uint32_t*)sink);
  return (int)hipGetLastError();
}

// Launch the matrix-core loop: `blocks` workgroups of 4 waves, `iters` rounds of
// 8 products each; flops = blocks * 4 * iters * 8 * 32768.
int peaks_mfma_loop(int blocks, int iters, void* sink, hipStream_t stream) {
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(blocks), dim3(256), 0, stream, iters, -1.2345e-30f, (float*)sink);
  return (int)hipGetLastError();
}

}  // extern "C"
