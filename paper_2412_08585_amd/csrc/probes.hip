// Measurement probes (not part of the method): the two ceilings the attention
// kernels are judged against, measured on the GPU itself.
//   * k_probe_mfma_i8: every wave runs chains of v_mfma_i32_16x16x64_i8 on
//     register operands -- the int8 matrix-core rate with no memory traffic
//     and no VALU work between the MFMAs;
//   * k_probe_read: a grid-stride streaming read of a device buffer (16-byte
//     loads, eight in flight per thread) -- the HBM read rate a kernel that
//     only reads can reach.
// Each folds its results into one word per work-group so nothing is
// eliminated, and that word is written.
#include "turbo_common.h"

namespace turbo {

constexpr int kProbeChains = 8;  // independent accumulator chains per wave

__global__ __launch_bounds__(256, 2) void k_probe_mfma_i8(int iters, int* sink) {
  const int lane = threadIdx.x & 63;
  v4i a = {lane, lane * 3, lane ^ 5, 7 - lane};
  v4i b = {lane + 1, lane * 5, lane ^ 9, 11 - lane};
  v4i acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) acc[c] = v4i{c, 0, 0, 0};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c) acc[c] = mfma16x16x64(a, b, acc[c]);
  }
  int x = 0;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) x ^= acc[c][0] ^ acc[c][1] ^ acc[c][2] ^ acc[c][3];
  x = wave_max_i(x);
  if (threadIdx.x == 0) sink[blockIdx.x] = x;
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void k_probe_read(const u32x4* src, long n16, unsigned* sink) {
  const long stride = (long)gridDim.x * blockDim.x;
  long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  unsigned x = 0;
  for (; i + 7 * stride < n16; i += 8 * stride) {
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < 8; ++u) x ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
  for (; i < n16; i += stride) {
    const u32x4 v = src[i];
    x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  x = (unsigned)wave_max_i((int)x);
  if ((threadIdx.x & 63) == 0) sink[blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6)] = x;
}

// Work-groups of the probes: two per CU for the MFMA loop (8 waves per CU,
// two per SIMD), eight per CU for the read.
constexpr int kProbeMfmaBlocks = 512;
constexpr int kProbeReadBlocks = 2048;

hipError_t launch_probe_mfma_i8(int iters, int* sink, hipStream_t stream) {
  hipLaunchKernelGGL(k_probe_mfma_i8, dim3(kProbeMfmaBlocks), dim3(256), 0, stream, iters, sink);
  return hipGetLastError();
}

hipError_t launch_probe_read(const void* src, size_t bytes, unsigned* sink, hipStream_t stream) {
  hipLaunchKernelGGL(k_probe_read, dim3(kProbeReadBlocks), dim3(256), 0, stream,
                     static_cast<const u32x4*>(src), (long)(bytes / 16), sink);
  return hipGetLastError();
}

}  // namespace turbo
