// Head-wise mixed precision (Sec. 3.2): the priority gap x std of each KV
// head, from the prefill keys of the whole batch.
//
// One workgroup of 1024 threads per KV head.  Thread (tl, cg) covers channels
// 4cg .. 4cg+3 (8 bytes of a 256-byte fp16 row, so a warp-row of 32 threads
// reads whole rows) of the tokens tl, tl + 32, ... of every sequence, keeping
// per-channel maxima and minima; the 32 token lanes are then merged through
// LDS, and one wave forms the channel gaps, their mean and spread.
#include "turbo_common.h"

namespace turbo {

struct PriorityArgs {
  const uint2* k;   // fp16 [B][Hkv][N][128] as 4-half units
  int B, Hkv, N;
  float* priority;  // [Hkv]
};

constexpr int kPrioThreads = 1024;
constexpr int kPrioTokenLanes = kPrioThreads / 32;

__global__ __launch_bounds__(kPrioThreads) void k_head_priority(PriorityArgs a) {
  __shared__ float smax[kPrioTokenLanes][128 + 4];
  __shared__ float smin[kPrioTokenLanes][128 + 4];
  const int h = blockIdx.x;
  const int tid = threadIdx.x;
  const int cg = tid & 31, tl = tid >> 5;
  float mx[4], mn[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    mx[e] = -INFINITY;
    mn[e] = INFINITY;
  }
  for (int b = 0; b < a.B; ++b) {
    const uint2* rows = a.k + ((long)b * a.Hkv + h) * a.N * 32 + cg;
    for (int t = tl; t < a.N; t += kPrioTokenLanes) {
      const f16x4_t v = __builtin_bit_cast(f16x4_t, rows[(long)t * 32]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        mx[e] = fmaxf(mx[e], (float)v[e]);
        mn[e] = fminf(mn[e], (float)v[e]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    smax[tl][4 * cg + e] = mx[e];
    smin[tl][4 * cg + e] = mn[e];
  }
  __syncthreads();
  if (tid < 64) {
    // lane c handles channels c and c + 64
    float gap[2], cmax[2], cmin[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = tid + 64 * u;
      cmax[u] = -INFINITY;
      cmin[u] = INFINITY;
      for (int l = 0; l < kPrioTokenLanes; ++l) {
        cmax[u] = fmaxf(cmax[u], smax[l][c]);
        cmin[u] = fminf(cmin[u], smin[l][c]);
      }
      gap[u] = cmax[u] - cmin[u];
    }
    const float gmax = wave_max(fmaxf(cmax[0], cmax[1]));
    const float gmin = -wave_max(-fminf(cmin[0], cmin[1]));
    float sum = gap[0] + gap[1];
    for (int m = 32; m >= 1; m >>= 1) sum += __shfl_xor(sum, m);
    const float mean = sum / 128.0f;
    const float d0 = gap[0] - mean, d1 = gap[1] - mean;
    float sq = d0 * d0 + d1 * d1;
    for (int m = 32; m >= 1; m >>= 1) sq += __shfl_xor(sq, m);
    if (tid == 0) a.priority[h] = (gmax - gmin) * sqrtf(sq / 128.0f);
  }
}

hipError_t launch_head_priority(const PriorityArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(k_head_priority, dim3(a.Hkv), dim3(kPrioThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace turbo
