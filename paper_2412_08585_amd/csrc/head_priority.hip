// Head-wise mixed precision (Sec. 3.2): the priority gap x std of each KV
// head, from the prefill keys of the whole batch.
//
// One workgroup of 1024 threads per KV head.  Thread (tl, cg) covers channels
// 8cg .. 8cg+7 (16 bytes of a 256-byte fp16 row, so 16 threads read a whole
// row) of the tokens tl, tl + 64, ... of every sequence, four rows in flight,
// keeping per-channel maxima and minima; the 64 token lanes are then merged
// through LDS, and one wave forms the channel gaps, their mean and spread.
#include "turbo_common.h"

namespace turbo {

struct PriorityArgs {
  const uint4* k;   // fp16 [B][Hkv][N][128] as 8-half units
  int B, Hkv, N;
  float* priority;  // [Hkv]
};

constexpr int kPrioThreads = 1024;
constexpr int kPrioTokenLanes = kPrioThreads / 16;

__global__ __launch_bounds__(kPrioThreads) void k_head_priority(PriorityArgs a) {
  __shared__ float smax[kPrioTokenLanes / 4][128 + 4];
  __shared__ float smin[kPrioTokenLanes / 4][128 + 4];
  const int h = blockIdx.x;
  const int tid = threadIdx.x;
  const int cg = tid & 15, tl = tid >> 4;
  float mx[8], mn[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    mx[e] = -INFINITY;
    mn[e] = INFINITY;
  }
  auto fold = [&](uint4 raw) {
    const f16x8_t v = __builtin_bit_cast(f16x8_t, raw);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mx[e] = fmaxf(mx[e], (float)v[e]);
      mn[e] = fminf(mn[e], (float)v[e]);
    }
  };
  for (int b = 0; b < a.B; ++b) {
    const uint4* rows = a.k + ((long)b * a.Hkv + h) * a.N * 16 + cg;
    int t = tl;
    for (; t + 3 * kPrioTokenLanes < a.N; t += 4 * kPrioTokenLanes) {
      const uint4 r0 = rows[(long)t * 16];
      const uint4 r1 = rows[(long)(t + kPrioTokenLanes) * 16];
      const uint4 r2 = rows[(long)(t + 2 * kPrioTokenLanes) * 16];
      const uint4 r3 = rows[(long)(t + 3 * kPrioTokenLanes) * 16];
      fold(r0);
      fold(r1);
      fold(r2);
      fold(r3);
    }
    for (; t < a.N; t += kPrioTokenLanes) fold(rows[(long)t * 16]);
  }
  // merge the 64 token lanes: four at a time through LDS
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], 16));
    mn[e] = fminf(mn[e], __shfl_xor(mn[e], 16));
    mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], 32));
    mn[e] = fminf(mn[e], __shfl_xor(mn[e], 32));
  }
  // lanes 0..15 of each wave now hold the wave's 4 token lanes merged
  const int wv = tid >> 6;
  if ((tid & 63) < 16) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      smax[wv][8 * cg + e] = mx[e];
      smin[wv][8 * cg + e] = mn[e];
    }
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
      for (int l = 0; l < kPrioTokenLanes / 4; ++l) {
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
