// Head-wise mixed precision (Sec. 3.2): the priority gap x std of each KV
// head, from the prefill keys of the whole batch.
//
// Two launches, so that the reads of the keys spread over the whole chip:
//   * k_head_minmax: one work-group of 256 threads per (KV head, sequence,
//     256-token slab).  Thread (row lane tl, channel group cg) covers channels
//     8cg .. 8cg+7 (16 bytes of a 256-byte fp16 row: 16 threads read a whole
//     row, a wave four consecutive rows) of rows tl, tl + 16, ..., sixteen
//     loads in flight at once; the 16 row lanes are merged through LDS and the
//     slab's per-channel maxima and minima go to the workspace.
//   * k_head_priority_final: one work-group of 1024 threads per KV head merges
//     its slabs (four threads per statistic, eight loads in flight each), then
//     one wave forms the channel gaps, their mean and spread.
#include "turbo_common.h"

namespace turbo {

struct PriorityArgs {
  const uint4* k;   // fp16 [B][Hkv][N][128] as 8-half units
  int B, Hkv, N;
  int nslab;        // 128-token slabs per sequence
  float* ws;        // [Hkv][B * nslab][256]: channel maxima, then minima
  float* priority;  // [Hkv]
};

constexpr int kPrioSlab = 256;  // tokens per slab
constexpr int kPrioRowLanes = 16;
constexpr int kPrioLoads = 16;  // rows per thread in flight at once

__global__ __launch_bounds__(256) void k_head_minmax(PriorityArgs a) {
  __shared__ float sx[kPrioRowLanes / 4][2][128 + 4];
  const int s = blockIdx.x % a.nslab;
  const int b = (blockIdx.x / a.nslab) % a.B;
  const int h = blockIdx.x / (a.nslab * a.B);
  const int tid = threadIdx.x;
  const int cg = tid & 15, tl = tid >> 4;
  float mx[8], mn[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    mx[e] = -INFINITY;
    mn[e] = INFINITY;
  }
  for (int r0 = 0; r0 < kPrioSlab; r0 += kPrioRowLanes * kPrioLoads) {
    const int t0 = s * kPrioSlab + r0 + tl;
    if (t0 >= a.N) break;
    const uint4* rows = a.k + (((long)b * a.Hkv + h) * a.N + t0) * 16 + cg;
    uint4 raw[kPrioLoads];
#pragma unroll
    for (int u = 0; u < kPrioLoads; ++u)  // rows past N read as -inf (max) and are skipped (min)
      raw[u] = t0 + kPrioRowLanes * u < a.N
                   ? rows[(long)u * kPrioRowLanes * 16]
                   : make_uint4(0xfc00fc00u, 0xfc00fc00u, 0xfc00fc00u, 0xfc00fc00u);
#pragma unroll
    for (int u = 0; u < kPrioLoads; ++u) {
      const bool ok = t0 + kPrioRowLanes * u < a.N;
      const f16x8_t v = __builtin_bit_cast(f16x8_t, raw[u]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        mx[e] = fmaxf(mx[e], (float)v[e]);
        mn[e] = ok ? fminf(mn[e], (float)v[e]) : mn[e];
      }
    }
  }
  // merge the 16 row lanes: the four of a wave by lane exchanges, the four
  // waves through LDS
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], 16));
    mn[e] = fminf(mn[e], __shfl_xor(mn[e], 16));
    mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], 32));
    mn[e] = fminf(mn[e], __shfl_xor(mn[e], 32));
  }
  const int wv = tid >> 6;
  if ((tid & 63) < 16) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      sx[wv][0][8 * cg + e] = mx[e];
      sx[wv][1][8 * cg + e] = mn[e];
    }
  }
  __syncthreads();
  // thread j: channel j & 127, maximum (j < 128) or minimum
  const int c = tid & 127, w = tid >> 7;
  float r = sx[0][w][c];
#pragma unroll
  for (int l = 1; l < 4; ++l) r = w ? fminf(r, sx[l][w][c]) : fmaxf(r, sx[l][w][c]);
  a.ws[((long)h * a.B * a.nslab + (long)b * a.nslab + s) * 256 + tid] = r;
}

__global__ __launch_bounds__(1024) void k_head_priority_final(PriorityArgs a) {
  __shared__ float part[4][256];
  __shared__ float cm[256];
  const int h = blockIdx.x;
  const int tid = threadIdx.x;
  const int j = tid & 255, q = tid >> 8;  // statistic j of slabs q, q + 4, ...
  const int w = j >> 7;                   // 0: maxima, 1: minima
  const long n = (long)a.B * a.nslab;
  const float* src = a.ws + (long)h * n * 256 + j;
  constexpr int kU = 8;  // loads in flight per thread
  float r[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) r[u] = w ? INFINITY : -INFINITY;
  long i = q;
  for (; i + 4 * (kU - 1) < n; i += 4 * kU) {
    float x[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) x[u] = src[(i + 4 * u) * 256];
#pragma unroll
    for (int u = 0; u < kU; ++u) r[u] = w ? fminf(r[u], x[u]) : fmaxf(r[u], x[u]);
  }
  for (; i < n; i += 4) r[0] = w ? fminf(r[0], src[i * 256]) : fmaxf(r[0], src[i * 256]);
#pragma unroll
  for (int u = 1; u < kU; ++u) r[0] = w ? fminf(r[0], r[u]) : fmaxf(r[0], r[u]);
  part[q][j] = r[0];
  __syncthreads();
  if (tid < 256) {
    float v = part[0][tid];
#pragma unroll
    for (int u = 1; u < 4; ++u) v = w ? fminf(v, part[u][tid]) : fmaxf(v, part[u][tid]);
    cm[tid] = v;
  }
  __syncthreads();
  if (tid < 64) {
    // lane c handles channels c and c + 64
    float gap[2], cmax[2], cmin[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      cmax[u] = cm[tid + 64 * u];
      cmin[u] = cm[128 + tid + 64 * u];
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

size_t head_priority_ws_bytes(int B, int Hkv, int N) {
  const long nslab = ceil_div(N, kPrioSlab);
  return (size_t)Hkv * B * nslab * 256 * sizeof(float);
}

hipError_t launch_head_priority(const PriorityArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(k_head_minmax, dim3(a.Hkv * a.B * a.nslab), dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_head_priority_final, dim3(a.Hkv), dim3(1024), 0, stream, a);
  return hipGetLastError();
}

}  // namespace turbo
