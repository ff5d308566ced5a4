// Algorithm 3 (Appendix B) on gfx950: the SAS softmax of every row of a
// float matrix, as a stand-alone operation.  Per row: m = max, e_c =
// SAS(x_c - m) (the same binary32 steps as the attention kernels: y = m - x,
// threshold, LUT[floor y] * POLY(y - floor y)), then e_c / sum_c e_c.
//
// The operation reads and writes each element once, so it is bound by HBM.
// Rows of up to 2048 values are held in the registers of one wave (four
// rows per work-group); longer rows use one 256-thread work-group, in
// registers up to 16384 values and in three streaming passes beyond.
#include "turbo_common.h"
#include "stream_loads.h"

namespace turbo {

struct SasSoftmaxArgs {
  const float* x;  // [rows][cols]
  float* y;        // [rows][cols]
  long rows;
  int cols;
  int vec;         // 1: cols % 4 == 0 and both pointers 16-byte aligned
};

__device__ __forceinline__ float wave_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xf, 0xf, false));
  const unsigned u = __float_as_uint(v);
  auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  return add_xor32(v);
}

// Loads of one row in chunks of four values: chunk i of thread t covers
// columns 4 (t + T i) .. +3; columns past the row read as -inf.  kNT: the row
// is read once (held in registers), so the vector loads stream.
template <int T, bool kNT = false>
__device__ __forceinline__ float4 load4(const float* xr, int C, int vec, int t, int i) {
  const int c = 4 * (t + T * i);
  if (vec && c + 3 < C) {
    if (kNT) {
      const u32x4_t u = load_nt4(xr + c);
      return make_float4(__uint_as_float(u.x), __uint_as_float(u.y), __uint_as_float(u.z),
                         __uint_as_float(u.w));
    }
    return *reinterpret_cast<const float4*>(xr + c);
  }
  float4 r;
  r.x = c < C ? xr[c] : -INFINITY;
  r.y = c + 1 < C ? xr[c + 1] : -INFINITY;
  r.z = c + 2 < C ? xr[c + 2] : -INFINITY;
  r.w = c + 3 < C ? xr[c + 3] : -INFINITY;
  return r;
}

// Stores of one output row in the same chunks.  The output is written once
// and not read again by this launch, so the vector stores stream
// (non-temporal): 3-4 % faster on the 2.7 GB workload.
typedef float f32x4_t __attribute__((ext_vector_type(4)));
template <int T>
__device__ __forceinline__ void store4(float* yr, int C, int vec, int t, int i, float4 v) {
  const int c = 4 * (t + T * i);
  if (vec && c + 3 < C) {
    __builtin_nontemporal_store(f32x4_t{v.x, v.y, v.z, v.w}, reinterpret_cast<f32x4_t*>(yr + c));
    return;
  }
  if (c < C) yr[c] = v.x;
  if (c + 1 < C) yr[c + 1] = v.y;
  if (c + 2 < C) yr[c + 2] = v.z;
  if (c + 3 < C) yr[c + 3] = v.w;
}

__device__ __forceinline__ float4 sas4(float m, float4 v, const float* lut) {
  return make_float4(sas_y(m - v.x, lut), sas_y(m - v.y, lut), sas_y(m - v.z, lut),
                     sas_y(m - v.w, lut));
}

__device__ __forceinline__ float4 div4(float4 v, float s) {
  return make_float4(v.x / s, v.y / s, v.z / s, v.w / s);
}

// One wave per row, the row in registers: NV chunks of four per lane.
template <int NV>
__global__ __launch_bounds__(256) void k_sas_softmax_wave(SasSoftmaxArgs a) {
  __shared__ float lut[8];
  if (threadIdx.x < 8) lut[threadIdx.x] = kLut[threadIdx.x];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= a.rows) return;  // wave-uniform; no barrier follows
  const float* xr = a.x + row * a.cols;
  float* yr = a.y + row * a.cols;
  float4 v[NV];
  float m = -INFINITY;
  // The row's loads are issued at raised priority, ahead of the arithmetic
  // of the other waves of the SIMD.
  __builtin_amdgcn_s_setprio(2);
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = load4<64, true>(xr, a.cols, a.vec, lane, i);
  __builtin_amdgcn_s_setprio(0);
#pragma unroll
  for (int i = 0; i < NV; ++i)
    m = fmaxf(m, fmaxf(fmaxf(v[i].x, v[i].y), fmaxf(v[i].z, v[i].w)));
  m = wave_max_fast(m);
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    v[i] = sas4(m, v[i], lut);
    s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
  }
  s = wave_sum(s);
#pragma unroll
  for (int i = 0; i < NV; ++i) store4<64>(yr, a.cols, a.vec, lane, i, div4(v[i], s));
}

__device__ __forceinline__ float block_reduce(float v, float* red, bool is_max) {
  v = is_max ? wave_max_fast(v) : wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  const float r = is_max ? fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]))
                         : (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

// One 256-thread work-group per row.  NV > 0: the row in registers (NV
// chunks of four per thread); NV == 0: three passes over memory.
template <int NV>
__global__ __launch_bounds__(256) void k_sas_softmax_block(SasSoftmaxArgs a) {
  __shared__ float lut[8];
  __shared__ float red[4];
  const int t = threadIdx.x;
  if (t < 8) lut[t] = kLut[t];
  __syncthreads();
  const long row = blockIdx.x;
  const float* xr = a.x + row * a.cols;
  float* yr = a.y + row * a.cols;
  const int C = a.cols;
  const int nch = (C + 1023) / 1024;  // chunks of four per thread
  if (NV > 0) {
    float4 v[NV > 0 ? NV : 1];
    float m = -INFINITY;
    __builtin_amdgcn_s_setprio(2);  // the row's loads first (2 % on 4096-column rows)
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] = load4<256, true>(xr, C, a.vec, t, i);
    __builtin_amdgcn_s_setprio(0);
#pragma unroll
    for (int i = 0; i < NV; ++i)
      m = fmaxf(m, fmaxf(fmaxf(v[i].x, v[i].y), fmaxf(v[i].z, v[i].w)));
    m = block_reduce(m, red, true);
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      v[i] = sas4(m, v[i], lut);
      s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
    }
    s = block_reduce(s, red, false);
#pragma unroll
    for (int i = 0; i < NV; ++i) store4<256>(yr, C, a.vec, t, i, div4(v[i], s));
  } else {
    float m = -INFINITY;
    for (int i = 0; i < nch; ++i) {
      const float4 v = load4<256>(xr, C, a.vec, t, i);
      m = fmaxf(m, fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w)));
    }
    m = block_reduce(m, red, true);
    float s = 0.0f;
    for (int i = 0; i < nch; ++i) {
      const float4 e = sas4(m, load4<256>(xr, C, a.vec, t, i), lut);
      s += (e.x + e.y) + (e.z + e.w);
    }
    s = block_reduce(s, red, false);
    for (int i = 0; i < nch; ++i)
      store4<256>(yr, C, a.vec, t, i, div4(sas4(m, load4<256>(xr, C, a.vec, t, i), lut), s));
  }
}

hipError_t launch_sas_softmax(const SasSoftmaxArgs& a, hipStream_t stream) {
  const int C = a.cols;
  if (C <= 2048) {
    const dim3 grid((unsigned)((a.rows + 3) / 4));
    if (C <= 256)
      hipLaunchKernelGGL(k_sas_softmax_wave<1>, grid, dim3(256), 0, stream, a);
    else if (C <= 512)
      hipLaunchKernelGGL(k_sas_softmax_wave<2>, grid, dim3(256), 0, stream, a);
    else if (C <= 1024)
      hipLaunchKernelGGL(k_sas_softmax_wave<4>, grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL(k_sas_softmax_wave<8>, grid, dim3(256), 0, stream, a);
  } else {
    const dim3 grid((unsigned)a.rows);
    if (C <= 4096)
      hipLaunchKernelGGL(k_sas_softmax_block<4>, grid, dim3(256), 0, stream, a);
    else if (C <= 8192)
      hipLaunchKernelGGL(k_sas_softmax_block<8>, grid, dim3(256), 0, stream, a);
    else if (C <= 16384)
      hipLaunchKernelGGL(k_sas_softmax_block<16>, grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL(k_sas_softmax_block<0>, grid, dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace turbo
