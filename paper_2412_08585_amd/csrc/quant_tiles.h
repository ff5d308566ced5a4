// FlashQ step 2 on an int8 block staged token-major in LDS, and the paged
// cache writes of its codes (Sec. 3.1 step 2, Algorithm 1): the routines the
// K/V quantization kernel and the fused QKV projection share.  Each routine is
// executed by all 256 threads of a work-group.
#pragma once

#include "turbo_common.h"

namespace turbo {

constexpr int kTileStride = 136;  // LDS row stride (bytes) of the int8 tile

// Step 2 for one channel group: thread (c = tid>>1, hh = tid&1) covers
// channel c, tokens 32hh..32hh+31 of the LDS tile.  Returns the codes of its
// 32 tokens in code[] and writes s/z to meta (hh == 0 threads).
static __device__ void step2_channel(const int8_t* tile, int bits, int8_t* meta_s, int8_t* meta_z,
                              int* code) {
  const int tid = threadIdx.x, c = tid >> 1, hh = tid & 1;
  int q[32];
  int mn = 127, mx = -128;
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    q[i] = tile[(32 * hh + i) * kTileStride + c];
    mn = min(mn, q[i]);
    mx = max(mx, q[i]);
  }
  mn = min(mn, __shfl_xor(mn, 1));
  mx = max(mx, __shfl_xor(mx, 1));
  const int levels = (1 << bits) - 1;
  const int s = max(1, (mx - mn + levels - 1) / levels);
  // floor(num / (2s)) for num <= 2*238 + 80 as (num * M) >> 20 with
  // M = 2^20 / (2s) + 1 (exact on that whole range).
  const int M = (1 << 20) / (2 * s) + 1;
#pragma unroll
  for (int i = 0; i < 32; ++i) code[i] = ((2 * (q[i] - mn) + s) * M) >> 20;
  if (hh == 0) {
    meta_s[c] = (int8_t)s;
    meta_z[c] = (int8_t)mn;
  }
}

// Step 2 of the K group staged token-major in `tile` (LDS), its group
// metadata and float scale, and the token-major packing of the codes into
// the four pages of the group (head region at head_off).
static __device__ void compress_k(const int8_t* tile, uint8_t* ctile, int bits, int8_t* meta,
                           float* gscale_k, float s, const long (&page)[4], uint8_t* pages,
                           int page_bytes, int head_off) {
  const int tid = threadIdx.x;
  int code[32];
  step2_channel(tile, bits, meta, meta + 128, code);
  if (tid == 0) *gscale_k = s;
  const int c = tid >> 1, hh = tid & 1;
#pragma unroll
  for (int i = 0; i < 32; ++i) ctile[(32 * hh + i) * kTileStride + c] = (uint8_t)code[i];
  __syncthreads();
  // token-major packing: thread (t = tid>>2, chunk = tid&3) packs 32 channels
  const int t = tid >> 2, ch = tid & 3;
  const uint8_t* src = ctile + t * kTileStride + 32 * ch;
  uint8_t* dst = pages + page[t >> 4] * page_bytes + head_off + (t & 15) * 16 * bits;
  if (bits == 4) {
    unsigned w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      unsigned x = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) x |= (unsigned)src[8 * i + e] << (4 * e);
      w[i] = x;
    }
    *reinterpret_cast<uint4*>(dst + 16 * ch) = make_uint4(w[0], w[1], w[2], w[3]);
  } else {
    unsigned w[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      unsigned x = 0;
#pragma unroll
      for (int e = 0; e < 16; ++e) x |= (unsigned)src[16 * i + e] << (2 * e);
      w[i] = x;
    }
    *reinterpret_cast<uint2*>(dst + 8 * ch) = make_uint2(w[0], w[1]);
  }
}

// Step 2 of the V group staged token-major in `tile`, its metadata and float
// scale, and the channel-major packing of the codes into the group's pages.
static __device__ void compress_v(const int8_t* tile, int bits, int8_t* meta, float* gscale_v, float s,
                           const long (&page)[4], uint8_t* pages, int page_bytes, int head_off) {
  const int tid = threadIdx.x;
  int code[32];
  step2_channel(tile, bits, meta + 256, meta + 384, code);
  if (tid == 0) *gscale_v = s;
  // channel-major packing: tokens 32hh..32hh+31 are pages 2hh, 2hh+1
  const int c = tid >> 1, hh = tid & 1;
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    uint8_t* dst = pages + page[2 * hh + pp] * page_bytes + head_off + 256 * bits + c * 2 * bits;
    if (bits == 4) {
      unsigned lo = 0, hi = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        lo |= (unsigned)code[16 * pp + e] << (4 * e);
        hi |= (unsigned)code[16 * pp + 8 + e] << (4 * e);
      }
      *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
    } else {
      unsigned x = 0;
#pragma unroll
      for (int e = 0; e < 16; ++e) x |= (unsigned)code[16 * pp + e] << (2 * e);
      *reinterpret_cast<unsigned*>(dst) = x;
    }
  }
}

}  // namespace turbo
