// FlashQ for K and V on gfx950: step 1 (symmetric int8 per 64-token block,
// eq. step1bpq) and step 2 (asymmetric int4/int2 per 64-token channel group,
// eq. step2bpq) with the cache writes of Algorithm 1.
//
// One workgroup of 256 threads handles one (sequence b, KV head h, 64-token
// block j) for both K and V.  The int8 block is staged token-major in LDS;
// step 2 then works channel by channel out of LDS.  k_quantize_kv_blocks is
// step 1 alone with blocks of 32 or 128 tokens (the B_c variants of Table 3);
// it keeps the 64-token storage layouts and writes no cache.
#include "turbo_common.h"
#include "quant_tiles.h"

namespace turbo {

constexpr int kQkvThreads = 256;

struct QuantArgs {
  const uint4* k;  // fp16 [B][Hkv][N][128]
  const uint4* v;
  int Hkv, N, nb;
  int8_t* k8;      // [B][Hkv][nb*64][128]
  int8_t* v8;      // [B][Hkv][nb][128][64]
  float* sk;       // [B][Hkv][nbc]
  float* sv;
  int bc, nbc;     // step-1 block (B_c) and blocks per (b, h): 64 and nb on the cache path
  // cache (pages == nullptr: no step 2)
  uint8_t* pages;
  int8_t* gmeta;
  float* gscale;
  long num_pages, num_slots;
  int page_bytes;
  unsigned long long int2_mask;  // bit h set: KV head h stored with 2 bits
  const int* block_table;        // [B][4*max_groups]
  const int* group_table;        // [B][max_groups]
  int max_groups;
};

// Block amax over the 256 threads (each passes its own max).
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  return r;
}

// Step 1 for one block of 16 kT tokens of one tensor.  Thread (ts = tid>>4,
// cg = tid&15) holds tokens ts + 16*tk (tk < kT) x channels 8cg..8cg+7.
// Writes the int8 tile into LDS (token-major) and returns the block scale;
// rows nr.. of the block are zero, and out_tokmajor receives rows < nw.
template <int kT>
__device__ float quant_block(const uint4* __restrict__ x, int nr, int8_t* tile, float* red,
                             int8_t* __restrict__ out_tokmajor, int nw = 16 * kT) {
  const int tid = threadIdx.x, ts = tid >> 4, cg = tid & 15;
  float f[kT][8];
  float amax = 0.0f;
#pragma unroll
  for (int tk = 0; tk < kT; ++tk) {
    const int t = ts + 16 * tk;
    uint4 raw = make_uint4(0, 0, 0, 0);
    if (t < nr) raw = x[t * 16 + cg];
    f16x8_t h = __builtin_bit_cast(f16x8_t, raw);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      f[tk][e] = (float)h[e];
      amax = fmaxf(amax, fabsf(f[tk][e]));
    }
  }
  amax = block_max(amax, red);
  float s = 0.0f, inv = 0.0f;
  if (amax > 0.0f) {
    s = amax / kQmax;
    inv = kQmax / amax;
  }
#pragma unroll
  for (int tk = 0; tk < kT; ++tk) {
    const int t = ts + 16 * tk;
    int q[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) q[e] = min(119, max(-119, rne_mul(f[tk][e], inv)));
    uint2 packed = make_uint2(pack4(q[0], q[1], q[2], q[3]), pack4(q[4], q[5], q[6], q[7]));
    *reinterpret_cast<uint2*>(tile + t * kTileStride + 8 * cg) = packed;
    if (out_tokmajor && t < nw)
      *reinterpret_cast<uint2*>(out_tokmajor + t * 128 + 8 * cg) = packed;
  }
  return s;
}

__global__ __launch_bounds__(kQkvThreads) void k_quantize_kv(QuantArgs a) {
  __shared__ int8_t tile[64 * kTileStride];
  __shared__ uint8_t ctile[64 * kTileStride];  // K codes, token-major
  __shared__ float red[4];

  const int j = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const long unit = (long)b * a.Hkv + h;
  const int r0 = j * 64;
  const int nr = min(64, a.N - r0);
  const long xoff = (unit * a.N + r0) * 16;  // in uint4 (8 halves)

  // cache destination of this group (full groups with valid table entries)
  bool do_cache = a.pages != nullptr && nr == 64;
  long page[4] = {0, 0, 0, 0};
  long slot = 0;
  if (do_cache) {
    const int* bt = a.block_table + (long)b * 4 * a.max_groups + 4 * j;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      page[p] = bt[p];
      do_cache = do_cache && page[p] >= 0 && page[p] < a.num_pages;
    }
    slot = a.group_table[(long)b * a.max_groups + j];
    do_cache = do_cache && slot >= 0 && slot < a.num_slots;
  }
  const int bits = ((a.int2_mask >> h) & 1ull) ? 2 : 4;
  const int head_off = 512 * (4 * h - 2 * __popcll(a.int2_mask & ((1ull << h) - 1ull)));
  int8_t* meta = a.gmeta + (slot * a.Hkv + h) * 512;

  // ---- K ----
  float s = quant_block<4>(a.k + xoff, nr, tile, red, a.k8 + (unit * a.nb + j) * 8192);
  if (tid == 0) a.sk[unit * a.nb + j] = s;
  __syncthreads();
  if (do_cache)
    compress_k(tile, ctile, bits, meta, a.gscale + (slot * a.Hkv + h) * 2 + 0, s, page, a.pages,
               a.page_bytes, head_off);
  __syncthreads();

  // ---- V ----
  s = quant_block<4>(a.v + xoff, nr, tile, red, nullptr);
  if (tid == 0) a.sv[unit * a.nb + j] = s;
  __syncthreads();
  {
    // channel-major int8 block: thread (c = tid>>1, hh) writes 32 tokens
    const int c = tid >> 1, hh = tid & 1;
    unsigned w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int t = 32 * hh + 4 * i;
      w[i] = pack4(tile[t * kTileStride + c], tile[(t + 1) * kTileStride + c],
                   tile[(t + 2) * kTileStride + c], tile[(t + 3) * kTileStride + c]);
    }
    uint4* dst = reinterpret_cast<uint4*>(a.v8 + (unit * a.nb + j) * 8192 + c * 64 + 32 * hh);
    dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
    dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
  }
  if (do_cache)
    compress_v(tile, bits, meta, a.gscale + (slot * a.Hkv + h) * 2 + 1, s, page, a.pages,
               a.page_bytes, head_off);
}

// Step 1 with BC-token blocks (BC = 32 or 128): one workgroup per (b, h,
// block jb), over the 64 nb rows of the 64-token layouts of k_quantize_kv
// (rows from N on are written as 0; a 32-token block past N writes only
// those zeros).  The scales are per BC block (jb < nbc).  A 128-token block
// whose second half lies past 64 nb writes its first half only.
template <int BC>
__global__ __launch_bounds__(kQkvThreads) void k_quantize_kv_blocks(QuantArgs a) {
  __shared__ int8_t tile[BC * kTileStride];
  __shared__ float red[4];
  const int jb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const long unit = (long)b * a.Hkv + h;
  const int r0 = jb * BC;
  const int nr = max(0, min(BC, a.N - r0));  // 0 for a block past N
  const int nw = min(BC, 64 * a.nb - r0);  // rows the 64-token buffers hold
  const long xoff = (unit * a.N + r0) * 16;
  float s = quant_block<BC / 16>(a.k + xoff, nr, tile, red, a.k8 + (unit * a.nb * 64 + r0) * 128,
                                 nw);
  if (tid == 0 && jb < a.nbc) a.sk[unit * a.nbc + jb] = s;
  __syncthreads();
  s = quant_block<BC / 16>(a.v + xoff, nr, tile, red, nullptr);
  if (tid == 0 && jb < a.nbc) a.sv[unit * a.nbc + jb] = s;
  __syncthreads();
  // channel-major int8 V: token t of the block is column (r0 + t) % 64 of
  // 64-token block (r0 + t) / 64; thread (c = tid>>1, hh) writes 16-token runs
  const int c = tid >> 1, hh = tid & 1;
#pragma unroll
  for (int run = hh; run < BC / 16; run += 2) {
    const int t = 16 * run;
    if (t >= nw) break;
    unsigned w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = pack4(tile[(t + 4 * i) * kTileStride + c], tile[(t + 4 * i + 1) * kTileStride + c],
                   tile[(t + 4 * i + 2) * kTileStride + c], tile[(t + 4 * i + 3) * kTileStride + c]);
    const int g = r0 + t;
    *reinterpret_cast<uint4*>(a.v8 + (unit * a.nb + g / 64) * 8192 + c * 64 + g % 64) =
        make_uint4(w[0], w[1], w[2], w[3]);
  }
}

hipError_t launch_quantize_kv(const QuantArgs& a, int B, hipStream_t stream) {
  // blocks covering the 64 nb buffer rows (2 nb of 32, ceil(nb / 2) of 128)
  if (a.bc == 32) {
    hipLaunchKernelGGL(k_quantize_kv_blocks<32>, dim3(2 * a.nb, a.Hkv, B), dim3(kQkvThreads), 0,
                       stream, a);
  } else if (a.bc == 128) {
    hipLaunchKernelGGL(k_quantize_kv_blocks<128>, dim3((a.nb + 1) / 2, a.Hkv, B),
                       dim3(kQkvThreads), 0, stream, a);
  } else {
    hipLaunchKernelGGL(k_quantize_kv, dim3(a.nb, a.Hkv, B), dim3(kQkvThreads), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace turbo
