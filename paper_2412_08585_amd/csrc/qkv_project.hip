// The QKV projection with FlashQ fused into its epilogue (Sec. 5.2: the
// quantization of Q, K and V is folded into the projection that produces
// them), on gfx950.
//
//   [Q | K | V] = X W^T,  X fp16 [B][N][D] (hidden states), W fp16 [F][D]
//   with F = (Hq + 2 Hkv) * 128 output features (query heads, then key
//   heads, then value heads, 128 channels each).
//
// The products accumulate in fp32 on v_mfma_f32_32x32x16_f16 and each output
// is rounded to fp16, the precision the unfused projection would store.  The
// epilogue then applies FlashQ step 1 to every (sequence, head, 64-token
// block) -- the same rule as the prefill prologue for Q and k_quantize_kv for
// K and V -- and, for K and V, step 2 with the paged cache write, through the
// same LDS-tile routines as k_quantize_kv.  Q, K and V never reach HBM in
// fp16.
//
// Tiling.  A work-group of four waves computes a 256-token x 256-feature tile
// (two heads).  The contraction runs in stages of 64 columns: the tile's 256
// X rows and 256 W rows of a stage (128 bytes each) sit in LDS at a 144-byte
// row pitch, so that the 16 lanes of each operand read hit 16 distinct
// 4-bank groups.  There are two LDS stages and two register sets: each
// thread loads its 16 chunks of stage k + 2 into registers at the top of
// stage k and stores them to LDS during stage k + 1, between its MFMA steps
// (one barrier per stage), which gives the loads -- a fifth of which miss
// the XCD's L2 -- more than a stage to land.  Wave (wm, wn) owns tokens
// 128 wm .. +127 and head wn of the pair: 4 x 4 MFMA blocks of 32 x 32, 256
// fp32 accumulators per lane, which live in the AGPR file (one wave per SIMD;
// this file is built as a translation unit of its own, without the VGPR-only
// MFMA form of the attention kernels).  Every operand byte leaves L2 once per
// work-group: X is read once per head pair and W once per 256-token tile.
#include "turbo_common.h"
#include "quant_tiles.h"
#include "qkv_project.h"

namespace turbo {

typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kProjThreads = 256;
constexpr int kPRow = 144;               // LDS bytes per staged row: 128 + 16 (bank spread)
constexpr int kPOp = 256 * kPRow;        // one operand (256 rows) of one stage
constexpr int kPStage = 2 * kPOp;        // X rows, then W rows
constexpr int kEpiTile = 64 * kTileStride;  // one 64 x 128 int8 block (k_quantize_kv layout)
constexpr int kQkvLds = 2 * kPStage;
static_assert(9 * kEpiTile <= kQkvLds, "the epilogue tiles fit in the stages");

__device__ __forceinline__ f32x16_t mfma_f16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8_t, a),
                                                __builtin_bit_cast(h8_t, b), c, 0, 0, 0);
}

// Raw buffer resource over `bytes` bytes at p (gfx9 descriptor word 3: 32-bit
// data format).  Loads at offsets >= bytes return zeros: the rows past N of
// the last token tile and past F of an odd head count.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, bytes, 0x00020000);
}

__device__ __forceinline__ uint4 bload(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// Work-group order.  The dispatcher hands work-group x to XCD x % 8.  When
// the token tiles are a multiple of 8, XCD k owns tiles k, k+8, ... and walks
// them in blocks of (all its tiles) x (8 head pairs): the 32 work-groups
// resident on an XCD then share 4 X tiles and 8 W pairs in its L2.
__device__ __forceinline__ void qkv_tile(int x, int ntiles, int npairs, int& tile, int& pair) {
  if (ntiles % 8 != 0) {
    pair = x % npairs;
    tile = x / npairs;
    return;
  }
  const int k = x % 8, i = x / 8;
  const int ntk = ntiles / 8;   // tiles of this XCD
  const int full = npairs / 8;  // complete groups of 8 pairs
  int tl;
  if (i < full * ntk * 8) {
    const int hg = i / (ntk * 8), rem = i % (ntk * 8);
    tl = rem / 8;
    pair = 8 * hg + rem % 8;
  } else {
    const int r = npairs - 8 * full, rem = i - full * ntk * 8;
    tl = rem / r;
    pair = 8 * full + rem % r;
  }
  tile = tl * 8 + k;
}

// kY = true only for the test hook that also stores the fp16 projection
// (the production instance carries no such store).
template <bool kY>
__global__ __launch_bounds__(kProjThreads, 1) __attribute__((amdgpu_waves_per_eu(1, 1))) void
k_qkv_project(QkvArgs a) {
  __shared__ __align__(16) uint8_t lds[kQkvLds];
  __shared__ float sblk[8];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int wm = wv & 1, wn = wv >> 1;
  const int m = lane & 31, hh = lane >> 5;
  const int nheads = a.Hq + 2 * a.Hkv;
  const int npairs = ceil_div(nheads, 2);
  const int F = 128 * nheads;
  int tile, pair;
  qkv_tile(blockIdx.x, a.B * a.ntile, npairs, tile, pair);
  const int b = tile / a.ntile;
  const int t0 = (tile % a.ntile) * kQkvTileTokens;

  // ---- staging: thread (row sr + 32 j, 16-byte chunk sc), j = 0..7 ---------
  // one load instruction reads 8 whole 128-byte rows of a stage
  const int sr = tid >> 3, sc = tid & 7;
  const unsigned D2 = 2u * (unsigned)a.D;  // bytes per row
  const __amdgpu_buffer_rsrc_t xrs =
      rows_rsrc(static_cast<const _Float16*>(a.x) + (long)b * a.N * a.D, a.N * (int)D2);
  const __amdgpu_buffer_rsrc_t wrs = rows_rsrc(a.w, F * (int)D2);
  const unsigned lv = (unsigned)sr * D2 + 16u * (unsigned)sc;  // lane part of both offsets
  const unsigned xs0 = (unsigned)t0 * D2, ws0 = (unsigned)(256 * pair) * D2;
  const unsigned sj = 32u * D2;  // 32 rows
  const int sdst = sr * kPRow + 16 * sc;

  // two register sets of a stage's 16 chunks (8 X, then 8 W): the loads of
  // stage k + 2 are issued at the top of stage k and stored to LDS during
  // stage k + 1
  uint4 g[2][16];
  auto gload = [&](auto setc, int kk) {
    constexpr int S = decltype(setc)::value;
    const unsigned kb = 128u * (unsigned)kk;  // 64 fp16 columns per stage
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      g[S][j] = bload(xrs, lv, xs0 + j * sj + kb);
      g[S][8 + j] = bload(wrs, lv, ws0 + j * sj + kb);
    }
  };
  f32x16_t acc[4][4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = f32x16_t{};

  // operand reads: A (X rows) row 128 wm + 32 mb + m, B (W rows) row
  // 128 wn + 32 nb + m; contraction slot (step s, lane half hh, element e) is
  // column 16 s + 8 hh + e of the stage for both operands
  const int aA = (128 * wm + m) * kPRow + 16 * hh;
  const int aB = kPOp + (128 * wn + m) * kPRow + 16 * hh;
  // one stage; the operands of step s + 1 are read while the 16 MFMAs of
  // step s run, and the next stage's chunks (register set S) are stored
  // into the other LDS buffer between the steps, so that the stores overlap
  // the MFMAs instead of stalling the barrier
  auto compute = [&](int st, auto setc) {
    constexpr int S = decltype(setc)::value;
    const uint8_t* sa = lds + st * kPStage + aA;
    const uint8_t* sb = lds + st * kPStage + aB;
    uint8_t* d = lds + (st ^ 1) * kPStage + sdst;
    uint4 A[2][4], Bo[2][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      A[0][i] = *reinterpret_cast<const uint4*>(sa + i * 32 * kPRow);
      Bo[0][i] = *reinterpret_cast<const uint4*>(sb + i * 32 * kPRow);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int cu = s & 1, nx = cu ^ 1;
      if (s < 3) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          A[nx][i] = *reinterpret_cast<const uint4*>(sa + i * 32 * kPRow + 32 * (s + 1));
          Bo[nx][i] = *reinterpret_cast<const uint4*>(sb + i * 32 * kPRow + 32 * (s + 1));
        }
      }
      // four of the next stage's 16 chunks per step: X chunks 0-3, X 4-7,
      // W 0-3, W 4-7
#pragma unroll
      for (int q = 4 * s; q < 4 * s + 4; ++q) {
        const int j = q & 7;
        *reinterpret_cast<uint4*>(d + (q < 8 ? 0 : kPOp) + j * 32 * kPRow) = g[S][q];
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = mfma_f16(A[cu][mb], Bo[cu][nb], acc[mb][nb]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  const int nk = a.D / 64;
  // every load is issued on every path (the stage index is clamped at the
  // end), so the waits the compiler places before each use stay exact
  gload(std::integral_constant<int, 0>{}, 0);
  {
    uint8_t* d = lds + sdst;  // stage 0 into LDS 0
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      *reinterpret_cast<uint4*>(d + j * 32 * kPRow) = g[0][j];
      *reinterpret_cast<uint4*>(d + kPOp + j * 32 * kPRow) = g[0][8 + j];
    }
  }
  gload(std::integral_constant<int, 1>{}, min(1, nk - 1));
  __syncthreads();
  for (int kk = 0; kk + 1 < nk; kk += 2) {
    // stage kk from LDS 0; set 0 (free) takes stage kk + 2; set 1 (stage
    // kk + 1) goes to LDS 1, whose last readers finished before the barrier
    gload(std::integral_constant<int, 0>{}, min(kk + 2, nk - 1));
    // keep the prefetch at the top (the scheduler would sink it to its use)
    __builtin_amdgcn_sched_barrier(0);
    compute(0, std::integral_constant<int, 1>{});
    __syncthreads();
    gload(std::integral_constant<int, 1>{}, min(kk + 3, nk - 1));
    __builtin_amdgcn_sched_barrier(0);
    compute(1, std::integral_constant<int, 0>{});
    __syncthreads();
  }
  if (nk & 1) compute(0, std::integral_constant<int, 1>{});  // the last stage of an odd count
  __syncthreads();

  // ---- epilogue: fp16 outputs, FlashQ step 1 per 64-token block --------------
  // lane (m, hh), register r of (mb, nb) <-> token 128 wm + 32 mb + 8 (r/4) +
  // 4 hh + r%4 of the tile, channel 32 nb + m of head 2 pair + wn; FlashQ
  // block i = mb >> 1 of the wave is block 2 wm + i of the tile
  const int head = 2 * pair + wn;
  const bool hv = head < nheads;  // wave-uniform (an odd head count leaves one out)
  // one block at a time (128 accumulators of a lane), which bounds the
  // registers the AGPR -> VGPR copies take; the stages are free for the tiles
  // since the loop's last barrier
  float sc_[2];
  // block i of the wave: kFull when all its 64 tokens are below N (the
  // common case: no per-element masking), else rows nv.. are masked out
  auto block = [&](auto ic, auto fullc) {
    constexpr int i = decltype(ic)::value;
    constexpr bool kFull = decltype(fullc)::value;
    const int nv = a.N - (t0 + 128 * wm + 64 * i);  // valid rows of the block
    // max |fp16(y)| = fp16(max |y|): rounding is monotone and symmetric, so
    // the first pass needs no conversion
    float amax = 0.0f;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = 32 * mi + 8 * (r >> 2) + 4 * hh + (r & 3);
          amax = fmaxf(amax, (kFull || row < nv) ? fabsf(acc[2 * i + mi][nb][r]) : 0.0f);
          if constexpr (kY) {
            if (hv && (kFull || row < nv))
              a.y[((long)b * a.N + t0 + 128 * wm + 64 * i + row) * (long)F + 128 * head + 32 * nb +
                  m] = (_Float16)acc[2 * i + mi][nb][r];
          }
        }
    amax = (float)(_Float16)amax;
    amax = wave_max_fast(amax);
    float inv = 0.0f;
    sc_[i] = 0.0f;
    if (amax > 0.0f) {
      sc_[i] = amax / kQmax;
      inv = kQmax / amax;
    }
    int8_t* tw = reinterpret_cast<int8_t*>(lds) + (4 * wn + 2 * wm + i) * kEpiTile;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = 32 * mi + 8 * (r >> 2) + 4 * hh + (r & 3);
          const float y = (float)(_Float16)acc[2 * i + mi][nb][r];
          const int q = min(119, max(-119, rne_mul(y, inv)));
          tw[row * kTileStride + 32 * nb + m] = (int8_t)((kFull || row < nv) ? q : 0);
        }
    if (lane == 0) sblk[4 * wn + 2 * wm + i] = sc_[i];
  };
  // (i a compile-time constant: acc is indexed with it)
  auto run = [&](auto ic) {
    constexpr int i = decltype(ic)::value;
    if (t0 + 128 * wm + 64 * i + 64 <= a.N)  // wave-uniform
      block(ic, std::true_type{});
    else
      block(ic, std::false_type{});
  };
  run(std::integral_constant<int, 0>{});
  // the next block's AGPR reads stay below this point
  __builtin_amdgcn_sched_barrier(0);
  run(std::integral_constant<int, 1>{});
  __syncthreads();

  // ---- Q8 / K8 / V8 and the block scales: each wave its own two tiles --------
  if (hv) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int8_t* tw = reinterpret_cast<const int8_t*>(lds) + (4 * wn + 2 * wm + i) * kEpiTile;
      const int jb = (t0 + 128 * wm + 64 * i) / 64;  // FlashQ block index in the sequence
      if (jb >= a.nb) continue;                      // wave-uniform
      if (head < a.Hq + a.Hkv) {
        // token-major int8 rows (Q8 or K8) and the block scale
        const bool isq = head < a.Hq;
        const int hq = isq ? head : head - a.Hq;
        const long unit = (long)b * (isq ? a.Hq : a.Hkv) + hq;
        int8_t* dst = (isq ? a.q8 : a.k8) + (unit * a.nb + jb) * 8192;
#pragma unroll
        for (int it = 0; it < 16; ++it) {
          const int row = 4 * it + (lane >> 4), c8 = lane & 15;
          *reinterpret_cast<uint2*>(dst + row * 128 + 8 * c8) =
              *reinterpret_cast<const uint2*>(tw + row * kTileStride + 8 * c8);
        }
        if (lane == 0) (isq ? a.sq : a.sk)[unit * a.nb + jb] = sc_[i];
      } else {
        // channel-major V8 block: lane = channel pair
        const long unit = (long)b * a.Hkv + (head - a.Hq - a.Hkv);
        int8_t* dst = a.v8 + (unit * a.nb + jb) * 8192;
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
          const int c = 2 * lane + cc;
          unsigned wd[16];
#pragma unroll
          for (int k = 0; k < 16; ++k) {
            const int t = 4 * k;
            wd[k] = pack4(tw[t * kTileStride + c], tw[(t + 1) * kTileStride + c],
                          tw[(t + 2) * kTileStride + c], tw[(t + 3) * kTileStride + c]);
          }
          uint4* o = reinterpret_cast<uint4*>(dst + c * 64);
#pragma unroll
          for (int k = 0; k < 4; ++k)
            o[k] = make_uint4(wd[4 * k], wd[4 * k + 1], wd[4 * k + 2], wd[4 * k + 3]);
        }
        if (lane == 0) a.sv[unit * a.nb + jb] = sc_[i];
      }
    }
  }

  // ---- step 2 and the cache write (K and V heads, full blocks) ---------------
  if (a.pages == nullptr) return;  // work-group uniform
  uint8_t* ctile = lds + 8 * kEpiTile;
  for (int hl = 0; hl < 2; ++hl) {
    const int hd = 2 * pair + hl;
    if (hd < a.Hq || hd >= nheads) continue;  // work-group uniform
    const bool isk = hd < a.Hq + a.Hkv;
    const int hkv = isk ? hd - a.Hq : hd - a.Hq - a.Hkv;
    const int bits = ((a.int2_mask >> hkv) & 1ull) ? 2 : 4;
    const int head_off = 512 * (4 * hkv - 2 * __popcll(a.int2_mask & ((1ull << hkv) - 1ull)));
    for (int w = 0; w < 4; ++w) {
      const int g = (t0 + 64 * w) / 64;
      if (t0 + 64 * w + 64 > a.N || g >= a.max_groups) break;  // uniform
      long page[4];
      bool ok = true;
      const int* bt = a.block_table + (long)b * 4 * a.max_groups + 4 * g;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        page[p] = bt[p];
        ok = ok && page[p] >= 0 && page[p] < a.num_pages;
      }
      const long slot = a.group_table[(long)b * a.max_groups + g];
      if (!ok || slot < 0 || slot >= a.num_slots) continue;  // uniform
      int8_t* meta = a.gmeta + (slot * a.Hkv + hkv) * 512;
      const int8_t* tb = reinterpret_cast<const int8_t*>(lds) + (4 * hl + w) * kEpiTile;
      if (isk)
        compress_k(tb, ctile, bits, meta, a.gscale + (slot * a.Hkv + hkv) * 2 + 0, sblk[4 * hl + w],
                   page, a.pages, a.page_bytes, head_off);
      else
        compress_v(tb, bits, meta, a.gscale + (slot * a.Hkv + hkv) * 2 + 1, sblk[4 * hl + w], page,
                   a.pages, a.page_bytes, head_off);
      __syncthreads();
    }
  }
}

hipError_t launch_qkv_project(const QkvArgs& a, hipStream_t stream) {
  const int total = a.B * a.ntile * ceil_div(a.Hq + 2 * a.Hkv, 2);
  if (a.y)
    hipLaunchKernelGGL(k_qkv_project<true>, dim3(total), dim3(kProjThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(k_qkv_project<false>, dim3(total), dim3(kProjThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace turbo
