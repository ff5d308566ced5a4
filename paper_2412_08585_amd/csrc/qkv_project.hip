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
// (two heads).  The contraction runs in stages of 32 columns: the tile's 256
// X rows and 256 W rows of a stage (64 bytes each, 16-byte chunks swizzled
// by row so that the operand reads are free of bank conflicts) are loaded
// straight into LDS by buffer loads, into a ring of four stage buffers, four
// stages ahead.  Each wave reads the next stage's operands into registers
// while the current stage's MFMAs run, and issues its part of the loads
// spread between those MFMAs; one barrier per stage.  Wave (wm, wn) owns
// tokens 128 wm .. +127 and head wn of the pair: 4 x 4 MFMA blocks of
// 32 x 32, 256 fp32 accumulators per lane, which live in the AGPR file (one
// wave per SIMD; this file is built as a translation unit of its own,
// without the VGPR-only MFMA form of the attention kernels).  Every operand
// byte leaves L2 once per work-group: X is read once per head pair and W
// once per 256-token tile.
#include "turbo_common.h"
#include "quant_tiles.h"
#include "qkv_project.h"

namespace turbo {

typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kProjThreads = 256;
constexpr int kPRow = 64;                // LDS bytes per staged row: 32 fp16 columns
constexpr int kPOp = 256 * kPRow;        // one operand (256 rows) of one stage
constexpr int kPStage = 2 * kPOp;        // X rows, then W rows
constexpr int kEpiTile = 64 * kTileStride;  // one 64 x 128 int8 block (k_quantize_kv layout)
static_assert(3 * kEpiTile <= kPStage, "three epilogue tiles fit in a stage");

__device__ __forceinline__ f32x16_t mfma_f16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8_t, a),
                                                __builtin_bit_cast(h8_t, b), c, 0, 0, 0);
}

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer resource over `bytes` bytes at p, as the four descriptor words
// (word 3: 32-bit data format).  Loads at offsets >= bytes return zeros: the
// rows past N of the last token tile and past F of an odd head count.
__device__ __forceinline__ i32x4 rows_words(const void* p, int bytes) {
  const unsigned long long a = (unsigned long long)p;
  return i32x4{(int)(unsigned)a, (int)((unsigned)(a >> 32) & 0xffffu), bytes, 0x00020000};
}

// 16 bytes per lane from the buffer (offsets voff + soff) into LDS at dst +
// 16 * lane (the wave-uniform LDS address goes through M0; the nop keeps the
// load one cycle away from the compiler's write of M0).
__device__ __forceinline__ void lds_load16(i32x4 r, unsigned voff, unsigned soff, uint8_t* dst) {
  const unsigned la = (unsigned)(unsigned long)(__attribute__((address_space(3))) uint8_t*)dst;
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :: "v"(voff), "s"(r), "s"(soff), "{m0}"(la) : "memory");
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
  // four stages, each its own array: the compiler then sees that the loads
  // into one stage and the operand reads of another do not overlap
  __shared__ __align__(16) uint8_t st0[kPStage], st1[kPStage], st2[kPStage], st3[kPStage];
  __shared__ float sblk[8];
  const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wv & 1, wn = wv >> 1;
  const int m = lane & 31, hh = lane >> 5;
  const int nheads = a.Hq + 2 * a.Hkv;
  const int npairs = ceil_div(nheads, 2);
  const int F = 128 * nheads;
  int tile, pair;
  qkv_tile(blockIdx.x, a.B * a.ntile, npairs, tile, pair);
  const int b = tile / a.ntile;
  const int t0 = (tile % a.ntile) * kQkvTileTokens;

  // ---- staging: buffer loads straight into LDS, four stages of 32 columns ----
  // chunk c of staged row r sits at chunk position c ^ ((r >> 2) & 3).  Per
  // stage a wave issues 4 X and 4 W loads; load i of wave w fills rows
  // 16 (4 w + i) .. +15 (1 KiB): lane L takes row + (L >> 2), position L & 3,
  // i.e. source chunk (L & 3) ^ ((L >> 4) & 3).
  const unsigned D2 = 2u * (unsigned)a.D;  // bytes per row
  const unsigned vo = (unsigned)(lane >> 2) * D2 + 16u * (unsigned)((lane & 3) ^ ((lane >> 4) & 3));
  const unsigned xs0 = (unsigned)t0 * D2, ws0 = (unsigned)(256 * pair) * D2;
  // The loads are written as inline assembly: the compiler then neither
  // waits for them before every LDS read nor counts them in its own waits
  // (no other vector-memory operation is in flight during the loop).
  const i32x4 xr = rows_words(static_cast<const _Float16*>(a.x) + (long)b * a.N * a.D, a.N * (int)D2);
  const i32x4 wr = rows_words(a.w, F * (int)D2);
  // load j (0..7) of this wave's part of a stage: X rows (j even) or W rows
  // (j odd) 16 (4 w + j / 2) .. +15
  auto dma_j = [&](uint8_t* st, int kk, int j) {
    const unsigned kb = 64u * (unsigned)kk;  // 32 fp16 columns per stage
    const int r0 = 16 * (4 * wv + (j >> 1));
    if (j & 1)
      lds_load16(wr, vo, ws0 + (unsigned)r0 * D2 + kb, st + kPOp + r0 * kPRow);
    else
      lds_load16(xr, vo, xs0 + (unsigned)r0 * D2 + kb, st + r0 * kPRow);
  };
  auto dma = [&](uint8_t* st, int kk) {
#pragma unroll
    for (int j = 0; j < 8; ++j) dma_j(st, kk, j);
  };
  f32x16_t acc[4][4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = f32x16_t{};

  // operand reads: row 128 wm + 32 mb + m (A) / 128 wn + 32 nb + m (B);
  // contraction slot (step s, half hh, element e) = column 16 s + 8 hh + e,
  // chunk 2 s + hh at position (2 s + hh) ^ ((m >> 2) & 3)
  const int sw = (m >> 2) & 3;
  const int ao0 = m * kPRow + 16 * ((0 + hh) ^ sw), ao1 = m * kPRow + 16 * ((2 + hh) ^ sw);
  const int aA = 128 * wm * kPRow, aB = kPOp + 128 * wn * kPRow;
  // operands of one stage in registers: [k-step][block]
  typedef uint4 StageOps[2][4];
  auto read_stage = [&](const uint8_t* st, StageOps& A, StageOps& Bo) {
    const uint8_t* sa = st + aA;
    const uint8_t* sb = st + aB;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      A[0][i] = *reinterpret_cast<const uint4*>(sa + ao0 + i * 32 * kPRow);
      Bo[0][i] = *reinterpret_cast<const uint4*>(sb + ao0 + i * 32 * kPRow);
      A[1][i] = *reinterpret_cast<const uint4*>(sa + ao1 + i * 32 * kPRow);
      Bo[1][i] = *reinterpret_cast<const uint4*>(sb + ao1 + i * 32 * kPRow);
    }
  };
  auto mma = [&](const StageOps& A, const StageOps& Bo, int s) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = mfma_f16(A[s][mb], Bo[s][nb], acc[mb][nb]);
  };
  const int nk = a.D / 32;
  // The loads write LDS behind the compiler's back: their completion is
  // waited for by hand (a wave's loads complete in order, eight per stage),
  // and a plain s_barrier then covers the other waves' parts (__syncthreads
  // would also wait for the loads still in flight).  Step k runs stage k's
  // MFMAs from registers, reads stage k + 1 into the other register set and
  // loads stage k + 4 into the slot of stage k; its closing barrier makes
  // stage k + 2 visible (16 loads, stages k + 3 and k + 4, may still be in
  // flight) and tells that every wave has read stage k + 1.  Past the end
  // the last stage is loaded again, so that every step issues the same
  // number of loads.
  StageOps A0, B0, A1, B1;
  dma(st0, 0);
  dma(st1, min(1, nk - 1));
  dma(st2, min(2, nk - 1));
  dma(st3, min(3, nk - 1));
  asm volatile("s_waitcnt vmcnt(24)\n\ts_barrier" ::: "memory");
  read_stage(st0, A0, B0);
  __builtin_amdgcn_s_waitcnt(0xC07F);
  asm volatile("s_waitcnt vmcnt(16)\n\ts_barrier" ::: "memory");
  // step k: the slot of stage k (in registers since step k - 1, and every
  // wave has passed the barrier after that read) takes stage k + 4
  auto step = [&](uint8_t* slot_k, const uint8_t* slot_k1, StageOps& Ak, StageOps& Bk,
                  StageOps& An, StageOps& Bn, int k) {
    // the stage's 32 MFMAs in eight groups of four, each followed by one
    // load of stage k + 4 and two operand reads of stage k + 1
    const uint8_t* sa = slot_k1 + aA;
    const uint8_t* sb = slot_k1 + aB;
    const int kn = min(k + 4, nk - 1);
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      const int s_ = g >> 2, q = g & 3;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) acc[q][nb] = mfma_f16(Ak[s_][q], Bk[s_][nb], acc[q][nb]);
      __builtin_amdgcn_sched_barrier(0);
      dma_j(slot_k, kn, g);
      // reads: group g fetches block (g >> 1) of k-step (g & 1), A and B
      const int rb = g >> 1, rs = g & 1;
      An[rs][rb] = *reinterpret_cast<const uint4*>(sa + (rs ? ao1 : ao0) + rb * 32 * kPRow);
      Bn[rs][rb] = *reinterpret_cast<const uint4*>(sb + (rs ? ao1 : ao0) + rb * 32 * kPRow);
      __builtin_amdgcn_sched_barrier(0);
    }
    // lgkmcnt(0) through the builtin, so that the compiler knows the operand
    // reads have landed; vmcnt(16) for the hidden loads by hand
    __builtin_amdgcn_s_waitcnt(0xC07F);
    asm volatile("s_waitcnt vmcnt(16)\n\ts_barrier" ::: "memory");
  };
  for (int k = 0; k < nk; k += 4) {
    step(st0, st1, A0, B0, A1, B1, k);
    if (k + 1 < nk) step(st1, st2, A1, B1, A0, B0, k + 1);
    if (k + 2 < nk) step(st2, st3, A0, B0, A1, B1, k + 2);
    if (k + 3 < nk) step(st3, st0, A1, B1, A0, B0, k + 3);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // ---- epilogue: fp16 outputs, FlashQ step 1 per 64-token block --------------
  // lane (m, hh), register r of (mb, nb) <-> token 128 wm + 32 mb + 8 (r/4) +
  // 4 hh + r%4 of the tile, channel 32 nb + m of head 2 pair + wn; FlashQ
  // block i = mb >> 1 of the wave is block 2 wm + i of the tile
  const int head = 2 * pair + wn;
  const bool hv = head < nheads;  // wave-uniform (an odd head count leaves one out)
  // epilogue tile t (0..8) in stage t / 3, slot t % 3
  auto etile = [&](int t) -> uint8_t* {
    uint8_t* st = t < 3 ? st0 : (t < 6 ? st1 : st2);
    return st + (t % 3) * kEpiTile;
  };
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
    int8_t* tw = reinterpret_cast<int8_t*>(etile(4 * wn + 2 * wm + i));
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
      const int8_t* tw = reinterpret_cast<const int8_t*>(etile(4 * wn + 2 * wm + i));
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
  uint8_t* ctile = etile(8);
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
      const int8_t* tb = reinterpret_cast<const int8_t*>(etile(4 * hl + w));
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
