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
// Work split.  A work-group of four waves owns 256 tokens of one sequence and
// one head (128 features); wave w owns the 64-token FlashQ block w, so the
// block maximum is a wave reduction.  Per 64-wide step of D, the W slice of
// the head (128 x 64 fp16) is staged in LDS (two stages) and shared by the
// four waves; each wave reads its own X rows straight into MFMA registers
// (one step ahead).  A lane's 32 contiguous halves of a row serve four
// k16-steps: contraction slot (step s, lane half h, element j) is column
// 32h + 8s + j of the slice, the same for both operands.
#include "turbo_common.h"

namespace turbo {

typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

struct QkvArgs {
  const uint4* x;  // fp16 [B][N][D]
  const uint4* w;  // fp16 [F][D]
  int B, N, D, Hq, Hkv, nb, ntile;
  int8_t* q8;      // [B][Hq][nb*64][128]
  float* sq;       // [B][Hq][nb]
  int8_t* k8;      // [B][Hkv][nb*64][128]
  int8_t* v8;      // [B][Hkv][nb][128][64]
  float* sk;       // [B][Hkv][nb]
  float* sv;
  // paged cache (pages == nullptr: none)
  uint8_t* pages;
  int8_t* gmeta;
  float* gscale;
  long num_pages, num_slots;
  int page_bytes;
  unsigned long long int2_mask;
  const int* block_table;  // [B][4*max_groups]
  const int* group_table;  // [B][max_groups]
  int max_groups;
  _Float16* y;     // test hook: the fp16 projection [B][N][F] (null: not written)
};

constexpr int kProjThreads = 256;
constexpr int kWRow = 144;                   // LDS bytes per W row: 128 + 16 (bank spread)
constexpr int kWStage = 128 * kWRow;         // one 128 x 64 fp16 slice
constexpr int kEpiTile = 64 * kTileStride;   // one 64 x 128 int8 block (k_quantize_kv layout)
constexpr int kQkvLds = (2 * kWStage > 5 * kEpiTile) ? 2 * kWStage : 5 * kEpiTile;

__device__ __forceinline__ f32x16_t mfma_f16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8_t, a),
                                                __builtin_bit_cast(h8_t, b), c, 0, 0, 0);
}

// Work-group order.  The dispatcher hands work-group x to XCD x % 8.  When
// the token tiles are a multiple of 8, XCD k owns tiles k, k+8, ... and walks
// them in blocks of (all its tiles) x (8 heads): the ~64 work-groups resident
// on an XCD then share 8 X tiles and 8 W heads in its L2, so X is fetched
// about nheads/8 times and W about ntiles/8 times in all (tile-major order
// would fetch all of W once per tile).
__device__ __forceinline__ void qkv_tile(int x, int ntiles, int nheads, int& tile, int& head) {
  if (ntiles % 8 != 0) {
    head = x % nheads;
    tile = x / nheads;
    return;
  }
  const int k = x % 8, i = x / 8;
  const int ntk = ntiles / 8;        // tiles of this XCD
  const int full = nheads / 8;       // complete groups of 8 heads
  int tl;
  if (i < full * ntk * 8) {
    const int hg = i / (ntk * 8), rem = i % (ntk * 8);
    tl = rem / 8;
    head = 8 * hg + rem % 8;
  } else {
    const int r = nheads - 8 * full, rem = i - full * ntk * 8;
    tl = rem / r;
    head = 8 * full + rem % r;
  }
  tile = tl * 8 + k;
}

// kY = true only for the test hook that also stores the fp16 projection
// (the production instance carries no such store).
template <bool kY>
__global__ __launch_bounds__(kProjThreads, 2) void k_qkv_project(QkvArgs a) {
  __shared__ __align__(16) uint8_t lds[kQkvLds];
  __shared__ float sblk[4];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int h = lane >> 5, m = lane & 31;
  const int nheads = a.Hq + 2 * a.Hkv;
  int tile, head;
  qkv_tile(blockIdx.x, a.B * a.ntile, nheads, tile, head);
  const int b = tile / a.ntile;
  const int t0 = (tile % a.ntile) * 256;
  const int n0 = t0 + 64 * wv;  // first token of this wave's block
  const int dq = a.D / 8;       // uint4 per row

  // this lane's two X rows (clamped into the sequence; rows >= N are masked
  // out in the epilogue) and the W row it stages
  const uint4* xr[2];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    const int n = min(n0 + 32 * mb + m, a.N - 1);
    xr[mb] = a.x + ((long)b * a.N + n) * dq + 4 * h;
  }
  // W staging: thread (row 32 j + tid/8, 16-byte chunk tid%8) for j = 0..3, so
  // one load instruction reads 8 whole 128-byte rows of the slice
  const int wrow = tid >> 3, wc = tid & 7;
  const uint4* wr = a.w + ((long)head * 128 + wrow) * dq + wc;
  const long wj = 32L * dq;  // 32 rows
  uint8_t* wdst = lds + wrow * kWRow + 16 * wc;

  f32x16_t acc[2][4];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = f32x16_t{};

  // X operands in two half-step register sets: P holds k16-slots 0-1 of a
  // step, R slots 2-3.  R is loaded at the top of its step and P (for the
  // next step) after slots 0-1 are done, so each load has half a step of
  // MFMAs to land, and each set is waited for only when it is used.  The W
  // slice of the next step is loaded at the top and stored to the other LDS
  // stage at the end of the step.
  uint4 P[2][2], R[2][2];
  const int nk = a.D / 64;
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) P[mb][j] = xr[mb][j];
  {
    const uint4 w0 = wr[0], w1 = wr[wj], w2 = wr[2 * wj], w3 = wr[3 * wj];
    *reinterpret_cast<uint4*>(wdst) = w0;
    *reinterpret_cast<uint4*>(wdst + 32 * kWRow) = w1;
    *reinterpret_cast<uint4*>(wdst + 64 * kWRow) = w2;
    *reinterpret_cast<uint4*>(wdst + 96 * kWRow) = w3;
  }
  __syncthreads();
  // every load is issued on every path (the index is clamped at the end), so
  // the waits the compiler places before each use stay exact
  for (int kk = 0; kk < nk; ++kk) {
    const int st = kk & 1, kn = min(kk + 1, nk - 1);
    const uint4* wn = wr + kn * 8;
    const uint4 w0 = wn[0], w1 = wn[wj], w2 = wn[2 * wj], w3 = wn[3 * wj];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) R[mb][j] = xr[mb][kk * 8 + 2 + j];
    // keep the prefetches where they are: issued early, their latency hides
    // behind MFMAs (the scheduler would otherwise sink them to their use)
    __builtin_amdgcn_sched_barrier(0);
    const uint8_t* base = lds + st * kWStage + m * kWRow + 64 * h;
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const uint4 bv = *reinterpret_cast<const uint4*>(base + nb * 32 * kWRow + 16 * s);
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) acc[mb][nb] = mfma_f16(P[mb][s], bv, acc[mb][nb]);
      }
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) P[mb][j] = xr[mb][kn * 8 + j];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 2; s < 4; ++s)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const uint4 bv = *reinterpret_cast<const uint4*>(base + nb * 32 * kWRow + 16 * s);
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) acc[mb][nb] = mfma_f16(R[mb][s - 2], bv, acc[mb][nb]);
      }
    uint8_t* d = wdst + (st ^ 1) * kWStage;
    *reinterpret_cast<uint4*>(d) = w0;
    *reinterpret_cast<uint4*>(d + 32 * kWRow) = w1;
    *reinterpret_cast<uint4*>(d + 64 * kWRow) = w2;
    *reinterpret_cast<uint4*>(d + 96 * kWRow) = w3;
    __syncthreads();
  }

  // ---- epilogue: fp16 outputs, FlashQ step 1 per 64-token block --------------
  // lane (m, h), register r of (mb, nb) <-> token n0 + 32 mb + 8 (r/4) + 4 h + r%4,
  // channel 32 nb + m
  float amax = 0.0f;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * mb + 8 * (r >> 2) + 4 * h + (r & 3);
        const float y = (float)(_Float16)acc[mb][nb][r];
        acc[mb][nb][r] = y;
        if (n0 + row < a.N) {
          amax = fmaxf(amax, fabsf(y));
          if constexpr (kY)
            a.y[((long)b * a.N + n0 + row) * (long)(128 * nheads) + 128 * head + 32 * nb + m] =
                (_Float16)y;
        }
      }
  amax = wave_max_fast(amax);
  float s = 0.0f, inv = 0.0f;
  if (amax > 0.0f) {
    s = amax / kQmax;
    inv = kQmax / amax;
  }
  __syncthreads();  // the W stages are reused as the epilogue tiles
  int8_t* tile_w = reinterpret_cast<int8_t*>(lds) + wv * kEpiTile;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * mb + 8 * (r >> 2) + 4 * h + (r & 3);
        const int q = n0 + row < a.N ? min(119, max(-119, rne_mul(acc[mb][nb][r], inv))) : 0;
        tile_w[row * kTileStride + 32 * nb + m] = (int8_t)q;
      }
  if (lane == 0) sblk[wv] = s;
  __syncthreads();

  const int jb = n0 / 64;  // FlashQ block index of this wave's block
  const bool live = jb < a.nb;
  if (head < a.Hq + a.Hkv) {
    // token-major int8 rows (Q8 or K8) and the block scale
    const bool isq = head < a.Hq;
    const int hh = isq ? head : head - a.Hq;
    const long unit = (long)b * (isq ? a.Hq : a.Hkv) + hh;
    int8_t* dst = (isq ? a.q8 : a.k8) + (unit * a.nb + jb) * 8192;
    if (live) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = 4 * i + (lane >> 4), c8 = lane & 15;
        *reinterpret_cast<uint2*>(dst + row * 128 + 8 * c8) =
            *reinterpret_cast<const uint2*>(tile_w + row * kTileStride + 8 * c8);
      }
      if (lane == 0) (isq ? a.sq : a.sk)[unit * a.nb + jb] = s;
    }
  } else {
    // channel-major V8 block: lane (channel pair) of each wave writes its
    // own block
    const int hh = head - a.Hq - a.Hkv;
    const long unit = (long)b * a.Hkv + hh;
    if (live) {
      int8_t* dst = a.v8 + (unit * a.nb + jb) * 8192;
#pragma unroll
      for (int cc = 0; cc < 2; ++cc) {
        const int c = 2 * lane + cc;
        unsigned wd[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int t = 4 * i;
          wd[i] = pack4(tile_w[t * kTileStride + c], tile_w[(t + 1) * kTileStride + c],
                        tile_w[(t + 2) * kTileStride + c], tile_w[(t + 3) * kTileStride + c]);
        }
        uint4* o = reinterpret_cast<uint4*>(dst + c * 64);
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = make_uint4(wd[4 * i], wd[4 * i + 1], wd[4 * i + 2], wd[4 * i + 3]);
      }
      if (lane == 0) a.sv[unit * a.nb + jb] = s;
    }
  }

  // ---- step 2 and the cache write (K and V heads, full blocks) ---------------
  if (a.pages == nullptr || head < a.Hq) return;  // work-group uniform
  const bool isk = head < a.Hq + a.Hkv;
  const int hkv = isk ? head - a.Hq : head - a.Hq - a.Hkv;
  const int bits = ((a.int2_mask >> hkv) & 1ull) ? 2 : 4;
  const int head_off = 512 * (4 * hkv - 2 * __popcll(a.int2_mask & ((1ull << hkv) - 1ull)));
  uint8_t* ctile = lds + 4 * kEpiTile;
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
    const int8_t* tb = reinterpret_cast<const int8_t*>(lds) + w * kEpiTile;
    if (isk)
      compress_k(tb, ctile, bits, meta, a.gscale + (slot * a.Hkv + hkv) * 2 + 0, sblk[w], page,
                 a.pages, a.page_bytes, head_off);
    else
      compress_v(tb, bits, meta, a.gscale + (slot * a.Hkv + hkv) * 2 + 1, sblk[w], page, a.pages,
                 a.page_bytes, head_off);
    __syncthreads();
  }
}

hipError_t launch_qkv_project(const QkvArgs& a, hipStream_t stream) {
  const int total = a.B * a.ntile * (a.Hq + 2 * a.Hkv);
  if (a.y)
    hipLaunchKernelGGL(k_qkv_project<true>, dim3(total), dim3(kProjThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(k_qkv_project<false>, dim3(total), dim3(kProjThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace turbo
