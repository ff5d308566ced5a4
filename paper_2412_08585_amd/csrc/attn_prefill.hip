// TurboAttention prefill on gfx950 (Algorithm 1): int8 QK^T and PV on the
// i8 MFMA, SAS online softmax in fp32 on the VALU.  Two kernels:
//   * k_attn_prefill16 (further below): B_r = B_c = 64, the paper's setting,
//     with four waves of 16 query rows -- the default, the pre-quantized-Q
//     path and the test hook;
//   * k_attn_prefill (this one): waves of 32 query rows, templated over
//     B_r in {32, 64, 128} and B_c in {32, 64, 128} for the other block sizes
//     of Table 3.
//
// k_attn_prefill: a workgroup of B_r / 32 waves owns one (sequence b, query
// head h, query block i of B_r rows); wave qh holds queries B_r i + 32qh ..
// +31 and all run over the key blocks j (those with a key at or before the
// block's last row when causal).  The Q scale and the P scale of Algorithm 1 cover the
// whole B_r x 64 tile, so the waves exchange their partial maxima through LDS
// (once for Q, once per tile for P).  32 queries per wave keep a wave under
// 256 VGPRs (two waves per SIMD, MFMA results in VGPRs).  With B_r = 128 the
// first waves of a diagonal block see no key of its last tile; their rows
// keep m and l unchanged there.
//
// Register layout.  The scores are computed transposed, S^T = K Q^T, so that
// each lane holds one query column:  for the 32x32 output block kb (32-key
// half kb), lane n + 32*hf, register r holds query n and key 32kb + 16hf + r.
// This is obtained by feeding A-operand row m of the K block with key
// 16*((m>>2)&1) + 4*(m>>3) + (m&3), the inverse of the MFMA output row map
// 8(r/4) + 4hf + r%4.  Consequently the 16 quantized P values of a lane are,
// byte for byte, its B-operand for O^T = V^T P^T with contraction index
// (hf, byte i) <-> key 16hf + i, and V^T is read as 16 contiguous bytes of
// the channel-major int8 V block.  Row max and row sum need one exchange
// between lanes n and n + 32 (v_permlane32_swap).
//
// The accumulator is kept as O = beta * Ost with a per-row factor beta, so
// the rescale by SAS(m_old - m_new) of Algorithm 1 multiplies beta instead of
// the 128 accumulator entries of a row; Ost is renormalized (a wave-uniform
// rare path) when beta underflows or the factor is 0.
#include "turbo_common.h"

namespace turbo {

struct PrefillArgs {
  const uint4* q;      // fp16 [B][Hq][N][128] (null when q8 is given)
  const int8_t* q8;    // pre-quantized Q: int8 [B][Hq][nb*64][128], scales sq [B][Hq][nb]
  const float* sq;
  const int8_t* k8;    // [B][Hkv][nb*64][128]
  const int8_t* v8;    // [B][Hkv][nb][128][64]
  const float* sk;     // [B][Hkv][nb]
  const float* sv;
  int B, Hq, Hkv, N, nb;
  int waves;           // 1, 2 or 4: B_r = 32 * waves
  int nbq;             // query blocks of B_r rows
  int bc, nbc;         // key block B_c (32, 64, 128) and key blocks per (b, h); sk, sv [..][nbc]
  float sm_scale;
  int causal;
  uint2* o;            // fp16 [B][Hq][N][128] (as 4-half units)
  float* lse;          // [B][Hq][N] or null
  unsigned char* trace;  // test hook: integers of tile (logical index tr_L, key block tr_j)
  int tr_L, tr_j;
};

// Logical work-group order L: longest causal query blocks first, and within
// a query block the G query heads of one KV head next to each other.  The
// dispatcher hands work-group x to XCD x % 8, so XCD k is given the units
// k, k + 8, k + 16, ... of G consecutive L: every XCD receives the same mix
// of row lengths (a contiguous split would leave one XCD with all the long
// rows) and the G heads reading the same K/V tiles run together on one
// XCD's L2.  Falls back to L = x (still interleaved) when 8G does not divide
// the grid.
__device__ __forceinline__ int prefill_order(int x, int total, int G) {
  if (total % (8 * G) != 0) return x;
  const int k = x % 8, n = x / 8;
  return (8 * (n / G) + k) * G + n % G;
}

// kTrace = true only for the test hook that also stores one tile's integers
// (the production instance carries no trace code).  kQ8: Q arrives already
// quantized (FlashQ step 1 of the fused projection), so the prologue only
// loads the int8 block and its scale.
//
// kBc = B_c: each online step (tile) covers kBc keys in kKb 32-key MFMA
// blocks.  B_c <= 64 keeps the whole pipeline in registers (K of the next
// tile loaded during the softmax); B_c = 128 would need 64 more registers for
// that, so its K is fetched in two 64-key halves after the tile's PV.
template <bool kTrace, bool kQ8, int kWaves, int kBc>
__global__ __launch_bounds__(64 * kWaves, 2) void k_attn_prefill(PrefillArgs a) {
  constexpr int kBr = 32 * kWaves;
  constexpr int kKb = kBc / 32;           // 32-key blocks per tile
  constexpr bool kSplitK = kKb > 2;       // B_c = 128
  constexpr int kKl = kSplitK ? 2 : kKb;  // 32-key K blocks held in registers
  __shared__ float lut[8];
  __shared__ float xmax[2][kWaves];  // per-wave P maxima, double-buffered
  const int tid = threadIdx.x;
  const int lane = tid & 63, qh = tid >> 6;
  if (tid < 8) lut[tid] = kLut[tid];
  __syncthreads();

  const int BH = a.B * a.Hq;
  const int L = prefill_order(blockIdx.x, BH * a.nbq, a.Hq / a.Hkv);
  const int i = a.nbq - 1 - L / BH;  // longest causal rows first
  const int b = (L % BH) / a.Hq, h = L % a.Hq;
  const int G = a.Hq / a.Hkv, kh = h / G;
  const int n = lane & 31, hf = lane >> 5;
  const int N = a.N;
  const int row0 = kBr * i + 32 * qh;  // first query row of this wave
  const int qrow = row0 + n;

  // ---- Q_i -> int8 (eq. step1bpq; scale over the 64-row block) ----------
  // lane (n + 32hf), k-step ks: channels 32ks + 16hf .. +15 of query qrow
  v4i qop[4];
  float sq;
  if (kQ8) {
    const int8_t* src = a.q8 + (((long)b * a.Hq + h) * a.nb * 64 + qrow) * 128 + 16 * hf;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) qop[ks] = *reinterpret_cast<const v4i*>(src + 32 * ks);
    sq = a.sq[((long)b * a.Hq + h) * a.nb + i];
  } else {
    uint4 raw[4][2];
    float amax = 0.0f;
    const uint4* src = a.q + (((long)b * a.Hq + h) * N + qrow) * 16;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        raw[ks][u] = qrow < N ? src[4 * ks + 2 * hf + u] : make_uint4(0, 0, 0, 0);
        f16x8_t hv = __builtin_bit_cast(f16x8_t, raw[ks][u]);
#pragma unroll
        for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)hv[e]));
      }
    amax = wave_max_fast(amax);
    if (kWaves > 1) {
      if (lane == 0) xmax[0][qh] = amax;
      __syncthreads();
      amax = xmax[0][0];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) amax = fmaxf(amax, xmax[0][w]);
      __syncthreads();
    }
    float inv = 0.0f;
    sq = 0.0f;
    if (amax > 0.0f) {
      sq = amax / kQmax;
      inv = kQmax / amax;
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      int w[4];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        f16x8_t hv = __builtin_bit_cast(f16x8_t, raw[ks][u]);
        int qv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) qv[e] = rne_mul((float)hv[e], inv);
        w[2 * u] = pack4(qv[0], qv[1], qv[2], qv[3]);
        w[2 * u + 1] = pack4(qv[4], qv[5], qv[6], qv[7]);
      }
      qop[ks] = v4i{w[0], w[1], w[2], w[3]};
    }
  }
  // wave-uniform; a key block the loop never reaches traces nothing
  const bool traced = kTrace && L == a.tr_L &&
                      a.tr_j <= (a.causal ? min(a.nbc - 1, (kBr * i + kBr - 1) / kBc) : a.nbc - 1);
  if constexpr (kTrace) {
    if (traced) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        *reinterpret_cast<v4i*>(a.trace + TURBO_TRACE_Q8 + (32 * qh + n) * 128 + 32 * ks +
                                16 * hf) = qop[ks];
      if (tid == 0) *reinterpret_cast<float*>(a.trace + TURBO_TRACE_SQ) = sq;
    }
  }

  const long kvu = (long)b * a.Hkv + kh;
  const float* skp = a.sk + kvu * a.nbc;
  const float* svp = a.sv + kvu * a.nbc;
  // A-operand row m of a 32-key block holds key kidx(m)
  const int m = lane & 31;
  const int kidx = 16 * ((m >> 2) & 1) + 4 * (m >> 3) + (m & 3);
  const int8_t* klane = a.k8 + kvu * a.nb * 8192 + kidx * 128 + 16 * hf;
  const int8_t* vlane = a.v8 + kvu * a.nb * 8192 + n * 64 + 16 * hf;
  // 32-key blocks the K8/V8 buffers hold (64 nb keys).  Only a 128-key tile
  // can reach past them; such blocks re-read the last one held, and their
  // keys (all >= N) are masked, so their scores and Q(P~) codes do not count.
  const int glast = 2 * a.nb - 1;
  auto blk = [&](int g) { return kSplitK ? min(g, glast) : g; };

  // K of the 32-key blocks g0 .. g0 + kKl - 1 (token-major, 128 B a key)
  auto load_k = [&](v4i (&kop)[kKl][4], int g0) {
#pragma unroll
    for (int kb = 0; kb < kKl; ++kb)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        kop[kb][ks] =
            *reinterpret_cast<const v4i*>(klane + (long)blk(g0 + kb) * 4096 + 32 * ks);
  };
  // V^T of the 32-key blocks g0 .. g0 + kKb - 1 (channel-major 64-key blocks)
  auto load_v = [&](v4i (&vop)[4][kKb], int g0) {
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int kb = 0; kb < kKb; ++kb) {
        const int g = blk(g0 + kb);
        vop[cb][kb] = *reinterpret_cast<const v4i*>(vlane + (long)(g >> 1) * 8192 +
                                                    32 * cb * 64 + 32 * (g & 1));
      }
  };
  // S^T of kKl 32-key blocks into S[off ..]
  auto qk = [&](v16i (&S)[kKb], int off, const v4i (&kop)[kKl][4]) {
#pragma unroll
    for (int kb = 0; kb < kKl; ++kb) {
      v16i acc = {};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) acc = mfma32x32x32(kop[kb][ks], qop[ks], acc);
      S[off + kb] = acc;
    }
  };

  float O[4][16];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) O[cb][r] = 0.0f;
  float mrow = -INFINITY, lhalf = 0.0f, beta = 1.0f;

  // last key tile: the one holding the block's last row when causal
  const int jend = a.causal ? min(a.nbc - 1, (kBr * i + kBr - 1) / kBc) : a.nbc - 1;
  // Software pipeline per tile j:  softmax of S_j on the VALU (K of tile j+1
  // already in flight) -> tile maximum exchange -> PV_j and then S_{j+1} on
  // the MFMA -> accumulator update on the VALU while S_{j+1} is computed.
  // B_c = 128: K_{j+1} is loaded during the accumulator update and S_{j+1}
  // computed after it.
  v4i kop[kKl][4];
  v4i vop[4][kKb];
  v16i S[kKb];
  load_k(kop, 0);
  qk(S, 0, kop);
  if constexpr (kSplitK) {
    load_k(kop, 2);
    qk(S, 2, kop);
  }
  load_v(vop, 0);
  float skj = skp[0], svj = svp[0];
  for (int j = 0; j <= jend; ++j) {
    const int jn = min(j + 1, jend);
    if constexpr (!kSplitK) load_k(kop, kKb * jn);
    const float skn = skp[jn], svn = svp[jn];
    const bool trace_tile = traced && j == a.tr_j;
    if constexpr (kTrace) {
      if (trace_tile) {
        int* ts = reinterpret_cast<int*>(a.trace + TURBO_TRACE_S) + (32 * qh + n) * kBc + 16 * hf;
#pragma unroll
        for (int kb = 0; kb < kKb; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) ts[32 * kb + r] = S[kb][r];
      }
    }
    // ---- scores, online max, SAS (Algorithm 1, statistics step) --------
    const float c = (sq * skj) * a.sm_scale;
    float P[kKb][16];
#pragma unroll
    for (int kb = 0; kb < kKb; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) P[kb][r] = (float)S[kb][r] * c;
    // masking only where a key can lie after one of this wave's rows (the
    // diagonal) and on tiles that reach past N
    if ((a.causal && kBc * j + kBc - 1 > row0) || (kBc * j + kBc > N) || (row0 + 32 > N)) {
#pragma unroll
      for (int kb = 0; kb < kKb; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kBc * j + 32 * kb + 16 * hf + r;
          const bool vis = key < N && qrow < N && (!a.causal || key <= qrow);
          P[kb][r] = vis ? P[kb][r] : -INFINITY;
        }
    }
    float smax = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < kKb; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) smax = fmaxf(smax, P[kb][r]);
    smax = max_xor32(smax);
    const float mold = mrow;
    const float mnew = fmaxf(mold, smax);
    float rs = 0.0f, pmax = 0.0f;
#pragma unroll
    for (int kb = 0; kb < kKb; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = sas_y(mnew - P[kb][r], lut);
        P[kb][r] = p;
        rs += p;
        pmax = fmaxf(pmax, p);
      }
    // SAS(m_old - m_new), 0 when m_old = -inf, and exactly 1 (e^0) for a row
    // whose maximum did not move.  A row that sees no key of the tile (with
    // B_r > B_c its keys can all follow the row) has only -inf scores, keeps
    // its maximum and adds nothing: it is left as it is.
    float alpha = sas_y(mnew - mold, lut);
    alpha = mnew > mold ? alpha : 1.0f;
    lhalf = alpha * lhalf + rs;
    mrow = mnew;
    // ---- tile maximum of P~ over the waves -----------------------------
    pmax = wave_max_fast(pmax);
    if (kWaves > 1) {
      if (lane == 0) xmax[j & 1][qh] = pmax;
      __syncthreads();
      pmax = xmax[j & 1][0];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) pmax = fmaxf(pmax, xmax[j & 1][w]);
    }
    // ---- rescale factor: O = beta * Ost --------------------------------
    float nbeta = beta * alpha;
    if (__builtin_amdgcn_ballot_w64(nbeta < 0x1p-64f) != 0) {  // rare: renormalize
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) O[cb][r] *= nbeta;
      nbeta = 1.0f;
    }
    beta = nbeta;
    // ---- Q(P~) with scale pmax/119 over the B_r x B_c tile --------------
    // (a tile with pmax = 0 gets inv = 0, Q(P~) = 0 and adds nothing)
    const float inv = pmax > 0.0f ? kQmax / pmax : 0.0f;
    const float g = ((pmax / kQmax) * svj) * __builtin_amdgcn_rcpf(beta);
    v4i pop[kKb];
#pragma unroll
    for (int kb = 0; kb < kKb; ++kb) {
      int w[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        w[u] = pack_lo4(rne_bits(P[kb][4 * u], inv), rne_bits(P[kb][4 * u + 1], inv),
                        rne_bits(P[kb][4 * u + 2], inv), rne_bits(P[kb][4 * u + 3], inv));
      pop[kb] = v4i{w[0], w[1], w[2], w[3]};
    }
    if constexpr (kTrace) {
      if (trace_tile) {
#pragma unroll
        for (int kb = 0; kb < kKb; ++kb)
          *reinterpret_cast<v4i*>(a.trace + TURBO_TRACE_P + (32 * qh + n) * kBc + 32 * kb +
                                  16 * hf) = pop[kb];
        if (tid == 0) *reinterpret_cast<float*>(a.trace + TURBO_TRACE_PMAX) = pmax;
      }
    }
    // ---- PV_j, then S_{j+1}, on the MFMA -------------------------------
    v16i acc[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      v16i t = {};
#pragma unroll
      for (int kb = 0; kb < kKb; ++kb) t = mfma32x32x32(vop[cb][kb], pop[kb], t);
      acc[cb] = t;
    }
    if constexpr (!kSplitK) {
      qk(S, 0, kop);
    } else {
      // keep the next tile's loads behind the PV (registers)
      __builtin_amdgcn_sched_barrier(0);
      load_k(kop, kKb * jn);
    }
    if constexpr (kTrace) {
      if (trace_tile) {
        // register r of channel block cb <-> channel 32cb + 8(r/4) + 4hf + r%4
        int* tp = reinterpret_cast<int*>(a.trace + TURBO_TRACE_PV) + (32 * qh + n) * 128;
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
#pragma unroll
          for (int r = 0; r < 16; ++r) tp[32 * cb + 8 * (r >> 2) + 4 * hf + (r & 3)] = acc[cb][r];
      }
    }
    // ---- Ost += (s_P s_V / beta) V_j^T Q(P~)^T ---------------------------
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) O[cb][r] = __builtin_fmaf(g, (float)acc[cb][r], O[cb][r]);
    if constexpr (kSplitK) {
      __builtin_amdgcn_sched_barrier(0);
      qk(S, 0, kop);
      __builtin_amdgcn_sched_barrier(0);
      load_k(kop, kKb * jn + 2);
      qk(S, 2, kop);
      __builtin_amdgcn_sched_barrier(0);
    }
    load_v(vop, kKb * jn);
    skj = skn;
    svj = svn;
  }

  // ---- epilogue: O / l (fp16), L = m + ln l ----------------------------
  const float l = add_xor32(lhalf);
  if (qrow < N) {
    const float f = beta / l;
    uint2* orow = a.o + (((long)b * a.Hq + h) * N + qrow) * 32;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        f16x4_t hv;
#pragma unroll
        for (int e = 0; e < 4; ++e) hv[e] = (_Float16)(O[cb][4 * g4 + e] * f);
        orow[(32 * cb + 8 * g4 + 4 * hf) / 4] = __builtin_bit_cast(uint2, hv);
      }
    if (a.lse && hf == 0) a.lse[((long)b * a.Hq + h) * N + qrow] = mrow + logf(l);
  }
}

// ---------------------------------------------------------------------------
// B_r = B_c = 64 (the paper's setting): four waves of 16 query rows.
//
// A 16-row wave holds half the accumulators of a 32-row one, which brings the
// kernel under 128 VGPRs: a SIMD then keeps four waves resident instead of
// two.  The softmax is bound by VALU issue, and one wave alone issues a VALU
// instruction only every few clocks, so more resident waves raise the rate.
// The work-group loads each K and V tile once into LDS (double-buffered) and
// the waves read their MFMA operands from there.
//
// v_mfma_i32_16x16x64_i8: output lane (n + 16g), register r = row 4g + r,
// column n.  S^T = K Q^T per 16-key block mb: A-operand row m holds key
// 16(m >> 2) + 4mb + (m & 3), so lane (n, g), register r of block mb is the
// score of query n and key 16g + 4mb + r.  The lane's 16 keys 16g .. 16g + 15
// are, byte for byte, its B-operand of O^T = V^T P^T with contraction slot
// (g, byte i) = key 16g + i, and the matching V^T bytes are 16 contiguous
// bytes of a channel row of the channel-major V block.  A query's 64 scores
// lie in lanes n, n + 16, n + 32, n + 48 (two exchanges per row reduction).
//
// LDS tiles without padding: 16-byte chunk c of K row t is stored at chunk
// c ^ kswz(t), chunk c of V row ch at c ^ vswz(ch), so that the lanes of
// each ds_read_b128 / ds_write_b128 pass hit distinct 4-bank groups.
//
// Per tile j (one barrier): QK_j from K buffer j&1; K_{j+1} (loaded a tile
// earlier) into K buffer (j+1)&1, whose last readers (QK_{j-1}) all finished
// before the previous barrier; softmax; tile maximum exchange + barrier; PV_j
// from V buffer j&1; V_{j+1} into V buffer (j+1)&1, whose last readers
// (PV_{j-1}) all finished before this tile's barrier.

// (conflict-free with 32 banks served 8 lanes per pass and with 64 banks
// served 16 lanes per pass; they depend only on key bits 0, 1, 4, 5 and
// channel bits 1 .. 3, so they are the same for every block mb and cb)
__device__ __forceinline__ int kswz(int t) {
  return ((t >> 1) & 1) | (((t >> 4) & 1) << 1) | ((((t >> 5) ^ t) & 1) << 2);
}
__device__ __forceinline__ int vswz(int ch) {
  return (((ch >> 1) ^ (ch >> 3)) & 1) | (((ch >> 2) & 1) << 1);
}

// Raw buffer resource over `bytes` bytes at p (gfx9 descriptor word 3).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t unit_rsrc(const int8_t* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(p), 0, bytes, 0x00020000);
}

__device__ __forceinline__ uint4 tile_load(__amdgpu_buffer_rsrc_t r, unsigned voff, int soff) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, soff, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

template <int kW>
struct Prefill16Lds {
  __attribute__((aligned(16))) int8_t k[2][64 * 128];   // [key][128 channels], swizzled
  __attribute__((aligned(16))) int8_t v[2][128 * 64];   // [channel][64 keys], swizzled
  float lut[8];
  float xmax[2][kW];
  float xq[kW];
};

// kW waves of 16 rows: B_r = 16 kW (4: the paper's 64; 8: Table 3's 128).
template <bool kTrace, bool kQ8, int kW>
__global__ __launch_bounds__(64 * kW, 4) void k_attn_prefill16(PrefillArgs a) {
  static_assert(kW == 4 || kW == 8, "B_r = 64 or 128");
  constexpr int kBr = 16 * kW;
  __shared__ Prefill16Lds<kW> L;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int n = lane & 15, g = lane >> 4;
  if (tid < 8) L.lut[tid] = kLut[tid];

  const int BH = a.B * a.Hq;
  const int Lx = prefill_order(blockIdx.x, BH * a.nbq, a.Hq / a.Hkv);
  const int i = a.nbq - 1 - Lx / BH;  // longest causal rows first
  const int b = (Lx % BH) / a.Hq, h = Lx % a.Hq;
  const int G = a.Hq / a.Hkv, kh = h / G;
  const int N = a.N;
  const int row0 = kBr * i + 16 * w;  // first query row of this wave
  const int qrow = row0 + n;
  const long kvu = (long)b * a.Hkv + kh;
  // the block scales are read-only here: read them through the constant
  // address space, which keeps these wave-uniform reads on the scalar unit
  typedef const __attribute__((address_space(4))) float cfloat;
  const cfloat* skp = (const cfloat*)(a.sk + kvu * a.nbc);
  const cfloat* svp = (const cfloat*)(a.sv + kvu * a.nbc);
  // last key tile: the one holding the block's last row when causal
  const int jend = a.causal ? min(a.nbc - 1, (kBr * i + kBr - 1) / 64) : a.nbc - 1;

  // ---- tile copies: the 512 16-byte chunks of a K (V) tile, one (kW = 8)
  // or two (kW = 4: tid and tid + 256) per thread --------------------------
  // wave-uniform tile bases; the lane adds its chunk index
  constexpr bool kTwo = kW == 4;
  const uint4* kg = reinterpret_cast<const uint4*>(a.k8 + kvu * a.nb * 8192);
  const uint4* vg = reinterpret_cast<const uint4*>(a.v8 + kvu * a.nb * 8192);
  const int c0 = tid, c1 = tid + 256;
  // buffer resources over this unit's K8 and V8 blocks (loads past them,
  // which never occur, would read 0)
  const __amdgpu_buffer_rsrc_t krs = unit_rsrc(a.k8 + kvu * a.nb * 8192, a.nb * 8192);
  const __amdgpu_buffer_rsrc_t vrs = unit_rsrc(a.v8 + kvu * a.nb * 8192, a.nb * 8192);
  const unsigned lane16 = 16u * (unsigned)tid;
  const int kdst0 = (c0 >> 3) * 128 + 16 * ((c0 & 7) ^ kswz(c0 >> 3));
  const int kdst1 = (c1 >> 3) * 128 + 16 * ((c1 & 7) ^ kswz(c1 >> 3));
  const int vdst0 = (c0 >> 2) * 64 + 16 * ((c0 & 3) ^ vswz(c0 >> 2));
  const int vdst1 = (c1 >> 2) * 64 + 16 * ((c1 & 3) ^ vswz(c1 >> 2));
  // K_{j+1} and V_{j+1} in flight (registers)
  uint4 kp0 = kg[tid], vp0 = vg[tid], kp1 = {}, vp1 = {};
  if constexpr (kTwo) {
    kp1 = kg[tid + 256];
    vp1 = vg[tid + 256];
  }
  *reinterpret_cast<uint4*>(&L.k[0][kdst0]) = kp0;
  *reinterpret_cast<uint4*>(&L.v[0][vdst0]) = vp0;
  if constexpr (kTwo) {
    *reinterpret_cast<uint4*>(&L.k[0][kdst1]) = kp1;
    *reinterpret_cast<uint4*>(&L.v[0][vdst1]) = vp1;
  }
  {
    const long o1 = (long)min(1, jend) * 512;
    kp0 = kg[o1 + tid];
    vp0 = vg[o1 + tid];
    if constexpr (kTwo) {
      kp1 = kg[o1 + tid + 256];
      vp1 = vg[o1 + tid + 256];
    }
  }

  // ---- Q_i -> int8 (eq. step1bpq; scale over the 64-row block) ----------
  // lane (n, g), k-step ks: channels 64ks + 16g .. +15 of query qrow
  v4i qop[2];
  float sq;
  if (kQ8) {
    const int8_t* src = a.q8 + (((long)b * a.Hq + h) * a.nb * 64 + row0) * 128 + (n * 128 + 16 * g);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) qop[ks] = *reinterpret_cast<const v4i*>(src + 64 * ks);
    sq = a.sq[((long)b * a.Hq + h) * a.nb + i];
    __syncthreads();
  } else {
    uint4 raw[2][2];
    float amax = 0.0f;
    // wave-uniform row base + a small lane offset: nothing per lane and
    // 64-bit stays live across the tile loop
    const uint4* src = a.q + (((long)b * a.Hq + h) * N + row0) * 16 + (n * 16 + 2 * g);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        raw[ks][u] = qrow < N ? src[8 * ks + u] : make_uint4(0, 0, 0, 0);
        f16x8_t hv = __builtin_bit_cast(f16x8_t, raw[ks][u]);
#pragma unroll
        for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)hv[e]));
      }
    amax = wave_max_fast(amax);
    if (lane == 0) L.xq[w] = amax;
    __syncthreads();
    amax = L.xq[0];
#pragma unroll
    for (int u = 1; u < kW; ++u) amax = fmaxf(amax, L.xq[u]);
    float inv = 0.0f;
    sq = 0.0f;
    if (amax > 0.0f) {
      sq = amax / kQmax;
      inv = kQmax / amax;
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      int wd[4];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        f16x8_t hv = __builtin_bit_cast(f16x8_t, raw[ks][u]);
        int qv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) qv[e] = rne_mul((float)hv[e], inv);
        wd[2 * u] = pack4(qv[0], qv[1], qv[2], qv[3]);
        wd[2 * u + 1] = pack4(qv[4], qv[5], qv[6], qv[7]);
      }
      qop[ks] = v4i{wd[0], wd[1], wd[2], wd[3]};
    }
  }
  // wave-uniform; a key block the loop never reaches traces nothing
  const bool traced = kTrace && Lx == a.tr_L && a.tr_j <= jend;
  if constexpr (kTrace) {
    if (traced) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
        *reinterpret_cast<v4i*>(a.trace + TURBO_TRACE_Q8 + (16 * w + n) * 128 + 64 * ks +
                                16 * g) = qop[ks];
      if (tid == 0) *reinterpret_cast<float*>(a.trace + TURBO_TRACE_SQ) = sq;
    }
  }

  // operand addresses in the tiles: K row 16(n>>2) + (n&3) (+ 4mb), chunk
  // 4ks + g; V row n (+ 16cb), chunk g
  const int kf = kswz(16 * (n >> 2) + (n & 3));  // the same for every block mb
  const int kbase0 = (16 * (n >> 2) + (n & 3)) * 128 + 16 * (g ^ kf);
  const int kbase1 = (16 * (n >> 2) + (n & 3)) * 128 + 16 * ((4 + g) ^ kf);
  const int vbase = n * 64 + 16 * (g ^ vswz(n));

  float O[8][4];
#pragma unroll
  for (int cb = 0; cb < 8; ++cb)
#pragma unroll
    for (int r = 0; r < 4; ++r) O[cb][r] = 0.0f;
  // The running maximum starts at -FLT_MAX rather than -inf: SAS of
  // m_new - (-FLT_MAX) is 0 as SAS(+inf) is, masked scores (-inf) still give
  // +inf and 0, and a row that has seen no key never reaches its maximum
  // (so the test below needs no separate -inf check).
  float mrow = -0x1.fffffep127f, lpart = 0.0f, beta = 1.0f, rbeta = 1.0f;  // rbeta ~ 1 / beta
  // 119 / pmax of the last tile that computed it, as wave-uniform bits
  unsigned pmax_prev = 0xffffffffu, inv_prev = 0u;
  float skj = skp[0], svj = svp[0];
  // sm_scale 2^26: (sq s_K) * (sm_scale 2^26) = ((sq s_K) * sm_scale) 2^26
  // exactly (a power-of-two factor; c cannot be subnormal for fp16 inputs)
  const float sm26 = a.sm_scale * 0x1p26f;

  // The tile step, unrolled by two over the LDS buffer index so that every
  // LDS address is a register plus an immediate offset.
  auto tile = [&](const int j, auto bufc) {
    constexpr int buf = decltype(bufc)::value;
    const float skn = skp[min(j + 1, jend)], svn = svp[min(j + 1, jend)];
    // ---- S^T_j = K_j Q^T on the MFMA -----------------------------------
    // The MFMA steps (operand reads, MFMAs, the next tiles' loads) run at
    // raised issue priority: a wave that reaches them goes ahead of the
    // softmax arithmetic of the other waves of its SIMD, so that its MFMAs
    // overlap their VALU work.
    v4i S[4];
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      const v4i k0 = *reinterpret_cast<const v4i*>(&L.k[buf][kbase0 + 512 * mb]);
      const v4i k1 = *reinterpret_cast<const v4i*>(&L.k[buf][kbase1 + 512 * mb]);
      v4i acc = {kAccSeed, kAccSeed, kAccSeed, kAccSeed};
      acc = mfma16x16x64(k0, qop[0], acc);
      acc = mfma16x16x64(k1, qop[1], acc);
      S[mb] = acc;
    }
    *reinterpret_cast<uint4*>(&L.k[buf ^ 1][kdst0]) = kp0;
    if constexpr (kTwo) *reinterpret_cast<uint4*>(&L.k[buf ^ 1][kdst1]) = kp1;
    // tile j + 2: buffer loads with the tile offset in a scalar register and
    // the lane's fixed offset in a vector register (no per-lane address
    // arithmetic per tile)
    const int o2 = min(j + 2, jend) * 8192;
    kp0 = tile_load(krs, lane16, o2);
    if constexpr (kTwo) kp1 = tile_load(krs, lane16 + 4096u, o2);
    __builtin_amdgcn_s_setprio(0);
    const bool trace_tile = traced && j == a.tr_j;
    if constexpr (kTrace) {
      if (trace_tile) {
        int* ts = reinterpret_cast<int*>(a.trace + TURBO_TRACE_S) + (16 * w + n) * 64 + 16 * g;
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
#pragma unroll
          for (int r = 0; r < 4; ++r) ts[4 * mb + r] = S[mb][r] - kAccSeed;
      }
    }
    // ---- scores, online max, SAS (Algorithm 1, statistics step) --------
    // (seed - S read as float) * (-c 2^26) = float(S) * c, rounded once
    const float nc26 = -((sq * skj) * sm26);
    float P[4][4];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) P[mb][r] = acc_unseed_neg(S[mb][r]) * nc26;
    // masking on the diagonal tile and where keys or rows reach past N
    if ((a.causal && 64 * j + 63 > row0) || (64 * j + 64 > N) || (row0 + 16 > N)) {
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = 64 * j + 16 * g + 4 * mb + r;
          const bool vis = key < N && qrow < N && (!a.causal || key <= qrow);
          P[mb][r] = vis ? P[mb][r] : -INFINITY;
        }
    }
    float smax = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) smax = fmaxf(smax, P[mb][r]);
    // scores and maxima are never NaN: maxima without canonicalization
    smax = max_xor32_nn(max_xor16_nn(smax));
    const float mold = mrow;
    const float mnew = max_nn(mold, smax);
    // A row whose maximum over this tile reaches its running maximum holds a
    // score with y = 0, whose P~ is SAS(0) = c0, and no P~ exceeds c0 (LUT[k]
    // <= 1 and POLY is decreasing from c0 on [0, 1)): the wave's P~ maximum
    // is then c0 without a reduction.
    const bool top = __builtin_amdgcn_ballot_w64(smax >= mold) != 0;
    float rs;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = sas_y(mnew - P[mb][r], L.lut);
        P[mb][r] = p;
        rs = (mb | r) ? rs + p : p;
      }
    // Rescale by SAS(m_old - m_new): 0 when m_old = -inf, exactly 1 (e^0)
    // for a row whose maximum did not move.  When no row of the wave moved
    // its maximum -- the common case away from the diagonal -- l, beta and
    // the accumulator stay as they are (wave-uniform branch).  Rows that see
    // no key of the tile (past N, or with B_r = 128 all before its keys) have
    // only -inf scores, keep their maximum and add nothing.
    const bool moved = __builtin_amdgcn_ballot_w64(mnew > mold) != 0;
    float alpha = 1.0f;
    if (moved) alpha = mnew > mold ? sas_y(mnew - mold, L.lut) : 1.0f;
    lpart = __builtin_fmaf(alpha, lpart, rs);  // alpha = 1: lpart + rs exactly
    mrow = mnew;
    // ---- tile maximum of P~ over the four waves ------------------------
    float pmax = kC0;
    if (!top) {  // wave-uniform
      // P~ >= 0: the maximum on the bits (integer order = float order)
      int pm = __float_as_int(P[0][0]);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int r = (mb == 0); r < 4; ++r) pm = max(pm, __float_as_int(P[mb][r]));
      pmax = wave_max_pos(__int_as_float(pm));
    }
    if (lane == 0) L.xmax[buf][w] = pmax;
    __syncthreads();
    {
      int pm = __float_as_int(L.xmax[buf][0]);
#pragma unroll
      for (int u = 1; u < kW; ++u) pm = max(pm, __float_as_int(L.xmax[buf][u]));
      pmax = __int_as_float(pm);
    }
    // ---- rescale factor: O = beta * Ost --------------------------------
    if (moved) {
      float nbeta = beta * alpha;
      if (__builtin_amdgcn_ballot_w64(nbeta < 0x1p-64f) != 0) {  // rare: renormalize
#pragma unroll
        for (int cb = 0; cb < 8; ++cb)
#pragma unroll
          for (int r = 0; r < 4; ++r) O[cb][r] *= nbeta;
        nbeta = 1.0f;
      }
      beta = nbeta;
      rbeta = __builtin_amdgcn_rcpf(beta);
    }
    // ---- Q(P~) with scale pmax/119 over the 64 x 64 tile ----------------
    // tile-uniform (scalar registers); the same pmax as the last tile (often
    // SAS(0), when a row sets its maximum in the tile) reuses the quotient
    const unsigned pbits = __builtin_amdgcn_readfirstlane(__float_as_uint(pmax));
    pmax = __uint_as_float(pbits);
    if (pbits != pmax_prev) {
      inv_prev = __builtin_amdgcn_readfirstlane(__float_as_uint(pmax > 0.0f ? kQmax / pmax : 0.0f));
      pmax_prev = pbits;
    }
    const float inv = __uint_as_float(inv_prev);
    // s_P = pmax / 119 only scales O (no code depends on it): the product
    // with the rounded reciprocal is within one ulp of the quotient; the
    // factor 2^26 undoes the accumulator seed
    const float ng26 = -(((pmax * (0x1p26f / kQmax)) * svj) * rbeta);
    v4i pop;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
      pop[mb] = pack_lo4(rne_bits(P[mb][0], inv), rne_bits(P[mb][1], inv),
                         rne_bits(P[mb][2], inv), rne_bits(P[mb][3], inv));
    if constexpr (kTrace) {
      if (trace_tile) {
        *reinterpret_cast<v4i*>(a.trace + TURBO_TRACE_P + (16 * w + n) * 64 + 16 * g) = pop;
        if (tid == 0) *reinterpret_cast<float*>(a.trace + TURBO_TRACE_PMAX) = pmax;
      }
    }
    // ---- PV_j on the MFMA; Ost += (s_P s_V / beta) V_j^T Q(P~)^T --------
    // in two halves of four channel blocks (operands and accumulators of
    // all eight at once would not fit beside O in 128 VGPRs)
#pragma unroll
    for (int hv = 0; hv < 2; ++hv) {
      v4i acc[4];
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const v4i vop = *reinterpret_cast<const v4i*>(&L.v[buf][vbase + 1024 * (4 * hv + c)]);
        const v4i z = {kAccSeed, kAccSeed, kAccSeed, kAccSeed};
        acc[c] = mfma16x16x64(vop, pop, z);
      }
      __builtin_amdgcn_s_setprio(0);
      if constexpr (kTrace) {
        if (trace_tile) {
          // register r of channel block cb <-> channel 16cb + 4g + r
          int* tp = reinterpret_cast<int*>(a.trace + TURBO_TRACE_PV) + (16 * w + n) * 128 + 4 * g;
#pragma unroll
          for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int r = 0; r < 4; ++r) tp[16 * (4 * hv + c) + r] = acc[c][r] - kAccSeed;
        }
      }
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          O[4 * hv + c][r] = __builtin_fmaf(ng26, acc_unseed_neg(acc[c][r]), O[4 * hv + c][r]);
      __builtin_amdgcn_sched_barrier(0);
    }
    *reinterpret_cast<uint4*>(&L.v[buf ^ 1][vdst0]) = vp0;
    if constexpr (kTwo) *reinterpret_cast<uint4*>(&L.v[buf ^ 1][vdst1]) = vp1;
    vp0 = tile_load(vrs, lane16, o2);
    if constexpr (kTwo) vp1 = tile_load(vrs, lane16 + 4096u, o2);
    skj = skn;
    svj = svn;
  };
  for (int j = 0; j <= jend; j += 2) {
    tile(j, std::integral_constant<int, 0>{});
    if (j + 1 <= jend) tile(j + 1, std::integral_constant<int, 1>{});
  }

  // ---- epilogue: O / l (fp16), L = m + ln l ----------------------------
  float l = lpart;
  {
    const unsigned u = __float_as_uint(l);
    auto r16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    l = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
  }
  l = add_xor32(l);
  // the lane index again, from an instruction the compiler cannot merge with
  // the prologue's: nothing lane-derived stays live across the tile loop
  // only for the epilogue (which kept three registers spilled)
  int lane_e;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane_e));
  const int ne = lane_e & 15, ge = lane_e >> 4;
  if (row0 + ne < N) {
    const float f = beta / l;
    uint2* orow = a.o + (((long)b * a.Hq + h) * N + row0) * 32 + ne * 32;
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      f16x4_t hv;
#pragma unroll
      for (int e = 0; e < 4; ++e) hv[e] = (_Float16)(O[cb][e] * f);
      orow[(16 * cb + 4 * ge) / 4] = __builtin_bit_cast(uint2, hv);
    }
    if (a.lse && ge == 0) a.lse[(((long)b * a.Hq + h) * N + row0) + ne] = mrow + logf(l);
  }
}

template <bool kTrace, int kWaves>
static void launch_bc(const PrefillArgs& a, int total, hipStream_t stream) {
  const dim3 grid(total), block(64 * kWaves);
  if (a.bc == 32)
    hipLaunchKernelGGL((k_attn_prefill<kTrace, false, kWaves, 32>), grid, block, 0, stream, a);
  else if (a.bc == 128)
    hipLaunchKernelGGL((k_attn_prefill<kTrace, false, kWaves, 128>), grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((k_attn_prefill<kTrace, false, kWaves, 64>), grid, block, 0, stream, a);
}

// (B_r, B_c) = (64, 64) and (128, 64) run on the 16-row-wave kernel, the
// other pairs on the 32-row-wave kernel; the test hook runs the same kernel
// as the plain call (its trace instance).
template <bool kTrace>
static void launch_prefill(const PrefillArgs& a, hipStream_t stream) {
  const int total = a.B * a.Hq * a.nbq;
  if (a.waves == 2 && a.bc == 64)
    hipLaunchKernelGGL((k_attn_prefill16<kTrace, false, 4>), dim3(total), dim3(256), 0, stream, a);
  else if (a.waves == 4 && a.bc == 64)
    hipLaunchKernelGGL((k_attn_prefill16<kTrace, false, 8>), dim3(total), dim3(512), 0, stream, a);
  else if (a.waves == 1)
    launch_bc<kTrace, 1>(a, total, stream);
  else if (a.waves == 4)
    launch_bc<kTrace, 4>(a, total, stream);
  else
    launch_bc<kTrace, 2>(a, total, stream);
}

hipError_t launch_attn_prefill(const PrefillArgs& a, hipStream_t stream) {
  if (a.q8)  // B_r = B_c = 64 only
    hipLaunchKernelGGL((k_attn_prefill16<false, true, 4>), dim3(a.B * a.Hq * a.nbq), dim3(256), 0,
                       stream, a);
  else if (a.trace)
    launch_prefill<true>(a, stream);
  else
    launch_prefill<false>(a, stream);
  return hipGetLastError();
}

}  // namespace turbo
