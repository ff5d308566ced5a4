// TurboAttention decode on gfx950 (Algorithm 2) over the paged int4/int2
// cache, with an optional split of the KV range into chunks (merged by
// k_decode_combine).
//
// One wave owns one (sequence b, KV head kh, chunk s) and all G query heads
// of kh.  Contractions run on the 16x16x64 i8 MFMA; the G query rows are the
// N columns (G <= 16).
//
// Layouts.  Lane = n + 16*g4 (n = lane & 15, g4 = lane >> 4).
//  * QK^T is computed transposed, S^T = K q^T.  A-operand row m of m-block mb
//    holds token 16*(m>>2) + 4*mb + (m&3) of the 64-token group, so that the
//    MFMA output of lane (n, g4), register r of m-block mb is the score of
//    query row n against token 16*g4 + 4*mb + r.  The 16 quantized P values
//    of a lane are then, in order, the scores of its row against the tokens
//    of page g4 -- exactly the B-operand of O^T = V^T P^T when the V^T
//    A-operand of lane (c, g4) is the 16 codes of channel c in page g4, which
//    is one contiguous 8-byte (int4) / 4-byte (int2) run of the
//    channel-major page.
//  * K is expanded to int8 in registers (code * s^int + z^int, Sec. 2.3);
//    the contraction index of k-step ks, byte i is channel 32*g4 + 16*ks + i.
//  * V is contracted on its raw codes and corrected per channel with the
//    exact integer identity sum_t p_t (c_t s + z) = s sum_t p_t c_t +
//    z sum_t p_t (eq. integer_inference of Sec. 2.3), so the int32 PV
//    accumulator equals the one over the int8-expanded V.
#include "turbo_common.h"

namespace turbo {

struct DecodeArgs {
  const uint4* q;            // fp16 [B][Hq][128]
  const uint8_t* pages;
  const int8_t* gmeta;       // [slots][Hkv][4][128]
  const float* gscale;       // [slots][Hkv][2]
  long num_pages, num_slots;
  int page_bytes;
  unsigned long long int2_mask;
  const int* seq_lens;       // [B]
  const int* block_table;    // [B][4*max_groups]
  const int* group_table;    // [B][max_groups]
  int max_groups;
  int B, Hq, Hkv, G;
  float sm_scale;
  int split;                 // groups per chunk
  int nsplit;                // chunks per sequence (grid dimension)
  float* ws;                 // [B][Hq][nsplit][132] when nsplit > 1: m, l, -, -, O[128]
  uint2* o;                  // fp16 [B][Hq][128]
  float* lse;                // [B][Hq] or null
};

constexpr int kWsStride = 132;  // m, l, two pad words, O[128] (16-byte aligned)
constexpr int kWsO = 4;

__device__ __forceinline__ int byte_of(const unsigned* w, int idx) {
  return (int)((w[idx >> 2] >> (8 * (idx & 3))) & 0xffu);
}

__device__ __forceinline__ int sbyte_of(const unsigned* w, int idx) {
  return (int)(int8_t)((w[idx >> 2] >> (8 * (idx & 3))) & 0xffu);
}

__global__ __launch_bounds__(64, 1) void k_attn_decode(DecodeArgs a) {
  __shared__ float lut[8];
  const int lane = threadIdx.x;
  if (lane < 8) lut[lane] = kLut[lane];
  __syncthreads();

  const int s = blockIdx.x % a.nsplit;
  const int kh = (blockIdx.x / a.nsplit) % a.Hkv;
  const int b = blockIdx.x / (a.nsplit * a.Hkv);
  const int n = lane & 15, g4 = lane >> 4;
  const int G = a.G;
  const bool rowok = n < G;
  const int h = kh * G + n;

  int ng = a.seq_lens[b] / 64;
  ng = min(max(ng, 0), a.max_groups);
  const int g0 = s * a.split;
  const int g1 = min(ng, g0 + a.split);

  const int bits = ((a.int2_mask >> kh) & 1ull) ? 2 : 4;
  const int head_off = 512 * (4 * kh - 2 * __popcll(a.int2_mask & ((1ull << kh) - 1ull)));

  // ---- q -> int8 per (b, query head) (Algorithm 2; eq. step1bpq) ---------
  v4i qop[2];
  float sq = 0.0f;
  {
    uint4 raw[2][2];
    float amax = 0.0f;
    const uint4* src = a.q + ((long)b * a.Hq + (rowok ? h : 0)) * 16;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        raw[ks][u] = rowok ? src[4 * g4 + 2 * ks + u] : make_uint4(0, 0, 0, 0);
        f16x8_t hv = __builtin_bit_cast(f16x8_t, raw[ks][u]);
#pragma unroll
        for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)hv[e]));
      }
    amax = fmaxf(amax, __shfl_xor(amax, 16));
    amax = fmaxf(amax, __shfl_xor(amax, 32));
    float inv = 0.0f;
    if (amax > 0.0f) {
      sq = amax / kQmax;
      inv = kQmax / amax;
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
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

  float O[8][4];
#pragma unroll
  for (int cb = 0; cb < 8; ++cb)
#pragma unroll
    for (int r = 0; r < 4; ++r) O[cb][r] = 0.0f;
  float mrow = -INFINITY, lpart = 0.0f;

  const int* bt = a.block_table + (long)b * 4 * a.max_groups;
  const int* gt = a.group_table + (long)b * a.max_groups;
  const int m = lane & 15;

  for (int g = g0; g < g1; ++g) {
    long pg[4];
    bool ok = true;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      pg[p] = bt[4 * g + p];
      ok = ok && pg[p] >= 0 && pg[p] < a.num_pages;
    }
    const long slot = gt[g];
    ok = ok && slot >= 0 && slot < a.num_slots;
    if (!ok) continue;  // caller error: this group is not read

    const int8_t* meta = a.gmeta + (slot * a.Hkv + kh) * 512;
    const float skg = a.gscale[(slot * a.Hkv + kh) * 2 + 0];
    const float svg = a.gscale[(slot * a.Hkv + kh) * 2 + 1];

    // K scale/zero of this lane's 32 channels 32g4 .. 32g4+31
    unsigned ksw[8], kzw[8];
    {
      const uint4* ms = reinterpret_cast<const uint4*>(meta + 32 * g4);
      const uint4* mz = reinterpret_cast<const uint4*>(meta + 128 + 32 * g4);
      uint4 t0 = ms[0], t1 = ms[1], z0 = mz[0], z1 = mz[1];
      ksw[0] = t0.x; ksw[1] = t0.y; ksw[2] = t0.z; ksw[3] = t0.w;
      ksw[4] = t1.x; ksw[5] = t1.y; ksw[6] = t1.z; ksw[7] = t1.w;
      kzw[0] = z0.x; kzw[1] = z0.y; kzw[2] = z0.z; kzw[3] = z0.w;
      kzw[4] = z1.x; kzw[5] = z1.y; kzw[6] = z1.z; kzw[7] = z1.w;
    }

    // ---- S^T = K^{q1} q^T ---------------------------------------------
    v4i sacc[4];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      const uint8_t* krow = a.pages + pg[m >> 2] * a.page_bytes + head_off +
                            (4 * mb + (m & 3)) * 16 * bits;
      int kv[32];  // int8 values of channels 32g4 + e
      if (bits == 4) {
        uint4 x = *reinterpret_cast<const uint4*>(krow + 16 * g4);
        unsigned xw[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int e = 0; e < 32; ++e) {
          const int code = (int)((xw[e >> 3] >> (4 * (e & 7))) & 15u);
          kv[e] = code * byte_of(ksw, e) + sbyte_of(kzw, e);
        }
      } else {
        uint2 x = *reinterpret_cast<const uint2*>(krow + 8 * g4);
        unsigned xw[2] = {x.x, x.y};
#pragma unroll
        for (int e = 0; e < 32; ++e) {
          const int code = (int)((xw[e >> 4] >> (2 * (e & 15))) & 3u);
          kv[e] = code * byte_of(ksw, e) + sbyte_of(kzw, e);
        }
      }
      v4i acc = {};
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        v4i kop = v4i{pack4(kv[16 * ks + 0], kv[16 * ks + 1], kv[16 * ks + 2], kv[16 * ks + 3]),
                      pack4(kv[16 * ks + 4], kv[16 * ks + 5], kv[16 * ks + 6], kv[16 * ks + 7]),
                      pack4(kv[16 * ks + 8], kv[16 * ks + 9], kv[16 * ks + 10], kv[16 * ks + 11]),
                      pack4(kv[16 * ks + 12], kv[16 * ks + 13], kv[16 * ks + 14], kv[16 * ks + 15])};
        acc = mfma16x16x64(kop, qop[ks], acc);
      }
      sacc[mb] = acc;
    }

    // ---- scores, online max, SAS (one row per lane column n) ----------
    const float c = (sq * skg) * a.sm_scale;
    float P[4][4];
    float smax = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        P[mb][r] = (float)sacc[mb][r] * c;
        smax = fmaxf(smax, P[mb][r]);
      }
    smax = fmaxf(smax, __shfl_xor(smax, 16));
    smax = fmaxf(smax, __shfl_xor(smax, 32));
    const float mnew = fmaxf(mrow, smax);
    float rs = 0.0f, pmax = 0.0f;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = sas_y(mnew - P[mb][r], lut);
        P[mb][r] = p;
        rs += p;
        pmax = fmaxf(pmax, p);
      }
    const float alpha = (mrow == -INFINITY) ? 0.0f : sas_y(mnew - mrow, lut);
    lpart = alpha * lpart + rs;
    mrow = mnew;
    pmax = fmaxf(pmax, __shfl_xor(pmax, 16));
    pmax = fmaxf(pmax, __shfl_xor(pmax, 32));
#pragma unroll
    for (int cb = 0; cb < 8; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r) O[cb][r] *= alpha;
    {
      // ---- Q(P~) with the row's scale pmax/119 over the group ----------
      // pmax differs between the rows of the wave and is 0 for a row whose
      // whole group lies more than 6 below its running maximum; such a row
      // gets Q(P~) = 0 and adds nothing (no branch: the shuffles and the
      // MFMA below need every lane).
      const float inv = pmax > 0.0f ? kQmax / pmax : 0.0f;
      const float spv = (pmax / kQmax) * svg;
      int qpw[4];
      int psum = 0;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        int qv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          qv[r] = rne_mul(P[mb][r], inv);
          psum += qv[r];
        }
        qpw[mb] = pack4(qv[0], qv[1], qv[2], qv[3]);
      }
      psum += __shfl_xor(psum, 16);
      psum += __shfl_xor(psum, 32);
      const v4i pop = v4i{qpw[0], qpw[1], qpw[2], qpw[3]};
      // ---- O^T += s_P s_V (s V^T_codes P^T + z sum P) --------------------
      const uint8_t* vreg = a.pages + pg[g4] * a.page_bytes + head_off + 256 * bits;
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) {
        const int ch = 16 * cb + n;  // A-operand row (channel) of this lane
        int w[4];
        if (bits == 4) {
          uint2 x = *reinterpret_cast<const uint2*>(vreg + ch * 8);
          unsigned xw[2] = {x.x, x.y};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const unsigned src = xw[u >> 1] >> (16 * (u & 1));
            w[u] = (int)((src & 15u) | (((src >> 4) & 15u) << 8) | (((src >> 8) & 15u) << 16) |
                         (((src >> 12) & 15u) << 24));
          }
        } else {
          const unsigned x = *reinterpret_cast<const unsigned*>(vreg + ch * 4);
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const unsigned src = x >> (8 * u);
            w[u] = (int)((src & 3u) | (((src >> 2) & 3u) << 8) | (((src >> 4) & 3u) << 16) |
                         (((src >> 6) & 3u) << 24));
          }
        }
        v4i acc = {};
        acc = mfma16x16x64(v4i{w[0], w[1], w[2], w[3]}, pop, acc);
        // output: lane (n, g4), register r <-> channel 16cb + 4g4 + r, row n
        const unsigned vs4 = *reinterpret_cast<const unsigned*>(meta + 256 + 16 * cb + 4 * g4);
        const unsigned vz4 = *reinterpret_cast<const unsigned*>(meta + 384 + 16 * cb + 4 * g4);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int sv_c = (int)((vs4 >> (8 * r)) & 0xffu);
          const int zv_c = (int)(int8_t)((vz4 >> (8 * r)) & 0xffu);
          const int pv = sv_c * acc[r] + zv_c * psum;
          O[cb][r] = __builtin_fmaf(spv, (float)pv, O[cb][r]);
        }
      }
    }
  }

  // ---- epilogue -----------------------------------------------------------
  float l = lpart + __shfl_xor(lpart, 16);
  l += __shfl_xor(l, 32);
  if (!rowok) return;
  if (a.nsplit == 1) {
    uint2* orow = a.o + ((long)b * a.Hq + h) * 32;
    const bool empty = g1 <= g0;
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      f16x4_t hv;
#pragma unroll
      for (int r = 0; r < 4; ++r) hv[r] = empty ? (_Float16)0.0f : (_Float16)(O[cb][r] / l);
      orow[(16 * cb + 4 * g4) / 4] = __builtin_bit_cast(uint2, hv);
    }
    if (a.lse && g4 == 0) a.lse[(long)b * a.Hq + h] = empty ? -INFINITY : mrow + logf(l);
  } else {
    if (g1 <= g0) return;  // chunk beyond this sequence: never read by the merge
    float* w = a.ws + (((long)b * a.Hq + h) * a.nsplit + s) * kWsStride;
    if (g4 == 0) {
      w[0] = mrow;
      w[1] = l;
    }
#pragma unroll
    for (int cb = 0; cb < 8; ++cb)
      *reinterpret_cast<float4*>(w + kWsO + 16 * cb + 4 * g4) =
          make_float4(O[cb][0], O[cb][1], O[cb][2], O[cb][3]);
  }
}

// Merge of the chunk states of one (b, query head): lane handles channels
// 2*lane, 2*lane + 1.
__global__ __launch_bounds__(64) void k_decode_combine(DecodeArgs a) {
  __shared__ float lut[8];
  const int lane = threadIdx.x;
  if (lane < 8) lut[lane] = kLut[lane];
  __syncthreads();
  const int bh = blockIdx.x;
  const int b = bh / a.Hq;
  int ng = a.seq_lens[b] / 64;
  ng = min(max(ng, 0), a.max_groups);
  const int ns = (ng + a.split - 1) / a.split;
  const float* w = a.ws + (long)bh * a.nsplit * kWsStride;
  float o0 = 0.0f, o1 = 0.0f, L = -INFINITY;
  if (ns == 1) {
    const float l = w[1];
    o0 = w[kWsO + 2 * lane] / l;
    o1 = w[kWsO + 1 + 2 * lane] / l;
    L = w[0] + logf(l);
  } else if (ns > 1) {
    float mstar = -INFINITY;
    for (int s = 0; s < ns; ++s) mstar = fmaxf(mstar, w[s * kWsStride]);
    float den = 0.0f, n0 = 0.0f, n1 = 0.0f;
    for (int s = 0; s < ns; ++s) {
      const float* ws = w + s * kWsStride;
      const float wt = sas_y(mstar - ws[0], lut);
      den = __builtin_fmaf(wt, ws[1], den);
      n0 = __builtin_fmaf(wt, ws[kWsO + 2 * lane], n0);
      n1 = __builtin_fmaf(wt, ws[kWsO + 1 + 2 * lane], n1);
    }
    o0 = n0 / den;
    o1 = n1 / den;
    L = mstar + logf(den);
  }
  _Float16 h2[2] = {(_Float16)o0, (_Float16)o1};
  reinterpret_cast<unsigned*>(a.o)[(long)bh * 64 + lane] = __builtin_bit_cast(unsigned, h2);
  if (a.lse && lane == 0) a.lse[bh] = L;
}

hipError_t launch_attn_decode(const DecodeArgs& a, hipStream_t stream) {
  const int total = a.B * a.Hkv * a.nsplit;
  hipLaunchKernelGGL(k_attn_decode, dim3(total), dim3(64), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.nsplit == 1) return e;
  hipLaunchKernelGGL(k_decode_combine, dim3(a.B * a.Hq), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace turbo
