// The int8 KV-cache buffer of Sec. 3.3 on gfx950: its start after a prefill,
// the append of one decoding step's key and value (with the flush of a full
// buffer into a step-2 group), and the decode of the buffered tokens as one
// more chunk of the split-KV merge.
#include "turbo_common.h"

namespace turbo {

// Universal-scale int8 code: nearest integer (ties to even) of the exact
// product x * inv, inv = 1/s in binary32, clamped to [-119, 119]; s = 0 gives
// 0.  The fp32 product only decides whether the code saturates (there the
// exact nearest integer is at least 120 in magnitude as well).
__device__ __forceinline__ int quant_univ(float x, float inv) {
  if (fabsf(x * inv) >= 120.0f) return x > 0.0f ? 119 : -119;
  return min(119, max(-119, rne_mul(x, inv)));
}

__device__ __forceinline__ float univ_inv(float s) { return s > 0.0f ? 1.0f / s : 0.0f; }

// ---- start of the buffer after a prefill ------------------------------------

struct TailInitArgs {
  const unsigned short* k;  // fp16 [B][Hkv][N][128]
  const unsigned short* v;
  const float* sk;          // [B][Hkv][nb]
  const float* sv;
  int Hkv, N, nb;
  int8_t* tk;               // [batch][Hkv][64][128]
  int8_t* tv;               // [batch][Hkv][128][64]
  float* tscale;            // [batch][Hkv][2]
};

__global__ __launch_bounds__(256) void k_tail_init(TailInitArgs a) {
  __shared__ float red[4];
  const long u = blockIdx.x;  // b * Hkv + h
  const int tid = threadIdx.x;
  float mk = 0.0f, mv = 0.0f;
  for (int j = tid; j < a.nb; j += 256) {
    mk = fmaxf(mk, a.sk[u * a.nb + j]);
    mv = fmaxf(mv, a.sv[u * a.nb + j]);
  }
  mk = block_max(mk, red);
  mv = block_max(mv, red);
  if (tid == 0) {
    a.tscale[2 * u] = mk;
    a.tscale[2 * u + 1] = mv;
  }
  const int ng = a.N / 64, nt = a.N - 64 * ng;
  const float ik = univ_inv(mk), iv = univ_inv(mv);
  const unsigned short* kr = a.k + (u * a.N + 64L * ng) * 128;
  const unsigned short* vr = a.v + (u * a.N + 64L * ng) * 128;
  {
    // K, token-major: thread (t = tid>>2, chunk = tid&3) codes 32 channels
    const int t = tid >> 2, c0 = 32 * (tid & 3);
    unsigned w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int q[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = c0 + 4 * i + e;
        q[e] = t < nt ? quant_univ((float)__builtin_bit_cast(_Float16, kr[t * 128 + c]), ik) : 0;
      }
      w[i] = pack4(q[0], q[1], q[2], q[3]);
    }
    uint4* dst = reinterpret_cast<uint4*>(a.tk + (u * 64 + t) * 128 + c0);
    dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
    dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
  }
  {
    // V, channel-major: thread (c = tid>>1, hh = tid&1) codes tokens 32hh..+31
    const int c = tid >> 1, t0 = 32 * (tid & 1);
    unsigned w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int q[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int t = t0 + 4 * i + e;
        q[e] = t < nt ? quant_univ((float)__builtin_bit_cast(_Float16, vr[t * 128 + c]), iv) : 0;
      }
      w[i] = pack4(q[0], q[1], q[2], q[3]);
    }
    uint4* dst = reinterpret_cast<uint4*>(a.tv + (u * 128 + c) * 64 + t0);
    dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
    dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
  }
}

hipError_t launch_tail_init(const TailInitArgs& a, int B, hipStream_t stream) {
  hipLaunchKernelGGL(k_tail_init, dim3(B * a.Hkv), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// ---- append of one decoding step (and flush of a full buffer) ---------------

struct AppendArgs {
  const unsigned short* knew;  // fp16 [B][Hkv][128]
  const unsigned short* vnew;
  const int* seq_lens;         // [B], lengths before the step
  int Hkv;
  int8_t* tk;
  int8_t* tv;
  const float* tscale;
  uint8_t* pages;
  int8_t* gmeta;
  float* gscale;
  long num_pages, num_slots;
  int page_bytes;
  unsigned long long int2_mask;
  const int* block_table;      // [B][4*max_groups]
  const int* group_table;      // [B][max_groups]
  int max_groups;
};

__global__ __launch_bounds__(256) void k_append_kv(AppendArgs a) {
  __shared__ int8_t tile[64 * kTileStride];
  __shared__ uint8_t ctile[64 * kTileStride];
  const long u = blockIdx.x;
  const int b = (int)(u / a.Hkv), h = (int)(u % a.Hkv);
  const int tid = threadIdx.x;
  const int p = a.seq_lens[b];
  if (p < 0) return;
  const int r = p & 63, g = p >> 6;
  const float sK = a.tscale[2 * u], sV = a.tscale[2 * u + 1];
  // threads 0..127: K channel tid; 128..255: V channel tid-128
  const int c = tid & 127;
  int qnew;
  if (tid < 128) {
    qnew = quant_univ((float)__builtin_bit_cast(_Float16, a.knew[u * 128 + c]), univ_inv(sK));
    a.tk[(u * 64 + r) * 128 + c] = (int8_t)qnew;
  } else {
    qnew = quant_univ((float)__builtin_bit_cast(_Float16, a.vnew[u * 128 + c]), univ_inv(sV));
    a.tv[(u * 128 + c) * 64 + r] = (int8_t)qnew;
  }
  // flush when this token is the buffer's 64th (workgroup-uniform)
  if (r != 63 || g >= a.max_groups) return;
  long page[4];
  bool ok = true;
  const int* bt = a.block_table + (long)b * 4 * a.max_groups + 4 * g;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    page[i] = bt[i];
    ok = ok && page[i] >= 0 && page[i] < a.num_pages;
  }
  const long slot = a.group_table[(long)b * a.max_groups + g];
  if (!ok || slot < 0 || slot >= a.num_slots) return;
  const int bits = ((a.int2_mask >> h) & 1ull) ? 2 : 4;
  const int head_off = 512 * (4 * h - 2 * __popcll(a.int2_mask & ((1ull << h) - 1ull)));
  int8_t* meta = a.gmeta + (slot * a.Hkv + h) * 512;
  // K buffer into the LDS tile (rows 0..62 from memory, row 63 the new codes)
  {
    const int t = tid >> 2, c0 = 32 * (tid & 3);
    if (t < 63) {
      const uint4* src = reinterpret_cast<const uint4*>(a.tk + (u * 64 + t) * 128 + c0);
      uint4* dst = reinterpret_cast<uint4*>(tile + t * kTileStride + c0);
      dst[0] = src[0];
      dst[1] = src[1];
    }
    if (tid < 128) tile[63 * kTileStride + c] = (int8_t)qnew;
  }
  __syncthreads();
  compress_k(tile, ctile, bits, meta, a.gscale + (slot * a.Hkv + h) * 2 + 0, sK, page, a.pages,
             a.page_bytes, head_off);
  __syncthreads();
  // V buffer (channel-major in memory) into the token-major tile
  {
    const int cc = tid >> 1, t0 = 32 * (tid & 1);
    const uint4* src = reinterpret_cast<const uint4*>(a.tv + (u * 128 + cc) * 64 + t0);
    const uint4 x0 = src[0], x1 = src[1];
    const unsigned w[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      const int t = t0 + i;
      if (t < 63) tile[t * kTileStride + cc] = (int8_t)(w[i >> 2] >> (8 * (i & 3)));
    }
    if (tid >= 128) tile[63 * kTileStride + c] = (int8_t)qnew;
  }
  __syncthreads();
  compress_v(tile, bits, meta, a.gscale + (slot * a.Hkv + h) * 2 + 1, sV, page, a.pages,
             a.page_bytes, head_off);
}

hipError_t launch_append_kv(const AppendArgs& a, int B, hipStream_t stream) {
  hipLaunchKernelGGL(k_append_kv, dim3(B * a.Hkv), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// ---- decode of the buffered tokens --------------------------------------
// One wave per (sequence b, KV head kh) and all G query rows of kh.  The
// buffer holds at most 63 tokens, so the integer products run on the VALU
// (v_dot4): lane t scores token t, then lane L accumulates channels 2L, 2L+1.
// The result is the buffer's chunk state (m, l, O) in workspace slot
// nchunk (after the group chunks), merged by k_decode_combine like the
// others (or written as the output when the sequence has no cached group).  It runs as the last B * Hkv
// work-groups of the k_attn_decode launch (work-group index bx among them),
// so it needs no launch of its own and fills the slots the group chunks
// leave free at the end.

template <int GP, bool kTrace>
__device__ void decode_tail_body(const DecodeArgs& a, int bx) {
  __shared__ float lut[8];
  __shared__ int q8s[GP][32];        // int8 query codes, 4 per word
  __shared__ float sqs[GP];
  __shared__ int p8s[GP][16];        // Q(P~) codes of the 64 slots, 4 per word
  __shared__ float4 rowv[GP];        // m, l, g = s_P s_V, -
  const int lane = threadIdx.x;
  if (lane < 8) lut[lane] = kLut[lane];
  const int b = bx / a.Hkv, kh = bx % a.Hkv;
  const int G = a.G;
  const DecodeSeq sq_ = decode_seq(a, b);
  const int ng = sq_.ng, nt = sq_.nt;
  if (nt == 0) return;
  const int sslot = sq_.nchunk;  // after the group chunks
  const long u = (long)b * a.Hkv + kh;
  const float sK = a.tscale[2 * u], sV = a.tscale[2 * u + 1];
  const int trow = kTrace && b == a.tr_b && kh == a.tr_h / G && a.tr_g == ng ? a.tr_h % G : -1;

  // ---- q -> int8 per query row (Algorithm 2; eq. step1bpq) ----------------
  for (int r = 0; r < G; ++r) {
    const unsigned qq = reinterpret_cast<const unsigned*>(a.q)[((long)b * a.Hq + kh * G + r) * 64 + lane];
    const float x0 = (float)__builtin_bit_cast(_Float16, (unsigned short)(qq & 0xffffu));
    const float x1 = (float)__builtin_bit_cast(_Float16, (unsigned short)(qq >> 16));
    const float amax = wave_max(fmaxf(fabsf(x0), fabsf(x1)));
    float inv = 0.0f, sq = 0.0f;
    if (amax > 0.0f) {
      sq = amax / kQmax;
      inv = kQmax / amax;
    }
    const int c0 = min(119, max(-119, rne_mul(x0, inv)));
    const int c1 = min(119, max(-119, rne_mul(x1, inv)));
    reinterpret_cast<int8_t*>(q8s[r])[2 * lane] = (int8_t)c0;
    reinterpret_cast<int8_t*>(q8s[r])[2 * lane + 1] = (int8_t)c1;
    if (lane == 0) sqs[r] = sq;
  }
  __syncthreads();
  if (kTrace && trow >= 0) {
    const int tr = trow >= 0 ? trow : 0;
    reinterpret_cast<unsigned short*>(a.trace + TURBO_TRACE_Q8)[lane] =
        reinterpret_cast<const unsigned short*>(q8s[tr])[lane];
    if (lane == 0) *reinterpret_cast<float*>(a.trace + TURBO_TRACE_SQ) = sqs[tr];
  }

  // ---- scores (lane t = buffer row t), online step from m = -inf ------------
  {
    const uint4* krow = reinterpret_cast<const uint4*>(a.tk + (u * 64 + lane) * 128);
    uint4 kw[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) kw[i] = krow[i];
    const bool vis = lane < nt;
    for (int r = 0; r < G; ++r) {
      int acc = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        acc = __builtin_amdgcn_sdot4(q8s[r][4 * i + 0], (int)kw[i].x, acc, false);
        acc = __builtin_amdgcn_sdot4(q8s[r][4 * i + 1], (int)kw[i].y, acc, false);
        acc = __builtin_amdgcn_sdot4(q8s[r][4 * i + 2], (int)kw[i].z, acc, false);
        acc = __builtin_amdgcn_sdot4(q8s[r][4 * i + 3], (int)kw[i].w, acc, false);
      }
      if (r == trow && vis) reinterpret_cast<int*>(a.trace + TURBO_TRACE_S)[lane] = acc;
      const float c = (sqs[r] * sK) * a.sm_scale;
      const float s = vis ? (float)acc * c : -INFINITY;
      const float m = wave_max(s);
      const float pt = vis ? sas_y(m - s, lut) : 0.0f;  // SAS(S - m)
      float l = pt;
      for (int o = 32; o >= 1; o >>= 1) l += __shfl_xor(l, o);
      const float pmax = wave_max(pt);
      const float inv = pmax > 0.0f ? kQmax / pmax : 0.0f;
      const int code = rne_bits(pt, inv) & 0xff;
      reinterpret_cast<uint8_t*>(p8s[r])[lane] = (uint8_t)code;
      if (r == trow) {
        a.trace[TURBO_TRACE_P + lane] = (unsigned char)code;
        if (lane == 0) *reinterpret_cast<float*>(a.trace + TURBO_TRACE_PMAX) = pmax;
      }
      if (lane == 0) rowv[r] = make_float4(m, l, (pmax / kQmax) * sV, 0.0f);
    }
  }
  __syncthreads();

  // ---- O = s_P s_V Q(P~) V^{q1} (lane L: channels 2L, 2L+1) ------------------
  {
    const uint4* v0 = reinterpret_cast<const uint4*>(a.tv + (u * 128 + 2 * lane) * 64);
    const uint4* v1 = reinterpret_cast<const uint4*>(a.tv + (u * 128 + 2 * lane + 1) * 64);
    uint4 w0[4], w1[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      w0[i] = v0[i];
      w1[i] = v1[i];
    }
    for (int r = 0; r < G; ++r) {
      int acc0 = 0, acc1 = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int* pw = p8s[r] + 4 * i;
        acc0 = __builtin_amdgcn_sdot4(pw[0], (int)w0[i].x, acc0, false);
        acc0 = __builtin_amdgcn_sdot4(pw[1], (int)w0[i].y, acc0, false);
        acc0 = __builtin_amdgcn_sdot4(pw[2], (int)w0[i].z, acc0, false);
        acc0 = __builtin_amdgcn_sdot4(pw[3], (int)w0[i].w, acc0, false);
        acc1 = __builtin_amdgcn_sdot4(pw[0], (int)w1[i].x, acc1, false);
        acc1 = __builtin_amdgcn_sdot4(pw[1], (int)w1[i].y, acc1, false);
        acc1 = __builtin_amdgcn_sdot4(pw[2], (int)w1[i].z, acc1, false);
        acc1 = __builtin_amdgcn_sdot4(pw[3], (int)w1[i].w, acc1, false);
      }
      if (r == trow)
        reinterpret_cast<int2*>(a.trace + TURBO_TRACE_PV)[lane] = make_int2(acc0, acc1);
      const float4 rv = rowv[r];
      const long bh = (long)b * a.Hq + kh * G + r;
      if (sq_.nparts == 1) {  // no cached group: the buffer's state is the result
        _Float16 h2[2] = {(_Float16)(rv.z * (float)acc0 / rv.y), (_Float16)(rv.z * (float)acc1 / rv.y)};
        reinterpret_cast<unsigned*>(a.o)[bh * 64 + lane] = __builtin_bit_cast(unsigned, h2);
        if (a.lse && lane == 0) a.lse[bh] = rv.x + logf(rv.y);
      } else {
        float* w = a.ws + (bh * a.nws + sslot) * kWsStride;
        *reinterpret_cast<float2*>(w + kWsO + 2 * lane) =
            make_float2(rv.z * (float)acc0, rv.z * (float)acc1);
        if (lane == 0) {
          w[0] = rv.x;
          w[1] = rv.y;
        }
      }
    }
  }
}


}  // namespace turbo
