// TurboAttention decode on gfx950 (Algorithm 2) over the paged int4/int2
// cache, with an optional split of the KV range into chunks (merged by
// k_decode_combine).
//
// One wave owns one (sequence b, KV head kh, chunk s) and all G query heads
// of kh (padded to GP = 1, 2, 4, 8 or 16 rows).  Per 64-token group:
//
//  * QK^T on the raw codes.  With w_c = q_c * s_c split exactly as
//    w = 128*hi + lo (lo in 0..127, hi in -75..74, both int8), the int32
//    accumulator of Algorithm 2, sum_c q_c (code_c s_c + z_c), equals
//    128 * sum hi*code + sum lo*code + sum_c q_c z_c  (eq. integer_inference
//    of Sec. 2.3 applied to the step-2 dequantization code*s + z).  Two
//    16x16x64 i8 MFMAs per k-step contract the unpacked 4/2-bit codes with
//    hi and lo; the zero-point term enters as the initial accumulator.  The
//    codes are only unpacked (mask/shift), never multiplied.
//    S^T = K q^T: A-operand row m of m-block mb holds token
//    16*(m>>2) + 4*mb + (m&3), so lane (n + 16*g4), register r of m-block mb
//    is the score of query row n and token 16*g4 + 4*mb + r.
//  * The GP x 64 scores go through LDS to a compact layout (lane L: row
//    L / (64/GP), GP consecutive tokens) where the SAS online softmax of
//    Algorithm 2 runs on useful values only; row reductions are DPP /
//    permlane within the row's 64/GP lanes.
//  * Q(P~) bytes return through LDS as the A-operand of O = P V (16x16x64
//    MFMA, K index = the tokens of page kg in the order the V codes unpack
//    to); the B-operand is the 16 codes of a channel in page kg, one
//    contiguous 8-byte (int4) / 4-byte (int2) run of the channel-major page.
//    PV is taken on the raw V codes and corrected per channel with
//    s * acc + z * sum(Q(P~)) (same identity), which equals the int32
//    accumulator over the int8-expanded V.  The GP x 128 result goes through
//    LDS to the compact layout (lane L: row L / (64/GP), 2*GP channels) for
//    the accumulator update.
//  * The accumulator is kept as O = beta * Ost (per-row beta) so the
//    rescale by SAS(m_old - m_new) touches one value per row.
//  * Every code byte is read once per launch, through streaming loads: the
//    waves spend their time waiting on these loads.
#include "turbo_common.h"
#include "stream_loads.h"

namespace turbo {

struct DecodeArgs {
  const uint4* q;            // fp16 [B][Hq][128]
  const uint8_t* pages;
  const int8_t* gmeta;       // [slots][Hkv][4][128]
  const float* gscale;       // [slots][Hkv][2]
  long num_pages, num_slots;
  int npages32, nslots32;    // min(num_pages, INT_MAX), min(num_slots, INT_MAX)
  int page_bytes;
  unsigned long long int2_mask;
  const int* seq_lens;       // [B]
  const int* block_table;    // [B][4*max_groups]
  const int* group_table;    // [B][max_groups]
  int max_groups;
  int B, Hq, Hkv, G;
  float sm_scale;
  int split;                 // groups per chunk; 0: decode_default_split of each sequence
  int nsplit;                // group chunks per (sequence, KV head) in the grid
  int nws;                   // workspace slots per row: nsplit, plus one with a tail
  float* ws;                 // [B][Hq][nws][132]: m, l, -, -, O[128] of each chunk
  const int8_t* tk;          // Sec. 3.3 buffer (null: none): [B][Hkv][64][128]
  const int8_t* tv;          //   [B][Hkv][128][64]
  const float* tscale;       //   [B][Hkv][2]
  uint2* o;                  // fp16 [B][Hq][128]
  float* lse;                // [B][Hq] or null
  unsigned char* trace;      // test hook: integers of (sequence tr_b, query head tr_h, group tr_g)
  int tr_b, tr_h, tr_g;
};

constexpr int kWsStride = 132;  // m, l, two pad words, O[128] (16-byte aligned)
constexpr int kWsO = 4;


// Chunk length (groups) that kv_split_groups = 0 gives a sequence of ng
// cached groups: one chunk up to 32 groups, chunks of 32 up to 128 groups,
// four equal chunks beyond.  It depends on the sequence alone, so a
// sequence's result does not depend on the batch it is decoded in.
__host__ __device__ constexpr int decode_default_split(int ng) {
  return ng <= 32 ? (ng > 0 ? ng : 1) : (ng <= 128 ? 32 : ceil_div(ng, 4));
}

// Chunks of a sequence with ng groups (chunk length split > 0 or the
// default rule), and the most any sequence of at most max_groups groups has.
__host__ __device__ constexpr int decode_chunks(int ng, int split) {
  return ng <= 0 ? 0 : ceil_div(ng, split > 0 ? split : decode_default_split(ng));
}
__host__ __device__ constexpr int decode_max_chunks(int max_groups, int split) {
  return max_groups <= 0 ? 0
         : split > 0     ? ceil_div(max_groups, split)
                         : (max_groups <= 32 ? 1 : (max_groups <= 128 ? ceil_div(max_groups, 32) : 4));
}

// The cached groups and buffered tokens decode attends for sequence b.
struct DecodeSeq {
  int ng;      // cached groups
  int split;   // chunk length
  int nchunk;  // group chunks
  int nt;      // buffered tokens (0 without a buffer)
  int nparts;  // nchunk + (nt > 0): states to merge
};

__device__ __forceinline__ DecodeSeq decode_seq(const DecodeArgs& a, int b) {
  DecodeSeq q;
  const int len = a.seq_lens[b];
  q.ng = min(max(len / 64, 0), a.max_groups);
  q.split = a.split > 0 ? a.split : decode_default_split(q.ng);
  q.nchunk = decode_chunks(q.ng, a.split);
  q.nt = a.tk ? min(max(len - 64 * q.ng, 0), 63) : 0;
  q.nparts = q.nchunk + (q.nt > 0);
  return q;
}

// o = 0 and lse = -inf for the G rows of (b, kh): a sequence with nothing to
// attend.
__device__ void decode_write_empty(const DecodeArgs& a, int b, int kh) {
  for (int r = 0; r < a.G; ++r) {
    const long bh = (long)b * a.Hq + kh * a.G + r;
    reinterpret_cast<unsigned*>(a.o)[bh * 64 + (threadIdx.x & 63)] = 0u;
    if (a.lse && (threadIdx.x & 63) == 0) a.lse[bh] = -INFINITY;
  }
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef short s16x2 __attribute__((ext_vector_type(2)));


// Reductions over the 64/GP consecutive lanes of a compact row (every lane
// of the row receives the result).
// Integer forms (the DPP moves fuse into the max / add).
template <int LPR>
__device__ __forceinline__ int row_max_i(int v) {
  if (LPR >= 2) v = max(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xf, 0xf, true));
  if (LPR >= 4) v = max(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xf, 0xf, true));
  if (LPR >= 8) v = max(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xf, 0xf, true));
  if (LPR >= 16) v = max(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xf, 0xf, true));
  if (LPR >= 32) {
    auto r = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
    v = max((int)r[0], (int)r[1]);
  }
  if (LPR >= 64) {
    auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
    v = max((int)r[0], (int)r[1]);
  }
  return v;
}

template <int LPR>
__device__ __forceinline__ int row_sum_i(int v) {
  if (LPR >= 2) v += __builtin_amdgcn_mov_dpp(v, 0xB1, 0xf, 0xf, true);
  if (LPR >= 4) v += __builtin_amdgcn_mov_dpp(v, 0x4E, 0xf, 0xf, true);
  if (LPR >= 8) v += __builtin_amdgcn_mov_dpp(v, 0x141, 0xf, 0xf, true);
  if (LPR >= 16) v += __builtin_amdgcn_mov_dpp(v, 0x140, 0xf, 0xf, true);
  if (LPR >= 32) {
    auto r = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
    v = (int)r[0] + (int)r[1];
  }
  if (LPR >= 64) {
    auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
    v = (int)r[0] + (int)r[1];
  }
  return v;
}

template <int LPR>
__device__ __forceinline__ float row_sum(float v) {
  if (LPR >= 2) v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xf, 0xf, false));
  if (LPR >= 4) v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xf, 0xf, false));
  if (LPR >= 8) v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xf, 0xf, false));
  if (LPR >= 16) v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xf, 0xf, false));
  if (LPR >= 32) {
    const unsigned u = __float_as_uint(v);
    auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  if (LPR >= 64) v = add_xor32(v);
  return v;
}

// Position of page token j in the order the V codes unpack to (see the PV
// step): int4 gives tokens {0,2,4,6},{1,3,5,7},{8,..},{9,..}; int2 gives
// {0,4,8,12},{1,5,9,13},...
template <int BITS>
__device__ __forceinline__ int vpos(int j) {
  if (BITS == 4) return (j & 8) + ((j & 1) << 2) + ((j & 7) >> 1);
  return 4 * (j & 3) + (j >> 2);
}

// LDS row strides (in ints) chosen for the bank pattern of the exchanges
// (64 banks of 4 bytes):
//  * scores: one row per MFMA column n (16), 68 ints apart, so the 16 lanes
//    of a column block store to 16 different banks;
//  * PV accumulators: GP + 2 ints per channel (an odd number of 8-byte
//    pairs), so lanes L = 0..15 reading channel rows 2L (+1) hit distinct
//    banks.  Lanes whose MFMA rows are unused (4*g4 >= GP) store to a
//    separate area instead, at one address for every channel block.
constexpr int kSbufStride = 68;
template <int GP>
constexpr int kObufStride = GP < 4 ? GP : GP + 2;
template <int GP>
constexpr int kOdumRows = GP < 4 ? 1 : (GP < 16 ? 64 - 4 * GP : 1);

// Rows of the w = q * s^int exchange: the GP query rows (at least 4, the
// rows one writer pass covers).
template <int GP>
constexpr int kWRows = GP < 4 ? 4 : GP;

template <int GP>
struct DecodeLds {
  float lut[8];
  float sq[16];
  __attribute__((aligned(16))) unsigned char whi[kWRows<GP>][128];  // hi bytes of w, B-operand order
  __attribute__((aligned(16))) unsigned char wlo[kWRows<GP>][128];  // lo bytes of w
  int wbias[kWRows<GP>];                // sum_c q_c z_c of each row
  signed char qbuf[kWRows<GP>][128];    // the int8 query rows
  __attribute__((aligned(16))) int sbuf[16][kSbufStride];  // scores, row n; rows >= GP unused
  unsigned char pbuf[GP + 1][64];   // Q(P~), per page in V-unpack order; row GP: read by
                                    // unused rows (their products are never kept)
  __attribute__((aligned(16))) int obuf[128][kObufStride<GP>];  // PV accumulators, channel-major
  __attribute__((aligned(16))) int odum[kOdumRows<GP>][4];     // stores of unused MFMA rows
  float4 rowv[GP];                  // per row: g = s_P s_V / beta, sum Q(P~), renorm, -
};

// K side of one group, loaded one group ahead of its step.  The table
// entries, the slot and the float scales are wave-uniform.  A group that is
// not live (past the chunk) or has an out-of-range entry (a caller error; it
// is skipped) still issues every load, from page 0 and slot 0, so that the
// number of memory operations in flight is the same on every path and the
// waits before each use stay exact.
//
// A-operand row m of m-block mb holds token 16*mb + m, so each m-block reads
// one page: its base address is wave-uniform and the lane adds its own
// offset (token row m, channel block g4).
template <int BITS>
struct GroupK {
  bool ok;
  int pg[4];                // page of each 16-token quarter (clamped into range)
  int vpg;                  // page of quarter g4 (this lane's PV K-chunk), clamped
  int slot;                 // group slot (clamped)
  float skg, svg;           // float scales s_K, s_V of the group
  unsigned kraw[4][BITS];   // K codes of the lane's 4 A-operand rows (32 channels each)
  // s^int and z^int bytes of the channels the lane writes w for (see
  // decode_groups): int4: 8 channels (2 dwords each), int2: their 16-channel
  // block (4 dwords each)
  unsigned ws[BITS == 4 ? 2 : 4], wz[BITS == 4 ? 2 : 4];
};

// V side of one group, loaded by the group's own step after its QK^T.
template <int BITS>
struct GroupV {
  unsigned vraw[8][BITS / 2];  // V codes of channel 16*cb + n in page g4
  unsigned vs4, vz4;           // V scales / zeros of channels 2L&~3 .. +3 (aligned dwords)
};

template <int BITS>
__device__ __forceinline__ void load_k(const DecodeArgs& a, int kh, int head_off, const int* bt,
                                       const int* gt, int g, bool live, GroupK<BITS>& K) {
  const int lane = threadIdx.x & 63;
  const int n = lane & 15, g4 = lane >> 4, m = lane & 15;
  g = live ? g : 0;
  bool ok = live;
  // the tables are read-only here: read them through the constant address
  // space, which keeps these wave-uniform reads on the scalar unit
  typedef const __attribute__((address_space(4))) int cint;
  const cint* btc = (const cint*)bt;
  const cint* gtc = (const cint*)gt;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int p = btc[4 * g + i];
    ok = ok && p >= 0 && p < a.npages32;
    K.pg[i] = p;
  }
  const int slot = gtc[g];
  ok = ok && slot >= 0 && slot < a.nslots32;
  K.ok = ok;
#pragma unroll
  for (int i = 0; i < 4; ++i) K.pg[i] = ok ? K.pg[i] : 0;
  K.slot = ok ? slot : 0;
  // this lane's V page, read by the lane itself (no per-lane choice among
  // the four uniform values)
  const int vp = bt[4 * g + g4];
  K.vpg = ok ? vp : 0;
  const int8_t* meta = a.gmeta + ((long)K.slot * a.Hkv + kh) * 512;
  typedef const __attribute__((address_space(4))) float cfloat;
  const cfloat* gs = (const cfloat*)(a.gscale + ((long)K.slot * a.Hkv + kh) * 2);
  K.skg = gs[0];
  K.svg = gs[1];
  const int koff = head_off + m * 16 * BITS + 4 * BITS * g4;
  // the codes are read once per launch: streaming loads.  The group's
  // metadata stays on ordinary loads, since its block is read twice (the K
  // scales and zeros here, the V ones by load_v)
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) {
    const uint8_t* krow = a.pages + (long)K.pg[mb] * a.page_bytes + koff;
    if constexpr (BITS == 4) {
      const u32x4_t x = load_nt4(krow);
      K.kraw[mb][0] = x.x; K.kraw[mb][1] = x.y; K.kraw[mb][2] = x.z; K.kraw[mb][3] = x.w;
    } else {
      const u32x2_t x = load_nt2(krow);
      K.kraw[mb][0] = x.x; K.kraw[mb][1] = x.y;
    }
  }
  // the lane writes w for 16-channel block k >> 1, half k & 1 (k = lane & 15)
  if constexpr (BITS == 4) {
    const uint2 x = *reinterpret_cast<const uint2*>(meta + 8 * n);
    const uint2 z = *reinterpret_cast<const uint2*>(meta + 128 + 8 * n);
    K.ws[0] = x.x; K.ws[1] = x.y;
    K.wz[0] = z.x; K.wz[1] = z.y;
  } else {
    const uint4 x = *reinterpret_cast<const uint4*>(meta + 16 * (n >> 1));
    const uint4 z = *reinterpret_cast<const uint4*>(meta + 128 + 16 * (n >> 1));
    K.ws[0] = x.x; K.ws[1] = x.y; K.ws[2] = x.z; K.ws[3] = x.w;
    K.wz[0] = z.x; K.wz[1] = z.y; K.wz[2] = z.z; K.wz[3] = z.w;
  }
}

template <int BITS>
__device__ __forceinline__ void load_v(const DecodeArgs& a, int kh, int head_off,
                                       const GroupK<BITS>& K, GroupV<BITS>& V) {
  const int lane = threadIdx.x & 63;
  const int n = lane & 15;
  const uint8_t* vrow = a.pages + (long)K.vpg * a.page_bytes + head_off + 256 * BITS + n * 2 * BITS;
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) {
    if constexpr (BITS == 4) {
      const u32x2_t x = load_nt2(vrow + cb * 32 * BITS);
      V.vraw[cb][0] = x.x; V.vraw[cb][1] = x.y;
    } else {
      V.vraw[cb][0] = load_nt1(vrow + cb * 32 * BITS);
    }
  }
  const int8_t* meta = a.gmeta + ((long)K.slot * a.Hkv + kh) * 512;
  V.vs4 = *reinterpret_cast<const unsigned*>(meta + 256 + 4 * (lane >> 1));
  V.vz4 = *reinterpret_cast<const unsigned*>(meta + 384 + 4 * (lane >> 1));
}

template <int GP, int BITS, bool kTrace>
__device__ __forceinline__ void decode_groups(const DecodeArgs& a, DecodeLds<GP>& L, int b, int kh,
                                              int g0, int g1, int head_off, float& mrow, float& lpart, float& beta,
                                              float (&O)[GP][2], float sq_row, int trow) {
  constexpr int LPR = 64 / GP;  // lanes per compact softmax row
  constexpr int d = BITS == 4 ? 2 : 4;
  const int lane = threadIdx.x & 63;
  const int n = lane & 15, g4 = lane >> 4;
  const int rr = lane / LPR, cc = lane % LPR;
  const int nrow = min(n, GP);  // P~ row this lane reads (GP: unused rows)
  // PV store target of this lane (GP >= 4): its 4 MFMA rows of channel
  // 16*cb + n, or (rows 4*g4.. unused) one spare slot for every cb
  const bool orows = 4 * g4 < GP;
  const int odi = min(max((g4 * 16 + n) - 4 * GP, 0), kOdumRows<GP> - 1);
  int* const obase = orows ? &L.obuf[n][4 * g4] : &L.odum[odi][0];
  const int ostep = orows ? 16 * kObufStride<GP> : 0;

  // ---- w = q * s^int, written by all lanes ------------------------------
  // The QK^T B-operand of lane (n, g4), k-step ks, is 16 bytes: dword j, byte
  // i holds channel 32*g4 + c0 + d*i with c0 = 16ks + 8(j>>1) + (j&1) (int4)
  // or 16ks + j (int2), the order the K codes unpack to.  Only GP of the 16
  // rows n are real, so instead of every lane building its own 32 values,
  // lane L builds those of unit U = L + 64t: row U >> 4, 8 channels given by
  // k = U & 15 -- dwords j = 2h, 2h+1 (h = k & 1) of block (g4 = k >> 2,
  // ks = (k >> 1) & 1) -- and writes their hi/lo bytes to byte 8k of the row.
  constexpr int kU = GP <= 4 ? 1 : GP / 4;  // writer units per lane
  const int k = lane & 15;
  const int cA = BITS == 4 ? 8 * k : 16 * (k >> 1) + 2 * (k & 1);  // channel of dword 2h, byte 0
  unsigned wq[kU][4];  // 16-bit q pairs (A0,A1) (A2,A3) (B0,B1) (B2,B3)
  int wqn[kU][2];      // the q bytes of dword A (= 2h) and B (= 2h + 1)
#pragma unroll
  for (int t = 0; t < kU; ++t) {
    const int r = (lane >> 4) + 4 * t;
    int qa[4], qb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      qa[i] = L.qbuf[r][cA + d * i];
      qb[i] = L.qbuf[r][cA + 1 + d * i];
    }
    wq[t][0] = ((unsigned)qa[0] & 0xffffu) | ((unsigned)qa[1] << 16);
    wq[t][1] = ((unsigned)qa[2] & 0xffffu) | ((unsigned)qa[3] << 16);
    wq[t][2] = ((unsigned)qb[0] & 0xffffu) | ((unsigned)qb[1] << 16);
    wq[t][3] = ((unsigned)qb[2] & 0xffffu) | ((unsigned)qb[3] << 16);
    wqn[t][0] = pack4(qa[0], qa[1], qa[2], qa[3]);
    wqn[t][1] = pack4(qb[0], qb[1], qb[2], qb[3]);
  }
  // int2: byte selectors of channel 2h (+1) in the four dwords of the block
  const unsigned h2 = 2u * (unsigned)(k & 1);
  const unsigned selA = h2 | (0x0cu << 8) | ((4u + h2) << 16) | (0x0cu << 24);
  const unsigned selZ1 = h2 | ((4u + h2) << 8) | 0x0c0c0000u;
  const unsigned selZ2 = 0x00000c0cu | (h2 << 16) | ((4u + h2) << 24);
  const int wrow = min(n, kWRows<GP> - 1);  // row this lane reads (unused rows: any)

  const int* bt = a.block_table + (long)b * 4 * a.max_groups;
  const int* gt = a.group_table + (long)b * a.max_groups;

  // Two K prefetch buffers used alternately (a copy cur = nxt between groups
  // would be a register move that waits for the prefetch to land).  A step
  // issues K of the next group first and V of its own group after its QK^T
  // MFMAs (V is not held during the QK^T phase); the softmax covers the V
  // latency.
  GroupK<BITS> KA, KB;
  load_k<BITS>(a, kh, head_off, bt, gt, g0, g0 < g1, KA);
  // Issue priority (s_setprio) is highest from a group's start until its V
  // loads are out, and for the K prefetch, lower in the softmax and lowest in
  // the PV and update steps: a wave on its way to a load goes ahead of the
  // other waves of its SIMD, and a wave nearer its next load ahead of one
  // that has just issued it, so the loads leave earlier.
  auto process = [&](const GroupK<BITS>& cur, int g) {
    if (cur.ok) {
      __builtin_amdgcn_s_setprio(2);
      // s^int pairs matching wq and z^int bytes matching wqn (see above)
      unsigned sA01, sA23, sB01, sB23, zA, zB;
      if constexpr (BITS == 4) {
        sA01 = __builtin_amdgcn_perm(0u, cur.ws[0], 0x0c020c00u);
        sA23 = __builtin_amdgcn_perm(0u, cur.ws[1], 0x0c020c00u);
        sB01 = __builtin_amdgcn_perm(0u, cur.ws[0], 0x0c030c01u);
        sB23 = __builtin_amdgcn_perm(0u, cur.ws[1], 0x0c030c01u);
        zA = __builtin_amdgcn_perm(cur.wz[1], cur.wz[0], 0x06040200u);
        zB = __builtin_amdgcn_perm(cur.wz[1], cur.wz[0], 0x07050301u);
      } else {
        sA01 = __builtin_amdgcn_perm(cur.ws[1], cur.ws[0], selA);
        sA23 = __builtin_amdgcn_perm(cur.ws[3], cur.ws[2], selA);
        sB01 = __builtin_amdgcn_perm(cur.ws[1], cur.ws[0], selA + 0x00010001u);
        sB23 = __builtin_amdgcn_perm(cur.ws[3], cur.ws[2], selA + 0x00010001u);
        zA = __builtin_amdgcn_perm(cur.wz[1], cur.wz[0], selZ1) |
             __builtin_amdgcn_perm(cur.wz[3], cur.wz[2], selZ2);
        zB = __builtin_amdgcn_perm(cur.wz[1], cur.wz[0], selZ1 + 0x0101u) |
             __builtin_amdgcn_perm(cur.wz[3], cur.wz[2], selZ2 + 0x01010000u);
      }
#pragma unroll
      for (int t = 0; t < kU; ++t) {
        const int r = (lane >> 4) + 4 * t;
        const unsigned sp[4] = {sA01, sA23, sB01, sB23};
        unsigned hx[4], lx[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const u16x2 w = __builtin_bit_cast(u16x2, wq[t][u]) * __builtin_bit_cast(u16x2, sp[u]);
          hx[u] = __builtin_bit_cast(unsigned, __builtin_bit_cast(s16x2, w) >> (short)7);
          lx[u] = __builtin_bit_cast(unsigned, w) & 0x007F007Fu;
        }
        *reinterpret_cast<uint2*>(&L.whi[r][8 * k]) =
            make_uint2(__builtin_amdgcn_perm(hx[1], hx[0], 0x06040200u),
                       __builtin_amdgcn_perm(hx[3], hx[2], 0x06040200u));
        *reinterpret_cast<uint2*>(&L.wlo[r][8 * k]) =
            make_uint2(__builtin_amdgcn_perm(lx[1], lx[0], 0x06040200u),
                       __builtin_amdgcn_perm(lx[3], lx[2], 0x06040200u));
        // zero-point term sum_c q_c z_c of row r: the unit's 8 channels, then
        // the 16 units of the row (one DPP row; exact: |sum| < 2^24)
        const int bp = __builtin_amdgcn_sdot4(wqn[t][0], (int)zA,
                                              __builtin_amdgcn_sdot4(wqn[t][1], (int)zB, 0, false),
                                              false);
        L.wbias[r] = row_sum_i<16>(bp);  // every lane of the row: the same value
      }
      wave_sync();
      v4i bhi[2], blo[2];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        bhi[ks] = *reinterpret_cast<const v4i*>(&L.whi[wrow][32 * g4 + 16 * ks]);
        blo[ks] = *reinterpret_cast<const v4i*>(&L.wlo[wrow][32 * g4 + 16 * ks]);
      }
      const int bias = L.wbias[wrow];
      // ---- S^T = K^{q1} q^T on the MFMA, scores to LDS -----------------
      int4 sv[4];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        v4i kop[2];
        if (BITS == 4) {
          unsigned u[8];
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            u[2 * w] = cur.kraw[mb][w] & 0x0F0F0F0Fu;
            u[2 * w + 1] = (cur.kraw[mb][w] >> 4) & 0x0F0F0F0Fu;
          }
          kop[0] = v4i{(int)u[0], (int)u[1], (int)u[2], (int)u[3]};
          kop[1] = v4i{(int)u[4], (int)u[5], (int)u[6], (int)u[7]};
        } else {
#pragma unroll
          for (int w = 0; w < 2; ++w)
            kop[w] = v4i{(int)(cur.kraw[mb][w] & 0x03030303u),
                         (int)((cur.kraw[mb][w] >> 2) & 0x03030303u),
                         (int)((cur.kraw[mb][w] >> 4) & 0x03030303u),
                         (int)((cur.kraw[mb][w] >> 6) & 0x03030303u)};
        }
        v4i lo = v4i{bias, bias, bias, bias};
        v4i hi = {};
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          lo = mfma16x16x64(kop[ks], blo[ks], lo);
          hi = mfma16x16x64(kop[ks], bhi[ks], hi);
        }
        sv[mb] = make_int4((hi[0] << 7) + lo[0], (hi[1] << 7) + lo[1], (hi[2] << 7) + lo[2],
                           (hi[3] << 7) + lo[3]);
      }
      GroupV<BITS> cv;
      load_v<BITS>(a, kh, head_off, cur, cv);
      __builtin_amdgcn_s_setprio(1);
      // lane (n, g4), register r of m-block mb: row n, token 16*mb + 4*g4 + r
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
        *reinterpret_cast<int4*>(&L.sbuf[n][16 * mb + 4 * g4]) = sv[mb];
      const bool trace_g = kTrace && trow >= 0 && g == a.tr_g;  // wave-uniform
      if (trace_g && n == trow) {
#pragma unroll
        for (int mb = 0; mb < 4; ++mb)
          reinterpret_cast<int4*>(a.trace + TURBO_TRACE_S)[4 * mb + g4] = sv[mb];
      }
      wave_sync();
      // ---- compact softmax: lane (rr, cc) holds tokens cc*GP .. +GP-1 -----
      bool renorm;
      {
        int si[GP];
        if (GP >= 4) {
#pragma unroll
          for (int e = 0; e < GP; e += 4) {
            const int4 t = *reinterpret_cast<const int4*>(&L.sbuf[rr][cc * GP + e]);
            si[e] = t.x; si[e + 1] = t.y; si[e + 2] = t.z; si[e + 3] = t.w;
          }
        } else {
#pragma unroll
          for (int e = 0; e < GP; ++e) si[e] = L.sbuf[rr][cc * GP + e];
        }
        // c >= 0 (sm_scale > 0, the scales are non-negative) and both
        // roundings of p = float(S) * c are monotonic: the row maximum of p is
        // float(max S) * c, taken on the integers
        const float c = (sq_row * cur.skg) * a.sm_scale;
        float p[GP];
        int imax = si[0];
#pragma unroll
        for (int e = 0; e < GP; ++e) {
          p[e] = (float)si[e] * c;
          imax = max(imax, si[e]);
        }
        const float smax = (float)row_max_i<LPR>(imax) * c;
        const float mnew = fmaxf(mrow, smax);
        float rs = 0.0f;
        int pbits = 0;  // the maximum of the p >= 0, on their bits (same order)
#pragma unroll
        for (int e = 0; e < GP; ++e) {
          p[e] = sas_y(mnew - p[e], L.lut);
          rs += p[e];
          pbits = max(pbits, __float_as_int(p[e]));
        }
        // SAS(m_old - m_new): 0 when m_old = -inf, exactly 1 (e^0) when the
        // row's maximum did not move
        const float alpha = mnew > mrow ? sas_y(mnew - mrow, L.lut) : 1.0f;
        lpart = alpha * lpart + rs;
        mrow = mnew;
        const float pmax = __int_as_float(row_max_i<LPR>(pbits));
        // rescale: O = beta * Ost; renormalize when beta underflows / is 0
        float nbeta = beta * alpha;
        renorm = __builtin_amdgcn_ballot_w64(nbeta < 0x1p-64f) != 0;
        const float rf = renorm ? nbeta : 1.0f;
        if (renorm) nbeta = 1.0f;
        beta = nbeta;
        // Q(P~) with the row's scale pmax/119 (a row whose group lies wholly
        // below the threshold has pmax = 0: inv = 0, Q(P~) = 0, adds nothing)
        const float inv = pmax > 0.0f ? kQmax / pmax : 0.0f;
        int ps = 0;
#pragma unroll
        for (int e = 0; e < GP; ++e) {
          const int code = rne_bits(p[e], inv) & 0xff;
          ps += code;
          const int t = cc * GP + e;  // token of the group
          L.pbuf[rr][16 * (t >> 4) + vpos<BITS>(t & 15)] = (unsigned char)code;
          if (trace_g && rr == trow) a.trace[TURBO_TRACE_P + t] = (unsigned char)code;
        }
        if (trace_g && rr == trow && cc == 0)
          *reinterpret_cast<float*>(a.trace + TURBO_TRACE_PMAX) = pmax;
        const int psum = row_sum_i<LPR>(ps);
        // s_P s_V / beta scales the fp32 accumulator only (no integer depends
        // on it): s_P as pmax times the binary32 1/119
        const float gsc = ((pmax * (1.0f / kQmax)) * cur.svg) * __builtin_amdgcn_rcpf(beta);
        // every lane of the row holds the same values
        L.rowv[rr] = make_float4(gsc, __int_as_float(psum), rf, 0.0f);
      }
      wave_sync();
      __builtin_amdgcn_s_setprio(0);
      // ---- O = Q(P~) V on the raw codes (A = P rows, B = V codes) -------
      const v4i pop = *reinterpret_cast<const v4i*>(&L.pbuf[nrow][16 * g4]);
      auto vop_of = [&](int cb) {
        if (BITS == 4) {
          const unsigned x0 = cv.vraw[cb][0], x1 = cv.vraw[cb][BITS / 2 - 1];
          return v4i{(int)(x0 & 0x0F0F0F0Fu), (int)((x0 >> 4) & 0x0F0F0F0Fu),
                     (int)(x1 & 0x0F0F0F0Fu), (int)((x1 >> 4) & 0x0F0F0F0Fu)};
        } else {
          const unsigned x = cv.vraw[cb][0];
          return v4i{(int)(x & 0x03030303u), (int)((x >> 2) & 0x03030303u),
                     (int)((x >> 4) & 0x03030303u), (int)((x >> 6) & 0x03030303u)};
        }
      };
      // lane (n, g4), register r <-> row 4*g4 + r, channel 16*cb + n
      auto store = [&](int cb, const v4i& acc) {
        if (GP >= 4) {
          int* dst = obase + cb * ostep;
          *reinterpret_cast<int2*>(dst) = make_int2(acc[0], acc[1]);
          *reinterpret_cast<int2*>(dst + 2) = make_int2(acc[2], acc[3]);
        } else if (g4 == 0) {
#pragma unroll
          for (int r = 0; r < GP; ++r) L.obuf[16 * cb + n][r] = acc[r];
        }
      };
      // two channel blocks per step: the second MFMA runs while the first
      // one's result is stored
#pragma unroll
      for (int cb = 0; cb < 8; cb += 2) {
        const v4i acc0 = mfma16x16x64(pop, vop_of(cb), v4i{});
        const v4i acc1 = mfma16x16x64(pop, vop_of(cb + 1), v4i{});
        store(cb, acc0);
        store(cb + 1, acc1);
      }
      wave_sync();
      // ---- accumulator update: lane L owns channels 2L, 2L+1 of all rows --
      {
        int acc[2][GP];
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
          if (GP >= 4) {
#pragma unroll
            for (int r = 0; r < GP; r += 2) {
              const int2 t = *reinterpret_cast<const int2*>(&L.obuf[2 * lane + c2][r]);
              acc[c2][r] = t.x; acc[c2][r + 1] = t.y;
            }
          } else {
#pragma unroll
            for (int r = 0; r < GP; ++r) acc[c2][r] = L.obuf[2 * lane + c2][r];
          }
        }
        const int sh = 16 * (lane & 1);  // channels 2L, 2L+1 within the dword
        const int s0 = (int)((cv.vs4 >> sh) & 0xffu), s1 = (int)((cv.vs4 >> (sh + 8)) & 0xffu);
        const int z0 = (int)(int8_t)((cv.vz4 >> sh) & 0xffu);
        const int z1 = (int)(int8_t)((cv.vz4 >> (sh + 8)) & 0xffu);
        if (renorm) {  // wave-uniform and rare: a branch (the empty asm keeps
                       // the compiler from turning it into selects)
          asm volatile("");
#pragma unroll
          for (int r = 0; r < GP; ++r) {
            const float rf = L.rowv[r].z;
            O[r][0] *= rf;
            O[r][1] *= rf;
          }
        }
#pragma unroll
        for (int r = 0; r < GP; ++r) {
          const float4 rv = L.rowv[r];
          const int psum = __float_as_int(rv.y);
          // exact int32 PV of Algorithm 2: s * sum P*code + z * sum P (every
          // factor fits 24 bits: s <= 80, |z| <= 127, sum P <= 64*119,
          // |sum P*code| <= 64*119*15)
          const int pv0 = __mul24(s0, acc[0][r]) + __mul24(z0, psum);
          const int pv1 = __mul24(s1, acc[1][r]) + __mul24(z1, psum);
          O[r][0] = __builtin_fmaf(rv.x, (float)pv0, O[r][0]);
          O[r][1] = __builtin_fmaf(rv.x, (float)pv1, O[r][1]);
          if (trace_g && r == trow)
            reinterpret_cast<int2*>(a.trace + TURBO_TRACE_PV)[lane] = make_int2(pv0, pv1);
        }
      }
    }
  };
  for (int g = g0; g < g1; g += 2) {
    __builtin_amdgcn_s_setprio(2);
    load_k<BITS>(a, kh, head_off, bt, gt, g + 1, g + 1 < g1, KB);
    __builtin_amdgcn_s_setprio(0);
    process(KA, g);
    if (g + 1 < g1) {
      __builtin_amdgcn_s_setprio(2);
      load_k<BITS>(a, kh, head_off, bt, gt, g + 2, g + 2 < g1, KA);
      __builtin_amdgcn_s_setprio(0);
      process(KB, g + 1);
    }
  }
}

// kTrace = true only for the test hook that also stores one group's integers
// (the production instances carry no trace code).
template <int GP, bool kTrace>
__device__ void decode_tail_body(const DecodeArgs& a, int bx);  // kv_tail.hip

// One wave per (b, KV head, chunk of groups); with several chunks each
// writes its state to the workspace and k_decode_combine merges them.
template <int GP, bool kTrace>
__global__ __launch_bounds__(64, (GP <= 8 && !kTrace) ? 3 : 2) void k_attn_decode(DecodeArgs a) {
  // the last B * Hkv work-groups (when there is a buffer): its chunk
  const int nmain = a.B * a.Hkv * a.nsplit;
  if ((int)blockIdx.x >= nmain) {
    decode_tail_body<GP, kTrace>(a, (int)blockIdx.x - nmain);
    return;
  }
  __shared__ DecodeLds<GP> L;
  const int s = blockIdx.x % a.nsplit;
  const int kh = (blockIdx.x / a.nsplit) % a.Hkv;
  const int b = blockIdx.x / (a.nsplit * a.Hkv);
  constexpr int LPR = 64 / GP;
  const int lane = threadIdx.x & 63;
  if (lane < 8) L.lut[lane] = kLut[lane];
  const int n = lane & 15, g4 = lane >> 4;
  const int rr = lane / LPR, cc = lane % LPR;
  const int G = a.G;

  const DecodeSeq sq_ = decode_seq(a, b);
  const int g0 = s * sq_.split;
  const int g1 = min(sq_.ng, g0 + sq_.split);
  if (g1 <= g0) {  // no group of this sequence in the chunk
    if (s == 0 && sq_.nparts == 0) decode_write_empty(a, b, kh);
    return;
  }

  float O[GP][2];
#pragma unroll
  for (int r = 0; r < GP; ++r) O[r][0] = O[r][1] = 0.0f;
  float mrow = -INFINITY, lpart = 0.0f, beta = 1.0f, l = 0.0f;
  {
    const int bits = ((a.int2_mask >> kh) & 1ull) ? 2 : 4;
    const int head_off = 512 * (4 * kh - 2 * __popcll(a.int2_mask & ((1ull << kh) - 1ull)));

    // ---- q -> int8 per (b, query head) (Algorithm 2; eq. step1bpq) -------
    // lane (n, g4) holds channels 32*g4 .. 32*g4+31 of row n (zero if n >= G)
    int q8w[8];
    {
      const bool rowok = n < G;
      uint4 raw[4];
      float amax = 0.0f;
      const uint4* src = a.q + ((long)b * a.Hq + kh * G + (rowok ? n : 0)) * 16;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        raw[u] = rowok ? src[4 * g4 + u] : make_uint4(0, 0, 0, 0);
        f16x8_t hv = __builtin_bit_cast(f16x8_t, raw[u]);
#pragma unroll
        for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)hv[e]));
      }
      amax = max_xor16(amax);
      amax = max_xor32(amax);
      float inv = 0.0f, sq = 0.0f;
      if (amax > 0.0f) {
        sq = amax / kQmax;
        inv = kQmax / amax;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        f16x8_t hv = __builtin_bit_cast(f16x8_t, raw[u]);
        int qv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) qv[e] = rne_mul((float)hv[e], inv);
        q8w[2 * u] = pack4(qv[0], qv[1], qv[2], qv[3]);
        q8w[2 * u + 1] = pack4(qv[4], qv[5], qv[6], qv[7]);
      }
      if (g4 == 0) L.sq[n] = sq;
      if (n < kWRows<GP>) {
#pragma unroll
        for (int i = 0; i < 8; ++i) *reinterpret_cast<int*>(&L.qbuf[n][32 * g4 + 4 * i]) = q8w[i];
      }
    }
    // traced row of this wave (-1: none); the wave whose chunk holds group tr_g
    const int trow = kTrace && b == a.tr_b && kh == a.tr_h / G && g0 <= a.tr_g && a.tr_g < g1
                         ? a.tr_h % G : -1;
    if (trow >= 0 && n == trow) {
#pragma unroll
      for (int i = 0; i < 8; ++i) reinterpret_cast<int*>(a.trace + TURBO_TRACE_Q8)[8 * g4 + i] = q8w[i];
      if (g4 == 0) *reinterpret_cast<float*>(a.trace + TURBO_TRACE_SQ) = L.sq[n];
    }
    wave_sync();
    const float sq_row = L.sq[rr];

    if (bits == 4)
      decode_groups<GP, 4, kTrace>(a, L, b, kh, g0, g1, head_off, mrow, lpart, beta, O, sq_row, trow);
    else
      decode_groups<GP, 2, kTrace>(a, L, b, kh, g0, g1, head_off, mrow, lpart, beta, O, sq_row, trow);

    // ---- epilogue: per-row (m, l, beta) from the softmax lanes -----------
    l = row_sum<LPR>(lpart);
    wave_sync();
    if (cc == 0) L.rowv[rr] = make_float4(mrow, l, beta, 0.0f);
    wave_sync();
  }
  if (sq_.nparts == 1) {  // the only state (chunk 0): O / l and L directly
#pragma unroll
    for (int r = 0; r < GP; ++r) {
      if (r >= G) break;
      const float4 rv = L.rowv[r];
      const float f = rv.z / rv.y;
      _Float16 h2[2] = {(_Float16)(O[r][0] * f), (_Float16)(O[r][1] * f)};
      reinterpret_cast<unsigned*>(a.o)[((long)b * a.Hq + kh * G + r) * 64 + lane] =
          __builtin_bit_cast(unsigned, h2);
    }
    if (a.lse && cc == 0 && rr < G)
      a.lse[(long)b * a.Hq + kh * G + rr] = mrow + logf(l);
    return;
  }
  // several states: O beta, m and l of each row, to the workspace
#pragma unroll
  for (int r = 0; r < GP; ++r) {
    if (r >= G) break;
    const float be = L.rowv[r].z;
    float* w = a.ws + (((long)b * a.Hq + kh * G + r) * a.nws + s) * kWsStride;
    *reinterpret_cast<float2*>(w + kWsO + 2 * lane) = make_float2(O[r][0] * be, O[r][1] * be);
  }
  if (cc == 0 && rr < G) {
    float* w = a.ws + (((long)b * a.Hq + kh * G + rr) * a.nws + s) * kWsStride;
    w[0] = mrow;
    w[1] = l;
  }
}

// Merge of the chunk states of one (b, query head) with more than one state
// (split-KV extension): m* = max m_s, w_s = SAS(m_s - m*) (exactly 1 for
// m_s = m*), O = sum w_s O_s / sum w_s l_s, L = m* + ln sum w_s l_s, chunks
// in ascending order (the buffer's state last).  A separate launch: the
// kernel boundary makes every chunk's state visible across the XCDs' L2
// caches.  Lane L handles channels 2L, 2L + 1.
__global__ __launch_bounds__(64) void k_decode_combine(DecodeArgs a) {
  __shared__ float lut[8];
  __shared__ float cwt[64], cl[64];  // merge weights and l of up to 64 chunks
  const int lane = threadIdx.x & 63;
  const int bh = blockIdx.x;
  const int b = bh / a.Hq;
  const int ns = decode_seq(a, b).nparts;
  if (ns < 2) return;  // written by the decode launch itself
  if (lane < 8) lut[lane] = kLut[lane];
  const float* w = a.ws + (long)bh * a.nws * kWsStride;
  // m* over the chunks, lane s reading chunk s (and s + 64, ...)
  float mstar = -INFINITY;
  for (int s = lane; s < ns; s += 64) mstar = fmaxf(mstar, w[(long)s * kWsStride]);
  mstar = wave_max(mstar);
  // ascending accumulation of w_s l_s and w_s O_s; the weights of 64 chunks
  // at a time go through LDS and four chunks' O loads are in flight at once
  float den = 0.0f, n0 = 0.0f, n1 = 0.0f;
  for (int s0 = 0; s0 < ns; s0 += 64) {
    const int cnt = min(64, ns - s0);
    __syncthreads();
    if (lane < cnt) {
      const float* ws = w + (long)(s0 + lane) * kWsStride;
      cwt[lane] = ws[0] < mstar ? sas_y(mstar - ws[0], lut) : 1.0f;  // e^0 for m_s = m*
      cl[lane] = ws[1];
    }
    __syncthreads();
    const float* wo = w + (long)s0 * kWsStride + kWsO + 2 * lane;
    int t = 0;
    for (; t + 4 <= cnt; t += 4) {
      float2 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) x[u] = *reinterpret_cast<const float2*>(wo + (t + u) * kWsStride);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        den = __builtin_fmaf(cwt[t + u], cl[t + u], den);
        n0 = __builtin_fmaf(cwt[t + u], x[u].x, n0);
        n1 = __builtin_fmaf(cwt[t + u], x[u].y, n1);
      }
    }
    for (; t < cnt; ++t) {
      const float2 x = *reinterpret_cast<const float2*>(wo + t * kWsStride);
      den = __builtin_fmaf(cwt[t], cl[t], den);
      n0 = __builtin_fmaf(cwt[t], x.x, n0);
      n1 = __builtin_fmaf(cwt[t], x.y, n1);
    }
  }
  _Float16 h2[2] = {(_Float16)(n0 / den), (_Float16)(n1 / den)};
  reinterpret_cast<unsigned*>(a.o)[(long)bh * 64 + lane] = __builtin_bit_cast(unsigned, h2);
  if (a.lse && lane == 0) a.lse[bh] = mstar + logf(den);
}

hipError_t launch_attn_decode(const DecodeArgs& a, hipStream_t stream) {
  const int gp = a.G <= 1 ? 1 : a.G <= 2 ? 2 : a.G <= 4 ? 4 : a.G <= 8 ? 8 : 16;
  // group chunks, then one work-group per (sequence, KV head) for the buffer
  const int total = a.B * a.Hkv * a.nsplit + (a.tk ? a.B * a.Hkv : 0);
  if (a.trace) {
    switch (gp) {
      case 1: hipLaunchKernelGGL((k_attn_decode<1, true>), dim3(total), dim3(64), 0, stream, a); break;
      case 2: hipLaunchKernelGGL((k_attn_decode<2, true>), dim3(total), dim3(64), 0, stream, a); break;
      case 4: hipLaunchKernelGGL((k_attn_decode<4, true>), dim3(total), dim3(64), 0, stream, a); break;
      case 8: hipLaunchKernelGGL((k_attn_decode<8, true>), dim3(total), dim3(64), 0, stream, a); break;
      default: hipLaunchKernelGGL((k_attn_decode<16, true>), dim3(total), dim3(64), 0, stream, a); break;
    }
  } else {
    switch (gp) {
      case 1: hipLaunchKernelGGL((k_attn_decode<1, false>), dim3(total), dim3(64), 0, stream, a); break;
      case 2: hipLaunchKernelGGL((k_attn_decode<2, false>), dim3(total), dim3(64), 0, stream, a); break;
      case 4: hipLaunchKernelGGL((k_attn_decode<4, false>), dim3(total), dim3(64), 0, stream, a); break;
      case 8: hipLaunchKernelGGL((k_attn_decode<8, false>), dim3(total), dim3(64), 0, stream, a); break;
      default: hipLaunchKernelGGL((k_attn_decode<16, false>), dim3(total), dim3(64), 0, stream, a); break;
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.nws < 2) return e;  // no sequence has two states to merge
  hipLaunchKernelGGL(k_decode_combine, dim3(a.B * a.Hq), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace turbo
