/*
 * turbo_oracle.c — plain, slow CPU oracle of TurboAttention (FlashQ + SAS).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  It shares no code,
 * header, table or constant with the GPU library; its constants are typed
 * here from the paper.
 *
 * Paper: Kang et al., "TurboAttention: Efficient attention approximation for
 * high throughputs LLMs", MLSys 2025.  Every function names the passage it
 * follows.  Readings of passages that are ambiguous or garbled are stated
 * where they are used.
 *
 * Precision.  The method's steps whose floating-point result decides an
 * integer (block scales, scores, row maxima, SAS values, the P scale and the
 * quantized P) are computed in IEEE binary32 exactly as written, one rounding
 * per operation (built with -ffp-contract=off, no fast-math).  A product that
 * is then rounded to an integer is formed exactly (in double, where the
 * product of two binary32 numbers is exact) and rounded once, ties to even.
 * The accumulators l and O, which decide no integer, are kept in double.
 *
 * Parity status: every function is pinned by the CPU tests (closed forms,
 * brute force, invariants, reduction to exact softmax attention), except the
 * size of the whole pipeline's error against exact softmax attention, which
 * the paper fixes only through task accuracy: parity unpinned, reported only.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---- constants typed from the paper ---------------------------------- */
/* Symmetric int8 divisor: Algorithms 1 and 2 divide max|X| by 119. */
#define OR_QMAX 119
/* SAS threshold n_r = -6 (Sec. 5.2). */
#define OR_NR 6
/* Query/key block B_r = B_c = 64 and step-2 group length (Sec. 5.2). */
#define OR_BS 64
/* Largest query block of the block-size variants (Table 3: B_r up to 128). */
#define OR_MAXBR 128
/* POLY(x) = -0.1025 x^3 + 0.4626 x^2 - 0.9922 x + 0.9996 (Sec. 4). */
static const float OR_C3 = -0.1025f, OR_C2 = 0.4626f, OR_C1 = -0.9922f, OR_C0 = 0.9996f;

/* Switches of the attention skeleton, for the error decomposition FlashQ
 * alone / SAS alone / both (the operator-level analogue of Appendix C,
 * Table 4) and for the reduction to exact softmax attention. */
typedef struct or_opts {
  int quant; /* 1: FlashQ int8 Q/K/V, quantized P, integer contractions */
  int sas;   /* 1: SAS in place of exp (with the n_r threshold)         */
} or_opts;

int or_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ---- SAS (Sec. 4; Appendix B, Algorithm 3) ---------------------------- */
/* LUT[k] = e^{-k} rounded to binary32 for the integer parts k = 0..6 that
 * survive the threshold (Algorithm 3's zero sentinel is the 0 returned for
 * dropped scores). */
float or_lut(int k) { return (float)exp(-(double)k); }

/* POLY by Horner's rule with fused multiply-adds in binary32. */
float or_poly(float f) {
  float p = fmaf(OR_C3, f, OR_C2);
  p = fmaf(p, f, OR_C1);
  return fmaf(p, f, OR_C0);
}

/* SAS of x = -y <= 0, written for y = m - s >= 0 (Sec. 4): 0 when x < n_r,
 * i.e. y > 6; otherwise LUT(integer part) * POLY(fractional part), with
 * k = floor(y) and f = y - k in [0, 1). */
float or_sas_y(float y) {
  if (!(y <= (float)OR_NR)) return 0.0f;
  float k = floorf(y);
  float f = y - k;
  return or_lut((int)k) * or_poly(f);
}

/* SAS(x) in the paper's sign convention, for x <= 0. */
float or_sas(float x) { return or_sas_y(-x); }

/* Algorithm 3 (offline SAS softmax of the rows of X [R][C]): subtract the
 * row maximum, apply SAS, divide by the row sum (sum and division in double). */
void or_sas_softmax_rows(const float* x, int R, int C, double* out) {
  for (int r = 0; r < R; ++r) {
    const float* xr = x + (size_t)r * C;
    float mx = -INFINITY;
    for (int c = 0; c < C; ++c) mx = xr[c] > mx ? xr[c] : mx;
    double sum = 0.0;
    for (int c = 0; c < C; ++c) {
      double e = or_sas_y(mx - xr[c]);
      out[(size_t)r * C + c] = e;
      sum += e;
    }
    for (int c = 0; c < C; ++c) out[(size_t)r * C + c] /= sum;
  }
}

/* ---- FlashQ step 1: symmetric int8 per block (eq. step1bpq; Alg. 1) --- */
/* s = max|x| / 119 and q = round(x / s), read as: q = nearest integer (ties
 * to even) of x * inv with inv = 119 / max|x| rounded to binary32 once per
 * block; s = max|x| / 119 in binary32.  A block of zeros gets s = 0, q = 0.
 * Returns s. */
float or_block_quant(const float* x, long n, int8_t* q) {
  float amax = 0.0f;
  for (long i = 0; i < n; ++i) {
    float a = fabsf(x[i]);
    amax = a > amax ? a : amax;
  }
  if (amax == 0.0f) {
    memset(q, 0, (size_t)n);
    return 0.0f;
  }
  const float s = amax / (float)OR_QMAX;
  const float inv = (float)OR_QMAX / amax;
  for (long i = 0; i < n; ++i) {
    double r = rint((double)x[i] * (double)inv);
    if (r > OR_QMAX) r = OR_QMAX;
    if (r < -OR_QMAX) r = -OR_QMAX;
    q[i] = (int8_t)r;
  }
  return s;
}

/* ---- FlashQ step 2: asymmetric int4/int2 per channel group ------------ */
/* eq. step2bpq (Sec. 3.1); the s^int, z^int and K^q2 writes of Algorithm 1;
 * the dequantization Q(Q(x)) * s^int + z^int of Sec. 2.3 and Algorithm 2.
 * Readings: the zero point is the group minimum in int8 units (so that the
 * dequantization is code*s + z as Sec. 2.3 and Algorithm 2 write it); the
 * integer scale is the range over 2^bits - 1 rounded up and at least 1, so
 * no code leaves 0..2^bits-1; the code is the nearest level with ties
 * rounded up, code = floor((2 (q - z) + s) / (2 s)).
 * The group is n values of one channel at `stride`; codes at code_stride. */
void or_step2_group(const int8_t* q1, int n, long stride, int bits, uint8_t* s_out,
                    int8_t* z_out, uint8_t* code, long code_stride) {
  int mn = 127, mx = -128;
  for (int i = 0; i < n; ++i) {
    int v = q1[(long)i * stride];
    mn = v < mn ? v : mn;
    mx = v > mx ? v : mx;
  }
  const int levels = (1 << bits) - 1;
  int s = (mx - mn + levels - 1) / levels;
  if (s < 1) s = 1;
  *s_out = (uint8_t)s;
  *z_out = (int8_t)mn;
  for (int i = 0; i < n; ++i) {
    int dlt = q1[(long)i * stride] - mn;
    code[(long)i * code_stride] = (uint8_t)((2 * dlt + s) / (2 * s));
  }
}

/* ---- FlashQ of a whole K/V cache -------------------------------------- */
/* k, v: float [B][Hkv][N][d] holding fp16 values; bits: int [Hkv] (4 or 2).
 * Outputs in natural logical layouts:
 *   k8, v8          int8  [B][Hkv][N][d]        (step 1, per 64-token block)
 *   sk, sv          float [B][Hkv][nb], nb = ceil(N/64)
 *   kc, vc          uint8 [B][Hkv][ng*64][d]    (step-2 codes), ng = floor(N/64)
 *   ks, kz, vs, vz  [B][Hkv][ng][d]             (uint8 scale, int8 zero)
 * kc == NULL skips step 2.  A partial last block (N % 64 rows) is quantized
 * over its valid rows only and gets no step-2 group. */
void or_quantize_kv(const float* k, const float* v, int B, int Hkv, int N, int d, const int* bits,
                    int8_t* k8, int8_t* v8, float* sk, float* sv, uint8_t* kc, uint8_t* vc,
                    uint8_t* ks, int8_t* kz, uint8_t* vs, int8_t* vz) {
  const int nb = (N + OR_BS - 1) / OR_BS, ng = N / OR_BS;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < Hkv; ++h) {
      const size_t u = (size_t)b * Hkv + h;
      const size_t base = u * (size_t)N * d;
      for (int j = 0; j < nb; ++j) {
        const int r0 = j * OR_BS, nr = (N - r0) < OR_BS ? (N - r0) : OR_BS;
        const size_t off = base + (size_t)r0 * d;
        sk[u * nb + j] = or_block_quant(k + off, (long)nr * d, k8 + off);
        sv[u * nb + j] = or_block_quant(v + off, (long)nr * d, v8 + off);
      }
      if (!kc) continue;
      for (int g = 0; g < ng; ++g)
        for (int c = 0; c < d; ++c) {
          const size_t src = base + (size_t)g * OR_BS * d + c;
          const size_t dst = u * (size_t)ng * OR_BS * d + (size_t)g * OR_BS * d + c;
          const size_t m = (u * ng + g) * (size_t)d + c;
          or_step2_group(k8 + src, OR_BS, d, bits[h], ks + m, kz + m, kc + dst, d);
          or_step2_group(v8 + src, OR_BS, d, bits[h], vs + m, vz + m, vc + dst, d);
        }
    }
}

/* Step 1 alone with key/value blocks of bc tokens (Table 3 varies B_c):
 * k8, v8 int8 [B][Hkv][N][d]; sk, sv float [B][Hkv][ceil(N/bc)].  The last
 * block is quantized over its valid rows only. */
void or_quantize_kv_blocks(const float* k, const float* v, int B, int Hkv, int N, int d, int bc,
                           int8_t* k8, int8_t* v8, float* sk, float* sv) {
  const int nbc = (N + bc - 1) / bc;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < Hkv; ++h) {
      const size_t u = (size_t)b * Hkv + h;
      for (int j = 0; j < nbc; ++j) {
        const int r0 = j * bc, nr = (N - r0) < bc ? (N - r0) : bc;
        const size_t off = (u * (size_t)N + r0) * d;
        sk[u * nbc + j] = or_block_quant(k + off, (long)nr * d, k8 + off);
        sv[u * nbc + j] = or_block_quant(v + off, (long)nr * d, v8 + off);
      }
    }
}

/* ---- the online softmax step shared by Algorithms 1 and 2 ------------- */
/* Exponential factor e^{-(hi - lo)} of the online softmax for hi >= lo.
 * With FlashQ on, hi and lo are binary32 values and their difference is
 * rounded to binary32 (as the scores are binary32); with FlashQ off the
 * difference stays in double.  SAS or exact exp per the options. */
static double or_e(const or_opts* o, double hi, double lo) {
  if (o->quant) {
    const float y = (float)hi - (float)lo;
    return o->sas ? (double)or_sas_y(y) : (double)(float)exp(-(double)y);
  }
  const double y = hi - lo;
  return o->sas ? (double)or_sas_y((float)y) : exp(-y);
}

/* Factor that rescales a running state (l, O of Algorithms 1 and 2; the
 * weight of a chunk in the split-KV merge) when the maximum it was taken
 * against moves from lo to hi >= lo.  Reading: SAS stands in for e^x; where
 * the maximum has not moved the exponent is exactly 0 and the factor is
 * e^0 = 1, so the state is left as it is.  Evaluating SAS there would give
 * the fit error POLY(0) = 0.9996 of Sec. 4, compounded once per online step,
 * which makes the result depend on how many steps (tiles, chunks) the keys
 * are cut into.  A moved maximum takes SAS (or exp) of the difference, and
 * lo = -inf (an empty state) gives 0.  The SAS value of an individual score
 * (P~ = SAS(0) for the row's maximum) is not a rescale and keeps POLY(0). */
static double or_rescale(const or_opts* o, double hi, double lo) {
  if (lo == -INFINITY) return 0.0;
  if (hi == lo) return 1.0;
  return or_e(o, hi, lo);
}

/* Running state of one query row: m (binary32-valued when FlashQ is on),
 * l and O (double). */
typedef struct or_row {
  double m, l;
  double* O;
} or_row;

/* Optional trace of one tile, for checking another implementation's
 * integers bit for bit: prefill selects (b, h, i, j) = (batch, query head,
 * query block of B_r rows, key block of B_c keys); decode selects (b, h, j) =
 * (batch, query head, group) and ignores i (B_r = 1, B_c = 64).  Buffers are
 * filled only for the selected tile:
 *   q8    int8  [B_r][d]   quantized query block (decode: row 0 only)
 *   sacc  int32 [B_r][B_c] QK^T accumulators (row r, key t) of visible pairs
 *   qp    int8  [B_r][B_c] Q(P~) (0 where not visible)
 *   pvacc int32 [B_r][d]   Q(P~) V^{q1} accumulators
 *   sq    query block scale; pmax tile maximum of P~ (decode: of the row). */
typedef struct or_trace {
  int b, h, i, j;
  int hit;
  int8_t* q8;
  int32_t* sacc;
  int8_t* qp;
  int32_t* pvacc;
  float sq, pmax;
} or_trace;

/* One key tile for a set of query rows (Algorithm 1 inner loop; Algorithm 2
 * with one row).  For row r and key t:
 *   sc[r*ldsc + t]  score S (binary32 value when FlashQ is on), valid where
 *                   vis[r*ldsc + t] != 0;
 *   V rows          vq (int8, FlashQ on, scaled by sv) or vf (float values,
 *                   FlashQ off), row t at vq/vf + t*d.
 * Steps, in the order of Algorithm 1:
 *   m_new = max(m_old, rowmax S);  P~ = SAS(S - m_new);
 *   alpha = SAS(m_old - m_new), 1 when m_new = m_old (or_rescale);
 *   l = alpha l + rowsum P~;
 *   s_P = max P~ / 119 over the tile, Q(P~) = round(P~ / s_P) (FlashQ on);
 *   O = alpha O + s_P s_V Q(P~) V^{q1}.
 * A row with no visible key is left untouched.  P scale granularity: the
 * whole tile (all processed rows and visible keys) for prefill (B_r x B_c,
 * Algorithm 1) and one row for decode (1 x B_c, Algorithm 2).
 * Work buffers p (float) and pd (double) hold nr*ldsc values; qp nr*ldsc. */
static void or_tile(const or_opts* o, or_row* rows, int nr, int nk, const double* sc,
                    const unsigned char* vis, int ldsc, const int8_t* vq, float sv,
                    const float* vf, int d, float* p, double* pd, int8_t* qp,
                    or_trace* tr) {
  double alpha[OR_MAXBR];
  int act[OR_MAXBR];
  float pmax = 0.0f;
  for (int r = 0; r < nr; ++r) {
    act[r] = 0;
    double smax = -INFINITY;
    for (int t = 0; t < nk; ++t)
      if (vis[r * ldsc + t]) {
        act[r] = 1;
        smax = sc[r * ldsc + t] > smax ? sc[r * ldsc + t] : smax;
      }
    if (!act[r]) continue;
    const double mold = rows[r].m;
    const double mnew = mold > smax ? mold : smax;
    double rowsum = 0.0;
    for (int t = 0; t < nk; ++t) {
      double e = vis[r * ldsc + t] ? or_e(o, mnew, sc[r * ldsc + t]) : 0.0;
      p[r * ldsc + t] = (float)e;
      pd[r * ldsc + t] = e;
      rowsum += e;
      if ((float)e > pmax) pmax = (float)e;
    }
    alpha[r] = or_rescale(o, mnew, mold);
    rows[r].l = alpha[r] * rows[r].l + rowsum;
    rows[r].m = mnew;
    for (int e = 0; e < d; ++e) rows[r].O[e] *= alpha[r];
  }
  if (tr) tr->pmax = pmax;
  if (o->quant) {
    if (!(pmax > 0.0f)) return; /* nothing survives: the tile adds no PV */
    const float inv = (float)OR_QMAX / pmax;
    const float sp = pmax / (float)OR_QMAX;
    const double spv = (double)(float)(sp * sv);
    for (int r = 0; r < nr; ++r) {
      if (!act[r]) continue;
      for (int t = 0; t < nk; ++t) {
        qp[r * ldsc + t] = (int8_t)rint((double)p[r * ldsc + t] * (double)inv);
        if (tr) tr->qp[r * ldsc + t] = vis[r * ldsc + t] ? qp[r * ldsc + t] : 0;
      }
      for (int e = 0; e < d; ++e) {
        int32_t acc = 0;
        for (int t = 0; t < nk; ++t)
          if (vis[r * ldsc + t]) acc += (int32_t)qp[r * ldsc + t] * (int32_t)vq[(size_t)t * d + e];
        rows[r].O[e] += spv * (double)acc;
        if (tr) tr->pvacc[(size_t)r * d + e] = acc;
      }
    }
  } else {
    for (int r = 0; r < nr; ++r) {
      if (!act[r]) continue;
      for (int e = 0; e < d; ++e) {
        double acc = 0.0;
        for (int t = 0; t < nk; ++t)
          if (vis[r * ldsc + t]) acc += pd[r * ldsc + t] * (double)vf[(size_t)t * d + e];
        rows[r].O[e] += acc;
      }
    }
  }
}

/* ---- Algorithm 1: prefill --------------------------------------------- */
/* q: float [B][Hq][N][d]; k, v: float [B][Hkv][N][d] (fp16 values).
 * Query head h uses KV head h / (Hq/Hkv).  causal: key t visible to query r
 * iff t <= r; a (row, tile) pair without a visible key is not processed.
 * Outputs: o double [B][Hq][N][d] = O / l before any rounding to fp16;
 * lse double [B][Hq][N] = m + ln l.  Only query blocks i0 <= i < i1 are
 * computed (i0 = i1 = -1: all); other rows of o and lse are not written.
 * Readings: the softmax temperature of eq. threesteps multiplies the scores,
 * S = fl(fl(acc) * fl(fl(s_Q * s_K) * sm_scale)); Algorithm 1 writes the
 * accumulator update with the inverse of diag(SAS(m_old - m_new)), which
 * would not compute a softmax and disagrees with the l update next to it, so
 * O is multiplied by that factor; when the maximum does not move the factor
 * is e^0 = 1 (or_rescale).
 * Block sizes (Table 3 varies them): Q is quantized per br rows of a head
 * (br = B_r in {32, 64, 128}); K and V are quantized per bc tokens (bc = B_c
 * in {32, 64, 128}), each online step covers bc keys and the P scale covers
 * the br x bc tile.  Query blocks i0..i1 count br-row blocks; the trace
 * selects a (br-row block, bc-key block) tile. */
void or_attn_prefill_blocks(const float* q, const float* k, const float* v, int B, int Hq,
                            int Hkv, int N, int d, float sm_scale, int causal, or_opts opts,
                            int br, int bc, double* o, double* lse, or_trace* tr, int i0,
                            int i1) {
  const int G = Hq / Hkv, nb = (N + bc - 1) / bc, nbq = (N + br - 1) / br;
#pragma omp parallel
  {
    int8_t* k8 = malloc((size_t)N * d + 1);
    int8_t* v8 = malloc((size_t)N * d + 1);
    float* sk = malloc(sizeof(float) * (nb + 1));
    float* sv = malloc(sizeof(float) * (nb + 1));
    int8_t* q8 = malloc((size_t)br * d);
    double* sc = malloc(sizeof(double) * br * bc);
    unsigned char* vis = malloc((size_t)br * bc);
    float* p = malloc(sizeof(float) * br * bc);
    double* pd = malloc(sizeof(double) * br * bc);
    int8_t* qp = malloc((size_t)br * bc);
    double* Obuf = malloc(sizeof(double) * br * d);
    or_row rows[OR_MAXBR];
#pragma omp for collapse(2) schedule(dynamic)
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < Hq; ++h) {
        const int kh = h / G;
        const float* kk = k + ((size_t)b * Hkv + kh) * (size_t)N * d;
        const float* vv = v + ((size_t)b * Hkv + kh) * (size_t)N * d;
        const float* qq = q + ((size_t)b * Hq + h) * (size_t)N * d;
        if (opts.quant)
          for (int j = 0; j < nb; ++j) { /* K_j^{q1}, V_j^{q1} (eq. step1bpq) */
            const int r0 = j * bc, nr = (N - r0) < bc ? (N - r0) : bc;
            sk[j] = or_block_quant(kk + (size_t)r0 * d, (long)nr * d, k8 + (size_t)r0 * d);
            sv[j] = or_block_quant(vv + (size_t)r0 * d, (long)nr * d, v8 + (size_t)r0 * d);
          }
        for (int i = i0 < 0 ? 0 : i0; i < (i1 < 0 || i1 > nbq ? nbq : i1); ++i) {
          const int q0 = i * br, nq = (N - q0) < br ? (N - q0) : br;
          float sq = 0.0f; /* Q_i^{q1} (eq. step1bpq) */
          if (opts.quant) sq = or_block_quant(qq + (size_t)q0 * d, (long)nq * d, q8);
          const int trq = tr && tr->b == b && tr->h == h && tr->i == i;
          if (trq) {
            memcpy(tr->q8, q8, (size_t)nq * d);
            tr->sq = sq;
          }
          for (int r = 0; r < nq; ++r) {
            rows[r].m = -INFINITY;
            rows[r].l = 0.0;
            rows[r].O = Obuf + (size_t)r * d;
          }
          memset(Obuf, 0, sizeof(double) * br * d);
          for (int j = 0; j < nb; ++j) {
            const int k0 = j * bc, nk = (N - k0) < bc ? (N - k0) : bc;
            if (causal && k0 > q0 + nq - 1) break;
            /* S_i^{(j)} = s_Q s_K Q_i^{q1} K_j^{q1 T} (times sm_scale) */
            const float c = (float)(sq * sk[j]) * sm_scale;
            for (int r = 0; r < nq; ++r)
              for (int t = 0; t < nk; ++t) {
                const int visible = !causal || (k0 + t <= q0 + r);
                vis[r * bc + t] = (unsigned char)visible;
                if (!visible) continue;
                if (opts.quant) {
                  int32_t acc = 0;
                  for (int e = 0; e < d; ++e)
                    acc += (int32_t)q8[(size_t)r * d + e] * (int32_t)k8[(size_t)(k0 + t) * d + e];
                  sc[r * bc + t] = (double)((float)acc * c);
                  if (trq && tr->j == j) tr->sacc[r * bc + t] = acc;
                } else {
                  double acc = 0.0;
                  for (int e = 0; e < d; ++e)
                    acc += (double)qq[(size_t)(q0 + r) * d + e] * (double)kk[(size_t)(k0 + t) * d + e];
                  sc[r * bc + t] = acc * (double)sm_scale;
                }
              }
            or_trace* tt = (trq && tr->j == j) ? tr : NULL;
            if (tt) tt->hit = 1;
            or_tile(&opts, rows, nq, nk, sc, vis, bc, v8 + (size_t)k0 * d, sv[j],
                    vv + (size_t)k0 * d, d, p, pd, qp, tt);
          }
          for (int r = 0; r < nq; ++r) {
            const size_t row = ((size_t)b * Hq + h) * (size_t)N + q0 + r;
            for (int e = 0; e < d; ++e) o[row * d + e] = rows[r].O[e] / rows[r].l;
            lse[row] = rows[r].m + log(rows[r].l);
          }
        }
      }
    free(k8); free(v8); free(sk); free(sv); free(q8); free(sc); free(vis); free(p); free(pd);
    free(qp); free(Obuf);
  }
}

/* Algorithm 1 with the paper's query/key blocks B_r = B_c = 64. */
void or_attn_prefill(const float* q, const float* k, const float* v, int B, int Hq, int Hkv,
                     int N, int d, float sm_scale, int causal, or_opts opts, double* o,
                     double* lse, or_trace* tr, int i0, int i1) {
  or_attn_prefill_blocks(q, k, v, B, Hq, Hkv, N, d, sm_scale, causal, opts, OR_BS, OR_BS, o, lse,
                         tr, i0, i1);
}

/* ---- Algorithm 2: decode over the compressed cache -------------------- */
/* q: float [B][Hq][d] (fp16 values).  Cache in the logical layouts written
 * by or_quantize_kv for length Nc: kc, vc uint8 [B][Hkv][Nc][d]; ks, kz, vs,
 * vz [B][Hkv][Nc/64][d]; sk, sv float [B][Hkv][Nc/64].  seq_lens[b] tokens
 * are cached for sequence b (only its floor(seq_len/64) full groups are
 * attended).  Steps (Algorithm 2): s_Q = max|q|/119 and q^{q1} per (b, query
 * head); per group j: K_j^{q1} = K_j^{q2} s^int + z^int and V_j^{q1} likewise
 * (Sec. 2.3 dequantization); S_j = s_Q s_K q^{q1} K_j^{q1 T} (times sm_scale);
 * the online SAS step with the P scale taken over the row's 64 keys.
 * Split-KV extension (not in the paper): chunks of `split` groups each run
 * the loop from m = -inf; with more than one chunk the states are merged in
 * ascending order with m* = max m_s, w_s = SAS(m_s - m*) (1 for m_s = m*),
 * O = sum w_s O_s / sum w_s l_s, L = m* + ln(sum w_s l_s).
 * No group: o = 0, lse = -inf.  Outputs o double [B][Hq][d], lse [B][Hq].
 * With the int8 buffer of Sec. 3.3 (tk != NULL): the seq_len - 64 ng newest
 * tokens (at most 63) sit in tk [B][Hkv][64][d] (token-major) and
 * tv [B][Hkv][d][64] (channel-major) with the universal scales tsk, tsv
 * [B][Hkv].  Reading: they are attended as one more chunk after the group
 * chunks (same online step, P scale over the row's buffered keys), merged
 * with the others as above. */
void or_attn_decode(const float* q, const uint8_t* kc, const uint8_t* vc, const uint8_t* ks,
                    const int8_t* kz, const uint8_t* vs, const int8_t* vz, const float* sk,
                    const float* sv, const int* seq_lens, int B, int Hq, int Hkv, int Nc, int d,
                    float sm_scale, int split, or_opts opts, double* o, double* lse,
                    or_trace* tr, const int8_t* tk, const int8_t* tv, const float* tsk,
                    const float* tsv) {
  const int G = Hq / Hkv, ngc = Nc / OR_BS;
#pragma omp parallel
  {
    int8_t* k1 = malloc((size_t)OR_BS * d);
    int8_t* v1 = malloc((size_t)OR_BS * d);
    int8_t q8[1024];
    double sc[OR_BS];
    unsigned char vis[OR_BS];
    float p[OR_BS];
    double pd[OR_BS];
    int8_t qp[OR_BS];
    double* Os = malloc(sizeof(double) * d);
    double* num = malloc(sizeof(double) * d);
    float* vf = malloc(sizeof(float) * OR_BS * d);
#pragma omp for collapse(2) schedule(dynamic)
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < Hq; ++h) {
        const int kh = h / G;
        const size_t u = (size_t)b * Hkv + kh;
        const size_t orow = (size_t)b * Hq + h;
        int ng = seq_lens[b] / OR_BS;
        if (ng > ngc) ng = ngc;
        if (ng < 0) ng = 0;
        const float* qq = q + orow * d;
        const float sq = or_block_quant(qq, d, q8);
        const int trq = tr && tr->b == b && tr->h == h;
        if (trq) {
          memcpy(tr->q8, q8, (size_t)d);
          tr->sq = sq;
        }
        /* the int8 buffer of Sec. 3.3 holds the seq_len - 64 ng newest tokens */
        int ntail = tk ? seq_lens[b] - ng * OR_BS : 0;
        if (ntail < 0) ntail = 0;
        if (ntail > OR_BS - 1) ntail = OR_BS - 1;
        const int ngchunks = ng == 0 ? 0 : (ng + split - 1) / split;
        const int nsplit = ngchunks + (ntail > 0);
        double mstar = -INFINITY, den = 0.0;
        for (int e = 0; e < d; ++e) num[e] = 0.0;
        /* first pass over chunks for m* (needed only when merging) */
        double* ms = malloc(sizeof(double) * (nsplit + 1));
        double* ls = malloc(sizeof(double) * (nsplit + 1));
        double* Oall = malloc(sizeof(double) * (size_t)(nsplit + 1) * d);
        for (int s = 0; s < nsplit; ++s) {
          or_row row = {-INFINITY, 0.0, Oall + (size_t)s * d};
          for (int e = 0; e < d; ++e) row.O[e] = 0.0;
          if (s == ngchunks) {
            /* the buffer: one more chunk of ntail int8 tokens with the
             * universal scales, merged like the others */
            const int8_t* kb = tk + u * (size_t)OR_BS * d;
            const int8_t* vbuf = tv + u * (size_t)d * OR_BS; /* channel-major */
            for (int t = 0; t < OR_BS; ++t)
              for (int e = 0; e < d; ++e) {
                k1[t * d + e] = t < ntail ? kb[(size_t)t * d + e] : 0;
                v1[t * d + e] = t < ntail ? vbuf[(size_t)e * OR_BS + t] : 0;
              }
            const float c = (float)(sq * tsk[u]) * sm_scale;
            for (int t = 0; t < OR_BS; ++t) {
              vis[t] = (unsigned char)(t < ntail);
              if (!vis[t]) continue;
              if (opts.quant) {
                int32_t acc = 0;
                for (int e = 0; e < d; ++e) acc += (int32_t)q8[e] * (int32_t)k1[t * d + e];
                sc[t] = (double)((float)acc * c);
                if (trq && tr->j == ng) tr->sacc[t] = acc;
              } else {
                double acc = 0.0;
                for (int e = 0; e < d; ++e) acc += (double)qq[e] * (double)k1[t * d + e] * tsk[u];
                sc[t] = acc * (double)sm_scale;
                for (int e = 0; e < d; ++e) vf[t * d + e] = (float)((double)v1[t * d + e] * tsv[u]);
              }
            }
            or_trace* tt = (trq && tr->j == ng) ? tr : NULL;
            if (tt) tt->hit = 1;
            or_tile(&opts, &row, 1, OR_BS, sc, vis, OR_BS, v1, tsv[u], vf, d, p, pd, qp, tt);
            ms[s] = row.m;
            ls[s] = row.l;
            if (row.m > mstar) mstar = row.m;
            continue;
          }
          const int g1 = (s + 1) * split < ng ? (s + 1) * split : ng;
          for (int g = s * split; g < g1; ++g) {
            const size_t cb = (u * (size_t)ngc * OR_BS + (size_t)g * OR_BS) * d;
            const size_t mb = (u * ngc + g) * (size_t)d;
            for (int t = 0; t < OR_BS; ++t)
              for (int e = 0; e < d; ++e) {
                /* K^{q1} = K^{q2} s^int + z^int, V^{q1} likewise */
                k1[t * d + e] = (int8_t)(kc[cb + (size_t)t * d + e] * ks[mb + e] + kz[mb + e]);
                v1[t * d + e] = (int8_t)(vc[cb + (size_t)t * d + e] * vs[mb + e] + vz[mb + e]);
              }
            const float c = (float)(sq * sk[u * ngc + g]) * sm_scale;
            for (int t = 0; t < OR_BS; ++t) {
              vis[t] = 1;
              if (opts.quant) {
                int32_t acc = 0;
                for (int e = 0; e < d; ++e) acc += (int32_t)q8[e] * (int32_t)k1[t * d + e];
                sc[t] = (double)((float)acc * c);
                if (trq && tr->j == g) tr->sacc[t] = acc;
              } else { /* dequantized cache values against the fp16 query */
                double acc = 0.0;
                const double skg = sk[u * ngc + g], svg = sv[u * ngc + g];
                for (int e = 0; e < d; ++e) acc += (double)qq[e] * (double)k1[t * d + e] * skg;
                sc[t] = acc * (double)sm_scale;
                for (int e = 0; e < d; ++e) vf[t * d + e] = (float)((double)v1[t * d + e] * svg);
              }
            }
            or_trace* tt = (trq && tr->j == g) ? tr : NULL;
            if (tt) tt->hit = 1;
            or_tile(&opts, &row, 1, OR_BS, sc, vis, OR_BS, v1, sv[u * ngc + g], vf, d, p, pd, qp, tt);
          }
          ms[s] = row.m;
          ls[s] = row.l;
          if (row.m > mstar) mstar = row.m;
        }
        if (nsplit == 0) {
          for (int e = 0; e < d; ++e) o[orow * d + e] = 0.0;
          lse[orow] = -INFINITY;
        } else if (nsplit == 1) {
          for (int e = 0; e < d; ++e) o[orow * d + e] = Oall[e] / ls[0];
          lse[orow] = ms[0] + log(ls[0]);
        } else {
          for (int s = 0; s < nsplit; ++s) {
            const double w = or_rescale(&opts, mstar, ms[s]);
            den += w * ls[s];
            for (int e = 0; e < d; ++e) num[e] += w * Oall[(size_t)s * d + e];
          }
          for (int e = 0; e < d; ++e) o[orow * d + e] = num[e] / den;
          lse[orow] = mstar + log(den);
        }
        free(ms); free(ls); free(Oall);
        (void)Os;
      }
    free(k1); free(v1); free(Os); free(num); free(vf);
  }
}

/* ---- exact softmax attention in double (eq. stdattn / threesteps) ----- */
/* The error reference: H = softmax(Q K^T * sm_scale) V row by row, on the
 * given values (fp16 inputs), with causal masking when requested.
 * q [B][Hq][Nq][d], k, v [B][Hkv][Nk][d].  Query row r sits at absolute
 * position r + (Nk - Nq) (so Nq = 1 with Nk keys is a decode step).
 * Outputs o [B][Hq][Nq][d], lse [B][Hq][Nq] (natural log). */
void or_attn_exact(const float* q, const float* k, const float* v, int B, int Hq, int Hkv, int Nq,
                   int Nk, int d, double sm_scale, int causal, double* o, double* lse) {
  const int G = Hq / Hkv;
#pragma omp parallel
  {
    double* s = malloc(sizeof(double) * (Nk + 1));
#pragma omp for collapse(3) schedule(dynamic)
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < Hq; ++h)
        for (int r = 0; r < Nq; ++r) {
          const float* kk = k + ((size_t)b * Hkv + h / G) * (size_t)Nk * d;
          const float* vv = v + ((size_t)b * Hkv + h / G) * (size_t)Nk * d;
          const float* qr = q + (((size_t)b * Hq + h) * Nq + r) * d;
          const int last = causal ? r + (Nk - Nq) : Nk - 1;
          double mx = -INFINITY;
          for (int t = 0; t <= last; ++t) {
            double acc = 0.0;
            for (int e = 0; e < d; ++e) acc += (double)qr[e] * (double)kk[(size_t)t * d + e];
            s[t] = acc * sm_scale;
            mx = s[t] > mx ? s[t] : mx;
          }
          double sum = 0.0;
          for (int t = 0; t <= last; ++t) {
            s[t] = exp(s[t] - mx);
            sum += s[t];
          }
          double* orow = o + (((size_t)b * Hq + h) * Nq + r) * d;
          for (int e = 0; e < d; ++e) {
            double acc = 0.0;
            for (int t = 0; t <= last; ++t) acc += s[t] * (double)vv[(size_t)t * d + e];
            orow[e] = acc / sum;
          }
          lse[((size_t)b * Hq + h) * Nq + r] = mx + log(sum);
        }
    free(s);
  }
}

/* ---- vector helpers for the Python wrapper ---------------------------- */
/* ---- Sec. 3.3: the int8 KV-cache buffer -------------------------------- */
/* Universal-scale int8 code of x (Sec. 3.3): nearest integer (ties to even)
 * of x * inv, inv = 1/s rounded to binary32, clamped to [-119, 119] (values
 * beyond the scale's range are clamped, as Sec. 3.3 prescribes); s = 0
 * gives 0. */
static int8_t or_quant_univ(float x, float s) {
  if (!(s > 0.0f)) return 0;
  const float inv = 1.0f / s;
  double r = rint((double)x * (double)inv);
  if (r > OR_QMAX) r = OR_QMAX;
  if (r < -OR_QMAX) r = -OR_QMAX;
  return (int8_t)r;
}

/* Start of the buffer after a prefill of N tokens (Sec. 3.3).  Reading: the
 * universal scale of (b, kv-head) is the largest step-1 block scale of its
 * prefill (sk, sv [B][Hkv][ceil(N/64)] from or_quantize_kv), so the prefill's
 * range is representable; the N mod 64 tokens that form no step-2 group are
 * the buffer's first entries, coded with that scale.  tk [B][Hkv][64][d]
 * token-major, tv [B][Hkv][d][64] channel-major; unused rows are 0. */
void or_tail_init(const float* k, const float* v, int B, int Hkv, int N, int d, const float* sk,
                  const float* sv, int8_t* tk, int8_t* tv, float* tsk, float* tsv) {
  const int nb = (N + OR_BS - 1) / OR_BS, ng = N / OR_BS, nt = N - ng * OR_BS;
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < Hkv; ++h) {
      const size_t u = (size_t)b * Hkv + h;
      float mk = 0.0f, mv = 0.0f;
      for (int j = 0; j < nb; ++j) {
        mk = sk[u * nb + j] > mk ? sk[u * nb + j] : mk;
        mv = sv[u * nb + j] > mv ? sv[u * nb + j] : mv;
      }
      tsk[u] = mk;
      tsv[u] = mv;
      for (int t = 0; t < OR_BS; ++t)
        for (int e = 0; e < d; ++e) {
          const size_t src = (u * (size_t)N + (size_t)ng * OR_BS + t) * d + e;
          tk[(u * OR_BS + t) * d + e] = t < nt ? or_quant_univ(k[src], mk) : 0;
          tv[(u * d + e) * OR_BS + t] = t < nt ? or_quant_univ(v[src], mv) : 0;
        }
    }
}

/* One decoding step's new key and value per (b, kv-head) (Sec. 3.3): the
 * token at position p = seq_lens[b] (before the append) goes to buffer row
 * p mod 64 with the universal scales.  When that row is the 64th, the buffer
 * is compressed like any other group (step 2, eq. step2bpq) into group
 * p / 64 of the cache, whose float scales are the universal scales; groups
 * at or beyond Nc/64 are not written (the caller's cache is full).
 * knew, vnew float [B][Hkv][d]; cache arrays as in or_quantize_kv with
 * Nc = ngc * 64 and sk, sv [B][Hkv][ngc]; bits int [Hkv]. */
void or_append_kv(const float* knew, const float* vnew, int B, int Hkv, int d,
                  const int* seq_lens, const int* bits, int Nc, uint8_t* kc, uint8_t* vc,
                  uint8_t* ks, int8_t* kz, uint8_t* vs, int8_t* vz, float* sk, float* sv,
                  int8_t* tk, int8_t* tv, const float* tsk, const float* tsv) {
  const int ngc = Nc / OR_BS;
  int8_t* col = malloc((size_t)OR_BS);
  for (int b = 0; b < B; ++b) {
    const int p = seq_lens[b];
    if (p < 0) continue;
    const int r = p % OR_BS, g = p / OR_BS;
    for (int h = 0; h < Hkv; ++h) {
      const size_t u = (size_t)b * Hkv + h;
      for (int e = 0; e < d; ++e) {
        tk[(u * OR_BS + r) * d + e] = or_quant_univ(knew[u * d + e], tsk[u]);
        tv[(u * d + e) * OR_BS + r] = or_quant_univ(vnew[u * d + e], tsv[u]);
      }
      if (r != OR_BS - 1 || g >= ngc) continue;
      for (int e = 0; e < d; ++e) {
        const size_t m = (u * ngc + g) * (size_t)d + e;
        const size_t dst = (u * (size_t)ngc * OR_BS + (size_t)g * OR_BS) * d + e;
        or_step2_group(tk + u * OR_BS * (size_t)d + e, OR_BS, d, bits[h], ks + m, kz + m, kc + dst, d);
        for (int t = 0; t < OR_BS; ++t) col[t] = tv[(u * d + e) * OR_BS + t];
        or_step2_group(col, OR_BS, 1, bits[h], vs + m, vz + m, vc + dst, d);
      }
      sk[u * ngc + g] = tsk[u];
      sv[u * ngc + g] = tsv[u];
    }
  }
  free(col);
}

/* ---- Sec. 3.2: head-wise mixed precision ------------------------------ */
/* Priority of KV head h (Sec. 3.2, the priority equation):
 *   gap_c   = max - min of channel c over every token of every sequence;
 *   gap^(h) = max - min over all channels (and tokens) of the head;
 *   std^(h) = standard deviation of the channel-wise gaps gap_c
 *             (population form: the mean of squared deviations);
 *   priority^(h) = gap^(h) * std^(h).
 * Readings: the statistics are taken on K, the tensor whose heads carry the
 * large-magnitude channels of Fig. 3 (V shows no outlier pattern), over the
 * whole prefill batch of one layer (the bit widths are per layer and head).
 * k: float [B][Hkv][N][d] (fp16 values).  Computed in double. */
void or_head_priority(const float* k, int B, int Hkv, int N, int d, double* prio) {
  double* gap = malloc(sizeof(double) * (size_t)d);
  for (int h = 0; h < Hkv; ++h) {
    double gmax = -INFINITY, gmin = INFINITY;
    for (int c = 0; c < d; ++c) {
      double cmax = -INFINITY, cmin = INFINITY;
      for (int b = 0; b < B; ++b)
        for (int t = 0; t < N; ++t) {
          const double x = k[(((size_t)b * Hkv + h) * N + t) * d + c];
          cmax = x > cmax ? x : cmax;
          cmin = x < cmin ? x : cmin;
        }
      gap[c] = cmax - cmin;
      gmax = cmax > gmax ? cmax : gmax;
      gmin = cmin < gmin ? cmin : gmin;
    }
    double mean = 0.0;
    for (int c = 0; c < d; ++c) mean += gap[c];
    mean /= d;
    double var = 0.0;
    for (int c = 0; c < d; ++c) var += (gap[c] - mean) * (gap[c] - mean);
    var /= d;
    prio[h] = (gmax - gmin) * sqrt(var);
  }
  free(gap);
}

/* Sec. 3.2 quantization strategy: the n_int2 heads of lowest priority (rank
 * <= n_h) get 2 bits, the others 4.  Equal priorities rank by head index. */
void or_int2_heads(const double* prio, int Hkv, int n_int2, uint8_t* bits) {
  for (int h = 0; h < Hkv; ++h) {
    int rank = 0; /* number of heads ranked before h */
    for (int g = 0; g < Hkv; ++g)
      if (prio[g] < prio[h] || (prio[g] == prio[h] && g < h)) ++rank;
    bits[h] = rank < n_int2 ? 2 : 4;
  }
}

void or_sas_y_vec(const float* y, long n, float* out) {
  for (long i = 0; i < n; ++i) out[i] = or_sas_y(y[i]);
}
void or_poly_vec(const float* f, long n, float* out) {
  for (long i = 0; i < n; ++i) out[i] = or_poly(f[i]);
}
/* Step 1 over nblk consecutive blocks of n values each. */
void or_block_quant_vec(const float* x, long nblk, long n, int8_t* q, float* s) {
  for (long b = 0; b < nblk; ++b) s[b] = or_block_quant(x + b * n, n, q + b * n);
}
/* Step 2 over ncol independent groups of n values (column-major groups:
 * group c is q1[c], q1[c + ncol], ...). */
void or_step2_vec(const int8_t* q1, int n, int ncol, int bits, uint8_t* s, int8_t* z,
                  uint8_t* code) {
  for (int c = 0; c < ncol; ++c) or_step2_group(q1 + c, n, ncol, bits, s + c, z + c, code + c, ncol);
}
