/*
 * Sanitizer driver of the CPU oracle (test infrastructure): built together
 * with oracle/turbo_oracle.c under AddressSanitizer and UndefinedBehavior-
 * Sanitizer, it runs every oracle routine on small ragged inputs (partial
 * blocks, empty sequences, int4 and int2 heads, every block size, the int8
 * buffer with a flush) so that an out-of-bounds access or undefined
 * arithmetic in the oracle aborts the run.  Exit status 0: clean.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct or_opts { int quant, sas; } or_opts;
typedef struct or_trace {
  int b, h, i, j, hit;
  int8_t *q8;
  int32_t *sacc;
  int8_t *qp;
  int32_t *pvacc;
  float sq, pmax;
} or_trace;

float or_sas_y(float y);
void or_sas_softmax_rows(const float* x, int R, int C, double* out);
float or_block_quant(const float* x, long n, int8_t* q);
void or_quantize_kv(const float* k, const float* v, int B, int Hkv, int N, int d, const int* bits,
                    int8_t* k8, int8_t* v8, float* sk, float* sv, uint8_t* kc, uint8_t* vc,
                    uint8_t* ks, int8_t* kz, uint8_t* vs, int8_t* vz);
void or_quantize_kv_blocks(const float* k, const float* v, int B, int Hkv, int N, int d, int bc,
                           int8_t* k8, int8_t* v8, float* sk, float* sv);
void or_attn_prefill_blocks(const float* q, const float* k, const float* v, int B, int Hq,
                            int Hkv, int N, int d, float sm_scale, int causal, or_opts opts,
                            int br, int bc, double* o, double* lse, or_trace* tr, int i0, int i1);
void or_attn_decode(const float* q, const uint8_t* kc, const uint8_t* vc, const uint8_t* ks,
                    const int8_t* kz, const uint8_t* vs, const int8_t* vz, const float* sk,
                    const float* sv, const int* seq_lens, int B, int Hq, int Hkv, int Nc, int d,
                    float sm_scale, int split, or_opts opts, double* o, double* lse,
                    or_trace* tr, const int8_t* tk, const int8_t* tv, const float* tsk,
                    const float* tsv);
void or_attn_exact(const float* q, const float* k, const float* v, int B, int Hq, int Hkv, int Nq,
                   int Nk, int d, double sm_scale, int causal, double* o, double* lse);
void or_tail_init(const float* k, const float* v, int B, int Hkv, int N, int d, const float* sk,
                  const float* sv, int8_t* tk, int8_t* tv, float* tsk, float* tsv);
void or_append_kv(const float* knew, const float* vnew, int B, int Hkv, int d,
                  const int* seq_lens, const int* bits, int Nc, uint8_t* kc, uint8_t* vc,
                  uint8_t* ks, int8_t* kz, uint8_t* vs, int8_t* vz, float* sk, float* sv,
                  int8_t* tk, int8_t* tv, const float* tsk, const float* tsv);
void or_head_priority(const float* k, int B, int Hkv, int N, int d, double* prio);
void or_int2_heads(const double* prio, int Hkv, int n_int2, uint8_t* bits);

#define D 128
static unsigned rng_state = 12345u;
static float frand(void) { /* xorshift32, values in [-2, 2) rounded to fp16-like grid */
  rng_state ^= rng_state << 13;
  rng_state ^= rng_state >> 17;
  rng_state ^= rng_state << 5;
  return (float)((int)(rng_state % 4096u) - 2048) / 1024.0f;
}
static float* fbuf(size_t n) {
  float* p = malloc(n * sizeof(float));
  for (size_t i = 0; i < n; ++i) p[i] = frand();
  return p;
}

int main(void) {
  const int B = 2, Hq = 4, Hkv = 2, N = 64 * 3 + 37, G = N / 64;
  const int bits[2] = {4, 2};
  const size_t nkv = (size_t)B * Hkv * N * D;
  float *q = fbuf((size_t)B * Hq * N * D), *k = fbuf(nkv), *v = fbuf(nkv);
  for (size_t i = 3; i < nkv; i += D) k[i] *= 10.0f; /* an outlier channel */
  const int nb = (N + 63) / 64;

  /* SAS, Algorithm 3 */
  float ys[5] = {0.0f, 0.5f, 5.999f, 6.0f, 1e30f};
  for (int i = 0; i < 5; ++i) (void)or_sas_y(ys[i]);
  double* sm = malloc(sizeof(double) * 3 * 70);
  or_sas_softmax_rows(q, 3, 70, sm);

  /* FlashQ steps 1 and 2 */
  int8_t *k8 = malloc(nkv), *v8 = malloc(nkv);
  float *sk = malloc(sizeof(float) * B * Hkv * nb), *sv = malloc(sizeof(float) * B * Hkv * nb);
  uint8_t *kc = malloc((size_t)B * Hkv * G * 64 * D), *vc = malloc((size_t)B * Hkv * G * 64 * D);
  uint8_t *ks = malloc((size_t)B * Hkv * G * D), *vs = malloc((size_t)B * Hkv * G * D);
  int8_t *kz = malloc((size_t)B * Hkv * G * D), *vz = malloc((size_t)B * Hkv * G * D);
  or_quantize_kv(k, v, B, Hkv, N, D, bits, k8, v8, sk, sv, kc, vc, ks, kz, vs, vz);
  (void)or_block_quant(q, 17, k8);

  /* Algorithm 1 at every block size, with a trace */
  double *o = malloc(sizeof(double) * B * Hq * N * D), *lse = malloc(sizeof(double) * B * Hq * N);
  int8_t tq8[128 * D], tqp[128 * 128];
  int32_t tsacc[128 * 128], tpv[128 * D];
  const int sizes[3] = {32, 64, 128};
  for (int a = 0; a < 3; ++a)
    for (int c = 0; c < 3; ++c) {
      or_trace tr = {1, 3, 1, 1, 0, tq8, tsacc, tqp, tpv, 0.0f, 0.0f};
      or_opts op = {1, 1};
      or_attn_prefill_blocks(q, k, v, B, Hq, Hkv, N, D, 0.088f, (a + c) % 2, op, sizes[a],
                             sizes[c], o, lse, &tr, -1, -1);
      int8_t *kb8 = malloc(nkv), *vb8 = malloc(nkv);
      const int nbc = (N + sizes[c] - 1) / sizes[c];
      float *skb = malloc(sizeof(float) * B * Hkv * nbc), *svb = malloc(sizeof(float) * B * Hkv * nbc);
      or_quantize_kv_blocks(k, v, B, Hkv, N, D, sizes[c], kb8, vb8, skb, svb);
      free(kb8); free(vb8); free(skb); free(svb);
    }
  for (int qu = 0; qu < 2; ++qu)
    for (int sa = 0; sa < 2; ++sa) {
      or_opts op = {qu, sa};
      or_attn_prefill_blocks(q, k, v, B, Hq, Hkv, N, D, 0.088f, 1, op, 64, 64, o, lse, NULL, 1, 3);
    }

  /* Algorithm 2 over the cache, split and unsplit, with the int8 buffer */
  const int Nc = G * 64;
  const int seq[2] = {N, 63};
  float* qd = fbuf((size_t)B * Hq * D);
  double *od = malloc(sizeof(double) * B * Hq * D), *ld = malloc(sizeof(double) * B * Hq);
  int8_t *tk = calloc((size_t)B * Hkv * 64 * D, 1), *tv = calloc((size_t)B * Hkv * 64 * D, 1);
  float tsk[4], tsv[4];
  or_tail_init(k, v, B, Hkv, N, D, sk, sv, tk, tv, tsk, tsv);
  float *skg = malloc(sizeof(float) * B * Hkv * G), *svg = malloc(sizeof(float) * B * Hkv * G);
  for (int u = 0; u < B * Hkv; ++u)
    for (int g = 0; g < G; ++g) {
      skg[u * G + g] = sk[u * nb + g];
      svg[u * G + g] = sv[u * nb + g];
    }
  for (int split = 1; split <= 4; split += 3) {
    or_trace tr = {0, 1, 0, 1, 0, tq8, tsacc, tqp, tpv, 0.0f, 0.0f};
    or_opts op = {1, 1};
    or_attn_decode(qd, kc, vc, ks, kz, vs, vz, skg, svg, seq, B, Hq, Hkv, Nc, D, 0.088f, split,
                   op, od, ld, &tr, tk, tv, tsk, tsv);
    or_attn_decode(qd, kc, vc, ks, kz, vs, vz, skg, svg, seq, B, Hq, Hkv, Nc, D, 0.088f, split,
                   op, od, ld, NULL, NULL, NULL, NULL, NULL);
  }
  /* appends up to a flush into a cache with room for one more group */
  {
    const int Nc2 = Nc + 64, G2 = G + 1;
    uint8_t *kc2 = calloc((size_t)B * Hkv * Nc2 * D, 1), *vc2 = calloc((size_t)B * Hkv * Nc2 * D, 1);
    uint8_t *ks2 = calloc((size_t)B * Hkv * G2 * D, 1), *vs2 = calloc((size_t)B * Hkv * G2 * D, 1);
    int8_t *kz2 = calloc((size_t)B * Hkv * G2 * D, 1), *vz2 = calloc((size_t)B * Hkv * G2 * D, 1);
    float *sk2 = calloc((size_t)B * Hkv * G2, 4), *sv2 = calloc((size_t)B * Hkv * G2, 4);
    int pos[2] = {N, N};
    for (int step = 0; step < 64 - (N % 64) + 1; ++step) {
      float *kn = fbuf((size_t)B * Hkv * D), *vn = fbuf((size_t)B * Hkv * D);
      or_append_kv(kn, vn, B, Hkv, D, pos, bits, Nc2, kc2, vc2, ks2, kz2, vs2, vz2, sk2, sv2, tk,
                   tv, tsk, tsv);
      pos[0]++;
      pos[1]++;
      free(kn);
      free(vn);
    }
    free(kc2); free(vc2); free(ks2); free(vs2); free(kz2); free(vz2); free(sk2); free(sv2);
  }

  /* exact attention (prefill and decode shapes), Sec. 3.2 priority */
  or_attn_exact(q, k, v, B, Hq, Hkv, N, N, D, 0.088, 1, o, lse);
  or_attn_exact(qd, k, v, B, Hq, Hkv, 1, N, D, 0.088, 0, od, ld);
  double prio[2];
  uint8_t hb[2];
  or_head_priority(k, B, Hkv, N, D, prio);
  or_int2_heads(prio, Hkv, 1, hb);

  printf("oracle sanitizer driver: ok (lse[0] = %.6f, priority %.3f %.3f)\n", lse[0], prio[0],
         prio[1]);
  free(q); free(k); free(v); free(sm); free(k8); free(v8); free(sk); free(sv); free(kc);
  free(vc); free(ks); free(vs); free(kz); free(vz); free(o); free(lse); free(qd); free(od);
  free(ld); free(tk); free(tv); free(skg); free(svg);
  return 0;
}
