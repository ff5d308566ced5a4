/*
 * turbo_attn.h — C ABI of the MI355X (gfx950) TurboAttention hot path.
 *
 * TurboAttention (Kang et al., MLSys 2025) replaces FP16 FlashAttention by
 *   - FlashQ: blockwise symmetric int8 quantization of Q, K and V tiles
 *     (Sec. 3.1, eq. step1bpq) followed, for K and V only, by channel-wise
 *     asymmetric int4 / int2 compression of the int8 values into a cache
 *     (Sec. 3.1, eq. step2bpq; Sec. 2.3 progressive quantization), with the
 *     bit width chosen per KV head (Sec. 3.2);
 *   - SAS: the exponential of the online softmax is replaced by a lookup
 *     table for the integer part and a cubic polynomial for the fractional
 *     part, and scores more than |n_r| = 6 below the running row maximum are
 *     dropped (Sec. 4; Appendix B, Algorithm 3);
 *   - integer QK^T and PV contractions inside a FlashAttention-style tiled
 *     loop (Appendix A, Algorithm 1 prefill, Algorithm 2 decode).
 *
 * This header declares the three calls of that path plus their helpers.
 *
 * General rules for every entry point
 *   - All tensor arguments are DEVICE pointers allocated and owned by the
 *     caller, unless stated "host".  The library never allocates, frees or
 *     synchronizes; every launch is queued on `stream` and outputs are valid
 *     once that stream has completed.
 *   - Return value: TURBO_OK (0) on success, a negative turbo_status
 *     otherwise.  All argument checks run on the host before any launch; on
 *     an error nothing is launched.  No C++ exception crosses this boundary.
 *   - fp16 means IEEE binary16 stored as 16-bit words.
 *   - Fixed constants: head dimension d = 128; query block B_r, key block
 *     B_c and the channel-group length of the int4/int2 step are all 64
 *     tokens (Sec. 5.2 fixes B_r = B_c = n_b = 64); cache pages hold 16
 *     tokens; the symmetric int8 divisor is 119 (Algorithms 1 and 2); the SAS
 *     threshold is n_r = -6 (Sec. 5.2).
 *   - Index types are int32 for shapes and table entries.
 */
#ifndef TURBO_ATTN_H
#define TURBO_ATTN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TURBO_ABI_VERSION 4

#define TURBO_HEAD_DIM 128       /* d */
#define TURBO_BLOCK 64           /* B_r = B_c = step-2 group length (tokens) */
#define TURBO_PAGE_TOKENS 16     /* tokens per cache page */
#define TURBO_PAGES_PER_GROUP 4  /* TURBO_BLOCK / TURBO_PAGE_TOKENS */
#define TURBO_MAX_KV_HEADS 64
#define TURBO_MAX_GQA 16         /* max query heads per KV head */

/* Layout of the tile trace written by the *_trace test hooks (bytes), for a
 * tile of B_r query rows and B_c keys (B_r, B_c <= 128; 64 x 64 for the
 * default prefill, one row of 64 keys for decode): */
#define TURBO_TRACE_Q8 0         /* int8  [B_r][128]  Q^{q1} rows of the block  */
#define TURBO_TRACE_S 16384      /* int32 [B_r][B_c]  QK^T accumulators         */
#define TURBO_TRACE_P 81920      /* int8  [B_r][B_c]  Q(P~) codes               */
#define TURBO_TRACE_PV 98304     /* int32 [B_r][128]  PV accumulators           */
#define TURBO_TRACE_SQ 163840    /* fp32              s_Q                       */
#define TURBO_TRACE_PMAX 163844  /* fp32              max P~ behind the P scale */
#define TURBO_TRACE_BYTES 163848

typedef enum turbo_status {
  TURBO_OK = 0,
  TURBO_ERR_INVALID_ARG = -1,         /* null pointer, bad shape, bad bits */
  TURBO_ERR_UNSUPPORTED = -2,         /* device is not gfx950 */
  TURBO_ERR_WORKSPACE_TOO_SMALL = -3, /* decode workspace smaller than needed */
  TURBO_ERR_HIP = -4                  /* a HIP runtime call or launch failed */
} turbo_status;

/*
 * Compressed paged KV cache (Sec. 3.1 eq. step2bpq; Sec. 2.3: the int4/int2
 * data with integer scale and zero point per group, plus the float scales of
 * the int8 step).  The cache is shared by all sequences of a batch: pages and
 * group slots are handed out through the block and group tables.
 *
 * pages        device, uint8 [num_pages][page_bytes].  A page holds 16
 *              consecutive tokens of one sequence for ALL KV heads.  KV head h
 *              occupies 512*bits_h bytes starting at byte offset
 *              sum_{h'<h} 512*bits_{h'}: first the K codes (256*bits_h bytes),
 *              then the V codes (256*bits_h bytes).
 *                K codes are token-major: token t (0..15) uses 16*bits_h
 *                bytes; int4: byte j holds channel 2j in bits 0-3 and channel
 *                2j+1 in bits 4-7; int2: byte j holds channels 4j..4j+3 in
 *                bits (0-1, 2-3, 4-5, 6-7).
 *                V codes are channel-major: channel c (0..127) uses 2*bits_h
 *                bytes for the page's 16 tokens; int4: byte j holds token 2j
 *                in bits 0-3 and token 2j+1 in bits 4-7; int2: byte j holds
 *                tokens 4j..4j+3 in bits (0-1, 2-3, 4-5, 6-7).
 *              Codes are the unsigned step-2 levels, 0 .. 2^bits-1.
 * group_meta   device, int8 [num_group_slots][num_kv_heads][4][128]: per
 *              64-token group and channel the integer step-2 parameters:
 *              [0] K scale s^int (stored as uint8, 1..255), [1] K zero point
 *              z^int (int8), [2] V scale (uint8), [3] V zero point (int8).
 *              The int8 value is recovered as code * s^int + z^int.
 * group_scale  device, fp32 [num_group_slots][num_kv_heads][2]: the step-1
 *              block scales s_K and s_V of the group (int8 value * s = real).
 * head_bits    HOST array inside the struct: 4 or 2 for each KV head.
 */
typedef struct turbo_kv_cache {
  uint8_t* pages;
  int8_t* group_meta;
  float* group_scale;
  int64_t num_pages;
  int64_t num_group_slots;
  int32_t num_kv_heads;
  int32_t head_dim;
  uint8_t head_bits[TURBO_MAX_KV_HEADS];
} turbo_kv_cache;

/*
 * int8 KV-cache buffer of Sec. 3.3: per (sequence b, KV head h) the newest
 * tokens that do not yet form a full 64-token group, kept as int8 under one
 * "universal" scale per (b, h) and tensor, so that appending a token never
 * re-quantizes the others.
 *
 * k      device int8 [batch][num_kv_heads][64][128], token-major: row r holds
 *        token 64*floor(len/64) + r of the sequence (r < len mod 64).
 * v      device int8 [batch][num_kv_heads][128][64], channel-major (element
 *        (token r, channel c) at [c][r]).
 * scale  device fp32 [batch][num_kv_heads][2]: universal scales s_K, s_V
 *        (int8 value * s = real value).
 * batch, num_kv_heads   the sizes the buffers are allocated for.
 */
typedef struct turbo_kv_tail {
  int8_t* k;
  int8_t* v;
  float* scale;
  int32_t batch;
  int32_t num_kv_heads;
} turbo_kv_tail;

/* ABI version of the loaded library (TURBO_ABI_VERSION). */
int turbo_abi_version(void);

/* Static description of a status code; never NULL. */
const char* turbo_strerror(int status);

/* Bytes of one cache page for the given host array of per-head bit widths
 * (sum over heads of 512*bits).  Returns 0 if any width is not 2 or 4 or
 * num_kv_heads is outside 1..TURBO_MAX_KV_HEADS. */
size_t turbo_page_bytes(const uint8_t* head_bits, int num_kv_heads);

/*
 * turbo_quantize_kv — FlashQ for K and V (Algorithm 1, the step-1 int8
 * quantization of K_j, V_j and the step-2 channel-wise int4/int2 compression
 * with its writes of K^q2, V^q2, s^int, z^int, s_K, s_V; eq. step1bpq and
 * step2bpq of Sec. 3.1).
 *
 * k, v        fp16 [B][Hkv][N][128].
 * k8          int8 [B][Hkv][Np][128], Np = 64*ceil(N/64), token-major; the
 *             int8 codes round(x * 119 / max|block|) of each 64-token block.
 *             Rows N..Np-1 are written as 0.
 * v8          int8 [B][Hkv][Np/64][128][64]: the same codes for V, stored
 *             channel-major inside each 64-token block (element (token t,
 *             channel c) at [t/64][c][t%64]); rows >= N are written as 0.
 * s_k, s_v    fp32 [B][Hkv][Np/64]: block scales max|block| / 119 (0 for an
 *             all-zero block).  A partial last block uses its valid rows only.
 * cache       may be NULL (no cache write).  Otherwise the full 64-token
 *             groups g = 0 .. floor(N/64)-1 of sequence b are compressed
 *             into pages block_table[b][4g .. 4g+3] and group slot
 *             group_table[b][g].  The N mod 64 trailing tokens stay in k8/v8
 *             only.  cache->num_kv_heads must equal Hkv.
 * block_table device int32 [B][4*max_groups_per_seq] (ignored if cache NULL).
 * group_table device int32 [B][max_groups_per_seq]   (ignored if cache NULL).
 *             Entries must lie in [0, num_pages) / [0, num_group_slots) and
 *             the pages and slots of different (b, g) must be distinct; the
 *             kernel skips the cache write of a group whose entries are out
 *             of range (never touching memory for it).
 * B, Hkv, N   B >= 0, 1 <= Hkv <= 64, N >= 0; B == 0 or N == 0 is a no-op.
 *             max_groups_per_seq >= floor(N/64) when cache != NULL.
 * d           must be 128.
 */
int turbo_quantize_kv(const void* k, const void* v, int B, int Hkv, int N, int d,
                      int8_t* k8, int8_t* v8, float* s_k, float* s_v,
                      const turbo_kv_cache* cache, const int32_t* block_table,
                      const int32_t* group_table, int max_groups_per_seq,
                      hipStream_t stream);

/*
 * turbo_quantize_kv_blocks — FlashQ step 1 of K and V (eq. step1bpq) with
 * key blocks of block_cols = B_c tokens, the block sizes Table 3 compares
 * (32, 64 or 128), for turbo_attn_prefill_blocks.  No cache write: the
 * step-2 groups of the cache stay 64 tokens (Sec. 3.3 fixes n_b = 64), so
 * the cache is written by turbo_quantize_kv only.
 *
 * k8, v8      the layouts of turbo_quantize_kv (64-token blocks, Np =
 *             64*ceil(N/64) rows; rows N..Np-1 written as 0), holding the
 *             codes of the B_c-token blocks.
 * s_k, s_v    fp32 [B][Hkv][ceil(N/B_c)]: max|block| / 119 of each B_c block.
 * block_cols  32, 64 or 128 (64: turbo_quantize_kv without a cache);
 *             INVALID_ARG otherwise.  Other arguments as turbo_quantize_kv.
 */
int turbo_quantize_kv_blocks(const void* k, const void* v, int B, int Hkv, int N, int d,
                             int block_cols, int8_t* k8, int8_t* v8, float* s_k, float* s_v,
                             hipStream_t stream);

/*
 * turbo_attn_prefill — Algorithm 1 (TurboAttention prefill): per 64-row query
 * block, int8 quantization of Q_i; for each key block j, int8 QK^T scaled by
 * s_Q * s_K * sm_scale, online row maximum, SAS in place of exp, running sum
 * of the unquantized SAS values, int8 quantization of the 64x64 SAS tile with
 * scale max/119, int8 PV scaled by s_P * s_V, and the rescale of the
 * accumulator by SAS(m_old - m_new) (exactly 1, e^0, for a row whose maximum
 * did not move); finally O / l and L = m + ln l.
 *
 * q           fp16 [B][Hq][N][128].
 * k8, v8, s_k, s_v  as written by turbo_quantize_kv for the same B, Hkv, N.
 * B, Hq, Hkv  Hq % Hkv == 0, Hq / Hkv <= 16; query head h reads KV head
 *             h / (Hq / Hkv).
 * sm_scale    the softmax temperature 1/sqrt(d) of eq. threesteps (any
 *             positive finite value is accepted).
 * causal      nonzero: key t is visible to query r only if t <= r.
 * o           fp16 [B][Hq][N][128] (output, round-to-nearest-even of O/l).
 * lse         fp32 [B][Hq][N] or NULL: L = m + ln(l).
 * B == 0 or N == 0 is a no-op.
 */
int turbo_attn_prefill(const void* q, const int8_t* k8, const int8_t* v8, const float* s_k,
                       const float* s_v, int B, int Hq, int Hkv, int N, int d, float sm_scale,
                       int causal, void* o, float* lse, hipStream_t stream);

/*
 * turbo_attn_prefill_blocks — turbo_attn_prefill with other block sizes
 * (B_r, B_c) (Table 3 evaluates seven pairs from {32, 64, 128}): Q is
 * quantized per block_rows rows of a head, each online step covers
 * block_cols keys, and the P scale covers the block_rows x block_cols tile.
 * k8, v8, s_k, s_v must come from turbo_quantize_kv_blocks with the same
 * block_cols (s_k, s_v [B][Hkv][ceil(N/block_cols)]).  (64, 64) is
 * turbo_attn_prefill.  With causal masking and B_r > B_c, a 32-row slice of
 * a block that sees no key of a tile leaves its rows untouched (Algorithm 1
 * processes no such pair).  INVALID_ARG for block sizes outside
 * {32, 64, 128}; other arguments and errors as turbo_attn_prefill.
 */
int turbo_attn_prefill_blocks(const void* q, const int8_t* k8, const int8_t* v8, const float* s_k,
                              const float* s_v, int B, int Hq, int Hkv, int N, int d,
                              float sm_scale, int causal, int block_rows, int block_cols, void* o,
                              float* lse, hipStream_t stream);

/*
 * turbo_attn_prefill_q8 — turbo_attn_prefill with Q already quantized
 * (FlashQ step 1 done by turbo_qkv_project): the prologue loads the int8
 * block and its scale instead of quantizing fp16 Q.  Given the codes and
 * scales the fp16 path would compute, the output is bit-identical to
 * turbo_attn_prefill's.
 *
 * q8          int8 [B][Hq][64*ceil(N/64)][128], rows >= N zero.
 * s_q         fp32 [B][Hq][ceil(N/64)]: the scale of each 64-row block.
 * Other arguments and errors as turbo_attn_prefill.
 */
int turbo_attn_prefill_q8(const int8_t* q8, const float* s_q, const int8_t* k8, const int8_t* v8,
                          const float* s_k, const float* s_v, int B, int Hq, int Hkv, int N,
                          int d, float sm_scale, int causal, void* o, float* lse,
                          hipStream_t stream);

/*
 * turbo_qkv_project — the QKV projection with FlashQ fused into it (Sec. 5.2
 * folds the quantization of Q, K and V into the projection that produces
 * them; Sec. 3.1 steps 1 and 2):
 *   Y = X W^T in fp32 (fp16 MFMA), each output rounded to fp16, then
 *   Q: int8 codes and scale per (sequence, query head, 64-row block), the rule
 *      of the prefill's Q quantization (so turbo_attn_prefill_q8 can use it);
 *   K, V: exactly what turbo_quantize_kv writes for the same fp16 K and V
 *      (k8, v8, s_k, s_v and, when cache != NULL, the int4/int2 groups).
 * Q, K and V are never stored in fp16.
 *
 * x           fp16 [B][N][D] hidden states, row-major; D % 64 == 0.
 * w           fp16 [(Hq + 2 Hkv) * 128][D]: output feature f < 128 Hq is
 *             channel f % 128 of query head f / 128; then the key heads, then
 *             the value heads (the rows of a fused QKV linear layer).
 * q8, s_q     int8 [B][Hq][64*ceil(N/64)][128] (rows >= N zero), fp32
 *             [B][Hq][ceil(N/64)].
 * k8, v8, s_k, s_v, cache, block_table, group_table, max_groups_per_seq
 *             as turbo_quantize_kv.
 * B, N        B == 0 or N == 0 is a no-op.  Errors: INVALID_ARG for null
 *             outputs, D not a positive multiple of 64, d != 128,
 *             Hq % Hkv != 0, Hkv outside 1..64, or a cache that
 *             turbo_quantize_kv would reject.
 */
int turbo_qkv_project(const void* x, const void* w, int B, int N, int D, int Hq, int Hkv, int d,
                      int8_t* q8, float* s_q, int8_t* k8, int8_t* v8, float* s_k, float* s_v,
                      const turbo_kv_cache* cache, const int32_t* block_table,
                      const int32_t* group_table, int max_groups_per_seq, hipStream_t stream);

/*
 * Test hook (not part of the method): turbo_qkv_project that also writes the
 * fp16 projection it quantizes, y fp16 [B][N][F] (F = (Hq + 2 Hkv) * 128,
 * feature order of w's rows), so that its codes, scales and cache bytes can
 * be checked bit for bit as FlashQ of that projection.  The same kernel
 * source runs (an instance with the extra stores).  INVALID_ARG also when
 * y is NULL.
 */
int turbo_qkv_project_trace(const void* x, const void* w, int B, int N, int D, int Hq, int Hkv,
                            int d, int8_t* q8, float* s_q, int8_t* k8, int8_t* v8, float* s_k,
                            float* s_v, const turbo_kv_cache* cache, const int32_t* block_table,
                            const int32_t* group_table, int max_groups_per_seq, void* y,
                            hipStream_t stream);

/*
 * Test hook (not part of the method): turbo_attn_prefill with the integers of
 * one (sequence tb, query head th, query block ti, key block tj) tile written
 * to `trace` (device, TURBO_TRACE_BYTES, layout above).  The same kernel runs;
 * the selected tile additionally stores
 *   Q8[r][c]   int8 Q code of query 64*ti + r, channel c (rows past N are 0);
 *   S[r][t]    int32 sum_c Q8[r][c] * K8[64*tj + t][c] for every (r, t) of
 *              the tile, masked entries included (they are excluded from the
 *              softmax, not from the product);
 *   P[r][t]    Q(P~) code (0 where masked);
 *   PV[r][c]   int32 sum_t P[r][t] * V8[64*tj + t][c];
 *   SQ, PMAX   s_Q of the block and the tile maximum of P~.
 * Nothing is written when tj is not processed for ti (tj > ti when causal).
 * INVALID_ARG also when trace is NULL or an index is out of range.
 */
int turbo_attn_prefill_trace(const void* q, const int8_t* k8, const int8_t* v8,
                             const float* s_k, const float* s_v, int B, int Hq, int Hkv, int N,
                             int d, float sm_scale, int causal, void* o, float* lse, int tb,
                             int th, int ti, int tj, void* trace, hipStream_t stream);

/*
 * Test hook (not part of the method): turbo_attn_prefill_blocks with the
 * integers of one tile -- query block ti of block_rows rows, key block tj of
 * block_cols keys -- written to `trace` as for turbo_attn_prefill_trace, with
 * B_r = block_rows rows and row strides B_c = block_cols for S and P.  Rows of
 * the tile that see no key of it (causal, B_r > B_c) store their products and
 * Q(P~) = 0, PV = 0.  Errors as turbo_attn_prefill_trace.
 */
int turbo_attn_prefill_blocks_trace(const void* q, const int8_t* k8, const int8_t* v8,
                                    const float* s_k, const float* s_v, int B, int Hq, int Hkv,
                                    int N, int d, float sm_scale, int causal, int block_rows,
                                    int block_cols, void* o, float* lse, int tb, int th, int ti,
                                    int tj, void* trace, hipStream_t stream);

/*
 * turbo_attn_decode — Algorithm 2 (TurboAttention decode): the new query of
 * each sequence is quantized to int8 per (b, query head); every cached
 * 64-token group is expanded from int4/int2 to int8 in the kernel with
 * code * s^int + z^int, and the same SAS online softmax as prefill runs with
 * one query row (P scale per row and group).
 *
 * The rescale factor SAS(m_old - m_new) of the online step is exactly 1
 * (e^0) when a row's maximum does not move (reading: SAS stands in for e^x,
 * and the exponent is exactly 0 there).
 *
 * Split-KV extension (not in the paper): the groups of a sequence are cut
 * into chunks of kv_split_groups groups (0: turbo_decode_default_split of
 * the sequence's own group count, so that a sequence's result does not
 * depend on the batch).  Each chunk runs the online loop from m = -inf; with
 * more than one chunk the partial states are merged with m* = max m_s,
 * w_s = SAS(m_s - m*) (1 for m_s = m*), O = sum w_s O_s / sum w_s l_s,
 * L = m* + ln(sum w_s l_s), chunks in ascending order (a second launch on
 * the same stream).  With one chunk the result is the unsplit Algorithm 2.
 * Different chunkings give different results (the n_r threshold drops
 * scores against the running maximum of each chunk).
 *
 * int8 buffer (Sec. 3.3): with tail != NULL the seq_len mod 64 newest tokens
 * (rows of the buffer) are attended as well.  Reading: the buffer is one more
 * chunk after the group chunks, running the same online step from m = -inf
 * with the universal scales (QK^T and PV on its int8 codes), merged with the
 * others as above.
 *
 * q               fp16 [B][Hq][128].
 * cache           as filled by turbo_quantize_kv / turbo_append_kv
 *                 (num_kv_heads = Hkv).
 * tail            NULL (groups only) or the Sec. 3.3 buffer (batch >= B,
 *                 num_kv_heads == Hkv).
 * seq_lens        device int32 [B]: tokens of each sequence.  The
 *                 floor(seq_len/64) full groups (at most max_groups_per_seq)
 *                 come from the cache; with a tail, the next seq_len mod 64
 *                 tokens (at most 63) from the buffer.  A sequence with
 *                 nothing to attend yields o = 0 and lse = -inf.
 * block_table,
 * group_table     as for turbo_quantize_kv.  A group whose page or slot entry
 *                 is out of range is skipped (its memory is never read).
 * B, Hq           Hq % Hkv == 0, Hq / Hkv <= 16.
 * kv_split_groups groups per chunk, >= 1, for every sequence; 0 selects
 *                 turbo_decode_default_split(ng) for each sequence of ng
 *                 cached groups.  turbo_decode_auto_split offers a chunk
 *                 length fitted to the batch's occupancy instead (pass it
 *                 explicitly; results then depend on the batch shape).
 * workspace       device scratch of at least turbo_decode_workspace_bytes()
 *                 bytes (with_tail = tail != NULL; may be NULL when that is
 *                 0): the chunk states, fully written before they are
 *                 read (no initialization needed).  Calls that share a
 *                 workspace must not overlap.
 * o               fp16 [B][Hq][128];  lse fp32 [B][Hq] or NULL.
 */
int turbo_attn_decode(const void* q, const turbo_kv_cache* cache, const turbo_kv_tail* tail,
                      const int32_t* seq_lens, const int32_t* block_table,
                      const int32_t* group_table, int max_groups_per_seq, int B, int Hq,
                      float sm_scale, int kv_split_groups, void* workspace,
                      size_t workspace_bytes, void* o, float* lse, hipStream_t stream);

/*
 * turbo_attn_decode_noalloc — turbo_attn_decode for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.  Same arguments, kernels and results as
 * turbo_attn_decode, without the workspace: the split-KV chunk states go to
 * a fixed device array of TURBO_DECODE_SCRATCH_BYTES inside the library
 * (one per GPU, held until the process ends; its address is looked up once
 * per device on the first call there).  The call itself allocates nothing.
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (other streams, other host threads) race and must be ordered by the
 * caller.  Nothing in the array needs clearing: each call writes every chunk
 * state before reading it.
 * Errors as turbo_attn_decode, plus TURBO_ERR_WORKSPACE_TOO_SMALL (before
 * any launch) when turbo_decode_workspace_bytes(B, Hq, Hkv,
 * max_groups_per_seq, kv_split_groups, tail != NULL) exceeds
 * TURBO_DECODE_SCRATCH_BYTES, e.g. B * Hq * chunks > 63550.
 */
#define TURBO_DECODE_SCRATCH_BYTES (32u << 20)
int turbo_attn_decode_noalloc(const void* q, const turbo_kv_cache* cache,
                              const turbo_kv_tail* tail, const int32_t* seq_lens,
                              const int32_t* block_table, const int32_t* group_table,
                              int max_groups_per_seq, int B, int Hq, float sm_scale,
                              int kv_split_groups, void* o, float* lse, hipStream_t stream);

/*
 * Test hook (not part of the method): turbo_attn_decode with the integers of
 * group tg of (sequence tb, query head th) written to `trace` (device,
 * TURBO_TRACE_BYTES, layout above; row 0 of each array is used):
 *   Q8[0][c]   int8 code of the query;
 *   S[0][t]    int32 sum_c Q8[c] * K^{q1}[t][c] with K^{q1} = code*s^int + z^int;
 *   P[0][t]    Q(P~) code of token t;
 *   PV[0][c]   int32 sum_t P[t] * V^{q1}[t][c];
 *   SQ, PMAX   s_Q and the group's maximum of P~.
 * With a tail, group tg = floor(seq_len/64) selects the buffer (K^{q1}, V^{q1}
 * its int8 codes).  Nothing is written when group tg is not attended (beyond
 * the sequence, or a table entry out of range).  INVALID_ARG also when trace
 * is NULL or an index is out of range.
 */
int turbo_attn_decode_trace(const void* q, const turbo_kv_cache* cache,
                            const turbo_kv_tail* tail, const int32_t* seq_lens,
                            const int32_t* block_table, const int32_t* group_table,
                            int max_groups_per_seq, int B, int Hq, float sm_scale,
                            int kv_split_groups, void* workspace, size_t workspace_bytes, void* o,
                            float* lse, int tb, int th, int tg, void* trace, hipStream_t stream);

/*
 * turbo_head_priority — head-wise mixed precision (Sec. 3.2, the priority
 * equation): for each KV head h of the prefill keys k (fp16 [B][Hkv][N][128],
 * all B sequences and N tokens of one layer),
 *   gap_c = max - min of channel c,  gap = max - min over all channels,
 *   std   = population standard deviation of the 128 gap_c,
 *   priority[h] = gap * std   (device fp32 [Hkv], written on `stream`).
 * workspace   device scratch of at least turbo_head_priority_workspace_bytes
 *             (per-slab channel maxima and minima; no initialization needed).
 * INVALID_ARG for B == 0 or N == 0 (no statistics), null pointers, d != 128;
 * WORKSPACE_TOO_SMALL for a missing or short workspace.
 */
int turbo_head_priority(const void* k, int B, int Hkv, int N, int d, void* workspace,
                        size_t workspace_bytes, float* priority, hipStream_t stream);

/* Workspace bytes of turbo_head_priority: fp32 [Hkv][B * ceil(N / 256)][256]
 * (0 for arguments < 1). */
size_t turbo_head_priority_workspace_bytes(int B, int Hkv, int N);

/*
 * turbo_int2_heads — the quantization strategy of Sec. 3.2 on the host:
 * head_bits[h] = 2 for the n_int2 heads of lowest priority (equal priorities
 * rank by head index), 4 for the others.  priority and head_bits are host
 * arrays of Hkv entries (the result feeds turbo_kv_cache.head_bits and
 * turbo_page_bytes).  INVALID_ARG for a NaN priority or n_int2 outside 0..Hkv.
 */
int turbo_int2_heads(const float* priority, int Hkv, int n_int2, uint8_t* head_bits);

/*
 * turbo_tail_init — start of the int8 buffer after a prefill (Sec. 3.3).
 * Reading: the universal scale of (b, h) is the largest step-1 block scale of
 * the prefill (max over j of s_k[b][h][j], likewise for V), so every prefill
 * value is representable; the N mod 64 trailing tokens, which form no step-2
 * group, become the buffer's first rows, coded as
 *   code = clamp(round_half_even(x * inv), -119, 119), inv = 1/s in binary32
 * (0 when s = 0).  Rows beyond N mod 64 are zeroed.
 *
 * k, v      fp16 [B][Hkv][N][128] (the prefill keys and values).
 * s_k, s_v  fp32 [B][Hkv][ceil(N/64)] as written by turbo_quantize_kv.
 * tail      buffers with batch >= B, num_kv_heads == Hkv.
 * B == 0 is a no-op; N == 0 is INVALID_ARG (no scale to start from).
 */
int turbo_tail_init(const void* k, const void* v, int B, int Hkv, int N, int d, const float* s_k,
                    const float* s_v, const turbo_kv_tail* tail, hipStream_t stream);

/*
 * turbo_append_kv — one decoding step's new key and value per sequence
 * (Sec. 3.3).  The token of sequence b at position p = seq_lens[b] (the
 * length BEFORE this step; p < 0 skips the sequence) goes to buffer row
 * p mod 64 with the universal scales and clamping (as in turbo_tail_init).
 * When that row is the 64th, the buffer is compressed like any other group:
 * step 2 (eq. step2bpq) into group g = p / 64 of the cache, pages
 * block_table[b][4g..4g+3], slot group_table[b][g], with the universal
 * scales as the group's s_K, s_V.  A flush whose group is >= max_groups_per_seq
 * or whose table entries are out of range is skipped (never touching memory).
 * The caller advances seq_lens afterwards.
 *
 * k_new, v_new  fp16 [B][Hkv][128].
 * cache, tail   cache->num_kv_heads == tail->num_kv_heads == Hkv, batch >= B.
 */
int turbo_append_kv(const void* k_new, const void* v_new, int B, int Hkv, int d,
                    const int32_t* seq_lens, const turbo_kv_cache* cache,
                    const turbo_kv_tail* tail, const int32_t* block_table,
                    const int32_t* group_table, int max_groups_per_seq, hipStream_t stream);

/*
 * turbo_sas_softmax — Algorithm 3 (Appendix B; SAS of Sec. 4) as a
 * stand-alone row softmax: for every row r of x (fp32 [rows][cols], row-major,
 * device), with m = max_c x[r][c]:
 *   e_c = SAS(x[r][c] - m): 0 when x - m < -6, else LUT[floor y] * POLY(y -
 *         floor y) with y = m - x in binary32, LUT[k] = e^-k in binary32 and
 *         POLY the cubic of Sec. 4 (Horner, fused multiply-adds);
 *   y[r][c] = e_c / sum_c e_c   (fp32, device; may alias x).
 * The e_c are the same binary32 values the attention kernels use; the row sum
 * is accumulated in fp32.  -inf entries contribute 0; a row without a finite
 * value gives NaN (0/0).  INVALID_ARG for null pointers, rows < 0,
 * rows > 2^31 - 1 or cols < 1.  rows == 0 is a no-op.
 */
int turbo_sas_softmax(const float* x, float* y, int64_t rows, int cols, hipStream_t stream);

/* The chunk length (in 64-token groups) that kv_split_groups = 0 gives a
 * sequence with ng cached groups: ng itself (one chunk) up to 32 groups,
 * 32 up to 128 groups (2 to 4 chunks), ceil(ng / 4) beyond (4 chunks).  It
 * depends on the sequence only.  Returns 1 for ng < 1. */
int turbo_decode_default_split(int ng);

/* A chunk length fitted to the occupancy of a decode batch of B sequences,
 * Hq query and Hkv KV heads and max_groups_per_seq (to be passed explicitly
 * as kv_split_groups).  The decode kernel keeps three waves per SIMD resident
 * when Hq / Hkv <= 8 and two otherwise (3072 or 2048 on 256 CUs); the
 * fewest chunks n whose B * Hkv * n waves fill at least two thirds of those
 * slots are chosen, with chunk length ceil(max_groups_per_seq / n) (the
 * whole sequence when B * Hkv already fills them), but never fewer than two
 * groups per chunk.  Since the chunked result merges SAS-weighted
 * partial states, the output then depends on the batch shape.
 * Returns 1 for arguments < 1. */
int turbo_decode_auto_split(int B, int Hq, int Hkv, int max_groups_per_seq);

/* Workspace bytes turbo_attn_decode needs for these arguments (0 when every
 * sequence fits one chunk and there is no tail): fp32 chunk states
 * [B][Hq][n][132] with n the most chunks a sequence of max_groups_per_seq
 * groups can have, plus one with_tail.  kv_split_groups as for
 * turbo_attn_decode. */
size_t turbo_decode_workspace_bytes(int B, int Hq, int Hkv, int max_groups_per_seq,
                                    int kv_split_groups, int with_tail);

/*
 * Measurement probes (not part of the method): the ceilings the attention
 * kernels are measured against, on the GPU at hand.
 *
 * turbo_probe_mfma_i8 — chains of v_mfma_i32_16x16x64_i8 on register
 * operands, `iters` rounds of 8 per wave, 2048 waves (two per SIMD of 256
 * CUs); no memory traffic.  *ops (host) receives the int8 ops the launch
 * performs (2 * 16 * 16 * 64 per MFMA); sink (device, int32 [512]) receives
 * one folded word per work-group.  The int8 MFMA rate is *ops / elapsed.
 *
 * turbo_probe_read — a streaming read of `bytes` (a multiple of 16 up to
 * 2^40, 16-byte aligned device buffer): one work-group of 256 threads per
 * 32 KiB chunk, eight nontemporal 16-byte loads in flight per thread; sink
 * (device, uint32 [1]) is written only if the folded data hit a fixed
 * pattern.  The read rate is bytes / elapsed.
 *
 * turbo_probe_valu — chains of fp32 FMAs (v_fma_f32, one value per lane),
 * `iters` rounds of 8 per wave, 4096 waves (four per SIMD of 256 CUs); no
 * memory traffic.  *insts (host) receives the wave-level vector ALU
 * instructions the launch issues; sink (device, float [1024]) is written
 * only if the folded chains hit a fixed value.  The vector ALU issue rate is
 * *insts / elapsed (one wave64 instruction occupies a SIMD for 4 clocks).
 *
 * All queue one launch on `stream`.  INVALID_ARG for iters < 1, null
 * pointers, or a misaligned / zero-sized buffer.
 */
int turbo_probe_mfma_i8(int iters, int* sink, int64_t* ops, hipStream_t stream);
int turbo_probe_read(const void* src, size_t bytes, unsigned* sink, hipStream_t stream);
int turbo_probe_valu(int iters, float* sink, int64_t* insts, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* TURBO_ATTN_H */
