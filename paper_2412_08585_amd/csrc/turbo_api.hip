// C ABI of the gfx950 TurboAttention hot path: argument checks on the host,
// then the kernel launches on the caller's stream.  No allocation, no
// synchronization, no exception crosses the boundary.
#include <algorithm>
#include <atomic>
#include <cstring>

#include "turbo_common.h"

// The library is one translation unit: the kernel sources (each with its
// argument struct and launcher) are included here.
#include "quantize_kv.hip"
#include "attn_prefill.hip"
#include "attn_decode.hip"
#include "head_priority.hip"
#include "kv_tail.hip"
#include "sas_softmax.hip"
#include "qkv_project.h"
#include "probes.hip"

namespace {

constexpr int kMaxDevices = 64;
// 0 unknown, 1 gfx950, -1 other; written once per device (benign race: every
// writer stores the same value).
std::atomic<int> g_arch_ok[kMaxDevices];

int check_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return TURBO_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return TURBO_ERR_UNSUPPORTED;
  int st = g_arch_ok[dev].load(std::memory_order_relaxed);
  if (st == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return TURBO_ERR_HIP;
    st = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : -1;
    g_arch_ok[dev].store(st, std::memory_order_relaxed);
  }
  return st == 1 ? TURBO_OK : TURBO_ERR_UNSUPPORTED;
}

// Scratch of turbo_attn_decode_noalloc: the split-KV chunk states live in a
// file-scope device array instead of a caller workspace.  Each GPU the
// library runs on holds its own copy until the process ends.  In host code
// `scratch` is only a stand-in for the symbol; its device address comes from
// hipGetSymbolAddress, once per device, and only that address is passed on.
constexpr size_t kDecodeScratchBytes = size_t(32) << 20;  // TURBO_DECODE_SCRATCH_BYTES
static_assert(kDecodeScratchBytes == TURBO_DECODE_SCRATCH_BYTES, "header and library agree");
static __device__ __align__(256) unsigned char scratch[kDecodeScratchBytes];
std::atomic<void*> g_scratch[kMaxDevices];

// Device address of this device's scratch (nullptr on failure).  Written once
// per device; concurrent first calls store the same address.
void* decode_scratch() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    g_scratch[dev].store(p, std::memory_order_release);
  }
  return p;
}

int check_cache(const turbo_kv_cache* c, int Hkv, unsigned long long* int2_mask,
                int* page_bytes) {
  if (!c || !c->pages || !c->group_meta || !c->group_scale) return TURBO_ERR_INVALID_ARG;
  if (c->num_kv_heads != Hkv || c->head_dim != TURBO_HEAD_DIM) return TURBO_ERR_INVALID_ARG;
  if (c->num_pages < 1 || c->num_group_slots < 1) return TURBO_ERR_INVALID_ARG;
  unsigned long long mask = 0;
  for (int h = 0; h < Hkv; ++h) {
    if (c->head_bits[h] == 2)
      mask |= 1ull << h;
    else if (c->head_bits[h] != 4)
      return TURBO_ERR_INVALID_ARG;
  }
  *int2_mask = mask;
  *page_bytes = (int)turbo_page_bytes(c->head_bits, Hkv);
  return TURBO_OK;
}

}  // namespace

extern "C" {

int turbo_abi_version(void) { return TURBO_ABI_VERSION; }

const char* turbo_strerror(int status) {
  switch (status) {
    case TURBO_OK: return "success";
    case TURBO_ERR_INVALID_ARG: return "invalid argument";
    case TURBO_ERR_UNSUPPORTED: return "unsupported device (gfx950 required)";
    case TURBO_ERR_WORKSPACE_TOO_SMALL: return "decode workspace too small";
    case TURBO_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

size_t turbo_page_bytes(const uint8_t* head_bits, int num_kv_heads) {
  if (!head_bits || num_kv_heads < 1 || num_kv_heads > TURBO_MAX_KV_HEADS) return 0;
  size_t total = 0;
  for (int h = 0; h < num_kv_heads; ++h) {
    if (head_bits[h] != 2 && head_bits[h] != 4) return 0;
    total += 512u * head_bits[h];
  }
  return total;
}

int turbo_quantize_kv(const void* k, const void* v, int B, int Hkv, int N, int d, int8_t* k8,
                      int8_t* v8, float* s_k, float* s_v, const turbo_kv_cache* cache,
                      const int32_t* block_table, const int32_t* group_table,
                      int max_groups_per_seq, hipStream_t stream) {
  if (B < 0 || N < 0 || Hkv < 1 || Hkv > TURBO_MAX_KV_HEADS || d != TURBO_HEAD_DIM)
    return TURBO_ERR_INVALID_ARG;
  if (B == 0 || N == 0) return TURBO_OK;
  if (!k || !v || !k8 || !v8 || !s_k || !s_v) return TURBO_ERR_INVALID_ARG;
  turbo::QuantArgs a{};
  if (cache) {
    if (!block_table || !group_table || max_groups_per_seq < N / TURBO_BLOCK)
      return TURBO_ERR_INVALID_ARG;
    int st = check_cache(cache, Hkv, &a.int2_mask, &a.page_bytes);
    if (st != TURBO_OK) return st;
    a.pages = cache->pages;
    a.gmeta = cache->group_meta;
    a.gscale = cache->group_scale;
    a.num_pages = cache->num_pages;
    a.num_slots = cache->num_group_slots;
    a.block_table = block_table;
    a.group_table = group_table;
    a.max_groups = max_groups_per_seq;
  }
  int st = check_device();
  if (st != TURBO_OK) return st;
  a.k = static_cast<const uint4*>(k);
  a.v = static_cast<const uint4*>(v);
  a.Hkv = Hkv;
  a.N = N;
  a.nb = turbo::ceil_div(N, TURBO_BLOCK);
  a.bc = TURBO_BLOCK;
  a.nbc = a.nb;
  a.k8 = k8;
  a.v8 = v8;
  a.sk = s_k;
  a.sv = s_v;
  return turbo::launch_quantize_kv(a, B, stream) == hipSuccess ? TURBO_OK : TURBO_ERR_HIP;
}

int turbo_quantize_kv_blocks(const void* k, const void* v, int B, int Hkv, int N, int d,
                             int block_cols, int8_t* k8, int8_t* v8, float* s_k, float* s_v,
                             hipStream_t stream) {
  if (block_cols == TURBO_BLOCK)
    return turbo_quantize_kv(k, v, B, Hkv, N, d, k8, v8, s_k, s_v, nullptr, nullptr, nullptr, 0,
                             stream);
  if (B < 0 || N < 0 || Hkv < 1 || Hkv > TURBO_MAX_KV_HEADS || d != TURBO_HEAD_DIM ||
      (block_cols != 32 && block_cols != 128))
    return TURBO_ERR_INVALID_ARG;
  if (B == 0 || N == 0) return TURBO_OK;
  if (!k || !v || !k8 || !v8 || !s_k || !s_v) return TURBO_ERR_INVALID_ARG;
  int st = check_device();
  if (st != TURBO_OK) return st;
  turbo::QuantArgs a{};
  a.k = static_cast<const uint4*>(k);
  a.v = static_cast<const uint4*>(v);
  a.Hkv = Hkv;
  a.N = N;
  a.nb = turbo::ceil_div(N, TURBO_BLOCK);
  a.bc = block_cols;
  a.nbc = turbo::ceil_div(N, block_cols);
  a.k8 = k8;
  a.v8 = v8;
  a.sk = s_k;
  a.sv = s_v;
  return turbo::launch_quantize_kv(a, B, stream) == hipSuccess ? TURBO_OK : TURBO_ERR_HIP;
}

static int attn_prefill_impl(const void* q, const int8_t* q8, const float* s_q,
                             const int8_t* k8, const int8_t* v8, const float* s_k,
                             const float* s_v, int B, int Hq, int Hkv, int N, int d,
                             float sm_scale, int causal, int block_rows, int block_cols,
                             void* o, float* lse, unsigned char* trace, int tr_L, int tr_j,
                             hipStream_t stream) {
  if (B < 0 || N < 0 || Hkv < 1 || Hq < 1 || Hq % Hkv != 0 || Hq / Hkv > TURBO_MAX_GQA ||
      d != TURBO_HEAD_DIM || !(sm_scale > 0.0f) || sm_scale > 3.0e38f)
    return TURBO_ERR_INVALID_ARG;
  if (B == 0 || N == 0) return TURBO_OK;
  if (!(q || (q8 && s_q)) || !k8 || !v8 || !s_k || !s_v || !o) return TURBO_ERR_INVALID_ARG;
  if (block_rows != 32 && block_rows != 64 && block_rows != 128) return TURBO_ERR_INVALID_ARG;
  if (block_cols != 32 && block_cols != 64 && block_cols != 128) return TURBO_ERR_INVALID_ARG;
  if (q8 && (block_rows != 64 || block_cols != 64)) return TURBO_ERR_INVALID_ARG;
  const long tiles = (long)B * Hq * (turbo::ceil_div(N, block_rows));
  if (tiles > 0x7fffffffL) return TURBO_ERR_INVALID_ARG;
  int st = check_device();
  if (st != TURBO_OK) return st;
  turbo::PrefillArgs a{};
  a.q = static_cast<const uint4*>(q);
  a.q8 = q ? nullptr : q8;
  a.sq = q ? nullptr : s_q;
  a.k8 = k8;
  a.v8 = v8;
  a.sk = s_k;
  a.sv = s_v;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.N = N;
  a.nb = turbo::ceil_div(N, TURBO_BLOCK);
  a.waves = block_rows / 32;
  a.nbq = turbo::ceil_div(N, block_rows);
  a.bc = block_cols;
  a.nbc = turbo::ceil_div(N, block_cols);
  a.sm_scale = sm_scale;
  a.causal = causal ? 1 : 0;
  a.o = static_cast<uint2*>(o);
  a.lse = lse;
  a.trace = trace;
  a.tr_L = tr_L;
  a.tr_j = tr_j;
  return turbo::launch_attn_prefill(a, stream) == hipSuccess ? TURBO_OK : TURBO_ERR_HIP;
}

int turbo_attn_prefill(const void* q, const int8_t* k8, const int8_t* v8, const float* s_k,
                       const float* s_v, int B, int Hq, int Hkv, int N, int d, float sm_scale,
                       int causal, void* o, float* lse, hipStream_t stream) {
  return attn_prefill_impl(q, nullptr, nullptr, k8, v8, s_k, s_v, B, Hq, Hkv, N, d, sm_scale,
                           causal, 64, 64, o, lse, nullptr, -1, -1, stream);
}

int turbo_attn_prefill_blocks(const void* q, const int8_t* k8, const int8_t* v8, const float* s_k,
                              const float* s_v, int B, int Hq, int Hkv, int N, int d,
                              float sm_scale, int causal, int block_rows, int block_cols,
                              void* o, float* lse, hipStream_t stream) {
  return attn_prefill_impl(q, nullptr, nullptr, k8, v8, s_k, s_v, B, Hq, Hkv, N, d, sm_scale,
                           causal, block_rows, block_cols, o, lse, nullptr, -1, -1, stream);
}

int turbo_attn_prefill_q8(const int8_t* q8, const float* s_q, const int8_t* k8, const int8_t* v8,
                          const float* s_k, const float* s_v, int B, int Hq, int Hkv, int N,
                          int d, float sm_scale, int causal, void* o, float* lse,
                          hipStream_t stream) {
  if (B > 0 && N > 0 && (!q8 || !s_q)) return TURBO_ERR_INVALID_ARG;
  return attn_prefill_impl(nullptr, q8, s_q, k8, v8, s_k, s_v, B, Hq, Hkv, N, d, sm_scale,
                           causal, 64, 64, o, lse, nullptr, -1, -1, stream);
}

static int qkv_project_impl(const void* x, const void* w, int B, int N, int D, int Hq, int Hkv,
                            int d, int8_t* q8, float* s_q, int8_t* k8, int8_t* v8, float* s_k,
                            float* s_v, const turbo_kv_cache* cache, const int32_t* block_table,
                            const int32_t* group_table, int max_groups_per_seq, void* y,
                            hipStream_t stream) {
  if (B < 0 || N < 0 || D < 64 || D % 64 != 0 || Hkv < 1 || Hkv > TURBO_MAX_KV_HEADS || Hq < 1 ||
      Hq % Hkv != 0 || d != TURBO_HEAD_DIM)
    return TURBO_ERR_INVALID_ARG;
  if (B == 0 || N == 0) return TURBO_OK;
  if (!x || !w || !q8 || !s_q || !k8 || !v8 || !s_k || !s_v) return TURBO_ERR_INVALID_ARG;
  const long ntile = turbo::ceil_div(N, turbo::kQkvTileTokens);
  const long npairs = turbo::ceil_div(Hq + 2 * Hkv, 2);
  // the kernel addresses one sequence of X and all of W (rounded up to whole
  // tiles) with 32-bit byte offsets
  if ((long)B * ntile * npairs > 0x7fffffffL || (long)B * N > 0x7fffffffL ||
      ntile * turbo::kQkvTileTokens * 2L * D > 0x7fffffffL || npairs * 256L * 2L * D > 0x7fffffffL)
    return TURBO_ERR_INVALID_ARG;
  turbo::QkvArgs a{};
  if (cache) {
    if (!block_table || !group_table || max_groups_per_seq < N / TURBO_BLOCK)
      return TURBO_ERR_INVALID_ARG;
    int st = check_cache(cache, Hkv, &a.int2_mask, &a.page_bytes);
    if (st != TURBO_OK) return st;
    a.pages = cache->pages;
    a.gmeta = cache->group_meta;
    a.gscale = cache->group_scale;
    a.num_pages = cache->num_pages;
    a.num_slots = cache->num_group_slots;
    a.block_table = block_table;
    a.group_table = group_table;
    a.max_groups = max_groups_per_seq;
  }
  int st = check_device();
  if (st != TURBO_OK) return st;
  a.x = x;
  a.w = w;
  a.B = B;
  a.N = N;
  a.D = D;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.nb = turbo::ceil_div(N, TURBO_BLOCK);
  a.ntile = (int)ntile;
  a.q8 = q8;
  a.sq = s_q;
  a.k8 = k8;
  a.v8 = v8;
  a.sk = s_k;
  a.sv = s_v;
  a.y = static_cast<_Float16*>(y);
  return turbo::launch_qkv_project(a, stream) == hipSuccess ? TURBO_OK : TURBO_ERR_HIP;
}

int turbo_qkv_project(const void* x, const void* w, int B, int N, int D, int Hq, int Hkv, int d,
                      int8_t* q8, float* s_q, int8_t* k8, int8_t* v8, float* s_k, float* s_v,
                      const turbo_kv_cache* cache, const int32_t* block_table,
                      const int32_t* group_table, int max_groups_per_seq, hipStream_t stream) {
  return qkv_project_impl(x, w, B, N, D, Hq, Hkv, d, q8, s_q, k8, v8, s_k, s_v, cache,
                          block_table, group_table, max_groups_per_seq, nullptr, stream);
}

int turbo_qkv_project_trace(const void* x, const void* w, int B, int N, int D, int Hq, int Hkv,
                            int d, int8_t* q8, float* s_q, int8_t* k8, int8_t* v8, float* s_k,
                            float* s_v, const turbo_kv_cache* cache, const int32_t* block_table,
                            const int32_t* group_table, int max_groups_per_seq, void* y,
                            hipStream_t stream) {
  if (B > 0 && N > 0 && !y) return TURBO_ERR_INVALID_ARG;
  return qkv_project_impl(x, w, B, N, D, Hq, Hkv, d, q8, s_q, k8, v8, s_k, s_v, cache,
                          block_table, group_table, max_groups_per_seq, y, stream);
}

int turbo_attn_prefill_blocks_trace(const void* q, const int8_t* k8, const int8_t* v8,
                                    const float* s_k, const float* s_v, int B, int Hq, int Hkv,
                                    int N, int d, float sm_scale, int causal, int block_rows,
                                    int block_cols, void* o, float* lse, int tb, int th, int ti,
                                    int tj, void* trace, hipStream_t stream) {
  if (block_rows != 32 && block_rows != 64 && block_rows != 128) return TURBO_ERR_INVALID_ARG;
  if (block_cols != 32 && block_cols != 64 && block_cols != 128) return TURBO_ERR_INVALID_ARG;
  const int nbq = N > 0 ? turbo::ceil_div(N, block_rows) : 0;
  const int nbc = N > 0 ? turbo::ceil_div(N, block_cols) : 0;
  if (!trace || tb < 0 || tb >= B || th < 0 || th >= Hq || ti < 0 || ti >= nbq || tj < 0 ||
      tj >= nbc)
    return TURBO_ERR_INVALID_ARG;
  // logical work index of (tb, th, ti): longest query blocks first
  const int tr_L = (nbq - 1 - ti) * B * Hq + tb * Hq + th;
  return attn_prefill_impl(q, nullptr, nullptr, k8, v8, s_k, s_v, B, Hq, Hkv, N, d, sm_scale,
                           causal, block_rows, block_cols, o, lse,
                           static_cast<unsigned char*>(trace), tr_L, tj, stream);
}

int turbo_attn_prefill_trace(const void* q, const int8_t* k8, const int8_t* v8,
                             const float* s_k, const float* s_v, int B, int Hq, int Hkv, int N,
                             int d, float sm_scale, int causal, void* o, float* lse, int tb,
                             int th, int ti, int tj, void* trace, hipStream_t stream) {
  return turbo_attn_prefill_blocks_trace(q, k8, v8, s_k, s_v, B, Hq, Hkv, N, d, sm_scale, causal,
                                         64, 64, o, lse, tb, th, ti, tj, trace, stream);
}

int turbo_decode_default_split(int ng) { return turbo::decode_default_split(ng); }

int turbo_decode_auto_split(int B, int Hq, int Hkv, int max_groups_per_seq) {
  if (B < 1 || Hq < 1 || Hkv < 1 || max_groups_per_seq < 1) return 1;
  // One wave per (sequence, KV head, chunk).  The decode kernel holds three
  // waves per SIMD when a KV head has at most 8 query heads and two
  // otherwise: 3072 or 2048 resident waves on the 256 CUs of gfx950.  A
  // wave's run time is set by its per-group latency chain, and the chunks of
  // a sequence are merged afterwards, so take the fewest chunks whose waves
  // fill at least two thirds of the resident slots (one chunk when the
  // sequences alone do), with the groups spread evenly over them.  A chunk
  // holds at least two groups: below that the fixed cost of a wave (query
  // quantization, state write) and of the merge outweigh the parallelism.
  const long slots = 1024L * ((Hq / Hkv) <= 8 ? 3 : 2);
  const long want = (2 * slots + 2) / 3;
  const long units = (long)B * Hkv, G = max_groups_per_seq;
  const long min_split = G < 2 ? G : 2;
  for (long n = 1; n <= G; ++n) {
    const long split = (G + n - 1) / n;
    if (split <= min_split || units * ((G + split - 1) / split) >= want)
      return (int)(split > min_split ? split : min_split);
  }
  return (int)min_split;
}

size_t turbo_decode_workspace_bytes(int B, int Hq, int Hkv, int max_groups_per_seq,
                                    int kv_split_groups, int with_tail) {
  if (B < 1 || Hq < 1 || Hkv < 1 || max_groups_per_seq < 1 || kv_split_groups < 0) return 0;
  const long nws = turbo::decode_max_chunks(max_groups_per_seq, kv_split_groups) +
                   (with_tail ? 1 : 0);
  if (nws <= 1) return 0;
  return (size_t)B * Hq * nws * turbo::kWsStride * sizeof(float);
}

static int check_tail(const turbo_kv_tail* tail, int B, int Hkv) {
  if (!tail) return TURBO_OK;
  if (!tail->k || !tail->v || !tail->scale || tail->batch < B || tail->num_kv_heads != Hkv)
    return TURBO_ERR_INVALID_ARG;
  return TURBO_OK;
}

static int attn_decode_impl(const void* q, const turbo_kv_cache* cache,
                            const turbo_kv_tail* tail, const int32_t* seq_lens,
                            const int32_t* block_table, const int32_t* group_table,
                            int max_groups_per_seq, int B, int Hq, float sm_scale,
                            int kv_split_groups, void* workspace, size_t workspace_bytes, void* o,
                            float* lse, unsigned char* trace, int tb, int th, int tg,
                            hipStream_t stream) {
  if (B < 0 || Hq < 1 || max_groups_per_seq < 1 || kv_split_groups < 0 || !cache ||
      !(sm_scale > 0.0f) || sm_scale > 3.0e38f)
    return TURBO_ERR_INVALID_ARG;
  const int Hkv = cache->num_kv_heads;
  if (Hkv < 1 || Hkv > TURBO_MAX_KV_HEADS || Hq % Hkv != 0 || Hq / Hkv > TURBO_MAX_GQA)
    return TURBO_ERR_INVALID_ARG;
  if (B == 0) return TURBO_OK;
  if (!q || !seq_lens || !block_table || !group_table || !o) return TURBO_ERR_INVALID_ARG;
  turbo::DecodeArgs a{};
  int st = check_cache(cache, Hkv, &a.int2_mask, &a.page_bytes);
  if (st != TURBO_OK) return st;
  st = check_tail(tail, B, Hkv);
  if (st != TURBO_OK) return st;
  const long nsplit = turbo::decode_max_chunks(max_groups_per_seq, kv_split_groups);
  if ((long)B * Hkv * (nsplit + (tail ? 1 : 0)) > 0x7fffffffL) return TURBO_ERR_INVALID_ARG;
  const size_t need = turbo_decode_workspace_bytes(B, Hq, Hkv, max_groups_per_seq,
                                                   kv_split_groups, tail != nullptr);
  if (need > 0 && (!workspace || workspace_bytes < need)) return TURBO_ERR_WORKSPACE_TOO_SMALL;
  st = check_device();
  if (st != TURBO_OK) return st;
  a.q = static_cast<const uint4*>(q);
  a.pages = cache->pages;
  a.gmeta = cache->group_meta;
  a.gscale = cache->group_scale;
  a.num_pages = cache->num_pages;
  a.num_slots = cache->num_group_slots;
  a.npages32 = (int)std::min<long>(cache->num_pages, 0x7fffffffL);
  a.nslots32 = (int)std::min<long>(cache->num_group_slots, 0x7fffffffL);
  a.seq_lens = seq_lens;
  a.block_table = block_table;
  a.group_table = group_table;
  a.max_groups = max_groups_per_seq;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.G = Hq / Hkv;
  a.sm_scale = sm_scale;
  a.split = kv_split_groups;
  a.nsplit = (int)nsplit;
  a.nws = (int)nsplit + (tail ? 1 : 0);
  a.ws = static_cast<float*>(workspace);
  if (tail) {
    a.tk = tail->k;
    a.tv = tail->v;
    a.tscale = tail->scale;
  }
  a.o = static_cast<uint2*>(o);
  a.lse = lse;
  a.trace = trace;
  a.tr_b = tb;
  a.tr_h = th;
  a.tr_g = tg;
  return turbo::launch_attn_decode(a, stream) == hipSuccess ? TURBO_OK : TURBO_ERR_HIP;
}

int turbo_attn_decode(const void* q, const turbo_kv_cache* cache, const turbo_kv_tail* tail,
                      const int32_t* seq_lens, const int32_t* block_table,
                      const int32_t* group_table, int max_groups_per_seq, int B, int Hq,
                      float sm_scale, int kv_split_groups, void* workspace,
                      size_t workspace_bytes, void* o, float* lse, hipStream_t stream) {
  return attn_decode_impl(q, cache, tail, seq_lens, block_table, group_table, max_groups_per_seq,
                          B, Hq, sm_scale, kv_split_groups, workspace, workspace_bytes, o, lse,
                          nullptr, -1, -1, -1, stream);
}

int turbo_attn_decode_noalloc(const void* q, const turbo_kv_cache* cache,
                              const turbo_kv_tail* tail, const int32_t* seq_lens,
                              const int32_t* block_table, const int32_t* group_table,
                              int max_groups_per_seq, int B, int Hq, float sm_scale,
                              int kv_split_groups, void* o, float* lse, hipStream_t stream) {
  if (!cache || B < 0 || Hq < 1 || max_groups_per_seq < 1 || kv_split_groups < 0)
    return TURBO_ERR_INVALID_ARG;
  const int Hkv = cache->num_kv_heads;
  if (Hkv < 1 || Hkv > TURBO_MAX_KV_HEADS || Hq % Hkv != 0) return TURBO_ERR_INVALID_ARG;
  const size_t need = turbo_decode_workspace_bytes(B, Hq, Hkv, max_groups_per_seq,
                                                   kv_split_groups, tail != nullptr);
  if (need > kDecodeScratchBytes) return TURBO_ERR_WORKSPACE_TOO_SMALL;
  void* ws = nullptr;
  if (need > 0 && B > 0) {
    const int st = check_device();  // before the symbol lookup on a foreign device
    if (st != TURBO_OK) return st;
    ws = decode_scratch();
    if (!ws) return TURBO_ERR_HIP;
  }
  return attn_decode_impl(q, cache, tail, seq_lens, block_table, group_table, max_groups_per_seq,
                          B, Hq, sm_scale, kv_split_groups, ws, ws ? kDecodeScratchBytes : 0, o,
                          lse, nullptr, -1, -1, -1, stream);
}

int turbo_attn_decode_trace(const void* q, const turbo_kv_cache* cache,
                            const turbo_kv_tail* tail, const int32_t* seq_lens,
                            const int32_t* block_table, const int32_t* group_table,
                            int max_groups_per_seq, int B, int Hq, float sm_scale,
                            int kv_split_groups, void* workspace, size_t workspace_bytes, void* o,
                            float* lse, int tb, int th, int tg, void* trace, hipStream_t stream) {
  if (!trace || tb < 0 || tb >= B || th < 0 || th >= Hq || tg < 0 || tg > max_groups_per_seq)
    return TURBO_ERR_INVALID_ARG;
  return attn_decode_impl(q, cache, tail, seq_lens, block_table, group_table, max_groups_per_seq,
                          B, Hq, sm_scale, kv_split_groups, workspace, workspace_bytes, o, lse,
                          static_cast<unsigned char*>(trace), tb, th, tg, stream);
}

size_t turbo_head_priority_workspace_bytes(int B, int Hkv, int N) {
  if (B < 1 || Hkv < 1 || N < 1) return 0;
  return turbo::head_priority_ws_bytes(B, Hkv, N);
}

int turbo_head_priority(const void* k, int B, int Hkv, int N, int d, void* workspace,
                        size_t workspace_bytes, float* priority, hipStream_t stream) {
  if (B < 0 || N < 0 || Hkv < 1 || Hkv > TURBO_MAX_KV_HEADS || d != TURBO_HEAD_DIM)
    return TURBO_ERR_INVALID_ARG;
  if (!k || !priority || B == 0 || N == 0) return TURBO_ERR_INVALID_ARG;
  const long nslab = turbo::ceil_div(N, turbo::kPrioSlab);
  if ((long)B * Hkv * N > 0x7fffffffL || (long)Hkv * B * nslab > 0x7fffffffL)
    return TURBO_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < turbo::head_priority_ws_bytes(B, Hkv, N))
    return TURBO_ERR_WORKSPACE_TOO_SMALL;
  int st = check_device();
  if (st != TURBO_OK) return st;
  turbo::PriorityArgs a{};
  a.k = static_cast<const uint4*>(k);
  a.B = B;
  a.Hkv = Hkv;
  a.N = N;
  a.nslab = (int)nslab;
  a.ws = static_cast<float*>(workspace);
  a.priority = priority;
  return turbo::launch_head_priority(a, stream) == hipSuccess ? TURBO_OK : TURBO_ERR_HIP;
}

int turbo_int2_heads(const float* priority, int Hkv, int n_int2, uint8_t* head_bits) {
  if (!priority || !head_bits || Hkv < 1 || Hkv > TURBO_MAX_KV_HEADS || n_int2 < 0 ||
      n_int2 > Hkv)
    return TURBO_ERR_INVALID_ARG;
  for (int h = 0; h < Hkv; ++h)
    if (!(priority[h] == priority[h])) return TURBO_ERR_INVALID_ARG;  // NaN
  for (int h = 0; h < Hkv; ++h) {
    int rank = 0;  // heads ranked before h: lower priority, or equal and lower index
    for (int g = 0; g < Hkv; ++g)
      if (priority[g] < priority[h] || (priority[g] == priority[h] && g < h)) ++rank;
    head_bits[h] = rank < n_int2 ? 2 : 4;
  }
  return TURBO_OK;
}

int turbo_sas_softmax(const float* x, float* y, int64_t rows, int cols, hipStream_t stream) {
  if (rows < 0 || rows > 0x7fffffffLL || cols < 1) return TURBO_ERR_INVALID_ARG;
  if (rows == 0) return TURBO_OK;
  if (!x || !y) return TURBO_ERR_INVALID_ARG;
  const int st = check_device();
  if (st != TURBO_OK) return st;
  turbo::SasSoftmaxArgs a{};
  a.x = x;
  a.y = y;
  a.rows = rows;
  a.cols = cols;
  a.vec = cols % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
          reinterpret_cast<uintptr_t>(y) % 16 == 0;
  return turbo::launch_sas_softmax(a, stream) == hipSuccess ? TURBO_OK : TURBO_ERR_HIP;
}

int turbo_tail_init(const void* k, const void* v, int B, int Hkv, int N, int d, const float* s_k,
                    const float* s_v, const turbo_kv_tail* tail, hipStream_t stream) {
  if (B < 0 || N < 0 || Hkv < 1 || Hkv > TURBO_MAX_KV_HEADS || d != TURBO_HEAD_DIM)
    return TURBO_ERR_INVALID_ARG;
  if (B == 0) return TURBO_OK;
  if (N == 0 || !k || !v || !s_k || !s_v || !tail) return TURBO_ERR_INVALID_ARG;
  int st = check_tail(tail, B, Hkv);
  if (st != TURBO_OK) return st;
  if ((long)B * Hkv * N > 0x7fffffffL) return TURBO_ERR_INVALID_ARG;
  st = check_device();
  if (st != TURBO_OK) return st;
  turbo::TailInitArgs a{};
  a.k = static_cast<const unsigned short*>(k);
  a.v = static_cast<const unsigned short*>(v);
  a.sk = s_k;
  a.sv = s_v;
  a.Hkv = Hkv;
  a.N = N;
  a.nb = turbo::ceil_div(N, TURBO_BLOCK);
  a.tk = tail->k;
  a.tv = tail->v;
  a.tscale = tail->scale;
  return turbo::launch_tail_init(a, B, stream) == hipSuccess ? TURBO_OK : TURBO_ERR_HIP;
}

int turbo_append_kv(const void* k_new, const void* v_new, int B, int Hkv, int d,
                    const int32_t* seq_lens, const turbo_kv_cache* cache,
                    const turbo_kv_tail* tail, const int32_t* block_table,
                    const int32_t* group_table, int max_groups_per_seq, hipStream_t stream) {
  if (B < 0 || Hkv < 1 || Hkv > TURBO_MAX_KV_HEADS || d != TURBO_HEAD_DIM ||
      max_groups_per_seq < 1)
    return TURBO_ERR_INVALID_ARG;
  if (B == 0) return TURBO_OK;
  if (!k_new || !v_new || !seq_lens || !cache || !tail || !block_table || !group_table)
    return TURBO_ERR_INVALID_ARG;
  turbo::AppendArgs a{};
  int st = check_cache(cache, Hkv, &a.int2_mask, &a.page_bytes);
  if (st != TURBO_OK) return st;
  st = check_tail(tail, B, Hkv);
  if (st != TURBO_OK) return st;
  st = check_device();
  if (st != TURBO_OK) return st;
  a.knew = static_cast<const unsigned short*>(k_new);
  a.vnew = static_cast<const unsigned short*>(v_new);
  a.seq_lens = seq_lens;
  a.Hkv = Hkv;
  a.tk = tail->k;
  a.tv = tail->v;
  a.tscale = tail->scale;
  a.pages = cache->pages;
  a.gmeta = cache->group_meta;
  a.gscale = cache->group_scale;
  a.num_pages = cache->num_pages;
  a.num_slots = cache->num_group_slots;
  a.block_table = block_table;
  a.group_table = group_table;
  a.max_groups = max_groups_per_seq;
  return turbo::launch_append_kv(a, B, stream) == hipSuccess ? TURBO_OK : TURBO_ERR_HIP;
}

int turbo_probe_mfma_i8(int iters, int* sink, int64_t* ops, hipStream_t stream) {
  if (iters < 1 || !sink || !ops) return TURBO_ERR_INVALID_ARG;
  const int st = check_device();
  if (st != TURBO_OK) return st;
  // 4 waves per work-group, kProbeChains MFMAs of 2 * 16 * 16 * 64 ops each
  *ops = (int64_t)turbo::kProbeMfmaBlocks * 4 * turbo::kProbeChains * iters * (2 * 16 * 16 * 64);
  return turbo::launch_probe_mfma_i8(iters, sink, stream) == hipSuccess ? TURBO_OK
                                                                         : TURBO_ERR_HIP;
}

int turbo_probe_valu(int iters, float* sink, int64_t* insts, hipStream_t stream) {
  if (iters < 1 || !sink || !insts) return TURBO_ERR_INVALID_ARG;
  const int st = check_device();
  if (st != TURBO_OK) return st;
  // 4 waves per work-group, kProbeChains FMAs per round
  *insts = (int64_t)turbo::kProbeValuBlocks * 4 * turbo::kProbeChains * iters;
  return turbo::launch_probe_valu(iters, sink, stream) == hipSuccess ? TURBO_OK : TURBO_ERR_HIP;
}

int turbo_probe_read(const void* src, size_t bytes, unsigned* sink, hipStream_t stream) {
  if (!src || !sink || bytes < 16 || bytes % 16 != 0 || bytes > (size_t(1) << 40) ||
      reinterpret_cast<uintptr_t>(src) % 16 != 0)
    return TURBO_ERR_INVALID_ARG;
  const int st = check_device();
  if (st != TURBO_OK) return st;
  return turbo::launch_probe_read(src, bytes, sink, stream) == hipSuccess ? TURBO_OK
                                                                          : TURBO_ERR_HIP;
}

}  // extern "C"
