// Sanitizer driver of the C ABI's host side (test infrastructure): the
// library's host code (argument checks, sizing helpers, the bit-width
// choice, error strings) built under AddressSanitizer and UndefinedBehavior-
// Sanitizer and called with valid, extreme and invalid arguments.  Calls that
// pass the checks stop at the device check when no GPU is present (or, with
// one, at launches that never happen because the checks come first for the
// invalid cases).  Exit status 0: clean.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <limits>

#include "turbo_attn.h"

static int fails = 0;
#define EXPECT(c)                                                      \
  do {                                                                 \
    if (!(c)) {                                                        \
      std::fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, \
                   __LINE__, #c);                                      \
      ++fails;                                                         \
    }                                                                  \
  } while (0)

int main() {
  EXPECT(turbo_abi_version() == TURBO_ABI_VERSION);
  for (int s = -10; s <= 10; ++s) EXPECT(turbo_strerror(s) != nullptr);

  uint8_t bits[TURBO_MAX_KV_HEADS + 1];
  for (auto& b : bits) b = 4;
  EXPECT(turbo_page_bytes(bits, TURBO_MAX_KV_HEADS) == 2048u * TURBO_MAX_KV_HEADS);
  EXPECT(turbo_page_bytes(bits, TURBO_MAX_KV_HEADS + 1) == 0);
  EXPECT(turbo_page_bytes(nullptr, 3) == 0);
  bits[1] = 3;
  EXPECT(turbo_page_bytes(bits, 2) == 0);
  bits[1] = 2;

  // sizing helpers over wide and extreme ranges (overflow is undefined
  // behaviour in the host arithmetic, which the sanitizer reports)
  const int vals[] = {-1, 0, 1, 2, 31, 32, 33, 127, 128, 129, 512, 4096, 1 << 20, 0x7fffffff};
  for (int a : vals) {
    (void)turbo_decode_default_split(a);
    for (int b : vals) {
      (void)turbo_decode_auto_split(a, 32, 8, b);
      (void)turbo_decode_workspace_bytes(a, 40, 10, b, 0, 1);
      (void)turbo_decode_workspace_bytes(a, 40, 10, b, 3, 0);
      (void)turbo_head_priority_workspace_bytes(a, 10, b);
    }
  }

  // the Sec. 3.2 bit choice: ties, NaN, bounds
  float prio[4] = {3.0f, 1.0f, 1.0f, 2.0f};
  uint8_t hb[4];
  EXPECT(turbo_int2_heads(prio, 4, 2, hb) == TURBO_OK && hb[1] == 2 && hb[2] == 2 && hb[0] == 4);
  EXPECT(turbo_int2_heads(prio, 4, 5, hb) == TURBO_ERR_INVALID_ARG);
  prio[3] = std::numeric_limits<float>::quiet_NaN();
  EXPECT(turbo_int2_heads(prio, 4, 1, hb) == TURBO_ERR_INVALID_ARG);

  // invalid arguments are rejected before any device call
  char dummy[256] = {};
  void* p = dummy;
  turbo_kv_cache cache{};
  cache.pages = reinterpret_cast<uint8_t*>(dummy);
  cache.group_meta = reinterpret_cast<int8_t*>(dummy);
  cache.group_scale = reinterpret_cast<float*>(dummy);
  cache.num_pages = 4;
  cache.num_group_slots = 1;
  cache.num_kv_heads = 2;
  cache.head_dim = 128;
  cache.head_bits[0] = 4;
  cache.head_bits[1] = 2;
  auto i8 = reinterpret_cast<int8_t*>(dummy);
  auto f = reinterpret_cast<float*>(dummy);
  auto i32 = reinterpret_cast<int32_t*>(dummy);
  EXPECT(turbo_quantize_kv(p, p, 1, 2, 64, 64, i8, i8, f, f, nullptr, nullptr, nullptr, 0,
                           nullptr) == TURBO_ERR_INVALID_ARG);
  EXPECT(turbo_quantize_kv(p, p, 1, 65, 64, 128, i8, i8, f, f, nullptr, nullptr, nullptr, 0,
                           nullptr) == TURBO_ERR_INVALID_ARG);
  EXPECT(turbo_quantize_kv(p, p, 1, 2, 128, 128, i8, i8, f, f, &cache, i32, i32, 1, nullptr) ==
         TURBO_ERR_INVALID_ARG);  // table shorter than the groups
  EXPECT(turbo_quantize_kv(p, p, 0, 2, 64, 128, nullptr, nullptr, nullptr, nullptr, nullptr,
                           nullptr, nullptr, 0, nullptr) == TURBO_OK);  // empty batch
  EXPECT(turbo_attn_prefill(p, i8, i8, f, f, 1, 3, 2, 64, 128, 0.1f, 1, p, nullptr, nullptr) ==
         TURBO_ERR_INVALID_ARG);  // Hq % Hkv
  EXPECT(turbo_attn_prefill(p, i8, i8, f, f, 1, 2, 2, 64, 128, -1.0f, 1, p, nullptr, nullptr) ==
         TURBO_ERR_INVALID_ARG);
  EXPECT(turbo_attn_prefill(p, i8, i8, f, f, 0x7fffffff, 64, 1, 0x7fffffff, 128, 0.1f, 1, p,
                            nullptr, nullptr) == TURBO_ERR_INVALID_ARG);  // too many tiles
  EXPECT(turbo_attn_prefill_blocks(p, i8, i8, f, f, 1, 2, 2, 64, 128, 0.1f, 1, 48, 64, p, nullptr,
                                   nullptr) == TURBO_ERR_INVALID_ARG);
  EXPECT(turbo_attn_prefill_trace(p, i8, i8, f, f, 1, 2, 2, 64, 128, 0.1f, 1, p, nullptr, 0, 0, 0,
                                  1, p, nullptr) == TURBO_ERR_INVALID_ARG);  // tile j >= nb
  EXPECT(turbo_attn_decode(p, &cache, nullptr, i32, i32, i32, 4, 1, 3, 0.1f, 0, nullptr, 0, p,
                           nullptr, nullptr) == TURBO_ERR_INVALID_ARG);  // Hq % Hkv
  EXPECT(turbo_attn_decode(p, &cache, nullptr, i32, i32, i32, 512, 64, 8, 0.1f, 0, nullptr, 0, p,
                           nullptr, nullptr) == TURBO_ERR_WORKSPACE_TOO_SMALL);
  EXPECT(turbo_attn_decode_noalloc(p, &cache, nullptr, i32, i32, i32, 512, 100000, 3, 0.1f, 0, p,
                                   nullptr, nullptr) == TURBO_ERR_INVALID_ARG);  // Hq % Hkv
  EXPECT(turbo_attn_decode_noalloc(p, &cache, nullptr, i32, i32, i32, 512, 4096, 32, 0.1f, 1, p,
                                   nullptr, nullptr) == TURBO_ERR_WORKSPACE_TOO_SMALL);
  EXPECT(turbo_qkv_project(p, p, 1, 64, 96, 2, 1, 128, i8, f, i8, i8, f, f, nullptr, nullptr,
                           nullptr, 0, nullptr) == TURBO_ERR_INVALID_ARG);  // D % 64
  EXPECT(turbo_qkv_project_trace(p, p, 1, 64, 64, 2, 1, 128, i8, f, i8, i8, f, f, nullptr,
                                 nullptr, nullptr, 0, nullptr, nullptr) == TURBO_ERR_INVALID_ARG);
  EXPECT(turbo_head_priority(p, 1, 2, 64, 128, p, 0, f, nullptr) ==
         TURBO_ERR_WORKSPACE_TOO_SMALL);
  EXPECT(turbo_sas_softmax(f, f, -1, 4, nullptr) == TURBO_ERR_INVALID_ARG);
  EXPECT(turbo_sas_softmax(f, f, 0, 4, nullptr) == TURBO_OK);
  turbo_kv_tail tail{i8, i8, f, 1, 2};
  EXPECT(turbo_tail_init(p, p, 2, 2, 64, 128, f, f, &tail, nullptr) == TURBO_ERR_INVALID_ARG);
  EXPECT(turbo_append_kv(p, p, 1, 2, 128, i32, &cache, &tail, i32, i32, 0, nullptr) ==
         TURBO_ERR_INVALID_ARG);
  EXPECT(turbo_probe_mfma_i8(0, i32, nullptr, nullptr) == TURBO_ERR_INVALID_ARG);
  EXPECT(turbo_probe_read(p, 17, reinterpret_cast<unsigned*>(dummy), nullptr) ==
         TURBO_ERR_INVALID_ARG);

  // valid arguments: without a GPU these stop at the device check
  int64_t ops = 0;
  const int st = turbo_probe_mfma_i8(1, nullptr, &ops, nullptr);
  EXPECT(st == TURBO_ERR_INVALID_ARG);
  std::printf("abi sanitizer driver: %s (%d failed expectations)\n", fails ? "FAILED" : "ok",
              fails);
  return fails ? 1 : 0;
}
