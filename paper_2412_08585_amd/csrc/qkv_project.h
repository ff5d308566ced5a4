// Arguments and launcher of the fused QKV projection (qkv_project.hip, a
// translation unit of its own: its accumulators live in the AGPR file, which
// the attention kernels are built not to use).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace turbo {

struct QkvArgs {
  const void* x;   // fp16 [B][N][D]
  const void* w;   // fp16 [F][D], F = (Hq + 2 Hkv) * 128
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

// Tokens per work-group tile (ntile = ceil(N / kQkvTileTokens)).
constexpr int kQkvTileTokens = 256;

hipError_t launch_qkv_project(const QkvArgs& a, hipStream_t stream);

}  // namespace turbo
