// Internal launch interface between the C ABI (pallas_api.hip) and the
// kernels.  Every launcher enqueues on `s` and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pallas {

// ----------------------------------------------------------------- KV copies
struct PoolGeom {
  char* base;         // bf16 [L][2][num_pages][page][Hkv][d]
  int32_t num_pages;
  int32_t page;
  int32_t lk;         // 2 * L: (layer, K|V) planes
  int32_t row_bytes;  // Hkv * d * 2, a multiple of 16
};

constexpr int kCopyMaxChunks = 128;   // chunks per copy launch
constexpr int kCopyTokens = 16;       // tokens per work unit

struct CopyChunk {
  int32_t start;       // first logical position
  int32_t count;       // positions
  uint64_t offset;     // byte offset of [2L][count][row] in the arena
};
struct CopyBatch {
  int32_t n;
  int32_t unit_prefix[kCopyMaxChunks + 1];  // work units before chunk j
  CopyChunk c[kCopyMaxChunks];
};

// Pack (pool -> arena) or assemble (arena -> pool) of up to kCopyMaxChunks
// chunks through one block table.
hipError_t launch_kv_copy(bool pack, const PoolGeom& pool, const int32_t* bt, char* arena,
                          const CopyBatch& b, int32_t* d_err, hipStream_t s);

}  // namespace pallas
