// Suffix-block extraction (pack) and assembly (scatter) between a paged KV
// pool and contiguous per-layer transfer chunks.
//
// Pool  bf16 [2L][P][page][row]   (row = Hkv * d elements, K after rotary)
// Chunk bf16 [2L][count][row]     at arena + offset
//
// One work unit is (chunk, layer-plane, run of up to 16 consecutive
// positions).  Each position's row is contiguous on both sides, and at page
// aligned runs so is the whole 16-position run, so the copy streams 16-byte
// vectors with every wave reading and writing contiguous memory.  The copy
// is a pure bit move: no conversion, bit-exact by construction.
#include "common.h"
#include "kernels.h"

namespace pallas {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 8;

template <bool kPack>
__global__ __launch_bounds__(kThreads) void kv_copy_kernel(PoolGeom pool,
                                                           const int32_t* __restrict__ bt,
                                                           char* __restrict__ arena,
                                                           CopyBatch b,
                                                           int32_t* __restrict__ err) {
  const int u = blockIdx.x;
  // chunk j: largest j with unit_prefix[j] <= u
  int lo = 0, hi = b.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (b.unit_prefix[mid] <= u) lo = mid; else hi = mid - 1;
  }
  const CopyChunk c = b.c[lo];
  const int local = u - b.unit_prefix[lo];
  const int nb = (c.count + kCopyTokens - 1) / kCopyTokens;
  const int plane = local / nb;
  const int t0 = (local - plane * nb) * kCopyTokens;
  const int nt = min(kCopyTokens, c.count - t0);
  const int vpr = pool.row_bytes >> 4;  // 16-byte vectors per row
  const int total = nt * vpr;

  const int64_t row = pool.row_bytes;
  char* chunk_plane = arena + c.offset + static_cast<int64_t>(plane) * c.count * row;
  char* pool_plane = pool.base + static_cast<int64_t>(plane) * pool.num_pages * pool.page * row;

  for (int e0 = threadIdx.x; e0 < total; e0 += kThreads * kUnroll) {
    u32x4 v[kUnroll];
    u32x4* dst[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      dst[k] = nullptr;
      const int e = e0 + k * kThreads;
      if (e < total) {
        const int i = e / vpr;
        const int w = e - i * vpr;
        const int t = c.start + t0 + i;
        const int pg = bt[t / pool.page];
        if (pg < 0 || pg >= pool.num_pages) {
          if (w == 0 && err) atomicOr(err, 1);
          continue;
        }
        u32x4* pp = reinterpret_cast<u32x4*>(
                        pool_plane + (static_cast<int64_t>(pg) * pool.page + t % pool.page) * row) + w;
        u32x4* cp = reinterpret_cast<u32x4*>(chunk_plane + static_cast<int64_t>(t0 + i) * row) + w;
        if (kPack) { v[k] = __builtin_nontemporal_load(pp); dst[k] = cp; }
        else       { v[k] = __builtin_nontemporal_load(cp); dst[k] = pp; }
      }
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k)
      if (dst[k]) __builtin_nontemporal_store(v[k], dst[k]);
  }
}

}  // namespace

hipError_t launch_kv_copy(bool pack, const PoolGeom& pool, const int32_t* bt, char* arena,
                          const CopyBatch& b, int32_t* d_err, hipStream_t s) {
  const int units = b.unit_prefix[b.n];
  if (units == 0) return hipSuccess;
  if (pack)
    kv_copy_kernel<true><<<units, kThreads, 0, s>>>(pool, bt, arena, b, d_err);
  else
    kv_copy_kernel<false><<<units, kThreads, 0, s>>>(pool, bt, arena, b, d_err);
  return hipGetLastError();
}

}  // namespace pallas
