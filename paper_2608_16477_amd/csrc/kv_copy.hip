// Suffix-block extraction (pack) and assembly (scatter) between a paged KV
// pool and contiguous per-layer transfer chunks.
//
// Pool  bf16 [2L][P][page][row]   (row = Hkv * d elements, K after rotary)
// Chunk bf16 [2L][count][row]     at arena + offset
//
// One work unit is (chunk, layer-plane, run of up to 16 consecutive
// positions).  Each position's row is contiguous on both sides, and at page
// aligned runs so is the whole 16-position run, so the copy streams 16-byte
// vectors with every wave reading and writing contiguous memory.  With pages
// of at least 16 slots a run touches at most two pages, whose table entries
// are read once per workgroup.  The copy
// is a pure bit move: no conversion, bit-exact by construction.
#include "common.h"
#include "kernels.h"

namespace pallas {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 8;
constexpr int64_t kNtStoreBytes = int64_t(512) << 20;   // payload bytes read per launch

// Stores: plain for launches up to kNtStoreBytes of payload (measured 74-80%
// of HBM peak at 262 MB, against 62-67% with non-temporal stores), non-
// temporal above it (68% against 65% at 1 GiB read + 1 GiB written).
// Loads are non-temporal in both.
template <bool kPack, bool kNtStore>
__global__ __launch_bounds__(kThreads) void kv_copy_kernel(PoolGeom pool,
                                                           const int32_t* __restrict__ bt,
                                                           char* __restrict__ arena,
                                                           CopyBatch b,
                                                           int32_t* __restrict__ err) {
  auto store = [](u32x4* d, const u32x4& v) {
    if (kNtStore) __builtin_nontemporal_store(v, d);
    else *d = v;
  };
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
  if (pool.page < kCopyTokens) {
    // Pages shorter than a run: look up each position's page.
    for (int e0 = threadIdx.x; e0 < total; e0 += kThreads * kUnroll) {
      u32x4 v[kUnroll];
      u32x4* dst[kUnroll];
#pragma unroll
      for (int k = 0; k < kUnroll; ++k) {
        dst[k] = nullptr;
        const int e = e0 + k * kThreads;
        if (e < total) {
          const int i = e / vpr, w = e - (e / vpr) * vpr;
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
        if (dst[k]) store(dst[k], v[k]);
    }
    return;
  }
  // The run's positions span at most two pages: read both table entries once.
  const int tf = c.start + t0;
  const int first_in = pool.page - tf % pool.page;   // positions on the first page
  const int pg0 = bt[tf / pool.page];
  const int pg1 = nt > first_in ? bt[(tf + nt - 1) / pool.page] : pg0;
  const bool ok0 = pg0 >= 0 && pg0 < pool.num_pages, ok1 = pg1 >= 0 && pg1 < pool.num_pages;
  if (err && threadIdx.x == 0 && (!ok0 || (nt > first_in && !ok1))) atomicOr(err, 1);
  // Pool byte offsets of the run's first slot on each page (the second page
  // starts at slot 0).
  const int64_t base0 = (static_cast<int64_t>(pg0) * pool.page + tf % pool.page) * row;
  const int64_t base1 = static_cast<int64_t>(pg1) * pool.page * row;

  // Thread element e = (row i, vector w); advance by kThreads per step
  // without dividing.
  int i = threadIdx.x / vpr, w = threadIdx.x - (threadIdx.x / vpr) * vpr;
  const int di = kThreads / vpr, dw = kThreads - di * vpr;
  for (int e0 = threadIdx.x; e0 < total; e0 += kThreads * kUnroll) {
    u32x4 v[kUnroll];
    u32x4* dst[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      dst[k] = nullptr;
      if (e0 + k * kThreads < total) {
        const bool second = i >= first_in;
        if (second ? ok1 : ok0) {
          u32x4* pp = reinterpret_cast<u32x4*>(
                          pool_plane + (second ? base1 + static_cast<int64_t>(i - first_in) * row
                                               : base0 + static_cast<int64_t>(i) * row)) + w;
          u32x4* cp = reinterpret_cast<u32x4*>(chunk_plane + static_cast<int64_t>(t0 + i) * row) + w;
          if (kPack) { v[k] = __builtin_nontemporal_load(pp); dst[k] = cp; }
          else       { v[k] = __builtin_nontemporal_load(cp); dst[k] = pp; }
        }
      }
      i += di;
      w += dw;
      if (w >= vpr) { w -= vpr; ++i; }
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k)
      if (dst[k]) store(dst[k], v[k]);
  }
}

}  // namespace

hipError_t launch_kv_copy(bool pack, const PoolGeom& pool, const int32_t* bt, char* arena,
                          const CopyBatch& b, int32_t* d_err, hipStream_t s) {
  const int units = b.unit_prefix[b.n];
  if (units == 0) return hipSuccess;
  int64_t payload = 0;
  for (int j = 0; j < b.n; ++j) payload += static_cast<int64_t>(b.c[j].count) * pool.lk * pool.row_bytes;
  const bool nt = payload > kNtStoreBytes;
  if (pack) {
    if (nt) kv_copy_kernel<true, true><<<units, kThreads, 0, s>>>(pool, bt, arena, b, d_err);
    else kv_copy_kernel<true, false><<<units, kThreads, 0, s>>>(pool, bt, arena, b, d_err);
  } else {
    if (nt) kv_copy_kernel<false, true><<<units, kThreads, 0, s>>>(pool, bt, arena, b, d_err);
    else kv_copy_kernel<false, false><<<units, kThreads, 0, s>>>(pool, bt, arena, b, d_err);
  }
  return hipGetLastError();
}

}  // namespace pallas
