// Skinny GEMM for decode (M <= 8 rows): C = X W^T streaming the weights once.
//
// A workgroup of 4 waves owns one 16-row weight tile (two for the gate|up
// projection: 16 gate rows and the matching 16 up rows) and splits K four
// ways.  Each wave streams its K range in steps of 64: one 128-byte line of
// each weight row and the matching 64 columns of X go straight from memory
// into a private LDS stage with buffer_load ... lds (three stages in
// flight), each load instruction covering whole lines of 8 rows.  Inside a
// stage the 16-byte slots are permuted so the v_mfma_f32_16x16x32_bf16
// operand reads (16 rows at one k) hit 16 distinct bank groups.  The four
// partial tiles are summed through LDS and the epilogue matches the prefill
// GEMM's.  Launches with fewer than two tiles per CU (O and down) also split
// K over up to kGemvMaxSplit workgroups per tile: each writes its partial
// sums with agent-scope stores and counts itself in a per-tile counter, and
// the last to arrive adds the splits in order and applies the epilogue.
#include <cmath>

#include "common.h"
#include "kernels.h"

namespace pallas {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kKStep = 64;        // k per stage: one 128-byte line per weight row
constexpr int kBlockSlots = 68;   // 8 rows x 8 slots of 16 B, plus 4 slots of padding

typedef __attribute__((address_space(3))) void lds_void;

template <int TILES>
struct GvLayout {
  static constexpr int kStages = 3;                                   // stages in flight per wave
  static constexpr int kWBlocks = 2 * TILES;                          // 8-row blocks per stage
  static constexpr int kStageSlots = kWBlocks * kBlockSlots + 64;     // + one X block
  static constexpr int kWaveSlots = kStages * kStageSlots;
  static constexpr int kLoads = kWBlocks + 1;                         // load instructions per stage
};

// Weight block slot of (row rr in 0..7, 16-byte chunk c in 0..7).
__device__ __forceinline__ int wslot(int rr, int c) {
  return (rr & 3) + 8 * (rr >> 2) + 4 * (c & 1) + 16 * (c >> 1);
}
// X block slot of (row r in 0..7, chunk c in 0..7).
__device__ __forceinline__ int xslot(int r, int c) { return r * 8 + (c ^ r); }

// K split over workgroups: workgroup (tile, ks) covers K range ks of S and
// writes float32 partial sums to part[ks][m][B row]; the last workgroup of
// a tile to finish (an atomic count in ctr[tile], which it resets to 0)
// adds the S partials in order and applies the epilogue.
struct GemvSplit {
  int S;
  float* part;   // [S][M][B rows]
  int* ctr;      // [tiles], zero on entry
  int nrows;     // B rows: N, or 2N for gate|up
};

template <int EPI, int TILES>
__global__ __launch_bounds__(kThreads) void gemv_kernel(const uint16_t* __restrict__ X, int ldx,
                                                        const uint16_t* __restrict__ W, int ldw,
                                                        void* __restrict__ C, int ldc, int M, int N,
                                                        int K, GemvSplit sp) {
  using L = GvLayout<TILES>;
  __shared__ __attribute__((aligned(16))) u32x4 lds[kWaves * L::kWaveSlots];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int li = lane & 15, kg = lane >> 4;
  const int tile = static_cast<int>(blockIdx.x) / sp.S, ks = static_cast<int>(blockIdx.x) % sp.S;

  // Weight tiles: first row and valid row count.
  int trow[TILES], tvalid[TILES];
  if (EPI == kEpiSwiGLU) {
    const int o0 = tile * 16;
    trow[0] = o0;
    trow[TILES - 1] = N + o0;
    tvalid[0] = tvalid[TILES - 1] = min(16, N - o0);
  } else {
#pragma unroll
    for (int t = 0; t < TILES; ++t) {
      trow[t] = (tile * TILES + t) * 16;
      // The same in every lane: keeps the descriptors in scalar registers.
      tvalid[t] = __builtin_amdgcn_readfirstlane(max(0, min(16, N - trow[t])));
    }
  }
  auto tile_rsrc = [&](int t) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)(W + static_cast<int64_t>(tvalid[t] > 0 ? trow[t] : 0) * ldw), 0,
                                             static_cast<uint32_t>(tvalid[t]) * ldw * 2u, 0x00020000);
  };
  const __amdgpu_buffer_rsrc_t rw0 = tile_rsrc(0), rw1 = tile_rsrc(TILES - 1);
  const __amdgpu_buffer_rsrc_t rx =
      __builtin_amdgcn_make_buffer_rsrc((void*)X, 0, static_cast<uint32_t>(M) * ldx * 2u, 0x00020000);
  constexpr uint32_t kOob = 0xFFFFFFF0u;

  // This workgroup's K range [kw0, kw1), then a quarter of it per wave.
  const int kper = ((K + sp.S * kKStep - 1) / (sp.S * kKStep)) * kKStep;
  const int kw0 = ks * kper, kw1 = min(K, kw0 + kper);
  const int kslice = ((max(kw1 - kw0, 0) + kWaves * kKStep - 1) / (kWaves * kKStep)) * kKStep;
  const int kb = kw0 + wave * kslice, ke = min(kw1, kb + kslice);
  const int nst = ke > kb ? (ke - kb + kKStep - 1) / kKStep : 0;

  // Per-lane load coordinates (fixed for every stage).
  // Weight block instruction: lane -> slot lane -> (row rr, chunk c).
  const int b = lane & 15;
  const int w_rr = (b & 3) | ((b >> 3) << 2);
  const int w_c = ((lane >> 4) << 1) | ((b >> 2) & 1);
  // X block instruction: lane -> row lane/8, chunk (lane%8) ^ row.
  const int x_r = lane >> 3;
  const int x_c = (lane & 7) ^ x_r;

  u32x4* wbase = lds + wave * L::kWaveSlots;
  auto issue = [&](int s) {
    const int k0 = kb + s * kKStep;
    u32x4* st = wbase + (s % L::kStages) * L::kStageSlots;
#pragma unroll
    for (int blk = 0; blk < L::kWBlocks; ++blk) {
      const int t = blk >> 1;
      const int row = (blk & 1) * 8 + w_rr;
      const int k = k0 + w_c * 8;
      const uint32_t off = k < ke ? static_cast<uint32_t>(row) * ldw * 2u + static_cast<uint32_t>(k) * 2u : kOob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(t == 0 ? rw0 : rw1, (lds_void*)(st + blk * kBlockSlots), 16, off, 0, 0, 0);
    }
    const int k = k0 + x_c * 8;
    const uint32_t off = (x_r < M && k < ke) ? static_cast<uint32_t>(x_r) * ldx * 2u + static_cast<uint32_t>(k) * 2u : kOob;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void*)(st + L::kWBlocks * kBlockSlots), 16, off, 0, 0, 0);
  };

  f32x4 acc[TILES];
#pragma unroll
  for (int t = 0; t < TILES; ++t) acc[t] = f32x4{0, 0, 0, 0};
  auto compute = [&](int s) {
    const u32x4* st = wbase + (s % L::kStages) * L::kStageSlots;
#pragma unroll
    for (int q = 0; q < kKStep / 32; ++q) {
      const int c = 4 * q + kg;
      const bf16x8 a = __builtin_bit_cast(bf16x8, st[L::kWBlocks * kBlockSlots + xslot(li & 7, c)]);
#pragma unroll
      for (int t = 0; t < TILES; ++t) {
        const bf16x8 w = __builtin_bit_cast(bf16x8, st[(2 * t + (li >> 3)) * kBlockSlots + wslot(li & 7, c)]);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, w, acc[t], 0, 0, 0);
      }
    }
  };

  for (int s = 0; s < L::kStages - 1 && s < nst; ++s) issue(s);
  for (int s = 0; s < nst; ++s) {
    asm volatile("" ::: "memory");
    if (s + L::kStages - 1 < nst) {
      issue(s + L::kStages - 1);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"((L::kStages - 1) * L::kLoads) : "memory");
    } else {
      // Tail: stages s+1 .. nst-1 may stay in flight.
      switch (nst - 1 - s) {
        case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
        case 1: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(L::kLoads) : "memory"); break;
        case 2: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * L::kLoads) : "memory"); break;
        case 3: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(3 * L::kLoads) : "memory"); break;
        default: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(4 * L::kLoads) : "memory"); break;
      }
    }
    compute(s);
  }

  // Sum the per-wave partial tiles.
  __syncthreads();
  f32x4* red = reinterpret_cast<f32x4*>(lds);
#pragma unroll
  for (int t = 0; t < TILES; ++t) red[(wave * TILES + t) * 64 + lane] = acc[t];
  __syncthreads();
  if (wave != 0) return;
  f32x4 sum[TILES];
#pragma unroll
  for (int t = 0; t < TILES; ++t) {
    sum[t] = red[t * 64 + lane];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) sum[t] += red[(w * TILES + t) * 64 + lane];
  }
  // lane holds column li and rows kg*4 + r
  if (sp.S > 1) {
    const bool col_ok = (EPI == kEpiSwiGLU ? tile * 16 : trow[0]) + li < N;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = kg * 4 + r;
      if (m >= M || !col_ok) continue;
#pragma unroll
      for (int t = 0; t < TILES; ++t)
        __hip_atomic_store(sp.part + (static_cast<int64_t>(ks) * M + m) * sp.nrows + trow[t] + li, sum[t][r],
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // The partials are agent-scope atomic stores, which write through this
    // XCD's L2 to the device-coherent level; once they have completed
    // (vmcnt 0), the count goes up.  The reader's agent-scope atomic loads
    // miss its own L2, and are issued only after the count they branch on
    // has returned.  That is the agent-scope release/acquire sequence of
    // the gfx950 memory model for data accessed only through agent-scope
    // atomics: its L2 write-back and invalidate act on non-atomic data
    // only, and as fences (__ATOMIC_RELEASE / __ATOMIC_ACQUIRE at agent
    // scope) they cost a whole L2 per workgroup: measured, a decode step
    // of the large model took 21.6 ms with them against 14.9 ms.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    int prev = 0;
    if (lane == 0) prev = __hip_atomic_fetch_add(sp.ctr + tile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    prev = __shfl(prev, 0, kWave);
    if (prev != sp.S - 1) return;
    asm volatile("" ::: "memory");
    // Last of the tile: the others' partials, read past this XCD's L2.
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = kg * 4 + r;
#pragma unroll
      for (int t = 0; t < TILES; ++t) {
        float v = 0.f;
        if (m < M && col_ok)
          for (int j = 0; j < sp.S; ++j)
            v += __hip_atomic_load(sp.part + (static_cast<int64_t>(j) * M + m) * sp.nrows + trow[t] + li,
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        sum[t][r] = v;
      }
    }
    if (lane == 0) __hip_atomic_store(sp.ctr + tile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int m = kg * 4 + r;
    if (m >= M) continue;
    if (EPI == kEpiSwiGLU) {
      const int col = tile * 16 + li;
      if (col < N) {
        const float gt = sum[0][r], up = sum[TILES - 1][r];
        static_cast<uint16_t*>(C)[static_cast<int64_t>(m) * ldc + col] = f2bf(swiglu(gt, up));
      }
    } else {
#pragma unroll
      for (int t = 0; t < TILES; ++t) {
        const int col = trow[t] + li;
        if (col >= N) continue;
        const float v = sum[t][r];
        const int64_t at = static_cast<int64_t>(m) * ldc + col;
        if (EPI == kEpiBf16) static_cast<uint16_t*>(C)[at] = f2bf(v);
        else if (EPI == kEpiAddF32) static_cast<float*>(C)[at] += v;
        else static_cast<float*>(C)[at] = v;
      }
    }
  }
}

__global__ void fill_zero_kernel(int* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

}  // namespace

int gemv_ksplit(int epi, int N, int K) {
  // Workgroups per tile, for launches of fewer than two tiles per CU (O and
  // down at the large shape: 320 tiles): the split whose workgroup count
  // divides most evenly over the 256 CUs, with at least four 64-wide
  // K-steps per wave and every workgroup resident at once (the LDS stages
  // hold four single-tile or two gate|up workgroups per CU), and only when it beats no
  // split by more than 5%.  Measured at the large shape, M = 1: O 21.6 ->
  // 18.8 us and down 64 -> 58 us with four splits, and three (960
  // workgroups) beat four (1280, a fifth of them in a second round): the
  // decode step 14.94 -> 14.63 ms.  Q|K|V (640 tiles) and gate|up (1600)
  // ran 10% slower split in two, so they do not split.
  const int tiles = (N + 15) / 16;
  if (tiles >= 512) return 1;
  const int resident = 256 * (epi == kEpiSwiGLU ? 2 : 4);
  auto eff = [&](int s) {
    const double per_cu = double(tiles) * s / 256.0;
    return per_cu / std::ceil(per_cu);
  };
  int best = 1;
  for (int s = 2; s <= kGemvMaxSplit; ++s) {
    if (K / (s * kWaves * kKStep) < 4 || tiles * s > resident) break;
    if (eff(s) > eff(best) + 0.05) best = s;
  }
  return best;
}

hipError_t launch_zero_counters(int* ctr, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  fill_zero_kernel<<<(n + 255) / 256, 256, 0, s>>>(ctr, n);
  return hipGetLastError();
}

hipError_t launch_gemv(int epi, const uint16_t* A, int lda, const uint16_t* B, int ldb, void* C,
                       int ldc, int M, int N, int K, float* part, size_t part_bytes, int* ctr,
                       int ctr_count, hipStream_t s) {
  if (M <= 0 || M > 8 || N <= 0 || K <= 0 || (K & 7) || (lda & 7) || (ldb & 7)) return hipErrorInvalidValue;
  // 32-bit buffer offsets: one 16-row weight tile and the X rows
  if (static_cast<int64_t>(16) * ldb * 2 >= (int64_t(1) << 32) || static_cast<int64_t>(8) * lda * 2 >= (int64_t(1) << 32))
    return hipErrorInvalidValue;
  const int tiles = (N + 15) / 16;
  GemvSplit sp;
  sp.S = gemv_ksplit(epi, N, K);
  sp.nrows = epi == kEpiSwiGLU ? 2 * N : N;
  sp.part = part;
  sp.ctr = ctr;
  if (sp.S > 1 && (!part || !ctr || ctr_count < tiles ||
                   part_bytes < size_t(sp.S) * M * sp.nrows * sizeof(float)))
    sp.S = 1;   // no room for the split: stream the whole K per tile
  const int grid = tiles * sp.S;
  switch (epi) {
    case kEpiBf16: gemv_kernel<kEpiBf16, 1><<<grid, kThreads, 0, s>>>(A, lda, B, ldb, C, ldc, M, N, K, sp); break;
    case kEpiAddF32: gemv_kernel<kEpiAddF32, 1><<<grid, kThreads, 0, s>>>(A, lda, B, ldb, C, ldc, M, N, K, sp); break;
    case kEpiF32: gemv_kernel<kEpiF32, 1><<<grid, kThreads, 0, s>>>(A, lda, B, ldb, C, ldc, M, N, K, sp); break;
    case kEpiSwiGLU: gemv_kernel<kEpiSwiGLU, 2><<<grid, kThreads, 0, s>>>(A, lda, B, ldb, C, ldc, M, N, K, sp); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace pallas
