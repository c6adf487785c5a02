// Skinny GEMM for decode (M <= 8 rows): C = X W^T streaming the weights once.
//
// A workgroup of 8 waves owns two 16-column tiles of W and splits K eight
// ways; each wave runs v_mfma_f32_16x16x32_bf16 with X (rows padded to 16
// with zeros) as the A operand and 16 weight rows, loaded straight from
// memory in operand layout, as the B operand.  The eight partial tiles are
// summed through LDS and the epilogue matches the prefill GEMM's.
#include "common.h"
#include "kernels.h"

namespace pallas {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kUnroll = 4;

template <int EPI>
__global__ __launch_bounds__(kThreads) void gemv_kernel(const uint16_t* __restrict__ X, int ldx,
                                                        const uint16_t* __restrict__ W, int ldw,
                                                        void* __restrict__ C, int ldc, int M, int N,
                                                        int K, int w_rows) {
  __shared__ f32x4 red[kWaves][2][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int li = lane & 15, kg = lane >> 4;
  // weight rows of the two tiles
  int wrow[2];
  if (EPI == kEpiSwiGLU) {
    const int o = blockIdx.x * 16 + li;
    wrow[0] = o < N ? o : -1;
    wrow[1] = o < N ? N + o : -1;
  } else {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int n = blockIdx.x * 32 + t * 16 + li;
      wrow[t] = n < N ? n : -1;
    }
  }
  (void)w_rows;
  const int kslice = ((K + kWaves * 32 - 1) / (kWaves * 32)) * 32;
  const int kb = wave * kslice, ke = min(K, kb + kslice);
  const bool xrow_ok = li < M;
  const uint16_t* xr = X + static_cast<int64_t>(xrow_ok ? li : 0) * ldx;
  const uint16_t* wr0 = W + static_cast<int64_t>(wrow[0] < 0 ? 0 : wrow[0]) * ldw;
  const uint16_t* wr1 = W + static_cast<int64_t>(wrow[1] < 0 ? 0 : wrow[1]) * ldw;

  f32x4 acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0};
  for (int k = kb; k < ke; k += 32 * kUnroll) {
    u32x4 xa[kUnroll], w0[kUnroll], w1[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int kk = k + u * 32 + kg * 8;
      const bool ok = kk < ke;
      xa[u] = (ok && xrow_ok) ? *reinterpret_cast<const u32x4*>(xr + kk) : u32x4{0, 0, 0, 0};
      w0[u] = (ok && wrow[0] >= 0) ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wr0 + kk))
                                   : u32x4{0, 0, 0, 0};
      w1[u] = (ok && wrow[1] >= 0) ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wr1 + kk))
                                   : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, xa[u]);
      acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, w0[u]), acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, w1[u]), acc1, 0, 0, 0);
    }
  }
  red[wave][0][lane] = acc0;
  red[wave][1][lane] = acc1;
  __syncthreads();
  if (wave != 0) return;
  f32x4 s0 = red[0][0][lane], s1 = red[0][1][lane];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) {
    s0 += red[w][0][lane];
    s1 += red[w][1][lane];
  }
  // lane holds column li and rows kg*4 + r
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int m = kg * 4 + r;
    if (m >= M) continue;
    if (EPI == kEpiSwiGLU) {
      const int col = blockIdx.x * 16 + li;
      if (col < N) {
        const float gt = s0[r], up = s1[r];
        static_cast<uint16_t*>(C)[static_cast<int64_t>(m) * ldc + col] = f2bf(gt / (1.0f + __expf(-gt)) * up);
      }
    } else {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int col = blockIdx.x * 32 + t * 16 + li;
        if (col >= N) continue;
        const float v = t == 0 ? s0[r] : s1[r];
        const int64_t at = static_cast<int64_t>(m) * ldc + col;
        if (EPI == kEpiBf16) static_cast<uint16_t*>(C)[at] = f2bf(v);
        else if (EPI == kEpiAddF32) static_cast<float*>(C)[at] += v;
        else static_cast<float*>(C)[at] = v;
      }
    }
  }
}

}  // namespace

hipError_t launch_gemv(int epi, const uint16_t* A, int lda, const uint16_t* B, int ldb, void* C,
                       int ldc, int M, int N, int K, hipStream_t s) {
  if (M <= 0 || M > 8) return hipErrorInvalidValue;
  const int w_rows = epi == kEpiSwiGLU ? 2 * N : N;
  switch (epi) {
    case kEpiBf16: gemv_kernel<kEpiBf16><<<(N + 31) / 32, kThreads, 0, s>>>(A, lda, B, ldb, C, ldc, M, N, K, w_rows); break;
    case kEpiAddF32: gemv_kernel<kEpiAddF32><<<(N + 31) / 32, kThreads, 0, s>>>(A, lda, B, ldb, C, ldc, M, N, K, w_rows); break;
    case kEpiF32: gemv_kernel<kEpiF32><<<(N + 31) / 32, kThreads, 0, s>>>(A, lda, B, ldb, C, ldc, M, N, K, w_rows); break;
    case kEpiSwiGLU: gemv_kernel<kEpiSwiGLU><<<(N + 15) / 16, kThreads, 0, s>>>(A, lda, B, ldb, C, ldc, M, N, K, w_rows); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace pallas
