// Token embedding, RMSNorm and the rotary angle table.
//
// RMSNorm: h = bf16(x * (mean(x^2) + eps)^(-1/2) * g) with x the float32
// residual row; one workgroup per row, float4 loads, a wave64 butterfly sum
// and a cross-wave sum through LDS.  Rows up to 8192 wide are held in
// registers between the two passes.
#include "common.h"
#include "kernels.h"

namespace pallas {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < kThreads / 64; ++i) t += sh[i];
  return t;
}

// Writes h[i..i+3] = bf16(x * inv * g)
__device__ __forceinline__ void store_norm4(uint16_t* h, const uint16_t* g, int i, f32x4 x, float inv) {
  const u32x2 gg = *reinterpret_cast<const u32x2*>(g + i);
  u32x2 out;
  out.x = pack_bf2(x.x * inv * bflo(gg.x), x.y * inv * bfhi(gg.x));
  out.y = pack_bf2(x.z * inv * bflo(gg.y), x.w * inv * bfhi(gg.y));
  *reinterpret_cast<u32x2*>(h + i) = out;
}

__global__ __launch_bounds__(kThreads) void embed_rmsnorm_kernel(
    const int32_t* __restrict__ ids, const uint16_t* __restrict__ E, const uint16_t* __restrict__ g,
    float* __restrict__ r, uint16_t* __restrict__ h, int H, float eps, int vocab, int32_t* err) {
  __shared__ float sh[kThreads / 64];
  const int t = blockIdx.x;
  int id = ids[t];
  if (id < 0 || id >= vocab) {
    if (threadIdx.x == 0 && err) atomicOr(err, static_cast<int32_t>(PALLAS_DEVERR_TOKEN));
    id = 0;
  }
  const uint16_t* e = E + static_cast<int64_t>(id) * H;
  float* rr = r + static_cast<int64_t>(t) * H;
  float ss = 0.f;
  for (int i = threadIdx.x * 4; i < H; i += kThreads * 4) {
    const u32x2 w = *reinterpret_cast<const u32x2*>(e + i);
    const f32x4 x = {bflo(w.x), bfhi(w.x), bflo(w.y), bfhi(w.y)};
    *reinterpret_cast<f32x4*>(rr + i) = x;
    ss += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
  }
  const float inv = rsqrtf(block_sum(ss, sh) / H + eps);
  uint16_t* hh = h + static_cast<int64_t>(t) * H;
  for (int i = threadIdx.x * 4; i < H; i += kThreads * 4) {
    const u32x2 w = *reinterpret_cast<const u32x2*>(e + i);
    const f32x4 x = {bflo(w.x), bfhi(w.x), bflo(w.y), bfhi(w.y)};
    store_norm4(hh, g, i, x, inv);
  }
}

// Rows of up to kRegVecs * kThreads * 4 elements stay in registers between
// the sum of squares and the scaling, so a row is read from memory once.
constexpr int kRegVecs = 8;

__global__ __launch_bounds__(kThreads) void rmsnorm_reg_kernel(const float* __restrict__ r,
                                                               const uint16_t* __restrict__ g,
                                                               uint16_t* __restrict__ h, int H,
                                                               float eps) {
  __shared__ float sh[kThreads / 64];
  const int t = blockIdx.x;
  const float* rr = r + static_cast<int64_t>(t) * H;
  f32x4 x[kRegVecs];
  float ss = 0.f;
#pragma unroll
  for (int v = 0; v < kRegVecs; ++v) {
    const int i = (v * kThreads + threadIdx.x) * 4;
    x[v] = i < H ? *reinterpret_cast<const f32x4*>(rr + i) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int v = 0; v < kRegVecs; ++v) ss += x[v].x * x[v].x + x[v].y * x[v].y + x[v].z * x[v].z + x[v].w * x[v].w;
  const float inv = rsqrtf(block_sum(ss, sh) / H + eps);
  uint16_t* hh = h + static_cast<int64_t>(t) * H;
#pragma unroll
  for (int v = 0; v < kRegVecs; ++v) {
    const int i = (v * kThreads + threadIdx.x) * 4;
    if (i < H) store_norm4(hh, g, i, x[v], inv);
  }
}

__global__ __launch_bounds__(kThreads) void rmsnorm_kernel(const float* __restrict__ r,
                                                           const uint16_t* __restrict__ g,
                                                           uint16_t* __restrict__ h, int H,
                                                           float eps) {
  __shared__ float sh[kThreads / 64];
  const int t = blockIdx.x;
  const float* rr = r + static_cast<int64_t>(t) * H;
  float ss = 0.f;
  for (int i = threadIdx.x * 4; i < H; i += kThreads * 4) {
    const f32x4 x = *reinterpret_cast<const f32x4*>(rr + i);
    ss += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
  }
  const float inv = rsqrtf(block_sum(ss, sh) / H + eps);
  uint16_t* hh = h + static_cast<int64_t>(t) * H;
  for (int i = threadIdx.x * 4; i < H; i += kThreads * 4)
    store_norm4(hh, g, i, *reinterpret_cast<const f32x4*>(rr + i), inv);
}

__global__ void rope_table_kernel(RowMap rm, int rows, int half, double log2_theta_over_half,
                                  float* __restrict__ tab) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * half) return;
  const int t = idx / half, i = idx - t * half;
  const int s = row_seq(rm, t);
  const double pos = double(rm.base_pos[s] + (t - rm.cu[s]));
  // theta^(-2i/d) = 2^(-i * log2(theta) / (d/2))
  const double inv_freq = exp2(-double(i) * log2_theta_over_half);
  double sn, cs;
  sincos(pos * inv_freq, &sn, &cs);
  tab[2 * idx] = static_cast<float>(cs);
  tab[2 * idx + 1] = static_cast<float>(sn);
}

}  // namespace

hipError_t launch_embed_rmsnorm(const int32_t* ids, const uint16_t* embed, const uint16_t* gain,
                                float* r, uint16_t* h, int rows, int H, float eps, int vocab,
                                int32_t* err, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  embed_rmsnorm_kernel<<<rows, kThreads, 0, s>>>(ids, embed, gain, r, h, H, eps, vocab, err);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const float* r, const uint16_t* gain, uint16_t* h, int rows, int H,
                          float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (H <= kRegVecs * kThreads * 4)
    rmsnorm_reg_kernel<<<rows, kThreads, 0, s>>>(r, gain, h, H, eps);
  else
    rmsnorm_kernel<<<rows, kThreads, 0, s>>>(r, gain, h, H, eps);
  return hipGetLastError();
}

hipError_t launch_rope_table(const RowMap& rm, int rows, int d, float theta, float* tab,
                             hipStream_t s) {
  const int half = d / 2;
  const int n = rows * half;
  if (n <= 0) return hipSuccess;
  rope_table_kernel<<<(n + 255) / 256, 256, 0, s>>>(rm, rows, half, log2(double(theta)) / half, tab);
  return hipGetLastError();
}

}  // namespace pallas
