// Causal grouped-query attention over the paged KV cache.
//
// Prefill: one workgroup per (sequence, 32-query block, KV head) with one
// wave per query head of the group, so each 64-key K/V tile is read from the
// pool once for all G query heads.  The score tile is computed transposed,
// S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: a lane then owns one query and
// 16 of its keys per 32-key block, so the online-softmax max and sum are
// register reductions plus one cross-half shuffle, and the rescale of the
// output accumulator is lane-uniform.  O^T = V^T P^T reuses the score
// registers as the B operand; the key order inside each 16-key MFMA step is
// permuted identically on both operands (a sum is order-free), which lets V
// be read from a transposed LDS tile with two 8-byte reads per step.
// Softmax runs in fp32 in the log2 domain (scores pre-scaled by
// log2(e)/sqrt(d)); P is rounded to bf16 for the PV product.
//
// Decode: one workgroup per (sequence, query head): scores of the n+1 keys
// into LDS, block max and sum, then the weighted sum of V rows.
#include "common.h"
#include "kernels.h"

namespace pallas {

namespace {

constexpr int QB = 32;  // queries per workgroup
constexpr int KB = 64;  // keys per tile
constexpr int VPAD = 4; // Vt row padding (elements): 136-byte rows spread banks

struct AttnSched {
  int32_t total;
  int32_t prefix[kMaxSeqs + 1];  // query blocks before sequence s
};

template <int D>
__device__ __forceinline__ int kswz(int key, int c) {
  return D == 128 ? (c ^ (key & 15)) : (c ^ ((key >> 1) & 7));
}

template <int D>
__global__ __launch_bounds__(512) void attn_prefill_kernel(AttnParams p, RowMap rm, AttnSched sch) {
  constexpr int CH = D / 8;  // 16-byte chunks per K/V row
  __shared__ __attribute__((aligned(16))) u32x4 Ks[KB * CH];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * (KB + VPAD)];

  const int G = p.Hq / p.Hkv;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = lane >> 5, l32 = lane & 31;
  const int kh = blockIdx.y;
  const int h = kh * G + wave;

  const int gidx = sch.total - 1 - static_cast<int>(blockIdx.x);  // longest blocks first
  int s = 0;
  while (s + 1 < rm.n_seqs && sch.prefix[s + 1] <= gidx) ++s;
  const int q0 = (gidx - sch.prefix[s]) * QB;
  const int len = rm.cu[s + 1] - rm.cu[s];
  const int row0 = rm.cu[s];
  const int32_t* bt = p.bt + static_cast<int64_t>(s) * p.max_pages;

  const int qpos = q0 + l32;
  const bool qvalid = qpos < len;
  bf16x8 qf[D / 16];
  {
    const uint16_t* qrow = p.q + (static_cast<int64_t>(row0 + (qvalid ? qpos : 0)) * p.Hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      u32x4 v = qvalid ? *reinterpret_cast<const u32x4*>(qrow + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t) oacc[t] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  const int kend = min(q0 + QB, len);
  const int ntiles = (kend + KB - 1) / KB;
  const int nthreads = G * 64;

  for (int kt = 0; kt < ntiles; ++kt) {
    const int k0 = kt * KB;
    __syncthreads();
    // Stage K (row-major, swizzled) and V (transposed) for keys k0..k0+63.
    for (int it = threadIdx.x; it < (KB / 2) * CH; it += nthreads) {
      const int kp = it % (KB / 2), ch = it / (KB / 2);
      u32x4 kv[2], vv[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int key = 2 * kp + e;
        const int pos = k0 + key;
        kv[e] = u32x4{0, 0, 0, 0};
        vv[e] = u32x4{0, 0, 0, 0};
        if (pos < len) {
          const int pg = bt[pos / p.page];
          if (pg >= 0 && pg < p.num_pages) {
            const int64_t off = ((static_cast<int64_t>(pg) * p.page + pos % p.page) * p.Hkv + kh) * D + ch * 8;
            kv[e] = *reinterpret_cast<const u32x4*>(p.k_plane + off);
            vv[e] = *reinterpret_cast<const u32x4*>(p.v_plane + off);
          }
        }
        Ks[key * CH + kswz<D>(key, ch)] = kv[e];
      }
      // Vt[dv][key]: pack keys (2kp, 2kp+1) for each of the 8 dv of this chunk
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t a = vv[0][e], b = vv[1][e];
        const uint32_t lo = (a & 0xFFFFu) | (b << 16);
        const uint32_t hi = (a >> 16) | (b & 0xFFFF0000u);
        *reinterpret_cast<uint32_t*>(&Vt[(ch * 8 + 2 * e) * (KB + VPAD) + 2 * kp]) = lo;
        *reinterpret_cast<uint32_t*>(&Vt[(ch * 8 + 2 * e + 1) * (KB + VPAD) + 2 * kp]) = hi;
      }
    }
    __syncthreads();

    // S^T for keys k0 + [0,32) and k0 + [32,64)
    f32x16 st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      st[t] = f32x16{};
      const int key = t * 32 + l32;
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        const bf16x8 a = __builtin_bit_cast(bf16x8, Ks[key * CH + kswz<D>(key, kk * 2 + g)]);
        st[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], st[t], 0, 0, 0);
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + t * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
        float v = st[t][r] * p.scale_log2;
        if (key > qpos || key >= len) v = -INFINITY;
        st[t][r] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    float rs = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = exp2f(st[t][r] - m_use);
        st[t][r] = e;
        rs += e;
      }
    rs += __shfl_xor(rs, 32, 64);
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < D / 32; ++t) oacc[t] *= alpha;

#pragma unroll
    for (int c = 0; c < KB / 16; ++c) {
      const int t = c >> 1, base = (c & 1) * 8;
      u32x4 pk;
#pragma unroll
      for (int e = 0; e < 4; ++e) pk[e] = pack_bf2(st[t][base + 2 * e], st[t][base + 2 * e + 1]);
      const bf16x8 pb = __builtin_bit_cast(bf16x8, pk);
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
        const uint16_t* vrow = &Vt[(dt * 32 + l32) * (KB + VPAD) + c * 16 + g * 4];
        const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + 8);
        const u32x4 av = {lo.x, lo.y, hi.x, hi.y};
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, av), pb,
                                                           oacc[dt], 0, 0, 0);
      }
    }
  }

  if (!qvalid) return;
  const float inv_l = l_run > 0.f ? 1.f / l_run : 0.f;
  uint16_t* orow = p.o + (static_cast<int64_t>(row0 + qpos) * p.Hq + h) * D;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int dv = dt * 32 + rg * 8 + g * 4;
      u32x2 w;
      w.x = pack_bf2(oacc[dt][rg * 4 + 0] * inv_l, oacc[dt][rg * 4 + 1] * inv_l);
      w.y = pack_bf2(oacc[dt][rg * 4 + 2] * inv_l, oacc[dt][rg * 4 + 3] * inv_l);
      *reinterpret_cast<u32x2*>(orow + dv) = w;
    }
}

constexpr int kDecThreads = 256;
constexpr int kDecMaxKeys = 16384;

template <int D>
__global__ __launch_bounds__(kDecThreads) void attn_decode_kernel(AttnParams p, RowMap rm) {
  __shared__ float sc[kDecMaxKeys];
  __shared__ float qs[D];
  __shared__ float red[kDecThreads];
  const int s = blockIdx.x / p.Hq, h = blockIdx.x % p.Hq;
  const int G = p.Hq / p.Hkv, kh = h / G;
  const int n = rm.base_pos[s];  // this token's position; keys [0, n]
  const int row = rm.cu[s];
  const int32_t* bt = p.bt + static_cast<int64_t>(s) * p.max_pages;
  const uint16_t* q = p.q + (static_cast<int64_t>(row) * p.Hq + h) * D;
  for (int i = threadIdx.x; i < D; i += kDecThreads) qs[i] = bf2f(q[i]);
  __syncthreads();

  float mx = -INFINITY;
  for (int j = threadIdx.x; j <= n; j += kDecThreads) {
    const int pg = bt[j / p.page];
    float v = -INFINITY;
    if (pg >= 0 && pg < p.num_pages) {
      const uint16_t* k = p.k_plane + ((static_cast<int64_t>(pg) * p.page + j % p.page) * p.Hkv + kh) * D;
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < D / 8; ++c) {
        const u32x4 w = *reinterpret_cast<const u32x4*>(k + c * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          acc += qs[c * 8 + 2 * e] * bflo(w[e]) + qs[c * 8 + 2 * e + 1] * bfhi(w[e]);
      }
      v = acc * p.scale_log2;
    }
    sc[j] = v;
    mx = fmaxf(mx, v);
  }
  mx = wave_max(mx);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float sum = 0.f;
  for (int j = threadIdx.x; j <= n; j += kDecThreads) {
    const float e = exp2f(sc[j] - mx);
    sc[j] = e;
    sum += e;
  }
  sum = wave_sum(sum);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = sum;
  __syncthreads();
  sum = red[0] + red[1] + red[2] + red[3];
  __syncthreads();

  constexpr int NG = kDecThreads / D;  // key groups
  const int dv = threadIdx.x % D, kg = threadIdx.x / D;
  float acc = 0.f;
  for (int j = kg; j <= n; j += NG) {
    const int pg = bt[j / p.page];
    if (pg < 0 || pg >= p.num_pages) continue;
    const uint16_t* v = p.v_plane + ((static_cast<int64_t>(pg) * p.page + j % p.page) * p.Hkv + kh) * D;
    acc += sc[j] * bf2f(v[dv]);
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  if (kg == 0) {
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < NG; ++i) t += red[i * D + dv];
    p.o[(static_cast<int64_t>(row) * p.Hq + h) * D + dv] = f2bf(t / sum);
  }
}

}  // namespace

hipError_t launch_attention_prefill(const AttnParams& p, const RowMap& rm, hipStream_t s) {
  AttnSched sch;
  sch.prefix[0] = 0;
  for (int i = 0; i < rm.n_seqs; ++i) {
    const int len = rm.cu[i + 1] - rm.cu[i];
    sch.prefix[i + 1] = sch.prefix[i] + (len + QB - 1) / QB;
  }
  sch.total = sch.prefix[rm.n_seqs];
  if (sch.total == 0) return hipSuccess;
  const int G = p.Hq / p.Hkv;
  dim3 grid(sch.total, p.Hkv);
  if (p.d == 128)
    attn_prefill_kernel<128><<<grid, G * 64, 0, s>>>(p, rm, sch);
  else if (p.d == 64)
    attn_prefill_kernel<64><<<grid, G * 64, 0, s>>>(p, rm, sch);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attention_decode(const AttnParams& p, const RowMap& rm, hipStream_t s) {
  for (int i = 0; i < rm.n_seqs; ++i)
    if (rm.base_pos[i] < 0 || rm.base_pos[i] >= kDecMaxKeys) return hipErrorInvalidValue;
  const int blocks = rm.n_seqs * p.Hq;
  if (p.d == 128)
    attn_decode_kernel<128><<<blocks, kDecThreads, 0, s>>>(p, rm);
  else if (p.d == 64)
    attn_decode_kernel<64><<<blocks, kDecThreads, 0, s>>>(p, rm);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pallas
