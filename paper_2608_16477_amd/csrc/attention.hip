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
// Decode: split over keys (64 per workgroup, all query heads of one KV
// head per workgroup), then a combine pass over the splits.
#include <algorithm>

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

template <int D, int G>
__global__ __launch_bounds__(G * 64) void attn_prefill_kernel(AttnParams p, RowMap rm, AttnSched sch) {
  constexpr int CH = D / 8;                   // 16-byte chunks per K/V row
  constexpr int ITEMS = (KB / 2) * CH;        // (key pair, chunk) staging items per tile
  constexpr int VROW = KB + VPAD;
  constexpr int nthreads = G * 64;
  constexpr int MAXIT = (ITEMS + nthreads - 1) / nthreads;
  __shared__ __attribute__((aligned(16))) u32x4 Ks[2][KB * CH];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[2][D * VROW];

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
  float m_run = -INFINITY, l_run = 0.f;   // running max of raw scores; running sum

  const int kend = min(q0 + QB, len);
  const int ntiles = (kend + KB - 1) / KB;
  // Staging registers: each thread owns MAXIT (key pair, chunk) items.
  u32x4 sk[MAXIT][2], sv[MAXIT][2];

  auto gload = [&](int k0) {
#pragma unroll
    for (int r = 0; r < MAXIT; ++r) {
      const int it = threadIdx.x + r * nthreads;
      if (it >= ITEMS) break;
      const int ch = it % CH, kp = it / CH;  // chunk fastest: lanes read whole head rows
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int pos = k0 + 2 * kp + e;
        sk[r][e] = u32x4{0, 0, 0, 0};
        sv[r][e] = u32x4{0, 0, 0, 0};
        if (pos < len) {
          const int pg = bt[pos / p.page];
          if (pg >= 0 && pg < p.num_pages) {
            const int64_t off = ((static_cast<int64_t>(pg) * p.page + pos % p.page) * p.Hkv + kh) * D + ch * 8;
            sk[r][e] = *reinterpret_cast<const u32x4*>(p.k_plane + off);
            sv[r][e] = *reinterpret_cast<const u32x4*>(p.v_plane + off);
          }
        }
      }
    }
  };
  auto swrite = [&](int buf) {
#pragma unroll
    for (int r = 0; r < MAXIT; ++r) {
      const int it = threadIdx.x + r * nthreads;
      if (it >= ITEMS) break;
      const int ch = it % CH, kp = it / CH;  // chunk fastest: lanes read whole head rows
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int key = 2 * kp + e;
        Ks[buf][key * CH + kswz<D>(key, ch)] = sk[r][e];
      }
      // Vt[dv][key]: keys (2kp, 2kp+1) packed per dv of this chunk
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t a = sv[r][0][e], b = sv[r][1][e];
        *reinterpret_cast<uint32_t*>(&Vt[buf][(ch * 8 + 2 * e) * VROW + 2 * kp]) = (a & 0xFFFFu) | (b << 16);
        *reinterpret_cast<uint32_t*>(&Vt[buf][(ch * 8 + 2 * e + 1) * VROW + 2 * kp]) = (a >> 16) | (b & 0xFFFF0000u);
      }
    }
  };

  if (ntiles > 0) {
    gload(0);
    swrite(0);
    if (ntiles > 1) gload(KB);
  }
  const float c = p.scale_log2;
  for (int kt = 0; kt < ntiles; ++kt) {
    const int buf = kt & 1;
    const int k0 = kt * KB;
    __syncthreads();  // tile kt resident; buffer buf^1 free
    const u32x4* Kb = Ks[buf];
    const uint16_t* Vb = Vt[buf];

    // S^T for keys k0 + [0,32) and k0 + [32,64)
    f32x16 st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      st[t] = f32x16{};
      const int key = t * 32 + l32;
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        const bf16x8 a = __builtin_bit_cast(bf16x8, Kb[key * CH + kswz<D>(key, kk * 2 + g)]);
        st[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], st[t], 0, 0, 0);
      }
    }
    // Masks only where the tile reaches the diagonal or the sequence end.
    if (k0 + KB - 1 > q0 || k0 + KB > len) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + t * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
          if (key > qpos || key >= len) st[t][r] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, st[t][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float mc = (m_new == -INFINITY) ? 0.f : m_new * c;
    const float alpha = __builtin_amdgcn_exp2f(fmaf(m_run, c, -mc));
    float rs = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = __builtin_amdgcn_exp2f(fmaf(st[t][r], c, -mc));
        st[t][r] = e;
        rs += e;
      }
    rs += __shfl_xor(rs, 32, 64);
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < D / 32; ++t) oacc[t] *= alpha;

#pragma unroll
    for (int cc = 0; cc < KB / 16; ++cc) {
      const int t = cc >> 1, base = (cc & 1) * 8;
      u32x4 pk;
#pragma unroll
      for (int e = 0; e < 4; ++e) pk[e] = pack_bf2(st[t][base + 2 * e], st[t][base + 2 * e + 1]);
      const bf16x8 pb = __builtin_bit_cast(bf16x8, pk);
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
        const uint16_t* vrow = &Vb[(dt * 32 + l32) * VROW + cc * 16 + g * 4];
        const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + 8);
        const u32x4 av = {lo.x, lo.y, hi.x, hi.y};
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, av), pb,
                                                           oacc[dt], 0, 0, 0);
      }
    }
    // Stage tile kt+1 (loaded during this tile) and start loading kt+2.
    if (kt + 1 < ntiles) {
      swrite(buf ^ 1);
      if (kt + 2 < ntiles) gload((kt + 2) * KB);
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
constexpr int kDecSplit = 64;   // keys per split
constexpr int kMaxG = 8;

// Decode attention, split over keys: workgroup (split of 64 keys, KV head,
// seq) scores its keys for all G query heads of the KV head (4 threads per
// key, each over a quarter of the head dimension, so every K row is read
// once), keeps the split's max, sum and unnormalised output per head in the
// partial buffer; decode_combine merges the splits.
template <int D>
__global__ __launch_bounds__(kDecThreads) void attn_decode_split_kernel(AttnParams p, RowMap rm,
                                                                        float* __restrict__ part,
                                                                        int max_splits) {
  constexpr int TPK = kDecThreads / kDecSplit;  // threads per key (4)
  constexpr int DPT = D / TPK;                  // dimensions per thread
  constexpr int NG = kDecThreads / D;           // key groups in the PV pass
  constexpr int KPG = kDecSplit / NG;           // keys per group
  __shared__ float qs[kMaxG][D];
  __shared__ float sc[kMaxG][kDecSplit];
  __shared__ float stat[kMaxG][2];
  __shared__ float oacc[NG][kMaxG][D];
  const int G = p.Hq / p.Hkv;
  const int split = blockIdx.x, kh = blockIdx.y, s = blockIdx.z;
  const int n = rm.base_pos[s];
  const int j0 = split * kDecSplit;
  if (j0 > n) return;
  const int jn = min(n + 1 - j0, kDecSplit);
  const int row = rm.cu[s];
  const int32_t* bt = p.bt + static_cast<int64_t>(s) * p.max_pages;
  for (int i = threadIdx.x; i < G * D; i += kDecThreads)
    qs[i / D][i % D] = bf2f(p.q[(static_cast<int64_t>(row) * p.Hq + kh * G + i / D) * D + i % D]);
  __syncthreads();

  // Scores: thread (key, quarter).
  const int key = threadIdx.x / TPK, qt = threadIdx.x % TPK;
  float acc[kMaxG];
#pragma unroll
  for (int g = 0; g < kMaxG; ++g) acc[g] = 0.f;
  bool valid = false;
  if (key < jn) {
    const int j = j0 + key;
    const int pg = bt[j / p.page];
    if (pg >= 0 && pg < p.num_pages) {
      valid = true;
      const uint16_t* k = p.k_plane + ((static_cast<int64_t>(pg) * p.page + j % p.page) * p.Hkv + kh) * D + qt * DPT;
      u32x4 w[DPT / 8];
#pragma unroll
      for (int c = 0; c < DPT / 8; ++c) w[c] = *reinterpret_cast<const u32x4*>(k + c * 8);
#pragma unroll
      for (int c = 0; c < DPT / 8; ++c) {
        float kf[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          kf[2 * e] = bflo(w[c][e]);
          kf[2 * e + 1] = bfhi(w[c][e]);
        }
#pragma unroll
        for (int g = 0; g < kMaxG; ++g) {
          if (g < G) {
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[g] += qs[g][qt * DPT + c * 8 + e] * kf[e];
          }
        }
      }
    }
  }
#pragma unroll
  for (int g = 0; g < kMaxG; ++g) {
    acc[g] += __shfl_xor(acc[g], 1, kWave);
    acc[g] += __shfl_xor(acc[g], 2, kWave);
  }
  if (qt == 0 && key < kDecSplit) {
#pragma unroll
    for (int g = 0; g < kMaxG; ++g)
      if (g < G) sc[g][key] = valid ? acc[g] * p.scale_log2 : -INFINITY;
  }
  __syncthreads();
  // Per-head max and sum over the split: wave w owns heads w, w + 4.
  {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    for (int g = wave; g < G; g += kDecThreads / 64) {
      const float v = sc[g][lane];
      const float m = wave_max(v);
      const float e = (m == -INFINITY) ? 0.f : exp2f(v - m);
      sc[g][lane] = e;
      const float l = wave_sum(e);
      if (lane == 0) {
        stat[g][0] = m;
        stat[g][1] = l;
      }
    }
  }
  __syncthreads();
  // Weighted sum of V: thread (dim dv, key group kg), eight V loads in flight.
  const int dv = threadIdx.x % D, kg = threadIdx.x / D;
  float o[kMaxG];
#pragma unroll
  for (int g = 0; g < kMaxG; ++g) o[g] = 0.f;
#pragma unroll
  for (int jb = 0; jb < KPG; jb += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int jj = kg * KPG + jb + u;
      v[u] = 0.f;
      if (jj < jn) {
        const int j = j0 + jj;
        const int pg = bt[j / p.page];
        if (pg >= 0 && pg < p.num_pages)
          v[u] = bf2f(p.v_plane[((static_cast<int64_t>(pg) * p.page + j % p.page) * p.Hkv + kh) * D + dv]);
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int jj = kg * KPG + jb + u;
#pragma unroll
      for (int g = 0; g < kMaxG; ++g)
        if (g < G) o[g] += sc[g][jj] * v[u];
    }
  }
#pragma unroll
  for (int g = 0; g < kMaxG; ++g)
    if (g < G) oacc[kg][g][dv] = o[g];
  __syncthreads();
  // partial record per (seq, head, split): [max, sum, o[0..D)]
  for (int i = threadIdx.x; i < G * D; i += kDecThreads) {
    const int g = i / D, e = i % D;
    float t = 0.f;
#pragma unroll
    for (int q = 0; q < NG; ++q) t += oacc[q][g][e];
    float* rec = part + ((static_cast<int64_t>(s) * p.Hq + kh * G + g) * max_splits + split) * (D + 2);
    rec[2 + e] = t;
    if (e == 0) {
      rec[0] = stat[g][0];
      rec[1] = stat[g][1];
    }
  }
}

template <int D>
__global__ __launch_bounds__(D) void attn_decode_combine_kernel(AttnParams p, RowMap rm,
                                                                const float* __restrict__ part,
                                                                int max_splits) {
  const int h = blockIdx.x, s = blockIdx.y;
  const int n = rm.base_pos[s];
  const int nsplit = n / kDecSplit + 1;
  const float* base = part + (static_cast<int64_t>(s) * p.Hq + h) * max_splits * (D + 2);
  // Online merge, eight split records per round so their loads overlap.
  constexpr int U = 8;
  float m = -INFINITY, l = 0.f, o = 0.f;
  for (int k0 = 0; k0 < nsplit; k0 += U) {
    float mk[U], lk[U], ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = k0 + u;
      mk[u] = -INFINITY;
      lk[u] = 0.f;
      ok[u] = 0.f;
      if (k < nsplit) {
        const float* rec = base + static_cast<int64_t>(k) * (D + 2);
        mk[u] = rec[0];
        lk[u] = rec[1];
        ok[u] = rec[2 + threadIdx.x];
      }
    }
    float mg = m;
#pragma unroll
    for (int u = 0; u < U; ++u) mg = fmaxf(mg, mk[u]);
    if (mg == -INFINITY) continue;
    const float sc = exp2f(m - mg);   // m = -inf -> 0
    l *= sc;
    o *= sc;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float w = exp2f(mk[u] - mg);
      l += w * lk[u];
      o += w * ok[u];
    }
    m = mg;
  }
  p.o[(static_cast<int64_t>(rm.cu[s]) * p.Hq + h) * D + threadIdx.x] = f2bf(l > 0.f ? o / l : 0.f);
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
#define PALLAS_ATTN_CASE(DD, GG) \
  if (p.d == DD && G == GG) { attn_prefill_kernel<DD, GG><<<grid, GG * 64, 0, s>>>(p, rm, sch); return hipGetLastError(); }
  PALLAS_ATTN_CASE(128, 1) PALLAS_ATTN_CASE(128, 2) PALLAS_ATTN_CASE(128, 4) PALLAS_ATTN_CASE(128, 8)
  PALLAS_ATTN_CASE(64, 1) PALLAS_ATTN_CASE(64, 2) PALLAS_ATTN_CASE(64, 4) PALLAS_ATTN_CASE(64, 8)
#undef PALLAS_ATTN_CASE
  return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attention_decode(const AttnParams& p, const RowMap& rm, float* partial,
                                   int max_splits, hipStream_t s) {
  int nmax = 0;
  for (int i = 0; i < rm.n_seqs; ++i) {
    if (rm.base_pos[i] < 0) return hipErrorInvalidValue;
    nmax = std::max(nmax, rm.base_pos[i]);
  }
  const int splits = nmax / kDecSplit + 1;
  if (splits > max_splits || p.Hq / p.Hkv > kMaxG) return hipErrorInvalidValue;
  dim3 grid(splits, p.Hkv, rm.n_seqs);
  dim3 cgrid(p.Hq, rm.n_seqs);
  if (p.d == 128) {
    attn_decode_split_kernel<128><<<grid, kDecThreads, 0, s>>>(p, rm, partial, max_splits);
    attn_decode_combine_kernel<128><<<cgrid, 128, 0, s>>>(p, rm, partial, max_splits);
  } else if (p.d == 64) {
    attn_decode_split_kernel<64><<<grid, kDecThreads, 0, s>>>(p, rm, partial, max_splits);
    attn_decode_combine_kernel<64><<<cgrid, 64, 0, s>>>(p, rm, partial, max_splits);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace pallas
