// Q/K/V epilogue of the fused projection: optional per-head RMSNorm of Q and
// K over the head dimension, rotary embedding at the row's absolute
// position, and the paged store of K and V:
//   pool[K|V][bt[seq][pos / page]][pos % page][kv_head][:]
// (K after rotary; V copied bit for bit).  Q goes to a [rows][Hq][d]
// buffer for the attention kernel.
//
// One workgroup per row; each lane handles four rotary pairs of one head.
#include "common.h"
#include "kernels.h"

namespace pallas {

namespace {

constexpr int kThreads = 256;
constexpr int kGroup = 5;   // passes whose loads are in flight together

// One workgroup per row.  A lane owns 4 rotary pairs: elements [4j, 4j+4)
// of the head's first half and their partners [4j+d/2, 4j+d/2+4), loaded as
// 8-byte vectors; d/8 lanes cover a head, so a workgroup works on
// 256 / (d/8) heads at a time and the head norm is a sum over d/8 lanes.
template <int D>
__global__ __launch_bounds__(kThreads) void qkv_rope_kernel(QkvParams p, RowMap rm, int heads) {
  constexpr int LPH = D / 8;            // lanes per head
  constexpr int HPB = kThreads / LPH;   // heads per pass
  constexpr int HALF = D / 2;
  const int row = blockIdx.x;
  const int j = threadIdx.x % LPH;      // pair group: pairs 4j .. 4j+3
  const int hsub = threadIdx.x / LPH;
  const int s = row_seq(rm, row);
  const int pos = rm.base_pos[s] + (row - rm.cu[s]);
  const int pg = p.bt[static_cast<int64_t>(s) * p.max_pages + pos / p.page];
  const bool page_ok = pg >= 0 && pg < p.num_pages;
  const int64_t slot = (static_cast<int64_t>(pg) * p.page + pos % p.page) * p.Hkv;
  const f32x4* rope = reinterpret_cast<const f32x4*>(p.rope + (static_cast<int64_t>(row) * HALF + 4 * j) * 2);
  const f32x4 cs01 = rope[0], cs23 = rope[1];   // (cos, sin) of pairs 4j .. 4j+3
  const float cs[4] = {cs01.x, cs01.z, cs23.x, cs23.z};
  const float sn[4] = {cs01.y, cs01.w, cs23.y, cs23.w};
  const uint16_t* src_row = p.qkv + static_cast<int64_t>(row) * p.qkv_ld;
  bool flagged = false;

  // The loads of kGroup passes are issued before any of their stores (the
  // stores may not alias them, but the compiler cannot know): one memory
  // round trip per group of passes instead of one per pass.
  for (int g0 = 0; g0 < heads; g0 += kGroup * HPB) {
  u32x2 lov[kGroup], hiv[kGroup];
#pragma unroll
  for (int ps = 0; ps < kGroup; ++ps) {
    const int hl = g0 + ps * HPB + hsub;
    lov[ps] = hiv[ps] = u32x2{0, 0};
    if (hl < heads) {
      const uint16_t* src = src_row + static_cast<int64_t>(hl) * D;
      lov[ps] = *reinterpret_cast<const u32x2*>(src + 4 * j);
      hiv[ps] = *reinterpret_cast<const u32x2*>(src + HALF + 4 * j);
    }
  }

#pragma unroll
  for (int ps = 0; ps < kGroup; ++ps) {
    const int hl = g0 + ps * HPB + hsub;        // local head index
    const bool active = hl < heads;
    const int hh = hl + (p.kv_only ? p.Hq : 0); // head in [0, Hq + 2 Hkv)
    const bool is_q = hh < p.Hq;
    const bool is_k = !is_q && hh < p.Hq + p.Hkv;
    const u32x2 lo = lov[ps], hi = hiv[ps];
    float x0[4] = {bflo(lo.x), bfhi(lo.x), bflo(lo.y), bfhi(lo.y)};
    float x1[4] = {bflo(hi.x), bfhi(hi.x), bflo(hi.y), bfhi(hi.y)};
    u32x2 olo = lo, ohi = hi;
    if (is_q || is_k) {
      if (p.qk_norm) {
        float ss = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) ss += x0[e] * x0[e] + x1[e] * x1[e];
        if constexpr (LPH == 16) {
          ss = row16_sum(ss);
        } else {
#pragma unroll
          for (int o = LPH / 2; o > 0; o >>= 1) ss += __shfl_xor(ss, o, kWave);
        }
        const float inv = rsqrtf(ss / D + p.eps);
        const uint16_t* gsrc = is_q ? p.q_gain : p.k_gain;
        const u32x2 g0 = *reinterpret_cast<const u32x2*>(gsrc + 4 * j);
        const u32x2 g1 = *reinterpret_cast<const u32x2*>(gsrc + HALF + 4 * j);
        const float ga[4] = {bflo(g0.x), bfhi(g0.x), bflo(g0.y), bfhi(g0.y)};
        const float gb[4] = {bflo(g1.x), bfhi(g1.x), bflo(g1.y), bfhi(g1.y)};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x0[e] = x0[e] * inv * ga[e];
          x1[e] = x1[e] * inv * gb[e];
        }
      }
      float y0[4], y1[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        y0[e] = x0[e] * cs[e] - x1[e] * sn[e];
        y1[e] = x1[e] * cs[e] + x0[e] * sn[e];
      }
      olo = u32x2{pack_bf2(y0[0], y0[1]), pack_bf2(y0[2], y0[3])};
      ohi = u32x2{pack_bf2(y1[0], y1[1]), pack_bf2(y1[2], y1[3])};
    }
    if (!active) continue;
    uint16_t* dst;
    if (is_q) {
      dst = p.q_out + (static_cast<int64_t>(row) * p.Hq + hh) * D;
    } else {
      if (!page_ok) {
        flagged = true;
        continue;
      }
      const int kh = is_k ? hh - p.Hq : hh - p.Hq - p.Hkv;
      dst = (is_k ? p.k_plane : p.v_plane) + (slot + kh) * D;
    }
    *reinterpret_cast<u32x2*>(dst + 4 * j) = olo;
    *reinterpret_cast<u32x2*>(dst + HALF + 4 * j) = ohi;
  }
  }
  if (flagged && j == 0 && p.err) atomicOr(p.err, static_cast<int32_t>(PALLAS_DEVERR_PAGE));
}

}  // namespace

hipError_t launch_qkv_rope(const QkvParams& p, const RowMap& rm, int rows, hipStream_t s) {
  const int heads = p.kv_only ? 2 * p.Hkv : p.Hq + 2 * p.Hkv;
  if (rows <= 0) return hipSuccess;
  if (p.d == 128)
    qkv_rope_kernel<128><<<rows, kThreads, 0, s>>>(p, rm, heads);
  else if (p.d == 64)
    qkv_rope_kernel<64><<<rows, kThreads, 0, s>>>(p, rm, heads);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pallas
