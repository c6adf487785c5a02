// Q/K/V epilogue of the fused projection: optional per-head RMSNorm of Q and
// K over the head dimension, rotary embedding at the row's absolute
// position, and the paged store of K and V:
//   pool[K|V][bt[seq][pos / page]][pos % page][kv_head][:]
// (K after rotary; V copied bit for bit).  Q goes to a [rows][Hq][d]
// buffer for the attention kernel.
//
// One wave per (row, head).  Lane i < d/2 holds the rotary pair (i, i+d/2),
// so the norm is one wave sum and the rotation is lane-local.
#include "common.h"
#include "kernels.h"

namespace pallas {

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void qkv_rope_kernel(QkvParams p, RowMap rm, int rows,
                                                            int heads) {
  const int wave_id = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (wave_id >= rows * heads) return;
  const int lane = threadIdx.x & 63;
  const int row = wave_id / heads;
  const int hh = wave_id - row * heads + (p.kv_only ? p.Hq : 0);  // head in [0, Hq + 2 Hkv)
  const int half = p.d >> 1;
  const bool active = lane < half;
  const int i = active ? lane : 0;

  const int col0 = (p.kv_only ? hh - p.Hq : hh) * p.d;
  const uint16_t* src = p.qkv + static_cast<int64_t>(row) * p.qkv_ld + col0;
  const uint16_t b0 = src[i], b1 = src[i + half];

  const bool is_q = hh < p.Hq;
  const bool is_k = !is_q && hh < p.Hq + p.Hkv;
  uint16_t o0 = b0, o1 = b1;
  if (is_q || is_k) {
    float x0 = bf2f(b0), x1 = bf2f(b1);
    if (p.qk_norm) {
      const float ss = wave_sum(active ? x0 * x0 + x1 * x1 : 0.f);
      const float inv = rsqrtf(ss / p.d + p.eps);
      const uint16_t* g = is_q ? p.q_gain : p.k_gain;
      x0 = x0 * inv * bf2f(g[i]);
      x1 = x1 * inv * bf2f(g[i + half]);
    }
    const float cs = p.rope[(static_cast<int64_t>(row) * half + i) * 2];
    const float sn = p.rope[(static_cast<int64_t>(row) * half + i) * 2 + 1];
    o0 = f2bf(x0 * cs - x1 * sn);
    o1 = f2bf(x1 * cs + x0 * sn);
  }
  if (!active) return;
  if (is_q) {
    uint16_t* dst = p.q_out + (static_cast<int64_t>(row) * p.Hq + hh) * p.d;
    dst[i] = o0;
    dst[i + half] = o1;
    return;
  }
  const int s = row_seq(rm, row);
  const int pos = rm.base_pos[s] + (row - rm.cu[s]);
  const int pg = p.bt[static_cast<int64_t>(s) * p.max_pages + pos / p.page];
  if (pg < 0 || pg >= p.num_pages) {
    if (lane == 0 && p.err) atomicOr(p.err, static_cast<int32_t>(PALLAS_DEVERR_PAGE));
    return;
  }
  const int kh = is_k ? hh - p.Hq : hh - p.Hq - p.Hkv;
  uint16_t* plane = is_k ? p.k_plane : p.v_plane;
  uint16_t* dst = plane + ((static_cast<int64_t>(pg) * p.page + pos % p.page) * p.Hkv + kh) * p.d;
  dst[i] = o0;
  dst[i + half] = o1;
}

}  // namespace

hipError_t launch_qkv_rope(const QkvParams& p, const RowMap& rm, int rows, hipStream_t s) {
  const int heads = p.kv_only ? 2 * p.Hkv : p.Hq + 2 * p.Hkv;
  const int waves = rows * heads;
  if (waves <= 0) return hipSuccess;
  const int per_block = kThreads / 64;
  qkv_rope_kernel<<<(waves + per_block - 1) / per_block, kThreads, 0, s>>>(p, rm, rows, heads);
  return hipGetLastError();
}

}  // namespace pallas
