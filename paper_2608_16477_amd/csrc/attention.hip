// Causal grouped-query attention over the paged KV cache.
//
// Prefill: one workgroup per (sequence, 32-query block, G query heads of one
// KV head) with one wave per query head, so each 64-key K/V tile is read
// from the pool once for the G heads.  G is the GQA group, except that in
// calls with too few query blocks to fill the chip a group of 8 at head_dim
// 128 is split over two 4-wave workgroups, two of which fit on a CU (under
// 224 registers, 74 KB of LDS each).  K and V tiles go from memory straight
// into LDS (buffer_load ... lds); V is read transposed for the PV product.
//
// The score tile is computed transposed, S^T = K Q^T, with
// v_mfma_f32_32x32x16_bf16: a lane then owns one query and
// 16 of its keys per 32-key block, so the online-softmax max and sum are
// register reductions plus one cross-half lane swap, and the rescale of the
// output accumulator is lane-uniform.  O^T = V^T P^T reuses the score
// registers as the B operand; the key order inside each 16-key MFMA step is
// permuted identically on both operands (a sum is order-free), which lets V
// be read from a transposed LDS tile with two 8-byte reads per step.
// Softmax runs in fp32 in the log2 domain (scores scaled by log2(e)/sqrt(d))
// against a reference max that is raised lazily; P is rounded to bf16 for
// the PV product.  The scores of tile j+1 are computed while tile j goes
// through softmax and PV, so MFMA and VALU work of one wave overlap.
//
// Decode: split over keys (64 per workgroup, all query heads of one KV
// head per workgroup), then a combine pass over the splits.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace pallas {

namespace {

constexpr int QB = 32;  // queries per workgroup
constexpr int KB = 64;  // keys per tile
constexpr int kPage = 16;     // tokens per cache page (the only page size the library accepts)
constexpr int KSTR = KB + 1;  // K tile chunk stride, in 16-byte slots
constexpr float kLazyLog2 = 8.f;  // lazy-rescale headroom, log2 units

typedef __attribute__((address_space(3))) void lds_void;

// Swizzle of a V tile row's 16-byte chunks: chunk c of key k sits in slot
// c ^ vswz(k).  The transposed PV reads of one instruction cover 8 keys
// (two groups of 4 consecutive ones) at 4 chunks each; the XOR puts keys
// k..k+3 on 4 different quarters of the 256-byte bank window, so 512 bytes
// read in two passes.
template <int CH>
__device__ __forceinline__ int vswz(int key) { return (4 * (key & 3)) & (CH - 1); }

// ds_read_b64_tr_b16 at byte `off` of an LDS tile: in each 16-lane group,
// lane i receives element i % 4 of the 64-bit words read by lanes i / 4,
// i / 4 + 4, i / 4 + 8 and i / 4 + 12 of the group, in that order.
__device__ __forceinline__ u32x2 lds_read_tr16(const u32x4* tile, uint32_t off) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
  typedef __attribute__((address_space(3))) char lds_char;
  const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)((lds_char*)tile + off));
  return __builtin_bit_cast(u32x2, v);
}

// Row-sum step: acc + lo + hi of a packed bf16 pair (a dot product with ones).
__device__ __forceinline__ float sum_bf2(uint32_t pair, float acc) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pair), ones, acc, false);
}

struct AttnSched {
  int32_t total;
  int32_t split_tiles;           // key tiles per split (split launches)
  int32_t last_block;            // largest absolute query block of the call
};

// Dispatch order of the (query block, head group) workgroups.  Workgroups
// start in linear grid order, each on the first CU of its XCD that frees
// up, so the order decides the balance: a query block's causal key range
// grows with its absolute block index, and ranking every block of every
// sequence by that index, largest first, with the head groups of a block
// consecutive, makes the dispatch longest-job-first over the whole call.
// Rank r is the block B with count(>= B) > r >= count(>= B + 1), where
// count(>= b) sums over sequences the blocks at index b or later; ties go
// in sequence order.
__host__ __device__ __forceinline__ void block_of_rank(const RowMap& rm, const AttnSched& sch, int r, int& s_out,
                                              int& b_out) {
  if (rm.n_seqs == 1) {
    s_out = 0;
    b_out = sch.last_block - r;
    return;
  }
  auto count_ge = [&](int b) {
    int c = 0;
    for (int s = 0; s < rm.n_seqs; ++s) {
      const int f = rm.base_pos[s] / QB, l = (rm.base_pos[s] + rm.cu[s + 1] - rm.cu[s] - 1) / QB;
      c += max(0, l - max(f, b) + 1);
    }
    return c;
  };
  int lo = 0, hi = sch.last_block + 1;   // count_ge(lo) > r >= count_ge(hi)
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (count_ge(mid) > r) lo = mid; else hi = mid;
  }
  int k = r - count_ge(lo + 1), s = 0;
  for (;; ++s) {
    const int f = rm.base_pos[s] / QB, l = (rm.base_pos[s] + rm.cu[s + 1] - rm.cu[s] - 1) / QB;
    if (f <= lo && lo <= l && k-- == 0) break;
  }
  s_out = s;
  b_out = lo;
}

// Full max / sum over the two 32-lane halves of a wave (the two key halves
// of one query in the S^T layout).
__device__ __forceinline__ float xhalf_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xhalf_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// kSplit: the key tiles of a query block are divided over gridDim.z
// workgroups of at most sch.split_tiles tiles each; a workgroup writes its
// unnormalised output, running max and sum to `part`, and
// attn_prefill_combine_kernel merges them.  Used when a call has too few
// query blocks to fill the chip (a 256-token chunk over a long prefix).
template <int D, int G, bool kSplit>
__global__ __launch_bounds__(G * 64, G == 4 ? 2 : 1) void attn_prefill_kernel(AttnParams p, RowMap rm, AttnSched sch,
                                                              float* __restrict__ part) {
  constexpr int CH = D / 8;                   // 16-byte chunks per K/V row
  constexpr int nthreads = G * 64;
  constexpr int RPI = 64 / CH;                // V rows per staging instruction (64 lanes x 16 B)
  constexpr int NV = KB / RPI;                // V staging instructions per tile
  static_assert(CH % G == 0, "each wave issues CH / G of a K tile's chunk loads");
  static_assert(NV % G == 0, "each wave issues NV / G of a V tile's row loads");
  // K tile as [chunk][key] with a chunk stride of KB + 1 slots: the score
  // MFMA reads 32 consecutive keys of one chunk.  V tile as [key][chunk]
  // (whole head rows) with the 16-byte chunk index XORed by vswz(key), read
  // transposed (ds_read_b64_tr_b16) into the PV operand.
  // Two buffers of each as separate arrays, chosen by a compile-time
  // parity, so the compiler can tell a tile loading into one from reads of
  // the other.
  __shared__ __attribute__((aligned(16))) u32x4 Ks0[CH * KSTR];
  __shared__ __attribute__((aligned(16))) u32x4 Ks1[CH * KSTR];
  __shared__ __attribute__((aligned(16))) u32x4 Vs0[KB * CH];
  __shared__ __attribute__((aligned(16))) u32x4 Vs1[KB * CH];
  __shared__ int32_t bts[kMaxPrefillLen / kPage];   // the sequence's block-table entries

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int g = lane >> 5, l32 = lane & 31;
  // Workgroup x is head group x mod (Hq / G), query block of rank
  // x / (Hq / G) (block_of_rank).  Head group y covers query heads
  // [y G, y G + G), all of one KV head (G divides the group size Hq / Hkv).
  const int ngroups = p.Hq / G;
  const int h = (static_cast<int>(blockIdx.x) % ngroups) * G + wave;
  const int kh = __builtin_amdgcn_readfirstlane(h / (p.Hq / p.Hkv));
  int s, qblock;
  block_of_rank(rm, sch, static_cast<int>(blockIdx.x) / ngroups, s, qblock);
  s = __builtin_amdgcn_readfirstlane(s);
  qblock = __builtin_amdgcn_readfirstlane(qblock);
  // Query blocks sit at absolute positions [32 b, 32 b + 32): the rows of
  // sequence s are positions [base, base + len), so with base > 0 (a chunk
  // over earlier chunks) the first block may be partly before the chunk.
  // Aligned blocks keep every key tile but the last wholly visible to
  // every query of the block, and give a query the same key tiles as an
  // undivided prefill would.
  const int base = rm.base_pos[s];
  const int len = rm.cu[s + 1] - rm.cu[s];
  const int q0 = qblock * QB;
  const int row0 = rm.cu[s] - base;   // row of absolute position a: row0 + a
  const int32_t* bt = p.bt + static_cast<int64_t>(s) * p.max_pages;

  const int qpos = q0 + l32;
  const bool qvalid = qpos >= base && qpos < base + len;
  bf16x8 qf[D / 16];
  {
    const uint16_t* qrow = p.q + (static_cast<int64_t>(row0 + (qvalid ? qpos : base)) * p.Hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      u32x4 v = qvalid ? *reinterpret_cast<const u32x4*>(qrow + kk * 16 + g * 8) : u32x4{0, 0, 0, 0};
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  const int kend = min(q0 + QB, base + len);
  const int ntiles_all = (kend + KB - 1) / KB;
  // This workgroup's key tiles [t0, t0 + ntiles).
  const int t0 = kSplit ? static_cast<int>(blockIdx.z) * sch.split_tiles : 0;
  const int ntiles = kSplit ? min(sch.split_tiles, ntiles_all - t0) : ntiles_all;
  // Split record of (row, head, split): D unnormalised outputs, then the
  // log2-domain max and the sum of this split's probabilities (D + 4
  // floats, so records stay 16-byte aligned).
  float* rec = nullptr;
  if (kSplit)
    rec = part + ((static_cast<int64_t>(row0 + (qvalid ? qpos : base)) * p.Hq + h) * gridDim.z + blockIdx.z) * (D + 4);
  if (kSplit && ntiles <= 0) {
    // Nothing of this block's keys falls in this split.
    if (qvalid && g == 0) {
      rec[D] = -INFINITY;
      rec[D + 1] = 0.f;
    }
    return;
  }
  const int kt0 = t0 * KB;
  {
    // This workgroup's block-table entries (keys [kt0, kend)), read once.
    const int pend = min((kt0 + ntiles * KB + kPage - 1) / kPage, (kend + kPage - 1) / kPage);
    for (int i = kt0 / kPage + static_cast<int>(threadIdx.x); i < pend; i += nthreads) bts[i] = bt[i];
    __syncthreads();
  }

  // Keys at or past kend are masked for every query of the block; they read
  // key kend - 1 instead (its table entry is staged, and a finite V row
  // times probability zero adds nothing).  A table entry outside the pool
  // reads page 0 (the K/V store reports such entries).  K and V planes are
  // addressed through buffer descriptors with 32-bit offsets (the host
  // keeps a plane under 4 GiB).
  const int64_t row_stride = static_cast<int64_t>(p.Hkv) * D;
  auto key_off = [&](int pos) -> uint32_t {   // byte offset of key `pos`'s head row in a plane
    const int pc = min(pos, kend - 1);
    int pg = bts[pc >> 4];
    pg = (pg >= 0 && pg < p.num_pages) ? pg : 0;
    return static_cast<uint32_t>((pg * kPage + (pc & (kPage - 1))) * row_stride * 2);
  };
  const uint32_t head_bytes = static_cast<uint32_t>(p.plane_bytes - static_cast<int64_t>(kh) * D * 2);
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.k_plane + kh * D), 0, head_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.v_plane + kh * D), 0, head_bytes, 0x00020000);
  // K tile straight from memory into LDS: instruction c (16-byte chunk c of
  // the head dimension) has lane l load key k0 + l, so its 64 lanes fill
  // the 64 consecutive slots of chunk c.  Each wave issues CH / G of them.
  auto dmaK = [&](u32x4* Kd, int k0) {
    const uint32_t off = key_off(k0 + lane);
#pragma unroll
    for (int i = 0; i < CH / G; ++i) {
      const int ch = wave * (CH / G) + i;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(Kd + ch * KSTR), 16, off + ch * 16, 0, 0, 0);
    }
  };
  // V tile straight into LDS as [key][chunk]: instruction n fills the RPI
  // rows RPI n .. RPI n + RPI - 1 (lane l: row l / CH, slot l % CH, which
  // holds logical chunk (l % CH) ^ vswz(row)).  Each wave issues NV / G.
  const int vrow = lane / CH;   // this lane's row within a staging instruction (RPI n + vrow = vrow mod 4)
  const uint32_t vcoff = static_cast<uint32_t>(((lane % CH) ^ vswz<CH>(vrow)) * 16);
  auto dmaV = [&](u32x4* Vd, int k0) {
#pragma unroll
    for (int i = 0; i < NV / G; ++i) {
      const int n = wave * (NV / G) + i;
      // key_off written out: the host pass of this compiler drops the
      // kernel when the lambda is called inside this loop
      const int pc = min(k0 + n * RPI + vrow, kend - 1);
      int pg = bts[pc >> 4];
      pg = (pg >= 0 && pg < p.num_pages) ? pg : 0;
      const uint32_t off = static_cast<uint32_t>((pg * kPage + (pc & (kPage - 1))) * row_stride * 2) + vcoff;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(Vd + n * 64), 16, off, 0, 0, 0);
    }
  };
  auto barrier = [] { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

  // S^T = K Q^T for one 64-key tile: keys t*32 + [0,32) in st[t].
  auto scores = [&](const u32x4* Ksrc, f32x16 (&st)[2]) {
    const u32x4* Kb = Ksrc + g * KSTR + l32;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const bf16x8 a = __builtin_bit_cast(bf16x8, Kb[kk * 2 * KSTR + t * 32]);
        st[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], kk == 0 ? f32x16{} : st[t], 0, 0, 0);
      }
  };

  f32x16 oacc[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t) oacc[t] = f32x16{};
  // Probabilities are exp2((s - m_ref) c).  m_ref is raised only when a
  // score exceeds it by more than kLazyLog2 / c, so probabilities stay below
  // 2^kLazyLog2 and the accumulator is rescaled only on those tiles.
  // Row sums: this lane's keys, in four running partials (one per packed
  // pair slot of the PV operand), summed over the bf16 probabilities the PV
  // product uses.
  float m_ref = -INFINITY;
  float lsum[4] = {0.f, 0.f, 0.f, 0.f};
  const float c = p.scale_log2;
  const float thr = kLazyLog2 / c;

  // Softmax of one tile in place (st becomes P); returns whether the
  // reference max moved, with the accumulator factor in `alpha`.
  auto softmax = [&](f32x16 (&st)[2], float& alpha) {
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, st[t][r]);
    mx = xhalf_max(mx);
    const bool raise = __builtin_amdgcn_ballot_w64(mx > m_ref + thr) != 0;
    const float m_new = raise ? fmaxf(m_ref, mx) : m_ref;
    const float mc = (m_new == -INFINITY) ? 0.f : m_new * c;
    alpha = raise ? __builtin_amdgcn_exp2f(fmaf(m_ref, c, -mc)) : 1.f;
    m_ref = m_new;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) st[t][r] = __builtin_amdgcn_exp2f(fmaf(st[t][r], c, -mc));
    return raise;
  };
  // PV operand A = V^T[dv][16 keys of step cc] from the [key][chunk] tile:
  // in each 16-lane group, lane j's 64-bit read covers key (4 (lane / 32) +
  // j / 4) at dimensions dv0 + 4 (j % 4) .. + 3 with dv0 = 32 dt + 16 (j16
  // % 2), and the transposed read hands lane j of the group that key
  // quartet's dimension dv0 + j: 4 consecutive keys of one output row.  Two
  // reads (keys + 0 and + 8) give the 8 keys the score registers hold for
  // that lane, in the same order.  Byte offsets within a tile, for cc = 0:
  const int j16 = lane & 15, grp = lane >> 4;
  uint32_t voff[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt) {
    const int key = 4 * g + j16 / 4;
    const int lc = dt * 4 + 2 * (grp & 1) + (j16 & 3) / 2;   // logical 16-byte chunk
    voff[dt] = static_cast<uint32_t>(key * D * 2 + ((lc ^ vswz<CH>(key)) * 16) + (j16 & 1) * 8);
  }
  auto pv = [&](const u32x4* Vsrc, const f32x16 (&st)[2]) {
#pragma unroll
    for (int cc = 0; cc < KB / 16; ++cc) {
      const int t = cc >> 1, base = (cc & 1) * 8;
      u32x4 pk;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pk[e] = pack_bf2(st[t][base + 2 * e], st[t][base + 2 * e + 1]);
        lsum[e] = sum_bf2(pk[e], lsum[e]);
      }
      const bf16x8 pb = __builtin_bit_cast(bf16x8, pk);
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
        const u32x2 l2 = lds_read_tr16(Vsrc, voff[dt] + cc * 16 * D * 2);
        const u32x2 h2 = lds_read_tr16(Vsrc, voff[dt] + (cc * 16 + 8) * D * 2);
        const u32x4 av = {l2.x, l2.y, h2.x, h2.y};
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, av), pb, oacc[dt], 0, 0, 0);
      }
    }
  };
  auto rescale = [&](float alpha) {
#pragma unroll
    for (int t = 0; t < D / 32; ++t) oacc[t] *= alpha;
#pragma unroll
    for (int e = 0; e < 4; ++e) lsum[e] *= alpha;
  };

  // Pipeline: while tile j's softmax runs, tile j+1's scores are computed
  // from its K tile (already in LDS).  K tiles go straight to LDS two tiles
  // ahead, V tiles one tile ahead.
  dmaK(Ks0, kt0);
  dmaV(Vs0, kt0);
  if (ntiles > 1) dmaK(Ks1, kt0 + KB);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  barrier();
  // One pipeline step: scores of tile j+1 into `nxt` while tile j (scores in
  // `cur`, wholly below the diagonal) goes through softmax and PV.  B = j % 2
  // is a template constant: K_j and V_j sit in buffer B, K_{j+1} in 1 - B.
  auto step = [&](auto parity, int j, f32x16 (&cur)[2], f32x16 (&nxt)[2]) {
    constexpr int B = decltype(parity)::value;
    u32x4* Kfree = B == 0 ? Ks0 : Ks1;
    const u32x4* Knext = B == 0 ? Ks1 : Ks0;
    const u32x4* Vcur = B == 0 ? Vs0 : Vs1;
    u32x4* Vnext = B == 0 ? Vs1 : Vs0;
    barrier();   // K_{j+1} and V_j resident; the buffers of K_j and V_{j-1} free
    if (j + 2 < ntiles) dmaK(Kfree, kt0 + (j + 2) * KB);
    dmaV(Vnext, kt0 + (j + 1) * KB);   // j + 1 < ntiles here
    scores(Knext, nxt);
    float alpha;
    if (softmax(cur, alpha)) rescale(alpha);
    pv(Vcur, cur);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // K_{j+2}, V_{j+1} land before the next barrier
  };
  f32x16 sa[2], sb[2];
  scores(Ks0, sa);
  int j = 0;
  for (; j + 2 < ntiles; j += 2) {
    step(std::integral_constant<int, 0>{}, j, sa, sb);
    step(std::integral_constant<int, 1>{}, j + 1, sb, sa);
  }
  if (j + 1 < ntiles) {
    step(std::integral_constant<int, 0>{}, j, sa, sb);
#pragma unroll
    for (int t = 0; t < 2; ++t) sa[t] = sb[t];
  }
  f32x16 (&st)[2] = sa;
  {
    // Last tile: it holds the diagonal and the sequence end (the mask is
    // empty for the last tile of a split before them).
    const int k0 = kt0 + (ntiles - 1) * KB;
    barrier();
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + t * 32 + (r >> 2) * 8 + g * 4 + (r & 3);
        if (key > qpos || key >= kend) st[t][r] = -INFINITY;
      }
    float alpha;
    if (softmax(st, alpha)) rescale(alpha);
    pv(((ntiles - 1) & 1) ? Vs1 : Vs0, st);
  }

  const float l_tot = xhalf_sum((lsum[0] + lsum[1]) + (lsum[2] + lsum[3]));
  if (!qvalid) return;
  if (kSplit) {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int dv = dt * 32 + rg * 8 + g * 4;
        *reinterpret_cast<f32x4*>(rec + dv) =
            f32x4{oacc[dt][rg * 4 + 0], oacc[dt][rg * 4 + 1], oacc[dt][rg * 4 + 2], oacc[dt][rg * 4 + 3]};
      }
    if (g == 0) {
      rec[D] = m_ref == -INFINITY ? -INFINITY : m_ref * c;
      rec[D + 1] = l_tot;
    }
    return;
  }
  const float inv_l = l_tot > 0.f ? 1.f / l_tot : 0.f;
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

// Merge of the split records of prefill attention: for (row, head), with
// M the largest split max, o = sum_j 2^(m_j - M) o_j / sum_j 2^(m_j - M) l_j.
// 32 threads per (row, head), four output dimensions each (D = 128; two
// threads' worth idle at D = 64).
template <int D>
__global__ __launch_bounds__(256) void attn_prefill_combine_kernel(const float* __restrict__ part, int rows,
                                                                   int Hq, int S, uint16_t* __restrict__ o) {
  const int pair = blockIdx.x * 8 + (threadIdx.x >> 5);
  const int t = threadIdx.x & 31;
  if (pair >= rows * Hq) return;
  const float* rec = part + static_cast<int64_t>(pair) * S * (D + 4);
  float M = -INFINITY;
  for (int j = 0; j < S; ++j) M = fmaxf(M, rec[j * (D + 4) + D]);
  f32x4 acc = {};
  float L = 0.f;
  for (int j = 0; j < S; ++j) {
    const float l = rec[j * (D + 4) + D + 1];
    if (!(l > 0.f)) continue;
    const float w = __builtin_amdgcn_exp2f(rec[j * (D + 4) + D] - M);
    L = fmaf(w, l, L);
    if (t * 4 < D) acc += w * *reinterpret_cast<const f32x4*>(rec + j * (D + 4) + t * 4);
  }
  if (t * 4 >= D) return;
  const float inv = L > 0.f ? 1.f / L : 0.f;
  u32x2 w;
  w.x = pack_bf2(acc[0] * inv, acc[1] * inv);
  w.y = pack_bf2(acc[2] * inv, acc[3] * inv);
  *reinterpret_cast<u32x2*>(o + static_cast<int64_t>(pair) * D + t * 4) = w;
}

constexpr int kDecThreads = 256;
constexpr int kDecSplit = 64;   // keys per split
constexpr int kMaxG = 8;
constexpr int kDecMaxSplitsLds = 1024;   // split records staged in LDS by the combine pass

// Decode attention, split over keys: workgroup (split of 64 keys, KV head,
// seq).  Every K and V row of the split and the G query rows are loaded into
// LDS at once (one table read and one 16-byte load per row chunk and
// thread, all in flight together); then scores (4 threads per key, a
// quarter of the head dimension each), the per-head max and sum over the
// split, and PV (each thread a few output dimensions of one head) run from
// LDS.  The partial record per (seq, head, split) is [max, sum, o[0..d)];
// decode_combine merges the splits.
template <int D>
__global__ __launch_bounds__(kDecThreads) void attn_decode_split_kernel(AttnParams p, RowMap rm,
                                                                        float* __restrict__ part,
                                                                        int max_splits) {
  constexpr int CH = D / 8;                        // 16-byte chunks per row
  constexpr int RPP = kDecThreads / CH;            // rows loaded per pass
  constexpr int NPASS = kDecSplit / RPP;           // load passes
  constexpr int KROW = D + 8;                      // padded LDS row (elements)
  constexpr int TPK = kDecThreads / kDecSplit;     // threads per key in the score pass
  constexpr int DPT = D / TPK;                     // dimensions per score thread
  constexpr int OPT = kMaxG * D / kDecThreads;     // PV outputs per thread
  constexpr int TPH = D / OPT;                     // PV threads per head
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kDecSplit * KROW];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[kDecSplit * KROW];
  __shared__ __attribute__((aligned(16))) float qs[kMaxG][D];
  __shared__ float sc[kMaxG][kDecSplit];
  __shared__ float stat[kMaxG][2];
  __shared__ int kok[kDecSplit];
  const int G = p.Hq / p.Hkv;
  const int split = blockIdx.x, kh = blockIdx.y, s = blockIdx.z;
  const int n = rm.base_pos[s];
  const int j0 = split * kDecSplit;
  if (j0 > n) return;
  const int jn = min(n + 1 - j0, kDecSplit);   // keys of this split at positions <= n
  const int row = rm.cu[s];
  const int32_t* bt = p.bt + static_cast<int64_t>(s) * p.max_pages;
  const int t = threadIdx.x;

  {
    // Keys past jn read key jn - 1 (their scores are masked); rows on a page
    // outside the pool load zeros and are masked.
    const int ch = t % CH, r0 = t / CH;
    u32x4 kv[NPASS], vv[NPASS];
    bool ok[NPASS];
#pragma unroll
    for (int i = 0; i < NPASS; ++i) {
      const int j = j0 + min(r0 + i * RPP, jn - 1);
      const int pg = bt[j / p.page];
      ok[i] = pg >= 0 && pg < p.num_pages;
      const int64_t off = ((static_cast<int64_t>(ok[i] ? pg : 0) * p.page + j % p.page) * p.Hkv + kh) * D + ch * 8;
      kv[i] = ok[i] ? *reinterpret_cast<const u32x4*>(p.k_plane + off) : u32x4{0, 0, 0, 0};
      vv[i] = ok[i] ? *reinterpret_cast<const u32x4*>(p.v_plane + off) : u32x4{0, 0, 0, 0};
    }
    const int qg = t / CH;
    u32x4 qv = {0, 0, 0, 0};
    if (qg < G) qv = *reinterpret_cast<const u32x4*>(p.q + (static_cast<int64_t>(row) * p.Hq + kh * G + qg) * D + ch * 8);
#pragma unroll
    for (int i = 0; i < NPASS; ++i) {
      const int r = r0 + i * RPP;
      *reinterpret_cast<u32x4*>(&Ks[r * KROW + ch * 8]) = kv[i];
      *reinterpret_cast<u32x4*>(&Vs[r * KROW + ch * 8]) = vv[i];
      if (ch == 0) kok[r] = ok[i] && r < jn;
    }
    if (qg < kMaxG) {
      float4* qd = reinterpret_cast<float4*>(&qs[qg][ch * 8]);
      qd[0] = float4{bflo(qv[0]), bfhi(qv[0]), bflo(qv[1]), bfhi(qv[1])};
      qd[1] = float4{bflo(qv[2]), bfhi(qv[2]), bflo(qv[3]), bfhi(qv[3])};
    }
  }
  __syncthreads();

  {
    // Scores: thread (key, part of the head dimension).
    const int key = t / TPK, qt = t % TPK;
    float acc[kMaxG];
#pragma unroll
    for (int g = 0; g < kMaxG; ++g) acc[g] = 0.f;
    const uint16_t* kr = &Ks[key * KROW + qt * DPT];
#pragma unroll
    for (int c = 0; c < DPT / 8; ++c) {
      const u32x4 w = *reinterpret_cast<const u32x4*>(kr + c * 8);
      float kf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        kf[2 * e] = bflo(w[e]);
        kf[2 * e + 1] = bfhi(w[e]);
      }
#pragma unroll
      for (int g = 0; g < kMaxG; ++g) {
        if (g < G) {
          const float4* q4 = reinterpret_cast<const float4*>(&qs[g][qt * DPT + c * 8]);
          const float4 a = q4[0], b = q4[1];
          acc[g] += a.x * kf[0] + a.y * kf[1] + a.z * kf[2] + a.w * kf[3] +
                    b.x * kf[4] + b.y * kf[5] + b.z * kf[6] + b.w * kf[7];
        }
      }
    }
    static_assert(TPK == 4, "a key's score threads are one quad");
#pragma unroll
    for (int g = 0; g < kMaxG; ++g) acc[g] = quad_sum(acc[g]);
    if (qt == 0) {
      const bool valid = kok[key] != 0;
#pragma unroll
      for (int g = 0; g < kMaxG; ++g)
        if (g < G) sc[g][key] = valid ? acc[g] * p.scale_log2 : -INFINITY;
    }
  }
  __syncthreads();
  {
    // Per-head max and sum over the split: wave w owns heads w, w + 4.
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6), lane = t & 63;
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
  {
    // PV: thread (head g, OPT consecutive output dimensions).
    const int g = t / TPH, dv0 = (t % TPH) * OPT;
    if (g >= G) return;
    float o[OPT];
#pragma unroll
    for (int e = 0; e < OPT; ++e) o[e] = 0.f;
    for (int key = 0; key < jn; ++key) {
      const float pw = sc[g][key];
      const uint16_t* vr = &Vs[key * KROW + dv0];
      if constexpr (OPT == 4) {
        const u32x2 v = *reinterpret_cast<const u32x2*>(vr);
        o[0] += pw * bflo(v.x);
        o[1] += pw * bfhi(v.x);
        o[2] += pw * bflo(v.y);
        o[3] += pw * bfhi(v.y);
      } else {
        const uint32_t v = *reinterpret_cast<const uint32_t*>(vr);
        o[0] += pw * bflo(v);
        o[OPT - 1] += pw * bfhi(v);
      }
    }
    float* rec = part + ((static_cast<int64_t>(s) * p.Hq + kh * G + g) * max_splits + split) * (D + 2);
#pragma unroll
    for (int e = 0; e < OPT; ++e) rec[2 + dv0 + e] = o[e];
    if (dv0 == 0) {
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
  // Global max over the splits' maxima, then one weighted pass; records are
  // read sixteen at a time so their loads overlap.
  __shared__ float ms[kDecMaxSplitsLds];
  __shared__ float ls[kDecMaxSplitsLds];
  for (int k = threadIdx.x; k < nsplit; k += D) {
    ms[k] = base[static_cast<int64_t>(k) * (D + 2)];
    ls[k] = base[static_cast<int64_t>(k) * (D + 2) + 1];
  }
  __syncthreads();
  float m = -INFINITY;
  for (int k = 0; k < nsplit; ++k) m = fmaxf(m, ms[k]);
  float l = 0.f, o = 0.f;
  if (m != -INFINITY) {
    constexpr int U = 16;
    for (int k0 = 0; k0 < nsplit; k0 += U) {
      float ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        ok[u] = k0 + u < nsplit ? base[static_cast<int64_t>(k0 + u) * (D + 2) + 2 + threadIdx.x] : 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (k0 + u < nsplit) {
          const float w = exp2f(ms[k0 + u] - m);   // a split with no valid key: max -inf, weight 0
          l += w * ls[k0 + u];
          o += w * ok[u];
        }
      }
    }
  }
  p.o[(static_cast<int64_t>(rm.cu[s]) * p.Hq + h) * D + threadIdx.x] = f2bf(l > 0.f ? o / l : 0.f);
}

}  // namespace

hipError_t launch_attention_prefill(const AttnParams& p, const RowMap& rm, float* part, size_t part_bytes,
                                   hipStream_t s) {
  AttnSched sch;
  sch.total = 0;
  int maxlen = 0;
  for (int i = 0; i < rm.n_seqs; ++i) {
    const int len = rm.cu[i + 1] - rm.cu[i], base = rm.base_pos[i];
    if (len < 1 || base < 0) return hipErrorInvalidValue;
    maxlen = std::max(maxlen, base + len);
    sch.total += (base + len + QB - 1) / QB - base / QB;
  }
  if (sch.total == 0) return hipSuccess;
  sch.last_block = (maxlen - 1) / QB;
  // Query heads per workgroup: the whole GQA group, except that a group of
  // 8 at head_dim 128 is split over two 4-wave workgroups (two of which fit
  // on a CU) when the call has fewer than 512 (query block, KV head) pairs,
  // too few to fill the chip twice.  Measured on one box: a 256-token chunk
  // over a 3000-token prefix runs its attention 20% faster split, while a
  // 3000-token prefill (752 pairs) runs 1% slower split.
  const int group = p.Hq / p.Hkv;
  const int G = (group == 8 && p.d == 128 && sch.total * p.Hkv < 512) ? 4 : group;
  if (maxlen > kMaxPrefillLen || p.page != kPage) return hipErrorInvalidValue;
  const int rows = rm.cu[rm.n_seqs];
  const int S = attn_prefill_splits(rows, sch.total * (p.Hq / G), (maxlen + KB - 1) / KB);
  sch.split_tiles = (((maxlen + KB - 1) / KB) + S - 1) / S;
  if (S > 1 && (!part || part_bytes < attn_prefill_split_bytes(rows, p.Hq, p.d)))
    return hipErrorInvalidValue;
  dim3 grid(sch.total * (p.Hq / G), 1, S);
#define PALLAS_ATTN_CASE(DD, GG)                                                                 \
  if (p.d == DD && G == GG) {                                                                    \
    if (S == 1) {                                                                                \
      attn_prefill_kernel<DD, GG, false><<<grid, GG * 64, 0, s>>>(p, rm, sch, nullptr);          \
      return hipGetLastError();                                                                  \
    }                                                                                            \
    attn_prefill_kernel<DD, GG, true><<<grid, GG * 64, 0, s>>>(p, rm, sch, part);                \
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;                             \
    attn_prefill_combine_kernel<DD><<<(rows * p.Hq + 7) / 8, 256, 0, s>>>(part, rows, p.Hq, S, p.o); \
    return hipGetLastError();                                                                    \
  }
  PALLAS_ATTN_CASE(128, 1) PALLAS_ATTN_CASE(128, 2) PALLAS_ATTN_CASE(128, 4) PALLAS_ATTN_CASE(128, 8)
  PALLAS_ATTN_CASE(64, 1) PALLAS_ATTN_CASE(64, 2) PALLAS_ATTN_CASE(64, 4) PALLAS_ATTN_CASE(64, 8)
#undef PALLAS_ATTN_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_attention_decode(const AttnParams& p, const RowMap& rm, float* partial,
                                   int max_splits, hipStream_t s) {
  int nmax = 0;
  for (int i = 0; i < rm.n_seqs; ++i) {
    if (rm.base_pos[i] < 0) return hipErrorInvalidValue;
    nmax = std::max(nmax, rm.base_pos[i]);
  }
  const int splits = nmax / kDecSplit + 1;
  if (splits > max_splits || splits > kDecMaxSplitsLds || p.Hq / p.Hkv > kMaxG) return hipErrorInvalidValue;
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
