// bf16 GEMM on gfx950 matrix cores: C = A * B^T with both operands K-major
// (activations [M][K], weights [N][K] as stored, [out][in]) and a float32
// accumulator, with the epilogue fused into the store.
//
// Tiling: a 256 x 256 output tile per workgroup of 8 waves (two per SIMD,
// so one wave's barrier and LDS waits overlap the other's MFMAs), each wave
// 128 x 64 as 8 x 4 blocks of v_mfma_f32_16x16x32_bf16.  The 16 x 16 x 32
// shape moves half the accumulator bits per FLOP of the 32 x 32 x 16 one,
// which matters because the chip runs these GEMMs at its power limit: a
// register-only loop of each over all CUs, with random operands, held
// 2.0 GHz and 1.99 PFLOP/s against 1.76 GHz and 1.80 PFLOP/s.  K advances 64 at
// a time through a double-buffered LDS stage (2 x (32 KiB A + 32 KiB B))
// filled by buffer loads that write LDS directly (no register staging);
// one barrier per step.  Step kt+2's loads are issued right after the
// barrier inside step kt that releases kt's slot, so they have a whole
// K-step to land (issued at the top of step kt+1 they had three quarters of
// one, and the loop waited on them).  64-element K-steps make
// every operand row segment a whole 128-byte line, so each L1 miss request
// carries 128 bytes: the kernel is bound by how many misses a CU keeps in
// flight against L2 latency, and full-line requests double the bytes per
// request.  The buffer range check turns rows past M/N and columns past K
// into zeros.
//
// Workgroups are dispatched round-robin over the 8 XCDs; the tile index is
// remapped so each XCD owns a contiguous run of tiles, M-tile fastest, so
// the workgroups sharing one weight panel run on one XCD and share its L2.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace pallas {

namespace {

constexpr int BK = 64;
constexpr int KK = BK / 32;              // MFMA K-substeps per K-step
constexpr int kThreads = 512;
constexpr int kChunks = BK / 8;          // 16-byte chunks per tile row
// Only waves 0-3 (one per SIMD) issue the operand loads: a wave blocked
// on a full L1 miss queue cannot issue MFMAs, and this keeps waves 4-7
// issuing MFMAs on every SIMD.
constexpr int kLoaderWaves = 4;
constexpr int kXcds = 8;
constexpr int kGroupM = 6;

// Tile shapes BM x BN (output rows x B rows), all with 8 waves and the
// same MFMA over the same K order, so an output element gets the same bits
// from any of them (a prefill's rows do not depend on its length):
//   256 x 256: waves 2 x 4, each 128 x 64 (8 x 4 blocks of 16 x 16), a
//              2-deep LDS ring of 64 KiB stages;
//   256 x 128: waves 4 x 2, each 64 x 64; a 3-deep ring of 48 KiB stages,
//              since a half-width step has half the MFMA work to hide its
//              loads behind;
//   192 x 256, 192 x 192, 192 x 128: waves 2 x 4, 2 x 4, 4 x 2, each 96 x 64,
//              96 x 48, 48 x 64; 2, 3 and 4-deep rings (56, 48, 40 KiB
//              stages; the smaller the tile, the less MFMA work a step
//              has to hide its loads behind).
// The 192-row shapes exist for row counts such as 1536 = 8 x 192, where
// 256-row tiles leave CUs idle (gemm_tile).
template <int BM_, int BN_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_;
  static constexpr int WAVES_N = BN_ == 128 ? 2 : 4;
  static constexpr int WAVES_M = 8 / WAVES_N;
  static constexpr int WM = BM_ / WAVES_M;        // rows per wave
  static constexpr int WN = BN_ / WAVES_N;        // B rows (columns) per wave
  static constexpr int IM = WM / 16, JN = WN / 16;
  static constexpr int kSlotsA = BM_ * kChunks, kSlotsB = BN_ * kChunks;   // 16-byte slots
  static constexpr int kStageBytes = (kSlotsA + kSlotsB) * 16;
  static constexpr int kStages = 4 * kStageBytes <= 160 * 1024 ? 4 : 3 * kStageBytes <= 150 * 1024 ? 3 : 2;
  static constexpr int kLoadsA = kSlotsA / (kLoaderWaves * 64);   // per loader thread
  static constexpr int kLoadsB = kSlotsB / (kLoaderWaves * 64);
  static_assert(WM % 16 == 0 && WN % 16 == 0, "whole 16 x 16 blocks per wave");
  static_assert(kLoadsA * kLoaderWaves * 64 == kSlotsA && kLoadsB * kLoaderWaves * 64 == kSlotsB,
                "the loader waves fill the tiles exactly");
};

typedef __attribute__((address_space(3))) void lds_void;

// 128-byte rows: two rows span the 64 banks; XOR the chunk with (row / 2)
// mod 8 so 16 consecutive rows read at one logical chunk hit 16 distinct
// 4-bank groups.
__device__ __forceinline__ int swz(int row, int c) { return row * kChunks + (c ^ ((row >> 1) & 7)); }

// Operand loads into LDS.  A loader wave issues N load instructions per
// operand tile and K-step; instruction i fills slots [(wave*N+i)*64, +64),
// tile rows 8 (wave N + i) + lane / 8.  The lane's chunk swizzle depends on
// i only through its parity, so the lane keeps two offsets, voff[0..1]
// (its row's byte offset plus its chunk's column offset for instructions
// 0 and 1), and instruction i adds the 8 (i - i mod 2) rows past those,
// `step` bytes each, in a vector register computed at the load (16 offsets
// kept live would cost registers that the accumulators need).  The range check thus sees the
// whole row offset: a row past the matrix reads zeros.  Without a K tail
// the step's column offset goes into the scalar offset; with one (K not a
// multiple of BK) each lane checks its column against K.
template <int N, bool kTail>
__device__ __forceinline__ void load_row_lds(__amdgpu_buffer_rsrc_t rsrc, uint32_t limit,
                                             const uint32_t* voff, const int* kcol, uint32_t step,
                                             int k0, int K, u32x4* lds_tile, int wave, int i) {
  lds_void* dst = (lds_void*)(lds_tile + (wave * N + i) * 64);
  const uint32_t vo = voff[i & 1] + static_cast<uint32_t>(i & ~1) * step;
  if (kTail) {
    const uint32_t off = kcol[i & 1] < K - k0 ? vo + static_cast<uint32_t>(k0) * 2u : limit;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, dst, 16, off, 0, 0, 0);
  } else {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, dst, 16, vo, k0 * 2, 0, 0);
  }
}
template <int N, bool kTail>
__device__ __forceinline__ void load_tile_lds(__amdgpu_buffer_rsrc_t rsrc, uint32_t limit,
                                              const uint32_t* voff, const int* kcol, uint32_t step,
                                              int k0, int K, u32x4* lds_tile, int wave) {
#pragma unroll
  for (int i = 0; i < N; ++i) load_row_lds<N, kTail>(rsrc, limit, voff, kcol, step, k0, K, lds_tile, wave, i);
}

template <int BM_, int BN_>
using LdsRing = u32x4[TileCfg<BM_, BN_>::kStages][TileCfg<BM_, BN_>::kSlotsA + TileCfg<BM_, BN_>::kSlotsB];
// ([stage][A slots, B slots])

// How a workgroup finds its work unit.  Workgroups are dealt round-robin
// over the 8 XCDs; XCD x owns the contiguous run of units
// [x tiles_per_xcd, +tiles_per_xcd).  kUnitsPlain: unit = (tile, K split)
// of one width.  kUnitsTailFull / kUnitsTailHalf (gemm_bf16_tail_kernel):
// the last tail_half full tiles of a run are split into two half-width
// units each, which follow the run's full tiles.
enum { kUnitsPlain = 0, kUnitsTailFull = 1, kUnitsTailHalf = 2 };

// One workgroup: its unit, then the output tile (M tile tm, column tile tn
// of BN_ B rows) over its K split, with its LDS ring `lds`.
template <int EPI, int BM_, int BN_, int kUnits>
__device__ __forceinline__ void gemm_workgroup(const GemmParams& p, LdsRing<BM_, BN_>& lds) {
  using T = TileCfg<BM_, BN_>;
  constexpr int BM = T::BM, BN = T::BN, IM = T::IM, JN = T::JN, WM = T::WM, WN = T::WN;
  constexpr int kSlotsA = T::kSlotsA;
  static_assert(EPI != kEpiSwiGLU || (JN % 2 == 0 && (BN / 2) % (8 * T::kLoadsB) == 0),
                "SwiGLU: gate and up blocks pair up, and a loader wave's B rows stay in one half");
  constexpr int kLoadsA = T::kLoadsA, kLoadsB = T::kLoadsB;
  constexpr int kStages = T::kStages, kLoadsStep = kLoadsA + kLoadsB;
  unsigned long long c0 = 0, w0 = 0;
  if (p.clk) {
    c0 = clock64();
    w0 = wall_clock64();
  }
  const int bid = blockIdx.x;
  const int loc = bid / kXcds;
  int t, ks = 0, half = 0;
  if (kUnits == kUnitsPlain) {
    if (loc >= p.tiles_per_xcd) return;
    const int u = (bid % kXcds) * p.tiles_per_xcd + loc;   // work unit: (tile, K split)
    if (u >= p.total_tiles * p.ksplit) return;
    t = u / p.ksplit;
    ks = u % p.ksplit;
  } else {
    const int full = p.tiles_per_xcd - p.tail_half;
    if (kUnits == kUnitsTailFull) {
      t = (bid % kXcds) * p.tiles_per_xcd + loc;
    } else {
      t = (bid % kXcds) * p.tiles_per_xcd + full + (loc - full) / 2;
      half = (loc - full) % 2;
    }
    if (t >= p.total_tiles) return;
  }
  // Grouped order: runs of group_m M-tiles, M fastest, so the ~32
  // workgroups an XCD runs at once cover about group_m x (32 / group_m)
  // tiles and share both operand panels in its L2.
  const int per_group = p.group_m * p.tiles_n;
  const int first_m = (t / per_group) * p.group_m;
  const int gsz = min(p.tiles_m - first_m, p.group_m);
  const int tm = first_m + (t % per_group) % gsz;
  const int tn = (kUnits == kUnitsTailHalf ? 2 : 1) * ((t % per_group) / gsz) + half;
  const int m0 = tm * BM;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // MFMA lane roles: lane l supplies row l mod 16 of a 16-row operand
  // block and its K elements [8 q4, 8 q4 + 8) of the 32-element substep;
  // accumulator register r holds row 4 q4 + r, column l mod 16.
  const int q4 = lane >> 4, l16 = lane & 15;

  // Per-thread load plan (load_tile_lds): the byte offsets of the lane's
  // row and column chunk for an even and an odd load instruction, and the
  // chunk's first column.  Rows past M (A) and past the weight's rows (B)
  // lie past the buffer's range and read zeros.  In the SwiGLU launch's
  // last column tile, gate rows past N read up rows instead: they feed
  // only output columns past N, which are never stored.  (A wave's B rows
  // lie all in the gate half or all in the up half.)
  uint32_t a_off[2], b_off[2];
  int kcol_a[2], kcol_b[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int s = (wave * kLoadsA + i) * 64 + lane;
    const int row = s / kChunks;
    const int chunk = (s % kChunks) ^ ((row >> 1) & 7);
    kcol_a[i] = chunk * 8;
    a_off[i] = static_cast<uint32_t>((m0 + row) * p.lda * 2 + chunk * 16);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int s = (wave * kLoadsB + i) * 64 + lane;
    const int row = s / kChunks;
    const int chunk = (s % kChunks) ^ ((row >> 1) & 7);
    kcol_b[i] = chunk * 8;
    int gn;
    if (EPI == kEpiSwiGLU) {
      // tile rows [0, BN/2): gate rows o0 + r; [BN/2, BN): up rows N + o0 + r - BN/2
      const int o = tn * (BN / 2) + (row & (BN / 2 - 1));
      gn = (row < BN / 2) ? o : p.N + o;
    } else {
      gn = tn * BN + row;
    }
    b_off[i] = static_cast<uint32_t>(gn * p.ldb * 2 + chunk * 16);
  }
  static_assert(kLoadsA % 2 == 0 && kLoadsB % 2 == 0, "loads come in even/odd pairs");
  const uint32_t a_step = 8u * p.lda * 2u, b_step = 8u * p.ldb * 2u;
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc((void*)p.A, 0, p.a_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc((void*)p.B, 0, p.b_bytes, 0x00020000);

  f32x4 acc[IM][JN];
#pragma unroll
  for (int i = 0; i < IM; ++i)
#pragma unroll
    for (int j = 0; j < JN; ++j) acc[i][j] = f32x4{};

  const int wm = wave / T::WAVES_N, wn = wave % T::WAVES_N;
  // LDS row of this lane's A fragment i, arow0 + 16 i, and B fragment j,
  // brow0 + bblk(j) (B rows follow the A slots).
  const int arow0 = wm * WM + l16;
  const int brow0 = (EPI == kEpiSwiGLU ? wn * (WN / 2) : wn * WN) + l16;
  auto bblk = [](int j) {
    return EPI == kEpiSwiGLU ? (j / (JN / 2)) * (BN / 2) + (j % (JN / 2)) * 16 : j * 16;
  };

  // K steps [kt0, kt0 + KT) of this unit: the whole K range, or split ks
  // of ksplit near-equal parts.
  const int KT_all = (p.K + BK - 1) / BK;
  const int kt0 = ks * KT_all / p.ksplit;
  const int KT = (ks + 1) * KT_all / p.ksplit - kt0;
  const int kb = kt0 * BK;
  // Prologue: steps 0 .. kStages-1 in flight; then step 0 resident.
  if (wave < kLoaderWaves) {
#pragma unroll
    for (int st = 0; st < kStages; ++st) {
      if (st < KT) {
        load_tile_lds<kLoadsA, true>(ra, p.a_bytes, a_off, kcol_a, a_step, kb + st * BK, p.K, lds[st], wave);
        load_tile_lds<kLoadsB, true>(rb, p.b_bytes, b_off, kcol_b, b_step, kb + st * BK, p.K, lds[st] + kSlotsA,
                                     wave);
      }
    }
  }
  // Wait for step 0; up to kStages - 1 later steps stay in flight.
  if (kStages == 4 && KT > 3) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(3 * kLoadsStep) : "memory");
  else if (kStages >= 3 && KT > 2) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kLoadsStep) : "memory");
  else if (KT > 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kLoadsStep) : "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();

  // Fragment registers.  B is double-buffered by substep parity, A is
  // single-buffered.  Substep 0 of step kt is read during the last
  // substep of step kt-1.  Every fragment row is congruent to l16 mod 16,
  // so the swizzle term (row / 2) mod 8 is the same for all of this lane's
  // blocks.
  // A fragment i of substep kk sits at slot's A base + arow0 rows +
  // ((4 kk + q4) XOR xsw) chunks + 16 i rows: one lane address per
  // (slot, substep) and an immediate offset per block.
  bf16x8 fa[IM], fb[2][JN];
  const int xsw = (l16 >> 1) & 7;
  auto abase = [&](int slot, int kk) { return lds[slot] + arow0 * kChunks + ((kk * 4 + q4) ^ xsw); };
  auto bbase = [&](int slot, int kk) { return lds[slot] + kSlotsA + brow0 * kChunks + ((kk * 4 + q4) ^ xsw); };
  auto frag = [](const u32x4* base, int rows) { return __builtin_bit_cast(bf16x8, base[rows * kChunks]); };
  {
    const u32x4* Ab = abase(0, 0);   // substep 0 of step 0 (slot 0)
    const u32x4* Bb = bbase(0, 0);
#pragma unroll
    for (int i = 0; i < IM; ++i) fa[i] = frag(Ab, i * 16);
#pragma unroll
    for (int j = 0; j < JN; ++j) fb[0][j] = frag(Bb, bblk(j));
  }
  // One substep: the MFMAs on fa and bc, in groups of one A block (JN
  // MFMAs), each followed by that block's re-read for the next substep
  // (substep kk of `slot`; its last use is just done), the next
  // substep's B blocks into bn (block i in group i, or JN / IM per group
  // when there are more B than A blocks), and, in a loader wave's refill
  // substep, an even share of its operand loads for K-step `kload` into
  // `lslot`, spread over the first half of the groups (issued earlier,
  // they gave 0.7% on gate|up against all groups).  A scheduling fence closes each group, so a block's re-read
  // cannot move above its MFMAs (which would need a second A buffer) and
  // the loads spread over the substep.
  auto substep = [&](const bf16x8* bc, int slot, int kk, bf16x8* bn, auto loads_tag, auto tail_tag, int kload,
                     int lslot) {
    constexpr bool kLoads = decltype(loads_tag)::value;
    constexpr bool kTail = decltype(tail_tag)::value;
    const u32x4* Ab = abase(slot, kk);
    const u32x4* Bb = bbase(slot, kk);
#pragma unroll
    for (int i = 0; i < IM; ++i) {
#pragma unroll
      for (int j = 0; j < JN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], bc[j], acc[i][j], 0, 0, 0);
      if constexpr (JN <= IM) {
        if (i < JN) bn[i] = frag(Bb, bblk(i));
      } else {
#pragma unroll
        for (int j = i * JN / IM; j < (i + 1) * JN / IM; ++j) bn[j] = frag(Bb, bblk(j));
      }
      fa[i] = frag(Ab, i * 16);
      if constexpr (kLoads) {
#pragma unroll
        for (int q = i * kLoadsStep / (IM / 2); q < (i + 1) * kLoadsStep / (IM / 2) && q < kLoadsStep; ++q) {
          if (q < kLoadsA)
            load_row_lds<kLoadsA, kTail>(ra, p.a_bytes, a_off, kcol_a, a_step, kload, p.K, lds[lslot], wave, q);
          else
            load_row_lds<kLoadsB, kTail>(rb, p.b_bytes, b_off, kcol_b, b_step, kload, p.K, lds[lslot] + kSlotsA,
                                         wave, q - kLoadsA);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // One K-step: the substeps of slot kt % kStages, each reading the next
  // one's fragments; before the last, wait for step kt+1 and barrier.
  // After that barrier no wave reads slot kt % kStages again, so step
  // kt+kStages's loads (kRefill) go there at once, spread over the last
  // substep, which also reads step kt+1's first substep.  While
  // refilling, the loads of steps kt+2 .. kt+kStages-1 may stay in flight
  // at the barrier; in the tail all land.
  auto step = [&](int kt, auto refill_tag, auto loader_tag, auto tail_tag) {
    constexpr bool kRefill = decltype(refill_tag)::value;
    constexpr bool kLoader = decltype(loader_tag)::value;
    const int slot = kStages == 2 ? (kt & 1) : kStages == 4 ? (kt & 3) : kt % kStages;
    const int next = kStages == 2 ? (slot ^ 1) : (slot + 1 == kStages ? 0 : slot + 1);
    // Opaque to the optimiser each step, so the per-load offset sums stay
    // at the loads instead of being hoisted out of the loop.
    if constexpr (kRefill && kLoader) asm volatile("" : "+v"(a_off[0]), "+v"(a_off[1]), "+v"(b_off[0]), "+v"(b_off[1]));
#pragma unroll
    for (int kk = 0; kk < KK - 1; ++kk)
      substep(fb[kk & 1], slot, kk + 1, fb[(kk + 1) & 1], std::false_type{}, tail_tag, 0, 0);
    // Step kt+1 must have landed; steps kt+2 .. kt+kStages-1 may not have.
    if (kRefill && kStages == 4) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kLoadsStep) : "memory");
    else if (kRefill && kStages == 3) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kLoadsStep) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    // Step kt+1 is resident; its slot index is valid even past the end
    // (the fragments are then unused).
    substep(fb[(KK - 1) & 1], next, 0, fb[KK & 1], std::integral_constant<bool, kRefill && kLoader>{}, tail_tag,
            kb + (kt + kStages) * BK, slot);
  };
  // The K-loop is specialised per role so the loader waves' loads sit in
  // the same scheduling region as their MFMAs.
  auto main_loop = [&](auto loader_tag, auto tail_tag) {
    int kt = 0;
    for (; kt + kStages < KT; ++kt) step(kt, std::true_type{}, loader_tag, tail_tag);
    for (; kt < KT; ++kt) step(kt, std::false_type{}, loader_tag, tail_tag);
  };
  // Only the loader waves issue loads, and only a K that is not a multiple
  // of BK needs the per-lane column check.
  if (wave >= kLoaderWaves) main_loop(std::false_type{}, std::false_type{});
  else if (p.K % BK == 0) main_loop(std::true_type{}, std::false_type{});
  else main_loop(std::true_type{}, std::true_type{});

  // Epilogue.  Accumulator register r of block (i, j) holds
  // row wm*WM + i*16 + 4*q4 + r and column (block col) + l16.  The lane
  // roles are derived again from an opaque copy of the thread index, so
  // nothing computed before the K-loop stays live through it for the
  // epilogue (the loop needs every register it has).
  int tid_e = static_cast<int>(threadIdx.x);
  asm volatile("" : "+v"(tid_e));
  const int q4e = (tid_e & 63) >> 4, l16e = tid_e & 15;
  if (p.ksplit > 1) {
    // Split K: the raw float32 sums go to part[ks][row][B row]; the reduce
    // kernel adds the splits in order and applies the epilogue.
    float* P = p.part + static_cast<int64_t>(ks) * p.M * p.part_ld;
#pragma unroll
    for (int j = 0; j < JN; ++j) {
      const int rr = (EPI == kEpiSwiGLU ? wn * (WN / 2) : wn * WN) + l16e + bblk(j);  // tile B row (output column) of this lane
      int col;
      bool ok;
      if (EPI == kEpiSwiGLU) {
        const int o = tn * (BN / 2) + (rr & (BN / 2 - 1));
        ok = o < p.N;
        col = (rr < BN / 2) ? o : p.N + o;
      } else {
        col = tn * BN + rr;
        ok = col < p.N;
      }
      if (!ok) continue;
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = m0 + wm * WM + i * 16 + q4e * 4 + r;
          if (row < p.M) P[static_cast<int64_t>(row) * p.part_ld + col] = acc[i][j][r];
        }
    }
  } else if (EPI == kEpiAddF32) {
    // Residual add through buffer accesses on this tile's rows: out-of-range
    // rows and columns get an offset past the range, so loads read 0 and
    // stores are dropped without a branch.  Written as C[i] += acc, a load
    // could not pass the previous store (they may alias) and each element
    // paid a memory round trip; here the residual values of the next half
    // block are loaded before the sums of this one are stored.
    // (readfirstlane keeps the descriptor in scalar registers; computed in
    // vector registers it would need a loop around every access)
    const int m0s = __builtin_amdgcn_readfirstlane(m0);
    const uint32_t c_bytes = static_cast<uint32_t>(min(p.M - m0s, BM)) * p.ldc * 4u;
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
        static_cast<float*>(p.C) + static_cast<int64_t>(m0s) * p.ldc, 0, c_bytes, 0x00020000);
    auto off = [&](int i, int r, int j) -> uint32_t {
      const int row = wm * WM + i * 16 + q4e * 4 + r;
      const int col = tn * BN + wn * WN + j * 16 + l16e;
      return col < p.N ? static_cast<uint32_t>(row * p.ldc + col) * 4u : c_bytes;
    };
    // Row blocks i are double buffered (2 x JN x 4 registers).
    float cv[2][JN][4];  // [buffer][j][r]
    auto load_block = [&](int i, float (*v)[4]) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int j = 0; j < JN; ++j)
          v[j][r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rc, off(i, r, j), 0, 0));
    };
    load_block(0, cv[0]);
#pragma unroll
    for (int i = 0; i < IM; ++i) {
      if (i + 1 < IM) load_block(i + 1, cv[(i + 1) & 1]);
      // The sums go back into the accumulators and are stored from there:
      // a store reads its data register late, so storing from cv would make
      // the loads of the next block wait for these stores.  (The sum goes
      // through a temporary: writing acc[i][j][r] and reading it back in
      // the same unrolled loop was miscompiled by the ROCm 7.2 clang; a
      // probe stored element 0's sum for every r.)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int j = 0; j < JN; ++j) {
          const float sum = cv[i & 1][j][r] + acc[i][j][r];
          acc[i][j][r] = sum;
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, sum), rc, off(i, r, j), 0, 0);
        }
    }
  } else {
#pragma unroll
  for (int i = 0; i < IM; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = m0 + wm * WM + i * 16 + q4e * 4 + r;
      if (row >= p.M) continue;
      if (EPI == kEpiSwiGLU) {
        // gate block j and up block j + JN/2 hold the same output columns
        uint16_t* C = static_cast<uint16_t*>(p.C) + static_cast<int64_t>(row) * p.ldc;
#pragma unroll
        for (int j = 0; j < JN / 2; ++j) {
          const int col = tn * (BN / 2) + wn * (WN / 2) + j * 16 + l16e;
          if (col < p.N) {
            const float gt = acc[i][j][r], up = acc[i][j + JN / 2][r];
            C[col] = f2bf(swiglu(gt, up));
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < JN; ++j) {
          const int col = tn * BN + wn * WN + j * 16 + l16e;
          if (col >= p.N) continue;
          if (EPI == kEpiF32) {
            float* C = static_cast<float*>(p.C) + static_cast<int64_t>(row) * p.ldc;
            C[col] = acc[i][j][r];
          } else {
            uint16_t* C = static_cast<uint16_t*>(p.C) + static_cast<int64_t>(row) * p.ldc;
            C[col] = f2bf(acc[i][j][r]);
          }
        }
      }
    }
  }
  }
  if (p.clk && threadIdx.x == 0) {
    const unsigned long long c1 = clock64(), w1 = wall_clock64();
    atomicAdd(&p.clk[0], c1 - c0);
    atomicAdd(&p.clk[1], w1 - w0);
    atomicAdd(&p.clk[2], 1ull);
  }
}

// Tiles of one width.
template <int EPI, int BM_, int BN_>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(16))) LdsRing<BM_, BN_> lds;
  gemm_workgroup<EPI, BM_, BN_, kUnitsPlain>(p, lds);
}

// Full-width tiles with a split tail: the last p.tail_half full tiles of
// each XCD's run (its last, partly filled round) run as two half-width
// tiles each, so that round ends sooner.  Same bits as full-width tiles.
template <int EPI>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_tail_kernel(GemmParams p) {
  static_assert(sizeof(LdsRing<256, 128>) >= sizeof(LdsRing<256, 256>), "the half-width ring is the larger");
  __shared__ __attribute__((aligned(16))) LdsRing<256, 128> lds;
  const int loc = static_cast<int>(blockIdx.x) / kXcds;
  if (loc >= p.tiles_per_xcd + p.tail_half) return;
  if (loc >= p.tiles_per_xcd - p.tail_half) gemm_workgroup<EPI, 256, 128, kUnitsTailHalf>(p, lds);
  else gemm_workgroup<EPI, 256, 256, kUnitsTailFull>(p, reinterpret_cast<LdsRing<256, 256>&>(lds));
}

// Split-K reduction: C = epilogue(sum over ks of part[ks]), the splits
// added in order (so the result is the same run to run), four columns per
// thread.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_reduce_kernel(const float* __restrict__ part, int S, int M,
                                                          int N, int ld, void* C, int ldc) {
  const int nq = N / 4;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<int64_t>(M) * nq) return;
  const int row = static_cast<int>(idx / nq), c = static_cast<int>(idx % nq) * 4;
  const int64_t split = static_cast<int64_t>(M) * ld;
  const float* src = part + static_cast<int64_t>(row) * ld + c;
  f32x4 a = *reinterpret_cast<const f32x4*>(src);
  f32x4 up = {};
  if (EPI == kEpiSwiGLU) up = *reinterpret_cast<const f32x4*>(src + N);
  for (int ks = 1; ks < S; ++ks) {
    a += *reinterpret_cast<const f32x4*>(src + ks * split);
    if (EPI == kEpiSwiGLU) up += *reinterpret_cast<const f32x4*>(src + ks * split + N);
  }
  if (EPI == kEpiAddF32) {
    f32x4* dst = reinterpret_cast<f32x4*>(static_cast<float*>(C) + static_cast<int64_t>(row) * ldc + c);
    *dst = *dst + a;
  } else if (EPI == kEpiF32) {
    *reinterpret_cast<f32x4*>(static_cast<float*>(C) + static_cast<int64_t>(row) * ldc + c) = a;
  } else {
    if (EPI == kEpiSwiGLU) {
#pragma unroll
      for (int e = 0; e < 4; ++e) a[e] = swiglu(a[e], up[e]);
    }
    u32x2 w;
    w.x = pack_bf2(a[0], a[1]);
    w.y = pack_bf2(a[2], a[3]);
    *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(C) + static_cast<int64_t>(row) * ldc + c) = w;
  }
}

// The instantiation for a tile shape (gemm_tile never picks 192-wide B
// tiles for the SwiGLU product, which has no such instantiation).
template <int EPI>
void launch_tiles(const GemmParams& p, int bm, int bn, int grid, hipStream_t s) {
  if (bm == 256 && bn == 128) gemm_bf16_kernel<EPI, 256, 128><<<grid, kThreads, 0, s>>>(p);
  else if (bm == 192 && bn == 256) gemm_bf16_kernel<EPI, 192, 256><<<grid, kThreads, 0, s>>>(p);
  else if (bm == 192 && bn == 128) gemm_bf16_kernel<EPI, 192, 128><<<grid, kThreads, 0, s>>>(p);
  else if constexpr (EPI != kEpiSwiGLU) {
    if (bm == 192 && bn == 192) {
      gemm_bf16_kernel<EPI, 192, 192><<<grid, kThreads, 0, s>>>(p);
      return;
    }
  }
  if (bm == 256 && bn == 256) {
    if (p.tail_half) gemm_bf16_tail_kernel<EPI><<<grid, kThreads, 0, s>>>(p);
    else gemm_bf16_kernel<EPI, 256, 256><<<grid, kThreads, 0, s>>>(p);
  }
}

}  // namespace

hipError_t launch_gemm(int epi, const uint16_t* A, int lda, const uint16_t* B, int ldb, void* C,
                       int ldc, int M, int N, int K, float* part, size_t part_bytes, hipStream_t s,
                       unsigned long long* clk) {
  const int64_t brows64 = epi == kEpiSwiGLU ? 2 * int64_t(N) : N;
  // byte offsets are 32-bit (buffer addressing): both operands below 2 GiB
  if (int64_t(M) * lda * 2 >= (int64_t(1) << 31) || brows64 * ldb * 2 >= (int64_t(1) << 31) ||
      M <= 0 || N <= 0 || K <= 0 || K % 8 != 0)
    return hipErrorInvalidValue;
  GemmParams p;
  p.A = A;
  p.B = B;
  p.C = C;
  p.M = M;
  p.N = N;
  p.K = K;
  p.lda = lda;
  p.ldb = ldb;
  p.ldc = ldc;
  p.ksplit = gemm_ksplit(epi, M, N, K);
  const GemmTile tile = p.ksplit == 1 ? gemm_tile(epi, M, N) : GemmTile{256, 256};
  const int bm = tile.bm, bn = tile.bn;
  p.tiles_m = (M + bm - 1) / bm;
  p.tiles_n = gemm_tiles_n(epi, N, bn);
  p.total_tiles = p.tiles_m * p.tiles_n;
  p.part = part;
  p.part_ld = epi == kEpiSwiGLU ? 2 * N : N;
  if (p.ksplit > 1 && (!part || part_bytes < gemm_split_bytes(epi, M, N, K) || ldc % 4 != 0 ||
                       (reinterpret_cast<uintptr_t>(part) & 15) != 0 ||
                       (reinterpret_cast<uintptr_t>(C) & 15) != 0))
    return hipErrorInvalidValue;
  p.tiles_per_xcd = (p.total_tiles * p.ksplit + kXcds - 1) / kXcds;
  // A last round that keeps at most half of an XCD's 32 CUs busy runs as
  // half-width tiles (full-width launches without a K split only).
  p.tail_half = 0;
  if (bm == 256 && bn == 256 && p.ksplit == 1) {
    const int rounds = (p.tiles_per_xcd + 31) / 32, last = p.tiles_per_xcd - 32 * (rounds - 1);
    if (rounds > 1 && last <= 16) p.tail_half = last;
  }
  p.group_m = std::min(p.tiles_m, kGroupM);
  p.a_bytes = static_cast<uint32_t>(int64_t(M) * lda * 2);
  const int64_t brows = epi == kEpiSwiGLU ? 2 * int64_t(N) : N;
  p.b_bytes = static_cast<uint32_t>(brows * ldb * 2);
  p.clk = clk;
  const int grid = (p.tiles_per_xcd + p.tail_half) * kXcds;
  switch (epi) {
    case kEpiBf16: launch_tiles<kEpiBf16>(p, bm, bn, grid, s); break;
    case kEpiAddF32: launch_tiles<kEpiAddF32>(p, bm, bn, grid, s); break;
    case kEpiSwiGLU: launch_tiles<kEpiSwiGLU>(p, bm, bn, grid, s); break;
    case kEpiF32: launch_tiles<kEpiF32>(p, bm, bn, grid, s); break;
    default: return hipErrorInvalidValue;
  }
  if (p.ksplit > 1) {
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    const int64_t threads = int64_t(M) * (N / 4);
    const int rgrid = static_cast<int>((threads + 255) / 256);
    switch (epi) {
      case kEpiBf16: gemm_reduce_kernel<kEpiBf16><<<rgrid, 256, 0, s>>>(part, p.ksplit, M, N, p.part_ld, C, ldc); break;
      case kEpiAddF32: gemm_reduce_kernel<kEpiAddF32><<<rgrid, 256, 0, s>>>(part, p.ksplit, M, N, p.part_ld, C, ldc); break;
      case kEpiSwiGLU: gemm_reduce_kernel<kEpiSwiGLU><<<rgrid, 256, 0, s>>>(part, p.ksplit, M, N, p.part_ld, C, ldc); break;
      case kEpiF32: gemm_reduce_kernel<kEpiF32><<<rgrid, 256, 0, s>>>(part, p.ksplit, M, N, p.part_ld, C, ldc); break;
    }
  }
  return hipGetLastError();
}

}  // namespace pallas
