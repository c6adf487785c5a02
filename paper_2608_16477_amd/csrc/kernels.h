// Internal launch interface between the C ABI (pallas_api.hip) and the
// kernels.  Every launcher enqueues on `s` and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pallas {

// ----------------------------------------------------------------- KV copies
struct PoolGeom {
  char* base;         // bf16 [L][2][num_pages][page][Hkv][d]
  int32_t num_pages;
  int32_t page;
  int32_t lk;         // 2 * L: (layer, K|V) planes
  int32_t row_bytes;  // Hkv * d * 2, a multiple of 16
};

constexpr int kCopyMaxChunks = 128;   // chunks per copy launch
constexpr int kCopyTokens = 16;       // tokens per work unit

struct CopyChunk {
  int32_t start;       // first logical position
  int32_t count;       // positions
  uint64_t offset;     // byte offset of [2L][count][row] in the arena
};
struct CopyBatch {
  int32_t n;
  int32_t unit_prefix[kCopyMaxChunks + 1];  // work units before chunk j
  CopyChunk c[kCopyMaxChunks];
};

// Pack (pool -> arena) or assemble (arena -> pool) of up to kCopyMaxChunks
// chunks through one block table.
hipError_t launch_kv_copy(bool pack, const PoolGeom& pool, const int32_t* bt, char* arena,
                          const CopyBatch& b, int32_t* d_err, hipStream_t s);

}  // namespace pallas

namespace pallas {

// ---------------------------------------------------------------- GEMM
enum GemmEpi : int {
  kEpiBf16 = 0,    // C bf16 [M][ldc] = A B^T
  kEpiAddF32 = 1,  // C f32 [M][ldc] += A B^T (residual add)
  kEpiSwiGLU = 2,  // C bf16 [M][ldc] = silu(A Bg^T) * (A Bu^T); B rows [0,N) gate, [N,2N) up
  kEpiF32 = 3,     // C f32 [M][ldc] = A B^T
};

struct GemmParams {
  const uint16_t* A;
  const uint16_t* B;
  void* C;
  int M, N, K;
  int lda, ldb, ldc;
  int tiles_m, tiles_n, total_tiles, tiles_per_xcd, group_m;
  int tail_half;        // full tiles per XCD run split into two half-width tiles (tail kernel)
  int ksplit;           // K-range splits per tile (1: none)
  float* part;          // split partial sums [ksplit][M][part_ld] (ksplit > 1)
  int part_ld;          // B rows: N, or 2N for the gate|up product
  uint32_t a_bytes, b_bytes;
  // Clock sampling (profiling only, else null): each workgroup adds its
  // shader-clock cycles, wall-clock ticks and 1 to clk[0], clk[1], clk[2].
  unsigned long long* clk;
};

// Output-column tiles for tiles of bn B rows (gate|up: bn/2 gate + bn/2
// up rows, so bn/2 output columns per tile).
inline int gemm_tiles_n(int epi, int N, int bn = 256) {
  const int cols = epi == kEpiSwiGLU ? bn / 2 : bn;
  return (N + cols - 1) / cols;
}
// Tile shape (output rows bm x B rows bn) of a launch without a K split.
// Every shape runs the same MFMA over the same K order, so the choice never
// changes an output bit.  A launch takes rounds of one workgroup per CU,
// dealt to the 8 XCDs' 32 CUs each; its time is modelled as rounds x tile
// area / the shape's FLOP rate per CU relative to 256 x 256, measured at
// the large and mid shapes (a 256 x 256 launch whose last round keeps at
// most half the CUs busy runs that round as half-width tiles, at
// 0.5 / 0.77 of a round).  The 192-row shapes fit row counts such as
// 1536 = 8 x 192 (the mid model: Q|K|V 144 tiles of 256 x 256 but 256 of
// 192 x 192; O and down 96 but 256 of 192 x 128).  A shape replaces the
// best so far only when modelled at least 1% cheaper, so near-ties keep
// the earlier (larger) tile: at the mid model's gate|up, 1536 rows, the
// split-tail 256 x 256 launch and 192 x 256 model within 0.1% of each
// other, and the 256 x 256 one measured 248-250 against 253 us.
struct GemmTile {
  int bm, bn;
};
inline GemmTile gemm_tile(int epi, int M, int N) {
  struct Cand {
    int bm, bn, rate;   // rate: FLOP rate per CU, percent of 256 x 256
  };
  static const Cand cands[] = {{256, 256, 100}, {256, 128, 77}, {192, 256, 85}, {192, 192, 80}, {192, 128, 70}};
  GemmTile best{256, 256};
  double best_cost = 0;
  for (const Cand& c : cands) {
    if (epi == kEpiSwiGLU && c.bn == 192) continue;   // gate and up blocks pair up
    const int tiles = ((M + c.bm - 1) / c.bm) * gemm_tiles_n(epi, N, c.bn);
    const int per_xcd = (tiles + 7) / 8, rounds = (per_xcd + 31) / 32;
    double r = rounds;
    if (c.bm == 256 && c.bn == 256 && rounds > 1 && per_xcd - 32 * (rounds - 1) <= 16) r = rounds - 1 + 0.5 / 0.77;
    const double cost = r * c.bm * c.bn / c.rate;
    if (best_cost == 0 || cost < 0.99 * best_cost) {
      best = {c.bm, c.bn};
      best_cost = cost;
    }
  }
  return best;
}

// K-range splits per tile.  Only GEMMs of a single 256-row M tile split
// (their few tiles would leave most of the 256 CUs idle): each split keeps
// at least 8 K-steps of 64 and the splits fill about 256 workgroups.  The
// factor depends on N and K alone within M <= 256, and is 1 above, so a
// row's arithmetic is the same in prefills of any two lengths on the same
// side of 256 rows.
inline int gemm_ksplit(int epi, int M, int N, int K) {
  if (M > 256 || N % 4 != 0) return 1;
  const int tiles = gemm_tiles_n(epi, N), steps = (K + 63) / 64;
  int s = 256 / tiles;
  if (s > steps / 8) s = steps / 8;
  if (s > 16) s = 16;
  return s < 1 ? 1 : s;
}
// Bytes of float32 partial sums a split GEMM needs (0 when it does not split).
inline size_t gemm_split_bytes(int epi, int M, int N, int K) {
  const int s = gemm_ksplit(epi, M, N, K);
  return s > 1 ? size_t(s) * M * (epi == kEpiSwiGLU ? 2 * size_t(N) : size_t(N)) * 4 : 0;
}

// A bf16 [M][lda] (K columns used), B bf16 [rows][ldb]; K a multiple of 8;
// A and B 16-byte aligned; M*lda*2 and rows*ldb*2 below 2 GiB.  When the
// GEMM splits K (gemm_ksplit > 1), `part` (16-byte aligned, at least
// gemm_split_bytes) receives the partial sums and a second kernel reduces
// them into C; ldc must then be a multiple of 4.
hipError_t launch_gemm(int epi, const uint16_t* A, int lda, const uint16_t* B, int ldb, void* C,
                       int ldc, int M, int N, int K, float* part, size_t part_bytes, hipStream_t s,
                       unsigned long long* clk = nullptr);

}  // namespace pallas

namespace pallas {

// ------------------------------------------------------------ row metadata
constexpr int kMaxSeqs = 64;
constexpr int kMaxPrefillLen = 32768;  // tokens per sequence in one prefill call

// Rows [cu[s], cu[s+1]) belong to sequence s and sit at positions
// base_pos[s] + (row - cu[s]); sequence s uses block-table row s.
struct RowMap {
  int32_t n_seqs;
  int32_t cu[kMaxSeqs + 1];
  int32_t base_pos[kMaxSeqs];
};

__host__ __device__ inline int row_seq(const RowMap& rm, int row) {
  int s = 0;
  while (s + 1 < rm.n_seqs && rm.cu[s + 1] <= row) ++s;
  return s;
}

// ------------------------------------------------------------ norms / embed
// r[t] = float(E[ids[t]]); h[t] = bf16(rmsnorm(r[t]) * g)
hipError_t launch_embed_rmsnorm(const int32_t* ids, const uint16_t* embed, const uint16_t* gain,
                                float* r, uint16_t* h, int rows, int H, float eps, int vocab,
                                int32_t* err, hipStream_t s);
// h[t] = bf16(rmsnorm(r[t]) * g)
hipError_t launch_rmsnorm(const float* r, const uint16_t* gain, uint16_t* h, int rows, int H,
                          float eps, hipStream_t s);

// ------------------------------------------------------------ rotary table
// tab[t][i] = (cos, sin)(pos(t) * theta^(-2i/d)), evaluated in double
hipError_t launch_rope_table(const RowMap& rm, int rows, int d, float theta, float* tab,
                             hipStream_t s);

// ------------------------------------------------------------ QKV epilogue
struct QkvParams {
  const uint16_t* qkv;     // [rows][qkv_ld]: Q heads, K heads, V heads (or K, V only)
  int qkv_ld;
  int kv_only;             // 1: qkv holds only the K and V heads
  const uint16_t* q_gain;  // [d] or null
  const uint16_t* k_gain;  // [d] or null
  const float* rope;       // [rows][d/2][2]
  uint16_t* q_out;         // [rows][Hq][d] (unused when kv_only)
  uint16_t* k_plane;       // pool K plane of this layer: [P][page][Hkv][d]
  uint16_t* v_plane;       // pool V plane
  const int32_t* bt;       // [n_seqs][max_pages]
  int max_pages, num_pages, page;
  int Hq, Hkv, d;
  float eps;
  int qk_norm;
  int32_t* err;
};
hipError_t launch_qkv_rope(const QkvParams& p, const RowMap& rm, int rows, hipStream_t s);

// ------------------------------------------------------------ attention
struct AttnParams {
  const uint16_t* q;       // [rows][Hq][d]
  const uint16_t* k_plane; // [P][page][Hkv][d]
  const uint16_t* v_plane;
  const int32_t* bt;
  int max_pages, num_pages, page;
  int64_t plane_bytes;     // bytes of one K (or V) plane: num_pages * page * Hkv * d * 2
  uint16_t* o;             // [rows][Hq * d]
  int Hq, Hkv, d;
  float scale_log2;        // log2(e) / sqrt(d)
};
// Key-range splits of prefill attention.  Only calls of at most 256 rows
// split (as the GEMMs, so longer prefills keep identical bytes per row),
// and only when their (query block, KV head) workgroups are too few to fill
// the chip: up to 8 splits of at least 2 key tiles of 64.
inline int attn_prefill_splits(int rows, int workgroups, int max_tiles) {
  if (rows > 256 || workgroups >= 256) return 1;
  int s = (512 + workgroups - 1) / workgroups;
  if (s > 8) s = 8;
  if (s > max_tiles / 2) s = max_tiles / 2;
  if (s < 1) return 1;
  const int per = (max_tiles + s - 1) / s;
  return (max_tiles + per - 1) / per;
}
// Bytes of split records the workspace holds for up to `rows` rows:
// [rows][Hq][8][d + 4] floats.
inline size_t attn_prefill_split_bytes(int rows, int Hq, int d) {
  return size_t(rows < 256 ? rows : 256) * Hq * 8 * (d + 4) * 4;
}
// Causal prefill attention: row t of sequence s is position base_pos[s] +
// (t - cu[s]) and attends to keys of its own table at positions <= its
// own, [0, base_pos[s]) written by earlier calls.  `part` (split records,
// attn_prefill_split_bytes) is used when the call splits its key ranges.
hipError_t launch_attention_prefill(const AttnParams& p, const RowMap& rm, float* part, size_t part_bytes,
                                    hipStream_t s);
// Decode attention: one row per sequence at position base_pos[s], keys
// [0, base_pos[s]] through the table, split in runs of 64 keys.  `partial`
// holds [n_seqs][Hq][max_splits][d + 2] floats; needs
// base_pos[s] / 64 < max_splits and Hq / Hkv <= 8.
hipError_t launch_attention_decode(const AttnParams& p, const RowMap& rm, float* partial,
                                   int max_splits, hipStream_t s);

// ------------------------------------------------------------ skinny GEMM
// C[m][n] (op) A[m] . B[n] for m < M <= 8 rows; epilogues as launch_gemm.
// With gemv_ksplit(epi, N, K) = S > 1 the K range of each 16-row tile is
// split over S workgroups: `part` needs S * M * (N, or 2N for gate|up)
// floats and `ctr` one int per tile, zero on entry and left zero (else, or
// with too little room, the launch does not split).
constexpr int kGemvMaxSplit = 8;
int gemv_ksplit(int epi, int N, int K);
hipError_t launch_gemv(int epi, const uint16_t* A, int lda, const uint16_t* B, int ldb, void* C,
                       int ldc, int M, int N, int K, float* part, size_t part_bytes, int* ctr,
                       int ctr_count, hipStream_t s);
// ctr[0..n) = 0 (a kernel, so it can sit in a captured graph).
hipError_t launch_zero_counters(int* ctr, int n, hipStream_t s);

}  // namespace pallas
