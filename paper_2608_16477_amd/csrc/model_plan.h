// Model handle and the per-call plan of the prefill and decode sequences.
#pragma once

#include <algorithm>
#include <vector>

#include "kernels.h"
#include "pallas.h"

struct pallas_model {
  pallas_model_config cfg;
  const void* embed;
  const void* final_norm;
  const void* lm_head;
  std::vector<pallas_layer_weights> layers;
};

namespace pallas {

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Workspace carve-up for `tokens` rows (prefill: sum of prefix lengths;
// decode: number of sequences).
struct Workspace {
  size_t resid, h, qkv, q, o, act, rope, part, split, split_bytes, attn_split, attn_split_bytes;
  size_t gemv_part, gemv_part_bytes, gemv_ctr;
  int gemv_ctr_count;
  int part_splits;   // decode attention records per (sequence, query head)
  size_t total;
};

// Decode positions are below this bound; decode attention keeps one partial
// record per 64-key split.
constexpr int kDecodeMaxPos = 16384;
constexpr int kDecodeMaxSplits = kDecodeMaxPos / 64;

inline Workspace workspace_layout(const pallas_model_config& c, int64_t tokens, int64_t seqs) {
  Workspace w;
  const int64_t qkv = int64_t(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  size_t at = 0;
  auto take = [&](size_t bytes) { size_t o = at; at = align_up(at + bytes, 256); return o; };
  w.resid = take(size_t(tokens) * c.hidden * 4);
  w.h = take(size_t(tokens) * c.hidden * 2);
  w.qkv = take(size_t(tokens) * qkv * 2);
  w.q = take(size_t(tokens) * c.n_q_heads * c.head_dim * 2);
  w.o = take(size_t(tokens) * c.n_q_heads * c.head_dim * 2);
  w.act = take(size_t(tokens) * c.ffn * 2);
  w.rope = take(size_t(tokens) * (c.head_dim / 2) * 8);  // (cos, sin) per row and pair
  w.part_splits = kDecodeMaxSplits;
  w.part = take(size_t(seqs) * c.n_q_heads * kDecodeMaxSplits * (c.head_dim + 2) * 4);
  // Split-K partial sums of the projections of up to 256 rows.
  {
    const int rows = static_cast<int>(tokens < 256 ? tokens : 256);
    const int H = c.hidden, QD = c.n_q_heads * c.head_dim, KVD = 2 * c.n_kv_heads * c.head_dim;
    size_t b = gemm_split_bytes(kEpiBf16, rows, static_cast<int>(qkv), H);
    b = std::max(b, gemm_split_bytes(kEpiBf16, rows, KVD, H));
    b = std::max(b, gemm_split_bytes(kEpiAddF32, rows, H, QD));
    b = std::max(b, gemm_split_bytes(kEpiSwiGLU, rows, c.ffn, H));
    b = std::max(b, gemm_split_bytes(kEpiAddF32, rows, H, c.ffn));
    b = std::max(b, gemm_split_bytes(kEpiF32, rows, c.vocab, H));
    w.split_bytes = b;
    w.split = take(b);
  }
  // Split records of prefill attention over up to 256 rows.
  w.attn_split_bytes = attn_prefill_split_bytes(static_cast<int>(tokens < 256 ? tokens : 256),
                                                c.n_q_heads, c.head_dim);
  w.attn_split = take(w.attn_split_bytes);
  // Decode projections (at most 8 rows) split over K: partial sums and one
  // arrival counter per 16-row weight tile.
  {
    const int64_t rows = std::max<int64_t>(
        std::max<int64_t>(qkv, 2 * int64_t(c.ffn)), std::max<int64_t>(c.hidden, c.vocab));
    const int64_t r8 = std::min<int64_t>(std::min<int64_t>(seqs, tokens), 8);
    w.gemv_part_bytes = size_t(kGemvMaxSplit) * r8 * rows * 4;
    w.gemv_part = take(w.gemv_part_bytes);
    w.gemv_ctr_count = static_cast<int>((rows + 15) / 16);
    w.gemv_ctr = take(size_t(w.gemv_ctr_count) * 4);
  }
  w.total = at;
  return w;
}

// The smallest layout a decode step of `seqs` <= 8 sequences needs, with
// positions up to `max_pos`: the activations, decode-attention records for
// max_pos / 64 + 1 splits, and the skinny projections' split partial sums
// and counters at exactly the split counts those projections take (so the
// arithmetic is that of a step in a full workspace).  No GEMM split-K or
// prefill-attention section: more than 8 rows are not served from it.
inline Workspace decode_layout(const pallas_model_config& c, int seqs, int max_pos) {
  Workspace w{};
  const int64_t QKV = int64_t(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  const int64_t QD = int64_t(c.n_q_heads) * c.head_dim;
  size_t at = 0;
  auto take = [&](size_t bytes) { size_t o = at; at = align_up(at + bytes, 256); return o; };
  w.resid = take(size_t(seqs) * c.hidden * 4);
  w.h = take(size_t(seqs) * c.hidden * 2);
  w.qkv = take(size_t(seqs) * QKV * 2);
  w.q = take(size_t(seqs) * QD * 2);
  w.o = take(size_t(seqs) * QD * 2);
  w.act = take(size_t(seqs) * c.ffn * 2);
  w.rope = take(size_t(seqs) * (c.head_dim / 2) * 8);
  w.part_splits = max_pos / 64 + 1;
  w.part = take(size_t(seqs) * c.n_q_heads * w.part_splits * (c.head_dim + 2) * 4);
  w.split = w.attn_split = 0;
  w.split_bytes = w.attn_split_bytes = 0;
  // (epi, N, K) of the five projections; B rows are 2N for gate|up.
  const int64_t proj[5][3] = {{kEpiBf16, QKV, c.hidden},
                              {kEpiAddF32, c.hidden, QD},
                              {kEpiSwiGLU, c.ffn, c.hidden},
                              {kEpiAddF32, c.hidden, c.ffn},
                              {kEpiF32, c.vocab, c.hidden}};
  size_t part = 0;
  int tiles = 0;
  for (const auto& pr : proj) {
    const int S = gemv_ksplit(int(pr[0]), int(pr[1]), int(pr[2]));
    if (S <= 1) continue;
    const int64_t nrows = pr[0] == kEpiSwiGLU ? 2 * pr[1] : pr[1];
    part = std::max(part, size_t(S) * seqs * nrows * 4);
    tiles = std::max(tiles, int((pr[1] + 15) / 16));
  }
  w.gemv_part_bytes = part;
  w.gemv_part = take(part);
  w.gemv_ctr_count = tiles;
  w.gemv_ctr = take(size_t(tiles) * 4);
  w.total = at;
  return w;
}

inline size_t workspace_bytes(const pallas_model_config& c, int32_t max_tokens, int32_t max_seqs) {
  return workspace_layout(c, max_tokens, max_seqs).total;
}

}  // namespace pallas
