// C ABI of the reconstruction library: argument checks, plans and launch
// sequences.  Every check runs before anything is enqueued, so a rejected
// call writes nothing.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <cmath>
#include <mutex>
#include <vector>

#include "pallas.h"
#include "kernels.h"
#include "model_plan.h"

static_assert(PALLAS_MAX_SEQS == pallas::kMaxSeqs, "sequence limit");
static_assert(PALLAS_MAX_PREFILL_LEN == pallas::kMaxPrefillLen, "prefill length limit");
static_assert(PALLAS_MAX_DECODE_POS == pallas::kDecodeMaxPos - 1, "decode position limit");
#include "profile.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* where) {
  return fail(PALLAS_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

int check_pool(const pallas_kv_pool* p, const char* what) {
  if (!p) return fail(PALLAS_ERR_INVALID_ARG, "%s: null pool", what);
  if (!p->base) return fail(PALLAS_ERR_INVALID_ARG, "%s: null pool base", what);
  if (p->num_pages <= 0 || p->page_size <= 0 || p->n_layers <= 0 || p->n_kv_heads <= 0 ||
      p->head_dim <= 0)
    return fail(PALLAS_ERR_INVALID_ARG, "%s: non-positive pool dimension", what);
  if ((reinterpret_cast<uintptr_t>(p->base) & 15) != 0)
    return fail(PALLAS_ERR_INVALID_ARG, "%s: pool base not 16-byte aligned", what);
  const int64_t row = int64_t(p->n_kv_heads) * p->head_dim * 2;
  if (row % 16 != 0 || row > (1 << 30))
    return fail(PALLAS_ERR_UNSUPPORTED, "%s: K/V row of %lld bytes is not a multiple of 16", what,
                (long long)row);
  return PALLAS_OK;
}

pallas::PoolGeom geom_of(const pallas_kv_pool* p) {
  pallas::PoolGeom g;
  g.base = static_cast<char*>(p->base);
  g.num_pages = p->num_pages;
  g.page = p->page_size;
  g.lk = 2 * p->n_layers;
  g.row_bytes = p->n_kv_heads * p->head_dim * 2;
  return g;
}

struct Span {
  int64_t a, b;
  int idx;
};

// Splits the non-empty ranges into launches of at most kCopyMaxChunks chunks.
int run_copies(bool pack, const pallas::PoolGeom& g, const int32_t* bt, char* arena,
               const std::vector<pallas::CopyChunk>& chunks, int32_t* d_err, hipStream_t s) {
  size_t i = 0;
  while (i < chunks.size()) {
    pallas::CopyBatch b;
    b.n = 0;
    b.unit_prefix[0] = 0;
    int64_t units = 0;
    for (; i < chunks.size() && b.n < pallas::kCopyMaxChunks; ++i) {
      const pallas::CopyChunk& c = chunks[i];
      const int64_t nb = (c.count + pallas::kCopyTokens - 1) / pallas::kCopyTokens;
      const int64_t add = nb * g.lk;
      if (b.n > 0 && units + add > (int64_t(1) << 30)) break;
      b.c[b.n] = c;
      units += add;
      b.n += 1;
      b.unit_prefix[b.n] = static_cast<int32_t>(units);
    }
    pallas::ProfScope ps(pack ? PALLAS_K_PACK : PALLAS_K_ASSEMBLE, s);
    hipError_t e = pallas::launch_kv_copy(pack, g, bt, arena, b, d_err, s);
    if (e != hipSuccess) return hip_fail(e, pack ? "pack launch" : "assemble launch");
  }
  return PALLAS_OK;
}

}  // namespace

extern "C" {

int32_t pallas_abi_version(void) { return PALLAS_ABI_VERSION; }

const char* pallas_last_error(void) { return g_err.c_str(); }

int pallas_check_coverage(int32_t prefix_len, const int32_t* h_starts, const int32_t* h_lens,
                          int32_t n_ranges, int32_t n) {
  if (n_ranges < 0 || (n_ranges > 0 && (!h_starts || !h_lens)))
    return fail(PALLAS_ERR_INVALID_ARG, "coverage: bad range arrays");
  if (prefix_len < 0 || n < 0 || prefix_len > n)
    return fail(PALLAS_ERR_COVERAGE, "coverage: prefix %d outside [0, %d]", prefix_len, n);
  std::vector<Span> spans;
  for (int j = 0; j < n_ranges; ++j) {
    if (h_lens[j] < 0) return fail(PALLAS_ERR_INVALID_ARG, "coverage: negative length");
    if (h_lens[j] == 0) continue;
    spans.push_back({h_starts[j], int64_t(h_starts[j]) + h_lens[j], j});
  }
  std::sort(spans.begin(), spans.end(), [](const Span& x, const Span& y) { return x.a < y.a; });
  int64_t at = prefix_len;
  for (const Span& sp : spans) {
    if (sp.a < at) return fail(PALLAS_ERR_COVERAGE, "coverage: position %lld claimed twice", (long long)sp.a);
    if (sp.a > at) return fail(PALLAS_ERR_COVERAGE, "coverage: gap at %lld", (long long)at);
    at = sp.b;
  }
  if (at != n) return fail(PALLAS_ERR_COVERAGE, "coverage: covered [0, %lld) of [0, %d)", (long long)at, n);
  return PALLAS_OK;
}

int pallas_pack_suffix_blocks(const pallas_kv_pool* src, const int32_t* d_src_block_table,
                              int32_t max_pages, const pallas_chunk_desc* h_descs,
                              int32_t n_descs, void* d_chunk_arena, size_t arena_bytes,
                              int32_t* d_err, void* stream) {
  if (int rc = check_pool(src, "pack")) return rc;
  if (!d_src_block_table || max_pages <= 0)
    return fail(PALLAS_ERR_INVALID_ARG, "pack: null block table or max_pages <= 0");
  if (n_descs < 0 || (n_descs > 0 && !h_descs))
    return fail(PALLAS_ERR_INVALID_ARG, "pack: bad descriptor array");
  const pallas::PoolGeom g = geom_of(src);
  const int64_t cap = int64_t(max_pages) * src->page_size;
  const int64_t tok_bytes = int64_t(g.lk) * g.row_bytes;
  std::vector<pallas::CopyChunk> chunks;
  std::vector<Span> spans;
  for (int j = 0; j < n_descs; ++j) {
    const pallas_chunk_desc& d = h_descs[j];
    if (d.start_pos < 0 || d.num_tokens < 0 || int64_t(d.start_pos) + d.num_tokens > cap)
      return fail(PALLAS_ERR_OUT_OF_RANGE, "pack: chunk %d range [%d, +%d) outside the table (%lld)",
                  j, d.start_pos, d.num_tokens, (long long)cap);
    if (d.num_tokens == 0) continue;
    if (d.arena_offset % 16 != 0)
      return fail(PALLAS_ERR_INVALID_ARG, "pack: chunk %d arena offset not 16-byte aligned", j);
    const uint64_t bytes = uint64_t(d.num_tokens) * tok_bytes;
    if (!d_chunk_arena || d.arena_offset > arena_bytes || bytes > arena_bytes - d.arena_offset)
      return fail(PALLAS_ERR_OUT_OF_RANGE, "pack: chunk %d leaves the arena", j);
    spans.push_back({int64_t(d.arena_offset), int64_t(d.arena_offset + bytes), j});
    chunks.push_back({d.start_pos, d.num_tokens, d.arena_offset});
  }
  std::sort(spans.begin(), spans.end(), [](const Span& x, const Span& y) { return x.a < y.a; });
  for (size_t k = 1; k < spans.size(); ++k)
    if (spans[k].a < spans[k - 1].b)
      return fail(PALLAS_ERR_INVALID_ARG, "pack: chunks %d and %d overlap in the arena",
                  spans[k - 1].idx, spans[k].idx);
  return run_copies(true, g, d_src_block_table, static_cast<char*>(d_chunk_arena), chunks, d_err,
                    static_cast<hipStream_t>(stream));
}

int pallas_assemble_kv(const pallas_kv_pool* dst, const int32_t* d_dst_block_table,
                       int32_t max_pages, const pallas_chunk_header* h_hdrs,
                       const void* d_chunk_arena, size_t arena_bytes, int32_t n_chunks,
                       uint64_t expected_request_id, uint64_t expected_epoch, int32_t* d_err,
                       void* stream) {
  if (int rc = check_pool(dst, "assemble")) return rc;
  if (!d_dst_block_table || max_pages <= 0)
    return fail(PALLAS_ERR_INVALID_ARG, "assemble: null block table or max_pages <= 0");
  if (n_chunks < 0 || (n_chunks > 0 && !h_hdrs))
    return fail(PALLAS_ERR_INVALID_ARG, "assemble: bad header array");
  for (int j = 0; j < n_chunks; ++j) {
    const pallas_chunk_header& h = h_hdrs[j];
    if (h.n_layers != dst->n_layers || h.n_kv_heads != dst->n_kv_heads ||
        h.head_dim != dst->head_dim || h.elem_bytes != 2)
      return fail(PALLAS_ERR_INVALID_ARG, "assemble: chunk %d shape differs from the pool", j);
  }
  for (int j = 0; j < n_chunks; ++j)
    if (h_hdrs[j].request_id != expected_request_id)
      return fail(PALLAS_ERR_WRONG_REQUEST, "assemble: chunk %d belongs to request %llu, not %llu", j,
                  (unsigned long long)h_hdrs[j].request_id, (unsigned long long)expected_request_id);
  for (int j = 0; j < n_chunks; ++j)
    if (h_hdrs[j].epoch != expected_epoch)
      return fail(PALLAS_ERR_STALE_EPOCH, "assemble: chunk %d has epoch %llu, expected %llu", j,
                  (unsigned long long)h_hdrs[j].epoch, (unsigned long long)expected_epoch);
  const pallas::PoolGeom g = geom_of(dst);
  const int64_t cap = int64_t(max_pages) * dst->page_size;
  const int64_t tok_bytes = int64_t(g.lk) * g.row_bytes;
  std::vector<pallas::CopyChunk> chunks;
  std::vector<Span> spans;
  for (int j = 0; j < n_chunks; ++j) {
    const pallas_chunk_header& h = h_hdrs[j];
    if (h.start_pos < 0 || h.num_tokens < 0 || int64_t(h.start_pos) + h.num_tokens > cap)
      return fail(PALLAS_ERR_OUT_OF_RANGE, "assemble: chunk %d range [%d, +%d) outside the table (%lld)",
                  j, h.start_pos, h.num_tokens, (long long)cap);
    if (h.num_tokens == 0) continue;
    const uint64_t bytes = uint64_t(h.num_tokens) * tok_bytes;
    if (!d_chunk_arena || h.arena_offset > arena_bytes || bytes > arena_bytes - h.arena_offset)
      return fail(PALLAS_ERR_OUT_OF_RANGE, "assemble: chunk %d payload leaves the arena", j);
    if (h.arena_offset % 16 != 0)
      return fail(PALLAS_ERR_INVALID_ARG, "assemble: chunk %d arena offset not 16-byte aligned", j);
    spans.push_back({h.start_pos, int64_t(h.start_pos) + h.num_tokens, j});
    chunks.push_back({h.start_pos, h.num_tokens, h.arena_offset});
  }
  std::sort(spans.begin(), spans.end(), [](const Span& x, const Span& y) { return x.a < y.a; });
  for (size_t k = 1; k < spans.size(); ++k)
    if (spans[k].a < spans[k - 1].b)
      return fail(PALLAS_ERR_COVERAGE, "assemble: chunks %d and %d both claim position %lld",
                  spans[k - 1].idx, spans[k].idx, (long long)spans[k].a);
  return run_copies(false, g, d_dst_block_table,
                    const_cast<char*>(static_cast<const char*>(d_chunk_arena)), chunks, d_err,
                    static_cast<hipStream_t>(stream));
}

}  // extern "C"

// ------------------------------------------------------------------ model
namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

int check_cfg(const pallas_model_config* c) {
  if (c->n_layers <= 0 || c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 ||
      c->head_dim <= 0 || c->ffn <= 0 || c->vocab <= 0 || c->page_size <= 0)
    return fail(PALLAS_ERR_INVALID_ARG, "model: non-positive dimension");
  if (c->n_q_heads % c->n_kv_heads != 0)
    return fail(PALLAS_ERR_INVALID_ARG, "model: query heads not a multiple of KV heads");
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f))
    return fail(PALLAS_ERR_INVALID_ARG, "model: bad eps or rope theta");
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(PALLAS_ERR_UNSUPPORTED, "model: head_dim %d (supported: 64, 128)", c->head_dim);
  if (c->page_size != 16)
    return fail(PALLAS_ERR_UNSUPPORTED, "model: page_size %d (supported: 16)", c->page_size);
  if (c->hidden % 64 != 0 || c->ffn % 16 != 0)
    return fail(PALLAS_ERR_UNSUPPORTED, "model: hidden must be a multiple of 64 and ffn of 16");
  const int grp = c->n_q_heads / c->n_kv_heads;
  if (grp != 1 && grp != 2 && grp != 4 && grp != 8)
    return fail(PALLAS_ERR_UNSUPPORTED, "model: %d query heads per KV head (supported: 1, 2, 4, 8)", grp);
  return PALLAS_OK;
}

}  // namespace

extern "C" {

int pallas_model_create(const pallas_model_config* cfg, const pallas_weights* w,
                        pallas_model** out) {
  if (!cfg || !w || !out) return fail(PALLAS_ERR_INVALID_ARG, "model: null argument");
  *out = nullptr;
  if (int rc = check_cfg(cfg)) return rc;
  if (!w->embed || !w->final_norm || !w->lm_head || !w->layers)
    return fail(PALLAS_ERR_INVALID_ARG, "model: null global weight");
  if (!aligned16(w->embed) || !aligned16(w->lm_head) || !aligned16(w->final_norm))
    return fail(PALLAS_ERR_INVALID_ARG, "model: weights must be 16-byte aligned");
  for (int l = 0; l < cfg->n_layers; ++l) {
    const pallas_layer_weights& L = w->layers[l];
    const void* need[] = {L.attn_norm, L.w_qkv, L.w_o, L.mlp_norm, L.w_gate_up, L.w_down};
    for (const void* p : need)
      if (!p || !aligned16(p)) return fail(PALLAS_ERR_INVALID_ARG, "model: layer %d weight null or unaligned", l);
    if (cfg->qk_norm && (!L.q_norm || !L.k_norm || !aligned16(L.q_norm) || !aligned16(L.k_norm)))
      return fail(PALLAS_ERR_INVALID_ARG, "model: layer %d QK-norm gains null or unaligned", l);
  }
  pallas_model* m = new pallas_model;
  m->cfg = *cfg;
  m->embed = w->embed;
  m->final_norm = w->final_norm;
  m->lm_head = w->lm_head;
  m->layers.assign(w->layers, w->layers + cfg->n_layers);
  *out = m;
  return PALLAS_OK;
}

void pallas_model_destroy(pallas_model* m) { delete m; }

}  // extern "C"

// ------------------------------------------------------------- prefill / decode
namespace {

int check_model_pool(const pallas_model* m, const pallas_kv_pool* pool, const char* what) {
  if (int rc = check_pool(pool, what)) return rc;
  const pallas_model_config& c = m->cfg;
  if (pool->n_layers != c.n_layers || pool->n_kv_heads != c.n_kv_heads ||
      pool->head_dim != c.head_dim || pool->page_size != c.page_size)
    return fail(PALLAS_ERR_INVALID_ARG, "%s: pool shape differs from the model", what);
  return PALLAS_OK;
}

int check_workspace(const pallas_model* m, const void* ws, size_t bytes, int64_t rows, int64_t seqs,
                    const char* what) {
  if (!ws) return fail(PALLAS_ERR_INVALID_ARG, "%s: null workspace", what);
  if ((reinterpret_cast<uintptr_t>(ws) & 255) != 0)
    return fail(PALLAS_ERR_INVALID_ARG, "%s: workspace not 256-byte aligned", what);
  const size_t need = pallas::workspace_layout(m->cfg, rows, seqs).total;
  if (bytes < need)
    return fail(PALLAS_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", what, bytes, need);
  return PALLAS_OK;
}

// The projections address their operands through buffer descriptors with
// 32-bit byte offsets, so every activation matrix a call feeds them and
// every weight matrix must stay below 2 GiB (the MFMA GEMM, for more than 8
// rows), or a 16-row weight tile and 8 activation rows below 4 GiB (the
// skinny kernel, which decode uses for up to 8 rows; prefill always runs
// the MFMA GEMM).  Checked here, on the host, so a call that would reach a
// limit mid-sequence is refused before layer 0 writes anything.
// `lm_head`: the call also projects the final norm onto the vocabulary
// (decode).
int check_gemm_extents(const pallas_model_config& c, int64_t rows, bool skinny, bool lm_head,
                       const char* what) {
  const int64_t H = c.hidden, QD = int64_t(c.n_q_heads) * c.head_dim, F = c.ffn;
  const int64_t QKV = int64_t(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  struct Op {
    const char* name;
    int64_t rows, ld;
  };
  const Op acts[] = {{"normalised activations", rows, H}, {"attention output", rows, QD},
                     {"SwiGLU product", rows, F}};
  const Op wts[] = {{"w_qkv", QKV, H},          {"w_o", H, QD},     {"w_gate_up", 2 * F, H},
                    {"w_down", H, F},           {"lm_head", lm_head ? int64_t(c.vocab) : 0, H}};
  if (!skinny) {
    const int64_t lim = int64_t(1) << 31;
    for (const Op& o : acts)
      if (o.rows * o.ld * 2 >= lim)
        return fail(PALLAS_ERR_UNSUPPORTED, "%s: %lld rows make the %s %lld bytes (at most 2 GiB - 1)", what,
                    (long long)rows, o.name, (long long)(o.rows * o.ld * 2));
    for (const Op& o : wts)
      if (o.rows * o.ld * 2 >= lim)
        return fail(PALLAS_ERR_UNSUPPORTED, "%s: %s of %lld bytes (at most 2 GiB - 1 for more than 8 rows)", what,
                    o.name, (long long)(o.rows * o.ld * 2));
  } else {
    const int64_t lim = int64_t(1) << 32;
    for (const Op& o : acts)
      if (8 * o.ld * 2 >= lim)
        return fail(PALLAS_ERR_UNSUPPORTED, "%s: %s rows of %lld bytes", what, o.name, (long long)(o.ld * 2));
    for (const Op& o : wts)
      if (o.rows > 0 && 16 * o.ld * 2 >= lim)
        return fail(PALLAS_ERR_UNSUPPORTED, "%s: %s rows of %lld bytes", what, o.name, (long long)(o.ld * 2));
  }
  return PALLAS_OK;
}

#define PALLAS_TRY(cls, expr, where)                  \
  do {                                                \
    pallas::ProfScope ps_(cls, s);                    \
    hipError_t e_ = (expr);                           \
    if (e_ != hipSuccess) return hip_fail(e_, where); \
  } while (0)

struct Planes {
  uint16_t* k;
  uint16_t* v;
};

Planes layer_planes(const pallas_kv_pool* pool, int l) {
  const int64_t plane = int64_t(pool->num_pages) * pool->page_size * pool->n_kv_heads * pool->head_dim;
  uint16_t* base = static_cast<uint16_t*>(pool->base) + int64_t(l) * 2 * plane;
  return {base, base + plane};
}

const uint16_t* u16(const void* p) { return static_cast<const uint16_t*>(p); }

// Projection of `rows` activation rows: the MFMA GEMM, or the skinny kernel
// for up to 8 rows.
// Scratch of the projections of one call: split-K partial sums of the
// GEMM, and partial sums plus arrival counters of the skinny kernel.
struct ProjScratch {
  float* split;
  size_t split_bytes;
  float* gv_part;
  size_t gv_part_bytes;
  int* gv_ctr;
  int gv_ctr_count;
};

hipError_t project(int epi, const uint16_t* A, int lda, const uint16_t* B, int ldb, void* C, int ldc,
                   int rows, int N, int K, const ProjScratch& sc, hipStream_t s) {
  if (rows <= 8)
    return pallas::launch_gemv(epi, A, lda, B, ldb, C, ldc, rows, N, K, sc.gv_part, sc.gv_part_bytes, sc.gv_ctr,
                               sc.gv_ctr_count, s);
  return pallas::launch_gemm(epi, A, lda, B, ldb, C, ldc, rows, N, K, sc.split, sc.split_bytes, s);
}

int run_prefill(const pallas_model* m, const pallas::RowMap& rm, int M, const int32_t* ids,
                const int32_t* bt, int max_pages, const pallas_kv_pool* pool, char* ws, int32_t* err,
                hipStream_t s) {
  const pallas_model_config& c = m->cfg;
  const pallas::Workspace w = pallas::workspace_layout(c, M, rm.n_seqs);
  float* r = reinterpret_cast<float*>(ws + w.resid);
  uint16_t* h = reinterpret_cast<uint16_t*>(ws + w.h);
  uint16_t* qkv = reinterpret_cast<uint16_t*>(ws + w.qkv);
  uint16_t* q = reinterpret_cast<uint16_t*>(ws + w.q);
  uint16_t* o = reinterpret_cast<uint16_t*>(ws + w.o);
  uint16_t* act = reinterpret_cast<uint16_t*>(ws + w.act);
  float* rope = reinterpret_cast<float*>(ws + w.rope);
  float* split = reinterpret_cast<float*>(ws + w.split);
  const size_t sb = w.split_bytes;
  const int H = c.hidden, d = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads, F = c.ffn;
  const int QKV = (Hq + 2 * Hkv) * d, QD = Hq * d, KVD = 2 * Hkv * d;

  PALLAS_TRY(PALLAS_K_ROPE_TABLE, pallas::launch_rope_table(rm, M, d, c.rope_theta, rope, s), "rope table");
  PALLAS_TRY(PALLAS_K_EMBED, pallas::launch_embed_rmsnorm(ids, u16(m->embed), u16(m->layers[0].attn_norm), r, h, M, H,
                                          c.rms_eps, c.vocab, err, s), "embed");
  pallas::QkvParams qp;
  qp.rope = rope;
  qp.q_out = q;
  qp.bt = bt;
  qp.max_pages = max_pages;
  qp.num_pages = pool->num_pages;
  qp.page = pool->page_size;
  qp.Hq = Hq;
  qp.Hkv = Hkv;
  qp.d = d;
  qp.eps = c.rms_eps;
  qp.qk_norm = c.qk_norm;
  qp.err = err;
  pallas::AttnParams ap;
  ap.q = q;
  ap.bt = bt;
  ap.max_pages = max_pages;
  ap.num_pages = pool->num_pages;
  ap.plane_bytes = int64_t(pool->num_pages) * pool->page_size * pool->n_kv_heads * pool->head_dim * 2;
  ap.page = pool->page_size;
  ap.o = o;
  ap.Hq = Hq;
  ap.Hkv = Hkv;
  ap.d = d;
  ap.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(double(d)));

  for (int l = 0; l < c.n_layers; ++l) {
    const pallas_layer_weights& L = m->layers[l];
    const bool last = l == c.n_layers - 1;
    const Planes pl = layer_planes(pool, l);
    if (l > 0) PALLAS_TRY(PALLAS_K_RMSNORM, pallas::launch_rmsnorm(r, u16(L.attn_norm), h, M, H, c.rms_eps, s), "rmsnorm");
    qp.q_gain = u16(L.q_norm);
    qp.k_gain = u16(L.k_norm);
    qp.k_plane = pl.k;
    qp.v_plane = pl.v;
    if (last) {
      // Only K and V of the last layer reach the cache.
      PALLAS_TRY(PALLAS_K_GEMM_QKV, pallas::launch_gemm(pallas::kEpiBf16, h, H, u16(L.w_qkv) + int64_t(QD) * H, H, qkv, KVD, M,
                                     KVD, H, split, sb, s), "kv gemm");
      qp.qkv = qkv;
      qp.qkv_ld = KVD;
      qp.kv_only = 1;
      PALLAS_TRY(PALLAS_K_QKV_EPI, pallas::launch_qkv_rope(qp, rm, M, s), "kv epilogue");
      break;
    }
    PALLAS_TRY(PALLAS_K_GEMM_QKV, pallas::launch_gemm(pallas::kEpiBf16, h, H, u16(L.w_qkv), H, qkv, QKV, M, QKV, H, split, sb, s,
                                                      pallas::profile_clock_slot(PALLAS_K_GEMM_QKV)), "qkv gemm");
    qp.qkv = qkv;
    qp.qkv_ld = QKV;
    qp.kv_only = 0;
    PALLAS_TRY(PALLAS_K_QKV_EPI, pallas::launch_qkv_rope(qp, rm, M, s), "qkv epilogue");
    ap.k_plane = pl.k;
    ap.v_plane = pl.v;
    PALLAS_TRY(PALLAS_K_ATTN, pallas::launch_attention_prefill(ap, rm, reinterpret_cast<float*>(ws + w.attn_split),
                                                               w.attn_split_bytes, s), "attention");
    PALLAS_TRY(PALLAS_K_GEMM_O, pallas::launch_gemm(pallas::kEpiAddF32, o, QD, u16(L.w_o), QD, r, H, M, H, QD, split, sb, s,
                                                     pallas::profile_clock_slot(PALLAS_K_GEMM_O)), "o gemm");
    PALLAS_TRY(PALLAS_K_RMSNORM, pallas::launch_rmsnorm(r, u16(L.mlp_norm), h, M, H, c.rms_eps, s), "rmsnorm");
    PALLAS_TRY(PALLAS_K_GEMM_GATE_UP, pallas::launch_gemm(pallas::kEpiSwiGLU, h, H, u16(L.w_gate_up), H, act, F, M, F, H, split, sb, s,
                                                         pallas::profile_clock_slot(PALLAS_K_GEMM_GATE_UP)),
               "gate_up gemm");
    PALLAS_TRY(PALLAS_K_GEMM_DOWN, pallas::launch_gemm(pallas::kEpiAddF32, act, F, u16(L.w_down), F, r, H, M, H, F, split, sb, s,
                                                        pallas::profile_clock_slot(PALLAS_K_GEMM_DOWN)), "down gemm");
  }
  return PALLAS_OK;
}

// One decode step with its intermediate values in `ws`, carved up by `w`
// (a full workspace's layout, or the compact decode layout).
int run_decode(const pallas_model* m, const pallas::RowMap& rm, const int32_t* tokens, const int32_t* bt,
               int max_pages, const pallas_kv_pool* pool, float* logits, char* ws, const pallas::Workspace& w,
               int32_t* err, hipStream_t s) {
  const pallas_model_config& c = m->cfg;
  const int B = rm.n_seqs;
  float* part = reinterpret_cast<float*>(ws + w.part);
  float* r = reinterpret_cast<float*>(ws + w.resid);
  uint16_t* h = reinterpret_cast<uint16_t*>(ws + w.h);
  uint16_t* qkv = reinterpret_cast<uint16_t*>(ws + w.qkv);
  uint16_t* q = reinterpret_cast<uint16_t*>(ws + w.q);
  uint16_t* o = reinterpret_cast<uint16_t*>(ws + w.o);
  uint16_t* act = reinterpret_cast<uint16_t*>(ws + w.act);
  float* rope = reinterpret_cast<float*>(ws + w.rope);
  float* split = reinterpret_cast<float*>(ws + w.split);
  const size_t sb = w.split_bytes;
  const int H = c.hidden, d = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads, F = c.ffn;
  const int QKV = (Hq + 2 * Hkv) * d, QD = Hq * d;

  const ProjScratch sc{split, sb, reinterpret_cast<float*>(ws + w.gemv_part), w.gemv_part_bytes,
                       reinterpret_cast<int*>(ws + w.gemv_ctr), w.gemv_ctr_count};
  if (hipError_t e = pallas::launch_zero_counters(sc.gv_ctr, sc.gv_ctr_count, s); e != hipSuccess)
    return hip_fail(e, "counters");
  PALLAS_TRY(PALLAS_K_ROPE_TABLE, pallas::launch_rope_table(rm, B, d, c.rope_theta, rope, s), "rope table");
  PALLAS_TRY(PALLAS_K_EMBED, pallas::launch_embed_rmsnorm(tokens, u16(m->embed), u16(m->layers[0].attn_norm), r, h, B, H,
                                          c.rms_eps, c.vocab, err, s), "embed");
  pallas::QkvParams qp;
  qp.rope = rope;
  qp.q_out = q;
  qp.bt = bt;
  qp.max_pages = max_pages;
  qp.num_pages = pool->num_pages;
  qp.page = pool->page_size;
  qp.Hq = Hq;
  qp.Hkv = Hkv;
  qp.d = d;
  qp.eps = c.rms_eps;
  qp.qk_norm = c.qk_norm;
  qp.err = err;
  qp.qkv = qkv;
  qp.qkv_ld = QKV;
  qp.kv_only = 0;
  pallas::AttnParams ap;
  ap.q = q;
  ap.bt = bt;
  ap.max_pages = max_pages;
  ap.num_pages = pool->num_pages;
  ap.plane_bytes = int64_t(pool->num_pages) * pool->page_size * pool->n_kv_heads * pool->head_dim * 2;
  ap.page = pool->page_size;
  ap.o = o;
  ap.Hq = Hq;
  ap.Hkv = Hkv;
  ap.d = d;
  ap.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(double(d)));
  for (int l = 0; l < c.n_layers; ++l) {
    const pallas_layer_weights& L = m->layers[l];
    const Planes pl = layer_planes(pool, l);
    if (l > 0) PALLAS_TRY(PALLAS_K_RMSNORM, pallas::launch_rmsnorm(r, u16(L.attn_norm), h, B, H, c.rms_eps, s), "rmsnorm");
    PALLAS_TRY(PALLAS_K_DECODE_PROJ, project(pallas::kEpiBf16, h, H, u16(L.w_qkv), H, qkv, QKV, B, QKV, H, sc, s), "qkv proj");
    qp.q_gain = u16(L.q_norm);
    qp.k_gain = u16(L.k_norm);
    qp.k_plane = pl.k;
    qp.v_plane = pl.v;
    PALLAS_TRY(PALLAS_K_QKV_EPI, pallas::launch_qkv_rope(qp, rm, B, s), "qkv epilogue");
    ap.k_plane = pl.k;
    ap.v_plane = pl.v;
    PALLAS_TRY(PALLAS_K_DECODE_ATTN, pallas::launch_attention_decode(ap, rm, part, w.part_splits, s), "decode attention");
    PALLAS_TRY(PALLAS_K_DECODE_PROJ, project(pallas::kEpiAddF32, o, QD, u16(L.w_o), QD, r, H, B, H, QD, sc, s), "o proj");
    PALLAS_TRY(PALLAS_K_RMSNORM, pallas::launch_rmsnorm(r, u16(L.mlp_norm), h, B, H, c.rms_eps, s), "rmsnorm");
    PALLAS_TRY(PALLAS_K_DECODE_PROJ, project(pallas::kEpiSwiGLU, h, H, u16(L.w_gate_up), H, act, F, B, F, H, sc, s), "gate_up proj");
    PALLAS_TRY(PALLAS_K_DECODE_PROJ, project(pallas::kEpiAddF32, act, F, u16(L.w_down), F, r, H, B, H, F, sc, s), "down proj");
  }
  PALLAS_TRY(PALLAS_K_RMSNORM, pallas::launch_rmsnorm(r, u16(m->final_norm), h, B, H, c.rms_eps, s), "final norm");
  PALLAS_TRY(PALLAS_K_DECODE_PROJ, project(pallas::kEpiF32, h, H, u16(m->lm_head), H, logits, c.vocab, B, c.vocab, H, sc, s), "lm_head");
  return PALLAS_OK;
}

}  // namespace

extern "C" {

size_t pallas_workspace_size(const pallas_model* m, int32_t max_tokens, int32_t max_seqs) {
  if (!m || max_tokens <= 0 || max_seqs <= 0) return 0;
  return pallas::workspace_bytes(m->cfg, max_tokens, max_seqs);
}

}  // extern "C"

namespace {

// Argument checks shared by both decode entry points; fills the row map.
int decode_checks(const pallas_model* m, int32_t num_seqs, const int32_t* d_tokens, const int32_t* h_positions,
                  const int32_t* d_block_tables, int32_t max_pages, const pallas_kv_pool* pool,
                  const float* d_logits, const char* what, pallas::RowMap& rm) {
  if (!m) return fail(PALLAS_ERR_INVALID_ARG, "%s: null model", what);
  if (num_seqs < 1 || num_seqs > PALLAS_MAX_SEQS)
    return fail(PALLAS_ERR_INVALID_ARG, "%s: num_seqs %d outside [1, %d]", what, num_seqs, PALLAS_MAX_SEQS);
  if (!d_tokens || !h_positions || !d_block_tables || !d_logits || max_pages <= 0)
    return fail(PALLAS_ERR_INVALID_ARG, "%s: null tokens, positions, tables or logits", what);
  if (int rc = check_model_pool(m, pool, what)) return rc;
  rm.n_seqs = num_seqs;
  const int64_t cap = int64_t(max_pages) * pool->page_size;
  for (int i = 0; i < num_seqs; ++i) {
    rm.cu[i] = i;
    const int n = h_positions[i];
    if (n < 0 || int64_t(n) + 1 > cap)
      return fail(PALLAS_ERR_OUT_OF_RANGE, "%s: position %d of sequence %d outside the table (%lld)", what, n, i,
                  (long long)cap);
    if (n >= pallas::kDecodeMaxPos)
      return fail(PALLAS_ERR_UNSUPPORTED, "%s: position %d beyond %d", what, n, pallas::kDecodeMaxPos - 1);
    rm.base_pos[i] = n;
  }
  rm.cu[num_seqs] = num_seqs;
  return check_gemm_extents(m->cfg, num_seqs, num_seqs <= 8, true, what);
}

// Scratch of pallas_decode_step_static: one copy per GPU, in the library's
// device code object, held until the process ends.  Host code never uses
// the array's name as an address: its device address on the current GPU is
// looked up once per device (hipGetSymbolAddress, on the first call that
// runs there) and kept in `g_scratch`.
static __device__ __align__(256) unsigned char scratch[PALLAS_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch[kMaxDevices];

int static_scratch(char** out) {
  int dev = -1;
  if (hipError_t e = hipGetDevice(&dev); e != hipSuccess) return hip_fail(e, "decode (static scratch): device");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(PALLAS_ERR_UNSUPPORTED, "decode (static scratch): device %d (at most %d devices)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)); e != hipSuccess)
      return hip_fail(e, "decode (static scratch): symbol address");
    if (!p || (reinterpret_cast<uintptr_t>(p) & 255) != 0)
      return fail(PALLAS_ERR_HIP, "decode (static scratch): bad scratch address");
    g_scratch[dev] = static_cast<char*>(p);
  }
  *out = g_scratch[dev];
  return PALLAS_OK;
}

// Shared by the whole-prefix and the chunked prefill: sequence i's ids sit
// at positions start[i] .. start[i] + p_i - 1 (start null: all 0).
int prefill_call(pallas_model* m, int32_t num_seqs, const int32_t* d_token_ids,
                 const int32_t* h_cu_seqlens, const int32_t* h_start_pos,
                 const int32_t* d_block_tables, int32_t max_pages, const pallas_kv_pool* pool,
                 void* d_workspace, size_t ws_bytes, int32_t* d_err, void* stream,
                 const char* what) {
  if (!m) return fail(PALLAS_ERR_INVALID_ARG, "%s: null model", what);
  if (num_seqs < 1 || num_seqs > PALLAS_MAX_SEQS)
    return fail(PALLAS_ERR_INVALID_ARG, "%s: num_seqs %d outside [1, %d]", what, num_seqs, PALLAS_MAX_SEQS);
  if (!d_token_ids || !h_cu_seqlens || !d_block_tables || max_pages <= 0)
    return fail(PALLAS_ERR_INVALID_ARG, "%s: null ids, cu_seqlens or block tables", what);
  if (int rc = check_model_pool(m, pool, what)) return rc;
  // Prefill attention loads K tiles through 32-bit offsets into a layer's K plane.
  const int64_t plane = int64_t(pool->num_pages) * pool->page_size * pool->n_kv_heads * pool->head_dim * 2;
  if (plane > int64_t(0xFFFFFFFFll))
    return fail(PALLAS_ERR_UNSUPPORTED, "%s: a layer's K plane of %lld bytes exceeds 4 GiB", what, (long long)plane);
  pallas::RowMap rm;
  rm.n_seqs = num_seqs;
  if (h_cu_seqlens[0] != 0) return fail(PALLAS_ERR_INVALID_ARG, "%s: cu_seqlens[0] must be 0", what);
  const int64_t cap = int64_t(max_pages) * pool->page_size;
  for (int i = 0; i <= num_seqs; ++i) rm.cu[i] = h_cu_seqlens[i];
  for (int i = 0; i < num_seqs; ++i) {
    const int64_t len = int64_t(h_cu_seqlens[i + 1]) - h_cu_seqlens[i];
    const int64_t start = h_start_pos ? h_start_pos[i] : 0;
    if (len < 1) return fail(PALLAS_ERR_INVALID_ARG, "%s: sequence %d has length %lld", what, i, (long long)len);
    if (start < 0) return fail(PALLAS_ERR_INVALID_ARG, "%s: sequence %d starts at %lld", what, i, (long long)start);
    if (start + len > cap)
      return fail(PALLAS_ERR_OUT_OF_RANGE, "%s: sequence %d positions [%lld, %lld) exceed the table (%lld)", what,
                  i, (long long)start, (long long)(start + len), (long long)cap);
    if (start + len > PALLAS_MAX_PREFILL_LEN)
      return fail(PALLAS_ERR_UNSUPPORTED, "%s: sequence %d reaches position %lld (at most %d)", what, i,
                  (long long)(start + len), PALLAS_MAX_PREFILL_LEN);
    rm.base_pos[i] = static_cast<int32_t>(start);
  }
  const int64_t M = h_cu_seqlens[num_seqs];
  if (M > (int64_t(1) << 24)) return fail(PALLAS_ERR_UNSUPPORTED, "%s: too many tokens", what);
  if (int rc = check_gemm_extents(m->cfg, M, false, false, what)) return rc;
  if (int rc = check_workspace(m, d_workspace, ws_bytes, M, num_seqs, what)) return rc;
  return run_prefill(m, rm, static_cast<int>(M), d_token_ids, d_block_tables, max_pages, pool,
                     static_cast<char*>(d_workspace), d_err, static_cast<hipStream_t>(stream));
}

}  // namespace

extern "C" {

int pallas_prefill_prefix(pallas_model* m, int32_t num_seqs, const int32_t* d_token_ids,
                          const int32_t* h_cu_seqlens, const int32_t* d_block_tables,
                          int32_t max_pages, const pallas_kv_pool* pool, void* d_workspace,
                          size_t ws_bytes, int32_t* d_err, void* stream) {
  return prefill_call(m, num_seqs, d_token_ids, h_cu_seqlens, nullptr, d_block_tables, max_pages,
                      pool, d_workspace, ws_bytes, d_err, stream, "prefill");
}

int pallas_prefill_chunk(pallas_model* m, int32_t num_seqs, const int32_t* d_token_ids,
                         const int32_t* h_cu_seqlens, const int32_t* h_start_pos,
                         const int32_t* d_block_tables, int32_t max_pages,
                         const pallas_kv_pool* pool, void* d_workspace, size_t ws_bytes,
                         int32_t* d_err, void* stream) {
  if (!h_start_pos) return fail(PALLAS_ERR_INVALID_ARG, "prefill chunk: null start positions");
  return prefill_call(m, num_seqs, d_token_ids, h_cu_seqlens, h_start_pos, d_block_tables, max_pages,
                      pool, d_workspace, ws_bytes, d_err, stream, "prefill chunk");
}

int pallas_decode_step(pallas_model* m, int32_t num_seqs, const int32_t* d_tokens,
                       const int32_t* h_positions, const int32_t* d_block_tables,
                       int32_t max_pages, const pallas_kv_pool* pool, float* d_logits,
                       void* d_workspace, size_t ws_bytes, int32_t* d_err, void* stream) {
  pallas::RowMap rm;
  if (int rc = decode_checks(m, num_seqs, d_tokens, h_positions, d_block_tables, max_pages, pool, d_logits,
                             "decode", rm))
    return rc;
  if (int rc = check_workspace(m, d_workspace, ws_bytes, num_seqs, num_seqs, "decode")) return rc;
  return run_decode(m, rm, d_tokens, d_block_tables, max_pages, pool, d_logits, static_cast<char*>(d_workspace),
                    pallas::workspace_layout(m->cfg, num_seqs, num_seqs), d_err,
                    static_cast<hipStream_t>(stream));
}

int pallas_decode_step_static(pallas_model* m, int32_t num_seqs, const int32_t* d_tokens,
                              const int32_t* h_positions, const int32_t* d_block_tables,
                              int32_t max_pages, const pallas_kv_pool* pool, float* d_logits,
                              int32_t* d_err, void* stream) {
  pallas::RowMap rm;
  if (int rc = decode_checks(m, num_seqs, d_tokens, h_positions, d_block_tables, max_pages, pool, d_logits,
                             "decode (static scratch)", rm))
    return rc;
  if (num_seqs > PALLAS_STATIC_DECODE_MAX_SEQS)
    return fail(PALLAS_ERR_UNSUPPORTED, "decode (static scratch): %d sequences (at most %d)", num_seqs,
                PALLAS_STATIC_DECODE_MAX_SEQS);
  int max_pos = 0;
  for (int i = 0; i < num_seqs; ++i) max_pos = std::max(max_pos, h_positions[i]);
  const pallas::Workspace w = pallas::decode_layout(m->cfg, num_seqs, max_pos);
  if (w.total > PALLAS_STATIC_SCRATCH_BYTES)
    return fail(PALLAS_ERR_UNSUPPORTED,
                "decode (static scratch): %d sequences up to position %d need %zu bytes of scratch (at most %zu)",
                num_seqs, max_pos, w.total, size_t(PALLAS_STATIC_SCRATCH_BYTES));
  char* ws = nullptr;
  if (int rc = static_scratch(&ws)) return rc;
  return run_decode(m, rm, d_tokens, d_block_tables, max_pages, pool, d_logits, ws, w, d_err,
                    static_cast<hipStream_t>(stream));
}

}  // extern "C"
