/*
 * pallas.h -- C ABI of the MI355X (gfx950) library for target-side KV-cache
 * reconstruction (Pallas, arXiv 2608.16477).
 *
 * The method (Section 4.3, "Parallel State Preparation"): at the trigger the
 * source splits the token sequence at position k; the target rebuilds the KV
 * cache of the stable prefix [0, k) by a local prefill; the source streams
 * the per-layer K/V of completed suffix blocks with their logical positions;
 * at handover the target copies them into a newly allocated block table
 * (Section 5), checks that [0, n) is covered with no gap or conflict and
 * that no block of a cancelled attempt (older migration epoch) enters the
 * request, and resumes decoding at position n.
 *
 * Calls:
 *   pallas_prefill_prefix      prefix prefill writing K/V into paged blocks
 *   pallas_prefill_chunk       the same, one chunk at a time over earlier chunks
 *   pallas_pack_suffix_blocks  gather suffix pages into transfer chunks
 *   pallas_assemble_kv         scatter chunks into the target block table
 *   pallas_decode_step         one decode step over an assembled cache
 *   pallas_check_coverage      host-only [0, n) coverage check
 *   pallas_window_*, pallas_ewma_update, pallas_admit, pallas_waste_bound
 *                              host-only Scheduler Engine (when to migrate)
 *
 * Conventions shared by every call:
 *   - Device pointers are named d_*, host pointers h_*.  All device memory
 *     (weights, pools, tables, chunk arenas, logits, workspace) belongs to the
 *     caller; the library allocates no device memory and keeps no pointer
 *     beyond a call, except the weight pointers kept by a model handle (and
 *     the opt-in profiling calls, which allocate a 312-byte counter array
 *     once per process).
 *   - Calls may come from several host threads at once.  A model handle is
 *     read-only after creation and may be shared; a workspace may not be
 *     used by two calls whose work is in flight at the same time unless
 *     they are ordered on one stream.
 *   - Host structs and arrays are read during the call only.
 *   - `stream` is a hipStream_t (NULL: the default stream).  Work is enqueued
 *     on it; calls return before the work completes and never synchronise.
 *   - A nonzero return is a pallas_status.  Every argument check is done
 *     before anything is enqueued, so a rejected call writes nothing.
 *     pallas_last_error() gives a message (thread-local, valid until the
 *     thread's next call).
 *   - Element type of weights, activations and the KV cache is bf16 (raw
 *     16-bit patterns); the residual stream is float32; logits are float32.
 *   - Results are bitwise reproducible run to run for the same inputs.
 */
#ifndef PALLAS_H
#define PALLAS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PALLAS_ABI_VERSION 3
#define PALLAS_MAX_SEQS 64 /* sequences per prefill or decode call */
#define PALLAS_MAX_PREFILL_LEN 32768 /* tokens per sequence in one prefill call */
#define PALLAS_MAX_DECODE_POS 16383  /* largest position a decode step accepts */

typedef enum {
  PALLAS_OK = 0,
  PALLAS_ERR_INVALID_ARG = 1,  /* null pointer, bad size, shape mismatch */
  PALLAS_ERR_OUT_OF_RANGE = 2, /* position or range outside a table / arena */
  PALLAS_ERR_COVERAGE = 3,     /* gap or two claims on one position */
  PALLAS_ERR_STALE_EPOCH = 4,  /* chunk of another migration epoch */
  PALLAS_ERR_WRONG_REQUEST = 5,/* chunk of another request */
  PALLAS_ERR_UNSUPPORTED = 6,  /* shape the library has no kernel for */
  PALLAS_ERR_HIP = 7,          /* a HIP runtime call failed */
  PALLAS_ERR_WORKSPACE = 8     /* workspace too small */
} pallas_status;

/* Device-side error bits written (OR-ed) into the optional d_err word. */
#define PALLAS_DEVERR_PAGE 1u  /* a block-table entry named no page of the pool;
                                  that position was skipped */
#define PALLAS_DEVERR_TOKEN 2u /* a token id outside [0, vocab) (prefill and
                                  decode); token 0's embedding row was used */

/* Decoder shape (Qwen3/Llama-style pre-norm decoder, Section 6.1 models). */
typedef struct {
  int32_t n_layers;
  int32_t hidden;     /* H */
  int32_t n_q_heads;  /* Hq */
  int32_t n_kv_heads; /* Hkv; Hq must be a multiple of it */
  int32_t head_dim;   /* d: 64 or 128 */
  int32_t ffn;        /* F */
  int32_t vocab;      /* V */
  float rms_eps;      /* RMSNorm epsilon (all norms) */
  float rope_theta;   /* rotary base */
  int32_t qk_norm;    /* 1: per-head RMSNorm of Q and K before rotary */
  int32_t page_size;  /* tokens per KV page; this build supports 16 */
} pallas_model_config;

/* Per-layer weights, device pointers to bf16, matrices row-major [out][in]:
 *   attn_norm [H]; w_qkv [(Hq + 2 Hkv) d][H] (rows: Q heads, K heads,
 *   V heads); q_norm [d]; k_norm [d] (ignored when qk_norm = 0);
 *   w_o [H][Hq d]; mlp_norm [H]; w_gate_up [2F][H] (rows: gate, then up);
 *   w_down [H][F].  Every pointer must be 16-byte aligned. */
typedef struct {
  const void* attn_norm;
  const void* w_qkv;
  const void* q_norm;
  const void* k_norm;
  const void* w_o;
  const void* mlp_norm;
  const void* w_gate_up;
  const void* w_down;
} pallas_layer_weights;

/* Global weights: embed [V][H], final_norm [H], lm_head [V][H] (device,
 * bf16); layers: host array of n_layers entries, copied at model creation. */
typedef struct {
  const void* embed;
  const void* final_norm;
  const void* lm_head;
  const pallas_layer_weights* layers;
} pallas_weights;

/* A paged KV pool: bf16 [n_layers][2 (K, V)][num_pages][page_size]
 * [n_kv_heads][head_dim] at `base` (device, 16-byte aligned).  K is stored
 * after rotary embedding. */
typedef struct {
  void* base;
  int32_t num_pages;
  int32_t page_size;
  int32_t n_layers;
  int32_t n_kv_heads;
  int32_t head_dim;
} pallas_kv_pool;

/* One transfer chunk to pack: positions [start_pos, start_pos + num_tokens)
 * of the source sequence, written as bf16 [L][2][num_tokens][Hkv][d] at byte
 * offset arena_offset (16-byte aligned) of the chunk arena. */
typedef struct {
  int32_t start_pos;
  int32_t num_tokens;
  uint64_t arena_offset;
} pallas_chunk_desc;

/* A received chunk: what the source sent with it (Section 4.3: logical
 * positions, request id, migration epoch) and where its payload
 * bf16 [n_layers][2][num_tokens][n_kv_heads][head_dim] sits in the arena. */
typedef struct {
  uint64_t request_id;
  uint64_t epoch;
  int32_t start_pos;
  int32_t num_tokens;
  uint64_t arena_offset;
  int32_t n_layers;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t elem_bytes;
} pallas_chunk_header;

typedef struct pallas_model pallas_model;

/* ABI version of the loaded library (PALLAS_ABI_VERSION). */
int32_t pallas_abi_version(void);

/* Message of the calling thread's last failed call ("" if none). */
const char* pallas_last_error(void);

/* Create a model handle over caller-owned weights (pointers are kept, bytes
 * are not copied).  Fails with INVALID_ARG on a null pointer or inconsistent
 * shape and UNSUPPORTED on a shape without kernels (head_dim other than 64 or
 * 128, page_size other than 16, hidden not a multiple of 64, ffn not a
 * multiple of 16, a GQA group other than 1, 2, 4 or 8 query heads per KV
 * head). */
int pallas_model_create(const pallas_model_config* cfg, const pallas_weights* w,
                        pallas_model** out);
void pallas_model_destroy(pallas_model* m);

/* Bytes of device workspace that prefill and decode need for up to
 * `max_tokens` tokens over up to `max_seqs` sequences in one call.
 *
 * The workspace (device, 256-byte aligned, owned by the caller) holds the
 * call's intermediate values.  One part of it is defined, for callers that
 * validate a model layer by layer: its first rows * hidden float32 values,
 * row-major [rows][hidden] in the call's row order, are the residual stream.
 * Once a call's work has completed they hold, after pallas_prefill_prefix
 * or pallas_prefill_chunk (rows = sum p_i), the residual entering the last
 * layer (the input of its RMSNorm), and after pallas_decode_step (rows =
 * num_seqs), the residual leaving the last layer (the input of the final
 * RMSNorm).  The rest of the workspace is undefined. */
size_t pallas_workspace_size(const pallas_model* m, int32_t max_tokens, int32_t max_seqs);

/* Prefix prefill (Section 4.3: the target rebuilds the KV cache of the
 * stable prefix by local prefill; Section 5: an ordinary prefill).
 *
 * Sequence i holds the ids d_token_ids[h_cu_seqlens[i] .. h_cu_seqlens[i+1])
 * (int32, device) at positions 0 .. p_i - 1.  For every layer, post-rotary K
 * and V of each token t are written to
 *   pool[l][0|1][bt_i[t / page]][t % page]
 * with bt_i = d_block_tables + i * max_pages (int32, device).  Nothing else
 * is written to the pool; no logits are produced.  num_seqs in
 * [1, PALLAS_MAX_SEQS]; 1 <= p_i <= PALLAS_MAX_PREFILL_LEN (UNSUPPORTED
 * beyond); sum p_i <= the workspace's max_tokens.  One layer's K plane of
 * the pool (num_pages * page * n_kv_heads * head_dim * 2 bytes) must not
 * exceed 4 GiB (UNSUPPORTED): attention addresses it with 32-bit offsets.
 * For the same reason the projections' bf16 operands must each stay below
 * 2 GiB (UNSUPPORTED): the call's activation matrices [M][hidden],
 * [M][n_q_heads * head_dim] and [M][ffn] with M = sum p_i, and the weight
 * matrices w_qkv, w_o, w_gate_up and w_down.  At hidden 5120, 64 query
 * heads of 128 and ffn 25600 that caps one call at 41,943 tokens.
 * Table entries outside [0, num_pages) are skipped and raise
 * PALLAS_DEVERR_PAGE, and token ids outside [0, vocab) raise
 * PALLAS_DEVERR_TOKEN, in *d_err (nullable, device, caller clears it). */
int pallas_prefill_prefix(pallas_model* m, int32_t num_seqs, const int32_t* d_token_ids,
                          const int32_t* h_cu_seqlens, const int32_t* d_block_tables,
                          int32_t max_pages, const pallas_kv_pool* pool, void* d_workspace,
                          size_t ws_bytes, int32_t* d_err, void* stream);

/* Chunked prefill (Section 4.5, contention with resident decoding: the
 * target interleaves prefix reconstruction with decode steps by prefilling
 * in chunks; the concurrency evaluation, Section 6.4, uses 256-token
 * chunks).
 *
 * As pallas_prefill_prefix, except that the ids of sequence i sit at
 * positions s_i .. s_i + p_i - 1 with s_i = h_start_pos[i] (host, >= 0), and
 * each of them attends to the K/V of positions [0, s_i) already in the pool
 * through the same block-table row (written by earlier calls, e.g. the
 * previous chunks) as well as to the chunk's own earlier positions.  Only
 * slots [s_i, s_i + p_i) are written.  A prefix prefilled chunk by chunk
 * gives the same cache, up to rounding, as one prefill over the whole
 * prefix.  Limits: s_i + p_i <= max_pages * page (OUT_OF_RANGE) and
 * <= PALLAS_MAX_PREFILL_LEN (UNSUPPORTED); sum p_i <= the workspace's
 * max_tokens; the 4 GiB K-plane and 2 GiB operand limits of
 * pallas_prefill_prefix.  Slots [0, s_i) are read, never checked: the
 * caller must have filled them. */
int pallas_prefill_chunk(pallas_model* m, int32_t num_seqs, const int32_t* d_token_ids,
                         const int32_t* h_cu_seqlens, const int32_t* h_start_pos,
                         const int32_t* d_block_tables, int32_t max_pages,
                         const pallas_kv_pool* pool, void* d_workspace, size_t ws_bytes,
                         int32_t* d_err, void* stream);

/* Suffix-block extraction (Section 4.3, Section 5: per-layer K/V of
 * completed blocks, taken by physical block id from the GPU cache).
 *
 * For each descriptor j and position t in [start, start + num_tokens):
 *   chunk_j[l][kv][t - start] = src[l][kv][bt[t / page]][t % page]
 * with bt = d_src_block_table (int32 [max_pages], device).  One launch covers
 * every descriptor.  Rejected (nothing written) when a range leaves
 * [0, max_pages * page), a chunk leaves the arena or two chunks overlap in
 * the arena.  Entries outside [0, num_pages) are skipped and raise
 * PALLAS_DEVERR_PAGE in *d_err (nullable). */
int pallas_pack_suffix_blocks(const pallas_kv_pool* src, const int32_t* d_src_block_table,
                              int32_t max_pages, const pallas_chunk_desc* h_descs,
                              int32_t n_descs, void* d_chunk_arena, size_t arena_bytes,
                              int32_t* d_err, void* stream);

/* Assembly into the target block table (Section 5: a new block table, then
 * a copy of the buffered suffix blocks; Section 4.3: state consistency).
 *
 * Host checks, in this order, each rejecting the whole call before anything
 * is enqueued: a header's shape differs from the pool (INVALID_ARG); its
 * request id differs from expected_request_id (WRONG_REQUEST); its epoch
 * differs from expected_epoch (STALE_EPOCH); its range leaves
 * [0, max_pages * page) or its payload leaves the arena (OUT_OF_RANGE); two
 * chunks claim one position (COVERAGE).  Then one launch writes
 *   dst[l][kv][bt[t / page]][t % page] = chunk[l][kv][t - start]
 * for every chunk and position; partial first and last pages are written
 * slot by slot and other slots of those pages keep their contents.  Table
 * entries outside [0, num_pages) are skipped and raise PALLAS_DEVERR_PAGE in
 * *d_err (nullable). */
int pallas_assemble_kv(const pallas_kv_pool* dst, const int32_t* d_dst_block_table,
                       int32_t max_pages, const pallas_chunk_header* h_hdrs,
                       const void* d_chunk_arena, size_t arena_bytes, int32_t n_chunks,
                       uint64_t expected_request_id, uint64_t expected_epoch,
                       int32_t* d_err, void* stream);

/* One decode step per sequence over its assembled cache (Section 4.3: the
 * target generates token n without repeating prefill over [0, n)).
 *
 * Sequence i feeds token d_tokens[i] (int32, device) at position
 * h_positions[i] = n_i; it attends to cached positions [0, n_i) and to
 * itself, writes its own K/V into slot n_i (the table needs capacity
 * n_i + 1), and the float32 logits of the next token go to
 * d_logits[i][0..V).  num_seqs in [1, PALLAS_MAX_SEQS]; 0 <= n_i <=
 * PALLAS_MAX_DECODE_POS (UNSUPPORTED beyond: decode attention keeps one
 * partial record per 64 keys in a workspace section of fixed size), and
 * n_i + 1 <= max_pages * page (OUT_OF_RANGE).  Up to 8 sequences run the
 * skinny projection kernel; more run the MFMA GEMM, whose 2 GiB operand
 * limit (see pallas_prefill_prefix) then also covers lm_head [V][hidden].
 * Table entries outside [0, num_pages) raise PALLAS_DEVERR_PAGE (the K/V
 * store of slot n_i is skipped; keys on such pages are masked), token ids
 * outside [0, vocab) PALLAS_DEVERR_TOKEN, in *d_err (nullable). */
int pallas_decode_step(pallas_model* m, int32_t num_seqs, const int32_t* d_tokens,
                       const int32_t* h_positions, const int32_t* d_block_tables,
                       int32_t max_pages, const pallas_kv_pool* pool, float* d_logits,
                       void* d_workspace, size_t ws_bytes, int32_t* d_err, void* stream);

/* Decode without a workspace, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  The same step as pallas_decode_step (the same checks,
 * kernels and results, bit for bit), with its intermediate values in a
 * scratch array of PALLAS_STATIC_SCRATCH_BYTES that the library keeps in
 * device memory on each GPU it runs on, from that GPU's first call until
 * the process ends.  The call allocates nothing; the caller still owns the
 * tokens, tables, pool and logits.  Every call on one GPU uses that GPU's
 * one array, so calls whose work overlaps on a GPU (different streams, or
 * host threads without ordering) race and give undefined results; calls
 * ordered on one stream do not.  Each call clears what must start at zero.
 * Limits, beyond those of pallas_decode_step (UNSUPPORTED): at most
 * PALLAS_STATIC_DECODE_MAX_SEQS sequences, and a scratch need within the
 * array: roughly num_seqs * n_q_heads * (max n_i / 64 + 1) * (head_dim + 2)
 * * 4 bytes of attention records plus the step's activations (at 64 query
 * heads of 128 and ffn 25600: 8 sequences up to position 15,743; fewer
 * up to 16,383).
 * HIP on a failed device query. */
#define PALLAS_STATIC_SCRATCH_BYTES (64u << 20)
#define PALLAS_STATIC_DECODE_MAX_SEQS 8
int pallas_decode_step_static(pallas_model* m, int32_t num_seqs, const int32_t* d_tokens,
                              const int32_t* h_positions, const int32_t* d_block_tables,
                              int32_t max_pages, const pallas_kv_pool* pool, float* d_logits,
                              int32_t* d_err, void* stream);

/* Coverage check (Section 4.3, "State consistency"), host only: returns
 * PALLAS_OK iff [0, prefix_len) and the ranges [h_starts[j], h_starts[j] +
 * h_lens[j]) together cover [0, n) exactly once (empty ranges are ignored),
 * PALLAS_ERR_COVERAGE otherwise, PALLAS_ERR_INVALID_ARG on null arrays with
 * n_ranges > 0 or negative lengths. */
int pallas_check_coverage(int32_t prefix_len, const int32_t* h_starts, const int32_t* h_lens,
                          int32_t n_ranges, int32_t n);

/* ------------------------------------------------------------------------
 * Scheduler Engine (host only, no GPU): when to start preparation.
 *
 * The prefetching-window model (Section 4.1, Eqs. 3-8) and its online
 * selection (Section 4.2, Eq. 9 and Algorithm 1).  For a candidate window
 * T_w (seconds before the predicted handover at which preparation starts),
 * with K_curr tokens in the context now and T_remain seconds predicted to
 * handover:
 *   L_hist  = K_curr + r_d (T_remain - T_w)          prefix at the trigger (Eq. 9)
 *   T_hist  = T_load + L_hist / r_p                   prefix reconstruction (Eq. 4)
 *   S_inc   = r_d T_w s_kv                            suffix bytes in the window (Eq. 3)
 *   T_res   = max(0, S_inc / B - T_w)                 suffix backlog at handover (Eq. 5)
 *   T_SIT   = T_0 + max(0, T_hist - T_w, T_res)       service interruption (Eq. 6)
 *   T_early = max(0, T_w - T_hist)                    early-preparation exposure (Eq. 7)
 *   J       = alpha T_SIT + (1 - alpha) T_early       objective (Eq. 8)
 * ------------------------------------------------------------------------ */
typedef struct {
  double r_p;     /* prefill throughput available to the migration at the target, tokens/s (> 0) */
  double r_d;     /* source-side decode throughput of the request, tokens/s (>= 0) */
  double goodput; /* inter-gNB goodput B available to the migration, bytes/s (> 0) */
  double s_kv;    /* KV-cache bytes per token, Eq. 1 (>= 0) */
  double t_load;  /* model load time at the target, s (>= 0; 0 when resident) */
  double t_0;     /* window-independent activation latency, s (>= 0) */
  double alpha;   /* objective weight in [0, 1] */
  double t_max;   /* largest window considered, s (>= 0) */
  double dt;      /* candidate grid step, s (> 0) */
} pallas_window_params;

typedef struct {
  double t_w;     /* the window */
  double cost;    /* J(t_w) */
  double t_sit;   /* T_SIT(t_w) */
  double t_early; /* T_early(t_w) */
  double t_hist;  /* T_hist(t_w) */
  double t_res;   /* T_res(t_w) */
  double l_hist;  /* L_hist(t_w), tokens */
  int32_t n_candidates; /* windows evaluated (selection only) */
  int32_t trigger;      /* selection only: 1 when T_remain <= t_w (start now), else 0 (defer) */
} pallas_window_decision;

/* The model at one window t_w (>= 0).  INVALID_ARG on a null pointer or a
 * parameter outside its range. */
int pallas_window_evaluate(const pallas_window_params* p, double k_curr, double t_remain, double t_w,
                           pallas_window_decision* out);

/* Algorithm 1's window decision: candidates {0, dt, 2 dt, ...} up to
 * T_limit = min(t_max, max(T_remain, 0)), plus T_limit itself when it is not
 * on the grid; the smallest J wins, the smallest window among equal J.
 * trigger = (T_remain <= t_w).  INVALID_ARG as above, or when the grid
 * would exceed 10^7 candidates. */
int pallas_window_select(const pallas_window_params* p, double k_curr, double t_remain,
                         pallas_window_decision* out);

/* Exponentially weighted moving average of a telemetry rate (Section 4.2:
 * r_p, r_d and B are smoothed): the first sample sets the value, later
 * ones move it by `weight` (in (0, 1]) towards the sample.  Returns the new
 * value (NaN and no change on a null pointer or a weight outside (0, 1]). */
typedef struct {
  double value;
  int32_t primed;
} pallas_ewma;
double pallas_ewma_update(pallas_ewma* e, double sample, double weight);

/* Admission (Section 4.2): 1 when the target runs a compatible model and
 * its free VRAM holds the request state expected at handover,
 * s_kv (K_curr + r_d max(T_remain, 0)) bytes; else 0. */
int32_t pallas_admit(int32_t model_compatible, double vram_free_bytes, double s_kv, double k_curr,
                     double r_d, double t_remain);

/* Bound on preparation discarded after wrong target predictions (Section
 * 4.4, Eq. 10): max(t_max + e_early - t_avail, 0) seconds. */
double pallas_waste_bound(double t_max, double e_early, double t_avail);

/* Per-kernel timing (tracing).  Kernel classes of the calls above: */
typedef enum {
  PALLAS_K_EMBED = 0,      /* token embedding + first RMSNorm */
  PALLAS_K_RMSNORM = 1,
  PALLAS_K_ROPE_TABLE = 2,
  PALLAS_K_GEMM_QKV = 3,   /* prefill Q|K|V projection (K|V only in the last layer) */
  PALLAS_K_QKV_EPI = 4,    /* QK-norm, rotary, paged K/V store */
  PALLAS_K_ATTN = 5,       /* prefill causal attention */
  PALLAS_K_GEMM_O = 6,     /* prefill output projection + residual */
  PALLAS_K_GEMM_GATE_UP = 7, /* prefill gate|up projection + SwiGLU */
  PALLAS_K_GEMM_DOWN = 8,  /* prefill down projection + residual */
  PALLAS_K_PACK = 9,
  PALLAS_K_ASSEMBLE = 10,
  PALLAS_K_DECODE_PROJ = 11, /* decode projections and lm_head */
  PALLAS_K_DECODE_ATTN = 12,
  PALLAS_K_COUNT = 13
} pallas_kernel_class;

/* Enable timing for the classes whose bit (1 << class) is set in
 * class_mask (0 disables).  Each timed launch is bracketed by two HIP events
 * recorded on the launch's stream; nothing else changes.  Process-wide and
 * serialised by a lock.  The first nonzero mask allocates the clock
 * counters (3 x PALLAS_K_COUNT uint64, kept until the process ends) on the
 * device current at that call; clock sampling covers launches on it. */
void pallas_profile_enable(uint32_t class_mask);

/* Wait for every recorded event pair, add its elapsed time to the class
 * totals, and copy the totals since the last reset: ms[k] (milliseconds) and
 * launches[k] for k < PALLAS_K_COUNT (host arrays of PALLAS_K_COUNT entries;
 * either may be NULL).  Returns PALLAS_ERR_HIP if an event query fails. */
int pallas_profile_read(double* ms, int64_t* launches);

/* Zero the class totals and drop pending event pairs. */
void pallas_profile_reset(void);

/* Mean shader clock inside the timed launches of one kernel class since the
 * last reset, in GHz (*mean_ghz; 0 when nothing was sampled), and the
 * number of workgroups sampled (*workgroups, nullable).  Each workgroup of
 * a sampled launch reads the shader-clock and constant-rate wall-clock
 * counters at its start and end; the ratio of the sums, scaled by the
 * wall-clock rate, is the clock the kernel actually ran at.  Sampled
 * classes: the prefill GEMMs.  Synchronizes the device.  INVALID_ARG for a
 * class outside [0, PALLAS_K_COUNT) or a null mean_ghz; HIP on a failed
 * copy. */
int pallas_profile_clock(int32_t kernel_class, double* mean_ghz, int64_t* workgroups);

#ifdef __cplusplus
}
#endif

#endif /* PALLAS_H */
