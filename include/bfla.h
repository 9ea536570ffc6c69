/*
 * bfla.h -- C ABI of the MI355X (gfx950) block-filtered sparse causal
 * prefill library (BFLA, "Block-Filtered Long-Context Attention
 * Mechanism", arXiv 2605.12193).
 *
 * The hot path is three stream-ordered calls:
 *
 *   bfla_estimate_mask   Stage 1 (Sec. 3.2): pooled block scores, block
 *                        softmax mass, keep-mass selection, GQA union
 *                        -> one keep mask per (request, KV head, query block).
 *   bfla_expand_rescue   Stage 2 tile mask (Sec. 3.2 end, Sec. 3.3): tile
 *                        expansion, local band, sink, stride and random
 *                        rescue -> compacted lists of kept KV tiles.
 *   bfla_sparse_prefill  Fused GQA prefill over the kept tiles only, exact
 *                        token-level causal attention inside them (eq27).
 *
 * plus bfla_dense_prefill, the same prefill over every causal tile (the
 * dense baseline, eq:vsa with a causal mask).
 *
 * Equations are named by their LaTeX labels in the paper (eq9 ... eq27 are
 * printed as (3) ... (21)).
 *
 * Conventions (all entry points):
 *  - Tensors are DEVICE pointers; structs and the arrays they point to are
 *    HOST memory read during the call only.  The caller owns all memory; the
 *    library never allocates or frees device memory.
 *  - bf16 is IEEE bfloat16 stored in 16 bits.  head_dim is always the
 *    contiguous (stride 1) dimension.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = default stream) and
 *    returns without synchronising.  Pointers must stay valid until the
 *    stream work completes.
 *  - Every argument check happens before any launch: on error nothing has
 *    been enqueued and the outputs are untouched.
 *  - Outputs are fully overwritten and bit-identical across runs (no
 *    floating-point atomics).
 *  - Calls only launch kernels (no allocation, memset, copy or
 *    synchronisation), so they can be captured into a HIP graph; run each
 *    kernel shape once outside capture first (its first launch sets the
 *    kernel's dynamic-LDS attribute).
 *  - No C++ exception crosses the ABI.  There is no global mutable state;
 *    the last error message is thread-local.
 */
#ifndef BFLA_H
#define BFLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BFLA_VERSION_STRING "0.2.0"
/* Maximum number of requests per call.  The kernels take the descriptors of
 * up to 32 requests in their arguments, so a larger batch launches each
 * kernel once per group of 32 requests. */
#define BFLA_MAX_BATCH 65536

typedef enum bfla_status {
  BFLA_OK = 0,
  BFLA_ERR_INVALID_ARG = 1,  /* null pointer, bad size, out-of-range value */
  BFLA_ERR_UNSUPPORTED = 2,  /* valid but not built: head_dim, tile, block, m */
  BFLA_ERR_WORKSPACE = 3,    /* workspace smaller than bfla_workspace_size */
  BFLA_ERR_CAPACITY = 4,     /* cols capacity below bfla_list_capacity */
  BFLA_ERR_HIP = 5           /* a HIP launch failed; see bfla_last_error */
} bfla_status;

/* Problem statement (eq2-eq3): head-first Q [H_q][N_q][C] and K/V
 * [H_kv][N_kv][C] per request, GQA group size m = H_q / H_kv (1 to 8 are
 * built); query head p reads KV head floor(p / m) (eq8).  Request r has N_q = n_q[r] query tokens
 * that are the LAST N_q of its N_kv = n_kv[r] tokens (chunked prefill with a
 * prefix of N_c = N_kv - N_q tokens, eq11). */
typedef struct bfla_problem {
  int32_t batch;        /* B, 1..BFLA_MAX_BATCH */
  int32_t h_q;          /* query heads */
  int32_t h_kv;         /* KV heads, h_q % h_kv == 0 */
  int32_t head_dim;     /* C: 64, 128 or 256 */
  const int32_t* n_q;   /* host [batch], >= 1 */
  const int32_t* n_kv;  /* host [batch], n_kv[r] >= n_q[r] */
} bfla_problem;

/* Addressing of a per-request [heads][tokens][head_dim] bf16 tensor (Q or
 * O): element (r, p, t, c) sits at
 *     data + off(r) + p * stride_head + t * stride_tok + c      (elements)
 * with off(r) = batch_offset[r] if batch_offset != NULL else
 * r * stride_batch.  This covers both a padded [B][H][N][C] tensor and a
 * packed token-major [sum N][H][C] varlen tensor. */
typedef struct bfla_view {
  void* data;                   /* device, bf16 */
  const int64_t* batch_offset;  /* host [batch] or NULL */
  int64_t stride_batch;
  int64_t stride_head;
  int64_t stride_tok;
} bfla_view;

enum { BFLA_KV_CONTIGUOUS = 0, BFLA_KV_PAGED = 1 };

/* K and V (same layout, separate base pointers).
 * CONTIGUOUS: element (r, h, t, c) at  base + off(r) + h*stride_head +
 *             t*stride_tok + c, off(r) as in bfla_view.  One KV head of one
 *             request must span less than 2 GiB.
 * PAGED (vLLM-style): token t of request r lives in page
 *             P = block_table[r * max_pages + t / page_size]
 *             at  base + P*page_stride + (t % page_size)*stride_tok +
 *             h*stride_head + c.  The pool holds n_pages pages and must be
 *             smaller than 2 GiB; a table entry outside [0, n_pages) reads as
 *             zeros (never out of bounds).  head_dim <= stride_tok < 2^24
 *             (BFLA_ERR_INVALID_ARG below, BFLA_ERR_UNSUPPORTED above). */
typedef struct bfla_kv {
  int32_t layout;               /* BFLA_KV_CONTIGUOUS or BFLA_KV_PAGED */
  const void* k;                /* device, bf16 */
  const void* v;                /* device, bf16 */
  const int64_t* batch_offset;  /* CONTIGUOUS: host [batch] or NULL */
  int64_t stride_batch;         /* CONTIGUOUS */
  int64_t stride_head;
  int64_t stride_tok;
  int32_t page_size;            /* PAGED: tokens per page, a power of two >= 16 */
  int32_t max_pages;            /* PAGED: row length of block_table */
  int64_t page_stride;          /* PAGED: elements between pages */
  const int32_t* block_table;   /* PAGED: device [batch][max_pages] */
  int64_t n_pages;              /* PAGED: pages in the pool */
} bfla_kv;

/* Method hyper-parameters. */
typedef struct bfla_params {
  int32_t block;    /* b, coarse block size (eq4); multiple of tile and group */
  int32_t group;    /* g, flattening group (eq6); b / g in {1, 2, 4, 8, 16} */
  int32_t tile;     /* T, attention tile (eq19); 64 */
  float gamma;      /* keep-mass threshold (eq17), 0 < gamma <= 1 */
  int32_t n_local;  /* local band (eq21): diagonal tile + n_local before it;
                       -1 switches the band off (diagonal included) */
  int32_t n_sink;   /* sink tiles kt < n_sink (eq22), >= 0 */
  int32_t eta;      /* stride rescue period (eq24), 0 = off */
  double rho;       /* random rescue probability (eq25), 0 <= rho <= 1 */
  uint64_t seed;    /* s, seed of chi and psi (eq24-eq25) */
  float scale;      /* alpha of eq15 and the 1/sqrt(C) of eq27; 0 -> 1/sqrt(C) */
} bfla_params;

/* ---------------------------------------------------------------------
 * Output layouts (all packed per request in request order):
 *  block_mask  uint8 [H_kv][L_q][L_kv] per request, L = ceil(N / b);
 *              request r starts at sum_{r'<r} H_kv*L_q(r')*L_kv(r').
 *              1 = keep, 0 = drop (also every non-causal cell).
 *  dbg_scores  float [H_q][L_q][L_kv] per request (block scores S of eq10,
 *              -inf where not causal, eq14).
 *  dbg_head_mask  uint8 [H_q][L_q][L_kv] per request, at the same element
 *              offsets as dbg_scores: the keep set of each query head
 *              before the GQA union (eq18), 1 = kept by that head.
 *  lists       rows ordered (request, KV head, q-tile): row index
 *              sum_{r'<r} H_kv*T_q(r') + h*T_q(r) + qt, T_q = ceil(N_q/T).
 *              row_ptr int32 [n_rows + 1] (row_ptr[0] = 0), cols int32
 *              ascending KV-tile indices of each row (local to the request).
 *  O           bf16 through its bfla_view, every query row written.
 *  lse         float [H_q][N_q] per request (natural-log log-sum-exp of the
 *              scaled logits of each query; -inf for a query that kept no
 *              key); request r starts at sum_{r'<r} H_q*N_q(r').
 * ------------------------------------------------------------------- */

enum { BFLA_WS_ESTIMATE = 1, BFLA_WS_EXPAND = 2 };

/* Bytes of device workspace the call `which` needs (0 is possible): for
 * BFLA_WS_ESTIMATE the split score GEMM's partial sums plus the block
 * scores (enough with or without dbg_scores); for BFLA_WS_EXPAND the row
 * counts and keep ballots of the tile stage. */
int bfla_workspace_size(const bfla_problem* prob, const bfla_params* params,
                        int which, size_t* bytes);

/* Sizes of the list outputs: n_rows (row_ptr has n_rows + 1 entries) and
 * max_cols, the number of causal tiles (an upper bound of every list total).
 * Also returns the sizes of block_mask (mask_bytes) and dbg_scores
 * (score_elems); any output pointer may be NULL. */
int bfla_list_capacity(const bfla_problem* prob, const bfla_params* params,
                       size_t* n_rows, size_t* max_cols, size_t* mask_bytes,
                       size_t* score_elems);

/* Stage 1, Sec. 3.2 (eq4-eq18) plus the GQA union: per request, query head
 * p and query block i, block scores S_{p,i,j} = max over group pairs of the
 * dot products of flattened g-token groups (eq9-eq10), causal blocks only
 * (eq11-eq14); block softmax A = softmax_j(alpha S) (eq15); keep the
 * shortest prefix of blocks in descending order whose mass reaches gamma
 * (eq16-eq18; ties: lower block index first; gamma >= 1 keeps all causal
 * blocks); OR over the m query heads of each KV head.
 *   q              Q view (bf16).
 *   kv             K (and V, unused here) descriptor.
 *   block_mask     out, device uint8, layout above.
 *   dbg_scores     out, device float or NULL (then the workspace holds them).
 *   dbg_head_mask  out, device uint8 or NULL: the per-query-head keep sets
 *                  of eq18 that the union combines (layout above).
 *   workspace      device scratch, 256-byte aligned, of
 *                  bfla_workspace_size(BFLA_WS_ESTIMATE) bytes: it holds the
 *                  partial sums of the score GEMM when the problem has too
 *                  few score tiles to fill the GPU and the GEMM's inner
 *                  dimension is split (added in a fixed order, so results
 *                  stay bit-identical run to run), then the block scores
 *                  when dbg_scores is NULL.  With dbg_scores given, only the
 *                  partial sums are needed (NULL / 0 is enough when there
 *                  are none).
 * Errors: INVALID_ARG, UNSUPPORTED (also: m > 8; more than 65536 KV blocks
 * per request; q rows of 256 * g consecutive tokens spanning 2 GiB or more,
 * i.e. (256 g - 1) * stride_tok + head_dim >= 2^30; paged K where
 * ceil(128 g / page_size) + 1 exceeds 2056 pages, e.g. g = 512 with 16-token
 * pages), WORKSPACE, HIP. */
int bfla_estimate_mask(const bfla_problem* prob, const bfla_params* params,
                       const bfla_view* q, const bfla_kv* kv,
                       uint8_t* block_mask, float* dbg_scores,
                       uint8_t* dbg_head_mask, void* workspace,
                       size_t ws_bytes, void* stream);

/* Stage 2 tile mask, eq19-eq26: tile (qt, kt) of KV head h inherits block
 * (qt / (b/T), kt / (b/T)) of block_mask, clipped to causal tiles; the
 * diagonal tile and n_local tiles before it (eq21) and KV tiles kt < n_sink
 * (eq22) are kept; each dropped causal tile (eq23) is rescued if
 * chi(qt, kt; s) mod eta == 0 (eq24) or psi(h, qt, kt; s) < rho (eq25),
 *   chi  = mix64(mix64(s)     ^ (qt << 21 | kt)),
 *   psi  = (mix64(mix64(s+1) ^ ((h+1) << 42 | qt << 21 | kt)) >> 40) / 2^24,
 * mix64 = the SplitMix64 output mix (Steele, Lea, Flood, OOPSLA 2014); the
 * final mask (eq26) is compacted into ascending lists.
 *   block_mask     in, device uint8 (layout above).
 *   row_ptr, cols  out, device int32 (layout above).
 *   cols_capacity  entries available at cols; must be >= max_cols of
 *                  bfla_list_capacity (else CAPACITY).
 *   workspace      device scratch of >= bfla_workspace_size(BFLA_WS_EXPAND),
 *                  8-byte aligned (else INVALID_ARG); holds per-row counts and
 *                  the keep / drop bits of every causal tile between passes.
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, CAPACITY, HIP. */
int bfla_expand_rescue(const bfla_problem* prob, const bfla_params* params,
                       const uint8_t* block_mask, int32_t* row_ptr,
                       int32_t* cols, size_t cols_capacity, void* workspace,
                       size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * bfla_expand_rescue with its workspace (per-row counts and keep ballots)
 * taken from a fixed scratch buffer that the library holds on each GPU it
 * runs on until the process ends, BFLA_EXPAND_SCRATCH_BYTES large; nothing
 * is allocated.  Same arguments, outputs and errors as bfla_expand_rescue
 * without the workspace; a problem whose workspace would exceed the scratch
 * (bfla_workspace_size(BFLA_WS_EXPAND) > BFLA_EXPAND_SCRATCH_BYTES) is
 * rejected with BFLA_ERR_WORKSPACE before anything is enqueued.
 *   stream  must belong to the current device (its scratch is used).
 * The scratch of a device is shared by every call on it and keeps the last
 * call's contents (nothing in it needs clearing: every call writes each
 * word it reads); calls that overlap on one GPU (different streams, or
 * threads without ordering between them) race on it and must be serialised
 * by the caller.  The first call on a device looks the buffer up
 * (hipGetSymbolAddress); make that call outside graph capture.
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, CAPACITY, HIP. */
#define BFLA_EXPAND_SCRATCH_BYTES (16u << 20)
int bfla_expand_rescue_noalloc(const bfla_problem* prob, const bfla_params* params,
                               const uint8_t* block_mask, int32_t* row_ptr,
                               int32_t* cols, size_t cols_capacity, void* stream);

/* Final sparse attention, eq27: for every query head p and query t (absolute
 * position N_c + t) of every request, softmax(scale * q.k) over the keys k
 * with k <= N_c + t whose tile is in the list of (request, floor(p/m),
 * floor(t/T)); O = weights * V.  Dropped tiles are never loaded.
 *   q, o     Q in, O out (bf16 views).
 *   kv       K/V descriptor.
 *   row_ptr, cols  lists from bfla_expand_rescue (or any ascending lists of
 *            causal tiles; an entry outside [0, ceil(N_kv/T)) contributes no
 *            key).  row_ptr must be non-decreasing with row_ptr[0] = 0.
 *   lse      out, device float or NULL.
 * A query that keeps no key gets O = 0 and lse = -inf.
 * Errors: INVALID_ARG, UNSUPPORTED, HIP. */
int bfla_sparse_prefill(const bfla_problem* prob, const bfla_params* params,
                        const bfla_view* q, const bfla_kv* kv,
                        const int32_t* row_ptr, const int32_t* cols,
                        const bfla_view* o, float* lse, void* stream);

/* Dense causal prefill (eq:vsa with the causal mask of the appendix): the
 * same kernel with every causal KV tile of each row.  Only params->tile and
 * params->scale are used (the other fields must still be valid).
 * Errors: INVALID_ARG, UNSUPPORTED, HIP. */
int bfla_dense_prefill(const bfla_problem* prob, const bfla_params* params,
                       const bfla_view* q, const bfla_kv* kv,
                       const bfla_view* o, float* lse, void* stream);

/* Static description of a status code. */
const char* bfla_status_string(int status);
/* Message of the last failing call on this thread ("" if none). */
const char* bfla_last_error(void);
/* Library version, BFLA_VERSION_STRING. */
const char* bfla_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BFLA_H */
