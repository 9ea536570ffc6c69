// C ABI of the BFLA sparse-prefill library: argument validation, output and
// workspace sizing, request descriptors, kernel dispatch.  Every check runs
// before the first launch; nothing here allocates device memory.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <string>
#include <vector>

#include "bfla.h"
#include "bfla_internal.h"

using namespace bfla;

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  g_last_error.clear();
  return BFLA_OK;
}

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

constexpr int kTile = 64;
constexpr int64_t kMaxTiles = int64_t(1) << 21;  // pack() field width of chi/psi
constexpr int64_t kMaxBlocksPerRow = 65536;       // keep bits of one row held in LDS

// Per-request sizes derived from the problem and parameters.
struct Sizes {
  int64_t n_rows = 0;      // list rows
  int64_t max_cols = 0;    // causal tiles
  int64_t mask_bytes = 0;  // block mask
  int64_t score_elems = 0; // block scores
  int64_t lse_elems = 0;
  int64_t max_t_kv = 0;    // KV tiles of the longest request
};

int64_t causal_tiles(int n_q, int n_kv, int T) {
  int64_t n_c = n_kv - n_q, total = 0;
  int64_t t_q = cdiv(n_q, T);
  for (int64_t qt = 0; qt < t_q; ++qt) {
    int64_t last = std::min<int64_t>(n_c + (qt + 1) * T - 1, n_kv - 1);
    total += last / T + 1;
  }
  return total;
}

int check_problem(const bfla_problem* prob, const bfla_params* pr) {
  if (!prob) return fail(BFLA_ERR_INVALID_ARG, "problem is NULL");
  if (!pr) return fail(BFLA_ERR_INVALID_ARG, "params is NULL");
  if (prob->batch < 1 || prob->batch > BFLA_MAX_BATCH)
    return fail(BFLA_ERR_INVALID_ARG, "batch %d outside [1, %d]", prob->batch, BFLA_MAX_BATCH);
  if (prob->h_q < 1 || prob->h_kv < 1)
    return fail(BFLA_ERR_INVALID_ARG, "head counts must be positive (h_q=%d h_kv=%d)",
                prob->h_q, prob->h_kv);
  if (prob->h_q % prob->h_kv)
    return fail(BFLA_ERR_INVALID_ARG, "h_q=%d is not a multiple of h_kv=%d", prob->h_q,
                prob->h_kv);
  if (prob->head_dim != 64 && prob->head_dim != 128 && prob->head_dim != 256)
    return fail(BFLA_ERR_UNSUPPORTED, "head_dim %d not in {64, 128, 256}", prob->head_dim);
  if (!prob->n_q || !prob->n_kv) return fail(BFLA_ERR_INVALID_ARG, "n_q / n_kv is NULL");
  if (pr->tile != kTile) return fail(BFLA_ERR_UNSUPPORTED, "tile %d != 64", pr->tile);
  if (pr->block < kTile || pr->block % kTile)
    return fail(BFLA_ERR_UNSUPPORTED, "block %d is not a positive multiple of tile 64",
                pr->block);
  if (pr->group < 1 || pr->block % pr->group)
    return fail(BFLA_ERR_INVALID_ARG, "block %d is not a multiple of group %d", pr->block,
                pr->group);
  if (!(pr->gamma > 0.f && pr->gamma <= 1.f))
    return fail(BFLA_ERR_INVALID_ARG, "gamma %g outside (0, 1]", (double)pr->gamma);
  if (pr->n_local < -1) return fail(BFLA_ERR_INVALID_ARG, "n_local %d < -1", pr->n_local);
  if (pr->n_sink < 0) return fail(BFLA_ERR_INVALID_ARG, "n_sink %d < 0", pr->n_sink);
  if (pr->eta < 0) return fail(BFLA_ERR_INVALID_ARG, "eta %d < 0", pr->eta);
  if (!(pr->rho >= 0.0 && pr->rho <= 1.0))
    return fail(BFLA_ERR_INVALID_ARG, "rho %g outside [0, 1]", pr->rho);
  if (!(pr->scale >= 0.f) || isinf(pr->scale))
    return fail(BFLA_ERR_INVALID_ARG, "scale %g must be finite and >= 0", (double)pr->scale);
  for (int r = 0; r < prob->batch; ++r) {
    int nq = prob->n_q[r], nkv = prob->n_kv[r];
    if (nq < 1 || nkv < nq)
      return fail(BFLA_ERR_INVALID_ARG, "request %d: need 1 <= n_q (%d) <= n_kv (%d)", r, nq,
                  nkv);
    if (cdiv(nkv, kTile) >= kMaxTiles)
      return fail(BFLA_ERR_UNSUPPORTED, "request %d: n_kv %d exceeds 2^21 tiles", r, nkv);
  }
  return BFLA_OK;
}

Sizes sizes_of(const bfla_problem* prob, const bfla_params* pr) {
  Sizes s;
  for (int r = 0; r < prob->batch; ++r) {
    int nq = prob->n_q[r], nkv = prob->n_kv[r];
    int64_t lq = cdiv(nq, pr->block), lkv = cdiv(nkv, pr->block);
    s.n_rows += prob->h_kv * cdiv(nq, pr->tile);
    s.max_cols += prob->h_kv * causal_tiles(nq, nkv, pr->tile);
    s.mask_bytes += prob->h_kv * lq * lkv;
    s.score_elems += prob->h_q * lq * lkv;
    s.lse_elems += (int64_t)prob->h_q * nq;
    s.max_t_kv = std::max<int64_t>(s.max_t_kv, cdiv(nkv, pr->tile));
  }
  return s;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

int check_view(const bfla_problem* prob, const bfla_view* v, const char* name) {
  if (!v) return fail(BFLA_ERR_INVALID_ARG, "%s view is NULL", name);
  if (!v->data) return fail(BFLA_ERR_INVALID_ARG, "%s data is NULL", name);
  if (!aligned16(v->data)) return fail(BFLA_ERR_INVALID_ARG, "%s data not 16-byte aligned", name);
  if (v->stride_head % 8 || v->stride_tok % 8 || v->stride_batch % 8)
    return fail(BFLA_ERR_INVALID_ARG, "%s strides must be multiples of 8 elements", name);
  if (v->stride_tok < 1 || v->stride_head < 1)
    return fail(BFLA_ERR_INVALID_ARG, "%s strides must be positive", name);
  if (v->batch_offset)
    for (int r = 0; r < prob->batch; ++r)
      if (v->batch_offset[r] < 0 || v->batch_offset[r] % 8)
        return fail(BFLA_ERR_INVALID_ARG, "%s batch_offset[%d] invalid", name, r);
  return BFLA_OK;
}

int check_kv(const bfla_problem* prob, const bfla_kv* kv, bool need_v) {
  if (!kv) return fail(BFLA_ERR_INVALID_ARG, "kv is NULL");
  if (!kv->k || (need_v && !kv->v)) return fail(BFLA_ERR_INVALID_ARG, "k / v is NULL");
  if (!aligned16(kv->k) || (need_v && !aligned16(kv->v)))
    return fail(BFLA_ERR_INVALID_ARG, "k / v not 16-byte aligned");
  if (kv->stride_head % 8 || kv->stride_tok % 8 || kv->stride_head < 1 || kv->stride_tok < 1)
    return fail(BFLA_ERR_INVALID_ARG, "kv strides must be positive multiples of 8");
  if (kv->layout == BFLA_KV_CONTIGUOUS) {
    if (kv->stride_batch % 8) return fail(BFLA_ERR_INVALID_ARG, "kv stride_batch %% 8 != 0");
    // one KV head of one request is read through a buffer descriptor whose
    // byte range is a signed 32-bit count
    for (int r = 0; r < prob->batch; ++r)
      if ((int64_t)(prob->n_kv[r] - 1) * kv->stride_tok + prob->head_dim >= (int64_t(1) << 30))
        return fail(BFLA_ERR_UNSUPPORTED, "request %d: one KV head spans >= 2 GiB", r);
    if (kv->batch_offset)
      for (int r = 0; r < prob->batch; ++r)
        if (kv->batch_offset[r] < 0 || kv->batch_offset[r] % 8)
          return fail(BFLA_ERR_INVALID_ARG, "kv batch_offset[%d] invalid", r);
  } else if (kv->layout == BFLA_KV_PAGED) {
    if (kv->page_size < 16 || (kv->page_size & (kv->page_size - 1)))
      return fail(BFLA_ERR_UNSUPPORTED, "page_size %d is not a power of two >= 16",
                  kv->page_size);
    if (kv->n_pages < 1) return fail(BFLA_ERR_INVALID_ARG, "n_pages %lld < 1",
                                     (long long)kv->n_pages);
    if ((kv->n_pages - 1) * kv->page_stride + (int64_t)kv->page_size * kv->stride_tok >=
        (int64_t(1) << 30))
      return fail(BFLA_ERR_UNSUPPORTED, "page pool spans >= 2 GiB");
    if (!kv->block_table) return fail(BFLA_ERR_INVALID_ARG, "block_table is NULL");
    if (kv->page_stride % 8 || kv->page_stride < 1)
      return fail(BFLA_ERR_INVALID_ARG, "page_stride must be a positive multiple of 8");
    // the prefill addresses a 64-token tile as if contiguous and maps it onto
    // its pages: token rows must not overlap and a tile must span < 2 GiB
    if (kv->stride_tok < prob->head_dim)
      return fail(BFLA_ERR_INVALID_ARG, "paged stride_tok %lld < head_dim %d",
                  (long long)kv->stride_tok, prob->head_dim);
    if (kv->stride_tok >= (int64_t(1) << 24))
      return fail(BFLA_ERR_UNSUPPORTED, "paged stride_tok %lld >= 2^24",
                  (long long)kv->stride_tok);
    for (int r = 0; r < prob->batch; ++r)
      if (cdiv(prob->n_kv[r], kv->page_size) > kv->max_pages)
        return fail(BFLA_ERR_INVALID_ARG, "request %d needs %lld pages > max_pages %d", r,
                    (long long)cdiv(prob->n_kv[r], kv->page_size), kv->max_pages);
  } else {
    return fail(BFLA_ERR_INVALID_ARG, "kv layout %d unknown", kv->layout);
  }
  return BFLA_OK;
}

KvAddr kv_addr(const bfla_kv* kv) {
  KvAddr a{};
  a.k = static_cast<const bf16_t*>(kv->k);
  a.v = static_cast<const bf16_t*>(kv->v);
  a.stride_head = kv->stride_head;
  a.stride_tok = kv->stride_tok;
  a.paged = kv->layout == BFLA_KV_PAGED;
  if (a.paged) {
    a.block_table = kv->block_table;
    a.page_stride = kv->page_stride;
    a.page_size = kv->page_size;
    a.max_pages = kv->max_pages;
    a.n_pages = (int32_t)kv->n_pages;
    a.pool_bytes = (uint32_t)(((kv->n_pages - 1) * kv->page_stride +
                               (int64_t)kv->page_size * kv->stride_tok) * 2);
  }
  return a;
}

int64_t view_off(const bfla_view* v, int r) {
  return v->batch_offset ? v->batch_offset[r] : (int64_t)r * v->stride_batch;
}

// Request descriptors in request order (offsets of every packed output).
std::vector<ReqDesc> make_batch(const bfla_problem* prob, const bfla_params* pr,
                                const bfla_view* q, const bfla_view* o, const bfla_kv* kv) {
  std::vector<ReqDesc> b((size_t)prob->batch);
  int64_t row = 0, mask = 0, score = 0, lse = 0;
  for (int r = 0; r < prob->batch; ++r) {
    ReqDesc& d = b[(size_t)r];
    d = ReqDesc{};
    d.n_q = prob->n_q[r];
    d.n_kv = prob->n_kv[r];
    d.l_q = (int32_t)cdiv(d.n_q, pr->block);
    d.l_kv = (int32_t)cdiv(d.n_kv, pr->block);
    d.t_q = (int32_t)cdiv(d.n_q, pr->tile);
    d.t_kv = (int32_t)cdiv(d.n_kv, pr->tile);
    d.q_off = q ? view_off(q, r) : 0;
    d.o_off = o ? view_off(o, r) : 0;
    d.kv_off = (kv && kv->layout == BFLA_KV_CONTIGUOUS)
                   ? (kv->batch_offset ? kv->batch_offset[r] : (int64_t)r * kv->stride_batch)
                   : 0;
    d.lse_off = lse;
    d.mask_off = mask;
    d.score_off = score;
    d.row_base = (int32_t)row;
    d.bt_row = r;
    row += (int64_t)prob->h_kv * d.t_q;
    mask += (int64_t)prob->h_kv * d.l_q * d.l_kv;
    score += (int64_t)prob->h_q * d.l_q * d.l_kv;
    lse += (int64_t)prob->h_q * d.n_q;
  }
  return b;
}

// Longest requests first (their rows are the longest work items).
std::vector<ReqDesc> longest_first(std::vector<ReqDesc> b) {
  std::stable_sort(b.begin(), b.end(),
                   [](const ReqDesc& x, const ReqDesc& y) { return x.n_kv > y.n_kv; });
  return b;
}

// Stage 1 runs once per group of kLaunchRequests requests (in request order),
// each group with its own split of the score GEMM; the groups share one
// partial-sum buffer in stream order, sized for the largest.
struct Stage1Layout {
  std::vector<int32_t> splits;
  size_t partial_bytes = 0;
};

Stage1Layout stage1_layout(const bfla_problem* prob, const bfla_params* pr) {
  Stage1Layout lay;
  for (int g0 = 0; g0 < prob->batch; g0 += kLaunchRequests) {
    const int n = std::min(kLaunchRequests, prob->batch - g0);
    const EstimatePlan plan = estimate_plan(prob->n_q + g0, prob->n_kv + g0, n, prob->h_q,
                                            prob->head_dim, pr->block, pr->group);
    lay.splits.push_back(plan.split);
    lay.partial_bytes = std::max(lay.partial_bytes, plan.partial_bytes);
  }
  return lay;
}

float scale_of(const bfla_problem* prob, const bfla_params* pr) {
  return pr->scale > 0.f ? pr->scale : 1.0f / sqrtf((float)prob->head_dim);
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(BFLA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

int check_rows_fit(const Sizes& s) {
  if (s.n_rows >= INT32_MAX || s.max_cols >= INT32_MAX)
    return fail(BFLA_ERR_UNSUPPORTED, "list sizes exceed int32");
  return BFLA_OK;
}

int prefill_common(const bfla_problem* prob, const bfla_params* pr, const bfla_view* q,
                   const bfla_kv* kv, const bfla_view* o, PrefillLaunch* L) {
  int st;
  if ((st = check_problem(prob, pr))) return st;
  if ((st = check_view(prob, q, "q"))) return st;
  if ((st = check_view(prob, o, "o"))) return st;
  if ((st = check_kv(prob, kv, true))) return st;
  if ((st = check_rows_fit(sizes_of(prob, pr)))) return st;
  if (!prefill_supported(prob->head_dim, prob->h_q / prob->h_kv))
    return fail(BFLA_ERR_UNSUPPORTED, "GQA group size %d not built (1 to 8)",
                prob->h_q / prob->h_kv);
  L->q = q->data;
  L->o = o->data;
  L->q_sh = q->stride_head;
  L->q_st = q->stride_tok;
  L->o_sh = o->stride_head;
  L->o_st = o->stride_tok;
  L->kv = kv_addr(kv);
  L->h_q = prob->h_q;
  L->h_kv = prob->h_kv;
  L->head_dim = prob->head_dim;
  L->scale = scale_of(prob, pr);
  L->reqs = longest_first(make_batch(prob, pr, q, o, kv));
  return BFLA_OK;
}

// Stage-1 workspace: the partial sums of a split score GEMM first, then the
// block scores when the caller passes no dbg_scores.
size_t estimate_ws_scores_offset(const Stage1Layout& plan) {
  return (plan.partial_bytes + 255) / 256 * 256;
}

int expand_common(const bfla_problem* prob, const bfla_params* params,
                  const uint8_t* block_mask, int32_t* row_ptr, int32_t* cols,
                  size_t cols_capacity, void* workspace, size_t ws_bytes, bool use_scratch,
                  void* stream) {
  int st;
  if ((st = check_problem(prob, params))) return st;
  if (!block_mask || !row_ptr || !cols)
    return fail(BFLA_ERR_INVALID_ARG, "block_mask / row_ptr / cols is NULL");
  Sizes s = sizes_of(prob, params);
  if ((st = check_rows_fit(s))) return st;
  if (cols_capacity < (size_t)s.max_cols)
    return fail(BFLA_ERR_CAPACITY, "cols capacity %zu < %lld causal tiles", cols_capacity,
                (long long)s.max_cols);
  size_t need = expand_workspace_bytes(s.n_rows, s.max_t_kv);
  if (use_scratch) {
    if (need > (size_t)BFLA_EXPAND_SCRATCH_BYTES)
      return fail(BFLA_ERR_WORKSPACE,
                  "tile stage needs %zu bytes of workspace, more than the %zu-byte scratch "
                  "of bfla_expand_rescue_noalloc", need, (size_t)BFLA_EXPAND_SCRATCH_BYTES);
    hipError_t e = expand_scratch(&workspace);
    if (e != hipSuccess) return hip_status(e, "expand_rescue_noalloc scratch lookup");
    ws_bytes = BFLA_EXPAND_SCRATCH_BYTES;
  }
  if (!workspace || ws_bytes < need)
    return fail(BFLA_ERR_WORKSPACE, "expand workspace %zu < %zu bytes", ws_bytes, need);
  if (reinterpret_cast<uintptr_t>(workspace) & 7)
    return fail(BFLA_ERR_INVALID_ARG, "expand workspace not 8-byte aligned");
  ExpandLaunch L{};
  L.block_mask = block_mask;
  L.row_ptr = row_ptr;
  L.cols = cols;
  L.counts = static_cast<int32_t*>(workspace);
  L.partial = L.counts + ((s.n_rows + 63) / 64) * 64;
  L.words_per_row = (int32_t)((s.max_t_kv + 63) / 64);
  L.bits = reinterpret_cast<uint64_t*>(L.partial + 64);
  L.n_rows = (int32_t)s.n_rows;
  L.h_kv = prob->h_kv;
  L.rb = params->block / params->tile;
  L.n_local = params->n_local;
  L.n_sink = params->n_sink;
  L.eta = params->eta;
  L.rho24 = (uint32_t)floor(params->rho * 16777216.0);
  L.seed = params->seed;
  L.reqs = make_batch(prob, params, nullptr, nullptr, nullptr);
  return hip_status(launch_expand(L, static_cast<hipStream_t>(stream)),
                    use_scratch ? "expand_rescue_noalloc" : "expand_rescue");
}

}  // namespace

extern "C" {

const char* bfla_version(void) { return BFLA_VERSION_STRING; }

const char* bfla_last_error(void) { return g_last_error.c_str(); }

const char* bfla_status_string(int status) {
  switch (status) {
    case BFLA_OK: return "ok";
    case BFLA_ERR_INVALID_ARG: return "invalid argument";
    case BFLA_ERR_UNSUPPORTED: return "unsupported configuration";
    case BFLA_ERR_WORKSPACE: return "workspace too small";
    case BFLA_ERR_CAPACITY: return "list capacity too small";
    case BFLA_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

int bfla_list_capacity(const bfla_problem* prob, const bfla_params* params, size_t* n_rows,
                       size_t* max_cols, size_t* mask_bytes, size_t* score_elems) {
  int st = check_problem(prob, params);
  if (st) return st;
  Sizes s = sizes_of(prob, params);
  if (n_rows) *n_rows = (size_t)s.n_rows;
  if (max_cols) *max_cols = (size_t)s.max_cols;
  if (mask_bytes) *mask_bytes = (size_t)s.mask_bytes;
  if (score_elems) *score_elems = (size_t)s.score_elems;
  return ok();
}

int bfla_workspace_size(const bfla_problem* prob, const bfla_params* params, int which,
                        size_t* bytes) {
  int st = check_problem(prob, params);
  if (st) return st;
  if (!bytes) return fail(BFLA_ERR_INVALID_ARG, "bytes is NULL");
  Sizes s = sizes_of(prob, params);
  if (which == BFLA_WS_ESTIMATE) {
    if (!estimate_supported(prob->head_dim, params->block, params->group))
      return fail(BFLA_ERR_UNSUPPORTED, "block %d / group %d not built for head_dim %d",
                  params->block, params->group, prob->head_dim);
    *bytes = estimate_ws_scores_offset(stage1_layout(prob, params)) +
             (size_t)s.score_elems * sizeof(float);
  } else if (which == BFLA_WS_EXPAND) {
    *bytes = expand_workspace_bytes(s.n_rows, s.max_t_kv);
  } else {
    return fail(BFLA_ERR_INVALID_ARG, "unknown workspace kind %d", which);
  }
  return ok();
}

int bfla_estimate_mask(const bfla_problem* prob, const bfla_params* params, const bfla_view* q,
                       const bfla_kv* kv, uint8_t* block_mask, float* dbg_scores,
                       uint8_t* dbg_head_mask, void* workspace, size_t ws_bytes,
                       void* stream) {
  int st;
  if ((st = check_problem(prob, params))) return st;
  if ((st = check_view(prob, q, "q"))) return st;
  if ((st = check_kv(prob, kv, false))) return st;
  if (!block_mask) return fail(BFLA_ERR_INVALID_ARG, "block_mask is NULL");
  if (prob->h_q / prob->h_kv > 8)
    return fail(BFLA_ERR_UNSUPPORTED, "GQA group size %d not built (1 to 8)",
                prob->h_q / prob->h_kv);
  if (!estimate_supported(prob->head_dim, params->block, params->group))
    return fail(BFLA_ERR_UNSUPPORTED, "block %d / group %d not built for head_dim %d",
                params->block, params->group, prob->head_dim);
  if (!estimate_q_fits(params->group, prob->head_dim, q->stride_tok))
    return fail(BFLA_ERR_UNSUPPORTED, "q stride_tok %lld too large for group %d",
                (long long)q->stride_tok, params->group);
  if (kv->layout == BFLA_KV_PAGED && !estimate_pages_fit(params->group, kv->page_size))
    return fail(BFLA_ERR_UNSUPPORTED, "group %d spans too many pages of size %d",
                params->group, kv->page_size);
  for (int r = 0; r < prob->batch; ++r)
    if (cdiv(prob->n_kv[r], params->block) > kMaxBlocksPerRow)
      return fail(BFLA_ERR_UNSUPPORTED, "request %d: more than %d KV blocks", r,
                  (int)kMaxBlocksPerRow);
  Sizes s = sizes_of(prob, params);
  Stage1Layout plan = stage1_layout(prob, params);
  const size_t off = estimate_ws_scores_offset(plan);
  const size_t need = dbg_scores ? plan.partial_bytes : off + (size_t)s.score_elems * sizeof(float);
  if (need > 0 && (!workspace || ws_bytes < need))
    return fail(BFLA_ERR_WORKSPACE, "estimate workspace %zu < %zu bytes", ws_bytes, need);
  if (need > 0 && (reinterpret_cast<uintptr_t>(workspace) & 255))
    return fail(BFLA_ERR_INVALID_ARG, "estimate workspace not 256-byte aligned");
  float* scores = dbg_scores ? dbg_scores
                             : reinterpret_cast<float*>(static_cast<char*>(workspace) + off);
  EstimateLaunch L{};
  L.q = q->data;
  L.q_sh = q->stride_head;
  L.q_st = q->stride_tok;
  L.kv = kv_addr(kv);
  L.block_mask = block_mask;
  L.scores = scores;
  L.partials = plan.partial_bytes > 0 ? static_cast<float*>(workspace) : nullptr;
  L.splits = std::move(plan.splits);
  L.head_mask = dbg_head_mask;
  L.h_q = prob->h_q;
  L.h_kv = prob->h_kv;
  L.head_dim = prob->head_dim;
  L.block = params->block;
  L.group = params->group;
  L.gamma = params->gamma;
  L.alpha = scale_of(prob, params);
  L.reqs = make_batch(prob, params, q, nullptr, kv);
  return hip_status(launch_estimate(L, static_cast<hipStream_t>(stream)), "estimate_mask");
}

int bfla_expand_rescue(const bfla_problem* prob, const bfla_params* params,
                       const uint8_t* block_mask, int32_t* row_ptr, int32_t* cols,
                       size_t cols_capacity, void* workspace, size_t ws_bytes, void* stream) {
  return expand_common(prob, params, block_mask, row_ptr, cols, cols_capacity, workspace,
                       ws_bytes, false, stream);
}

int bfla_expand_rescue_noalloc(const bfla_problem* prob, const bfla_params* params,
                               const uint8_t* block_mask, int32_t* row_ptr, int32_t* cols,
                               size_t cols_capacity, void* stream) {
  return expand_common(prob, params, block_mask, row_ptr, cols, cols_capacity, nullptr, 0,
                       true, stream);
}

int bfla_sparse_prefill(const bfla_problem* prob, const bfla_params* params, const bfla_view* q,
                        const bfla_kv* kv, const int32_t* row_ptr, const int32_t* cols,
                        const bfla_view* o, float* lse, void* stream) {
  PrefillLaunch L{};
  int st = prefill_common(prob, params, q, kv, o, &L);
  if (st) return st;
  if (!row_ptr || !cols) return fail(BFLA_ERR_INVALID_ARG, "row_ptr / cols is NULL");
  L.row_ptr = row_ptr;
  L.cols = cols;
  L.lse = lse;
  return hip_status(launch_prefill(L, static_cast<hipStream_t>(stream)), "sparse_prefill");
}

int bfla_dense_prefill(const bfla_problem* prob, const bfla_params* params, const bfla_view* q,
                       const bfla_kv* kv, const bfla_view* o, float* lse, void* stream) {
  PrefillLaunch L{};
  int st = prefill_common(prob, params, q, kv, o, &L);
  if (st) return st;
  L.row_ptr = nullptr;
  L.cols = nullptr;
  L.lse = lse;
  return hip_status(launch_prefill(L, static_cast<hipStream_t>(stream)), "dense_prefill");
}

}  // extern "C"
