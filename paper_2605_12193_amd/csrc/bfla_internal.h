// Host-side launcher interface between the C ABI (api.cpp) and the kernels.
// The shape predicates and workspace sizes are host code (shapes.cpp); the
// launch_* functions live beside their kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <vector>

#include "bfla_device.h"

namespace bfla {

// Stage-1 score tiles: kScoreTileM query groups x kScoreTileN key groups,
// kScoreChunk inner elements per LDS stage; the page numbers one tile of a
// paged cache spans are resolved into LDS, at most kScorePagesMax of them.
constexpr int kScoreTileM = 256;
constexpr int kScoreTileN = 128;
constexpr int kScoreChunk = 64;
constexpr int kScorePagesMax = 2056;
// stages per inner accumulation chain of the score GEMM (summed into a
// second accumulator; a split of the inner dimension cuts between chains)
constexpr int kScoreChain = 8;

// How Stage 1 runs a problem: score tiles in the launch (all, and those
// holding a causal block pair), the split of the inner dimension (1: none;
// S > 1: S workgroups per tile, each a run of whole chains, whose raw group
// sums a second kernel adds in a fixed order before the max pool), and the
// workspace bytes those partial sums take.  A function of the problem only,
// so results do not depend on the device.
struct EstimatePlan {
  int32_t split;
  int64_t total_tiles;
  int64_t causal_tiles;
  size_t partial_bytes;
};
EstimatePlan estimate_plan(const int32_t* n_q, const int32_t* n_kv, int batch, int h_q,
                           int head_dim, int block, int group);

struct PrefillLaunch {
  const void* q;
  void* o;
  float* lse;
  const int32_t* row_ptr;  // null -> dense (every causal tile)
  const int32_t* cols;
  int64_t q_sh, q_st, o_sh, o_st;
  KvAddr kv;
  int32_t h_q, h_kv, head_dim;
  float scale;
  std::vector<ReqDesc> reqs;  // every request, in launch order (longest first)
};

bool prefill_supported(int head_dim, int m);
hipError_t launch_prefill(const PrefillLaunch& L, hipStream_t stream);

struct ExpandLaunch {
  const uint8_t* block_mask;
  int32_t* row_ptr;
  int32_t* cols;
  int32_t* counts;   // workspace [n_rows]
  int32_t* partial;  // workspace [scan blocks]
  uint64_t* bits;    // workspace [n_rows][words_per_row]: keep ballots of 64 tiles
  int32_t words_per_row;
  int32_t n_rows;
  int32_t h_kv;
  int32_t rb;        // b / T
  int32_t n_local, n_sink, eta;
  uint32_t rho24;    // floor(rho * 2^24); 1<<24 means every dropped tile
  uint64_t seed;
  std::vector<ReqDesc> reqs;  // every request, in request order
};

hipError_t launch_expand(const ExpandLaunch& L, hipStream_t stream);
// The current device's fixed tile-stage scratch (BFLA_EXPAND_SCRATCH_BYTES),
// looked up once per device.
hipError_t expand_scratch(void** ptr);
size_t expand_workspace_bytes(int64_t n_rows, int64_t max_t_kv);

struct EstimateLaunch {
  const void* q;
  int64_t q_sh, q_st;
  KvAddr kv;
  uint8_t* block_mask;
  float* scores;      // [per request H_q x L_q x L_kv], workspace or dbg output
  float* partials;    // split > 1: [split][tiles][kScoreTileM][kScoreTileN] raw group sums
  uint8_t* head_mask; // [per request H_q x L_q x L_kv] per-head keep sets, or null
  int32_t h_q, h_kv, head_dim;
  int32_t block, group;
  float gamma;
  float alpha;
  std::vector<ReqDesc> reqs;    // every request, in request order
  std::vector<int32_t> splits;  // split of each group of kLaunchRequests requests
};

bool estimate_supported(int head_dim, int block, int group);
// Stage-1 address limits: the query rows of one score tile must span < 2 GiB,
// and one tile's keys of a paged cache at most kScorePagesMax pages.
bool estimate_q_fits(int group, int head_dim, int64_t q_stride_tok);
bool estimate_pages_fit(int group, int page_size);
hipError_t launch_estimate(const EstimateLaunch& L, hipStream_t stream);

}  // namespace bfla
