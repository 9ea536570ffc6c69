// Host-side shape predicates and workspace sizes of the kernels: which
// (head dim, block, group, GQA group) combinations are built, the address
// limits of the Stage-1 score tiles, and the tile-stage workspace layout.
// Kept apart from the kernel sources so the C ABI layer builds and runs
// without device code (the sanitizer build of the ABI links this file).
#include <algorithm>

#include "bfla_internal.h"

namespace bfla {

bool estimate_supported(int head_dim, int block, int group) {
  if (head_dim != 64 && head_dim != 128 && head_dim != 256) return false;
  if (group < 1 || block % group) return false;
  const int G = block / group;
  if (G != 1 && G != 2 && G != 4 && G != 8 && G != 16) return false;
  return ((int64_t)group * head_dim) % kScoreChunk == 0;
}

bool estimate_q_fits(int group, int head_dim, int64_t q_stride_tok) {
  // one score tile reads kScoreTileM query groups of g tokens through one
  // buffer descriptor with a signed 32-bit byte range
  return ((int64_t)kScoreTileM * group - 1) * q_stride_tok + head_dim < (int64_t(1) << 30);
}

bool estimate_pages_fit(int group, int page_size) {
  // a tile of kScoreTileN key groups covers kScoreTileN * g tokens: at most
  // kScoreTileN * g / page_size + 1 pages
  return ((int64_t)kScoreTileN * group + page_size - 1) / page_size + 1 <= kScorePagesMax;
}

EstimatePlan estimate_plan(const int32_t* n_q, const int32_t* n_kv, int batch, int h_q,
                           int head_dim, int block, int group) {
  EstimatePlan p{};
  const int G = block / group;
  for (int r = 0; r < batch; ++r) {
    const int64_t nqg = (n_q[r] + group - 1) / group, nkg = (n_kv[r] + group - 1) / group;
    const int64_t rt = (nqg + kScoreTileM - 1) / kScoreTileM;
    const int64_t ct = (nkg + kScoreTileN - 1) / kScoreTileN;
    p.total_tiles += (int64_t)h_q * rt * ct;
    // tile (ti, tj) holds a causal block pair iff its first KV block starts
    // at or before the end of its last query block: tj * kScoreTileN / G <= E
    // with E = e_i / b, i.e. tj <= E * G / kScoreTileN
    const int64_t n_c = n_kv[r] - n_q[r];
    for (int64_t ti = 0; ti < rt; ++ti) {
      const int64_t i_max = (std::min(nqg, (ti + 1) * kScoreTileM) - 1) / G;
      const int64_t e_i = std::min(n_c + (i_max + 1) * block - 1, (int64_t)n_kv[r] - 1);
      p.causal_tiles += (int64_t)h_q * std::min(ct, (e_i / block) * G / kScoreTileN + 1);
    }
  }
  // Estimated time of split S (whole chains per part only): a launch of T
  // causal tiles runs ceil(S T / 256) rounds of workgroups (one per compute
  // unit of an MI355X) of n_stage / S stages each, a stage of a 256 x 128
  // tile taking about 1.3 us (its 48 KiB of loads are bound by misses in
  // flight); a split also writes and re-reads 128 KiB of partial sums per
  // tile and part, at about 5 TB/s.
  constexpr int kCUs = 256;
  constexpr double kStageUs = 1.3, kPartialUs = 2.0 * 128 * 1024 / 5e6;
  const int n_stage = group * head_dim / kScoreChunk;
  auto cost = [&](int s) {
    const double rounds = (double)((p.causal_tiles * s + kCUs - 1) / kCUs);
    return rounds * (n_stage / s) * kStageUs +
           (s > 1 ? (double)s * (double)p.causal_tiles * kPartialUs : 0.0);
  };
  // a split must save at least 10 % of the estimate to be taken
  double best = 0.9 * cost(1);
  p.split = 1;
  for (int s = 2; s <= 8; s *= 2) {
    if (n_stage % (s * kScoreChain) != 0) break;
    const double c = cost(s);
    if (c < best) {
      best = c;
      p.split = s;
    }
  }
  p.partial_bytes = p.split > 1 ? (size_t)p.split * (size_t)p.total_tiles * kScoreTileM *
                                      kScoreTileN * sizeof(float)
                                : 0;
  return p;
}

// counts [n_rows rounded up to 64] + scan partials [64] (int32), then the
// keep ballots [n_rows][ceil(max_t_kv / 64)] (uint64, at a 256-byte offset)
size_t expand_workspace_bytes(int64_t n_rows, int64_t max_t_kv) {
  return (size_t)(((n_rows + 63) / 64) * 64 + 64) * sizeof(int32_t) +
         (size_t)n_rows * (size_t)((max_t_kv + 63) / 64) * sizeof(uint64_t);
}

bool prefill_supported(int head_dim, int m) {
  bool c_ok = head_dim == 64 || head_dim == 128 || head_dim == 256;
  bool m_ok = m >= 1 && m <= 8;
  return c_ok && m_ok;
}

}  // namespace bfla
