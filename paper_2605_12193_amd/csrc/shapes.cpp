// Host-side shape predicates and workspace sizes of the kernels: which
// (head dim, block, group, GQA group) combinations are built, the address
// limits of the Stage-1 score tiles, and the tile-stage workspace layout.
// Kept apart from the kernel sources so the C ABI layer builds and runs
// without device code (the sanitizer build of the ABI links this file).
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
