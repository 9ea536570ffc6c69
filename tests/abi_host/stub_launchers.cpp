// Host-only stand-ins for the kernel launchers of the BFLA library.  Linked
// with the real C ABI layer (api.cpp, shapes.cpp) into a sanitizer build that
// needs no GPU: each launcher counts its call, checks on the host that the
// launch descriptor the ABI layer built is consistent with the problem, and
// returns success without reading or writing any device pointer.
#include <stdint.h>

#include <vector>

#include "bfla_internal.h"

namespace {

int g_launches[3];  // prefill, expand, estimate
int g_bad;          // descriptors that failed a consistency check

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

void check_batch(const std::vector<bfla::ReqDesc>& b, int block) {
  if (b.empty() || b.size() > BFLA_MAX_BATCH) {
    ++g_bad;
    return;
  }
  std::vector<bool> seen(b.size(), false);
  for (size_t r = 0; r < b.size(); ++r) {
    const bfla::ReqDesc& d = b[r];
    if (d.n_q < 1 || d.n_kv < d.n_q) ++g_bad;
    if (d.t_q != cdiv(d.n_q, 64) || d.t_kv != cdiv(d.n_kv, 64)) ++g_bad;
    if (block > 0 && (d.l_q != cdiv(d.n_q, block) || d.l_kv != cdiv(d.n_kv, block))) ++g_bad;
    if (d.q_off < 0 || d.o_off < 0 || d.kv_off < 0 || d.lse_off < 0 || d.mask_off < 0 ||
        d.score_off < 0 || d.row_base < 0)
      ++g_bad;
    if (d.bt_row < 0 || d.bt_row >= (int)b.size() || seen[d.bt_row]) {
      ++g_bad;
      continue;
    }
    seen[d.bt_row] = true;
  }
}

}  // namespace

extern "C" int stub_launches(int which) { return which >= 0 && which < 3 ? g_launches[which] : -1; }
extern "C" int stub_bad_descriptors(void) { return g_bad; }

namespace bfla {

hipError_t launch_prefill(const PrefillLaunch& L, hipStream_t) {
  ++g_launches[0];
  check_batch(L.reqs, 0);
  if (!L.q || !L.o || !L.kv.k || !L.kv.v || L.h_q % L.h_kv || !prefill_supported(L.head_dim, L.h_q / L.h_kv))
    ++g_bad;
  if ((L.row_ptr == nullptr) != (L.cols == nullptr)) ++g_bad;
  // longest requests first
  for (size_t r = 1; r < L.reqs.size(); ++r)
    if (L.reqs[r].n_kv > L.reqs[r - 1].n_kv) ++g_bad;
  return hipSuccess;
}

hipError_t launch_expand(const ExpandLaunch& L, hipStream_t) {
  ++g_launches[1];
  check_batch(L.reqs, L.rb * 64);
  if (L.partial != L.counts + ((int64_t)L.n_rows + 63) / 64 * 64) ++g_bad;
  if (reinterpret_cast<const int32_t*>(L.bits) != L.partial + 64) ++g_bad;
  if (reinterpret_cast<uintptr_t>(L.bits) & 7) ++g_bad;
  int64_t rows = 0;
  for (const ReqDesc& d : L.reqs) {
    if (d.row_base != rows) ++g_bad;
    rows += (int64_t)L.h_kv * d.t_q;
    if (cdiv(d.t_kv, 64) > L.words_per_row) ++g_bad;
  }
  if (rows != L.n_rows) ++g_bad;
  return hipSuccess;
}

hipError_t expand_scratch(void** ptr) {
  // a fake, aligned device address: the stub launchers never dereference it
  *ptr = reinterpret_cast<void*>(uintptr_t(1) << 32);
  return hipSuccess;
}

hipError_t launch_estimate(const EstimateLaunch& L, hipStream_t) {
  ++g_launches[2];
  check_batch(L.reqs, L.block);
  if (!L.block_mask || !L.scores || !L.q || !L.kv.k) ++g_bad;
  if (L.splits.size() != (L.reqs.size() + kLaunchRequests - 1) / kLaunchRequests) ++g_bad;
  for (int32_t sp : L.splits)
    if (sp < 1 || (sp > 1 && !L.partials)) ++g_bad;
  if (!estimate_supported(L.head_dim, L.block, L.group) || L.h_q / L.h_kv > 8) ++g_bad;
  int64_t mask = 0, score = 0;
  for (const ReqDesc& d : L.reqs) {
    if (d.mask_off != mask || d.score_off != score) ++g_bad;
    mask += (int64_t)L.h_kv * d.l_q * d.l_kv;
    score += (int64_t)L.h_q * d.l_q * d.l_kv;
  }
  return hipSuccess;
}

}  // namespace bfla
