// Stage 2 tile mask and list compaction (eq19-eq26), integer only.
//
// One wave per list row (request, KV head, q-tile).  Lanes walk the causal
// KV tiles of the row 64 at a time; each decides keep / drop for its tile:
//   kept    = block mask of (qt / rb, kt / rb)          (eq20)
//           | local band kt in [kt_diag - n_local, kt_diag]   (eq21)
//           | sink kt < n_sink                            (eq22)
//   rescued = !kept & (chi(qt, kt; s) mod eta == 0        (eq24)
//                      | psi(h, qt, kt; s) < rho)         (eq25)
// Pass 1 stores the wave ballots (one 64-bit word per 64 tiles of a row) and
// the row counts; pass 2 is an exclusive scan of the counts in one
// workgroup; pass 3 reads the ballots back and writes each kept tile at its
// list position, so every keep / drop decision is taken once.
#include <algorithm>
#include <atomic>

#include "bfla_device.h"
#include "bfla_internal.h"

// Workspace of bfla_expand_rescue_noalloc: one copy per device, for the life
// of the process.  Host code never passes `scratch` itself to a kernel (on
// the host it names a stand-in, not device memory): expand_scratch() looks up
// each device's address once and every launch uses that.
static __device__ __align__(256) uint8_t scratch[BFLA_EXPAND_SCRATCH_BYTES];

namespace bfla {
namespace {

constexpr int TILE = 64;
constexpr int ROWS_PER_WG = 4;
constexpr int SCAN_THREADS = 1024;

struct ExpandArgs {
  const uint8_t* block_mask;
  int32_t* row_ptr;
  int32_t* cols;
  int32_t* counts;
  uint64_t* bits;
  int32_t words_per_row;
  int32_t n_rows;
  int32_t h_kv, rb;
  int32_t n_local, n_sink, eta;
  uint32_t eta_mask;  // eta - 1 when eta is a power of two, else 0
  uint32_t rho24;
  uint64_t chi_key;  // mix64(s)
  uint64_t psi_key;  // mix64(s + 1)
  int32_t row_lo, row_hi;  // list rows of this launch's requests
  Batch batch;
};

// SplitMix64 output mix (Steele, Lea and Flood, OOPSLA 2014).
__host__ __device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

struct RowCtx {
  const uint8_t* blk_row;  // block mask row of this q-tile's query block
  int h, qt, kt_diag, n_tiles;
};

__device__ __forceinline__ bool row_ctx(const ExpandArgs& a, int row, RowCtx* c) {
  if (row >= a.row_hi) return false;
  // the request owning the row: row_base ascends over the launch's requests
  int ri = 0;
#pragma unroll
  for (int step = kLaunchRequests / 2; step >= 1; step >>= 1)
    if (ri + step < a.batch.n_req && row >= a.batch.r[ri + step].row_base) ri += step;
  const ReqDesc& R = a.batch.r[ri];
  int local = row - R.row_base;
  c->h = local / R.t_q;
  c->qt = local % R.t_q;
  int n_c = R.n_kv - R.n_q;
  int last = min(n_c + (c->qt + 1) * TILE - 1, R.n_kv - 1);
  c->kt_diag = last / TILE;
  c->n_tiles = c->kt_diag + 1;
  c->blk_row = a.block_mask + R.mask_off +
               ((int64_t)c->h * R.l_q + c->qt / a.rb) * R.l_kv;
  return true;
}

__device__ __forceinline__ bool keep_tile(const ExpandArgs& a, const RowCtx& c, int kt) {
  if (kt > c.kt_diag) return false;
  bool kept = c.blk_row[kt / a.rb] != 0;
  kept |= (a.n_local >= 0) && (kt >= c.kt_diag - a.n_local);
  kept |= kt < a.n_sink;
  if (kept) return true;
  const uint64_t key = ((uint64_t)c.qt << 21) | (uint64_t)kt;
  if (a.eta > 0) {
    // chi mod eta == 0; for a power-of-two eta the low bits decide it (the
    // same test without a 64-bit division)
    const uint64_t chi = mix64(a.chi_key ^ key);
    if (a.eta_mask != 0 ? (chi & a.eta_mask) == 0 : chi % (uint64_t)a.eta == 0) return true;
  }
  if (a.rho24 > 0) {
    uint64_t hk = key | ((uint64_t)(c.h + 1) << 42);
    if ((uint32_t)(mix64(a.psi_key ^ hk) >> 40) < a.rho24) return true;
  }
  return false;
}

__global__ void __launch_bounds__(64 * ROWS_PER_WG) count_kernel(ExpandArgs a) {
  const int lane = threadIdx.x & 63;
  const int row = a.row_lo + blockIdx.x * ROWS_PER_WG + (threadIdx.x >> 6);
  RowCtx c;
  if (!row_ctx(a, row, &c)) return;
  uint64_t* bits = a.bits + (int64_t)row * a.words_per_row;
  int total = 0;
  for (int k0 = 0; k0 < c.n_tiles; k0 += 64) {
    const uint64_t b = __ballot(keep_tile(a, c, k0 + lane));
    if (lane == 0) bits[k0 >> 6] = b;
    total += __popcll(b);
  }
  if (lane == 0) a.counts[row] = total;
}

__global__ void __launch_bounds__(SCAN_THREADS) scan_kernel(const int32_t* counts,
                                                            int32_t* row_ptr, int n) {
  __shared__ int32_t wsum[SCAN_THREADS / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int per = (n + SCAN_THREADS - 1) / SCAN_THREADS;
  const int beg = min(n, tid * per), end = min(n, beg + per);
  int s = 0;
  for (int i = beg; i < end; ++i) s += counts[i];
  // inclusive scan of s across the workgroup
  int x = s;
  for (int d = 1; d < 64; d <<= 1) {
    int y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  if (wave == 0) {
    int v = lane < SCAN_THREADS / 64 ? wsum[lane] : 0;
    for (int d = 1; d < 64; d <<= 1) {
      int y = __shfl_up(v, d);
      if (lane >= d) v += y;
    }
    if (lane < SCAN_THREADS / 64) wsum[lane] = v;
  }
  __syncthreads();
  int excl = x - s + (wave > 0 ? wsum[wave - 1] : 0);
  for (int i = beg; i < end; ++i) {
    row_ptr[i] = excl;
    excl += counts[i];
  }
  if (tid == SCAN_THREADS - 1) row_ptr[n] = wsum[SCAN_THREADS / 64 - 1];
}

__global__ void __launch_bounds__(64 * ROWS_PER_WG) scatter_kernel(ExpandArgs a) {
  const int lane = threadIdx.x & 63;
  const int row = a.row_lo + blockIdx.x * ROWS_PER_WG + (threadIdx.x >> 6);
  RowCtx c;
  if (!row_ctx(a, row, &c)) return;
  const uint64_t* bits = a.bits + (int64_t)row * a.words_per_row;
  int pos = a.row_ptr[row];
  for (int k0 = 0; k0 < c.n_tiles; k0 += 64) {
    const int kt = k0 + lane;
    const uint64_t b = bits[k0 >> 6];   // pass 1's ballot of these 64 tiles
    const bool keep = (b >> lane) & 1;
    int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32),
                                           __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0));
    if (keep) a.cols[pos + before] = kt;
    pos += __popcll(b);
  }
}

}  // namespace

namespace {
constexpr int kMaxDevices = 256;
std::atomic<uintptr_t> g_scratch[kMaxDevices];  // device address, 0 = not looked up yet
}  // namespace

hipError_t expand_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  uintptr_t p = g_scratch[dev].load(std::memory_order_acquire);
  if (p == 0) {
    // with this device current: its own copy of the array
    void* addr = nullptr;
    e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (addr == nullptr) return hipErrorInvalidSymbol;
    p = reinterpret_cast<uintptr_t>(addr);
    g_scratch[dev].store(p, std::memory_order_release);
  }
  *ptr = reinterpret_cast<void*>(p);
  return hipSuccess;
}

hipError_t launch_expand(const ExpandLaunch& L, hipStream_t stream) {
  if (L.n_rows == 0) return hipSuccess;
  ExpandArgs a;
  a.block_mask = L.block_mask;
  a.row_ptr = L.row_ptr;
  a.cols = L.cols;
  a.counts = L.counts;
  a.bits = L.bits;
  a.words_per_row = L.words_per_row;
  a.n_rows = L.n_rows;
  a.h_kv = L.h_kv;
  a.rb = L.rb;
  a.n_local = L.n_local;
  a.n_sink = L.n_sink;
  a.eta = L.eta;
  a.eta_mask = (L.eta > 1 && (L.eta & (L.eta - 1)) == 0) ? (uint32_t)(L.eta - 1) : 0u;
  a.rho24 = L.rho24;
  a.chi_key = mix64(L.seed);
  a.psi_key = mix64(L.seed + 1);
  // count and scatter once per group of kLaunchRequests requests (each over
  // its own rows), one scan over every row in between
  auto for_each_group = [&](auto&& launch) -> hipError_t {
    for (size_t g0 = 0; g0 < L.reqs.size(); g0 += kLaunchRequests) {
      const int n = (int)std::min<size_t>(kLaunchRequests, L.reqs.size() - g0);
      a.batch.n_req = n;
      for (int i = 0; i < n; ++i) a.batch.r[i] = L.reqs[g0 + i];
      const ReqDesc& last = a.batch.r[n - 1];
      a.row_lo = a.batch.r[0].row_base;
      a.row_hi = last.row_base + L.h_kv * last.t_q;
      if (a.row_hi == a.row_lo) continue;
      const int grid = (a.row_hi - a.row_lo + ROWS_PER_WG - 1) / ROWS_PER_WG;
      launch(grid);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  };
  hipError_t e = for_each_group([&](int grid) {
    hipLaunchKernelGGL(count_kernel, dim3(grid), dim3(64 * ROWS_PER_WG), 0, stream, a);
  });
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(SCAN_THREADS), 0, stream, a.counts, a.row_ptr,
                     a.n_rows);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return for_each_group([&](int grid) {
    hipLaunchKernelGGL(scatter_kernel, dim3(grid), dim3(64 * ROWS_PER_WG), 0, stream, a);
  });
}

}  // namespace bfla
