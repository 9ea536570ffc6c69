// Stage 1: block-level importance estimation (Sec. 3.2, eq4-eq18) + GQA
// union.  gfx950 / CDNA4, wave64.
//
// Kernel 1 (scores): for every query head p the group-score matrix
//   S_groups[gi][gj] = PhiQ_p[gi] . PhiK_h[gj]       (eq9)
// is a GEMM whose rows are flattened g-token query groups and whose columns
// are flattened key groups (inner dimension g*C; a flattened group of a
// row-major [N][C] head is g consecutive token rows, so no copy is made,
// eq6-eq7).  128 x 128 output tiles, 4 waves of 64 x 64, bf16 MFMA
// 32x32x16, K/Q chunks staged through LDS with register double buffering;
// only tiles holding a causal block pair are computed (eq11-eq14).  The
// epilogue max-pools each G x G group block into the block score (eq10)
// and stores it as float.  Accumulation is two-level: chains of 32 MFMA
// steps (512 products) are summed into a second float accumulator, which
// keeps the score error well inside the near-tie band of the selection.
//
// Kernel 2 (select): one workgroup per (request, KV head, query block),
// one wave per query head of the group: block softmax over the causal KV
// blocks (eq15), keep-mass selection by repeated arg-max in the order
// (score descending, block index ascending) with a sequential float
// running mass (eq16-eq18), then OR of the m heads into the u8 mask row.
#include "bfla_device.h"
#include "bfla_internal.h"

namespace bfla {
namespace {

constexpr int BM = 128;     // query groups per tile
constexpr int BN = 128;     // key groups per tile
constexpr int BK = 64;      // inner elements per stage
constexpr int PITCH = BK + 8;
constexpr int NT = 256;
constexpr int CHAIN = 8;    // stages per inner accumulation chain (32 MFMA k-steps)
constexpr int MAX_LKV = 65536;

struct ScoreArgs {
  const bf16_t* q;
  int64_t q_sh, q_st;
  KvAddr kv;
  float* scores;
  int32_t h_q, h_kv, m;
  int32_t C, g, b, G;
  int32_t gc;        // g * C
  Batch batch;       // work_begin = first tile of request r
};

struct SelectArgs {
  const float* scores;
  float* dbg;        // non-null: also fill non-causal entries with -inf
  uint8_t* block_mask;
  int32_t h_q, h_kv, m, b;
  float gamma, alpha;
  Batch batch;       // work_begin = first (h, i) row of request r
};

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint4 ld16(const bf16_t* p) {
  return *reinterpret_cast<const uint4*>(p);
}

__host__ __device__ __forceinline__ int tiles_of(int groups) { return (groups + BM - 1) / BM; }

template <int G>
__global__ void __launch_bounds__(NT, 2) scores_kernel(ScoreArgs a) {
  __shared__ __align__(16) bf16_t sa[2][BM * PITCH];
  __shared__ __align__(16) bf16_t sb[2][BN * PITCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hi = lane >> 5;
  const int wi = wave >> 1, wj = wave & 1;

  // ---- tile decode: (request, tile rank, head) with the KV head fastest ----
  const int ri = find_req(a.batch, blockIdx.x);
  const ReqDesc& R = a.batch.r[ri];
  const int local = blockIdx.x - R.work_begin;
  const int nqg = (R.n_q + a.g - 1) / a.g;    // query groups
  const int nkg = (R.n_kv + a.g - 1) / a.g;   // key groups
  const int ntj = tiles_of(nkg);
  const int h = local % a.h_kv;
  const int pm = (local / a.h_kv) % a.m;
  const int rank = local / a.h_q;
  const int ti = rank / ntj, tj = rank % ntj;
  const int p = h * a.m + pm;
  const int n_c = R.n_kv - R.n_q;

  // skip tiles without any causal block pair
  {
    int gi_last = min(nqg, (ti + 1) * BM) - 1;
    int i_max = gi_last / G;
    int e_i = min(n_c + (i_max + 1) * a.b - 1, R.n_kv - 1);
    int j_min = (tj * BN) / G;
    if (j_min * a.b > e_i) return;
  }

  const bf16_t* qbase = a.q + R.q_off + (int64_t)p * a.q_sh;
  const int n_stage = a.gc / BK;

  // loader mapping: 1024 16-byte chunks per operand tile, 4 per thread
  uint4 ra[4], rbv[4];
  auto load = [&](int st) {
    const int k0 = st * BK;
    const int tok_in = k0 / a.C, ch = k0 % a.C;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + i * NT;
      const int row = e >> 3, ce = e & 7;
      const int gi = ti * BM + row;
      const int tq = gi * a.g + tok_in;
      ra[i] = (gi < nqg && tq < R.n_q)
                  ? ld16(qbase + (int64_t)tq * a.q_st + ch + 8 * ce)
                  : make_uint4(0, 0, 0, 0);
      const int gj = tj * BN + row;
      const int tk = gj * a.g + tok_in;
      rbv[i] = (gj < nkg && tk < R.n_kv)
                   ? ld16(a.kv.k + kv_elem(a.kv, R, h, tk) + ch + 8 * ce)
                   : make_uint4(0, 0, 0, 0);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + i * NT;
      const int row = e >> 3, ce = e & 7;
      *reinterpret_cast<uint4*>(&sa[buf][row * PITCH + 8 * ce]) = ra[i];
      *reinterpret_cast<uint4*>(&sb[buf][row * PITCH + 8 * ce]) = rbv[i];
    }
  };

  f32x16 acc[2][2], tot[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int r = 0; r < 16; ++r) { acc[x][y][r] = 0.f; tot[x][y][r] = 0.f; }

  load(0);
  store(0);
  __syncthreads();
  for (int st = 0; st < n_stage; ++st) {
    const bool more = st + 1 < n_stage;
    if (more) load(st + 1);
    const bf16_t* A = sa[st & 1];
    const bf16_t* B = sb[st & 1];
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 af[2], bf[2];
#pragma unroll
      for (int x = 0; x < 2; ++x)
        af[x] = __builtin_bit_cast(bf16x8, ld16(A + (64 * wi + 32 * x + l32) * PITCH + 16 * ks + 8 * hi));
#pragma unroll
      for (int y = 0; y < 2; ++y)
        bf[y] = __builtin_bit_cast(bf16x8, ld16(B + (64 * wj + 32 * y + l32) * PITCH + 16 * ks + 8 * hi));
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = mfma32(af[x], bf[y], acc[x][y]);
    }
    if ((st + 1) % CHAIN == 0 || !more) {
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
          for (int r = 0; r < 16; ++r) { tot[x][y][r] += acc[x][y][r]; acc[x][y][r] = 0.f; }
    }
    if (more) store((st + 1) & 1);
    __syncthreads();
  }

  // ---- epilogue: drop padded groups, G x G max pool, causal store ----
  // D[row = query group][col = key group]; lane: col l32, rows 8(r/4)+4hi+r%4
  float* srow_base = a.scores + R.score_off + (int64_t)p * R.l_q * R.l_kv;
#pragma unroll
  for (int x = 0; x < 2; ++x) {
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      const int gj = tj * BN + 64 * wj + 32 * y + l32;
      f32x16 v = tot[x][y];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int gi = ti * BM + 64 * wi + 32 * x + 8 * (r >> 2) + 4 * hi + (r & 3);
        if (gi >= nqg || gj >= nkg) v[r] = -INFINITY;
      }
      // pool over G consecutive query-group rows
      float pr[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) pr[r] = v[r];
      if (G >= 2) {
#pragma unroll
        for (int r = 0; r < 16; r += 2) pr[r] = fmaxf(pr[r], pr[r + 1]);
      }
      if (G >= 4) {
#pragma unroll
        for (int r = 0; r < 16; r += 4) pr[r] = fmaxf(pr[r], pr[r + 2]);
      }
      if (G >= 8) {
#pragma unroll
        for (int r = 0; r < 16; r += 4) pr[r] = fmaxf(pr[r], __shfl_xor(pr[r], 32));
      }
      // pool over G consecutive key-group columns (lanes)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (G >= 2) pr[r] = fmaxf(pr[r], __shfl_xor(pr[r], 1));
        if (G >= 4) pr[r] = fmaxf(pr[r], __shfl_xor(pr[r], 2));
        if (G >= 8) pr[r] = fmaxf(pr[r], __shfl_xor(pr[r], 4));
      }
      if ((l32 % G) != 0 || (G >= 8 && hi != 0)) continue;
      const int j = gj / G;
      if (j >= R.l_kv) continue;
#pragma unroll
      for (int r = 0; r < 16; r += (G >= 4 ? 4 : G)) {
        const int gi = ti * BM + 64 * wi + 32 * x + 8 * (r >> 2) + 4 * hi + (r & 3);
        const int i = gi / G;
        if (i >= R.l_q) continue;
        const int e_i = min(n_c + (i + 1) * a.b - 1, R.n_kv - 1);
        if (j * a.b <= e_i) srow_base[(int64_t)i * R.l_kv + j] = pr[r];
      }
    }
  }
}

// Total order of the keep ranking: score descending, then index ascending.
__device__ __forceinline__ bool better(float s1, int j1, float s2, int j2) {
  return s1 > s2 || (s1 == s2 && j1 < j2);
}

__global__ void __launch_bounds__(512) select_kernel(SelectArgs a) {
  __shared__ uint32_t keep_bits[MAX_LKV / 32];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ri = find_req(a.batch, blockIdx.x);
  const ReqDesc& R = a.batch.r[ri];
  const int local = blockIdx.x - R.work_begin;
  const int h = local / R.l_q, i = local % R.l_q;
  const int p = h * a.m + wave;
  const int n_c = R.n_kv - R.n_q;
  const int e_i = min(n_c + (i + 1) * a.b - 1, R.n_kv - 1);
  const int n_causal = e_i / a.b + 1;
  const int words = (R.l_kv + 31) / 32;

  for (int w = tid; w < words; w += blockDim.x) keep_bits[w] = 0u;
  __syncthreads();

  const float* row = a.scores + R.score_off + ((int64_t)p * R.l_q + i) * R.l_kv;

  if (a.gamma >= 1.0f) {
    for (int j = tid; j < n_causal; j += blockDim.x) atomicOr(&keep_bits[j >> 5], 1u << (j & 31));
  } else {
    // softmax statistics (eq15)
    float mx = -INFINITY;
    for (int j = lane; j < n_causal; j += 64) mx = fmaxf(mx, row[j]);
    for (int d = 32; d >= 1; d >>= 1) mx = fmaxf(mx, __shfl_xor(mx, d));
    float z = 0.f;
    for (int j = lane; j < n_causal; j += 64) z += expf(a.alpha * (row[j] - mx));
    for (int d = 32; d >= 1; d >>= 1) z += __shfl_xor(z, d);

    // keep-mass selection (eq16-eq18): repeated arg-max below the last pick
    float mass = 0.f;
    float s_prev = INFINITY;
    int j_prev = -1;
    for (int taken = 0; taken < n_causal; ++taken) {
      float bs = -INFINITY;
      int bj = INT_MAX;
      for (int j = lane; j < n_causal; j += 64) {
        const float s = row[j];
        if (better(s_prev, j_prev, s, j) && better(s, j, bs, bj)) { bs = s; bj = j; }
      }
      for (int d = 32; d >= 1; d >>= 1) {
        const float os = __shfl_xor(bs, d);
        const int oj = __shfl_xor(bj, d);
        if (better(os, oj, bs, bj)) { bs = os; bj = oj; }
      }
      if (bj >= n_causal) break;  // only with non-finite scores: nothing left to rank
      if (lane == 0) atomicOr(&keep_bits[bj >> 5], 1u << (bj & 31));
      mass += expf(a.alpha * (bs - mx)) / z;
      if (mass >= a.gamma) break;
      s_prev = bs;
      j_prev = bj;
    }
  }
  __syncthreads();

  uint8_t* mrow = a.block_mask + R.mask_off + ((int64_t)h * R.l_q + i) * R.l_kv;
  for (int j = tid; j < R.l_kv; j += blockDim.x) mrow[j] = (keep_bits[j >> 5] >> (j & 31)) & 1u;
  if (a.dbg) {
    float* drow = a.dbg + R.score_off + ((int64_t)p * R.l_q + i) * R.l_kv;
    for (int j = n_causal + lane; j < R.l_kv; j += 64) drow[j] = -INFINITY;
  }
}

template <int G>
hipError_t launch_scores(const ScoreArgs& a, int n_tiles, hipStream_t s) {
  hipLaunchKernelGGL(scores_kernel<G>, dim3(n_tiles), dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace

bool estimate_supported(int head_dim, int block, int group) {
  if (head_dim != 64 && head_dim != 128 && head_dim != 256) return false;
  if (group < 1 || block % group) return false;
  const int G = block / group;
  if (G != 1 && G != 2 && G != 4 && G != 8) return false;
  return ((int64_t)group * head_dim) % BK == 0;
}

hipError_t launch_estimate(const EstimateLaunch& L, hipStream_t stream) {
  const int m = L.h_q / L.h_kv;
  if (m > 8) return hipErrorInvalidValue;
  ScoreArgs a;
  a.q = static_cast<const bf16_t*>(L.q);
  a.q_sh = L.q_sh;
  a.q_st = L.q_st;
  a.kv = L.kv;
  a.scores = L.scores;
  a.h_q = L.h_q;
  a.h_kv = L.h_kv;
  a.m = m;
  a.C = L.head_dim;
  a.g = L.group;
  a.b = L.block;
  a.G = L.block / L.group;
  a.gc = L.group * L.head_dim;
  a.batch = L.batch;
  int n_tiles = 0;
  for (int r = 0; r < a.batch.n_req; ++r) {
    ReqDesc& d = a.batch.r[r];
    if (d.l_kv > MAX_LKV) return hipErrorInvalidValue;
    d.work_begin = n_tiles;
    const int nqg = (d.n_q + a.g - 1) / a.g, nkg = (d.n_kv + a.g - 1) / a.g;
    n_tiles += a.h_q * tiles_of(nqg) * tiles_of(nkg);
  }
  hipError_t e;
  switch (a.G) {
    case 1: e = launch_scores<1>(a, n_tiles, stream); break;
    case 2: e = launch_scores<2>(a, n_tiles, stream); break;
    case 4: e = launch_scores<4>(a, n_tiles, stream); break;
    case 8: e = launch_scores<8>(a, n_tiles, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;

  SelectArgs s;
  s.scores = L.scores;
  s.dbg = L.scores;  // always fill the non-causal entries (cheap, defined output)
  s.block_mask = L.block_mask;
  s.h_q = L.h_q;
  s.h_kv = L.h_kv;
  s.m = m;
  s.b = L.block;
  s.gamma = L.gamma;
  s.alpha = L.alpha;
  s.batch = L.batch;
  int n_rows = 0;
  for (int r = 0; r < s.batch.n_req; ++r) {
    s.batch.r[r].work_begin = n_rows;
    n_rows += L.h_kv * s.batch.r[r].l_q;
  }
  hipLaunchKernelGGL(select_kernel, dim3(n_rows), dim3(64 * m), 0, stream, s);
  return hipGetLastError();
}

}  // namespace bfla
