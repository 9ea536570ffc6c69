// Stage 1: block-level importance estimation (Sec. 3.2, eq4-eq18) + GQA
// union.  gfx950 / CDNA4, wave64.
//
// Kernel 1 (scores): for every query head p the group-score matrix
//   S_groups[gi][gj] = PhiQ_p[gi] . PhiK_h[gj]       (eq9)
// is a GEMM whose rows are flattened g-token query groups and whose columns
// are flattened key groups (inner dimension g*C; a flattened group of a
// row-major [N][C] head is g consecutive token rows, so no copy is made,
// eq6-eq7).  256 x 128 output tiles, 8 waves of 32 x 128, bf16 MFMA
// 32x32x16; Q/K chunks of 64 inner elements go from buffer loads straight
// into a 3-slot LDS ring (two chunks in flight, one workgroup per CU);
// only tiles holding a causal block pair are computed (eq11-eq14).  The
// epilogue max-pools each G x G group block into the block score (eq10)
// and stores it as float.  Accumulation is two-level: chains of 32 MFMA
// steps (512 products) are summed into a second float accumulator, which
// keeps the score error well inside the near-tie band of the selection.
// When a problem has too few tiles to fill the chip (a split S > 1 from
// estimate_plan), each tile runs as S workgroups over consecutive runs of
// whole chains that store their raw group sums; pool_kernel adds the S sums
// in part order, then pools and stores as the epilogue would.
//
// Kernel 2 (select): one workgroup per (request, KV head, query block),
// one wave per query head of the group: block softmax over the causal KV
// blocks (eq15), keep-mass selection by repeated arg-max in the order
// (score descending, block index ascending) with a sequential float
// running mass (eq16-eq18), then OR of the m heads into the u8 mask row.
// On request each wave also stores its own head's keep set (eq18).
#include <algorithm>

#include "bfla_device.h"
#include "bfla_internal.h"

namespace bfla {
namespace {

constexpr int BM = kScoreTileM;   // query groups per tile (32 per wave)
constexpr int BN = kScoreTileN;   // key groups per tile
constexpr int BK = kScoreChunk;   // inner elements per stage
// 8 waves (two per SIMD): each keeps its own DMA loads in flight, and the
// kernel is bound by the memory requests in flight (4 waves of 64 x 128
// outputs each were 12 % slower)
constexpr int NW = 8;
constexpr int NT = 64 * NW;
constexpr int XB = BM / NW / 32;   // 32-row MFMA blocks per wave
constexpr int CHAIN = kScoreChain;  // stages per inner accumulation chain (32 MFMA k-steps)
constexpr int MAX_LKV = 65536;

struct ScoreArgs {
  const bf16_t* q;
  int64_t q_sh, q_st;
  KvAddr kv;
  float* scores;
  float* partials;   // split > 1: raw group sums [split][tiles][BM][BN]
  int32_t h_q, h_kv, m;
  int32_t C, g, b, G;
  int32_t gc;        // g * C
  int32_t split;     // workgroups per tile, each part_stages stages
  int32_t part_stages;
  int32_t total_tiles;
  Batch batch;       // work_begin = first tile of request r
};

struct SelectArgs {
  const float* scores;
  float* dbg;        // non-null: also fill non-causal entries with -inf
  uint8_t* block_mask;
  uint8_t* head_mask;  // non-null: per-query-head keep sets, score layout
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

__host__ __device__ __forceinline__ int row_tiles(int groups) { return (groups + BM - 1) / BM; }
__host__ __device__ __forceinline__ int col_tiles(int groups) { return (groups + BN - 1) / BN; }

// One ring stage: the Q tile (BM rows) and the K tile (BN rows) of 64 bf16
// each (128 B per row, no padding).  Rows are XOR-swizzled in 16-byte chunks
// (physical chunk = logical chunk ^ ((row / 2) % 8)) so that the 32x32
// fragment reads of 16 consecutive rows hit 16 distinct bank groups.
constexpr int A_ELEMS = BM * BK;
constexpr int B_ELEMS = BN * BK;
constexpr int NSTAGE = 3;     // ring depth: loads run NSTAGE - 1 stages ahead
constexpr int A_LOADS = BM / 8 / NW;   // 1 KB loads per wave per stage (8 rows each)
constexpr int B_LOADS = BN / 8 / NW;
constexpr int VM_STAGE = A_LOADS + B_LOADS;
constexpr uint32_t RSRC_WORD3 = 0x00020000u;
constexpr int PT_MAX = kScorePagesMax;  // page-table entries one tile of a paged cache may span
constexpr uint32_t BAD_PAGE = 0xFFFFFFFFu;

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer descriptor (stride 0, byte range [0, bytes)): offsets at or past
// `bytes` read as zeros.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)b);
  r[1] = __builtin_amdgcn_readfirstlane((int)(uint32_t)(b >> 32) & 0xFFFF);
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = (int)RSRC_WORD3;
  return r;
}

// 16 bytes per lane from a buffer straight into LDS: lane l writes
// [lds + 16 l, +16).  Issued as inline assembly so that the compiler adds no
// waits of its own; the caller waits (vmcnt) and synchronises before the
// data are read.
__device__ __forceinline__ void dma16(i32x4 rs, uint32_t lds, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rs)
               : "memory", "m0");
}

#define LDS_ADDR(arr) ((uint32_t)(uintptr_t)(lds_ptr_t)(arr))

template <int G, bool PAGED>
__global__ void __launch_bounds__(NT, 1) scores_kernel(ScoreArgs a) {
  // ring slot s: Q tile at ring[s][0 .. A_ELEMS), K tile after it
  __shared__ __align__(1024) bf16_t ring[NSTAGE][A_ELEMS + B_ELEMS];
  __shared__ uint32_t page_base[PAGED ? PT_MAX : 1];  // byte offset of each page, or BAD_PAGE

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hi = lane >> 5;

  // ---- tile decode: (split part, request, tile rank, head) with the KV
  // head fastest and the part slowest ----
  const int part = blockIdx.x / a.total_tiles;
  const int tile_id = blockIdx.x - part * a.total_tiles;
  const int ri = find_req(a.batch, tile_id);
  const ReqDesc& R = a.batch.r[ri];
  const int n_q = R.n_q, n_kv = R.n_kv;
  const int64_t q_off = R.q_off, kv_off = R.kv_off;
  const int bt_row = R.bt_row;
  const int local = tile_id - R.work_begin;
  const int nqg = (n_q + a.g - 1) / a.g;    // query groups
  const int nkg = (n_kv + a.g - 1) / a.g;   // key groups
  const int ntj = col_tiles(nkg);
  const int h = local % a.h_kv;
  const int pm = (local / a.h_kv) % a.m;
  const int rank = local / a.h_q;
  const int ti = rank / ntj, tj = rank % ntj;
  const int p = h * a.m + pm;
  const int n_c = n_kv - n_q;

  // skip tiles without any causal block pair
  {
    int gi_last = min(nqg, (ti + 1) * BM) - 1;
    int i_max = gi_last / G;
    int e_i = min(n_c + (i_max + 1) * a.b - 1, n_kv - 1);
    int j_min = (tj * BN) / G;
    if (j_min * a.b > e_i) return;
  }

  // ---- direct global -> LDS loads through buffer descriptors ----
  // Wave w, load i fills rows [8 (NW i + w), +8) of the Q (i < A_LOADS) or K
  // (i < B_LOADS) tile: lane l writes LDS chunk l % 8 of row 8 (NW i + w) +
  // l / 8 and fetches the logical chunk that the swizzle places there.  Out-of-range offsets
  // (padding groups, tokens past the end, bad pages) read as zeros.  The Q
  // descriptor starts at the tile's first query token, so it spans at most
  // BM * g token rows.
  const int q_tok0 = ti * BM * a.g;
  const int q_tile_tok = min(n_q - q_tok0, BM * a.g);
  const i32x4 qrs =
      make_rsrc(a.q + q_off + (int64_t)p * a.q_sh + (int64_t)q_tok0 * a.q_st,
                (uint32_t)(((int64_t)(q_tile_tok - 1) * a.q_st + a.C) * 2));
  const i32x4 krs =
      make_rsrc(a.kv.k + (PAGED ? 0 : kv_off) + (int64_t)h * a.kv.stride_head,
                PAGED ? a.kv.pool_bytes
                      : (uint32_t)(((int64_t)(n_kv - 1) * a.kv.stride_tok + a.C) * 2));
  const int ps_shift = PAGED ? __builtin_ctz(a.kv.page_size) : 0;
  const int k_tok0 = tj * BN * a.g;                 // first key token of the tile (< n_kv)
  const int first_page = k_tok0 >> ps_shift;
  if (PAGED) {
    // the pages this tile's keys live in, resolved once: byte offset of each
    // page in the pool, or BAD_PAGE for an entry outside [0, n_pages)
    const int32_t* bt = a.kv.block_table + (int64_t)bt_row * a.kv.max_pages;
    const int n_pt = ((min(n_kv, k_tok0 + BN * a.g) - 1) >> ps_shift) - first_page + 1;
    const uint32_t page_bytes = (uint32_t)(a.kv.page_stride * 2);
    for (int e = tid; e < n_pt; e += NT) {
      const int pg = bt[first_page + e];
      page_base[e] = (unsigned)pg < (unsigned)a.kv.n_pages ? (uint32_t)pg * page_bytes : BAD_PAGE;
    }
    __syncthreads();
  }
  const int row_sub = lane >> 3, pch = lane & 7;
  int q_row_tok[A_LOADS], k_row_tok[B_LOADS];   // first token of each loaded row's group
  int lch[A_LOADS];                             // logical chunk fetched by this lane
  bool q_ok[A_LOADS], k_ok[B_LOADS];
#pragma unroll
  for (int i = 0; i < A_LOADS; ++i) {
    const int row = 8 * (NW * i + wave) + row_sub;   // the K rows are the first B_LOADS of these
    lch[i] = swz(row, pch);
    q_ok[i] = ti * BM + row < nqg;
    q_row_tok[i] = row * a.g;   // relative to q_tok0
    if (i < B_LOADS) {
      const int gj = tj * BN + row;
      k_ok[i] = gj < nkg;
      k_row_tok[i] = gj * a.g;
    }
  }
  const uint32_t ring_lds = LDS_ADDR(&ring[0][0]) + (uint32_t)wave * 1024;
  constexpr uint32_t SLOT_BYTES = (A_ELEMS + B_ELEMS) * 2;
  auto issue = [&](int st) __attribute__((always_inline)) {
    const uint32_t la = ring_lds + (uint32_t)(st % NSTAGE) * SLOT_BYTES;
    const uint32_t lb = la + A_ELEMS * 2;
    const int k0 = st * BK;
    const int tok_in = k0 / a.C, ch = k0 % a.C;
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
      const int tq = q_row_tok[i] + tok_in;
      const uint32_t qo = (q_ok[i] && tq < q_tile_tok)
                              ? (uint32_t)(((int64_t)tq * a.q_st + ch + 8 * lch[i]) * 2)
                              : 0x80000000u;
      dma16(qrs, la + i * (NW * 1024), qo);
    }
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
      const int tk = k_row_tok[i] + tok_in;
      uint32_t ko = 0x80000000u;
      if (k_ok[i] && tk < n_kv) {
        if (PAGED) {
          const uint32_t pb = page_base[(tk >> ps_shift) - first_page];
          if (pb != BAD_PAGE)
            ko = pb + (uint32_t)((((tk & (a.kv.page_size - 1)) * a.kv.stride_tok) + ch +
                                  8 * lch[i]) * 2);
        } else {
          ko = (uint32_t)(((int64_t)tk * a.kv.stride_tok + ch + 8 * lch[i]) * 2);
        }
      }
      dma16(krs, lb + i * (NW * 1024), ko);
    }
  };

  // wave w: query-group rows [32 w, +32) x all BN key-group columns
  f32x16 acc[XB][4], tot[XB][4];
#pragma unroll
  for (int x = 0; x < XB; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y)
#pragma unroll
      for (int r = 0; r < 16; ++r) { acc[x][y][r] = 0.f; tot[x][y][r] = 0.f; }

  // this workgroup's stages: a run of whole chains
  const int st_begin = part * a.part_stages;
  const int st_end = st_begin + a.part_stages;
  auto compute = [&](const bf16_t* A, const bf16_t* B) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 af[XB], bf[4];
#pragma unroll
      for (int x = 0; x < XB; ++x) {
        const int row = (BM / NW) * wave + 32 * x + l32;
        af[x] = __builtin_bit_cast(bf16x8, ld16(A + row * BK + 8 * swz(row, 2 * ks + hi)));
      }
#pragma unroll
      for (int y = 0; y < 4; ++y) {
        const int row = 32 * y + l32;
        bf[y] = __builtin_bit_cast(bf16x8, ld16(B + row * BK + 8 * swz(row, 2 * ks + hi)));
      }
#pragma unroll
      for (int x = 0; x < XB; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) acc[x][y] = mfma32(af[x], bf[y], acc[x][y]);
    }
  };
  // s_waitcnt immediates: vmcnt(n) with the other counters left free
  constexpr int VM_AHEAD = 0x0F70 | VM_STAGE, VM0 = 0x0F70;
  static_assert(NSTAGE == 3 && VM_STAGE < 16, "one stage ahead, vmcnt below 16");

  // prologue: stages st_begin .. st_begin + NSTAGE - 2 in flight
  for (int st = st_begin; st < st_begin + NSTAGE - 1 && st < st_end; ++st) issue(st);
  for (int c0 = st_begin; c0 < st_end; c0 += CHAIN) {
    const int c1 = min(c0 + CHAIN, st_end);
    for (int st = c0; st < c1; ++st) {
      // this wave's loads of stage st are done once at most the loads of the
      // stage after it (VM_STAGE) remain; the barrier then makes every wave's
      // part visible, and also tells that every wave is done reading the slot
      // refilled next (stage st - 1's)
      if (st + 1 < st_end) __builtin_amdgcn_s_waitcnt(VM_AHEAD);
      else __builtin_amdgcn_s_waitcnt(VM0);
      // plain barrier: a __syncthreads() fence would also wait for the
      // loads still in flight for the later stages
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      if (st + NSTAGE - 1 < st_end) issue(st + NSTAGE - 1);
      const int slot = st % NSTAGE;
      compute(&ring[slot][0], &ring[slot][A_ELEMS]);
    }
    // close the chain: fold it into the running total
#pragma unroll
    for (int x = 0; x < XB; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y)
#pragma unroll
        for (int r = 0; r < 16; ++r) { tot[x][y][r] += acc[x][y][r]; acc[x][y][r] = 0.f; }
  }

  // ---- split: store this part's raw group sums (pool_kernel finishes) ----
  // D[row = query group][col = key group]; lane: col l32, rows 8(r/4)+4hi+r%4
  if (a.split > 1) {
    float* dst = a.partials + (int64_t)blockIdx.x * (BM * BN);
#pragma unroll
    for (int x = 0; x < XB; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = (BM / NW) * wave + 32 * x + 8 * (r >> 2) + 4 * hi + (r & 3);
          dst[row * BN + 32 * y + l32] = tot[x][y][r];
        }
    return;
  }

  // ---- epilogue: drop padded groups, G x G max pool, causal store ----
  float* srow_base = a.scores + R.score_off + (int64_t)p * R.l_q * R.l_kv;
#pragma unroll
  for (int x = 0; x < XB; ++x) {
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      const int gj = tj * BN + 32 * y + l32;
      f32x16 v = tot[x][y];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int gi = ti * BM + (BM / NW) * wave + 32 * x + 8 * (r >> 2) + 4 * hi + (r & 3);
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
      if (G >= 16) {   // rows 8 (r / 4) .. +7 -> 16 consecutive rows
#pragma unroll
        for (int r = 0; r < 16; r += 8) pr[r] = fmaxf(pr[r], pr[r + 4]);
      }
      // pool over G consecutive key-group columns (lanes)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (G >= 2) pr[r] = fmaxf(pr[r], __shfl_xor(pr[r], 1));
        if (G >= 4) pr[r] = fmaxf(pr[r], __shfl_xor(pr[r], 2));
        if (G >= 8) pr[r] = fmaxf(pr[r], __shfl_xor(pr[r], 4));
        if (G >= 16) pr[r] = fmaxf(pr[r], __shfl_xor(pr[r], 8));
      }
      if ((l32 % G) != 0 || (G >= 8 && hi != 0)) continue;
      const int j = gj / G;
      if (j >= R.l_kv) continue;
#pragma unroll
      for (int r = 0; r < 16; r += (G >= 16 ? 8 : G >= 4 ? 4 : G)) {
        const int gi = ti * BM + (BM / NW) * wave + 32 * x + 8 * (r >> 2) + 4 * hi + (r & 3);
        const int i = gi / G;
        if (i >= R.l_q) continue;
        const int e_i = min(n_c + (i + 1) * a.b - 1, R.n_kv - 1);
        if (j * a.b <= e_i) srow_base[(int64_t)i * R.l_kv + j] = pr[r];
      }
    }
  }
}

// Finish of a split score tile, POOL_ROWS group rows per workgroup: the
// group sums of the `split` parts are added in part order (into LDS), then
// padded groups are dropped, each G x G group block is max-pooled into its
// block score (eq10) and the causal blocks are stored (eq11-eq14) -- what
// the epilogue of an unsplit tile does.
constexpr int POOL_ROWS = 32;
constexpr int POOL_THREADS = 256;

template <int G>
__global__ void __launch_bounds__(POOL_THREADS) pool_kernel(ScoreArgs a) {
  __shared__ float sum[POOL_ROWS][BN + 4];
  constexpr int CHUNKS = BM / POOL_ROWS;
  const int tile_id = blockIdx.x / CHUNKS;
  const int chunk = blockIdx.x % CHUNKS;
  const int ri = find_req(a.batch, tile_id);
  const ReqDesc& R = a.batch.r[ri];
  const int n_q = R.n_q, n_kv = R.n_kv;
  const int local = tile_id - R.work_begin;
  const int nqg = (n_q + a.g - 1) / a.g;
  const int nkg = (n_kv + a.g - 1) / a.g;
  const int ntj = col_tiles(nkg);
  const int h = local % a.h_kv;
  const int pm = (local / a.h_kv) % a.m;
  const int rank = local / a.h_q;
  const int ti = rank / ntj, tj = rank % ntj;
  const int p = h * a.m + pm;
  const int n_c = n_kv - n_q;
  {
    int gi_last = min(nqg, (ti + 1) * BM) - 1;
    int i_max = gi_last / G;
    int e_i = min(n_c + (i_max + 1) * a.b - 1, n_kv - 1);
    int j_min = (tj * BN) / G;
    if (j_min * a.b > e_i) return;   // no causal block pair: no part ran
  }
  const int row0 = chunk * POOL_ROWS;             // first group row of this chunk
  if (ti * BM + row0 >= nqg) return;              // only padding rows
  const int64_t part_stride = (int64_t)a.total_tiles * (BM * BN);
  const float* src = a.partials + (int64_t)tile_id * (BM * BN) + (int64_t)row0 * BN;
  // 1. the parts' group sums, in part order, 4 columns per thread
  for (int e = threadIdx.x; e < POOL_ROWS * (BN / 4); e += POOL_THREADS) {
    const int r = e / (BN / 4), c4 = e % (BN / 4);
    const float* s0 = src + r * BN + 4 * c4;
    float4 v = *reinterpret_cast<const float4*>(s0);
    for (int q = 1; q < a.split; ++q) {
      const float4 w = *reinterpret_cast<const float4*>(s0 + q * part_stride);
      v.x += w.x;
      v.y += w.y;
      v.z += w.z;
      v.w += w.w;
    }
    sum[r][4 * c4] = v.x;
    sum[r][4 * c4 + 1] = v.y;
    sum[r][4 * c4 + 2] = v.z;
    sum[r][4 * c4 + 3] = v.w;
  }
  __syncthreads();
  // 2. G x G max pool of real groups, causal store
  float* srow_base = a.scores + R.score_off + (int64_t)p * R.l_q * R.l_kv;
  constexpr int PI = POOL_ROWS / G, PJ = BN / G;
  for (int o = threadIdx.x; o < PI * PJ; o += POOL_THREADS) {
    const int ii = o / PJ, jj = o % PJ;
    const int i = (ti * BM + row0) / G + ii, j = tj * PJ + jj;
    if (i >= R.l_q || j >= R.l_kv) continue;
    const int e_i = min(n_c + (i + 1) * a.b - 1, n_kv - 1);
    if (j * a.b > e_i) continue;
    float best = -INFINITY;
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const int gi = ti * BM + row0 + ii * G + u;
#pragma unroll
      for (int v = 0; v < G; ++v) {
        const int gj = tj * BN + jj * G + v;
        if (gi < nqg && gj < nkg) best = fmaxf(best, sum[ii * G + u][jj * G + v]);
      }
    }
    srow_base[(int64_t)i * R.l_kv + j] = best;
  }
}

// Total order of the keep ranking: score descending, then index ascending.
__device__ __forceinline__ bool better(float s1, int j1, float s2, int j2) {
  return s1 > s2 || (s1 == s2 && j1 < j2);
}

// Wave-wide reductions without LDS round trips.  Step k hands every lane
// the partial result of a partner lane in another group of 2^k lanes:
// lane ^ 1 and lane ^ 2 (DPP quad permutations), the lane mirrored in its
// 8 and in its 16 (DPP row_half_mirror, row_mirror), then lane ^ 16 and
// lane ^ 32 (v_permlane16_swap / v_permlane32_swap, which deliver both
// lanes of the pair).  Partners hold the same set of lanes, and a + b ==
// b + a exactly, so every lane ends with the bit-identical result.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, CTRL, 0xF, 0xF, false);
}
constexpr int DPP_XOR1 = 0xB1, DPP_XOR2 = 0x4E, DPP_HALF_MIRROR = 0x141, DPP_MIRROR = 0x140;

template <typename Op>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t x, Op op) {
  x = op(x, dpp_u32<DPP_XOR1>(x));
  x = op(x, dpp_u32<DPP_XOR2>(x));
  x = op(x, dpp_u32<DPP_HALF_MIRROR>(x));
  x = op(x, dpp_u32<DPP_MIRROR>(x));
  const auto p = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = op((uint32_t)p[0], (uint32_t)p[1]);
  const auto q = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return op((uint32_t)q[0], (uint32_t)q[1]);
}
__device__ __forceinline__ float wave_max(float x) {
  return __builtin_bit_cast(float, wave_reduce_u32(__builtin_bit_cast(uint32_t, x),
      [](uint32_t a, uint32_t b) {
        return __builtin_bit_cast(uint32_t, fmaxf(__builtin_bit_cast(float, a),
                                                  __builtin_bit_cast(float, b)));
      }));
}
__device__ __forceinline__ float wave_sum(float x) {
  return __builtin_bit_cast(float, wave_reduce_u32(__builtin_bit_cast(uint32_t, x),
      [](uint32_t a, uint32_t b) {
        return __builtin_bit_cast(uint32_t, __builtin_bit_cast(float, a) +
                                                __builtin_bit_cast(float, b));
      }));
}
// (score, block) pair that ranks first under better(), in every lane
__device__ __forceinline__ void wave_best(float& s, int& j) {
  auto step = [&](float os, int oj) {
    if (better(os, oj, s, j)) { s = os; j = oj; }
  };
  auto sw = [](float x) { return __builtin_bit_cast(uint32_t, x); };
  auto fl = [](uint32_t x) { return __builtin_bit_cast(float, x); };
  step(fl(dpp_u32<DPP_XOR1>(sw(s))), (int)dpp_u32<DPP_XOR1>((uint32_t)j));
  step(fl(dpp_u32<DPP_XOR2>(sw(s))), (int)dpp_u32<DPP_XOR2>((uint32_t)j));
  step(fl(dpp_u32<DPP_HALF_MIRROR>(sw(s))), (int)dpp_u32<DPP_HALF_MIRROR>((uint32_t)j));
  step(fl(dpp_u32<DPP_MIRROR>(sw(s))), (int)dpp_u32<DPP_MIRROR>((uint32_t)j));
  {
    const auto ps = __builtin_amdgcn_permlane16_swap(sw(s), sw(s), false, false);
    const auto pj = __builtin_amdgcn_permlane16_swap((uint32_t)j, (uint32_t)j, false, false);
    s = fl((uint32_t)ps[0]);
    j = (int)pj[0];
    step(fl((uint32_t)ps[1]), (int)pj[1]);
  }
  {
    const auto ps = __builtin_amdgcn_permlane32_swap(sw(s), sw(s), false, false);
    const auto pj = __builtin_amdgcn_permlane32_swap((uint32_t)j, (uint32_t)j, false, false);
    s = fl((uint32_t)ps[0]);
    j = (int)pj[0];
    step(fl((uint32_t)ps[1]), (int)pj[1]);
  }
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

  // this head's own keep set: cleared here (every head keeps all causal
  // blocks when gamma >= 1); the barrier below orders these stores before
  // the picks that lane 0 stores during the selection
  uint8_t* hrow = a.head_mask
                      ? a.head_mask + R.score_off + ((int64_t)p * R.l_q + i) * R.l_kv
                      : nullptr;
  if (hrow)
    for (int j = lane; j < R.l_kv; j += 64) hrow[j] = (a.gamma >= 1.0f && j < n_causal) ? 1 : 0;
  for (int w = tid; w < words; w += blockDim.x) keep_bits[w] = 0u;
  __syncthreads();

  const float* row = a.scores + R.score_off + ((int64_t)p * R.l_q + i) * R.l_kv;

  if (a.gamma >= 1.0f) {
    for (int j = tid; j < n_causal; j += blockDim.x) atomicOr(&keep_bits[j >> 5], 1u << (j & 31));
  } else {
    // Rows of up to 64 * ROW_REGS causal blocks (every row up to 128K tokens
    // at b = 128) are read once into registers, lane l holding blocks
    // l, l + 64, ...; longer rows are re-read from memory on every pass.  Both
    // paths visit the blocks in the same per-lane order, so the statistics and
    // the picks are bit-identical.
    constexpr int ROW_REGS = 16;
    const bool in_regs = n_causal <= 64 * ROW_REGS;
    float rv[ROW_REGS];
#pragma unroll
    for (int k = 0; k < ROW_REGS; ++k) {
      const int j = lane + 64 * k;
      rv[k] = (in_regs && j < n_causal) ? row[j] : -INFINITY;
    }
    // f(j, s) for every causal block j of this lane, in increasing j
    auto for_each = [&](auto&& f) __attribute__((always_inline)) {
      if (in_regs) {
#pragma unroll
        for (int k = 0; k < ROW_REGS; ++k)
          if (lane + 64 * k < n_causal) f(lane + 64 * k, rv[k]);
      } else {
        for (int j = lane; j < n_causal; j += 64) f(j, row[j]);
      }
    };
    // softmax statistics (eq15)
    float mx = -INFINITY;
    for_each([&](int, float s) { mx = fmaxf(mx, s); });
    mx = wave_max(mx);
    float z = 0.f;
    for_each([&](int, float s) { z += expf(a.alpha * (s - mx)); });
    z = wave_sum(z);

    // keep-mass selection (eq16-eq18): repeated arg-max below the last pick
    float mass = 0.f;
    float s_prev = INFINITY;
    int j_prev = -1;
    for (int taken = 0; taken < n_causal; ++taken) {
      float bs = -INFINITY;
      int bj = INT_MAX;
      for_each([&](int j, float s) {
        if (better(s_prev, j_prev, s, j) && better(s, j, bs, bj)) { bs = s; bj = j; }
      });
      wave_best(bs, bj);
      if (bj >= n_causal) break;  // only with non-finite scores: nothing left to rank
      if (lane == 0) {
        atomicOr(&keep_bits[bj >> 5], 1u << (bj & 31));
        if (hrow) hrow[bj] = 1;
      }
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
  const dim3 grid((unsigned)((int64_t)n_tiles * a.split));
  if (a.kv.paged)
    hipLaunchKernelGGL((scores_kernel<G, true>), grid, dim3(NT), 0, s, a);
  else
    hipLaunchKernelGGL((scores_kernel<G, false>), grid, dim3(NT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.split == 1) return e;
  hipLaunchKernelGGL((pool_kernel<G>), dim3((unsigned)n_tiles * (BM / POOL_ROWS)),
                     dim3(POOL_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_estimate(const EstimateLaunch& L, hipStream_t stream) {
  const int m = L.h_q / L.h_kv;
  if (m > 8) return hipErrorInvalidValue;
  ScoreArgs a;
  a.q = static_cast<const bf16_t*>(L.q);
  a.q_sh = L.q_sh;
  a.q_st = L.q_st;
  a.kv = L.kv;
  a.scores = L.scores;
  a.partials = L.partials;
  a.h_q = L.h_q;
  a.h_kv = L.h_kv;
  a.m = m;
  a.C = L.head_dim;
  a.g = L.group;
  a.b = L.block;
  a.G = L.block / L.group;
  a.gc = L.group * L.head_dim;
  const int n_stage = a.gc / BK;

  SelectArgs s;
  s.scores = L.scores;
  s.dbg = L.scores;  // always fill the non-causal entries (cheap, defined output)
  s.block_mask = L.block_mask;
  s.head_mask = L.head_mask;
  s.h_q = L.h_q;
  s.h_kv = L.h_kv;
  s.m = m;
  s.b = L.block;
  s.gamma = L.gamma;
  s.alpha = L.alpha;

  // scores (and their pooling when split) then the selection, once per group
  // of kLaunchRequests requests; the groups share the partial-sum buffer in
  // stream order
  const size_t n_groups = (L.reqs.size() + kLaunchRequests - 1) / kLaunchRequests;
  if (L.splits.size() != n_groups) return hipErrorInvalidValue;
  for (size_t gi = 0; gi < n_groups; ++gi) {
    const size_t g0 = gi * kLaunchRequests;
    const int n = (int)std::min<size_t>(kLaunchRequests, L.reqs.size() - g0);
    a.batch.n_req = n;
    int n_tiles = 0;
    for (int r = 0; r < n; ++r) {
      ReqDesc& d = a.batch.r[r];
      d = L.reqs[g0 + r];
      if (d.l_kv > MAX_LKV) return hipErrorInvalidValue;
      d.work_begin = n_tiles;
      const int nqg = (d.n_q + a.g - 1) / a.g, nkg = (d.n_kv + a.g - 1) / a.g;
      n_tiles += a.h_q * row_tiles(nqg) * col_tiles(nkg);
    }
    a.split = L.splits[gi];
    a.total_tiles = n_tiles;
    if (a.split < 1 || (a.split > 1 && (n_stage % (a.split * CHAIN) != 0 || !a.partials)))
      return hipErrorInvalidValue;
    a.part_stages = n_stage / a.split;
    hipError_t e;
    switch (a.G) {
      case 1: e = launch_scores<1>(a, n_tiles, stream); break;
      case 2: e = launch_scores<2>(a, n_tiles, stream); break;
      case 4: e = launch_scores<4>(a, n_tiles, stream); break;
      case 8: e = launch_scores<8>(a, n_tiles, stream); break;
      case 16: e = launch_scores<16>(a, n_tiles, stream); break;
      default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;

    s.batch.n_req = n;
    int n_rows = 0;
    for (int r = 0; r < n; ++r) {
      s.batch.r[r] = L.reqs[g0 + r];
      s.batch.r[r].work_begin = n_rows;
      n_rows += L.h_kv * s.batch.r[r].l_q;
    }
    hipLaunchKernelGGL(select_kernel, dim3(n_rows), dim3(64 * m), 0, stream, s);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace bfla
