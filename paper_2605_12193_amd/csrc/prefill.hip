// Fused GQA flash-style causal prefill over kept KV tiles (eq27), and the
// dense causal baseline (every causal tile).  gfx950 / CDNA4, wave64.
//
// Work item = one list row (request r, KV head h, query tile qt): all m
// query heads of the GQA group share every K/V tile load.  At head dims 64
// and 128 (prefill_kernel) each wave owns 32 queries of one head: 2 waves per
// head (2m per workgroup), or, for the half-tile shapes (m > 4), one wave per
// head over half the q-tile, two work items per row.
//
// Per KV tile (T = 64 keys):
//   S^T[key][query] = K_tile . Q^T   v_mfma_f32_32x32x16_bf16, K from LDS
//                                   (A operand), Q held in registers (B)
//   In the 32x32 accumulator layout a lane owns one query column and 16 key
//   rows, so the row max / row sum of the online softmax are in-lane plus a
//   single exchange with lane ^ 32.
//   O^T[chan][query] += V^T_tile . P^T  P comes straight from the S^T
//                                   accumulators (as bf16) as the B operand;
//   V is staged transposed in LDS with the key order inside every 16-key
//   chunk permuted (bits 2 and 3 of the key offset swapped) so that the
//   accumulator's key order and the A operand's agree.
// K/V tiles go from memory into registers and from there into LDS stages
// (three in the ping-pong schedule of the 8-wave shapes, two otherwise), the
// staging instructions placed between the MFMAs of a stream: two iterations
// ahead through two register sets in the ping-pong, one ahead otherwise.
// K/V are read through buffer descriptors whose range check returns zeros
// past the last key or page, so loads carry no branches.
//
// The lane ^ 32 exchanges of the row max and sum use v_permlane32_swap.
//
// Head dim 256 runs prefill_q16_kernel instead: 16-query waves on
// v_mfma_f32_16x16x32_bf16 over a whole, half or quarter q-tile (at most 8
// waves), K and V in separate two-slot rings offset by one tile (three
// combined stages of 256 channels would not fit the LDS); the same ping-pong
// at GQA 2, all waves in one phase otherwise.
//
// The online softmax keeps a stale running max and takes no max reduction in
// the common case: a tile's weights are computed against the running max and
// kept when every row's weight sum over the tile is <= 2^RESCALE_LOG2 (so is
// every weight).  Otherwise, and on a row's first tile, the tile's max is
// taken, the running max moves up to it where it is larger (O and l
// rescaled) and the weights are recomputed (all <= 1).  O and l always refer
// to the same max, so O / l is exact.
#include <algorithm>
#include <atomic>
#include <utility>

#include "bfla_device.h"
#include "bfla_internal.h"

namespace bfla {
namespace {

constexpr int TILE = 64;
constexpr float LOG2E = 1.4426950408889634f;
constexpr int RESCALE_LOG2 = 8;
constexpr float RESCALE_SUM = float(1 << RESCALE_LOG2);
constexpr uint32_t RSRC_WORD3 = 0x00020000u;  // raw buffer, 32-bit data format
constexpr int VMCNT0 = 0x0F70;                // s_waitcnt vmcnt(0), other counters free

template <int C>
struct Cfg {
  static constexpr int KROW = C + 8;          // K tile row pitch (bf16), padded
  static constexpr int VROW = TILE + 8;       // V^T row pitch (bf16), padded
  static constexpr int K_ELEMS = TILE * KROW;
  static constexpr int V_ELEMS = C * VROW;
  static constexpr int STAGE = K_ELEMS + V_ELEMS;
  // three stages (ping-pong schedule) when they fit the 160 KB of LDS
  static constexpr bool PING_PONG = 3 * STAGE * 2 <= 160 * 1024;
  static constexpr int K_CHUNKS = TILE * C / 8;   // 16-byte chunks per K tile
  static constexpr int V_UNITS = (TILE / 2) * (C / 8);  // key pairs x 8 channels
};

struct PrefillArgs {
  const bf16_t* q;
  bf16_t* o;
  float* lse;
  const int32_t* row_ptr;  // sparse lists (unused when dense)
  const int32_t* cols;
  int64_t q_sh, q_st, o_sh, o_st;
  KvAddr kv;
  int32_t h_q, h_kv, m;
  float scale;
  Batch batch;
};

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint4 ld16(const bf16_t* p) {
  return *reinterpret_cast<const uint4*>(p);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Two floats -> two bf16 (round to nearest even) in one word.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 x = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2));
}

// max / sum of x over lanes l and l ^ 32, in every lane, without going
// through LDS: v_permlane32_swap leaves x of lane l % 32 in one result and
// x of lane 32 + l % 32 in the other.
__device__ __forceinline__ f32x2 lane32_pair(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x),
                                                  __builtin_bit_cast(uint32_t, x), false, false);
  return f32x2{__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1])};
}
__device__ __forceinline__ float max_lane32(float x) {
  const f32x2 p = lane32_pair(x);
  return fmaxf(p[0], p[1]);
}
__device__ __forceinline__ float add_lane32(float x) {
  const f32x2 p = lane32_pair(x);
  return p[0] + p[1];
}

// Position of key offset k (0..63) inside the permuted V^T row.
__device__ __forceinline__ int vperm(int k) {
  return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

// Uniform reads of the tile lists through the constant address space, so
// they become scalar loads (a vector load would be waited on together with the
// in-flight K/V prefetch).
typedef const __attribute__((address_space(4))) int32_t* const_i32_ptr;
__device__ __forceinline__ int uniform_load(const int32_t* p, int i) {
  return ((const_i32_ptr)p)[i];
}

// A block-table entry at byte offset e of a row, read as a scalar.  Through
// readfirstlane: a plain load that feeds a select is sunk into a branch of
// its own, and loads between branches are not issued together, which costs
// one round trip per entry.
__device__ __forceinline__ uint32_t table_entry(const int32_t* row, uint32_t e) {
  typedef const __attribute__((address_space(4))) char* const_byte_ptr;
  return (uint32_t)__builtin_amdgcn_readfirstlane(*(const_i32_ptr)((const_byte_ptr)row + e));
}

// Paged K/V: a 64-key tile spans up to four pages (pages hold >= 16 tokens).
// Its keys are addressed as if the tile were contiguous, boff = (kr * st +
// 8 ce) * 2 for key kr, plus the base of the key's page slot j = kr / ps
// (0 when ps >= 64): base_j = pg_j * page_bytes + (tok0 % ps) * st * 2 -
// j * ps * st * 2.  An entry outside [0, n_pages) gives 2^31, past every
// descriptor's range, so its keys read zeros; rows counts the keys of the
// tile below N_kv, and V units past it are zeroed the same way.  (Named
// fields, not an array: per-lane picks among them must stay selects between
// registers, not indexed scratch loads.)
struct PageBases {
  uint32_t b0, b1, b2, b3;
  int rows;
};
// Tile kt of a request whose block-table row is bt (N_kv >= 1).  Tiles
// outside [0, T_kv) (past the end of a list, or malformed lists) get rows = 0
// and bases of 2^31: their loads read zeros without memory traffic.  The
// four entries from the tile's first page on are read unconditionally,
// clamped to the request's last page, and issued together; slots past the
// tile or past N_kv are never used for keys below N_kv.
__device__ __forceinline__ PageBases page_bases(const int32_t* bt, int kt, int t_kv, int n_kv,
                                                int ps_shift, uint32_t n_pages,
                                                uint32_t page_bytes, uint32_t tok_bytes) {
  const bool ok = (unsigned)kt < (unsigned)t_kv;
  const int tok0 = ok ? kt * TILE : 0;
  PageBases pb;
  pb.rows = ok ? min(n_kv - tok0, TILE) : 0;
  const uint32_t in_page = (uint32_t)(tok0 & ((1 << ps_shift) - 1)) * tok_bytes;
  const uint32_t slot_step = tok_bytes << ps_shift;
  const uint32_t e0 = (uint32_t)(tok0 >> ps_shift) * 4u;
  const uint32_t last_e = (uint32_t)((n_kv - 1) >> ps_shift) * 4u;
  uint32_t pg[4], b[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) pg[j] = table_entry(bt, min(e0 + 4u * j, last_e));
#pragma unroll
  for (int j = 0; j < 4; ++j)
    b[j] = ok && pg[j] < n_pages ? pg[j] * page_bytes + in_page - (uint32_t)j * slot_step
                                 : 0x80000000u;
  pb.b0 = b[0];
  pb.b1 = b[1];
  pb.b2 = b[2];
  pb.b3 = b[3];
  return pb;
}
// The four bases in lanes 0-3 of one register, written whatever the exec
// mask (the other lanes are unused): a wave whose K rows of a round lie in
// one page reads its base with one readlane.
__device__ __forceinline__ int page_lanes(const PageBases pb) {
  int vb;
  asm("v_writelane_b32 %0, %1, 0" : "=v"(vb) : "s"(pb.b0));
  asm("v_writelane_b32 %0, %1, 1" : "+v"(vb) : "s"(pb.b1));
  asm("v_writelane_b32 %0, %1, 2" : "+v"(vb) : "s"(pb.b2));
  asm("v_writelane_b32 %0, %1, 3" : "+v"(vb) : "s"(pb.b3));
  return vb;
}
// V: a thread's key pair (2 j, 2 j + 1) lies in one page slot (hi, lo bits
// of the slot index, fixed per thread); the base of each key, or 2^31 for a
// key past N_kv.
__device__ __forceinline__ void v_pair_bases(const PageBases pb, bool hi, bool lo, int key0,
                                             uint32_t& b_first, uint32_t& b_second) {
  const uint32_t bv = hi ? (lo ? pb.b3 : pb.b2) : (lo ? pb.b1 : pb.b0);
  b_first = key0 < pb.rows ? bv : 0x80000000u;
  b_second = key0 + 1 < pb.rows ? bv : 0x80000000u;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           (int)RSRC_WORD3);
}

__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}

// every lambda of the kernel body is inlined (the loop calls some of them
// from several places, which the inliner would otherwise turn into calls)
#define INLINE __attribute__((always_inline))

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;
#define LDS_ADDR(arr) ((uint32_t)(uintptr_t)(lds_ptr_t)(arr))

// f(std::integral_constant<int, 0>) ... f(std::integral_constant<int, N - 1>),
// so that the body can use its index as a constant (immediate operands).
template <typename F, int... I>
__device__ __forceinline__ void static_for_seq(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_seq(f, std::make_integer_sequence<int, N>{});
}

// 16-byte LDS read issued exactly where it stands.  The result is in flight
// until a later lgkm_wait on the same value; the compiler does not track it.
template <int OFF>
__device__ __forceinline__ void lds_read(u32x4& r, uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds_read offset field is 16 bits");
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF) : "memory");
}
// Wait until at most N LDS/scalar-memory operations are outstanding.  r is an
// in/out operand so that no use of r can move above the wait.  LDS operations
// complete in issue order, so waiting for N leaves only the last N reads
// pending; other LDS or scalar loads in flight can only make it stricter.
template <int N>
__device__ __forceinline__ void lgkm_wait(u32x4& r) {
  static_assert(N >= 0 && N < 16, "lgkmcnt field is 4 bits");
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(r) : "i"(N));
}

// Shapes whose 2m-wave workgroup would cap registers below what the loop
// needs run half q-tiles instead: m waves of 32 queries, one per head, still
// sharing every K/V tile across the group.  At C <= 128 that is m > 4 (more
// than two waves on a SIMD).
__host__ __device__ constexpr bool half_shape(int c, int m) { return m > 4; }
// Head dim 256 runs on 16-query waves (a 32-query wave's 256-channel O, Q and
// S would leave one wave per SIMD), prefill_q16_kernel.  A work item covers
// QB 16-query blocks of one q-tile for all m heads, so that it has
// m * QB <= 8 waves: the whole tile at m <= 2, half at m = 3, 4, a quarter
// at m >= 5.
__host__ __device__ constexpr int q16_blocks(int m) { return m <= 2 ? 4 : m <= 4 ? 2 : 1; }
// work items per list row (request, KV head, q-tile)
__host__ __device__ constexpr int parts_per_row(int c, int m) {
  return c == 256 ? 4 / q16_blocks(m) : half_shape(c, m) ? 2 : 1;
}
template <int C, int M>
struct Shape {
  static constexpr bool HALF = half_shape(C, M);
  static constexpr int WAVES = HALF ? M : 2 * M;
};

template <int C, int M, bool DENSE, bool PAGED>
__global__ void __launch_bounds__(64 * (Shape<C, M>::WAVES))
prefill_kernel(PrefillArgs a) {
  using CF = Cfg<C>;
  constexpr bool HALF = Shape<C, M>::HALF;
  // ping-pong needs two groups of 4 waves, one wave of each per SIMD
  constexpr bool PP = CF::PING_PONG && Shape<C, M>::WAVES == 8;
  constexpr int NT = 64 * Shape<C, M>::WAVES;
  constexpr int KC_PER_T = (CF::K_CHUNKS + NT - 1) / NT;
  constexpr int VU_PER_T = (CF::V_UNITS + NT - 1) / NT;
  constexpr int NKC = C / 16;   // 16-channel chunks of the QK^T contraction
  constexpr int NCB = C / 32;   // 32-channel blocks of O^T

  extern __shared__ __align__(16) bf16_t lds[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int hi = lane >> 5;

  // ---- work item -> (request, kv head, q-tile), longest rows first ----
  const int w = blockIdx.x;
  const int ri = find_req(a.batch, w);
  const ReqDesc& Rd = a.batch.r[ri];
  const int n_q = Rd.n_q, n_kv = Rd.n_kv, t_q = Rd.t_q, t_kv = Rd.t_kv;
  const int64_t q_off = Rd.q_off, o_off = Rd.o_off, kv_off = Rd.kv_off, lse_off = Rd.lse_off;
  const int bt_row = Rd.bt_row;
  const int local = w - Rd.work_begin;
  const int h = local % a.h_kv;
  const int rank = local / a.h_kv;
  const int qt = t_q - 1 - (HALF ? rank >> 1 : rank);
  const int row = Rd.row_base + h * t_q + qt;
  const int n_c = n_kv - n_q;

  int list_begin = 0, n_tiles;
  if (DENSE) {
    n_tiles = min(n_c + (qt + 1) * TILE - 1, n_kv - 1) / TILE + 1;
  } else {
    list_begin = uniform_load(a.row_ptr, row);
    n_tiles = uniform_load(a.row_ptr, row + 1) - list_begin;
  }

  // ---- this wave's queries ----
  const int p = h * a.m + (HALF ? wave : wave >> 1);
  const int half = HALF ? (rank & 1) : (wave & 1);
  const int t = qt * TILE + half * 32 + l32;          // query index in request
  const bool q_ok = t < n_q;
  const int q_pos = n_c + t;                          // absolute position
  const int wave_q0 = n_c + qt * TILE + half * 32;
  const int key_lim = min(q_pos, n_kv - 1);           // last admissible key

  // Q is fetched as whole rows (C / 8 lanes per row, 16 bytes per lane; a
  // lane's MFMA fragments are 16-byte pieces of one row, and loading those
  // directly makes every load touch 32 rows), then redistributed through the
  // still-empty K/V stages by q_from_lds().  Both prologues issue their
  // first tile fetches before that call, so the Q and K/V round trips
  // overlap.
  bf16x8 qf[NKC];
  constexpr int QROW = C + 8, QLPR = C / 8, QRPI = 64 / QLPR;
  uint4 qv[32 / QRPI];
  {
    const int r0 = lane / QLPR, ch = 8 * (lane % QLPR);
    const int t0 = qt * TILE + half * 32;
    const bf16_t* const qb = a.q + q_off + (int64_t)p * a.q_sh;
#pragma unroll
    for (int i = 0; i < 32 / QRPI; ++i) {
      // rows past N_q (never stored) repeat the last query: the loads need
      // no branch, and the compiler then issues them back to back
      const int r = min(t0 + r0 + QRPI * i, n_q - 1);
      qv[i] = ld16(qb + (int64_t)r * a.q_st + ch);
    }
  }
  auto q_from_lds = [&]() INLINE {
    bf16_t* const qs = lds + wave * 32 * QROW;
    const int r0 = lane / QLPR, ch = 8 * (lane % QLPR);
#pragma unroll
    for (int i = 0; i < 32 / QRPI; ++i)
      *reinterpret_cast<uint4*>(qs + (r0 + QRPI * i) * QROW + ch) = qv[i];
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc)
      qf[kc] = as_bf16x8(*reinterpret_cast<const uint4*>(qs + l32 * QROW + 16 * kc + 8 * hi));
    __syncthreads();   // every wave holds its Q before the K/V stages are written
  };

  // ---- K/V addressing ----
  // Contiguous: one descriptor per head spanning its N_kv rows.  Paged: one
  // descriptor over the whole pool (offset by the head); keys past N_kv and
  // table entries outside the pool land outside the range and read zeros.
  const int64_t st = a.kv.stride_tok;
  __amdgpu_buffer_rsrc_t krs, vrs;
  if (!PAGED) {
    const int64_t head_off = kv_off + (int64_t)h * a.kv.stride_head;
    const uint32_t bytes = (uint32_t)(((int64_t)(n_kv - 1) * st + C) * 2);
    krs = make_rsrc(a.kv.k + head_off, bytes);
    vrs = make_rsrc(a.kv.v + head_off, bytes);
  } else {
    const int64_t head_off = (int64_t)h * a.kv.stride_head;
    krs = make_rsrc(a.kv.k + head_off, a.kv.pool_bytes);
    vrs = make_rsrc(a.kv.v + head_off, a.kv.pool_bytes);
  }
  const int ps = a.kv.page_size;  // power of two >= 16
  const int ps_shift = __builtin_ctz(ps);
  const uint32_t page_bytes = (uint32_t)(a.kv.page_stride * 2);
  const int32_t* bt = a.kv.block_table + (int64_t)bt_row * a.kv.max_pages;
  // Per-thread constant parts of the staging pattern.  A thread stages K
  // chunks e = tid + i NT (row e / (C / 8), channels 8 (e % (C / 8)) on) and
  // V units u = tid + i NT (key pair u % 32, fastest, so that the 16 lanes of
  // one LDS store phase write 16 consecutive words of one V^T row; channels
  // 8 (u / 32) on).  NT is a multiple of C / 8 and of 32, so round i only
  // moves the K row by i K_ROW_STEP and the V channel group by i V_CE_STEP:
  // one register holds each offset of round 0 and the steps are scalars or
  // immediates (offsets kept per round would hold KC_PER_T + VU_PER_T VGPRs
  // for the whole kernel).
  constexpr int K_ROW_STEP = NT / (C / 8), V_CE_STEP = NT / (TILE / 2);
  static_assert(NT % (C / 8) == 0 && NT % (TILE / 2) == 0, "rounds must keep a thread's column");
  const int k_row = tid / (C / 8), k_ce = tid % (C / 8);
  const uint32_t k_boff = (uint32_t)(((int64_t)k_row * st + 8 * k_ce) * 2);  // round 0, in a tile
  const uint32_t k_step = (uint32_t)(K_ROW_STEP * st * 2);
  const int v_j = tid % (TILE / 2), v_ce = tid / (TILE / 2);
  const uint32_t v_boff = (uint32_t)(((int64_t)(2 * v_j) * st + 8 * v_ce) * 2);
  constexpr uint32_t V_STEP = V_CE_STEP * 8 * 2;
  const uint32_t tile_bytes = (uint32_t)(TILE * st * 2);
  const uint32_t st_bytes = (uint32_t)(st * 2);
  // page slot (0-3) inside a tile of this wave's K rows in round i, and of
  // this thread's V key pair (paged K/V)
  int kj[KC_PER_T];
  {
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
#pragma unroll
    for (int i = 0; i < KC_PER_T; ++i)
      kj[i] = ps < TILE ? ((wave_u * 64 + i * NT) / (C / 8)) >> ps_shift : 0;
  }
  const int v_slot = ps < TILE ? (2 * v_j) >> ps_shift : 0;
  const bool vj_hi = (v_slot & 2) != 0, vj_lo = (v_slot & 1) != 0;

  // Ping-pong shapes split the staging between the groups instead: group A
  // (waves 0-3) stages every V unit of a tile, group B (waves 4-7) every K
  // chunk, each with the pattern above over its GT threads.
  constexpr int GT = NT / 2;
  constexpr int KC_B = PP ? CF::K_CHUNKS / GT : 0, VU_A = PP ? CF::V_UNITS / GT : 0;
  static_assert(!PP || (CF::K_CHUNKS % GT == 0 && CF::V_UNITS % GT == 0), "group staging");
  constexpr int K_ROW_STEP_G = GT / (C / 8), V_CE_STEP_G = GT / (TILE / 2);
  const int gtid = tid & (GT - 1);
  const int k_row_g = gtid / (C / 8), k_ce_g = gtid % (C / 8);
  const uint32_t k_boff_g = (uint32_t)(((int64_t)k_row_g * st + 8 * k_ce_g) * 2);
  const uint32_t k_step_g = (uint32_t)(K_ROW_STEP_G * st * 2);
  const int v_ce_g = gtid / (TILE / 2);   // v_j is the same as above
  const uint32_t v_boff_g = (uint32_t)(((int64_t)(2 * v_j) * st + 8 * v_ce_g) * 2);
  constexpr uint32_t V_STEP_G = V_CE_STEP_G * 8 * 2;
  int kj_g[KC_B > 0 ? KC_B : 1];   // group B: page slot of the wave's K rows in round i
  {
    const int wave_g = __builtin_amdgcn_readfirstlane(wave) & 3;
#pragma unroll
    for (int i = 0; i < KC_B; ++i)
      kj_g[i] = ps < TILE ? ((wave_g * 64 + i * GT) / (C / 8)) >> ps_shift : 0;
  }

  // Five- and six-wave work items (GQA 5; GQA 3 and 6): the waves sit on
  // four SIMDs, waves w and w + 4 on the same one (w = 0, and 1 with six
  // waves), which therefore carries twice the MFMA and softmax work.  Only
  // the waves alone on their SIMD (1-3, or 2-3) stage tiles, with the same
  // pattern over their threads, so the doubled SIMDs carry no staging.  (With
  // seven waves one wave would stage a whole tile: 128 VGPRs of staging.)
  constexpr bool SOLO = !PP && (Shape<C, M>::WAVES == 5 || Shape<C, M>::WAVES == 6);
  constexpr int SW0 = Shape<C, M>::WAVES - 4;   // first staging wave
  constexpr int SNT = (4 - SW0) * 64;
  constexpr int KC_S = SOLO ? (CF::K_CHUNKS + SNT - 1) / SNT : 0, VU_S = SOLO ? (CF::V_UNITS + SNT - 1) / SNT : 0;
  constexpr int K_ROW_STEP_S = SNT / (C / 8), V_CE_STEP_S = SNT / (TILE / 2);
  const int sidx = tid - 64 * SW0;   // 0 .. SNT - 1 on the staging waves
  const bool stager = SOLO && __builtin_amdgcn_readfirstlane(wave) >= SW0 &&
                      __builtin_amdgcn_readfirstlane(wave) <= 3;
  const int k_row_s = sidx / (C / 8), k_ce_s = sidx % (C / 8);
  const uint32_t k_boff_s = (uint32_t)(((int64_t)k_row_s * st + 8 * k_ce_s) * 2);
  const uint32_t k_step_s = (uint32_t)(K_ROW_STEP_S * st * 2);
  const int v_ce_s = sidx / (TILE / 2);
  const uint32_t v_boff_s = (uint32_t)(((int64_t)(2 * v_j) * st + 8 * v_ce_s) * 2);
  constexpr uint32_t V_STEP_S = V_CE_STEP_S * 8 * 2;
  int kj_s[KC_S > 0 ? KC_S : 1];
  {
    const int wave_s = __builtin_amdgcn_readfirstlane(wave) - SW0;
#pragma unroll
    for (int i = 0; i < KC_S; ++i)
      kj_s[i] = ps < TILE ? ((wave_s * 64 + i * SNT) / (C / 8)) >> ps_shift : 0;
  }
  // one K/V tile on its way from memory to LDS, in registers
  constexpr int KS0 = KC_PER_T > KC_B ? KC_PER_T : KC_B, VS0 = VU_PER_T > VU_A ? VU_PER_T : VU_A;
  constexpr int KS = KS0 > KC_S ? KS0 : KC_S, VS = VS0 > VU_S ? VS0 : VU_S;
  struct Staged {
    uint4 k[KS];
    uint4 v[VS][2];
  };

  // the page bases of tile kt (paged; scalars)
  const uint32_t n_pages_u = (uint32_t)a.kv.n_pages;
  auto paged_tile = [&](int kt) INLINE -> PageBases {
    return page_bases(bt, kt, t_kv, n_kv, ps_shift, n_pages_u, page_bytes, st_bytes);
  };
  // Fetch this thread's K chunks (part & 1) and/or V units (part & 2) of
  // tile kt into sg.
  auto load_part_pt = [&](int kt, const PageBases pt, Staged& sg, auto part) INLINE {
    constexpr bool LK = (decltype(part)::value & 1) != 0, LV = (decltype(part)::value & 2) != 0;
    // tiles outside [0, T_kv) (malformed lists) load nothing
    const bool ok = (unsigned)kt < (unsigned)t_kv;
    if (!PAGED) {
      // past-the-end offsets (and 2^31 for a bad tile) read as zeros
      const uint32_t base = ok ? (uint32_t)kt * tile_bytes : 0x80000000u;
#pragma unroll
      for (int i = 0; i < KC_PER_T; ++i)
        if (LK && (CF::K_CHUNKS % NT == 0 || tid + i * NT < CF::K_CHUNKS))
          sg.k[i] = bload16(krs, (base + i * k_step) + k_boff);
#pragma unroll
      for (int i = 0; i < VU_PER_T; ++i)
        if (LV && (CF::V_UNITS % NT == 0 || tid + i * NT < CF::V_UNITS)) {
          sg.v[i][0] = bload16(vrs, base + v_boff + i * V_STEP);
          sg.v[i][1] = bload16(vrs, (base + st_bytes) + v_boff + i * V_STEP);
        }
      return;
    }
    // K: the keys one wave fetches in a round are 512 / C consecutive rows
    // of the tile, inside one page, so the wave reads the base of that page
    // (slot kj[i], fixed per wave) from page_lanes().  Keys past N_kv need no
    // zeros: their scores are masked before the softmax.  V: a thread's key
    // pair is the same in every round, so its bases are picked once per
    // tile; values past N_kv read as zeros.
    if constexpr (LK) {
      const int vb = page_lanes(pt);
#pragma unroll
      for (int i = 0; i < KC_PER_T; ++i)
        if (CF::K_CHUNKS % NT == 0 || tid + i * NT < CF::K_CHUNKS)
          sg.k[i] = bload16(krs, ((uint32_t)__builtin_amdgcn_readlane(vb, kj[i]) + i * k_step) + k_boff);
    }
    if constexpr (LV) {
      uint32_t b0, b1;
      v_pair_bases(pt, vj_hi, vj_lo, 2 * v_j, b0, b1);
      b0 += v_boff;
      b1 += v_boff + st_bytes;
#pragma unroll
      for (int i = 0; i < VU_PER_T; ++i)
        if (CF::V_UNITS % NT == 0 || tid + i * NT < CF::V_UNITS) {
          sg.v[i][0] = bload16(vrs, b0 + i * V_STEP);
          sg.v[i][1] = bload16(vrs, b1 + i * V_STEP);
        }
    }
  };
  auto load_part = [&](int kt, Staged& sg, auto part) INLINE {
    if constexpr (PAGED) load_part_pt(kt, paged_tile(kt), sg, part);
    else load_part_pt(kt, PageBases{}, sg, part);
  };
  const std::integral_constant<int, 1> K_PART;
  const std::integral_constant<int, 2> V_PART;
  const std::integral_constant<int, 3> KV_PARTS;
  auto load_tile = [&](int kt, Staged& sg) INLINE { load_part(kt, sg, KV_PARTS); };

  // One V unit (keys 2 v_j, 2 v_j + 1 x channels 8 ce .. 8 ce + 7) written
  // transposed into the V^T rows of stage stg.
  auto put_v = [&](bf16_t* stg, const uint4 (&u)[2], int ce) INLINE {
    const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&u[0]);
    const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&u[1]);
    bf16_t* col = stg + CF::K_ELEMS + 8 * ce * CF::VROW + vperm(2 * v_j);
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      // channels 8ce + 2e2 (low halves) and 8ce + 2e2 + 1 (high halves)
      const uint32_t lo = __builtin_amdgcn_perm(r1[e2], r0[e2], 0x05040100u);
      const uint32_t hi2 = __builtin_amdgcn_perm(r1[e2], r0[e2], 0x07060302u);
      *reinterpret_cast<uint32_t*>(col + (2 * e2) * CF::VROW) = lo;
      *reinterpret_cast<uint32_t*>(col + (2 * e2 + 1) * CF::VROW) = hi2;
    }
  };
  // The staging stores of one thread, as pieces that can be placed apart:
  // K chunk i, and V unit i (two keys x 8 channels, transposed on the way).
  auto store_k = [&](bf16_t* stg, const Staged& sg, int i) INLINE {
    if (CF::K_CHUNKS % NT == 0 || tid + i * NT < CF::K_CHUNKS)
      *reinterpret_cast<uint4*>(stg + k_row * CF::KROW + 8 * k_ce + i * K_ROW_STEP * CF::KROW) = sg.k[i];
  };
  auto store_v = [&](bf16_t* stg, const Staged& sg, int i) INLINE {
    if (CF::V_UNITS % NT == 0 || tid + i * NT < CF::V_UNITS) {
      put_v(stg, sg.v[i], v_ce + i * V_CE_STEP);
    }
  };
  auto store_tile = [&](bf16_t* stg, const Staged& sg) INLINE {
#pragma unroll
    for (int i = 0; i < KC_PER_T; ++i) store_k(stg, sg, i);
#pragma unroll
    for (int i = 0; i < VU_PER_T; ++i) store_v(stg, sg, i);
  };
  // ping-pong group staging: B fetches / stores K chunk i (i < KC_B), A V
  // unit i (i < VU_A)
  auto load_k_b = [&](int kt, const PageBases pt, Staged& sg) INLINE {
    if constexpr (PAGED) {
      const int vb = page_lanes(pt);
#pragma unroll
      for (int i = 0; i < KC_B; ++i)
        sg.k[i] = bload16(krs, ((uint32_t)__builtin_amdgcn_readlane(vb, kj_g[i]) + i * k_step_g) + k_boff_g);
    } else {
      const uint32_t base = (unsigned)kt < (unsigned)t_kv ? (uint32_t)kt * tile_bytes : 0x80000000u;
#pragma unroll
      for (int i = 0; i < KC_B; ++i) sg.k[i] = bload16(krs, (base + i * k_step_g) + k_boff_g);
    }
  };
  auto load_v_a = [&](int kt, const PageBases pt, Staged& sg) INLINE {
    uint32_t b0, b1;
    if constexpr (PAGED) {
      v_pair_bases(pt, vj_hi, vj_lo, 2 * v_j, b0, b1);
    } else {
      b0 = b1 = (unsigned)kt < (unsigned)t_kv ? (uint32_t)kt * tile_bytes : 0x80000000u;
    }
    b0 += v_boff_g;
    b1 += v_boff_g + st_bytes;
#pragma unroll
    for (int i = 0; i < VU_A; ++i) {
      sg.v[i][0] = bload16(vrs, b0 + i * V_STEP_G);
      sg.v[i][1] = bload16(vrs, b1 + i * V_STEP_G);
    }
  };
  auto store_k_b = [&](bf16_t* stg, const Staged& sg, int i) INLINE {
    *reinterpret_cast<uint4*>(stg + k_row_g * CF::KROW + 8 * k_ce_g + i * K_ROW_STEP_G * CF::KROW) = sg.k[i];
  };
  auto store_v_a = [&](bf16_t* stg, const Staged& sg, int i) INLINE {
    put_v(stg, sg.v[i], v_ce_g + i * V_CE_STEP_G);
  };

  // ---- online softmax state (one query per lane; both lane halves agree) ----
  const float c2 = a.scale * LOG2E;
  float m_run = -INFINITY;   // stale running max of the raw scores
  float l_run = 0.f;
  bool max_ok = false;       // every lane of the wave has a finite m_run
  f32x16 acc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[cb][r] = 0.f;

  // Staging by the waves alone on their SIMD (five and six waves): fetch /
  // store K chunk i (i < KC_S) and V unit i (i < VU_S) of their pattern
  auto load_s = [&](int kt, Staged& sg) INLINE {
    PageBases pt{};
    if constexpr (PAGED) pt = paged_tile(kt);
    uint32_t kbase[KC_S > 0 ? KC_S : 1];
    uint32_t b0, b1;
    if constexpr (PAGED) {
      const int vb = page_lanes(pt);
#pragma unroll
      for (int i = 0; i < KC_S; ++i) kbase[i] = (uint32_t)__builtin_amdgcn_readlane(vb, kj_s[i]);
      v_pair_bases(pt, vj_hi, vj_lo, 2 * v_j, b0, b1);
    } else {
      const uint32_t base = (unsigned)kt < (unsigned)t_kv ? (uint32_t)kt * tile_bytes : 0x80000000u;
#pragma unroll
      for (int i = 0; i < KC_S; ++i) kbase[i] = base;
      b0 = b1 = base;
    }
#pragma unroll
    for (int i = 0; i < KC_S; ++i)
      if (CF::K_CHUNKS % SNT == 0 || sidx + i * SNT < CF::K_CHUNKS)
        sg.k[i] = bload16(krs, (kbase[i] + i * k_step_s) + k_boff_s);
    b0 += v_boff_s;
    b1 += v_boff_s + st_bytes;
#pragma unroll
    for (int i = 0; i < VU_S; ++i)
      if (CF::V_UNITS % SNT == 0 || sidx + i * SNT < CF::V_UNITS) {
        sg.v[i][0] = bload16(vrs, b0 + i * V_STEP_S);
        sg.v[i][1] = bload16(vrs, b1 + i * V_STEP_S);
      }
  };
  auto store_k_s = [&](bf16_t* stg, const Staged& sg, int i) INLINE {
    if (CF::K_CHUNKS % SNT == 0 || sidx + i * SNT < CF::K_CHUNKS)
      *reinterpret_cast<uint4*>(stg + k_row_s * CF::KROW + 8 * k_ce_s + i * K_ROW_STEP_S * CF::KROW) = sg.k[i];
  };
  auto store_v_s = [&](bf16_t* stg, const Staged& sg, int i) INLINE {
    if (CF::V_UNITS % SNT == 0 || sidx + i * SNT < CF::V_UNITS) {
      put_v(stg, sg.v[i], v_ce_s + i * V_CE_STEP_S);
    }
  };
  // (the index is made explicitly uniform: inside the unrolled ping-pong loop
  // the compiler no longer proves it so and would emit a vector load)
  auto tile_at = [&](int i) INLINE -> int {
    return DENSE ? i : uniform_load(a.cols, __builtin_amdgcn_readfirstlane(list_begin + i));
  };
  auto stage = [&](int slot) INLINE -> bf16_t* { return lds + slot * CF::STAGE; };
  // List entry i, or -1 (a tile that loads zeros) past the end.  The list
  // read itself is unconditional (index clamped) so that it stays a scalar
  // load: a vector load would share vmcnt with the K/V prefetch.
  auto tile_or_none = [&](int i) INLINE -> int {
    // (through readfirstlane: a plain load feeding the select would be sunk
    // into a branch of its own)
    const int t = __builtin_amdgcn_readfirstlane(tile_at(min(i, n_tiles - 1)));
    return i < n_tiles ? t : -1;
  };
  // entries first .. first + N - 1, all read before the first is used (one
  // round trip instead of N)
  auto tiles_or_none = [&](int first, auto& kt) INLINE {
    constexpr int N = sizeof(kt) / sizeof(kt[0]);
#pragma unroll
    for (int j = 0; j < N; ++j)
      kt[j] = __builtin_amdgcn_readfirstlane(tile_at(min(first + j, n_tiles - 1)));
#pragma unroll
    for (int j = 0; j < N; ++j) kt[j] = first + j < n_tiles ? kt[j] : -1;
  };

  // ---- MFMA streams fed from LDS ----
  // S^T = K . Q^T (two 32-key blocks, Q held in registers) and
  // O^T += V^T . P^T (channel block fastest, so consecutive MFMAs accumulate
  // into different registers).  One stream runs the PV product of one tile
  // and/or the QK product of another.  Its operand fragments are read
  // DEPTH ahead in exactly the order the MFMAs consume them, with the waits
  // placed by hand: left to the scheduler, the reads of a ring get reordered
  // and every few MFMAs wait on a read issued just before them.
  constexpr int DEPTH = 4;
  const uint32_t lds_base = LDS_ADDR(lds);
  const uint32_t k_lane = lds_base + (uint32_t)((l32 * CF::KROW + 8 * hi) * 2);
  const uint32_t v_lane = lds_base + (uint32_t)((CF::K_ELEMS + l32 * CF::VROW + 8 * hi) * 2);
  f32x16 s0, s1;
  bf16x8 pf[4];   // P^T of the tile being multiplied by V
  auto no_hook = [](auto) INLINE {};
  // hook(step) runs after the read of each step: other work placed between
  // the MFMAs of the stream
  auto stream = [&](auto do_pv, auto do_qk, int v_slot, int k_slot, auto&& hook) INLINE {
    constexpr int NV = decltype(do_pv)::value ? 4 * NCB : 0;   // V^T fragments
    constexpr int NK = decltype(do_qk)::value ? 2 * NKC : 0;   // K fragments
    constexpr int N = NV + NK;
    const uint32_t va = v_lane + (uint32_t)(v_slot * CF::STAGE * 2);
    const uint32_t ka = k_lane + (uint32_t)(k_slot * CF::STAGE * 2);
    u32x4 ring[DEPTH];
    // fragment j < NV: V^T rows 32 (j % NCB).., keys 16 (j / NCB)..;
    // else j' = j - NV: K rows 32 (j' % 2).., channels 16 (j' / 2)..
    auto issue = [&](auto jc) INLINE {
      constexpr int j = decltype(jc)::value;
      if constexpr (j < NV)
        lds_read<(32 * (j % NCB) * CF::VROW + 16 * (j / NCB)) * 2>(ring[j % DEPTH], va);
      else
        lds_read<(((j - NV) & 1) * 32 * CF::KROW + 16 * ((j - NV) >> 1)) * 2>(ring[j % DEPTH], ka);
    };
    static_for<(DEPTH < N ? DEPTH : N)>(issue);
    const f32x16 zero = {};
    static_for<N>([&](auto jc) {
      constexpr int j = decltype(jc)::value;
      // reads issued after fragment j so far: min(N, DEPTH + j) - j - 1
      lgkm_wait<(N - 1 - j < DEPTH - 1 ? N - 1 - j : DEPTH - 1)>(ring[j % DEPTH]);
      const bf16x8 a = __builtin_bit_cast(bf16x8, ring[j % DEPTH]);
      if constexpr (j < NV) {
        acc[j % NCB] = mfma32(a, pf[j / NCB], acc[j % NCB]);
      } else if constexpr (((j - NV) & 1) != 0) {
        s1 = mfma32(a, qf[(j - NV) >> 1], j - NV < 2 ? zero : s1);   // S starts at 0
      } else {
        s0 = mfma32(a, qf[(j - NV) >> 1], j - NV < 2 ? zero : s0);
      }
      if constexpr (j + DEPTH < N) issue(std::integral_constant<int, j + DEPTH>{});
      hook(jc);
      // keep every MFMA between its own wait and the next read (the 2-stage
      // shapes stage whole tiles through registers and need the scheduler's
      // freedom to fit them)
      if constexpr (PP) __builtin_amdgcn_sched_barrier(0);
    });
  };
  const std::true_type YES;
  const std::false_type NO;

  // online softmax of the scores of KV tile kt -> bf16 P^T operands
  // P = exp2(S c2 + moff) as bf16 B operands (16-key chunk q = regs 8(q%2)..
  // of block q/2); returns this lane's fp32 sum of the weights.
  auto exp_pack = [&](float moff) INLINE -> float {
    float r0 = 0.f, r1 = 0.f;
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const f32x16& sb = (qq < 2) ? s0 : s1;
      const int base = 8 * (qq & 1);
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(sb[base + 2 * e], c2, moff));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(sb[base + 2 * e + 1], c2, moff));
        w[e] = pack_bf16x2(p0, p1);
        r0 += p0;
        r1 += p1;
      }
      pf[qq] = as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
    }
    return r0 + r1;
  };
  auto softmax = [&](int kt_s) INLINE {
    // token-level causal mask and key bound, only on tiles that need it; a
    // list entry outside [0, T_kv) contributes nothing
    const int key0 = kt_s * TILE;
    if ((unsigned)kt_s >= (unsigned)t_kv || key0 + TILE - 1 > wave_q0 || key0 + TILE > n_kv) {
      const int lim = ((unsigned)kt_s >= (unsigned)t_kv ? -1 : key_lim) - key0 - 4 * hi;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kk = 8 * (r >> 2) + (r & 3);
        s0[r] = kk <= lim ? s0[r] : -INFINITY;
        s1[r] = kk + 32 <= lim ? s1[r] : -INFINITY;
      }
    }
    // Common case: weights against the stale max, accepted when the row's
    // weight sum for this tile stays <= 2^RESCALE_LOG2 (so does every weight).
    bool done = false;
    float rs = 0.f;
    if (max_ok) {
      rs = add_lane32(exp_pack(-m_run * c2));
      done = !__builtin_amdgcn_ballot_w64(!(rs <= RESCALE_SUM));
    }
    if (!done) {
      // row max over this lane's 32 keys: a chain of 3-input max
      float mx = fmaxf(s0[0], s1[0]);
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(fmaxf(mx, s0[r]), s1[r]);
      mx = max_lane32(mx);
      const bool grow = mx > m_run;
      if (__builtin_amdgcn_ballot_w64(grow)) {
        const float m_new = grow ? mx : m_run;
        const float corr = grow ? __builtin_amdgcn_exp2f((m_run - m_new) * c2) : 1.f;
        m_run = m_new;
        l_run *= corr;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[cb][r] *= corr;
      }
      max_ok = !__builtin_amdgcn_ballot_w64(m_run == -INFINITY);
      rs = add_lane32(exp_pack((m_run == -INFINITY) ? 0.f : -m_run * c2));
    }
    l_run += rs;
  };

  if (PP) {
    // Ping-pong over 3 LDS stages.  Group A (waves 0-3 of every 8) runs half
    // an iteration ahead of group B (waves 4-7); each SIMD hosts one wave of
    // each group, so in every phase one of them issues MFMAs while the other
    // runs the softmax.  Tile i lives in stage i % 3.
    //   phase Y_i:   A PV(i), QK(i+1)      | B softmax(i)
    //   phase X_i+1: A softmax(i+1)        | B PV(i), QK(i+1); both store
    //                their part of tile i+2
    // Stage (i+2) % 3 == (i-1) % 3 is last read by B in phase X_i.  Each
    // group runs one PV+QK stream per iteration; the QK of the last one reads
    // a stage no one writes any more and its scores are never used.
    //   Tile i + 4 is fetched into registers in phase X_i+1 and stored in
    // X_i+3: two register sets, the loop unrolled by two so each is fixed.
    // Past the end of the list the loads read zeros (no memory traffic) and
    // the stores fill a stage no one reads, so the loop body has no branches
    // around its memory operations.
    if (n_tiles <= 0) q_from_lds();
    if (n_tiles > 0) {
      Staged sg0, sg1;
      int kt[5];  // tiles i .. i+4
      tiles_or_none(0, kt);
      PageBases pt4{};
      // Each group runs its own copy of the prologue and the loop (same
      // barriers in the same order), so that the compiler sees one group's
      // loads and stores as straight-line code and waits for exactly the
      // older register set.
      auto run = [&](auto is_a) INLINE {
        constexpr bool A = decltype(is_a)::value;
        auto pp_load = [&](int t, Staged& sg) INLINE {
          PageBases pt{};
          if constexpr (PAGED) pt = paged_tile(t);
          if constexpr (A) load_v_a(t, pt, sg);
          else load_k_b(t, pt, sg);
        };
        auto pp_store = [&](bf16_t* stg, const Staged& sg) INLINE {
          if constexpr (A) {
#pragma unroll
            for (int i = 0; i < VU_A; ++i) store_v_a(stg, sg, i);
          } else {
#pragma unroll
            for (int i = 0; i < KC_B; ++i) store_k_b(stg, sg, i);
          }
        };
        pp_load(kt[0], sg0);
        pp_load(kt[1], sg1);
        q_from_lds();
        pp_store(stage(0), sg0);
        pp_store(stage(1), sg1);
        pp_load(kt[2], sg0);
        pp_load(kt[3], sg1);
        // the page bases of tile i + 4, read outside the MFMA streams
        if constexpr (PAGED) pt4 = paged_tile(kt[4]);
        __syncthreads();
        // phase X_0 (A starts half an iteration ahead with QK(0))
        if (A) stream(NO, YES, 0, 0, no_hook);
        __syncthreads();
        if (A) softmax(kt[0]);
        else stream(NO, YES, 0, 0, no_hook);
        __syncthreads();
        int slot = 0;  // i % 3
        int it = 0;
        // one iteration: phases Y_i and X_i+1, staging through sg
        auto iteration = [&](Staged& sg) INLINE {
          const int slot1 = slot == 2 ? 0 : slot + 1;   // (i + 1) % 3
          const int slot2 = slot1 == 2 ? 0 : slot1 + 1; // (i + 2) % 3 == (i - 1) % 3
          bf16_t* const dst = stage(slot2);
          const int kt_load = kt[4];
          // Each group stages its part of tile i + 2 (into the stage no one
          // reads in either phase) and fetches that part of tile i + 4: B the
          // K chunks, between the MFMAs of its stream, where its LDS and
          // memory ports are otherwise idle; A the V units (transposed on the
          // way, VALU work) in its softmax phase.  B's waves are the younger
          // ones and lose the issue arbitration, so its phases run longer:
          // leaving it no VALU staging balances them (each group staging half
          // of both parts was 2.4-3.2 % slower).
          auto stage_hook = [&](auto jc) INLINE {
            constexpr int j = decltype(jc)::value;
            constexpr int K0 = 2, L0 = K0 + 2 * KC_B;
            if constexpr (!A) {
              if constexpr (j >= K0 && j < L0 && (j - K0) % 2 == 0) store_k_b(dst, sg, (j - K0) / 2);
              if constexpr (j == L0) load_k_b(kt_load, pt4, sg);
            }
          };
          auto softmax_v = [&](int kt_s) INLINE {
            if constexpr (A) {
#pragma unroll
              for (int u = 0; u < VU_A; ++u) store_v_a(dst, sg, u);
              load_v_a(kt_load, pt4, sg);
            }
            softmax(kt_s);
          };
          // phase Y_i: A streams PV(i), QK(i+1); B takes the softmax of tile i
          if (A) stream(YES, YES, slot, slot1, stage_hook);
          else softmax_v(kt[0]);
          __syncthreads();
          // phase X_i+1: B streams PV(i), QK(i+1); A the softmax of tile i+1
          if (!A) {
            stream(YES, YES, slot, slot1, stage_hook);
          } else {
#pragma unroll
            for (int u = 0; u < VU_A; ++u) store_v_a(dst, sg, u);
            load_v_a(kt_load, pt4, sg);
            if (it + 1 < n_tiles) softmax(kt[1]);
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) kt[j] = kt[j + 1];
          kt[4] = tile_or_none(it + 5);
          if constexpr (PAGED) pt4 = paged_tile(kt[4]);
          slot = slot1;
          __syncthreads();
        };
        for (; it + 1 < n_tiles; it += 2) {
          iteration(sg0);
          ++it;
          iteration(sg1);
          --it;
        }
        if (it < n_tiles) iteration(sg0);
      };
      // group A = waves 0-3, B = waves 4-7 (one wave of each per SIMD)
      if (__builtin_amdgcn_readfirstlane(wave) < 4) run(YES);
      else run(NO);
    }
  } else {
    // Two LDS stages, every wave in the same phase.  Tile i + 1 (fetched into
    // registers during iteration i - 1) is stored into the free stage, and
    // tile i + 2 fetched, between the MFMAs of the PV stream of iteration i,
    // where the wave's VALU and LDS ports are otherwise idle.  Past the end of
    // the list the loads read zeros and the stores fill the unused stage.
    if (n_tiles <= 0) q_from_lds();
    if (n_tiles > 0) {
      Staged sg;
      int kt01[2];   // list entries 0 and 1
      tiles_or_none(0, kt01);
      if constexpr (SOLO) {
        Staged sg1;
        if (stager) {
          load_s(kt01[0], sg);
          load_s(kt01[1], sg1);
        }
        q_from_lds();
        if (stager) {
#pragma unroll
          for (int i = 0; i < KC_S; ++i) store_k_s(stage(0), sg, i);
#pragma unroll
          for (int i = 0; i < VU_S; ++i) store_v_s(stage(0), sg, i);
        }
        sg = sg1;
      } else if constexpr (HALF) {
        // half-tile shapes (GQA 6-8): tile 1 joins the same round trip
        // (measured faster there, slower for the 2-wave GQA 1 shape)
        Staged sg1;
        load_tile(kt01[0], sg);
        load_tile(kt01[1], sg1);
        q_from_lds();
        store_tile(stage(0), sg);
        sg = sg1;
      } else {
        load_tile(kt01[0], sg);
        q_from_lds();   // overlaps the first tile's round trip
        store_tile(stage(0), sg);
        load_tile(kt01[1], sg);
      }
      __syncthreads();
      // tiles it and it + 1; each entry is read once, as the fetch of
      // iteration it - 2 (entry it) and carried
      int kt_cur = kt01[0], kt_next = kt01[1];
      for (int it = 0; it < n_tiles; ++it) {
        bf16_t* const dst = stage((it + 1) & 1);
        const int kt_load = tile_or_none(it + 2);
        auto stage_hook = [&](auto jc) INLINE {
          constexpr int j = decltype(jc)::value;
          if constexpr (SOLO) {
            constexpr int K0 = 1, V0 = K0 + KC_S, L0 = V0 + VU_S;
            static_assert(L0 < 4 * NCB, "staging pieces must fit the PV stream");
            if constexpr (j >= K0 && j < V0) { if (stager) store_k_s(dst, sg, j - K0); }
            if constexpr (j >= V0 && j < L0) { if (stager) store_v_s(dst, sg, j - V0); }
            if constexpr (j == L0) { if (stager) load_s(kt_load, sg); }
          } else {
            constexpr int K0 = 1, V0 = K0 + KC_PER_T, L0 = V0 + VU_PER_T;
            static_assert(L0 < 4 * NCB, "staging pieces must fit the PV stream");
            if constexpr (j >= K0 && j < V0) store_k(dst, sg, j - K0);
            if constexpr (j >= V0 && j < L0) store_v(dst, sg, j - V0);
            if constexpr (j == L0) load_tile(kt_load, sg);
          }
        };
        stream(NO, YES, 0, it & 1, no_hook);
        softmax(kt_cur);
        stream(YES, NO, it & 1, 0, stage_hook);
        kt_cur = kt_next;
        kt_next = kt_load;
        __syncthreads();
      }
    }
  }

  // ---- epilogue: O = O^T / l, LSE ----
  // A lane holds 4-channel pieces of one query row, so storing the O^T
  // accumulators directly makes every store touch 32 rows.  Each wave
  // instead writes its 32 x C block into LDS (the K/V stages are free once
  // every wave has left the tile loop) and stores whole rows from there,
  // 16 bytes per lane and C / 8 lanes per row.  A wave reads back only its
  // own rows, which its LDS stores precede in order.
  constexpr int OROW = C + 8;                    // bf16 row pitch of the staged block
  constexpr int LDS_BYTES = (PP ? 3 : 2) * CF::STAGE * 2;
  static_assert(Shape<C, M>::WAVES * 32 * OROW * 2 <= LDS_BYTES, "O staging exceeds the LDS");
  const float inv = (l_run > 0.f) ? 1.f / l_run : 0.f;
  __syncthreads();
  bf16_t* const ow = lds + wave * 32 * OROW;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      uint2 u;
      u.x = pack_bf16x2(acc[cb][4 * rg + 0] * inv, acc[cb][4 * rg + 1] * inv);
      u.y = pack_bf16x2(acc[cb][4 * rg + 2] * inv, acc[cb][4 * rg + 3] * inv);
      *reinterpret_cast<uint2*>(ow + l32 * OROW + 32 * cb + 8 * rg + 4 * hi) = u;
    }
  }
  {
    constexpr int LPR = C / 8, RPI = 64 / LPR;   // lanes per row, rows per store
    const int r0 = lane / LPR, ch = 8 * (lane % LPR);
    const int t0 = qt * TILE + half * 32;
    bf16_t* const ob = a.o + o_off + (int64_t)p * a.o_sh;
#pragma unroll
    for (int i = 0; i < 32 / RPI; ++i) {
      const int r = r0 + RPI * i;
      const uint4 u = *reinterpret_cast<const uint4*>(ow + r * OROW + ch);
      if (t0 + r < n_q) *reinterpret_cast<uint4*>(ob + (int64_t)(t0 + r) * a.o_st + ch) = u;
    }
  }
  if (a.lse && hi == 0 && q_ok) {
    float v = (l_run > 0.f) ? m_run * a.scale + logf(l_run) : -INFINITY;
    a.lse[lse_off + (int64_t)p * n_q + t] = v;
  }
}

template <bool PAGED>
struct KvTiles {
  int t_kv, n_kv;
  uint32_t tile_bytes;     // contiguous: bytes per 64-key tile
  const int32_t* bt;       // paged: this request's block-table row
  int ps_shift;
  uint32_t n_pages, page_bytes, tok_bytes;
  int64_t st;              // elements per token

  // Contiguous: b0 is the tile's first byte (2^31 for a tile outside
  // [0, T_kv), so its loads read zeros).  Paged: page_bases().
  __device__ __forceinline__ PageBases locate(int kt) const {
    if (PAGED) return page_bases(bt, kt, t_kv, n_kv, ps_shift, n_pages, page_bytes, tok_bytes);
    PageBases pb{};
    pb.b0 = (unsigned)kt < (unsigned)t_kv ? (uint32_t)kt * tile_bytes : 0x80000000u;
    return pb;
  }
};
template <int C, bool PAGED>
__device__ __forceinline__ KvTiles<PAGED> kv_tiles(const PrefillArgs& a, const ReqDesc& Rd, int h,
                                                   __amdgpu_buffer_rsrc_t& krs,
                                                   __amdgpu_buffer_rsrc_t& vrs) {
  KvTiles<PAGED> kt;
  kt.t_kv = Rd.t_kv;
  kt.n_kv = Rd.n_kv;
  kt.st = a.kv.stride_tok;
  kt.tile_bytes = (uint32_t)(TILE * kt.st * 2);
  if (!PAGED) {
    const int64_t head_off = Rd.kv_off + (int64_t)h * a.kv.stride_head;
    const uint32_t bytes = (uint32_t)(((int64_t)(Rd.n_kv - 1) * kt.st + C) * 2);
    krs = make_rsrc(a.kv.k + head_off, bytes);
    vrs = make_rsrc(a.kv.v + head_off, bytes);
    kt.bt = nullptr;
    kt.ps_shift = 0;
    kt.n_pages = kt.page_bytes = kt.tok_bytes = 0;
  } else {
    const int64_t head_off = (int64_t)h * a.kv.stride_head;
    krs = make_rsrc(a.kv.k + head_off, a.kv.pool_bytes);
    vrs = make_rsrc(a.kv.v + head_off, a.kv.pool_bytes);
    kt.bt = a.kv.block_table + (int64_t)Rd.bt_row * a.kv.max_pages;
    kt.ps_shift = __builtin_ctz(a.kv.page_size);   // power of two >= 16
    kt.n_pages = (uint32_t)a.kv.n_pages;
    kt.page_bytes = (uint32_t)(a.kv.page_stride * 2);
    kt.tok_bytes = (uint32_t)(kt.st * 2);
  }
  return kt;
}

// ---- head dim 256: 16-query waves on v_mfma_f32_16x16x32_bf16 ----
__device__ __forceinline__ f32x4 mfma16x16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x2 lane16_pair(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, x),
                                                  __builtin_bit_cast(uint32_t, x), false, false);
  return f32x2{__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1])};
}
__device__ __forceinline__ float max_lane4(float x) {
  const f32x2 p = lane32_pair(x);
  const f32x2 q = lane16_pair(fmaxf(p[0], p[1]));
  return fmaxf(q[0], q[1]);
}
__device__ __forceinline__ float add_lane4(float x) {
  const f32x2 p = lane32_pair(x);
  const f32x2 q = lane16_pair(p[0] + p[1]);
  return q[0] + q[1];
}
// key 32 c + 16 h + 4 g + r of a tile sits at 32 c + 8 g + 4 h + r of a V^T
// row: the k order of the 16x16x32 B operand built from the S layout
__device__ __forceinline__ int vperm16(int k) {
  return (k & 32) | (((k >> 2) & 3) << 3) | (((k >> 4) & 1) << 2) | (k & 3);
}

// A work item holds QB 16-query blocks (q16_blocks) of one q-tile for all m
// heads of the GQA group: wave w owns head w / QB and block w % QB.  With
// 32-query waves these shapes need one wave per SIMD at 512 VGPRs (and spill
// at m = 1 and m > 2); 16-query waves halve O, Q and S per wave.  K and V
// live in separate two-slot rings offset by one tile (three combined stages
// of 256 channels, 212 KiB, would not fit the LDS; the rings take 141 KiB).
//
// GQA 2 (eight waves): the ping-pong, group A = head 0 (waves 0-3), group
// B = head 1 (waves 4-7), one wave of each per SIMD.  In the phases of
// iteration i the streams read K(i+1) and V(i), while K(i+2) and V(i+1) are
// staged into the other slots.
// Other group sizes: all waves run the same phase, one barrier per tile.
// Iteration i streams PV(i - 1) and QK(i) and takes the softmax of tile i;
// between the MFMAs each thread stores its chunks of K(i + 1) and V(i) and
// then fetches those of K(i + 2) and V(i + 1).
template <int C, int M, bool DENSE, bool PAGED>
__global__ void __launch_bounds__(64 * M * q16_blocks(M)) prefill_q16_kernel(PrefillArgs a) {
  constexpr int QB = q16_blocks(M), PARTS = 4 / QB;
  constexpr int NW = M * QB, NT = 64 * NW;
  // GQA 2: ping-pong between the two heads' waves (one of each per SIMD)
  constexpr bool PP = M == 2;
  // Five waves, list-driven: a thread stages 7 K chunks and 4 V units of a
  // tile (60 VGPRs).  Held together across the softmax they push the sparse
  // kernel past 256 VGPRs (65 spilled), so the two sets take turns: V(i) is
  // fetched at the end of iteration i - 1 and stored halfway through the QK
  // MFMAs of iteration i, K(i + 1) is fetched right after those stores and
  // stored after the softmax of iteration i.  The dense kernel fits with
  // both sets held and keeps the common schedule.
  constexpr bool ALT = !PP && !DENSE && M * q16_blocks(M) == 5;
  constexpr int KROW = C + 8, VROW = TILE + 8;
  constexpr int K_SLOT = TILE * KROW, V_SLOT = C * VROW;
  constexpr int K_CHUNKS = TILE * C / 8, V_UNITS = (TILE / 2) * (C / 8);
  constexpr int KC_PER_T = (K_CHUNKS + NT - 1) / NT;
  constexpr int VU_PER_T = (V_UNITS + NT - 1) / NT;
  constexpr int NKC = C / 32, NCB = C / 16;
  extern __shared__ __align__(16) bf16_t lds[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l16 = lane & 15;
  const int g = lane >> 4;

  const int w = blockIdx.x;
  const int ri = find_req(a.batch, w);
  const ReqDesc& Rd = a.batch.r[ri];
  const int n_q = Rd.n_q, n_kv = Rd.n_kv, t_q = Rd.t_q, t_kv = Rd.t_kv;
  const int64_t q_off = Rd.q_off, o_off = Rd.o_off, lse_off = Rd.lse_off;
  const int local = w - Rd.work_begin;
  const int h = local % a.h_kv;
  const int rank = local / a.h_kv;
  const int qt = t_q - 1 - rank / PARTS;
  const int row = Rd.row_base + h * t_q + qt;
  const int n_c = n_kv - n_q;
  int list_begin = 0, n_tiles;
  if (DENSE) {
    n_tiles = min(n_c + (qt + 1) * TILE - 1, n_kv - 1) / TILE + 1;
  } else {
    list_begin = uniform_load(a.row_ptr, row);
    n_tiles = uniform_load(a.row_ptr, row + 1) - list_begin;
  }
  const int p = h * M + wave / QB;
  const int q16 = qt * TILE + (rank % PARTS) * 16 * QB + (wave % QB) * 16;  // the wave's first query
  const int t = q16 + l16;                                         // this lane's query
  const int wave_q0 = n_c + q16;

  bf16x8 qf[NKC];
  {
    // queries past N_q (never stored) repeat the last one: no branch
    const bf16_t* qp = a.q + q_off + (int64_t)p * a.q_sh + (int64_t)min(t, n_q - 1) * a.q_st + 8 * g;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) qf[kc] = as_bf16x8(ld16(qp + 32 * kc));
  }
  __builtin_amdgcn_s_waitcnt(VMCNT0);

  __amdgpu_buffer_rsrc_t krs, vrs;
  const KvTiles<PAGED> kvt = kv_tiles<C, PAGED>(a, Rd, h, krs, vrs);
  const int64_t st = a.kv.stride_tok;
  // staging pattern as in prefill_kernel: round i moves a thread's K row by
  // i K_ROW_STEP and its V channel group by i V_CE_STEP
  constexpr int K_ROW_STEP = NT / (C / 8), V_CE_STEP = NT / (TILE / 2);
  static_assert(NT % (C / 8) == 0 && NT % (TILE / 2) == 0, "rounds must keep a thread's column");
  const int k_row = tid / (C / 8), k_ce = tid % (C / 8);
  const uint32_t k_boff = (uint32_t)(((int64_t)k_row * st + 8 * k_ce) * 2);
  const uint32_t k_step = (uint32_t)(K_ROW_STEP * st * 2);
  const int v_j = tid % (TILE / 2), v_ce = tid / (TILE / 2);
  const uint32_t v_boff = (uint32_t)(((int64_t)(2 * v_j) * st + 8 * v_ce) * 2);
  constexpr uint32_t V_STEP = V_CE_STEP * 8 * 2;
  auto k_mine = [&](int i) INLINE { return K_CHUNKS % NT == 0 || tid + i * NT < K_CHUNKS; };
  auto v_mine = [&](int i) INLINE { return V_UNITS % NT == 0 || tid + i * NT < V_UNITS; };
  const uint32_t st_bytes = (uint32_t)(st * 2);
  struct KSet { uint4 k[KC_PER_T]; };
  struct VSet { uint4 v[VU_PER_T][2]; };
  // Paged: the page slot (0-3) of this wave's K rows in round i (two
  // consecutive rows, inside one page) and of this thread's V key pair.
  int kj[KC_PER_T];
  bool vj_hi = false, vj_lo = false;
  if constexpr (PAGED) {
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const bool paged_slots = kvt.ps_shift < 6;   // pages shorter than a tile
#pragma unroll
    for (int i = 0; i < KC_PER_T; ++i)
      kj[i] = paged_slots ? ((wave_u * 64 + i * NT) / (C / 8)) >> kvt.ps_shift : 0;
    const int v_slot = paged_slots ? (2 * v_j) >> kvt.ps_shift : 0;
    vj_hi = (v_slot & 2) != 0;
    vj_lo = (v_slot & 1) != 0;
  }
  auto locate = [&](int kt) INLINE -> PageBases { return kvt.locate(kt); };
  auto load_k_at = [&](const PageBases at, KSet& sk) INLINE {
    if constexpr (PAGED) {
      const int vb = page_lanes(at);
#pragma unroll
      for (int i = 0; i < KC_PER_T; ++i)
        if (k_mine(i))
          sk.k[i] = bload16(krs, ((uint32_t)__builtin_amdgcn_readlane(vb, kj[i]) + i * k_step) + k_boff);
    } else {
#pragma unroll
      for (int i = 0; i < KC_PER_T; ++i)
        if (k_mine(i)) sk.k[i] = bload16(krs, (at.b0 + i * k_step) + k_boff);
    }
  };
  auto load_v_at = [&](const PageBases at, VSet& sv) INLINE {
    uint32_t b0 = at.b0, b1 = at.b0;
    if constexpr (PAGED) v_pair_bases(at, vj_hi, vj_lo, 2 * v_j, b0, b1);
    b0 += v_boff;
    b1 += v_boff + st_bytes;
#pragma unroll
    for (int i = 0; i < VU_PER_T; ++i)
      if (v_mine(i)) {
        sv.v[i][0] = bload16(vrs, b0 + i * V_STEP);
        sv.v[i][1] = bload16(vrs, b1 + i * V_STEP);
      }
  };
  auto load_k = [&](int kt, KSet& sk) INLINE { load_k_at(kvt.locate(kt), sk); };
  auto load_v = [&](int kt, VSet& sv) INLINE { load_v_at(kvt.locate(kt), sv); };
  bf16_t* const kring = lds;                  // [2][K_SLOT]
  bf16_t* const vring = lds + 2 * K_SLOT;     // [2][V_SLOT]
  auto store_k = [&](int slot, const KSet& sk, int i) INLINE {
    if (k_mine(i))
      *reinterpret_cast<uint4*>(kring + slot * K_SLOT + k_row * KROW + 8 * k_ce + i * K_ROW_STEP * KROW) = sk.k[i];
  };
  auto store_v = [&](int slot, const VSet& sv, int i) INLINE {
    if (!v_mine(i)) return;
    const int pos = vperm16(2 * v_j);
    const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&sv.v[i][0]);
    const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&sv.v[i][1]);
    bf16_t* col = vring + slot * V_SLOT + 8 * v_ce * VROW + pos + i * 8 * V_CE_STEP * VROW;
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const uint32_t lo = __builtin_amdgcn_perm(r1[e2], r0[e2], 0x05040100u);
      const uint32_t hi2 = __builtin_amdgcn_perm(r1[e2], r0[e2], 0x07060302u);
      *reinterpret_cast<uint32_t*>(col + (2 * e2) * VROW) = lo;
      *reinterpret_cast<uint32_t*>(col + (2 * e2 + 1) * VROW) = hi2;
    }
  };
  auto tile_or_none = [&](int i) INLINE -> int {
    if (DENSE) return i < n_tiles ? i : -1;
    const int tt = __builtin_amdgcn_readfirstlane(
        uniform_load(a.cols, __builtin_amdgcn_readfirstlane(list_begin + min(i, n_tiles - 1))));
    return i < n_tiles ? tt : -1;
  };
  // entries 0 .. N - 1, all read before the first is used
  auto first_tiles = [&](auto& kt) INLINE {
    constexpr int N = sizeof(kt) / sizeof(kt[0]);
#pragma unroll
    for (int j = 0; j < N; ++j)
      kt[j] = DENSE ? j : __builtin_amdgcn_readfirstlane(uniform_load(
                              a.cols, __builtin_amdgcn_readfirstlane(list_begin + min(j, n_tiles - 1))));
#pragma unroll
    for (int j = 0; j < N; ++j) kt[j] = j < n_tiles ? kt[j] : -1;
  };

  const float c2 = a.scale * LOG2E;
  float m_run = -INFINITY, l_run = 0.f;
  bool max_ok = false;
  f32x4 acc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 sc[4];     // keys 16 kb + 4 g + r of the tile, this lane's query
  bf16x8 pf[2];    // P^T B operands, 32-key chunks

  constexpr int DEPTH = 4;
  const uint32_t lds_base = LDS_ADDR(lds);
  const uint32_t k_lane = lds_base + (uint32_t)((l16 * KROW + 8 * g) * 2);
  const uint32_t v_lane = lds_base + (uint32_t)((2 * K_SLOT + l16 * VROW + 8 * g) * 2);
  // PV of the tile in V slot v_slot (P in pf) and/or QK of the tile in K slot
  // k_slot (S into sc); one LDS fragment per MFMA, read DEPTH ahead
  auto stream = [&](auto do_pv, auto do_qk, int v_slot, int k_slot, auto&& hook) INLINE {
    constexpr int NV = decltype(do_pv)::value ? 2 * NCB : 0;   // (cb, 32-key chunk)
    constexpr int NK = decltype(do_qk)::value ? 4 * NKC : 0;   // (kb, 32-channel chunk)
    constexpr int N = NV + NK;
    const uint32_t va = v_lane + (uint32_t)(v_slot * V_SLOT * 2);
    const uint32_t ka = k_lane + (uint32_t)(k_slot * K_SLOT * 2);
    u32x4 ring[DEPTH];
    auto issue = [&](auto jc) INLINE {
      constexpr int j = decltype(jc)::value;
      if constexpr (j < NV)
        lds_read<(16 * (j % NCB) * VROW + 32 * (j / NCB)) * 2>(ring[j % DEPTH], va);
      else
        lds_read<(16 * ((j - NV) & 3) * KROW + 32 * ((j - NV) >> 2)) * 2>(ring[j % DEPTH], ka);
    };
    static_for<(DEPTH < N ? DEPTH : N)>(issue);
    const f32x4 zero = {};
    static_for<N>([&](auto jc) INLINE {
      constexpr int j = decltype(jc)::value;
      lgkm_wait<(N - 1 - j < DEPTH - 1 ? N - 1 - j : DEPTH - 1)>(ring[j % DEPTH]);
      const bf16x8 av = __builtin_bit_cast(bf16x8, ring[j % DEPTH]);
      if constexpr (j < NV) {
        acc[j % NCB] = mfma16x16(av, pf[j / NCB], acc[j % NCB]);
      } else {
        constexpr int kb = (j - NV) & 3;
        sc[kb] = mfma16x16(av, qf[(j - NV) >> 2], (j - NV) < 4 ? zero : sc[kb]);
      }
      if constexpr (j + DEPTH < N) issue(std::integral_constant<int, j + DEPTH>{});
      hook(jc);
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  const std::true_type YES;
  const std::false_type NO;
  auto no_hook = [](auto) INLINE {};

  auto exp_pack = [&](float moff) INLINE -> float {
    float r0 = 0.f, r1 = 0.f;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      uint32_t wd[4];
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        const f32x4& v = sc[2 * c + hb];
        const float p0 = __builtin_amdgcn_exp2f(fmaf(v[0], c2, moff));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(v[1], c2, moff));
        const float p2 = __builtin_amdgcn_exp2f(fmaf(v[2], c2, moff));
        const float p3 = __builtin_amdgcn_exp2f(fmaf(v[3], c2, moff));
        wd[2 * hb] = pack_bf16x2(p0, p1);
        wd[2 * hb + 1] = pack_bf16x2(p2, p3);
        r0 += p0;
        r1 += p1;
        r0 += p2;
        r1 += p3;
      }
      pf[c] = as_bf16x8(make_uint4(wd[0], wd[1], wd[2], wd[3]));
    }
    return r0 + r1;
  };
  auto softmax = [&](int kt_s) INLINE {
    const int key0 = kt_s * TILE;
    if ((unsigned)kt_s >= (unsigned)t_kv || key0 + TILE - 1 > wave_q0 || key0 + TILE > n_kv) {
      const int lim = ((unsigned)kt_s >= (unsigned)t_kv ? -1 : min(n_c + t, n_kv - 1)) - key0 - 4 * g;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) sc[kb][r] = 16 * kb + r <= lim ? sc[kb][r] : -INFINITY;
    }
    bool done = false;
    float rs = 0.f;
    if (max_ok) {
      rs = add_lane4(exp_pack(-m_run * c2));
      done = !__builtin_amdgcn_ballot_w64(!(rs <= RESCALE_SUM));
    }
    if (!done) {
      float x = sc[0][0];
#pragma unroll
      for (int i = 1; i < 16; ++i) x = fmaxf(x, sc[i / 4][i % 4]);
      const float mx = max_lane4(x);
      const bool grow = mx > m_run;
      if (__builtin_amdgcn_ballot_w64(grow)) {
        const float m_new = grow ? mx : m_run;
        const float corr = grow ? __builtin_amdgcn_exp2f((m_run - m_new) * c2) : 1.f;
        m_run = m_new;
        l_run *= corr;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[cb][r] *= corr;
      }
      max_ok = !__builtin_amdgcn_ballot_w64(m_run == -INFINITY);
      rs = add_lane4(exp_pack((m_run == -INFINITY) ? 0.f : -m_run * c2));
    }
    l_run += rs;
  };

  if constexpr (PP) {
    if (n_tiles > 0) {
      // sk holds the K part of tile i + 2, sv the V part of tile i + 1
      KSet sk;
      VSet sv;
      int kt[5];   // tiles i .. i + 4
      first_tiles(kt);
      load_k(kt[0], sk);
      load_v(kt[0], sv);
  #pragma unroll
      for (int i = 0; i < KC_PER_T; ++i) store_k(0, sk, i);
  #pragma unroll
      for (int i = 0; i < VU_PER_T; ++i) store_v(0, sv, i);
      load_k(kt[1], sk);
  #pragma unroll
      for (int i = 0; i < KC_PER_T; ++i) store_k(1, sk, i);
      load_k(kt[2], sk);
      load_v(kt[1], sv);
      // where the next fetches go, K of tile i + 3 and V of tile i + 2, read
      // at the end of the previous iteration (paged: outside the MFMA streams)
      PageBases at_k = locate(kt[3]), at_v = locate(kt[2]);
      __syncthreads();
      auto run = [&](auto is_a) INLINE {
        constexpr bool A = decltype(is_a)::value;
        if (A) stream(NO, YES, 0, 0, no_hook);
        __syncthreads();
        if (A) softmax(kt[0]);
        else stream(NO, YES, 0, 0, no_hook);
        __syncthreads();
        int it = 0;
        // iteration i (tile parity ip = i & 1): phases Y_i, X_i+1.  The streams
        // read V(i) (V slot ip) and K(i+1) (K slot 1 - ip); each thread stages
        // its K chunks of tile i + 2 into K slot ip between the MFMAs of its
        // stream and then fetches those of tile i + 3, and in its softmax phase
        // stores its V units of tile i + 1 into V slot 1 - ip and fetches those
        // of tile i + 2.
        auto iteration = [&](auto ipc) INLINE {
          constexpr int ip = decltype(ipc)::value;
          auto stage_hook = [&](auto jc) INLINE {
            constexpr int j = decltype(jc)::value;
            if constexpr (j >= 2 && j < 2 + 2 * KC_PER_T && (j - 2) % 2 == 0) store_k(ip, sk, (j - 2) / 2);
            if constexpr (j == 2 + 2 * KC_PER_T) load_k_at(at_k, sk);
          };
          auto softmax_v = [&](int kt_s) INLINE {
  #pragma unroll
            for (int u = 0; u < VU_PER_T; ++u) store_v(1 - ip, sv, u);
            load_v_at(at_v, sv);
            softmax(kt_s);
          };
          if (A) stream(YES, YES, ip, 1 - ip, stage_hook);
          else softmax_v(kt[0]);
          __syncthreads();
          if (!A) {
            stream(YES, YES, ip, 1 - ip, stage_hook);
          } else {
  #pragma unroll
            for (int u = 0; u < VU_PER_T; ++u) store_v(1 - ip, sv, u);
            load_v_at(at_v, sv);
            if (it + 1 < n_tiles) softmax(kt[1]);
          }
  #pragma unroll
          for (int j = 0; j < 4; ++j) kt[j] = kt[j + 1];
          kt[4] = tile_or_none(it + 5);
          at_v = at_k;
          at_k = locate(kt[3]);
          __syncthreads();
        };
        const std::integral_constant<int, 0> P0;
        const std::integral_constant<int, 1> P1;
        for (; it + 1 < n_tiles; it += 2) {
          iteration(P0);
          ++it;
          iteration(P1);
          --it;
        }
        if (it < n_tiles) iteration(P0);
      };
      if (__builtin_amdgcn_readfirstlane(wave) < 4) run(YES);
      else run(NO);
    }
  } else if constexpr (ALT) {
    if (n_tiles > 0) {
      // entering iteration i: K(i) is in K slot i & 1 and V(i - 1) in V slot
      // (i - 1) & 1; sv holds V(i), sk nothing; kt[j] is tile i + j and at1
      // locates tile i + 1
      KSet sk;
      VSet sv;
      int kt[2];
      first_tiles(kt);
      PageBases at1 = locate(kt[0]);
      load_k_at(at1, sk);
  #pragma unroll
      for (int i = 0; i < KC_PER_T; ++i) store_k(0, sk, i);
      load_v_at(at1, sv);
      at1 = locate(kt[1]);
      __syncthreads();
      // iteration i (parity ip): PV(i - 1) from V slot 1 - ip and QK(i) from
      // K slot ip; V(i) goes into V slot ip, K(i + 1) into K slot 1 - ip
      auto iteration = [&](auto ipc, auto pv, auto qk, int i) INLINE {
        constexpr int ip = decltype(ipc)::value;
        constexpr bool QK = decltype(qk)::value;
        constexpr int N = (decltype(pv)::value ? 2 * NCB : 0) + 4 * NKC;
        constexpr int S0 = N / 2;
        static_assert(S0 + 2 * VU_PER_T < N, "staging must fit between the MFMAs");
        auto stage_hook = [&](auto jc) INLINE {
          constexpr int j = decltype(jc)::value;
          if constexpr (QK) {
            if constexpr (j >= S0 && j < S0 + 2 * VU_PER_T && (j - S0) % 2 == 0)
              store_v(ip, sv, (j - S0) / 2);
            if constexpr (j == S0 + 2 * VU_PER_T) load_k_at(at1, sk);
          }
        };
        stream(pv, qk, 1 - ip, ip, stage_hook);
        if constexpr (QK) {
          softmax(kt[0]);
          __builtin_amdgcn_sched_barrier(0);
  #pragma unroll
          for (int u = 0; u < KC_PER_T; ++u) store_k(1 - ip, sk, u);
          __builtin_amdgcn_sched_barrier(0);
          load_v_at(at1, sv);
          kt[0] = kt[1];
          kt[1] = tile_or_none(i + 2);
          at1 = locate(kt[1]);
          __syncthreads();
        }
      };
      const std::integral_constant<int, 0> P0;
      const std::integral_constant<int, 1> P1;
      iteration(P0, NO, YES, 0);
      int it = 1;
      for (; it + 1 < n_tiles; it += 2) {
        iteration(P1, YES, YES, it);
        iteration(P0, YES, YES, it + 1);
      }
      if (it < n_tiles) {
        iteration(P1, YES, YES, it);
        iteration(P0, YES, NO, it + 1);
      } else {
        iteration(P1, YES, NO, it);
      }
    }
  } else {
    if (n_tiles > 0) {
      // entering iteration i: K(i) is in K slot i & 1 and V(i - 1) in V slot
      // (i - 1) & 1; sk holds K(i + 1), sv holds V(i); kt[j] is tile i + j,
      // at1 / at2 locate tiles i + 1 / i + 2
      KSet sk;
      VSet sv;
      int kt[3];
      first_tiles(kt);
      PageBases at1 = locate(kt[0]);
      load_k_at(at1, sk);
  #pragma unroll
      for (int i = 0; i < KC_PER_T; ++i) store_k(0, sk, i);
      load_v_at(at1, sv);
      at1 = locate(kt[1]);
      PageBases at2 = locate(kt[2]);
      load_k_at(at1, sk);
      __syncthreads();
      constexpr int L0 = 2 + 2 * (KC_PER_T + VU_PER_T);
      static_assert(L0 < 4 * NKC, "staging must fit between the QK MFMAs");
      // iteration i (parity ip): PV(i - 1) from V slot 1 - ip and QK(i) from
      // K slot ip; K(i + 1) goes into K slot 1 - ip and V(i) into V slot ip
      auto iteration = [&](auto ipc, auto pv, auto qk, int i) INLINE {
        constexpr int ip = decltype(ipc)::value;
        constexpr bool QK = decltype(qk)::value;
        auto stage_hook = [&](auto jc) INLINE {
          constexpr int j = decltype(jc)::value;
          if constexpr (QK) {
            if constexpr (j >= 2 && j < 2 + 2 * KC_PER_T && j % 2 == 0) store_k(1 - ip, sk, (j - 2) / 2);
            if constexpr (j >= 2 + 2 * KC_PER_T && j < L0 && j % 2 == 0)
              store_v(ip, sv, (j - 2 - 2 * KC_PER_T) / 2);
            if constexpr (j == L0) {
              load_k_at(at2, sk);
              load_v_at(at1, sv);
            }
          }
        };
        stream(pv, qk, 1 - ip, ip, stage_hook);
        if constexpr (QK) {
          softmax(kt[0]);
          kt[0] = kt[1];
          kt[1] = kt[2];
          kt[2] = tile_or_none(i + 3);
          at1 = at2;
          at2 = locate(kt[2]);
          __syncthreads();
        }
      };
      const std::integral_constant<int, 0> P0;
      const std::integral_constant<int, 1> P1;
      iteration(P0, NO, YES, 0);
      int it = 1;
      for (; it + 1 < n_tiles; it += 2) {
        iteration(P1, YES, YES, it);
        iteration(P0, YES, YES, it + 1);
      }
      if (it < n_tiles) {
        iteration(P1, YES, YES, it);
        iteration(P0, YES, NO, it + 1);
      } else {
        iteration(P1, YES, NO, it);
      }
    }
  }

  // O through LDS as in prefill_kernel: each wave stages its 16 x C block
  // (the K/V rings are free once every wave has left the tile loop) and
  // stores whole rows, 16 bytes per lane.
  constexpr int OROW = C + 8;
  constexpr int LDS_BYTES = (2 * TILE * (C + 8) + 2 * C * (TILE + 8)) * 2;
  static_assert(NW * 16 * OROW * 2 <= LDS_BYTES, "O staging exceeds the LDS");
  const float inv = (l_run > 0.f) ? 1.f / l_run : 0.f;
  __syncthreads();
  bf16_t* const ow = lds + wave * 16 * OROW;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    uint2 u;
    u.x = pack_bf16x2(acc[cb][0] * inv, acc[cb][1] * inv);
    u.y = pack_bf16x2(acc[cb][2] * inv, acc[cb][3] * inv);
    *reinterpret_cast<uint2*>(ow + l16 * OROW + 16 * cb + 4 * g) = u;
  }
  {
    constexpr int LPR = C / 8, RPI = 64 / LPR;   // lanes per row, rows per store
    const int r0 = lane / LPR, ch = 8 * (lane % LPR);
    bf16_t* const ob = a.o + o_off + (int64_t)p * a.o_sh;
#pragma unroll
    for (int i = 0; i < 16 / RPI; ++i) {
      const int r = r0 + RPI * i;
      const uint4 u = *reinterpret_cast<const uint4*>(ow + r * OROW + ch);
      if (q16 + r < n_q) *reinterpret_cast<uint4*>(ob + (int64_t)(q16 + r) * a.o_st + ch) = u;
    }
  }
  if (a.lse && g == 0 && t < n_q) {
    float v = (l_run > 0.f) ? m_run * a.scale + logf(l_run) : -INFINITY;
    a.lse[lse_off + (int64_t)p * n_q + t] = v;
  }
}

// Launch one instantiation with `lds` bytes of dynamic LDS.  The kernel's
// dynamic-LDS limit is raised once per device (bit d of its mask); setting
// it is idempotent, so two threads racing on a device both set it.
template <auto KERN>
hipError_t launch_kernel(const PrefillArgs& a, int n_work, int threads, int lds, hipStream_t s) {
  static std::atomic<uint64_t> attr_set{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? uint64_t(1) << dev : 0;
  if (!bit || !(attr_set.load(std::memory_order_acquire) & bit)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(KERN),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr_set.fetch_or(bit, std::memory_order_release);
  }
  hipLaunchKernelGGL(KERN, dim3(n_work), dim3(threads), lds, s, a);
  return hipGetLastError();
}

template <int C, int M, bool DENSE, bool PAGED>
hipError_t launch_one(const PrefillArgs& a, int n_work, hipStream_t s) {
  // three stages for the ping-pong schedule, two otherwise (so that two
  // workgroups of a small shape can share a CU)
  constexpr bool pp = Cfg<C>::PING_PONG && Shape<C, M>::WAVES == 8;
  constexpr int lds = (pp ? 3 : 2) * Cfg<C>::STAGE * 2;
  static_assert(lds <= 160 * 1024, "LDS budget");
  return launch_kernel<prefill_kernel<C, M, DENSE, PAGED>>(a, n_work, 64 * Shape<C, M>::WAVES, lds, s);
}

template <int C, int M, bool DENSE, bool PAGED>
hipError_t launch_q16(const PrefillArgs& a, int n_work, hipStream_t s) {
  constexpr int lds = (2 * TILE * (C + 8) + 2 * C * (TILE + 8)) * 2;   // two K and two V slots
  static_assert(lds <= 160 * 1024, "LDS budget");
  return launch_kernel<prefill_q16_kernel<C, M, DENSE, PAGED>>(a, n_work, 64 * M * q16_blocks(M), lds, s);
}

template <int C, int M>
hipError_t launch_c_m(const PrefillArgs& a, bool dense, int n_work, hipStream_t s) {
  const bool paged = a.kv.paged != 0;
  if constexpr (C == 256) {
    if (dense) return paged ? launch_q16<C, M, true, true>(a, n_work, s)
                            : launch_q16<C, M, true, false>(a, n_work, s);
    return paged ? launch_q16<C, M, false, true>(a, n_work, s)
                 : launch_q16<C, M, false, false>(a, n_work, s);
  } else {
    if (dense) return paged ? launch_one<C, M, true, true>(a, n_work, s)
                            : launch_one<C, M, true, false>(a, n_work, s);
    return paged ? launch_one<C, M, false, true>(a, n_work, s)
                 : launch_one<C, M, false, false>(a, n_work, s);
  }
}

template <int C>
hipError_t launch_c(const PrefillArgs& a, bool dense, int n_work, hipStream_t s) {
  switch (a.m) {
    case 1: return launch_c_m<C, 1>(a, dense, n_work, s);
    case 2: return launch_c_m<C, 2>(a, dense, n_work, s);
    case 4: return launch_c_m<C, 4>(a, dense, n_work, s);
    case 3: return launch_c_m<C, 3>(a, dense, n_work, s);
    case 5: return launch_c_m<C, 5>(a, dense, n_work, s);
    case 6: return launch_c_m<C, 6>(a, dense, n_work, s);
    case 7: return launch_c_m<C, 7>(a, dense, n_work, s);
    case 8: return launch_c_m<C, 8>(a, dense, n_work, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillLaunch& L, hipStream_t stream) {
  PrefillArgs a;
  a.q = static_cast<const bf16_t*>(L.q);
  a.o = static_cast<bf16_t*>(L.o);
  a.lse = L.lse;
  a.row_ptr = L.row_ptr;
  a.cols = L.cols;
  a.q_sh = L.q_sh;
  a.q_st = L.q_st;
  a.o_sh = L.o_sh;
  a.o_st = L.o_st;
  a.kv = L.kv;
  a.h_q = L.h_q;
  a.h_kv = L.h_kv;
  a.m = L.h_q / L.h_kv;
  a.scale = L.scale;
  // work items per (request, KV head, q-tile): two for the half-tile shapes
  const int per_row = parts_per_row(L.head_dim, a.m);
  const bool dense = L.row_ptr == nullptr;
  // one launch per group of kLaunchRequests requests (longest first)
  for (size_t g0 = 0; g0 < L.reqs.size(); g0 += kLaunchRequests) {
    const int n = (int)std::min<size_t>(kLaunchRequests, L.reqs.size() - g0);
    a.batch.n_req = n;
    int n_work = 0;
    for (int i = 0; i < n; ++i) {
      a.batch.r[i] = L.reqs[g0 + i];
      a.batch.r[i].work_begin = n_work;
      n_work += per_row * a.h_kv * a.batch.r[i].t_q;
    }
    if (n_work == 0) continue;
    hipError_t e;
    switch (L.head_dim) {
      case 64: e = launch_c<64>(a, dense, n_work, stream); break;
      case 128: e = launch_c<128>(a, dense, n_work, stream); break;
      case 256: e = launch_c<256>(a, dense, n_work, stream); break;
      default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace bfla
