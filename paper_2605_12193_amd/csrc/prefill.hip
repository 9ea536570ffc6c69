// Fused GQA flash-style causal prefill over kept KV tiles (eq27), and the
// dense causal baseline (every causal tile).  gfx950 / CDNA4, wave64.
//
// Work item = one list row (request r, KV head h, query tile qt): all m
// query heads of the GQA group share every K/V tile load.  Each wave owns 32
// queries of one head (2 waves per head, 2m waves per workgroup).
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
// K/V tiles are double-buffered: the next list entry's tile is fetched into
// registers while the current one is consumed from LDS.
#include "bfla_device.h"
#include "bfla_internal.h"

namespace bfla {
namespace {

constexpr int TILE = 64;
constexpr float LOG2E = 1.4426950408889634f;

template <int C>
struct Cfg {
  static constexpr int KROW = C + 8;          // K tile row pitch (bf16), padded
  static constexpr int VROW = TILE + 8;       // V^T row pitch (bf16), padded
  static constexpr int K_ELEMS = TILE * KROW;
  static constexpr int V_ELEMS = C * VROW;
  static constexpr int STAGE = K_ELEMS + V_ELEMS;
  static constexpr int LDS_BYTES = 2 * STAGE * 2;
  static constexpr int K_CHUNKS = TILE * C / 8;   // 16-byte chunks per K tile
  static constexpr int V_UNITS = (TILE / 2) * (C / 8);  // key pairs x 8 channels
};

struct PrefillArgs {
  const bf16_t* q;
  bf16_t* o;
  float* lse;
  const int32_t* row_ptr;  // null -> dense
  const int32_t* cols;
  int64_t q_sh, q_st, o_sh, o_st;
  KvAddr kv;
  int32_t h_q, h_kv, m;
  float scale;
  Batch batch;
};

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint4 ld16(const bf16_t* p) {
  return *reinterpret_cast<const uint4*>(p);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

// Round-to-nearest-even float -> bf16 bits (inputs here are finite or 0).
__device__ __forceinline__ uint32_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f2bf(lo) | (f2bf(hi) << 16);
}

// Position of key offset k (0..63) inside the permuted V^T row.
__device__ __forceinline__ int vperm(int k) {
  return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

template <int C, int M>
__global__ void __launch_bounds__(128 * M)
prefill_kernel(PrefillArgs a) {
  using CF = Cfg<C>;
  constexpr int NT = 128 * M;
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
  const ReqDesc& R = a.batch.r[ri];
  const int local = w - R.work_begin;
  const int h = local % a.h_kv;
  const int qt = R.t_q - 1 - local / a.h_kv;
  const int n_c = R.n_kv - R.n_q;
  const int row = R.row_base + h * R.t_q + qt;

  int list_begin, list_end;
  if (a.row_ptr) {
    list_begin = a.row_ptr[row];
    list_end = a.row_ptr[row + 1];
  } else {
    int last = min(n_c + (qt + 1) * TILE - 1, R.n_kv - 1);
    list_begin = 0;
    list_end = last / TILE + 1;
  }
  const int n_tiles = list_end - list_begin;

  // ---- this wave's queries ----
  const int p = h * a.m + (wave >> 1);
  const int t = qt * TILE + (wave & 1) * 32 + l32;   // query index in request
  const bool q_ok = t < R.n_q;
  const int q_pos = n_c + t;                          // absolute position
  const int wave_q0 = n_c + qt * TILE + (wave & 1) * 32;

  bf16x8 qf[NKC];
  {
    const bf16_t* qp = a.q + R.q_off + (int64_t)p * a.q_sh + (int64_t)t * a.q_st + 8 * hi;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      uint4 v = q_ok ? ld16(qp + 16 * kc) : make_uint4(0, 0, 0, 0);
      qf[kc] = as_bf16x8(v);
    }
  }

  // ---- tile staging (global -> registers -> LDS) ----
  uint4 kreg[KC_PER_T];
  uint4 vreg[VU_PER_T][2];

  auto tile_of = [&](int i) -> int {
    return a.row_ptr ? a.cols[list_begin + i] : i;
  };

  auto load_tile = [&](int kt) {
#pragma unroll
    for (int i = 0; i < KC_PER_T; ++i) {
      int e = tid + i * NT;
      kreg[i] = make_uint4(0, 0, 0, 0);
      if (e < CF::K_CHUNKS) {
        int kr = e / (C / 8), ce = e % (C / 8);
        int key = kt * TILE + kr;
        if ((unsigned)key < (unsigned)R.n_kv)
          kreg[i] = ld16(a.kv.k + kv_elem(a.kv, R, h, key) + 8 * ce);
      }
    }
#pragma unroll
    for (int i = 0; i < VU_PER_T; ++i) {
      int u = tid + i * NT;
      vreg[i][0] = make_uint4(0, 0, 0, 0);
      vreg[i][1] = make_uint4(0, 0, 0, 0);
      if (u < CF::V_UNITS) {
        int ce = u % (C / 8), j = u / (C / 8);
        int key = kt * TILE + 2 * j;
        if ((unsigned)key < (unsigned)R.n_kv)
          vreg[i][0] = ld16(a.kv.v + kv_elem(a.kv, R, h, key) + 8 * ce);
        if ((unsigned)(key + 1) < (unsigned)R.n_kv)
          vreg[i][1] = ld16(a.kv.v + kv_elem(a.kv, R, h, key + 1) + 8 * ce);
      }
    }
  };

  auto store_tile = [&](bf16_t* st) {
    bf16_t* ks = st;
    bf16_t* vs = st + CF::K_ELEMS;
#pragma unroll
    for (int i = 0; i < KC_PER_T; ++i) {
      int e = tid + i * NT;
      if (e < CF::K_CHUNKS) {
        int kr = e / (C / 8), ce = e % (C / 8);
        *reinterpret_cast<uint4*>(ks + kr * CF::KROW + 8 * ce) = kreg[i];
      }
    }
#pragma unroll
    for (int i = 0; i < VU_PER_T; ++i) {
      int u = tid + i * NT;
      if (u < CF::V_UNITS) {
        int ce = u % (C / 8), j = u / (C / 8);
        int pos = vperm(2 * j);
        const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&vreg[i][0]);
        const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&vreg[i][1]);
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          // channels 8ce + 2e2 (low halves) and 8ce + 2e2 + 1 (high halves)
          uint32_t lo = (r0[e2] & 0xFFFFu) | (r1[e2] << 16);
          uint32_t hi2 = (r0[e2] >> 16) | (r1[e2] & 0xFFFF0000u);
          *reinterpret_cast<uint32_t*>(vs + (8 * ce + 2 * e2) * CF::VROW + pos) = lo;
          *reinterpret_cast<uint32_t*>(vs + (8 * ce + 2 * e2 + 1) * CF::VROW + pos) = hi2;
        }
      }
    }
  };

  // ---- online softmax state (one query per lane; both lane halves agree) ----
  const float c2 = a.scale * LOG2E;
  float m_run = -INFINITY;
  float l_run = 0.f;
  f32x16 acc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[cb][r] = 0.f;

  if (n_tiles > 0) {
    load_tile(tile_of(0));
    store_tile(lds);
  }
  __syncthreads();

  for (int it = 0; it < n_tiles; ++it) {
    const int kt = tile_of(it);
    const bool more = it + 1 < n_tiles;
    if (more) load_tile(tile_of(it + 1));

    const bf16_t* ks = lds + (it & 1) * CF::STAGE;
    const bf16_t* vs = ks + CF::K_ELEMS;

    // S^T = K . Q^T  (two 32-key blocks)
    f32x16 s0, s1;
#pragma unroll
    for (int r = 0; r < 16; ++r) { s0[r] = 0.f; s1[r] = 0.f; }
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      bf16x8 a0 = as_bf16x8(ld16(ks + l32 * CF::KROW + 16 * kc + 8 * hi));
      bf16x8 a1 = as_bf16x8(ld16(ks + (32 + l32) * CF::KROW + 16 * kc + 8 * hi));
      s0 = mfma32(a0, qf[kc], s0);
      s1 = mfma32(a1, qf[kc], s1);
    }

    // token-level causal mask and key bound, only where the tile needs it;
    // a list entry outside [0, T_kv) contributes nothing
    const int key0 = kt * TILE;
    if ((unsigned)kt >= (unsigned)R.t_kv || key0 + TILE - 1 > wave_q0 || key0 + TILE > R.n_kv) {
      const bool bad = (unsigned)kt >= (unsigned)R.t_kv;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int kk = key0 + 8 * (r >> 2) + 4 * hi + (r & 3);
        if (bad || kk > q_pos || kk >= R.n_kv) s0[r] = -INFINITY;
        kk += 32;
        if (bad || kk > q_pos || kk >= R.n_kv) s1[r] = -INFINITY;
      }
    }

    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, fmaxf(s0[r], s1[r]));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float corr = __builtin_amdgcn_exp2f((m_run - m_use) * c2);
    const float moff = -m_use * c2;
    float rs = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s0[r] = __builtin_amdgcn_exp2f(fmaf(s0[r], c2, moff));
      s1[r] = __builtin_amdgcn_exp2f(fmaf(s1[r], c2, moff));
      rs += s0[r] + s1[r];
    }
    rs += __shfl_xor(rs, 32);
    l_run = l_run * corr + rs;
    m_run = m_new;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[cb][r] *= corr;

    // P^T (bf16) as B operands: 16-key chunk q = regs 8(q%2).. of block q/2
    bf16x8 pf[4];
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const f32x16& sb = (qq < 2) ? s0 : s1;
      const int base = 8 * (qq & 1);
      uint4 u;
      u.x = pack_bf16x2(sb[base + 0], sb[base + 1]);
      u.y = pack_bf16x2(sb[base + 2], sb[base + 3]);
      u.z = pack_bf16x2(sb[base + 4], sb[base + 5]);
      u.w = pack_bf16x2(sb[base + 6], sb[base + 7]);
      pf[qq] = as_bf16x8(u);
    }

    // O^T += V^T . P^T
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        bf16x8 av = as_bf16x8(ld16(vs + (32 * cb + l32) * CF::VROW + 16 * qq + 8 * hi));
        acc[cb] = mfma32(av, pf[qq], acc[cb]);
      }
    }

    if (more) store_tile(lds + ((it + 1) & 1) * CF::STAGE);
    __syncthreads();
  }

  // ---- epilogue: O = O^T / l, LSE ----
  if (!q_ok) return;
  const float inv = (l_run > 0.f) ? 1.f / l_run : 0.f;
  bf16_t* op = a.o + R.o_off + (int64_t)p * a.o_sh + (int64_t)t * a.o_st;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      uint2 u;
      u.x = pack_bf16x2(acc[cb][4 * rg + 0] * inv, acc[cb][4 * rg + 1] * inv);
      u.y = pack_bf16x2(acc[cb][4 * rg + 2] * inv, acc[cb][4 * rg + 3] * inv);
      *reinterpret_cast<uint2*>(op + 32 * cb + 8 * rg + 4 * hi) = u;
    }
  }
  if (a.lse && hi == 0) {
    float v = (l_run > 0.f) ? m_run * a.scale + logf(l_run) : -INFINITY;
    a.lse[R.lse_off + (int64_t)p * R.n_q + t] = v;
  }
}

template <int C, int M>
hipError_t launch_c_m(const PrefillArgs& a, int n_work, hipStream_t s) {
  auto kern = prefill_kernel<C, M>;
  constexpr int lds = Cfg<C>::LDS_BYTES;
  static_assert(lds <= 160 * 1024, "LDS budget");
  static bool attr_set = false;  // idempotent; a benign race sets it twice
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3(n_work), dim3(128 * M), lds, s, a);
  return hipGetLastError();
}

template <int C>
hipError_t launch_c(const PrefillArgs& a, int n_work, hipStream_t s) {
  switch (a.m) {
    case 1: return launch_c_m<C, 1>(a, n_work, s);
    case 2: return launch_c_m<C, 2>(a, n_work, s);
    case 4: return launch_c_m<C, 4>(a, n_work, s);
    case 5: return launch_c_m<C, 5>(a, n_work, s);
    case 8: return launch_c_m<C, 8>(a, n_work, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool prefill_supported(int head_dim, int m) {
  bool c_ok = head_dim == 64 || head_dim == 128 || head_dim == 256;
  bool m_ok = m == 1 || m == 2 || m == 4 || m == 5 || m == 8;
  return c_ok && m_ok;
}

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
  a.batch = L.batch;
  int n_work = 0;
  for (int i = 0; i < a.batch.n_req; ++i) {
    a.batch.r[i].work_begin = n_work;
    n_work += a.h_kv * a.batch.r[i].t_q;
  }
  if (n_work == 0) return hipSuccess;
  switch (L.head_dim) {
    case 64: return launch_c<64>(a, n_work, stream);
    case 128: return launch_c<128>(a, n_work, stream);
    case 256: return launch_c<256>(a, n_work, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bfla
