// Device-side types shared by the HIP kernels and their host launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bfla.h"

namespace bfla {

typedef uint16_t bf16_t;  // raw bfloat16 bits

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// One request as the kernels see it (element / byte offsets already
// resolved on the host).
struct ReqDesc {
  int64_t q_off;      // element offset of (r, head 0, token 0) in Q
  int64_t o_off;      // same in O
  int64_t kv_off;     // same in contiguous K/V (0 when paged)
  int64_t lse_off;    // float offset of request r in lse
  int64_t mask_off;   // byte offset of request r in block_mask
  int64_t score_off;  // float offset of request r in the score buffer
  int32_t n_q, n_kv;  // tokens
  int32_t l_q, l_kv;  // coarse blocks
  int32_t t_q, t_kv;  // attention tiles
  int32_t row_base;   // first list row of this request
  int32_t work_begin; // first work item of this request in the launch
  int32_t bt_row;     // row of the block table (original request index)
  int32_t pad_;
};

// Requests per kernel launch: their descriptors travel in the kernel
// arguments, so a call with more requests launches each kernel once per
// group of this many (in the launch order of its entry point).
constexpr int kLaunchRequests = 32;

struct Batch {
  int32_t n_req;
  int32_t pad_[3];
  ReqDesc r[kLaunchRequests];
};

// K/V addressing shared by every kernel that reads keys or values.
struct KvAddr {
  const bf16_t* k;
  const bf16_t* v;
  const int32_t* block_table;
  int64_t stride_head, stride_tok;
  int64_t page_stride;
  int32_t page_size, max_pages;
  int32_t paged;
  uint32_t pool_bytes;  // paged: bytes from the pool base to the end of its last page
  int32_t n_pages;      // paged: valid page numbers are [0, n_pages)
  int32_t pad_;
};

// Request owning work item `w`: the last request whose first item is at or
// before w (work_begin ascends over the requests of a launch); a binary
// search over at most kLaunchRequests descriptors.
__device__ __forceinline__ int find_req(const Batch& b, int w) {
  int r = 0;
#pragma unroll
  for (int step = kLaunchRequests / 2; step >= 1; step >>= 1)
    if (r + step < b.n_req && w >= b.r[r + step].work_begin) r += step;
  return r;
}

}  // namespace bfla
