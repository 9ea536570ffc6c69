/* A plain C host program that drives the library through include/bfla.h and
 * the HIP runtime's C API only (no C++, no Python, no torch): one request,
 * Stage 1, the tile lists, the sparse prefill and the dense prefill, with
 * every buffer sized by the library's own size queries.
 *
 * usage: bfla_c_driver IN OUT N H_Q H_KV C
 *   IN   raw bf16: Q [H_Q][N][C], then K [H_KV][N][C], then V [H_KV][N][C]
 *   OUT  int64 mask_bytes, n_rows, n_cols; then block_mask (uint8),
 *        row_ptr (int32, n_rows + 1), cols (int32, n_cols), sparse O (bf16),
 *        LSE (float, H_Q * N), dense O (bf16)
 * Hyper-parameters: b = 128, g = 64, T = 64, gamma = 0.9, n_local = 2,
 * n_sink = 1, eta = 16, rho = 0.1, seed = 7, default scale.
 * Prints "c driver ok" and exits 0, or names the failing call and exits 1. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "bfla.h"

#define HIP_OK(call)                                                        \
  do {                                                                      \
    hipError_t e_ = (call);                                                 \
    if (e_ != hipSuccess) {                                                 \
      fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));     \
      return 1;                                                             \
    }                                                                       \
  } while (0)

#define BFLA_OK_(call)                                                      \
  do {                                                                      \
    int s_ = (call);                                                        \
    if (s_ != BFLA_OK) {                                                    \
      fprintf(stderr, "%s failed: %s (%s)\n", #call, bfla_status_string(s_), \
              bfla_last_error());                                           \
      return 1;                                                             \
    }                                                                       \
  } while (0)

static int write_all(FILE* f, const void* p, size_t bytes) {
  return fwrite(p, 1, bytes, f) == bytes ? 0 : 1;
}

int main(int argc, char** argv) {
  if (argc != 7) {
    fprintf(stderr, "usage: %s IN OUT N H_Q H_KV C\n", argv[0]);
    return 1;
  }
  const int32_t n = atoi(argv[3]), h_q = atoi(argv[4]), h_kv = atoi(argv[5]),
                c = atoi(argv[6]);
  if (n < 1 || h_q < 1 || h_kv < 1 || c < 1) {
    fprintf(stderr, "bad sizes\n");
    return 1;
  }
  const size_t q_elems = (size_t)h_q * n * c, kv_elems = (size_t)h_kv * n * c;
  uint16_t* host = (uint16_t*)malloc((q_elems + 2 * kv_elems) * 2);
  FILE* in = fopen(argv[1], "rb");
  if (!host || !in || fread(host, 2, q_elems + 2 * kv_elems, in) != q_elems + 2 * kv_elems) {
    fprintf(stderr, "cannot read %s\n", argv[1]);
    return 1;
  }
  fclose(in);

  const bfla_problem prob = {1, h_q, h_kv, c, &n, &n};
  const bfla_params prm = {128, 64, 64, 0.9f, 2, 1, 16, 0.1, 7u, 0.0f};
  size_t n_rows = 0, max_cols = 0, mask_bytes = 0, score_elems = 0, ws_est = 0, ws_exp = 0;
  BFLA_OK_(bfla_list_capacity(&prob, &prm, &n_rows, &max_cols, &mask_bytes, &score_elems));
  BFLA_OK_(bfla_workspace_size(&prob, &prm, BFLA_WS_ESTIMATE, &ws_est));
  BFLA_OK_(bfla_workspace_size(&prob, &prm, BFLA_WS_EXPAND, &ws_exp));

  void *q, *k, *v, *o_sparse, *o_dense, *mask, *w_est, *w_exp;
  int32_t *row_ptr, *cols;
  float* lse;
  HIP_OK(hipMalloc(&q, q_elems * 2));
  HIP_OK(hipMalloc(&k, kv_elems * 2));
  HIP_OK(hipMalloc(&v, kv_elems * 2));
  HIP_OK(hipMalloc(&o_sparse, q_elems * 2));
  HIP_OK(hipMalloc(&o_dense, q_elems * 2));
  HIP_OK(hipMalloc(&mask, mask_bytes));
  HIP_OK(hipMalloc(&w_est, ws_est > 0 ? ws_est : 256));
  HIP_OK(hipMalloc(&w_exp, ws_exp > 0 ? ws_exp : 256));
  HIP_OK(hipMalloc((void**)&row_ptr, (n_rows + 1) * sizeof(int32_t)));
  HIP_OK(hipMalloc((void**)&cols, (max_cols > 0 ? max_cols : 1) * sizeof(int32_t)));
  HIP_OK(hipMalloc((void**)&lse, (size_t)h_q * n * sizeof(float)));
  HIP_OK(hipMemcpy(q, host, q_elems * 2, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(k, host + q_elems, kv_elems * 2, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(v, host + q_elems + kv_elems, kv_elems * 2, hipMemcpyHostToDevice));

  /* head-first [H][N][C] views */
  const bfla_view qv = {q, NULL, 0, (int64_t)n * c, c};
  const bfla_view osv = {o_sparse, NULL, 0, (int64_t)n * c, c};
  const bfla_view odv = {o_dense, NULL, 0, (int64_t)n * c, c};
  const bfla_kv kv = {BFLA_KV_CONTIGUOUS, k, v, NULL, 0, (int64_t)n * c, c, 0, 0, 0, NULL, 0};

  BFLA_OK_(bfla_estimate_mask(&prob, &prm, &qv, &kv, (uint8_t*)mask, NULL, NULL, w_est,
                              ws_est > 0 ? ws_est : 256, NULL));
  BFLA_OK_(bfla_expand_rescue(&prob, &prm, (const uint8_t*)mask, row_ptr, cols, max_cols, w_exp,
                              ws_exp > 0 ? ws_exp : 256, NULL));
  BFLA_OK_(bfla_sparse_prefill(&prob, &prm, &qv, &kv, row_ptr, cols, &osv, lse, NULL));
  BFLA_OK_(bfla_dense_prefill(&prob, &prm, &qv, &kv, &odv, NULL, NULL));
  HIP_OK(hipDeviceSynchronize());

  uint8_t* h_mask = (uint8_t*)malloc(mask_bytes);
  int32_t* h_rp = (int32_t*)malloc((n_rows + 1) * sizeof(int32_t));
  uint16_t* h_os = (uint16_t*)malloc(q_elems * 2);
  uint16_t* h_od = (uint16_t*)malloc(q_elems * 2);
  float* h_lse = (float*)malloc((size_t)h_q * n * sizeof(float));
  if (!h_mask || !h_rp || !h_os || !h_od || !h_lse) return 1;
  HIP_OK(hipMemcpy(h_mask, mask, mask_bytes, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_rp, row_ptr, (n_rows + 1) * sizeof(int32_t), hipMemcpyDeviceToHost));
  const int64_t n_cols = h_rp[n_rows];
  if (n_cols < 0 || (size_t)n_cols > max_cols) {
    fprintf(stderr, "list total %lld outside [0, %zu]\n", (long long)n_cols, max_cols);
    return 1;
  }
  int32_t* h_cols = (int32_t*)malloc((n_cols > 0 ? n_cols : 1) * sizeof(int32_t));
  if (!h_cols) return 1;
  HIP_OK(hipMemcpy(h_cols, cols, n_cols * sizeof(int32_t), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_os, o_sparse, q_elems * 2, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_od, o_dense, q_elems * 2, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_lse, lse, (size_t)h_q * n * sizeof(float), hipMemcpyDeviceToHost));

  FILE* out = fopen(argv[2], "wb");
  const int64_t header[3] = {(int64_t)mask_bytes, (int64_t)n_rows, n_cols};
  if (!out || write_all(out, header, sizeof header) || write_all(out, h_mask, mask_bytes) ||
      write_all(out, h_rp, (n_rows + 1) * sizeof(int32_t)) ||
      write_all(out, h_cols, n_cols * sizeof(int32_t)) || write_all(out, h_os, q_elems * 2) ||
      write_all(out, h_lse, (size_t)h_q * n * sizeof(float)) || write_all(out, h_od, q_elems * 2)) {
    fprintf(stderr, "cannot write %s\n", argv[2]);
    return 1;
  }
  fclose(out);
  printf("c driver ok: %zu rows, %lld kept tiles, library %s\n", n_rows, (long long)n_cols,
         bfla_version());
  return 0;
}
