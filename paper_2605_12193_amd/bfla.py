"""Python binding of libbfla.so (the C ABI declared in include/bfla.h).

Argument marshalling only: torch provides device memory and the current
stream; every step of the path runs in the library's HIP kernels.  Importing
this module does not load the library; the first call does, and raises if
libbfla.so has not been built (there is no fallback).
"""
from __future__ import annotations

import ctypes as C
import math
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

import torch

from .abi import (BFLA_ERR_CAPACITY, BFLA_ERR_HIP, BFLA_ERR_INVALID_ARG,  # noqa: F401
                  BFLA_ERR_UNSUPPORTED, BFLA_ERR_WORKSPACE, BFLA_KV_CONTIGUOUS, BFLA_KV_PAGED,
                  BFLA_OK, BFLA_WS_ESTIMATE, BFLA_WS_EXPAND, EXPAND_SCRATCH_BYTES, EXPORTS,
                  MAX_BATCH, bfla_kv,
                  bfla_params, bfla_problem, bfla_view)
from .abi import SIGS as _SIGS  # noqa: F401
from .abi import bind as _bind

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbfla.so")


class BflaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"bfla status {status}: {message}")
        self.status = status


_lib = None


def lib():
    """The loaded library (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2605_12193_amd.build`")
        _lib = _bind(_LIB_PATH)
    return _lib


def _check(status: int) -> None:
    if status != BFLA_OK:
        raise BflaError(status, lib().bfla_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream) -> C.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


# ---------------------------------------------------------------------------
# Host-side descriptions (they own the arrays the C structs point to)
# ---------------------------------------------------------------------------

class Problem:
    def __init__(self, n_q: Sequence[int], n_kv: Sequence[int], h_q: int, h_kv: int,
                 head_dim: int):
        self.n_q = list(n_q)
        self.n_kv = list(n_kv)
        self._nq = (C.c_int32 * len(self.n_q))(*self.n_q)
        self._nkv = (C.c_int32 * len(self.n_kv))(*self.n_kv)
        self.c = bfla_problem(len(self.n_q), h_q, h_kv, head_dim, self._nq, self._nkv)

    @property
    def batch(self):
        return self.c.batch


def params(block=128, group=64, tile=64, gamma=0.9, n_local=2, n_sink=1, eta=16,
           rho=0.0, seed=0, scale=0.0) -> bfla_params:
    return bfla_params(block, group, tile, gamma, n_local, n_sink, eta, rho, seed, scale)


class View:
    """bfla_view of a bf16 tensor whose last dim is head_dim."""

    def __init__(self, t: torch.Tensor, stride_head: int, stride_tok: int,
                 stride_batch: int = 0, batch_offsets: Optional[Sequence[int]] = None):
        self.t = t
        self._off = None
        if batch_offsets is not None:
            self._off = (C.c_int64 * len(batch_offsets))(*batch_offsets)
        self.c = bfla_view(t.data_ptr(), self._off, stride_batch, stride_head, stride_tok)


def view_hnc(t: torch.Tensor) -> View:
    """[H][N][C] (one request) or [B][H][N][C]."""
    if t.dim() == 3:
        return View(t, t.stride(0), t.stride(1))
    return View(t, t.stride(1), t.stride(2), t.stride(0))


def view_packed(t: torch.Tensor, token_starts: Sequence[int]) -> View:
    """Packed token-major varlen [sum N][H][C]; request r starts at token_starts[r]."""
    return View(t, t.stride(1), t.stride(0),
                batch_offsets=[int(s) * t.stride(0) for s in token_starts])


class KV:
    """bfla_kv of K and V, which share one set of strides (the library reads
    both through the same addressing); a paged table is int32 [B][max_pages]."""

    def __init__(self, k: torch.Tensor, v: torch.Tensor, *, paged: bool = False,
                 block_table: Optional[torch.Tensor] = None,
                 batch_offsets: Optional[Sequence[int]] = None):
        if k.shape != v.shape or k.stride() != v.stride():
            raise ValueError(f"k {tuple(k.shape)}/{tuple(k.stride())} and v "
                             f"{tuple(v.shape)}/{tuple(v.stride())} need the same shape "
                             "and strides")
        if paged:
            if k.dim() != 4:
                raise ValueError("paged k / v must be [pages][page_size][H_kv][C]")
            if block_table is None or block_table.dtype != torch.int32 \
                    or block_table.dim() != 2 or not block_table.is_contiguous():
                raise ValueError("block_table must be a contiguous int32 [batch][max_pages] "
                                 "tensor")
            if block_table.device != k.device:
                raise ValueError("block_table must be on the same device as k / v")
        self.k, self.v, self.block_table = k, v, block_table
        self._off = None
        if paged:
            # pools [pages][page_size][H_kv][C]
            self.c = bfla_kv(BFLA_KV_PAGED, k.data_ptr(), v.data_ptr(), None, 0,
                             k.stride(2), k.stride(1), k.shape[1], block_table.shape[1],
                             k.stride(0), block_table.data_ptr(), k.shape[0])
        else:
            if batch_offsets is not None:
                self._off = (C.c_int64 * len(batch_offsets))(*batch_offsets)
            if k.dim() == 3:   # [H][N][C]
                sb, sh, st = 0, k.stride(0), k.stride(1)
            else:              # [B][H][N][C]
                sb, sh, st = k.stride(0), k.stride(1), k.stride(2)
            self.c = bfla_kv(BFLA_KV_CONTIGUOUS, k.data_ptr(), v.data_ptr(), self._off,
                             sb, sh, st, 0, 0, 0, None, 0)


# ---------------------------------------------------------------------------
# Entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def bfla_version() -> str:
    return lib().bfla_version().decode()


def bfla_status_string(status: int) -> str:
    return lib().bfla_status_string(status).decode()


@dataclass
class Capacity:
    n_rows: int
    max_cols: int
    mask_bytes: int
    score_elems: int


def bfla_list_capacity(prob: Problem, prm: bfla_params) -> Capacity:
    vals = [C.c_size_t() for _ in range(4)]
    _check(lib().bfla_list_capacity(C.byref(prob.c), C.byref(prm), *[C.byref(v) for v in vals]))
    return Capacity(*[v.value for v in vals])


def bfla_workspace_size(prob: Problem, prm: bfla_params, which: int) -> int:
    n = C.c_size_t()
    _check(lib().bfla_workspace_size(C.byref(prob.c), C.byref(prm), which, C.byref(n)))
    return n.value


def bfla_estimate_mask(prob: Problem, prm: bfla_params, q: View, kv: KV,
                       block_mask: torch.Tensor, dbg_scores: Optional[torch.Tensor] = None,
                       dbg_head_mask: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().bfla_estimate_mask(C.byref(prob.c), C.byref(prm), C.byref(q.c), C.byref(kv.c),
                                    _ptr(block_mask), _ptr(dbg_scores), _ptr(dbg_head_mask),
                                    _ptr(workspace), ws_bytes, _stream(stream)))


def bfla_expand_rescue(prob: Problem, prm: bfla_params, block_mask: torch.Tensor,
                       row_ptr: torch.Tensor, cols: torch.Tensor, workspace: torch.Tensor,
                       stream=None) -> None:
    _check(lib().bfla_expand_rescue(C.byref(prob.c), C.byref(prm), _ptr(block_mask),
                                    _ptr(row_ptr), _ptr(cols), cols.numel(), _ptr(workspace),
                                    workspace.numel() * workspace.element_size(),
                                    _stream(stream)))


def bfla_expand_rescue_noalloc(prob: Problem, prm: bfla_params, block_mask: torch.Tensor,
                               row_ptr: torch.Tensor, cols: torch.Tensor, stream=None) -> None:
    """bfla_expand_rescue with the library's fixed per-device scratch in place of
    a workspace (no allocation anywhere)."""
    _check(lib().bfla_expand_rescue_noalloc(C.byref(prob.c), C.byref(prm), _ptr(block_mask),
                                            _ptr(row_ptr), _ptr(cols), cols.numel(),
                                            _stream(stream)))


def bfla_sparse_prefill(prob: Problem, prm: bfla_params, q: View, kv: KV,
                        row_ptr: torch.Tensor, cols: torch.Tensor, o: View,
                        lse: Optional[torch.Tensor] = None, stream=None) -> None:
    _check(lib().bfla_sparse_prefill(C.byref(prob.c), C.byref(prm), C.byref(q.c), C.byref(kv.c),
                                     _ptr(row_ptr), _ptr(cols), C.byref(o.c), _ptr(lse),
                                     _stream(stream)))


def bfla_dense_prefill(prob: Problem, prm: bfla_params, q: View, kv: KV, o: View,
                       lse: Optional[torch.Tensor] = None, stream=None) -> None:
    _check(lib().bfla_dense_prefill(C.byref(prob.c), C.byref(prm), C.byref(q.c), C.byref(kv.c),
                                    C.byref(o.c), _ptr(lse), _stream(stream)))


# ---------------------------------------------------------------------------
# Convenience: buffers for a whole pass
# ---------------------------------------------------------------------------

class Buffers:
    """Device buffers of one sparse-prefill pass (allocated once, reused)."""

    def __init__(self, prob: Problem, prm: bfla_params, device="cuda", lse=True):
        cap = bfla_list_capacity(prob, prm)
        self.cap = cap
        self.block_mask = torch.empty(max(cap.mask_bytes, 1), dtype=torch.uint8, device=device)
        self.scores = torch.empty(max(cap.score_elems, 1), dtype=torch.float32, device=device)
        self.row_ptr = torch.empty(cap.n_rows + 1, dtype=torch.int32, device=device)
        self.cols = torch.empty(max(cap.max_cols, 1), dtype=torch.int32, device=device)
        ws = bfla_workspace_size(prob, prm, BFLA_WS_EXPAND)
        self.ws_expand = torch.empty(max(ws, 16), dtype=torch.uint8, device=device)
        ws = bfla_workspace_size(prob, prm, BFLA_WS_ESTIMATE)
        self.ws_estimate = torch.empty(max(ws, 16), dtype=torch.uint8, device=device)
        n_lse = sum(prob.c.h_q * n for n in prob.n_q)
        self.lse = torch.empty(n_lse, dtype=torch.float32, device=device) if lse else None


def sparse_pass(prob: Problem, prm: bfla_params, q: View, kv: KV, o: View, buf: Buffers,
                stream=None) -> None:
    """Stage 1 -> tile lists -> sparse prefill, all enqueued on one stream."""
    bfla_estimate_mask(prob, prm, q, kv, buf.block_mask, dbg_scores=buf.scores,
                       workspace=buf.ws_estimate, stream=stream)
    bfla_expand_rescue(prob, prm, buf.block_mask, buf.row_ptr, buf.cols, buf.ws_expand,
                       stream=stream)
    bfla_sparse_prefill(prob, prm, q, kv, buf.row_ptr, buf.cols, o, buf.lse, stream=stream)
