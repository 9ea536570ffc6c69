"""Helpers shared by the GPU parity tests: device packing of seeded inputs,
calls through the C ABI, the comparison bars, and canary bands around every
output buffer (4 KiB of a fixed byte pattern before and after it, checked
after each entry point: a write out of bounds changes a band)."""
from __future__ import annotations

import numpy as np
import torch

from oracle import bfla_oracle as O
from paper_2605_12193_amd import bfla, synth

# Output bar for bf16 outputs against the float64 oracle on the same lists.
MAX_ABS = 2e-2
REL_L2 = 5e-3

GUARD_BYTES = 4096
GUARD_BYTE = 0xA5


class Guarded:
    """A device buffer of n elements between two 4 KiB canary bands; ``t`` is
    the buffer itself (16-byte aligned like any fresh allocation)."""

    def __init__(self, n, dtype, fill=None, device="cuda"):
        item = torch.empty((), dtype=dtype).element_size()
        pad = GUARD_BYTES // item
        self._raw = torch.empty(n + 2 * pad, dtype=dtype, device=device)
        self._raw.view(torch.uint8).fill_(GUARD_BYTE)
        self.t = self._raw[pad:pad + n]
        if fill is not None:
            self.t.fill_(fill)

    def check(self, what):
        b = self._raw.view(torch.uint8)
        for name, band in (("before", b[:GUARD_BYTES]), ("after", b[-GUARD_BYTES:])):
            bad = torch.nonzero(band != GUARD_BYTE).flatten()
            assert bad.numel() == 0, (f"{what}: canary band {name} the buffer overwritten at "
                                      f"{bad[:8].tolist()} ({bad.numel()} bytes)")


class GuardedBuffers:
    """The buffers of one pass (as bfla.Buffers), each between canary bands;
    optionally the per-query-head keep sets of Stage 1."""

    def __init__(self, prob, prm, head_mask=False):
        cap = bfla.bfla_list_capacity(prob, prm)
        self.cap = cap
        ws = bfla.bfla_workspace_size(prob, prm, bfla.BFLA_WS_EXPAND)
        ws_est = bfla.bfla_workspace_size(prob, prm, bfla.BFLA_WS_ESTIMATE)
        n_lse = sum(prob.c.h_q * n for n in prob.n_q)
        self.g = {
            "block_mask": Guarded(max(cap.mask_bytes, 1), torch.uint8, fill=9),
            "scores": Guarded(max(cap.score_elems, 1), torch.float32, fill=float("nan")),
            "row_ptr": Guarded(cap.n_rows + 1, torch.int32, fill=-5),
            "cols": Guarded(max(cap.max_cols, 1), torch.int32, fill=-7),
            "ws_expand": Guarded(max(ws, 16), torch.uint8),
            "ws_estimate": Guarded(max(ws_est, 16), torch.uint8),
            "lse": Guarded(n_lse, torch.float32, fill=float("nan")),
        }
        if head_mask:
            self.g["head_mask"] = Guarded(max(cap.score_elems, 1), torch.uint8, fill=9)
        for k, v in self.g.items():
            setattr(self, k, v.t)
        if not head_mask:
            self.head_mask = None

    def check(self, what=""):
        for k, v in self.g.items():
            v.check(f"{what} {k}")


class DeviceBatch:
    """Requests packed per head along the token axis: Q [H_q][sum N_q][C],
    K/V [H_kv][sum N_kv][C]; request r is addressed by element offsets."""

    def __init__(self, seqs, n_q=None):
        self.seqs = seqs
        h_q, _, c = seqs[0].q.shape
        h_kv = seqs[0].k.shape[0]
        self.n_kv = [s.k.shape[1] for s in seqs]
        self.n_q = list(n_q) if n_q is not None else [s.q.shape[1] for s in seqs]
        # queries of a chunked request are its LAST n_q tokens
        qs = [s.q[:, s.q.shape[1] - nq:] for s, nq in zip(seqs, self.n_q)]
        self.q = torch.cat(qs, dim=1).contiguous().cuda()
        self.k = torch.cat([s.k for s in seqs], dim=1).contiguous().cuda()
        self.v = torch.cat([s.v for s in seqs], dim=1).contiguous().cuda()
        self.o_guard = Guarded(self.q.numel(), self.q.dtype, fill=float("nan"))
        self.o = self.o_guard.t.view(self.q.shape)
        self.q_start = np.concatenate([[0], np.cumsum(self.n_q)[:-1]]).astype(int)
        self.kv_start = np.concatenate([[0], np.cumsum(self.n_kv)[:-1]]).astype(int)
        self.prob = bfla.Problem(self.n_q, self.n_kv, h_q, h_kv, c)
        self.qv = bfla.View(self.q, self.q.stride(0), self.q.stride(1),
                            batch_offsets=[int(s) * c for s in self.q_start])
        self.ov = bfla.View(self.o, self.o.stride(0), self.o.stride(1),
                            batch_offsets=[int(s) * c for s in self.q_start])
        self.kv = bfla.KV(self.k, self.v, batch_offsets=[int(s) * c for s in self.kv_start])
        self.h_q, self.h_kv, self.c = h_q, h_kv, c

    def host(self, r):
        s = self.seqs[r]
        nq = self.n_q[r]
        q = s.q[:, s.q.shape[1] - nq:].double().numpy()
        return q, s.k.double().numpy(), s.v.double().numpy()

    def o_of(self, r):
        a = self.q_start[r]
        return self.o[:, a:a + self.n_q[r]].float().cpu().numpy()


class PagedBatch:
    """Packed token-major Q/O [sum N_q][H_q][C]; K/V in page pools."""

    def __init__(self, seqs, n_q, page_size, seed):
        self.n_kv = [s.k.shape[1] for s in seqs]
        self.n_q = list(n_q)
        h_q, _, c = seqs[0].q.shape
        h_kv = seqs[0].k.shape[0]
        qs = [s.q[:, s.q.shape[1] - nq:].transpose(0, 1) for s, nq in zip(seqs, self.n_q)]
        self.q = torch.cat(qs, dim=0).contiguous().cuda()          # [sum N_q][H_q][C]
        self.o_guard = Guarded(self.q.numel(), self.q.dtype, fill=float("nan"))
        self.o = self.o_guard.t.view(self.q.shape)
        starts = np.concatenate([[0], np.cumsum(self.n_q)[:-1]]).astype(int)
        table, total = synth.page_table(seed, self.n_kv, page_size)
        kp, vp = synth.to_paged(seqs, table, total, page_size)
        self.kp, self.vp = kp.cuda(), vp.cuda()
        self.table = torch.from_numpy(table).cuda()
        self.prob = bfla.Problem(self.n_q, self.n_kv, h_q, h_kv, c)
        self.qv = bfla.view_packed(self.q, starts)
        self.ov = bfla.view_packed(self.o, starts)
        self.kv = bfla.KV(self.kp, self.vp, paged=True, block_table=self.table)
        self.starts = starts

    def o_of(self, r):
        a = self.starts[r]
        return self.o[a:a + self.n_q[r]].transpose(0, 1).float().cpu().numpy()


def lists_to_device(row_ptr, cols):
    rp = torch.from_numpy(np.asarray(row_ptr, np.int32)).cuda()
    cl = torch.from_numpy(np.asarray(cols, np.int32) if len(cols) else np.zeros(1, np.int32)).cuda()
    return rp, cl


def request_rows(db: DeviceBatch, r: int, T: int = 64):
    base = sum(db.h_kv * -(-n // T) for n in db.n_q[:r])
    return base


def compare_outputs(got: np.ndarray, want: np.ndarray, what: str):
    """The bar for a bf16 output against the oracle: max-abs and rel-L2."""
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - want)
    max_abs = float(err.max()) if err.size else 0.0
    rel = float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-30))
    assert max_abs <= MAX_ABS, f"{what}: max-abs {max_abs:.3e} > {MAX_ABS}"
    assert rel <= REL_L2, f"{what}: rel-L2 {rel:.3e} > {REL_L2}"
    return max_abs, rel


def oracle_lists_for(db: DeviceBatch, masks, prm_kw):
    return O.expand_rescue(masks, db.n_q, db.n_kv, prm_kw["block"], prm_kw["tile"],
                           prm_kw["n_local"], prm_kw["n_sink"], prm_kw["eta"],
                           prm_kw["rho"], prm_kw["seed"])


def head_mask_compare(gpu_head: np.ndarray, head_keep: np.ndarray, head_tie: np.ndarray,
                      gpu_mask: np.ndarray = None):
    """Per-query-head keep sets (eq18) against the oracle's: every cell that
    is not a near-tie for its head must match; returns the near-tie cells
    that differ.  Given the GPU's block mask, it must be the OR of the GPU's
    own head sets over each GQA group, bit for bit."""
    assert set(np.unique(gpu_head)) <= {0, 1}, "head mask holds values other than 0 / 1"
    got = gpu_head.astype(bool)
    bad = np.argwhere(~head_tie & (got != head_keep))
    assert bad.size == 0, (f"per-head mismatches on {len(bad)} non-tie cells "
                           f"(e.g. {bad[:5].tolist()})")
    if gpu_mask is not None:
        h_kv = gpu_mask.shape[0]
        union = got.reshape(h_kv, -1, *got.shape[1:]).any(axis=1)
        assert np.array_equal(union, gpu_mask.astype(bool)), "block mask != OR of head masks"
    return int((head_tie & (got != head_keep)).sum())


def mask_compare(gpu_mask: np.ndarray, oracle_mask: np.ndarray, status: np.ndarray):
    """Block-mask parity with near-tie accounting: every sure cell must
    match; returns the number of near-tie cells where the two differ."""
    keep_sure = status == O.KEEP_SURE
    drop_sure = status == O.DROP_SURE
    bad_keep = np.argwhere(keep_sure & (gpu_mask == 0))
    bad_drop = np.argwhere(drop_sure & (gpu_mask != 0))
    assert bad_keep.size == 0 and bad_drop.size == 0, (
        f"sure-cell mismatches: {len(bad_keep)} kept->dropped (e.g. {bad_keep[:5].tolist()}), "
        f"{len(bad_drop)} dropped->kept (e.g. {bad_drop[:5].tolist()})")
    return int(((status == O.TIE) & ((gpu_mask != 0) != (oracle_mask != 0))).sum())
