"""Helpers shared by the GPU parity tests: device packing of seeded inputs,
calls through the C ABI, and the comparison bars."""
from __future__ import annotations

import numpy as np
import torch

from oracle import bfla_oracle as O
from paper_2605_12193_amd import bfla, synth

# Output bar for bf16 outputs against the float64 oracle on the same lists.
MAX_ABS = 2e-2
REL_L2 = 5e-3


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
        self.o = torch.full_like(self.q, float("nan"))
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
        self.o = torch.full_like(self.q, float("nan"))
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
