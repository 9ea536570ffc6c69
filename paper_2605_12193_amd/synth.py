"""Seeded synthetic inputs for the block-filtered sparse prefill path.

This module only draws tensors; it contains none of the method's arithmetic
(no scores, masks, hashes or attention).  Both the HIP path (through the
tests and the benchmark) and the CPU oracle consume what it returns, so it
imports neither of them.

Recipe (the same for every workload, parameters in ``WORKLOADS``):

* ``numpy.random.Generator(PCG64(seed))``; a paged batch draws sequence ``s``
  from ``PCG64([seed, s])`` and its page permutation from ``PCG64(seed)``.
* Draw order: a unit direction ``d_h`` per KV head, then Q, K, V as
  N(0, 1) float32, then the heavy-hitter positions.
* Every query of head ``p`` is shifted by ``beta * d_{p // m}`` (the shared
  direction of its KV head, ``beta = 3``).
* ``round(0.01 * N)`` heavy-hitter keys per KV head, uniform without
  replacement over positions ``[4, N)``, are shifted by ``3 * d_h`` (+3 sigma).
* Optional slow positional drift (wide-head workload): every key gets
  ``0.5 * cos(2 pi t / 8192) * d_h``.
* Sinks, set last: keys 0..3 of KV head ``h`` become ``4 * u_h`` where
  ``u_h`` is the unit mean query direction of the head's query group.
* V carries no structure.
* Everything is rounded once to bfloat16 (round-to-nearest-even, torch CPU).

The shapes are those of the attention layers the paper evaluates on
(Llama-3.1-8B: 32/8 heads, head dim 128; Gemma/Qwen-style wide heads:
16/8, head dim 256; a vLLM-style paged batch); the planted sinks, heavy
hitters and drift stand in for real prompts, which are not used.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np
import torch

# Method hyper-parameters shared by every workload: coarse block b, pooling
# group g, attention tile T, sink tiles, local band (tiles before the
# diagonal), stride-rescue period eta.
COMMON = dict(block=128, group=64, tile=64, n_sink=1, n_local=2, eta=16)

WORKLOADS = {
    # 2K, 4 query / 2 KV heads, head dim 64: small enough for a full oracle run.
    "tiny_2k": dict(seqlens=[2048], h_q=4, h_kv=2, head_dim=64, seed=0,
                    gamma=0.9, rho=0.0, drift=0.0),
    # Llama-3.1-8B-shaped layer at 32K.
    "llama_32k": dict(seqlens=[32768], h_q=32, h_kv=8, head_dim=128, seed=1,
                      gamma=0.9, rho=0.0, drift=0.0),
    # Same layer at 128K; all rescues on (stride and random, rho = 0.1).
    "llama_128k": dict(seqlens=[131072], h_q=32, h_kv=8, head_dim=128, seed=2,
                       gamma=0.9, rho=0.1, drift=0.0),
    # Gemma/Qwen-style wide heads at 64K with positional drift.
    "wide_64k": dict(seqlens=[65536], h_q=16, h_kv=8, head_dim=256, seed=3,
                     gamma=0.9, rho=0.0, drift=0.5),
    # vLLM-style paged batch of four requests, 16-token pages.
    "paged_4x": dict(seqlens=[16384, 32768, 65536, 131072], h_q=40, h_kv=8,
                     head_dim=128, seed=4, gamma=0.9, rho=0.1, drift=0.0,
                     page_size=16),
}


@dataclasses.dataclass
class Sequence:
    """One request: head-first bf16 tensors on the CPU."""
    q: torch.Tensor  # [h_q, n, C]
    k: torch.Tensor  # [h_kv, n, C]
    v: torch.Tensor  # [h_kv, n, C]


def draw_sequence(rng: np.random.Generator, n: int, h_q: int, h_kv: int,
                  head_dim: int, *, beta: float = 3.0, hh_frac: float = 0.01,
                  hh_amp: float = 3.0, sink_amp: float = 4.0, n_sinks: int = 4,
                  drift: float = 0.0, drift_period: int = 8192) -> Sequence:
    """Draw one request with the planted structure described in the module doc."""
    if h_q % h_kv:
        raise ValueError("h_q must be a multiple of h_kv")
    m = h_q // h_kv
    c = head_dim
    d = rng.standard_normal((h_kv, c))
    d /= np.linalg.norm(d, axis=1, keepdims=True)
    q = rng.standard_normal((h_q, n, c), dtype=np.float32)
    k = rng.standard_normal((h_kv, n, c), dtype=np.float32)
    v = rng.standard_normal((h_kv, n, c), dtype=np.float32)
    n_hh = int(round(hh_frac * n))
    lo = min(n_sinks, n)
    for h in range(h_kv):
        if n_hh > 0 and n - lo >= n_hh:
            pos = rng.choice(np.arange(lo, n), size=n_hh, replace=False)
            k[h, pos] += np.float32(hh_amp) * d[h].astype(np.float32)
    for p in range(h_q):
        q[p] += np.float32(beta) * d[p // m].astype(np.float32)
    if drift != 0.0:
        t = np.arange(n, dtype=np.float64)
        w = (drift * np.cos(2.0 * math.pi * t / drift_period)).astype(np.float32)
        for h in range(h_kv):
            k[h] += w[:, None] * d[h].astype(np.float32)[None, :]
    for h in range(h_kv):
        mean = q[h * m:(h + 1) * m].astype(np.float64).mean(axis=(0, 1))
        u = mean / np.linalg.norm(mean)
        k[h, :min(n_sinks, n)] = (sink_amp * u).astype(np.float32)
    to_bf16 = lambda a: torch.from_numpy(a).to(torch.bfloat16)
    return Sequence(q=to_bf16(q), k=to_bf16(k), v=to_bf16(v))


@dataclasses.dataclass
class Workload:
    name: str
    seqlens: List[int]
    h_q: int
    h_kv: int
    head_dim: int
    seed: int
    gamma: float
    rho: float
    drift: float
    block: int
    group: int
    tile: int
    n_sink: int
    n_local: int
    eta: int
    page_size: Optional[int] = None

    @property
    def batch(self) -> int:
        return len(self.seqlens)


def workload(name: str, **overrides) -> Workload:
    spec = dict(COMMON)
    spec.update(WORKLOADS[name])
    spec.update(overrides)
    return Workload(name=name, **spec)


def make_inputs(wl: Workload, seqlens: Optional[List[int]] = None) -> List[Sequence]:
    """Draw every request of a workload (optionally with other lengths)."""
    lens = list(seqlens if seqlens is not None else wl.seqlens)
    if len(lens) == 1:
        rngs = [np.random.Generator(np.random.PCG64(wl.seed))]
    else:
        rngs = [np.random.Generator(np.random.PCG64([wl.seed, s]))
                for s in range(len(lens))]
    return [draw_sequence(r, n, wl.h_q, wl.h_kv, wl.head_dim, drift=wl.drift)
            for r, n in zip(rngs, lens)]


def page_table(seed: int, seqlens: List[int], page_size: int):
    """Scatter the pages of every request over one pool by a seeded permutation.

    Returns ``(block_table [B][max_pages] int32, n_pages_total)``; unused
    entries of short requests are -1.
    """
    pages = [(n + page_size - 1) // page_size for n in seqlens]
    total = int(sum(pages))
    perm = np.random.Generator(np.random.PCG64(seed)).permutation(total)
    max_pages = max(pages)
    table = np.full((len(seqlens), max_pages), -1, dtype=np.int32)
    off = 0
    for s, np_ in enumerate(pages):
        table[s, :np_] = perm[off:off + np_]
        off += np_
    return table, total


def to_paged(seqs: List[Sequence], block_table: np.ndarray, n_pages: int,
             page_size: int):
    """Scatter per-request K/V into vLLM-style pools [pages][page_size][h_kv][C]."""
    h_kv, _, c = seqs[0].k.shape
    kp = torch.zeros((n_pages, page_size, h_kv, c), dtype=torch.bfloat16)
    vp = torch.zeros_like(kp)
    for s, seq in enumerate(seqs):
        n = seq.k.shape[1]
        for pg in range((n + page_size - 1) // page_size):
            t0, t1 = pg * page_size, min(n, (pg + 1) * page_size)
            dst = int(block_table[s, pg])
            kp[dst, :t1 - t0] = seq.k[:, t0:t1].transpose(0, 1)
            vp[dst, :t1 - t0] = seq.v[:, t0:t1].transpose(0, 1)
    return kp, vp


def random_block_mask(seed: int, h_kv: int, n_q: int, n_kv: int, block: int,
                      density: float) -> np.ndarray:
    """A seeded random 0/1 block mask [h_kv][L_q][L_kv] for isolated tests of
    the tile stage (no causal clipping: the consumer must apply it)."""
    lq = (n_q + block - 1) // block
    lkv = (n_kv + block - 1) // block
    rng = np.random.Generator(np.random.PCG64(seed))
    return (rng.random((h_kv, lq, lkv)) < density).astype(np.uint8)
