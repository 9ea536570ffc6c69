"""Drop-in block-filtered sparse causal prefill attention for PyTorch.

`BlockFilteredAttention` (a torch.nn.Module) and `block_filtered_attention`
take bf16 Q [B, H_q, N_q, C] and K, V [B, H_kv, N_kv, C] (or the same without
the batch dimension) and return the causal prefill output O, shaped like Q,
computed by the method of Sec. 3: Stage 1 block scores and keep-mass
selection (eq9-eq18) with the GQA union, the tile expansion with the sink,
local-band and rescue rules (eq19-eq26), and exact attention restricted to
the retained tiles (eq27).  N_q < N_kv is a chunked prefill: the queries are
the last N_q positions of the sequence.

Two more layouts take variable-length batches: `forward_varlen` (packed
token-major Q [sum N_q, H_q, C] and K, V [sum N_kv, H_kv, C] with cumulative
sequence lengths, as flash-attention's varlen interface) and `forward_paged`
(packed Q with K, V in page pools [pages, page_size, H_kv, C] addressed
through an int32 block table, as vLLM's cache).  Request r's queries are the
last N_q(r) positions of its N_kv(r) keys.

Every step runs in the library's HIP kernels, enqueued on the current torch
stream; this module only checks shapes, keeps the device buffers of the last
shape and passes pointers.
"""
from typing import List, Optional, Sequence, Tuple

import torch

from . import bfla


def _layout(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor):
    if q.dim() not in (3, 4) or k.dim() != q.dim() or v.shape != k.shape:
        raise ValueError("expected q [B, H_q, N_q, C] and k, v [B, H_kv, N_kv, C] "
                         "(or all without B)")
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dtype != torch.bfloat16:
            raise ValueError(f"{name} must be bfloat16, got {t.dtype}")
        if t.stride(-1) != 1:
            raise ValueError(f"{name} must have a contiguous last dimension")
    # the library addresses K and V with one set of strides
    if v.stride() != k.stride():
        raise ValueError(f"v strides {tuple(v.stride())} differ from k strides "
                         f"{tuple(k.stride())}")
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not t.is_cuda:
            raise ValueError(f"{name} must be on the GPU")
    batch = q.shape[0] if q.dim() == 4 else 1
    h_q, n_q, c = q.shape[-3:]
    h_kv, n_kv, c_k = k.shape[-3:]
    if (q.dim() == 4 and k.shape[0] != batch) or c_k != c:
        raise ValueError("q and k disagree on batch or head_dim")
    if h_q % h_kv:
        raise ValueError(f"H_q = {h_q} is not a multiple of H_kv = {h_kv}")
    if n_kv < n_q:
        raise ValueError(f"N_kv = {n_kv} < N_q = {n_q}")
    return batch, h_q, h_kv, n_q, n_kv, c


def _host_ints(x, name: str) -> List[int]:
    """Lengths size the launch, so they are read on the host: a sequence or a
    CPU tensor (a GPU tensor would force a synchronisation here)."""
    if isinstance(x, torch.Tensor):
        if x.is_cuda:
            raise ValueError(f"{name} must be a host sequence or CPU tensor")
        x = x.tolist()
    return [int(e) for e in x]


def _lengths(cu: Sequence[int], total: int, name: str) -> List[int]:
    if len(cu) < 2 or cu[0] != 0 or cu[-1] != total:
        raise ValueError(f"{name} must start at 0 and end at {total}, got {list(cu)}")
    n = [b - a for a, b in zip(cu[:-1], cu[1:])]
    if min(n) < 1:
        raise ValueError(f"{name} holds an empty or negative length: {n}")
    return n


def _packed(name: str, t: torch.Tensor) -> None:
    if t.dim() != 3 or t.dtype != torch.bfloat16 or not t.is_cuda or t.stride(-1) != 1:
        raise ValueError(f"{name} must be a bf16 [tokens, heads, C] GPU tensor with a "
                         "contiguous last dimension")


def _varlen_layout(q, n_q: Sequence[int], n_kv: Sequence[int], h_kv: int, c_k: int):
    _packed("q", q)
    _, h_q, c = q.shape
    if c_k != c:
        raise ValueError(f"q and k disagree on head_dim ({c} vs {c_k})")
    if h_q % h_kv:
        raise ValueError(f"H_q = {h_q} is not a multiple of H_kv = {h_kv}")
    if len(n_q) != len(n_kv):
        raise ValueError(f"{len(n_q)} query lengths for {len(n_kv)} key lengths")
    for r, (a, b) in enumerate(zip(n_q, n_kv)):
        if a > b:
            raise ValueError(f"request {r}: N_q = {a} > N_kv = {b}")
    return h_q, c


class _Pass:
    """The buffers of one (lengths, heads, C, device) shape, kept between calls."""

    def __init__(self):
        self.key = None
        self.prob: Optional[bfla.Problem] = None
        self.buf: Optional[bfla.Buffers] = None

    def get(self, prm, n_q, n_kv, h_q, h_kv, c, device):
        key = (tuple(n_q), tuple(n_kv), h_q, h_kv, c, device)
        if key != self.key:
            self.prob = bfla.Problem(list(n_q), list(n_kv), h_q, h_kv, c)
            self.buf = bfla.Buffers(self.prob, prm, device=device)
            self.key = key
        return self.prob, self.buf


def _lse_views(lse: torch.Tensor, h_q: int, n_q: Sequence[int]) -> Tuple[torch.Tensor, ...]:
    """Per-request [H_q, N_q(r)] views of the library's LSE (request r after
    the H_q * N_q of the requests before it)."""
    out, off = [], 0
    for n in n_q:
        out.append(lse[off:off + h_q * n].view(h_q, n))
        off += h_q * n
    return tuple(out)


class BlockFilteredAttention(torch.nn.Module):
    """Sparse causal prefill attention with BFLA's block filter.

    Parameters follow the method's notation: block b, flattening group g,
    keep-mass threshold gamma, n_local band tiles before the diagonal (-1
    turns the band off), n_sink sink tiles, stride rescue eta (0 off),
    random rescue rho (0 off) with its seed, and the softmax scale (0 means
    1/sqrt(C)).  The attention tile is 64.
    """

    def __init__(self, block: int = 128, group: int = 64, gamma: float = 0.9,
                 n_local: int = 2, n_sink: int = 1, eta: int = 16, rho: float = 0.0,
                 seed: int = 0, scale: float = 0.0, return_lse: bool = False):
        super().__init__()
        self.prm = bfla.params(block=block, group=group, tile=64, gamma=gamma,
                               n_local=n_local, n_sink=n_sink, eta=eta, rho=rho, seed=seed,
                               scale=scale)
        self.return_lse = return_lse
        self._key = None
        self._buf: Optional[bfla.Buffers] = None
        self._prob: Optional[bfla.Problem] = None
        self._varlen, self._paged = _Pass(), _Pass()

    def _pass_buffers(self, batch, h_q, h_kv, n_q, n_kv, c, device):
        key = (batch, h_q, h_kv, n_q, n_kv, c, device)
        if key != self._key:
            self._prob = bfla.Problem([n_q] * batch, [n_kv] * batch, h_q, h_kv, c)
            self._buf = bfla.Buffers(self._prob, self.prm, device=device)
            self._key = key
        return self._prob, self._buf

    def forward(self, q: torch.Tensor, k: torch.Tensor,
                v: torch.Tensor) -> torch.Tensor | Tuple[torch.Tensor, torch.Tensor]:
        batch, h_q, h_kv, n_q, n_kv, c = _layout(q, k, v)
        prob, buf = self._pass_buffers(batch, h_q, h_kv, n_q, n_kv, c, q.device)
        o = torch.empty_like(q)
        bfla.sparse_pass(prob, self.prm, bfla.view_hnc(q), bfla.KV(k, v), bfla.view_hnc(o), buf)
        if not self.return_lse:
            return o
        lse = buf.lse.view(batch, h_q, n_q).clone()
        return o, (lse if q.dim() == 4 else lse[0])

    def forward_varlen(self, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                       cu_seqlens_q, cu_seqlens_k):
        """Packed variable-length batch: q [sum N_q, H_q, C], k / v [sum N_kv,
        H_kv, C] (same strides), cu_seqlens_* the cumulative lengths (host ints,
        B + 1 of them, from 0).  Returns O like q (and, with return_lse, one
        [H_q, N_q(r)] LSE view per request)."""
        _packed("k", k)
        if v.shape != k.shape or v.stride() != k.stride():
            raise ValueError("v must have k's shape and strides")
        cq = _host_ints(cu_seqlens_q, "cu_seqlens_q")
        ck = _host_ints(cu_seqlens_k, "cu_seqlens_k")
        n_q = _lengths(cq, q.shape[0], "cu_seqlens_q")
        n_kv = _lengths(ck, k.shape[0], "cu_seqlens_k")
        h_q, c = _varlen_layout(q, n_q, n_kv, k.shape[1], k.shape[2])
        prob, buf = self._varlen.get(self.prm, n_q, n_kv, h_q, k.shape[1], c, q.device)
        o = torch.empty_like(q)
        kv = bfla.KV(k.transpose(0, 1), v.transpose(0, 1),
                     batch_offsets=[s * k.stride(0) for s in ck[:-1]])
        bfla.sparse_pass(prob, self.prm, bfla.view_packed(q, cq[:-1]), kv,
                         bfla.view_packed(o, cq[:-1]), buf)
        return (o, _lse_views(buf.lse, h_q, n_q)) if self.return_lse else o

    def forward_paged(self, q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                      block_table: torch.Tensor, seqlens_k, cu_seqlens_q):
        """Packed queries over a paged cache: q [sum N_q, H_q, C]; k_cache /
        v_cache [pages, page_size, H_kv, C] (same strides, page_size a power of
        two >= 16); block_table int32 [B, max_pages] on the GPU, row r listing
        request r's pages in order; seqlens_k the N_kv(r) and cu_seqlens_q the
        cumulative query lengths (host ints).  Returns O like q (and the LSE
        views with return_lse)."""
        if k_cache.dim() != 4 or k_cache.dtype != torch.bfloat16 or not k_cache.is_cuda:
            raise ValueError("k_cache must be a bf16 [pages, page_size, H_kv, C] GPU tensor")
        cq = _host_ints(cu_seqlens_q, "cu_seqlens_q")
        n_q = _lengths(cq, q.shape[0], "cu_seqlens_q")
        n_kv = _host_ints(seqlens_k, "seqlens_k")
        if block_table.dim() != 2 or block_table.shape[0] != len(n_kv):
            raise ValueError(f"block_table needs one row per request ({len(n_kv)})")
        h_q, c = _varlen_layout(q, n_q, n_kv, k_cache.shape[2], k_cache.shape[3])
        prob, buf = self._paged.get(self.prm, n_q, n_kv, h_q, k_cache.shape[2], c, q.device)
        o = torch.empty_like(q)
        kv = bfla.KV(k_cache, v_cache, paged=True, block_table=block_table)
        bfla.sparse_pass(prob, self.prm, bfla.view_packed(q, cq[:-1]), kv,
                         bfla.view_packed(o, cq[:-1]), buf)
        return (o, _lse_views(buf.lse, h_q, n_q)) if self.return_lse else o


def block_filtered_attention(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, **kw):
    """One call of `BlockFilteredAttention(**kw)` (buffers are not kept)."""
    return BlockFilteredAttention(**kw)(q, k, v)
