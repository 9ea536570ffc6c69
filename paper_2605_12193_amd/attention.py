"""Drop-in block-filtered sparse causal prefill attention for PyTorch.

`BlockFilteredAttention` (a torch.nn.Module) and `block_filtered_attention`
take bf16 Q [B, H_q, N_q, C] and K, V [B, H_kv, N_kv, C] (or the same without
the batch dimension) and return the causal prefill output O, shaped like Q,
computed by the method of Sec. 3: Stage 1 block scores and keep-mass
selection (eq9-eq18) with the GQA union, the tile expansion with the sink,
local-band and rescue rules (eq19-eq26), and exact attention restricted to
the retained tiles (eq27).  N_q < N_kv is a chunked prefill: the queries are
the last N_q positions of the sequence.

Every step runs in the library's HIP kernels, enqueued on the current torch
stream; this module only checks shapes, keeps the device buffers of the last
shape and passes pointers.
"""
from typing import Optional, Tuple

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


def block_filtered_attention(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, **kw):
    """One call of `BlockFilteredAttention(**kw)` (buffers are not kept)."""
    return BlockFilteredAttention(**kw)(q, k, v)
