"""The PyTorch drop-in on the GPU: outputs against the oracle, an all-keep
configuration equal to the dense kernel bit for bit, buffer reuse and a
chunked call; the packed variable-length entry against the head-first
library run and the oracle, and the paged-cache entry against it."""
import numpy as np
import pytest
import torch

from oracle import bfla_oracle as O
from paper_2605_12193_amd import bfla, synth
from paper_2605_12193_amd.attention import BlockFilteredAttention
from parity_util import DeviceBatch, PagedBatch, compare_outputs

pytestmark = pytest.mark.gpu


def _qkv(batch, n, h_q, h_kv, c, seed):
    wl = synth.workload("llama_32k", h_q=h_q, h_kv=h_kv, head_dim=c, seed=seed)
    seqs = [synth.make_inputs(wl, seqlens=[n])[0] if b == 0 else
            synth.make_inputs(synth.workload("llama_32k", h_q=h_q, h_kv=h_kv, head_dim=c,
                                             seed=seed + b), seqlens=[n])[0]
            for b in range(batch)]
    q = torch.stack([s.q for s in seqs]).cuda()
    k = torch.stack([s.k for s in seqs]).cuda()
    v = torch.stack([s.v for s in seqs]).cuda()
    return seqs, q, k, v


def test_module_matches_oracle():
    seqs, q, k, v = _qkv(2, 1500, 8, 2, 128, 11)
    att = BlockFilteredAttention(gamma=0.9, rho=0.1, seed=3, return_lse=True)
    o, lse = att(q, k, v)
    torch.cuda.synchronize()
    prm = dict(block=128, group=64, tile=64, gamma=0.9, n_local=2, n_sink=1, eta=16, rho=0.1,
               seed=3)
    alpha = O.default_scale(128)
    for b, s in enumerate(seqs):
        qh, kh, vh = (x.double().numpy() for x in (s.q, s.k, s.v))
        # the lists come from the GPU mask (near-tie cells may differ); rebuild them
        # from the module's own Stage-1 output through the oracle's tile stage
        n_cells = att._buf.block_mask.numel() // 2
        mask = att._buf.block_mask[b * n_cells:(b + 1) * n_cells].cpu().numpy()
        mask = mask.reshape(2, 12, 12)
        st = O.estimate_mask(qh, kh, 128, 64, 0.9, alpha)
        keep_sure = st["status"] == O.KEEP_SURE
        drop_sure = st["status"] == O.DROP_SURE
        assert np.all(mask[keep_sure] == 1) and np.all(mask[drop_sure] == 0)
        rp, cols, _ = O.expand_rescue([mask], [1500], [1500], 128, 64, 2, 1, 16, 0.1, 3)
        want, want_lse = O.attention(qh, kh, vh, 64, alpha, rp, cols, 0)
        compare_outputs(o[b].float().cpu().numpy(), want, f"batch {b}")
        np.testing.assert_allclose(lse[b].cpu().numpy(), want_lse, rtol=0, atol=2e-4)


def test_all_keep_equals_dense_kernel():
    _, q, k, v = _qkv(1, 1300, 8, 2, 128, 5)
    att = BlockFilteredAttention(gamma=1.0, eta=0, rho=0.0)
    o = att(q, k, v)
    prob = bfla.Problem([1300], [1300], 8, 2, 128)
    od = torch.empty_like(q)
    bfla.bfla_dense_prefill(prob, bfla.params(), bfla.view_hnc(q), bfla.KV(k, v),
                            bfla.view_hnc(od))
    torch.cuda.synchronize()
    assert torch.equal(o, od)


def test_buffers_reused_and_chunked_call():
    _, q, k, v = _qkv(1, 1200, 4, 2, 64, 9)
    att = BlockFilteredAttention()
    o1 = att(q, k, v)
    buf = att._buf
    o2 = att(q, k, v)
    torch.cuda.synchronize()
    assert att._buf is buf and torch.equal(o1, o2)
    # chunked: the last 300 queries against all 1200 keys
    qc = q[:, :, 900:].contiguous()
    oc = att(qc, k, v)
    torch.cuda.synchronize()
    assert att._buf is not buf and oc.shape == qc.shape
    s = synth.make_inputs(synth.workload("llama_32k", h_q=4, h_kv=2, head_dim=64, seed=9),
                          seqlens=[1200])[0]
    qh, kh, vh = (x.double().numpy() for x in (s.q, s.k, s.v))
    qh = qh[:, 900:]
    alpha = O.default_scale(64)
    mask = att._buf.block_mask.cpu().numpy().reshape(2, 3, 10)
    rp, cols, _ = O.expand_rescue([mask], [300], [1200], 128, 64, 2, 1, 16, 0.0, 0)
    want, _ = O.attention(qh, kh, vh, 64, alpha, rp, cols, 0)
    compare_outputs(oc[0].float().cpu().numpy(), want, "chunked")


def _packed_requests(n_kv, n_q, h_q, h_kv, c):
    wl = synth.workload("paged_4x", seqlens=n_kv, h_q=h_q, h_kv=h_kv, head_dim=c)
    seqs = synth.make_inputs(wl)
    q = torch.cat([s.q[:, s.q.shape[1] - nq:].transpose(0, 1) for s, nq in zip(seqs, n_q)])
    k = torch.cat([s.k.transpose(0, 1) for s in seqs])
    v = torch.cat([s.v.transpose(0, 1) for s in seqs])
    cu_q = np.concatenate([[0], np.cumsum(n_q)]).tolist()
    cu_k = np.concatenate([[0], np.cumsum(n_kv)]).tolist()
    return seqs, q.contiguous().cuda(), k.contiguous().cuda(), v.contiguous().cuda(), cu_q, cu_k


VARLEN = ([700, 1500, 900], [700, 1500, 200], 8, 2, 128)   # the third request is chunked


def test_varlen_matches_head_first_batch_and_oracle():
    n_kv, n_q, h_q, h_kv, c = VARLEN
    seqs, q, k, v, cu_q, cu_k = _packed_requests(n_kv, n_q, h_q, h_kv, c)
    att = BlockFilteredAttention(gamma=0.9, rho=0.1, seed=3, return_lse=True)
    o, lses = att.forward_varlen(q, k, v, cu_q, cu_k)
    torch.cuda.synchronize()
    assert o.shape == q.shape and len(lses) == 3
    # the same requests head-first through the library: bit for bit
    db = DeviceBatch(seqs, n_q)
    prm = bfla.params(gamma=0.9, rho=0.1, seed=3)
    buf = bfla.Buffers(db.prob, prm)
    bfla.sparse_pass(db.prob, prm, db.qv, db.kv, db.ov, buf)
    torch.cuda.synchronize()
    assert torch.equal(att._varlen.buf.block_mask, buf.block_mask)
    for r in range(3):
        got = o[cu_q[r]:cu_q[r + 1]].transpose(0, 1).float().cpu().numpy()
        assert np.array_equal(got, db.o_of(r))
    # and the oracle on the module's own mask
    mask = att._varlen.buf.block_mask.cpu().numpy()
    alpha, off, masks = O.default_scale(c), 0, []
    for r, s in enumerate(seqs):
        lq, lkv = -(-n_q[r] // 128), -(-n_kv[r] // 128)
        masks.append(mask[off:off + h_kv * lq * lkv].reshape(h_kv, lq, lkv))
        off += h_kv * lq * lkv
    rp, cols, _ = O.expand_rescue(masks, n_q, n_kv, 128, 64, 2, 1, 16, 0.1, 3)
    base = 0
    for r, s in enumerate(seqs):
        qh = s.q[:, n_kv[r] - n_q[r]:].double().numpy()
        want, want_lse = O.attention(qh, s.k.double().numpy(), s.v.double().numpy(), 64, alpha,
                                     rp, cols, base)
        base += h_kv * -(-n_q[r] // 64)
        got = o[cu_q[r]:cu_q[r + 1]].transpose(0, 1).float().cpu().numpy()
        compare_outputs(got, want, f"varlen request {r}")
        np.testing.assert_allclose(lses[r].cpu().numpy(), want_lse, rtol=0, atol=2e-4)


def test_paged_cache_equals_varlen():
    n_kv, n_q, h_q, h_kv, c = VARLEN
    seqs, q, k, v, cu_q, cu_k = _packed_requests(n_kv, n_q, h_q, h_kv, c)
    att = BlockFilteredAttention(gamma=0.9, rho=0.1, seed=3)
    o_var = att.forward_varlen(q, k, v, cu_q, cu_k)
    pb = PagedBatch(seqs, n_q, page_size=16, seed=5)
    assert torch.equal(pb.q, q)
    o_pg = att.forward_paged(pb.q, pb.kp, pb.vp, pb.table, n_kv, torch.tensor(cu_q))
    o_again = att.forward_paged(pb.q, pb.kp, pb.vp, pb.table, n_kv, cu_q)
    torch.cuda.synchronize()
    assert torch.equal(o_pg, o_var) and torch.equal(o_again, o_pg)
