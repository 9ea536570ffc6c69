"""Degenerate and boundary inputs through the whole path against the oracle:
sequences of 1, 2 and around one tile / one block, a single query against a
long prefix, a batch of 32 requests of mixed lengths (one launch group of
request descriptors), and batches of 40 and 70 requests that every kernel
runs as several launch groups (contiguous and paged K/V)."""
import numpy as np
import pytest
import torch

from oracle import bfla_oracle as O
from paper_2605_12193_amd import bfla, synth
from parity_util import (DeviceBatch, GuardedBuffers, PagedBatch, compare_outputs,
                         head_mask_compare, mask_compare, oracle_lists_for)

pytestmark = pytest.mark.gpu

KW = dict(block=128, group=64, tile=64, gamma=0.9, n_local=2, n_sink=1, eta=16, rho=0.1,
          seed=11)


def _run(seqlens, n_q=None, h_q=4, h_kv=2, c=64, seed=0, page_size=None):
    wl = synth.workload("tiny_2k", h_q=h_q, h_kv=h_kv, head_dim=c, seed=seed)
    seqs = synth.make_inputs(wl, seqlens=seqlens)
    if page_size is None:
        db = DeviceBatch(seqs, n_q)
    else:
        db = PagedBatch(seqs, n_q if n_q is not None else seqlens, page_size, seed)
        s0 = seqs
        db.h_q, db.h_kv, db.c = h_q, h_kv, c
        db.host = lambda r: (s0[r].q[:, s0[r].q.shape[1] - db.n_q[r]:].double().numpy(),
                             s0[r].k.double().numpy(), s0[r].v.double().numpy())
    prm = bfla.params(**KW)
    buf = GuardedBuffers(db.prob, prm, head_mask=True)
    bfla.bfla_estimate_mask(db.prob, prm, db.qv, db.kv, buf.block_mask, dbg_scores=buf.scores,
                            dbg_head_mask=buf.head_mask, workspace=buf.ws_estimate)
    torch.cuda.synchronize()
    buf.check("estimate_mask")
    bfla.bfla_expand_rescue(db.prob, prm, buf.block_mask, buf.row_ptr, buf.cols, buf.ws_expand)
    torch.cuda.synchronize()
    buf.check("expand_rescue")
    rp_gpu = buf.row_ptr.cpu().numpy()
    assert rp_gpu[0] == 0 and np.all(np.diff(rp_gpu) >= 0) and rp_gpu[-1] <= buf.cols.numel()
    bfla.bfla_sparse_prefill(db.prob, prm, db.qv, db.kv, buf.row_ptr, buf.cols, db.ov, buf.lse)
    torch.cuda.synchronize()
    buf.check("sparse_prefill")
    db.o_guard.check("sparse_prefill O")
    alpha = O.default_scale(c)
    gm_all = buf.block_mask.cpu().numpy()
    gh_all = buf.head_mask.cpu().numpy()
    masks, off, hoff = [], 0, 0
    for r in range(len(seqs)):
        q, k, _ = db.host(r)
        st = O.estimate_mask(q, k, KW["block"], KW["group"], KW["gamma"], alpha)
        gm = gm_all[off:off + st["mask"].size].reshape(st["mask"].shape)
        gh = gh_all[hoff:hoff + st["scores"].size].reshape(st["scores"].shape)
        off += st["mask"].size
        hoff += st["scores"].size
        mask_compare(gm, st["mask"], st["status"])
        head_mask_compare(gh, st["head_keep"], st["head_tie"], gm)
        masks.append(gm)
    rp, cols, _ = oracle_lists_for(db, masks, KW)
    assert np.array_equal(rp_gpu, rp)
    assert np.array_equal(buf.cols.cpu().numpy()[:rp[-1]], cols)
    lse = buf.lse.cpu().numpy()
    lse_off = 0
    for r in range(len(seqs)):
        q, k, v = db.host(r)
        base = sum(db.h_kv * -(-n // 64) for n in db.n_q[:r])
        want, want_lse = O.attention(q, k, v, 64, alpha, rp, cols, base)
        compare_outputs(db.o_of(r), want, f"request {r} of {len(seqs)}")
        got = lse[lse_off:lse_off + h_q * db.n_q[r]].reshape(h_q, db.n_q[r])
        lse_off += h_q * db.n_q[r]
        np.testing.assert_allclose(got, want_lse, rtol=0, atol=2e-4)
    # the dense kernel on the same batch
    db.o.fill_(float("nan"))
    bfla.bfla_dense_prefill(db.prob, prm, db.qv, db.kv, db.ov)
    torch.cuda.synchronize()
    db.o_guard.check("dense_prefill O")
    for r in range(len(seqs)):
        q, k, v = db.host(r)
        want, _ = O.attention(q, k, v, 64, alpha)
        compare_outputs(db.o_of(r), want, f"dense request {r} of {len(seqs)}")


# (C, H_q) with two KV heads: C = 256 with GQA 2 runs the 16-query ping-pong
# kernel; GQA 1 and 5 the 16-query kernel over whole and quarter q-tiles
SHAPES = [(64, 4), (256, 4), (256, 2), (256, 10)]
SHAPE_IDS = ["c64", "c256_gqa2", "c256_gqa1", "c256_gqa5"]


@pytest.mark.parametrize("c,h_q", SHAPES, ids=SHAPE_IDS)
@pytest.mark.parametrize("n", [1, 2, 63, 64, 65, 127, 128, 129])
def test_short_sequences(n, c, h_q):
    _run([n], h_q=h_q, c=c)


@pytest.mark.parametrize("c,h_q", [(64, 8), (128, 8)] + SHAPES[1:],
                         ids=["c64", "c128"] + SHAPE_IDS[1:])
def test_single_query_after_long_prefix(c, h_q):
    _run([1000], n_q=[1], h_q=h_q, h_kv=2, c=c)


@pytest.mark.parametrize("c,h_q", SHAPES, ids=SHAPE_IDS)
def test_max_batch_of_32_requests(c, h_q):
    rng = np.random.default_rng(3)
    seqlens = [int(x) for x in rng.integers(1, 700, size=32)]
    n_q = [max(1, int(n * f)) for n, f in zip(seqlens, rng.uniform(0.3, 1.0, size=32))]
    _run(seqlens, n_q=n_q, h_q=h_q, c=c)


@pytest.mark.parametrize("c,h_q", [(64, 4), (128, 8)], ids=["c64", "c128_gqa4"])
def test_batch_of_70_requests_spans_three_launch_groups(c, h_q):
    rng = np.random.default_rng(7)
    seqlens = [int(x) for x in rng.integers(1, 500, size=70)]
    n_q = [max(1, int(n * f)) for n, f in zip(seqlens, rng.uniform(0.3, 1.0, size=70))]
    _run(seqlens, n_q=n_q, h_q=h_q, c=c)


def test_paged_batch_of_40_requests_gqa5():
    # the paged workload's shape (GQA 5, head dim 128, 16-token pages) over
    # two launch groups of request descriptors
    rng = np.random.default_rng(8)
    seqlens = [int(x) for x in rng.integers(1, 700, size=40)]
    _run(seqlens, h_q=10, h_kv=2, c=128, page_size=16)
