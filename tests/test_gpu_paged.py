"""vLLM-style paged K/V (16-token pages scattered by a seeded block table) with a
packed token-major Q/O batch: the paged run must equal the contiguous run of
the same requests bit for bit (block masks, lists, O, LSE) and match the
oracle."""
import numpy as np
import pytest
import torch

from oracle import bfla_oracle as O
from paper_2605_12193_amd import bfla, synth
from parity_util import DeviceBatch, PagedBatch, compare_outputs, mask_compare

pytestmark = pytest.mark.gpu


SHAPES = [
    # (seqlens, n_q, h_q, h_kv, C)
    ([700, 1500, 333], [700, 1500, 333], 10, 2, 128),      # GQA 5 as in the paged workload
    ([1200, 900], [1200, 200], 8, 2, 128),                 # a chunked request (prefix in cache)
    ([1000, 513], [1000, 513], 4, 2, 64),
]


@pytest.mark.parametrize("shape", SHAPES, ids=["gqa5", "chunked", "c64"])
def test_paged_equals_contiguous_and_oracle(shape):
    seqlens, n_q, h_q, h_kv, c = shape
    wl = synth.workload("paged_4x", seqlens=seqlens, h_q=h_q, h_kv=h_kv, head_dim=c)
    seqs = synth.make_inputs(wl)
    pb = PagedBatch(seqs, n_q, wl.page_size, wl.seed)
    db = DeviceBatch(seqs, n_q)
    prm = bfla.params(block=wl.block, group=wl.group, tile=wl.tile, gamma=wl.gamma,
                      n_local=wl.n_local, n_sink=wl.n_sink, eta=wl.eta, rho=wl.rho,
                      seed=wl.seed)
    outs = []
    for b in (pb, db):
        buf = bfla.Buffers(b.prob, prm)
        bfla.bfla_estimate_mask(b.prob, prm, b.qv, b.kv, buf.block_mask, dbg_scores=buf.scores,
                                workspace=buf.ws_estimate)
        bfla.bfla_expand_rescue(b.prob, prm, buf.block_mask, buf.row_ptr, buf.cols,
                                buf.ws_expand)
        torch.cuda.synchronize()
        rp = buf.row_ptr.cpu().numpy()
        assert rp[0] == 0 and np.all(np.diff(rp) >= 0)
        bfla.bfla_sparse_prefill(b.prob, prm, b.qv, b.kv, buf.row_ptr, buf.cols, b.ov, buf.lse)
        torch.cuda.synchronize()
        outs.append(dict(mask=buf.block_mask.cpu().numpy(), scores=buf.scores.cpu().numpy(),
                         rp=rp, cols=buf.cols[:int(rp[-1])].cpu().numpy(),
                         lse=buf.lse.cpu().numpy(),
                         o=[b.o_of(r) for r in range(len(seqs))]))
    p, d = outs
    for key in ("mask", "scores", "rp", "cols", "lse"):
        assert np.array_equal(p[key], d[key], equal_nan=True), key
    for r in range(len(seqs)):
        assert np.array_equal(p["o"][r], d["o"][r])
    # oracle: Stage 1 per request on sure cells, lists, outputs
    alpha = O.default_scale(c)
    off = 0
    masks = []
    for r, s in enumerate(seqs):
        qh = s.q[:, s.q.shape[1] - n_q[r]:].double().numpy()
        kh = s.k.double().numpy()
        st = O.estimate_mask(qh, kh, wl.block, wl.group, wl.gamma, alpha)
        gm = p["mask"][off:off + st["mask"].size].reshape(st["mask"].shape)
        off += st["mask"].size
        mask_compare(gm, st["mask"], st["status"])
        masks.append(gm)
    rp, cols, _ = O.expand_rescue(masks, n_q, seqlens, wl.block, wl.tile, wl.n_local,
                                  wl.n_sink, wl.eta, wl.rho, wl.seed)
    assert np.array_equal(rp, p["rp"]) and np.array_equal(cols, p["cols"])
    base = 0
    for r, s in enumerate(seqs):
        qh = s.q[:, s.q.shape[1] - n_q[r]:].double().numpy()
        want, _ = O.attention(qh, s.k.double().numpy(), s.v.double().numpy(), wl.tile, alpha,
                              rp, cols, base)
        base += h_kv * -(-n_q[r] // wl.tile)
        compare_outputs(p["o"][r], want, f"paged request {r}")


def test_paged_dense_equals_contiguous():
    seqlens, n_q, h_q, h_kv, c = SHAPES[0]
    wl = synth.workload("paged_4x", seqlens=seqlens, h_q=h_q, h_kv=h_kv, head_dim=c)
    seqs = synth.make_inputs(wl)
    pb = PagedBatch(seqs, n_q, wl.page_size, wl.seed)
    db = DeviceBatch(seqs, n_q)
    prm = bfla.params()
    for b in (pb, db):
        bfla.bfla_dense_prefill(b.prob, prm, b.qv, b.kv, b.ov)
    torch.cuda.synchronize()
    alpha = O.default_scale(c)
    for r, s in enumerate(seqs):
        assert np.array_equal(pb.o_of(r), db.o_of(r))
        want, _ = O.attention(s.q.double().numpy(), s.k.double().numpy(), s.v.double().numpy(),
                              64, alpha)
        compare_outputs(pb.o_of(r), want, f"paged dense request {r}")


def test_paged_stage1_with_wide_groups():
    # b = g = 256 over 16-token pages: one score tile's keys (128 groups of
    # 256 tokens) span 2048 pages, the most the paged score kernel resolves
    # for the paper's widest group; masks and scores equal the contiguous
    # run bit for bit and the oracle on sure cells
    n, h_q, h_kv, c = 33000, 2, 1, 64
    wl = synth.workload("paged_4x", seqlens=[n], h_q=h_q, h_kv=h_kv, head_dim=c)
    seqs = synth.make_inputs(wl)
    pb = PagedBatch(seqs, [n], 16, wl.seed)
    db = DeviceBatch(seqs, [n])
    prm = bfla.params(block=256, group=256, gamma=0.95)
    got = []
    for b in (pb, db):
        buf = bfla.Buffers(b.prob, prm)
        bfla.bfla_estimate_mask(b.prob, prm, b.qv, b.kv, buf.block_mask, dbg_scores=buf.scores,
                                workspace=buf.ws_estimate)
        torch.cuda.synchronize()
        got.append((buf.block_mask.cpu().numpy(), buf.scores.cpu().numpy()))
    assert np.array_equal(got[0][0], got[1][0])
    assert np.array_equal(got[0][1], got[1][1], equal_nan=True)
    s = seqs[0]
    st = O.estimate_mask(s.q.double().numpy(), s.k.double().numpy(), 256, 256, 0.95,
                         O.default_scale(c))
    mask_compare(got[0][0][:st["mask"].size].reshape(st["mask"].shape), st["mask"],
                 st["status"])


def test_out_of_range_table_entries_read_as_zeros():
    # A block-table entry outside [0, n_pages) reads as zeros in every kernel:
    # the paged run with such entries equals, bit for bit, the contiguous run
    # whose K/V rows of those pages are zero (Stage 1 scores and masks, tile
    # lists, sparse and dense outputs, LSE), and the sparse output matches
    # the oracle on the zeroed inputs.  Bad pages sit in the first, a middle
    # and the last (partial) tile, and one spans a whole 64-key tile.
    seqlens, n_q, h_q, h_kv, c = [700, 333], [700, 333], 10, 2, 128
    wl = synth.workload("paged_4x", seqlens=seqlens, h_q=h_q, h_kv=h_kv, head_dim=c)
    seqs = synth.make_inputs(wl)
    pb = PagedBatch(seqs, n_q, 16, wl.seed)
    n_pages = int(pb.kp.shape[0])
    bad = {0: {0: -1, 17: n_pages, 20: n_pages + 5, 21: -7, 22: 2 ** 30, 23: -(2 ** 31), 43: n_pages},
           1: {5: -1, 20: n_pages + 1}}
    table = pb.table.cpu().numpy()
    zeroed = []
    for r, s in enumerate(seqs):
        k, v = s.k.clone(), s.v.clone()
        for page, val in bad[r].items():
            assert page * 16 < seqlens[r]
            table[r, page] = val
            k[:, page * 16:(page + 1) * 16] = 0
            v[:, page * 16:(page + 1) * 16] = 0
        zeroed.append(synth.Sequence(q=s.q, k=k, v=v))
    pb.table.copy_(torch.from_numpy(table))
    db = DeviceBatch(zeroed, n_q)
    prm = bfla.params(block=wl.block, group=wl.group, tile=wl.tile, gamma=wl.gamma,
                      n_local=wl.n_local, n_sink=wl.n_sink, eta=wl.eta, rho=wl.rho,
                      seed=wl.seed)
    outs = []
    for b in (pb, db):
        buf = bfla.Buffers(b.prob, prm)
        bfla.bfla_estimate_mask(b.prob, prm, b.qv, b.kv, buf.block_mask, dbg_scores=buf.scores,
                                workspace=buf.ws_estimate)
        bfla.bfla_expand_rescue(b.prob, prm, buf.block_mask, buf.row_ptr, buf.cols,
                                buf.ws_expand)
        bfla.bfla_sparse_prefill(b.prob, prm, b.qv, b.kv, buf.row_ptr, buf.cols, b.ov, buf.lse)
        torch.cuda.synchronize()
        rp = buf.row_ptr.cpu().numpy()
        sparse = [b.o_of(r) for r in range(len(seqs))]
        bfla.bfla_dense_prefill(b.prob, prm, b.qv, b.kv, b.ov)
        torch.cuda.synchronize()
        outs.append(dict(mask=buf.block_mask.cpu().numpy(), scores=buf.scores.cpu().numpy(),
                         rp=rp, cols=buf.cols[:int(rp[-1])].cpu().numpy(),
                         lse=buf.lse.cpu().numpy(), sparse=sparse,
                         dense=[b.o_of(r) for r in range(len(seqs))]))
    p, d = outs
    for key in ("mask", "scores", "rp", "cols", "lse"):
        assert np.array_equal(p[key], d[key], equal_nan=True), key
    for r in range(len(seqs)):
        assert np.array_equal(p["sparse"][r], d["sparse"][r]), f"sparse request {r}"
        assert np.array_equal(p["dense"][r], d["dense"][r]), f"dense request {r}"
    alpha = O.default_scale(c)
    base = 0
    for r, s in enumerate(zeroed):
        want, _ = O.attention(s.q.double().numpy(), s.k.double().numpy(), s.v.double().numpy(),
                              wl.tile, alpha, p["rp"], p["cols"], base)
        base += h_kv * -(-n_q[r] // wl.tile)
        compare_outputs(p["sparse"][r], want, f"request {r} with bad pages")
