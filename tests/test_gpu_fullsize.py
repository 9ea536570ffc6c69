"""GPU parity at the full workload sizes, in the launch configuration bench.py
times (same entry points, same shapes).  The oracle checks everything it can
afford at each size:

* llama_32k and wide_64k: all of Stage 1 (scores, per-head keep sets, the
  union mask) and every list, plus sampled sparse and dense output rows;
* llama_128k at gamma in {0.8, 0.9, 0.95} x rho in {0, 0.1}: sampled query
  blocks (scores, per-head keep sets, union) of two KV heads, every list of
  two KV heads, sampled output rows;
* paged_4x (four requests of 16K-128K tokens, GQA 5, 16-token pages): per
  request, sampled Stage-1 rows, every list of two KV heads, sampled output
  rows;
* b = 64 on 96K tokens: rows of up to 1536 causal blocks, beyond what the
  selection keeps in registers (1024), so its memory path runs; sampled rows
  on both sides of that limit.

Lists are compared with the oracle's tile stage applied to the GPU's own
block mask, outputs with the oracle's attention over the GPU's lists."""
import numpy as np
import pytest
import torch

from oracle import bfla_oracle as O
from paper_2605_12193_amd import bfla, synth
from parity_util import (PagedBatch, compare_outputs, head_mask_compare, mask_compare)

pytestmark = pytest.mark.gpu


def _kw(wl):
    return dict(block=wl.block, group=wl.group, tile=wl.tile, gamma=wl.gamma,
                n_local=wl.n_local, n_sink=wl.n_sink, eta=wl.eta, rho=wl.rho, seed=wl.seed)


class Contig:
    """One head-first request on the GPU with the buffers of a whole pass."""

    def __init__(self, wl, seq=None):
        self.wl = wl
        seq = seq if seq is not None else synth.make_inputs(wl)[0]
        self.q, self.k, self.v = (t.cuda().contiguous() for t in (seq.q, seq.k, seq.v))
        self.o = torch.empty_like(self.q)
        self.n = self.q.shape[1]
        self.prob = bfla.Problem([self.n], [self.n], wl.h_q, wl.h_kv, wl.head_dim)
        self.qv, self.ov, self.kv = bfla.view_hnc(self.q), bfla.view_hnc(self.o), \
            bfla.KV(self.k, self.v)
        self.host = tuple(t.float().numpy() for t in (seq.q, seq.k, seq.v))

    def run(self, **over):
        kw = _kw(self.wl)
        kw.update(over)
        prm = bfla.params(**kw)
        buf = bfla.Buffers(self.prob, prm)
        head = torch.empty(max(buf.cap.score_elems, 1), dtype=torch.uint8, device="cuda")
        bfla.bfla_estimate_mask(self.prob, prm, self.qv, self.kv, buf.block_mask,
                                dbg_scores=buf.scores, dbg_head_mask=head,
                                workspace=buf.ws_estimate)
        bfla.bfla_expand_rescue(self.prob, prm, buf.block_mask, buf.row_ptr, buf.cols,
                                buf.ws_expand)
        torch.cuda.synchronize()
        rp = buf.row_ptr.cpu().numpy()
        t_kv = -(-self.n // 64)
        cols = buf.cols[:int(rp[-1])].cpu().numpy()
        assert rp[0] == 0 and np.all(np.diff(rp) >= 0)
        assert np.all((cols >= 0) & (cols < t_kv))
        bfla.bfla_sparse_prefill(self.prob, prm, self.qv, self.kv, buf.row_ptr, buf.cols,
                                 self.ov, buf.lse)
        torch.cuda.synchronize()
        b = kw["block"]
        lq = -(-self.n // b)
        wl = self.wl
        res = dict(kw=kw, prm=prm, rp=rp, cols=cols,
                   mask=buf.block_mask.cpu().numpy().reshape(wl.h_kv, lq, lq),
                   scores=buf.scores.cpu().numpy().reshape(wl.h_q, lq, lq),
                   head=head.cpu().numpy()[:wl.h_q * lq * lq].reshape(wl.h_q, lq, lq),
                   o=self.o.float().cpu().numpy() if self.n <= 65536 else None)
        return res


def check_stage1_rows(q, k, m, kw, alpha, mask, scores, head, rows):
    """Stage 1 of sampled (KV head, query block) rows: query block i of the m
    heads of KV head h against its causal prefix of keys, through the oracle;
    scores within 1e-4 in alpha S, union exact on sure cells, per-head keep
    sets exact on their non-tie cells, nothing kept past the diagonal."""
    b, g, gamma = kw["block"], kw["group"], kw["gamma"]
    n = q.shape[1]
    ties = 0
    for h, i in rows:
        qb = q[h * m:(h + 1) * m, i * b:min(n, (i + 1) * b)].astype(np.float64)
        kb = k[h:h + 1, :min(n, (i + 1) * b)].astype(np.float64)
        st = O.estimate_mask(qb, kb, b, g, gamma, alpha)
        w = st["mask"].shape[2]
        ties += mask_compare(mask[h, i:i + 1, :w][None], st["mask"], st["status"])
        ties += head_mask_compare(head[h * m:(h + 1) * m, i:i + 1, :w], st["head_keep"],
                                  st["head_tie"], mask[h, i:i + 1, :w][None])
        assert not mask[h, i, w:].any() and not head[h * m:(h + 1) * m, i, w:].any()
        gs = scores[h * m:(h + 1) * m, i, :w].astype(np.float64)
        assert np.abs(gs - st["scores"][:, 0]).max() * alpha < 1e-4
    return ties


def check_lists(mask, n, kw, rp, cols, heads, row_base=0, h_kv=None):
    """Every list of the given KV heads equals the oracle's tile stage
    (eq19-eq26) applied to the GPU block mask."""
    t_q = -(-n // 64)
    for h in heads:
        tm = O.tile_mask(mask[h], n, n, kw["block"], 64, kw["n_local"], kw["n_sink"],
                         kw["eta"], kw["rho"], kw["seed"], h)
        for qt in range(t_q):
            r = row_base + h * t_q + qt
            assert np.array_equal(cols[rp[r]:rp[r + 1]], np.flatnonzero(tm[qt])), (h, qt)


def check_rows_out(host, m, alpha, get_rows, rp, cols, rows, what, row_base=0, dense=False):
    """Sampled output rows (all m query heads of (h, qt)) against the oracle's
    attention over the GPU lists (or every causal key when dense)."""
    q, k, v = host
    t_q = -(-q.shape[1] // 64)
    got_all, want_all = [], []
    for h, qt in rows:
        r = row_base + h * t_q + qt
        tiles = None if dense else cols[rp[r]:rp[r + 1]]
        for pp in range(m):
            p = h * m + pp
            want, _ = O.attention_rows(q, k, v, p, qt, 64, alpha, tiles)
            got_all.append(get_rows(p, qt * 64, qt * 64 + want.shape[0]))
            want_all.append(want)
    return compare_outputs(np.concatenate(got_all), np.concatenate(want_all), what)


def sample_rows(rng, h_kv, t_q, count):
    return [(int(h), int(qt)) for h, qt in zip(rng.integers(0, h_kv, count),
                                               np.linspace(0, t_q - 1, count).astype(int))]


def _full_stage1_and_lists(wl, c, res):
    """All of Stage 1 and every list of a single request against the oracle."""
    q, k, _ = c.host
    alpha = O.default_scale(wl.head_dim)
    st = O.estimate_mask(q.astype(np.float64), k.astype(np.float64), wl.block, wl.group,
                         res["kw"]["gamma"], alpha)
    fin = np.isfinite(st["scores"])
    assert np.array_equal(np.isfinite(res["scores"]), fin)
    err = np.abs(res["scores"][fin].astype(np.float64) - st["scores"][fin]) * alpha
    assert err.max() < 1e-4
    ties = mask_compare(res["mask"], st["mask"], st["status"])
    head_ties = head_mask_compare(res["head"], st["head_keep"], st["head_tie"], res["mask"])
    kw = res["kw"]
    want_rp, want_cols, _ = O.expand_rescue([res["mask"]], [c.n], [c.n], kw["block"], 64,
                                            kw["n_local"], kw["n_sink"], kw["eta"], kw["rho"],
                                            kw["seed"])
    assert np.array_equal(res["rp"], want_rp) and np.array_equal(res["cols"], want_cols)
    print(f"{wl.name}: near-tie mismatches {ties} (per head {head_ties}); "
          f"kept {want_rp[-1]} tiles", flush=True)


def test_llama_32k_all_masks_and_lists_sampled_outputs():
    wl = synth.workload("llama_32k")
    c = Contig(wl)
    res = c.run()
    _full_stage1_and_lists(wl, c, res)
    m = wl.h_q // wl.h_kv
    alpha = O.default_scale(wl.head_dim)
    rng = np.random.default_rng(0)
    rows = sample_rows(rng, wl.h_kv, c.n // 64, 24)
    o = res["o"]
    get = lambda oo: (lambda p, a, b: oo[p, a:b])
    check_rows_out(c.host, m, alpha, get(o), res["rp"], res["cols"], rows, "32K sparse rows")
    # dense on a few rows, in the same launch configuration
    od = torch.empty_like(c.o)
    bfla.bfla_dense_prefill(c.prob, res["prm"], c.qv, c.kv, bfla.view_hnc(od))
    torch.cuda.synchronize()
    check_rows_out(c.host, m, alpha, get(od.float().cpu().numpy()), None, None, rows[::4],
                   "32K dense rows", dense=True)


def test_wide_64k_all_masks_and_lists_sampled_outputs():
    # head dim 256, GQA 2, positional drift: the 16-query ping-pong kernel
    wl = synth.workload("wide_64k")
    c = Contig(wl)
    res = c.run()
    _full_stage1_and_lists(wl, c, res)
    m = wl.h_q // wl.h_kv
    alpha = O.default_scale(wl.head_dim)
    rng = np.random.default_rng(4)
    rows = sample_rows(rng, wl.h_kv, c.n // 64, 16)
    get = lambda oo: (lambda p, a, b: oo[p, a:b])
    check_rows_out(c.host, m, alpha, get(res["o"]), res["rp"], res["cols"], rows,
                   "wide 64K sparse rows")
    od = torch.empty_like(c.o)
    bfla.bfla_dense_prefill(c.prob, res["prm"], c.qv, c.kv, bfla.view_hnc(od))
    torch.cuda.synchronize()
    check_rows_out(c.host, m, alpha, get(od.float().cpu().numpy()), None, None, rows[::4],
                   "wide 64K dense rows", dense=True)


@pytest.fixture(scope="module")
def llama_128k():
    wl = synth.workload("llama_128k")
    return wl, Contig(wl)


@pytest.mark.parametrize("gamma,rho", [(0.8, 0.0), (0.8, 0.1), (0.9, 0.0), (0.9, 0.1),
                                       (0.95, 0.0), (0.95, 0.1)])
def test_llama_128k_sampled(llama_128k, gamma, rho):
    wl, c = llama_128k
    res = c.run(gamma=gamma, rho=rho)
    q, k, _ = c.host
    n, m = c.n, wl.h_q // wl.h_kv
    alpha = O.default_scale(wl.head_dim)
    rng = np.random.default_rng(int(gamma * 100) + int(rho * 10))
    lq = n // wl.block
    rows = [(h, int(i)) for h in (0, 5) for i in list(rng.integers(0, lq, 5)) + [lq - 1]]
    ties = check_stage1_rows(q, k, m, res["kw"], alpha, res["mask"], res["scores"],
                             res["head"], rows)
    check_lists(res["mask"], n, res["kw"], res["rp"], res["cols"], heads=(2, 7))
    orows = sample_rows(rng, wl.h_kv, n // 64, 16)
    o = c.o
    get = lambda p, a, b: o[p, a:b].float().cpu().numpy()
    err = check_rows_out(c.host, m, alpha, get, res["rp"], res["cols"], orows,
                         f"128K gamma {gamma} rho {rho} sparse rows")
    causal = wl.h_kv * (n // 64) * (n // 64 + 1) // 2
    print(f"128K gamma {gamma} rho {rho}: keep {res['rp'][-1] / causal:.4f}, near-tie "
          f"mismatches {ties}, max-abs {err[0]:.2e} rel-L2 {err[1]:.2e}", flush=True)


def test_llama_128k_dense_sampled(llama_128k):
    # the dense baseline at the headline size, in its launch configuration:
    # sampled rows (early, middle, last q-tiles) against the oracle over every
    # causal key
    wl, c = llama_128k
    m = wl.h_q // wl.h_kv
    alpha = O.default_scale(wl.head_dim)
    od = torch.empty_like(c.o)
    bfla.bfla_dense_prefill(c.prob, bfla.params(**_kw(wl)), c.qv, c.kv, bfla.view_hnc(od))
    torch.cuda.synchronize()
    t_q = c.n // 64
    rows = [(0, 0), (3, t_q // 3), (6, t_q // 2 + 7), (7, t_q - 1)]
    get = lambda p, a, b: od[p, a:b].float().cpu().numpy()
    check_rows_out(c.host, m, alpha, get, None, None, rows, "128K dense rows", dense=True)


def test_paged_4x_per_request():
    wl = synth.workload("paged_4x")
    seqs = synth.make_inputs(wl)
    n = [s.q.shape[1] for s in seqs]
    pb = PagedBatch(seqs, n, page_size=wl.page_size, seed=wl.seed)
    kw = _kw(wl)
    prm = bfla.params(**kw)
    buf = bfla.Buffers(pb.prob, prm)
    head = torch.empty(buf.cap.score_elems, dtype=torch.uint8, device="cuda")
    bfla.bfla_estimate_mask(pb.prob, prm, pb.qv, pb.kv, buf.block_mask, dbg_scores=buf.scores,
                            dbg_head_mask=head, workspace=buf.ws_estimate)
    bfla.bfla_expand_rescue(pb.prob, prm, buf.block_mask, buf.row_ptr, buf.cols, buf.ws_expand)
    torch.cuda.synchronize()
    rp = buf.row_ptr.cpu().numpy()
    cols = buf.cols[:int(rp[-1])].cpu().numpy()
    assert rp[0] == 0 and np.all(np.diff(rp) >= 0)
    bfla.bfla_sparse_prefill(pb.prob, prm, pb.qv, pb.kv, buf.row_ptr, buf.cols, pb.ov, buf.lse)
    torch.cuda.synchronize()
    pb.o_guard.check("paged_4x O")
    gm, gs, gh = (t.cpu().numpy() for t in (buf.block_mask, buf.scores, head))
    m = wl.h_q // wl.h_kv
    alpha = O.default_scale(wl.head_dim)
    rng = np.random.default_rng(9)
    moff = soff = row_base = 0
    for r, s in enumerate(seqs):
        nr = n[r]
        lq, t_q = nr // wl.block, nr // 64
        mask = gm[moff:moff + wl.h_kv * lq * lq].reshape(wl.h_kv, lq, lq)
        scores = gs[soff:soff + wl.h_q * lq * lq].reshape(wl.h_q, lq, lq)
        heads = gh[soff:soff + wl.h_q * lq * lq].reshape(wl.h_q, lq, lq)
        host = tuple(t.float().numpy() for t in (s.q, s.k, s.v))
        rows = [(h, int(i)) for h in (1, 6) for i in list(rng.integers(0, lq, 3)) + [lq - 1]]
        ties = check_stage1_rows(host[0], host[1], m, kw, alpha, mask, scores, heads, rows)
        check_lists(mask, nr, kw, rp, cols, heads=(0, 4), row_base=row_base)
        a = int(pb.starts[r])
        get = lambda p, t0, t1, a=a: pb.o[a + t0:a + t1, p].float().cpu().numpy()
        orows = sample_rows(rng, wl.h_kv, t_q, 16)
        err = check_rows_out(host, m, alpha, get, rp, cols, orows,
                             f"paged request {r} ({nr} tokens) sparse rows", row_base=row_base)
        print(f"paged request {r}: {nr} tokens, near-tie mismatches {ties}, "
              f"max-abs {err[0]:.2e} rel-L2 {err[1]:.2e}", flush=True)
        moff += wl.h_kv * lq * lq
        soff += wl.h_q * lq * lq
        row_base += wl.h_kv * t_q


def test_select_memory_path_rows_beyond_1024_blocks():
    # b = g = 64 on 96K tokens: 1536 causal blocks in the last rows; the
    # selection keeps rows of up to 1024 blocks in registers and re-reads
    # longer ones from memory
    wl = synth.workload("llama_32k", seqlens=[98304], h_q=8, h_kv=2)
    c = Contig(wl)
    res = c.run(block=64, group=64, gamma=0.95, rho=0.0)
    q, k, _ = c.host
    m = wl.h_q // wl.h_kv
    alpha = O.default_scale(wl.head_dim)
    lq = c.n // 64
    rows = [(h, i) for h in (0, 1) for i in (100, 1023, 1024, 1025, 1300, lq - 1)]
    ties = check_stage1_rows(q, k, m, res["kw"], alpha, res["mask"], res["scores"],
                             res["head"], rows)
    check_lists(res["mask"], c.n, res["kw"], res["rp"], res["cols"], heads=(1,))
    print(f"b=64 96K: near-tie mismatches {ties}", flush=True)
