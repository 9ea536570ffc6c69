"""Every (head dim, GQA group) shape the prefill kernels instantiate, against
the oracle: C in {64, 128, 256} x m in 1..8.  Each runs a ragged
333-token request (five full tiles and a 13-token tail) through the sparse
prefill on the oracle's own lists and through the dense prefill.  This covers
the ping-pong shapes (m = 4, 8 at C <= 128), the two-stage shapes, the
half-tile shapes (m > 4 at C <= 128) and, at C = 256, the 16-query kernels
over whole (m <= 2), half (m = 3, 4) and quarter (m >= 5) q-tiles.  The
paged cases run the same shapes on K/V in 16-token pages with two KV heads."""
import numpy as np
import pytest
import torch

from oracle import bfla_oracle as O
from paper_2605_12193_amd import bfla, synth
from parity_util import (DeviceBatch, Guarded, PagedBatch, compare_outputs, lists_to_device,
                         oracle_lists_for)

pytestmark = pytest.mark.gpu

N = 333
CASES = [(c, m) for c in (64, 128, 256) for m in range(1, 9)]
IDS = [f"c{c}_m{m}" for c, m in CASES]


def _batch(c, m):
    wl = synth.workload("tiny_2k", h_q=m, h_kv=1, head_dim=c, seed=100 + c + m)
    return DeviceBatch(synth.make_inputs(wl, seqlens=[N]), None)


def _params():
    kw = dict(block=128, group=64, tile=64, gamma=0.9, n_local=2, n_sink=1, eta=16,
              rho=0.1, seed=5)
    return kw, bfla.params(**kw)


def _check_lse(got, want):
    np.testing.assert_allclose(got.reshape(want.shape), want, rtol=0, atol=2e-4)


@pytest.mark.parametrize("c,m", CASES, ids=IDS)
def test_sparse_shape(c, m):
    db = _batch(c, m)
    kw, prm = _params()
    q, k, v = db.host(0)
    st = O.estimate_mask(q, k, kw["block"], kw["group"], kw["gamma"], O.default_scale(c))
    rp, cols, _ = oracle_lists_for(db, [st["mask"]], kw)
    drp, dcols = lists_to_device(rp, cols)
    lg = Guarded(m * N, torch.float32, fill=float("nan"))
    lse = lg.t
    bfla.bfla_sparse_prefill(db.prob, prm, db.qv, db.kv, drp, dcols, db.ov, lse)
    torch.cuda.synchronize()
    lg.check("sparse lse")
    db.o_guard.check("sparse O")
    want, want_lse = O.attention(q, k, v, 64, O.default_scale(c), rp, cols, 0)
    compare_outputs(db.o_of(0), want, f"sparse C={c} m={m}")
    _check_lse(lse.cpu().numpy(), want_lse)


@pytest.mark.parametrize("c,m", CASES, ids=IDS)
def test_dense_shape(c, m):
    db = _batch(c, m)
    _, prm = _params()
    lg = Guarded(m * N, torch.float32, fill=float("nan"))
    lse = lg.t
    bfla.bfla_dense_prefill(db.prob, prm, db.qv, db.kv, db.ov, lse)
    torch.cuda.synchronize()
    lg.check("dense lse")
    db.o_guard.check("dense O")
    q, k, v = db.host(0)
    want, want_lse = O.attention(q, k, v, 64, O.default_scale(c))
    compare_outputs(db.o_of(0), want, f"dense C={c} m={m}")
    _check_lse(lse.cpu().numpy(), want_lse)


PAGED_CASES = [(256, m) for m in range(1, 9)] + [(128, 1), (128, 4), (128, 5), (64, 8)]


# pages larger than a tile: a tile starts inside its page
BIG_PAGE_CASES = [(128, 4, 128), (128, 4, 256), (128, 5, 256), (64, 1, 128), (256, 2, 256),
                  (256, 3, 128), (256, 5, 256)]


@pytest.mark.parametrize("c,m", PAGED_CASES, ids=[f"c{c}_m{m}" for c, m in PAGED_CASES])
def test_paged_shape(c, m):
    _paged_case(c, m, 16)


@pytest.mark.parametrize("c,m,ps", BIG_PAGE_CASES,
                         ids=[f"c{c}_m{m}_p{p}" for c, m, p in BIG_PAGE_CASES])
def test_paged_shape_big_pages(c, m, ps):
    _paged_case(c, m, ps)


def _paged_case(c, m, page_size):
    """Sparse (oracle lists) and dense prefill on paged K/V, two KV heads."""
    wl = synth.workload("tiny_2k", h_q=2 * m, h_kv=2, head_dim=c, seed=200 + c + m)
    seqs = synth.make_inputs(wl, seqlens=[N])
    pb = PagedBatch(seqs, [N], page_size=page_size, seed=7 + m)
    kw, prm = _params()
    s = seqs[0]
    q, k, v = s.q.double().numpy(), s.k.double().numpy(), s.v.double().numpy()
    alpha = O.default_scale(c)
    masks = O.estimate_mask(q, k, kw["block"], kw["group"], kw["gamma"], alpha)["mask"]
    rp, cols, _ = O.expand_rescue([masks], [N], [N], kw["block"], kw["tile"], kw["n_local"],
                                  kw["n_sink"], kw["eta"], kw["rho"], kw["seed"])
    drp, dcols = lists_to_device(rp, cols)
    lg = Guarded(2 * m * N, torch.float32, fill=float("nan"))
    lse = lg.t
    bfla.bfla_sparse_prefill(pb.prob, prm, pb.qv, pb.kv, drp, dcols, pb.ov, lse)
    torch.cuda.synchronize()
    lg.check("paged sparse lse")
    pb.o_guard.check("paged sparse O")
    want, want_lse = O.attention(q, k, v, 64, alpha, rp, cols, 0)
    compare_outputs(pb.o_of(0), want, f"paged sparse C={c} m={m}")
    _check_lse(lse.cpu().numpy(), want_lse)
    lse.fill_(float("nan"))
    bfla.bfla_dense_prefill(pb.prob, prm, pb.qv, pb.kv, pb.ov, lse)
    torch.cuda.synchronize()
    lg.check("paged dense lse")
    pb.o_guard.check("paged dense O")
    want, want_lse = O.attention(q, k, v, 64, alpha)
    compare_outputs(pb.o_of(0), want, f"paged dense C={c} m={m}")
    _check_lse(lse.cpu().numpy(), want_lse)


# Long rows: the steady state of each schedule's tile loop (both tile
# parities, many iterations) on lists up to 40 tiles long, contiguous and
# paged; the five-wave head-dim-256 kernel stages K and V in turns.
LONG_N = 2500
LONG_CASES = [(256, 5, False), (256, 5, True), (256, 2, False), (256, 3, True), (128, 4, False),
              (128, 5, True), (64, 8, False)]


@pytest.mark.parametrize("c,m,paged", LONG_CASES,
                         ids=[f"c{c}_m{m}_{'paged' if p else 'contig'}" for c, m, p in LONG_CASES])
def test_sparse_long_rows(c, m, paged):
    wl = synth.workload("tiny_2k", h_q=2 * m, h_kv=2, head_dim=c, seed=300 + c + m)
    seqs = synth.make_inputs(wl, seqlens=[LONG_N])
    kw, prm = _params()
    s = seqs[0]
    q, k, v = s.q.double().numpy(), s.k.double().numpy(), s.v.double().numpy()
    alpha = O.default_scale(c)
    mask = O.estimate_mask(q, k, kw["block"], kw["group"], kw["gamma"], alpha)["mask"]
    rp, cols, _ = O.expand_rescue([mask], [LONG_N], [LONG_N], kw["block"], kw["tile"],
                                  kw["n_local"], kw["n_sink"], kw["eta"], kw["rho"], kw["seed"])
    assert np.diff(rp).max() >= 20
    drp, dcols = lists_to_device(rp, cols)
    b = PagedBatch(seqs, [LONG_N], page_size=16, seed=11) if paged else DeviceBatch(seqs, None)
    lg = Guarded(2 * m * LONG_N, torch.float32, fill=float("nan"))
    bfla.bfla_sparse_prefill(b.prob, prm, b.qv, b.kv, drp, dcols, b.ov, lg.t)
    torch.cuda.synchronize()
    lg.check("long-row lse")
    b.o_guard.check("long-row O")
    want, want_lse = O.attention(q, k, v, 64, alpha, rp, cols, 0)
    compare_outputs(b.o_of(0), want, f"long rows C={c} m={m} paged={paged}")
    _check_lse(lg.t.cpu().numpy(), want_lse)
