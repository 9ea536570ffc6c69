"""GPU parity of every stage against the CPU oracle, through the C ABI.

Each stage is first fed the oracle's own inputs (oracle lists for the
prefill, the oracle block mask for the tile stage), so errors never
compound; then the whole pipeline runs end to end.  Bars: lists bit-exact;
block mask exact on every cell that is not a near-tie; bf16 outputs within
max-abs 2e-2 and rel-L2 5e-3 of the float64 oracle on the same lists."""
import numpy as np
import pytest
import torch

from oracle import bfla_oracle as O
from paper_2605_12193_amd import bfla, synth
from parity_util import (DeviceBatch, Guarded, GuardedBuffers, compare_outputs,
                         head_mask_compare, lists_to_device, mask_compare, oracle_lists_for)

pytestmark = pytest.mark.gpu

# (name, seqlens, n_q (None = full prefill), h_q, h_kv, C)
SHAPES = [
    ("tiny_2k", [2048], None, 4, 2, 64),
    ("ragged_1000", [1000], None, 4, 2, 64),
    ("llama_gqa4", [1536 + 37], None, 8, 2, 128),
    ("wide_c256", [700], None, 4, 2, 256),
    ("chunked", [1100], [300], 4, 2, 64),
    ("gqa5", [777], None, 10, 2, 128),
    ("mha_m1", [512 + 64 + 5], None, 2, 2, 128),
    ("gqa8", [640], None, 8, 1, 64),
    ("batch3", [900, 300, 1200], [900, 100, 1200], 4, 2, 64),
    ("gqa4_c64_chunked", [1300], [700], 8, 2, 64),
    ("gqa8_c128", [900], None, 8, 1, 128),
    ("wide_gqa4", [700], [500], 8, 2, 256),
]
IDS = [s[0] for s in SHAPES]


def _make(name, seqlens, n_q, h_q, h_kv, c, seed=0):
    wl = synth.workload("tiny_2k", h_q=h_q, h_kv=h_kv, head_dim=c, seed=seed)
    seqs = synth.make_inputs(wl, seqlens=seqlens)
    return DeviceBatch(seqs, n_q)


def _params(**kw):
    base = dict(block=128, group=64, tile=64, gamma=0.9, n_local=2, n_sink=1, eta=16,
                rho=0.1, seed=7)
    base.update(kw)
    return base, bfla.params(**base)


def _oracle_stage1(db, kw):
    out = []
    for r in range(len(db.seqs)):
        q, k, _ = db.host(r)
        out.append(O.estimate_mask(q, k, kw["block"], kw["group"], kw["gamma"],
                                   O.default_scale(db.c)))
    return out


def _check_outputs(db, row_ptr, cols, T=64, lse=None):
    for r in range(len(db.seqs)):
        q, k, v = db.host(r)
        base = sum(db.h_kv * -(-n // T) for n in db.n_q[:r])
        want, want_lse = O.attention(q, k, v, T, O.default_scale(db.c), row_ptr, cols, base)
        compare_outputs(db.o_of(r), want, f"request {r}")
        if lse is not None:
            off = sum(db.h_q * n for n in db.n_q[:r])
            got = lse[off:off + db.h_q * db.n_q[r]].reshape(db.h_q, db.n_q[r])
            np.testing.assert_allclose(got, want_lse, rtol=0, atol=2e-4)


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_dense_prefill_matches_oracle(shape):
    db = _make(*shape)
    kw, prm = _params()
    lse = torch.full((db.h_q * sum(db.n_q),), float("nan"), device="cuda")
    bfla.bfla_dense_prefill(db.prob, prm, db.qv, db.kv, db.ov, lse)
    torch.cuda.synchronize()
    lse = lse.cpu().numpy()
    for r in range(len(db.seqs)):
        q, k, v = db.host(r)
        want, want_lse = O.attention(q, k, v, 64, O.default_scale(db.c))
        compare_outputs(db.o_of(r), want, f"dense request {r}")
        off = sum(db.h_q * n for n in db.n_q[:r])
        got = lse[off:off + db.h_q * db.n_q[r]].reshape(db.h_q, db.n_q[r])
        np.testing.assert_allclose(got, want_lse, rtol=0, atol=2e-4)


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_sparse_prefill_on_oracle_lists(shape):
    db = _make(*shape)
    kw, prm = _params()
    st = _oracle_stage1(db, kw)
    rp, cols, _ = oracle_lists_for(db, [s["mask"] for s in st], kw)
    drp, dcols = lists_to_device(rp, cols)
    lse = torch.full((db.h_q * sum(db.n_q),), float("nan"), device="cuda")
    bfla.bfla_sparse_prefill(db.prob, prm, db.qv, db.kv, drp, dcols, db.ov, lse)
    torch.cuda.synchronize()
    _check_outputs(db, rp, cols, lse=lse.cpu().numpy())


def test_sparse_prefill_empty_rows_and_band_off():
    db = _make("x", [640], None, 4, 2, 64)
    kw, prm = _params(n_local=-1, n_sink=0, eta=0, rho=0.0)
    # keep nothing in half of the rows: those queries must get O = 0, lse = -inf
    masks = [np.zeros((2, 5, 5), np.uint8)]
    masks[0][0, 2:, :2] = 1
    rp, cols, _ = oracle_lists_for(db, masks, kw)
    assert np.any(np.diff(rp) == 0)
    drp, dcols = lists_to_device(rp, cols)
    lse = torch.zeros(4 * 640, device="cuda")
    bfla.bfla_sparse_prefill(db.prob, prm, db.qv, db.kv, drp, dcols, db.ov, lse)
    torch.cuda.synchronize()
    _check_outputs(db, rp, cols, lse=lse.cpu().numpy())


@pytest.mark.parametrize("cfg", [
    dict(),
    dict(n_local=-1, n_sink=0, eta=0, rho=0.0),
    dict(n_local=0, n_sink=3, eta=3, rho=0.0),
    dict(n_local=5, n_sink=1, eta=0, rho=1.0),
    dict(block=256, n_local=8, eta=16, rho=0.37, seed=123456789),
    # the stride test on the low bits of chi (eta a power of two) and by
    # division (other eta), and eta = 1 rescuing every dropped tile
    dict(n_local=0, n_sink=0, eta=1, rho=0.0),
    dict(n_local=1, eta=2, rho=0.0, seed=99),
    dict(n_local=1, eta=12, rho=0.05, seed=7),
])
@pytest.mark.parametrize("shape", [SHAPES[0], SHAPES[4], SHAPES[8]], ids=["tiny", "chunked", "batch3"])
def test_expand_rescue_bit_exact(shape, cfg):
    db = _make(*shape)
    kw, prm = _params(**cfg)
    rng = np.random.default_rng(5)
    masks = []
    for r in range(len(db.seqs)):
        lq, lkv = -(-db.n_q[r] // kw["block"]), -(-db.n_kv[r] // kw["block"])
        masks.append((rng.random((db.h_kv, lq, lkv)) < 0.3).astype(np.uint8))
    rp, cols, _ = oracle_lists_for(db, masks, kw)
    buf = bfla.Buffers(db.prob, prm)
    flat = torch.from_numpy(np.concatenate([m.ravel() for m in masks])).cuda()
    buf.block_mask[:flat.numel()].copy_(flat)
    buf.cols.fill_(-7)
    bfla.bfla_expand_rescue(db.prob, prm, buf.block_mask, buf.row_ptr, buf.cols, buf.ws_expand)
    torch.cuda.synchronize()
    got_rp = buf.row_ptr.cpu().numpy()
    assert np.array_equal(got_rp, rp)
    got_cols = buf.cols.cpu().numpy()[:rp[-1]]
    assert np.array_equal(got_cols, cols)


@pytest.mark.parametrize("shape", [SHAPES[0], SHAPES[1], SHAPES[2], SHAPES[3], SHAPES[4],
                                   SHAPES[5], SHAPES[8]],
                         ids=["tiny", "ragged", "llama", "wide", "chunked", "gqa5", "batch3"])
@pytest.mark.parametrize("gamma", [0.9, 0.5, 1.0])
def test_estimate_mask_matches_oracle(shape, gamma):
    db = _make(*shape)
    kw, prm = _params(gamma=gamma)
    st = _oracle_stage1(db, kw)
    buf = GuardedBuffers(db.prob, prm, head_mask=True)
    bfla.bfla_estimate_mask(db.prob, prm, db.qv, db.kv, buf.block_mask, dbg_scores=buf.scores,
                            dbg_head_mask=buf.head_mask, workspace=buf.ws_estimate)
    torch.cuda.synchronize()
    buf.check("estimate_mask")
    got_mask = buf.block_mask.cpu().numpy()
    got_s = buf.scores.cpu().numpy()
    got_h = buf.head_mask.cpu().numpy()
    alpha = O.default_scale(db.c)
    mo = so = 0
    ties = head_ties = 0
    for r, s in enumerate(st):
        n_m, n_s = s["mask"].size, s["scores"].size
        gm = got_mask[mo:mo + n_m].reshape(s["mask"].shape)
        gs = got_s[so:so + n_s].reshape(s["scores"].shape)
        gh = got_h[so:so + n_s].reshape(s["scores"].shape)
        mo += n_m
        so += n_s
        assert np.array_equal(np.isinf(gs), np.isinf(s["scores"]))
        fin = np.isfinite(s["scores"])
        err = np.abs(gs[fin].astype(np.float64) - s["scores"][fin]) * alpha
        assert err.max() < 1e-4, f"alpha*S error {err.max():.2e}"
        assert set(np.unique(gm)) <= {0, 1}
        ties += mask_compare(gm, s["mask"], s["status"])
        head_ties += head_mask_compare(gh, s["head_keep"], s["head_tie"], gm)
    print(f"near-tie mismatches: {ties} (per head: {head_ties})")


def test_head_mask_is_optional_and_changes_nothing():
    """The per-head output is a debug view: the block mask and scores are the
    same bit for bit with and without it, and without dbg_scores the scores
    go to the workspace, after the split score GEMM's partial sums."""
    db = _make(*SHAPES[5])
    kw, prm = _params()
    a = GuardedBuffers(db.prob, prm, head_mask=True)
    b = GuardedBuffers(db.prob, prm)
    n_ws = bfla.bfla_workspace_size(db.prob, prm, bfla.BFLA_WS_ESTIMATE)
    ws = Guarded(n_ws, torch.uint8)
    bfla.bfla_estimate_mask(db.prob, prm, db.qv, db.kv, a.block_mask, dbg_scores=a.scores,
                            dbg_head_mask=a.head_mask, workspace=a.ws_estimate)
    bfla.bfla_estimate_mask(db.prob, prm, db.qv, db.kv, b.block_mask, workspace=ws.t)
    torch.cuda.synchronize()
    a.check("with head mask")
    b.check("without")
    ws.check("estimate workspace")
    assert torch.equal(a.block_mask, b.block_mask)
    n_s = a.cap.score_elems
    in_ws = ws.t[n_ws - 4 * n_s:].view(torch.int32)
    assert torch.equal(a.scores.view(torch.int32), in_ws)


@pytest.mark.parametrize("shape", [SHAPES[0], SHAPES[2], SHAPES[4], SHAPES[8]],
                         ids=["tiny", "llama", "chunked", "batch3"])
def test_end_to_end_pipeline(shape):
    db = _make(*shape)
    kw, prm = _params()
    buf = GuardedBuffers(db.prob, prm)
    bfla.bfla_estimate_mask(db.prob, prm, db.qv, db.kv, buf.block_mask, dbg_scores=buf.scores,
                            workspace=buf.ws_estimate)
    torch.cuda.synchronize()
    buf.check("estimate_mask")
    bfla.bfla_expand_rescue(db.prob, prm, buf.block_mask, buf.row_ptr, buf.cols, buf.ws_expand)
    torch.cuda.synchronize()
    buf.check("expand_rescue")
    _host_check_lists(db, buf)
    bfla.bfla_sparse_prefill(db.prob, prm, db.qv, db.kv, buf.row_ptr, buf.cols, db.ov, buf.lse)
    torch.cuda.synchronize()
    buf.check("sparse_prefill")
    db.o_guard.check("sparse_prefill O")
    # lists == oracle tile stage applied to the GPU's own block mask
    gm = buf.block_mask.cpu().numpy()
    masks, off = [], 0
    for r in range(len(db.seqs)):
        lq, lkv = -(-db.n_q[r] // 128), -(-db.n_kv[r] // 128)
        masks.append(gm[off:off + db.h_kv * lq * lkv].reshape(db.h_kv, lq, lkv))
        off += db.h_kv * lq * lkv
    rp, cols, _ = oracle_lists_for(db, masks, kw)
    assert np.array_equal(buf.row_ptr.cpu().numpy(), rp)
    assert np.array_equal(buf.cols.cpu().numpy()[:rp[-1]], cols)
    # the GPU mask agrees with the oracle's on every sure cell
    st = _oracle_stage1(db, kw)
    for r, s in enumerate(st):
        mask_compare(masks[r], s["mask"], s["status"])
    _check_outputs(db, rp, cols, lse=buf.lse.cpu().numpy())


def _host_check_lists(db, buf, T=64):
    """Lists produced on the GPU are well formed before a kernel reads them."""
    rp = buf.row_ptr.cpu().numpy()
    assert rp[0] == 0 and np.all(np.diff(rp) >= 0) and rp[-1] <= buf.cols.numel()
    cols = buf.cols.cpu().numpy()[:rp[-1]]
    row = 0
    for r in range(len(db.seqs)):
        t_kv = -(-db.n_kv[r] // T)
        n_rows = db.h_kv * -(-db.n_q[r] // T)
        seg = cols[rp[row]:rp[row + n_rows]]
        assert np.all((seg >= 0) & (seg < t_kv))
        row += n_rows


def test_runs_are_bit_identical():
    db = _make(*SHAPES[2])
    kw, prm = _params()
    outs = []
    for _ in range(2):
        buf = bfla.Buffers(db.prob, prm)
        db.o.fill_(0)
        bfla.bfla_estimate_mask(db.prob, prm, db.qv, db.kv, buf.block_mask, dbg_scores=buf.scores,
                                workspace=buf.ws_estimate)
        bfla.bfla_expand_rescue(db.prob, prm, buf.block_mask, buf.row_ptr, buf.cols,
                                buf.ws_expand)
        torch.cuda.synchronize()
        _host_check_lists(db, buf)
        bfla.bfla_sparse_prefill(db.prob, prm, db.qv, db.kv, buf.row_ptr, buf.cols, db.ov,
                                 buf.lse)
        torch.cuda.synchronize()
        n = int(buf.row_ptr[-1])
        outs.append((db.o.clone(), buf.block_mask.clone(), buf.row_ptr.clone(),
                     buf.cols[:n].clone(), buf.scores.clone(), buf.lse.clone()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)
