"""Pins for the oracle's tile stage: expansion, band, sink, stride and random
rescue, compaction into lists."""
import os

import numpy as np
import pytest

from oracle import bfla_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_splitmix():
    with open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt")) as f:
        lines = [l.strip() for l in f if l.strip() and not l.startswith("#")]
    seed = int(lines[0].split()[1])
    return seed, [int(x) for x in lines[1:]]


def test_mix64_reproduces_published_splitmix64_outputs():
    seed, want = _golden_splitmix()
    assert O.splitmix64_stream(seed, len(want)) == want


def test_mix64_fixes_zero_and_is_injective_on_a_sample():
    assert int(O.mix64(np.uint64(0))) == 0
    x = np.arange(1, 200001, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15)
    y = O.mix64(x)
    assert np.unique(y).size == x.size


def _plain(n, b=128, T=64, **kw):
    args = dict(n_local=-1, n_sink=0, eta=0, rho=0.0, seed=0, h=0)
    args.update(kw)
    return lambda bm: O.tile_mask(bm, n, n, b, T, **args)


def test_expansion_count_closed_form():
    # rho_b = 2, N_c = 0, whole blocks: every kept off-diagonal block gives 4
    # tiles, every kept diagonal block 3 causal tiles.
    rng = np.random.default_rng(0)
    L = 24
    bm = np.tril(rng.random((L, L)) < 0.3).astype(np.uint8)
    tm = _plain(L * 128)(bm)
    diag = np.trace(bm)
    assert int(tm.sum()) == 4 * int(bm.sum()) - int(diag)
    # each kept tile comes from a kept block and is causal
    qt, kt = np.nonzero(tm)
    assert np.all(bm[qt // 2, kt // 2] == 1) and np.all(kt <= qt)


def test_band_and_sink_always_kept():
    n, T = 40 * 64 + 17, 64          # ragged tail
    bm = np.zeros((-(-n // 128), -(-n // 128)), np.uint8)
    tm = O.tile_mask(bm, n, n, 128, T, n_local=2, n_sink=1, eta=0, rho=0.0,
                     seed=0, h=0)
    for qt in range(tm.shape[0]):
        diag = qt
        want = set(range(max(0, diag - 2), diag + 1)) | {0}
        assert set(np.flatnonzero(tm[qt])) == want


def test_band_follows_diagonal_in_chunked_prefill():
    n_q, n_kv, T = 3 * 64, 10 * 64 + 5, 64
    bm = np.zeros((2, 6), np.uint8)
    tm = O.tile_mask(bm, n_q, n_kv, 128, T, n_local=1, n_sink=2, eta=0,
                     rho=0.0, seed=0, h=0)
    n_c = n_kv - n_q
    for qt in range(3):
        last = min(n_c + (qt + 1) * T - 1, n_kv - 1)
        d = last // T
        assert set(np.flatnonzero(tm[qt])) == {0, 1, d - 1, d}


def test_rescue_is_subset_of_dropped_and_rates_are_binomial():
    L = 64                                   # 128 x 128 tiles
    rng = np.random.default_rng(1)
    bm = np.tril(rng.random((L, L)) < 0.05).astype(np.uint8)
    base = O.tile_mask(bm, L * 128, L * 128, 128, 64, n_local=2, n_sink=1,
                       eta=0, rho=0.0, seed=5, h=3)
    causal = np.tril(np.ones_like(base))
    dropped = causal & ~base
    nd = dropped.sum()
    for eta, rho in [(16, 0.0), (0, 0.1), (7, 0.0), (0, 0.37)]:
        tm = O.tile_mask(bm, L * 128, L * 128, 128, 64, n_local=2, n_sink=1,
                         eta=eta, rho=rho, seed=5, h=3)
        assert np.all(tm >= base) and not np.any(tm & ~causal)
        resc = tm & ~base
        assert np.all(resc <= dropped)
        p = 1.0 / eta if eta else rho
        mean, sd = nd * p, np.sqrt(nd * p * (1 - p))
        assert abs(resc.sum() - mean) <= 5 * sd, (eta, rho, resc.sum(), mean)


def test_rescue_decision_independent_of_mass_mask_and_seeded():
    L = 32
    rng = np.random.default_rng(2)
    b1 = np.tril(rng.random((L, L)) < 0.1).astype(np.uint8)
    b2 = np.tril(rng.random((L, L)) < 0.2).astype(np.uint8)
    kw = dict(n_local=2, n_sink=1, eta=16, rho=0.1)
    t1 = O.tile_mask(b1, L*128, L*128, 128, 64, seed=9, h=1, **kw)
    t2 = O.tile_mask(b2, L*128, L*128, 128, 64, seed=9, h=1, **kw)
    e1 = O.tile_mask(b1, L*128, L*128, 128, 64, seed=9, h=1, **dict(kw, eta=0, rho=0.0))
    e2 = O.tile_mask(b2, L*128, L*128, 128, 64, seed=9, h=1, **dict(kw, eta=0, rho=0.0))
    both_dropped = np.tril(np.ones_like(t1)) & ~e1 & ~e2
    assert np.array_equal(t1 & both_dropped, t2 & both_dropped)
    # deterministic per seed, different across seeds and heads
    t1b = O.tile_mask(b1, L*128, L*128, 128, 64, seed=9, h=1, **kw)
    assert np.array_equal(t1, t1b)
    t3 = O.tile_mask(b1, L*128, L*128, 128, 64, seed=10, h=1, **kw)
    t4 = O.tile_mask(b1, L*128, L*128, 128, 64, seed=9, h=2, **kw)
    assert not np.array_equal(t1, t3) and not np.array_equal(t1, t4)
    # stride rescue carries no head index (chi(i, j; s)), random rescue does
    s1 = O.tile_mask(b1, L*128, L*128, 128, 64, seed=9, h=1, **dict(kw, rho=0.0))
    s2 = O.tile_mask(b1, L*128, L*128, 128, 64, seed=9, h=5, **dict(kw, rho=0.0))
    assert np.array_equal(s1, s2)


def test_rho_threshold_integer_compare():
    assert O.rho_threshold(0.0) == 0
    assert O.rho_threshold(1.0) == 1 << 24
    assert O.rho_threshold(0.1) == 1677721
    # psi24 is a 24-bit integer
    v = O.psi24(0, np.arange(1000)[:, None], np.arange(1000)[None, :], 3)
    assert v.max() < (1 << 24)
    assert abs(float((v < O.rho_threshold(0.25)).mean()) - 0.25) < 0.005


def test_random_rescue_threshold_is_strict():
    # eq25 rescues a dropped tile iff psi < rho: with rho set to exactly the
    # tile's psi the tile stays dropped, one step of 2^-24 above it is rescued
    n, h, seed = 3 * 64, 1, 77
    bm = np.zeros((2, 2), np.uint8)
    v = int(O.psi24(h, 2, 0, seed))
    args = dict(n_local=-1, n_sink=0, eta=0, seed=seed, h=h)
    at = O.tile_mask(bm, n, n, 128, 64, rho=v / 16777216.0, **args)
    above = O.tile_mask(bm, n, n, 128, 64, rho=(v + 1) / 16777216.0, **args)
    assert O.rho_threshold(v / 16777216.0) == v
    assert not at[2, 0] and above[2, 0]


def test_lists_are_ascending_rows_in_order():
    n = [300, 1000]
    masks = [np.tril(np.ones((3, 3), np.uint8))[None].repeat(2, 0) * 0,
             np.random.default_rng(3).integers(0, 2, (2, 8, 8)).astype(np.uint8)]
    rp, cols, tms = O.expand_rescue(masks, n, n, 128, 64, 2, 1, 16, 0.1, 4)
    t_q = [5, 16]
    assert rp.size == 2 * t_q[0] + 2 * t_q[1] + 1
    row = 0
    for r in range(2):
        for h in range(2):
            for qt in range(t_q[r]):
                c = cols[rp[row]:rp[row + 1]]
                assert np.all(np.diff(c) > 0)
                assert np.array_equal(c, np.flatnonzero(tms[r][h, qt]))
                row += 1
