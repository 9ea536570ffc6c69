"""Pins for the oracle's Stage 1 (block scores, causal mask, block softmax,
keep-mass selection, GQA union) against independent computations."""
import itertools

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

from oracle import bfla_oracle as O


def _rand(seed, *shape):
    return np.random.default_rng(seed).standard_normal(shape)


def trace_scores(q, k, b, g):
    """Independent block scores: the full QK^T from a library float64 matmul;
    each group pair scores the trace of its g x g sub-block (only real
    tokens: zero padding adds nothing); fully padded groups are skipped;
    causal pairs are found by brute force over token pairs."""
    n_q, n_kv = q.shape[0], k.shape[0]
    qk = (torch.from_numpy(q).double() @ torch.from_numpy(k).double().T).numpy()
    n_c = n_kv - n_q
    lq, lkv, G = -(-n_q // b), -(-n_kv // b), b // g
    s = np.full((lq, lkv), -np.inf)
    for i in range(lq):
        for j in range(lkv):
            qs = np.arange(i * b, min(n_q, (i + 1) * b))
            ks = np.arange(j * b, min(n_kv, (j + 1) * b))
            if not (ks[:, None] <= n_c + qs[None, :]).any():
                continue
            best = -np.inf
            for u in range(G):
                for v in range(G):
                    r0, c0 = i * b + u * g, j * b + v * g
                    if r0 >= n_q or c0 >= n_kv:
                        continue
                    tr = sum(qk[r0 + t, c0 + t] for t in range(g)
                             if r0 + t < n_q and c0 + t < n_kv)
                    best = max(best, tr)
            s[i, j] = best
    return s


@pytest.mark.parametrize("n_q,n_kv,c,b,g", [
    (64, 64, 4, 16, 4),        # whole blocks, G = 4
    (50, 50, 3, 16, 8),        # ragged tail: partial and fully padded groups
    (40, 72, 5, 16, 4),        # chunked prefill, N_c = 32
    (33, 97, 2, 8, 2),         # chunked, ragged both sides
])
def test_block_scores_equal_subblock_traces(n_q, n_kv, c, b, g):
    q, k = _rand(1, n_q, c), _rand(2, n_kv, c)
    got = O.block_scores(q, k, b, g)
    want = trace_scores(q, k, b, g)
    assert np.array_equal(np.isinf(got), np.isinf(want))
    fin = np.isfinite(want)
    np.testing.assert_allclose(got[fin], want[fin], rtol=1e-12, atol=1e-10)


def test_g1_is_blockwise_max_of_qk():
    q, k = _rand(3, 48, 6), _rand(4, 48, 6)
    b = 16
    got = O.block_scores(q, k, b, 1)
    qk = q @ k.T
    for i in range(3):
        for j in range(3):
            if j > i:
                assert got[i, j] == -np.inf
            else:
                # g = 1: groups are single tokens -> max over the b x b block
                assert np.isclose(got[i, j], qk[i*b:(i+1)*b, j*b:(j+1)*b].max(), rtol=1e-12)


def test_g_equals_b_is_full_block_trace():
    q, k = _rand(5, 64, 3), _rand(6, 64, 3)
    b = 32
    got = O.block_scores(q, k, b, b)
    qk = q @ k.T
    for i in range(2):
        for j in range(i + 1):
            assert np.isclose(got[i, j], np.trace(qk[i*b:(i+1)*b, j*b:(j+1)*b]), rtol=1e-12)


@pytest.mark.parametrize("lq", [1, 2, 7, 16, 1024])
def test_causal_block_count_closed_form(lq):
    b = 128
    m = O.causal_block_mask(lq * b, lq * b, b)
    assert m.sum() == lq * (lq + 1) // 2
    assert np.array_equal(m, np.tril(np.ones((lq, lq), bool)))


def test_causal_block_mask_chunked_matches_token_brute_force():
    b = 8
    for n_q, n_kv in [(8, 24), (13, 29), (1, 17), (24, 24), (5, 5)]:
        m = O.causal_block_mask(n_q, n_kv, b)
        n_c = n_kv - n_q
        for i in range(m.shape[0]):
            for j in range(m.shape[1]):
                qs = np.arange(i * b, min(n_q, (i + 1) * b)) + n_c
                ks = np.arange(j * b, min(n_kv, (j + 1) * b))
                assert m[i, j] == bool((ks[:, None] <= qs[None, :]).any())


def test_block_probs_sum_to_one_and_match_library_softmax():
    rng = np.random.default_rng(7)
    s = (rng.standard_normal((50, 40)) * 80).astype(np.float32)
    s[:, 30:] = -np.inf
    alpha = 1 / np.sqrt(128)
    a = O.block_probs(s, alpha)
    np.testing.assert_allclose(a.astype(np.float64).sum(axis=1), 1.0, atol=2e-6)
    assert np.all(a[:, 30:] == 0)
    ref = torch.softmax(torch.from_numpy(s[:, :30].astype(np.float64)) * alpha, dim=1).numpy()
    # float32 against float64: well inside the 1e-5 near-tie band (measured 3.2e-6)
    np.testing.assert_allclose(a[:, :30], ref, rtol=4e-6, atol=1e-37)
    # adding a constant to a row leaves the probabilities unchanged
    a2 = O.block_probs(s + np.float32(64.0), alpha)
    np.testing.assert_allclose(a2, a, rtol=1e-5, atol=1e-7)


def test_block_probs_scale_enters_linearly():
    # alpha doubles -> logits double: A(2 alpha, S) == A(alpha, 2 S)
    s = (np.random.default_rng(9).standard_normal((4, 9)) * 10).astype(np.float32)
    a1 = O.block_probs(s, 0.25)
    a2 = O.block_probs(2 * s, 0.125)
    np.testing.assert_allclose(a1, a2, rtol=1e-6, atol=1e-9)


def _brute_min_subset(a, gamma):
    """Minimum number of blocks whose float64 mass reaches gamma (exhaustive)."""
    n = len(a)
    for r in range(1, n + 1):
        best = max(sum(a[list(c)]) for c in itertools.combinations(range(n), r))
        if best >= gamma:
            return r
    return n


@settings(max_examples=60, deadline=None)
@given(seed=st.integers(0, 10_000), n=st.integers(1, 10),
       gamma=st.sampled_from([0.3, 0.5, 0.8, 0.9, 0.95, 0.99]),
       spread=st.sampled_from([1.0, 5.0, 20.0]))
def test_keep_mass_is_minimum_cardinality(seed, n, gamma, spread):
    rng = np.random.default_rng(seed)
    s = np.full((1, 12), -np.inf, np.float32)
    s[0, :n] = (rng.standard_normal(n) * spread / 0.1).astype(np.float32)
    alpha = 0.1
    keep, tie, r = O.keep_mass(s, gamma, alpha)
    if tie.any():
        return
    a = O.block_probs(s, alpha)[0, :n].astype(np.float64)
    assert r[0] == keep[0].sum()
    assert r[0] == _brute_min_subset(a, gamma)
    # the kept set is a top set: every kept mass >= every dropped mass
    kept, dropped = a[keep[0, :n]], a[~keep[0, :n]]
    if dropped.size:
        assert kept.min() >= dropped.max()
    assert kept.sum() >= gamma * (1 - 1e-6)


def test_keep_mass_limits():
    rng = np.random.default_rng(11)
    s = (rng.standard_normal((20, 16)) * 30).astype(np.float32)
    s[np.triu_indices(16, 1)[0] % 20, np.triu_indices(16, 1)[1]] = -np.inf
    causal = np.isfinite(s)
    keep1, _, _ = O.keep_mass(s, 1.0, 0.1)
    assert np.array_equal(keep1, causal)        # gamma = 1 keeps everything causal
    keep0, _, r0 = O.keep_mass(s, 1e-9, 0.1)
    assert np.all(r0 == 1)                      # gamma -> 0+ keeps exactly the argmax
    am = np.argmax(np.where(causal, s, -np.inf), axis=1)
    assert np.array_equal(np.argmax(keep0, axis=1), am)
    assert np.all(keep0.sum(axis=1) == 1)


def test_gamma_one_keeps_every_block_even_when_the_float_mass_saturates():
    # one block carries all but ~1e-43 of the mass: its float32 mass rounds to
    # 1.0, so a float running sum reaches gamma = 1 after one block; in exact
    # arithmetic only the full set reaches 1, so all four are kept
    s = np.array([[100.0, 0.0, 0.0, 0.0, -np.inf]], np.float32)
    assert O.block_probs(s, 1.0)[0, 0] == np.float32(1.0)
    keep, _, r = O.keep_mass(s, 1.0, 1.0)
    assert r[0] == 4 and keep[0].tolist() == [True, True, True, True, False]
    # just below 1 the saturated float mass already reaches gamma
    keep, _, r = O.keep_mass(s, 0.999999, 1.0)
    assert r[0] == 1


def test_keep_mass_tie_break_by_index():
    s = np.array([[5.0, 7.0, 7.0, 7.0, -np.inf]], np.float32)
    keep, tie, r = O.keep_mass(s, 0.5, 1.0)
    # three equal maxima: order (7,j=1),(7,j=2),(7,j=3); 2 of them reach 0.5
    assert r[0] == 2 and keep[0].tolist() == [False, True, True, False, False]
    assert tie[0, 1:4].all()                    # equal masses straddle the cut


def test_threshold_tie_is_flagged():
    # two blocks of mass exactly 1/2: the mass before the second one equals
    # gamma = 0.5, so its inclusion flips under any perturbation
    s = np.array([[3.0, 3.0]], np.float32)
    keep, tie, r = O.keep_mass(s, 0.5, 1.0)
    assert r[0] == 1 and tie[0, 1]


def test_gqa_union_contains_every_head_and_m1_is_identity():
    rng = np.random.default_rng(12)
    q = rng.standard_normal((4, 256, 8)) + 0.5
    k = rng.standard_normal((2, 256, 8))
    st_ = O.estimate_mask(q, k, 32, 8, 0.8, 1 / np.sqrt(8))
    for p in range(4):
        assert np.all(st_["mask"][p // 2] >= st_["head_keep"][p])
    assert np.array_equal(st_["mask"].astype(bool),
                          st_["head_keep"].reshape(2, 2, 8, 8).any(axis=1))
    st1 = O.estimate_mask(q[:2], k, 32, 8, 0.8, 1 / np.sqrt(8))
    assert np.array_equal(st1["mask"].astype(bool), st1["head_keep"])
    # the diagonal block always enters the softmax and rows are never empty
    assert np.all(st_["head_keep"].sum(axis=-1) >= 1)


def test_padded_groups_never_win_the_max_when_every_real_pair_is_negative():
    # n = 192 with b = 128, g = 64: the last block holds one real group and
    # one group that starts at n (all padding); every real group pair scores
    # -g*C, so a padded group's zero dot product must not enter the max
    c, b, g, n = 4, 128, 64, 192
    q, k = np.ones((n, c)), -np.ones((n, c))
    s = O.block_scores(q, k, b, g)
    assert np.isfinite(s).sum() == 3
    assert np.all(s[np.isfinite(s)] == -g * c)
    # the same with a chunked prefix: 64 queries after 128 keys
    s = O.block_scores(q[:64], k, b, g)
    assert np.all(s[np.isfinite(s)] == -g * c)


def test_unreached_threshold_keeps_every_block():
    # the float32 masses of this row add up to 0.99999994 in keep order; a
    # gamma below 1 whose float32 rounding is 1 is never reached, and then
    # every causal block is kept (eq17 has no shorter prefix)
    s = np.array([[-1.3, 0.7, -np.inf]], np.float32)
    a = O.block_probs(s, 1.0)
    assert np.float32(a[0, 1]) + np.float32(a[0, 0]) < np.float32(1.0)
    gamma = 1.0 - 2.0 ** -26
    assert gamma < 1.0 and np.float32(gamma) == np.float32(1.0)
    keep, _, r = O.keep_mass(s, gamma, 1.0)
    assert r[0] == 2 and keep[0].tolist() == [True, True, False]


def test_gamma_is_compared_in_float32():
    # reading R16: the running mass and gamma are both float32; a gamma a
    # hair above the first block's float32 mass (same float32 value) is
    # reached by that block alone, while a float64 comparison would take two
    s = np.array([[-1.3, 0.7]], np.float32)
    a0 = float(O.block_probs(s, 1.0)[0, 1])
    gamma = a0 + 1e-9
    assert np.float32(gamma) == np.float32(a0) and gamma > a0
    _, _, r = O.keep_mass(s, gamma, 1.0)
    assert r[0] == 1


def test_threshold_tie_band_is_one_part_in_1e5():
    # two blocks, alpha = 1: the mass before the second block is a0; gamma a
    # relative 3e-6 above a0 puts the second block inside the near-tie band,
    # 3e-5 above leaves it a sure keep
    s = np.array([[1.0, 0.0]], np.float32)
    a0 = float(O.block_probs(s, 1.0)[0, 0])
    _, tie, r = O.keep_mass(s, a0 * (1 + 3e-6), 1.0)
    assert r[0] == 2 and tie[0, 1]
    _, tie, r = O.keep_mass(s, a0 * (1 + 3e-5), 1.0)
    assert r[0] == 2 and not tie[0].any()


def test_a_cell_kept_only_as_a_near_tie_is_not_sure():
    # b = g = 1, C = 1: block scores are q_i * k_j.  Query 3 of head 0 scores
    # [5, 3, 3, 0]: at gamma 0.85 it keeps block 0 and, of the two equal 3s,
    # block 1 (index order); head 1 scores [-5, -3, -3, 0] and keeps block 3
    # alone.  Block 1 of the union is kept only through an order tie: the
    # smallest change to k[2] moves it to block 2, so neither is sure.
    q = np.array([[[1.0], [1.0], [1.0], [1.0]], [[-1.0], [-1.0], [-1.0], [-1.0]]])
    k = np.array([[[5.0], [3.0], [3.0], [0.0]]])
    st_ = O.estimate_mask(q, k, 1, 1, 0.85, 1.0)
    assert st_["mask"][0, 3].tolist() == [1, 1, 0, 1]
    assert st_["status"][0, 3].tolist() == [O.KEEP_SURE, O.TIE, O.TIE, O.KEEP_SURE]
    k2 = k.copy()
    k2[0, 2, 0] = 3.0 * (1 + 1e-6)
    st2 = O.estimate_mask(q, k2, 1, 1, 0.85, 1.0)
    assert st2["mask"][0, 3].tolist() == [1, 0, 1, 1]
    # every sure cell of the first call keeps its decision under the change
    sure = st_["status"] != O.TIE
    assert np.array_equal(st_["mask"][sure], st2["mask"][sure])
