"""Pins for the oracle's attention (eq27 sparse, eq:vsa dense) and for the
whole oracle pipeline."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import bfla_oracle as O
from paper_2605_12193_amd import synth


def _qkv(seed, h_q, h_kv, n_q, n_kv, c):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((h_q, n_q, c))
    k = rng.standard_normal((h_kv, n_kv, c))
    v = rng.standard_normal((h_kv, n_kv, c))
    return q, k, v


def _sdpa(q, k, v, allowed, scale):
    """Library attention in float64 with an explicit boolean mask [H_q, N_q, N_kv]."""
    h_q, h_kv = q.shape[0], k.shape[0]
    m = h_q // h_kv
    kk = torch.from_numpy(np.repeat(k, m, axis=0))
    vv = torch.from_numpy(np.repeat(v, m, axis=0))
    return F.scaled_dot_product_attention(torch.from_numpy(q), kk, vv,
                                          attn_mask=torch.from_numpy(allowed),
                                          scale=scale).numpy()


def _allowed_from_lists(rp, cols, h_q, h_kv, n_q, n_kv, T, row_base=0):
    m = h_q // h_kv
    n_c = n_kv - n_q
    t_q = -(-n_q // T)
    allowed = np.zeros((h_q, n_q, n_kv), bool)
    for p in range(h_q):
        for qt in range(t_q):
            r = row_base + (p // m) * t_q + qt
            for kt in cols[rp[r]:rp[r + 1]]:
                allowed[p, qt * T:(qt + 1) * T, kt * T:(kt + 1) * T] = True
    pos = n_c + np.arange(n_q)
    allowed &= np.arange(n_kv)[None, None, :] <= pos[None, :, None]
    return allowed


@pytest.mark.parametrize("n_q,n_kv", [(200, 200), (130, 330), (64, 64)])
def test_dense_matches_library_sdpa(n_q, n_kv):
    q, k, v = _qkv(0, 4, 2, n_q, n_kv, 16)
    scale = 0.25
    o, lse = O.attention(q, k, v, 32, scale)
    pos = (n_kv - n_q) + np.arange(n_q)
    allowed = np.broadcast_to(np.arange(n_kv)[None, :] <= pos[:, None], (4, n_q, n_kv))
    np.testing.assert_allclose(o, _sdpa(q, k, v, allowed.copy(), scale), rtol=1e-10, atol=1e-12)
    if n_q == n_kv:
        ref = F.scaled_dot_product_attention(
            torch.from_numpy(q), torch.from_numpy(np.repeat(k, 2, 0)),
            torch.from_numpy(np.repeat(v, 2, 0)), is_causal=True, scale=scale).numpy()
        np.testing.assert_allclose(o, ref, rtol=1e-10, atol=1e-12)
    # LSE: log-sum-exp of the admissible scaled logits
    m = 2
    logits = scale * np.einsum("pqc,pkc->pqk", q, np.repeat(k, m, 0))
    ref_lse = torch.logsumexp(torch.from_numpy(np.where(allowed, logits, -np.inf)), -1).numpy()
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-12, atol=1e-12)


def test_sparse_matches_library_sdpa_with_explicit_mask():
    n, T = 512 + 40, 32
    q, k, v = _qkv(1, 6, 3, n, n, 8)
    bms = [np.random.default_rng(2).integers(0, 2, (3, 9, 9)).astype(np.uint8)]
    rp, cols, _ = O.expand_rescue(bms, [n], [n], 64, T, 1, 1, 5, 0.2, 7)
    scale = 0.3
    o, _ = O.attention(q, k, v, T, scale, rp, cols)
    allowed = _allowed_from_lists(rp, cols, 6, 3, n, n, T)
    np.testing.assert_allclose(o, _sdpa(q, k, v, allowed, scale), rtol=1e-10, atol=1e-12)


def _pipeline(q, k, v, b, g, T, gamma, n_local, n_sink, eta, rho, seed):
    alpha = O.default_scale(q.shape[-1])
    st = O.estimate_mask(q, k, b, g, gamma, alpha)
    n_q, n_kv = q.shape[1], k.shape[1]
    rp, cols, _ = O.expand_rescue([st["mask"]], [n_q], [n_kv], b, T, n_local,
                                  n_sink, eta, rho, seed)
    return O.attention(q, k, v, T, alpha, rp, cols), (rp, cols, st)


def test_gamma_one_reproduces_dense():
    seq = synth.make_inputs(synth.workload("tiny_2k"), seqlens=[700])[0]
    q, k, v = (x.double().numpy() for x in (seq.q, seq.k, seq.v))
    (o, lse), _ = _pipeline(q, k, v, 128, 64, 64, 1.0, 2, 1, 0, 0.0, 0)
    od, lsed = O.attention(q, k, v, 64, O.default_scale(64))
    np.testing.assert_allclose(o, od, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, lsed, rtol=1e-12, atol=1e-12)


def test_convex_combination_row0_and_future_independence():
    seq = synth.make_inputs(synth.workload("tiny_2k"), seqlens=[600])[0]
    q, k, v = (x.double().numpy() for x in (seq.q, seq.k, seq.v))
    (o, _), (rp, cols, _) = _pipeline(q, k, v, 128, 64, 64, 0.8, 1, 1, 16, 0.1, 3)
    allowed = _allowed_from_lists(rp, cols, 4, 2, 600, 600, 64)
    vv = np.repeat(v, 2, 0)
    for p in range(4):
        for t in range(0, 600, 37):
            sel = vv[p, allowed[p, t]]
            assert np.all(o[p, t] <= sel.max(0) + 1e-12)
            assert np.all(o[p, t] >= sel.min(0) - 1e-12)
        # row 0 attends only to key 0
        np.testing.assert_allclose(o[p, 0], vv[p, 0], rtol=0, atol=1e-12)
    # perturbing keys/values after position 300 leaves rows <= 300 unchanged
    k2, v2 = k.copy(), v.copy()
    k2[:, 301:] += 5.0
    v2[:, 301:] -= 3.0
    o2, _ = O.attention(q, k2, v2, 64, O.default_scale(64), rp, cols)
    np.testing.assert_array_equal(o2[:, :301], o[:, :301])


def test_dropped_tiles_do_not_matter():
    n, T = 640, 64
    q, k, v = _qkv(4, 2, 1, n, n, 16)
    bm = [np.tril(np.random.default_rng(5).integers(0, 2, (1, 5, 5))).astype(np.uint8)]
    rp, cols, tms = O.expand_rescue(bm, [n], [n], 128, T, 0, 1, 0, 0.0, 0)
    o, _ = O.attention(q, k, v, T, 0.25, rp, cols)
    qt = 9
    row = cols[rp[qt]:rp[qt + 1]]
    drop = [kt for kt in range(qt + 1) if kt not in set(row.tolist())]
    assert drop, "need a dropped tile"
    k2, v2 = k.copy(), v.copy()
    for kt in drop:
        k2[:, kt * T:(kt + 1) * T] = 100.0
        v2[:, kt * T:(kt + 1) * T] = -100.0
    o2, _ = O.attention(q, k2, v2, T, 0.25, rp, cols)
    np.testing.assert_array_equal(o2[:, qt * T:(qt + 1) * T], o[:, qt * T:(qt + 1) * T])


def test_empty_row_gives_zero_and_minus_inf():
    n, T = 256, 64
    q, k, v = _qkv(6, 1, 1, n, n, 8)
    rp = np.array([0, 1, 1, 2, 3], np.int32)     # q-tile 1 keeps nothing
    cols = np.array([0, 2, 3], np.int32)
    o, lse = O.attention(q, k, v, T, 0.3, rp, cols)
    assert np.all(o[0, 64:128] == 0) and np.all(np.isneginf(lse[0, 64:128]))


def test_dual_stage_error_bound_holds():
    """Appendix bound: ||O - O_s||_F <= (||D^-1 D_s - I||_F ||Z||_F +
    ||Z - Z_s||_F) ||A||_F ||V||_F, A = D_s^-1 exp(QK^T / sqrt(C))."""
    n, c, T = 256, 16, 32
    q, k, v = _qkv(8, 1, 1, n, n, c)
    q *= 0.5
    bm = [np.tril(np.random.default_rng(9).integers(0, 2, (1, 4, 4))).astype(np.uint8)]
    rp, cols, _ = O.expand_rescue(bm, [n], [n], 64, T, 0, 1, 0, 0.0, 0)
    scale = 1 / np.sqrt(c)
    o, _ = O.attention(q, k, v, T, scale, rp, cols)
    o_s, _ = O.attention(q, k, v, T, scale)
    z = _allowed_from_lists(rp, cols, 1, 1, n, n, T)[0].astype(np.float64)
    z_s = np.tril(np.ones((n, n)))
    e = np.exp(scale * q[0] @ k[0].T)
    d = (e * z).sum(1)
    d_s = (e * z_s).sum(1)
    a = e / d_s[:, None]
    alpha = np.linalg.norm(np.diag(d_s / d) - np.eye(n)) * np.linalg.norm(z) \
        + np.linalg.norm(z - z_s)
    lhs = np.linalg.norm(o[0] - o_s[0])
    assert lhs > 0
    assert lhs <= alpha * np.linalg.norm(a) * np.linalg.norm(v[0])


def test_default_scale_is_the_library_default():
    # alpha = 1/sqrt(C) (eq15, eq27) is also scaled-dot-product attention's
    # default scale: the oracle with its default equals the library without one
    q, k, v = _qkv(21, 2, 2, 48, 48, 16)
    o, _ = O.attention(q, k, v, 16, O.default_scale(16))
    ref = F.scaled_dot_product_attention(torch.from_numpy(q), torch.from_numpy(k),
                                         torch.from_numpy(v), is_causal=True).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-10, atol=1e-12)
