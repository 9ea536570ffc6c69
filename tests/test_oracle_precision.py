"""Pin of the oracle's float32 keep-mass decision against exact arithmetic.

The oracle takes the block softmax (eq15), the running mass and the
threshold test (eq16-eq17) in float32, from float64 scores rounded once.
Here an independent decision in float64 -- float64 scores, float64 softmax,
a float64 running mass summed one block at a time in the keep order (score
descending, block index ascending) -- is taken on the same rows, and every
block the oracle does not flag as a near-tie must be kept or dropped by both
alike.  The rows cover the tiny workload in full, sampled block rows of the
32K Llama-shaped layer at three thresholds, every configuration of the
paper's mask-density table (Sec. 5) on a 4.5K-token request, late rows of a
128K request at gamma = 0.999, and rows of 512 blocks with a flat block
softmax whose kept prefix holds hundreds of blocks.
"""
import numpy as np
import pytest

from oracle import bfla_oracle as O
from paper_2605_12193_amd import synth


def fp64_keep(s64: np.ndarray, gamma: float, alpha: float) -> np.ndarray:
    """Exact-arithmetic stand-in for eq15-eq18 on one row of float64 scores
    (-inf = not causal): a one-block-at-a-time float64 running mass."""
    causal = np.flatnonzero(np.isfinite(s64))
    keep = np.zeros(s64.shape, dtype=bool)
    if gamma >= 1.0:
        keep[causal] = True
        return keep
    s = s64[causal]
    mx = s.max()
    w = np.exp(alpha * (s - mx))
    a = w / w.sum()
    # s is in index order, so a stable sort on -s gives (score desc, index asc)
    order = np.argsort(-s, kind="stable")
    mass = 0.0
    for t in order:
        keep[causal[t]] = True
        mass += a[t]
        if mass >= gamma:
            break
    return keep


def check_rows(s64: np.ndarray, gamma: float, alpha: float):
    """Compare the oracle's float32 decision with the float64 one on rows of
    float64 scores [R, L]; returns (r_star per row, near-tie cells)."""
    keep, tie, r_star = O.keep_mass(s64.astype(np.float32), gamma, alpha)
    for row in range(s64.shape[0]):
        want = fp64_keep(s64[row], gamma, alpha)
        bad = np.flatnonzero((keep[row] != want) & ~tie[row])
        assert bad.size == 0, (
            f"row {row}: float32 and float64 decisions differ on non-tie blocks {bad[:8]} "
            f"(gamma {gamma}, r* {r_star[row]})")
    return r_star, int(tie.sum())


def block_rows(q, k, m, b, g, rows):
    """Float64 block scores of sampled (KV head, query block) rows: every
    query head of the group, block i against the (i + 1) b keys before its
    end (the causal prefix), returned as [rows * m, L] padded with -inf."""
    width = max(i for _, i in rows) + 1
    out = []
    for h, i in rows:
        qb = q[h * m:(h + 1) * m, i * b:(i + 1) * b]
        kb = k[h, :(i + 1) * b]
        for p in range(m):
            s = O.block_scores(qb[p], kb, b, g)[0]
            row = np.full(width, -np.inf)
            row[:s.size] = s
            out.append(row)
    return np.stack(out)


def _host(wl):
    seq = synth.make_inputs(wl)[0]
    return seq.q.double().numpy(), seq.k.double().numpy()


def test_tiny_2k_all_rows():
    wl = synth.workload("tiny_2k")
    q, k = _host(wl)
    m = wl.h_q // wl.h_kv
    alpha = O.default_scale(wl.head_dim)
    rows = []
    for p in range(wl.h_q):
        rows.append(O.block_scores(q[p], k[p // m], wl.block, wl.group))
    for gamma in (0.8, 0.9, 0.95, 0.999):
        check_rows(np.concatenate(rows), gamma, alpha)


@pytest.fixture(scope="module")
def llama_32k():
    wl = synth.workload("llama_32k")
    return wl, _host(wl)


@pytest.mark.parametrize("gamma", [0.8, 0.9, 0.95])
def test_llama_32k_sampled_rows(llama_32k, gamma):
    wl, (q, k) = llama_32k
    m = wl.h_q // wl.h_kv
    rng = np.random.default_rng(3)
    lq = q.shape[1] // wl.block
    rows = [(int(h), int(i)) for h, i in zip(rng.integers(0, wl.h_kv, 16),
                                             rng.integers(0, lq, 16))]
    rows += [(h, lq - 1) for h in range(wl.h_kv)]   # the longest rows of every KV head
    s = block_rows(q, k, m, wl.block, wl.group, rows)   # 24 x 4 = 96 rows
    check_rows(s, gamma, O.default_scale(wl.head_dim))


# (b, g, gamma) of every row of the paper's mask-density table (Sec. 5);
# n_local, rho and eta act after Stage 1
TABLE5_STAGE1 = sorted({(256, 64, 0.95), (256, 64, 0.999), (256, 64, 0.98),
                        (256, 64, 0.99), (128, 64, 0.99), (256, 256, 0.99),
                        (512, 64, 0.99), (512, 128, 0.99), (1024, 64, 0.99)})


def test_table5_configurations_on_4500_tokens():
    wl = synth.workload("llama_32k", seqlens=[4500], h_q=8, h_kv=2)
    q, k = _host(wl)
    m = wl.h_q // wl.h_kv
    alpha = O.default_scale(wl.head_dim)
    for b, g, gamma in TABLE5_STAGE1:
        rows = [O.block_scores(q[p], k[p // m], b, g) for p in range(wl.h_q)]
        check_rows(np.concatenate(rows), gamma, alpha)


def test_long_rows_with_hundreds_of_kept_blocks():
    # 128K tokens at b = 256: rows of up to 512 causal blocks; at gamma = 0.999
    # the kept prefixes of the planted-structure rows reach about 90 blocks
    wl = synth.workload("llama_128k", h_q=4, h_kv=1)
    q, k = _host(wl)
    lq = q.shape[1] // 256
    rows = [(0, i) for i in (lq - 1, lq - 2, lq - 40, lq // 2)]
    s = block_rows(q, k, 4, 256, 64, rows)
    r_real, _ = check_rows(s, 0.999, O.default_scale(wl.head_dim))
    assert r_real.max() >= 50
    # flat rows: queries scaled by 1/8 so that alpha S has unit spread; a row of
    # 512 causal blocks then keeps hundreds of them before the mass reaches gamma
    rng = np.random.default_rng(5)
    c, b, g, n = 128, 128, 64, 65536
    kk = rng.standard_normal((1, n, c))
    qq = rng.standard_normal((4, n, c)) / 8.0
    flat = block_rows(qq, kk, 4, b, g, [(0, n // b - 1), (0, n // b - 2), (0, n // (2 * b))])
    for gamma in (0.9, 0.99, 0.999):
        r_flat, _ = check_rows(flat, gamma, 1.0 / np.sqrt(c))
        if gamma == 0.999:
            assert r_flat.max() >= 300, f"longest kept prefix only {r_flat.max()} blocks"
