"""CPU oracle for BFLA block-filtered sparse causal prefill.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the tests, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg use it.  It shares no code with the HIP
library and imports nothing from it.

It is a plain, slow, step-by-step reading of the method in
"BFLA: Block-Filtered Long-Context Attention Mechanism" (arXiv 2605.12193).
Equations are cited by their LaTeX labels (``eq9`` ... ``eq33``); the
labelled equations eq9..eq33 are printed as (3)..(27).

Precision:
* Scores and attention are accumulated in float64 from the exact bf16 inputs
  (one library matmul per head; no blocking or reordering of the method).
* The keep-mass selection (softmax over blocks, cumulative mass, threshold
  test) is an integer decision taken from floating point; it is taken in
  float32 -- the precision the GPU kernel takes it in, since the paper fixes
  none -- starting from the float64 scores rounded once to float32.
* Blocks whose inclusion could flip under a relative perturbation of 1e-5
  are flagged as near-ties (see ``keep_mass``).

Readings of points where the paper is silent or garbled (each is repeated at
the function that applies it):
* zero padding of the last block; fully padded groups never win the max pool;
* the diagonal block keeps all group pairs (the causal mask is block level);
* alpha = 1/sqrt(C) (the scale printed with the block softmax);
* keep order = score descending, then KV block index ascending;
* gamma >= 1 keeps every causal block; if no prefix reaches gamma, all are kept;
* the per-query-head masks of a GQA group are united (OR) per KV head;
* tile expansion is clipped to the causal tile triangle;
* local band = the diagonal tile and the ``n_local`` tiles before it;
  sink = the first ``n_sink`` KV tiles;
* dropped set D = causal and not kept; final = kept OR (D and stride) OR
  (D and random);
* chi / psi use the SplitMix64 output mix (Steele, Lea and Flood, OOPSLA
  2014) of a packed (head, q-tile, kv-tile) key; see ``mix64``.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# Relative width of the near-tie band around the keep-mass threshold.
TIE_REL = 1e-5

# Union status codes for a (KV head, query block, KV block) cell.
DROP_SURE, KEEP_SURE, TIE = 0, 1, 2


def cdiv(a: int, b: int) -> int:
    return -(-a // b)


# ---------------------------------------------------------------------------
# Stage 1: block-level importance estimation (Sec. 3.2)
# ---------------------------------------------------------------------------

def kv_head_of(p: int, m: int) -> int:
    """GQA head grouping (eq8): query head p belongs to KV head floor(p / m)."""
    return p // m


def causal_block_mask(n_q: int, n_kv: int, b: int) -> np.ndarray:
    """Causal block mask (eq11-eq13).

    Query block i ends at absolute position e_i = min(N_c + (i+1) b - 1,
    N_kv - 1) with N_c = N_kv - N_q; KV block j starts at p_j = j b; the pair
    is causal iff p_j <= e_i.  Returns bool [L_q, L_kv].
    """
    n_c = n_kv - n_q
    i = np.arange(cdiv(n_q, b))[:, None]
    j = np.arange(cdiv(n_kv, b))[None, :]
    e = np.minimum(n_c + (i + 1) * b - 1, n_kv - 1)
    return (j * b) <= e


def block_scores(q_p: np.ndarray, k_h: np.ndarray, b: int, g: int) -> np.ndarray:
    """Block importance scores of one query head against its KV head.

    q_p: [N_q, C], k_h: [N_kv, C] (any float dtype; computed in float64).
    Steps: zero-pad to whole blocks (eq5); split each block into G = b/g
    groups and flatten each group into a g*C vector (eq6-eq7); group-level
    scores are dot products of flattened groups (eq9); the block score is the
    max over the G x G group pairs (eq10); non-causal pairs get -inf (eq14).
    Groups that lie entirely in the padding are left out of the max
    (a zero-padded group would otherwise score 0).  Returns float64
    [L_q, L_kv].
    """
    n_q, c = q_p.shape
    n_kv = k_h.shape[0]
    if b % g:
        raise ValueError("b must be a multiple of g")
    G = b // g
    l_q, l_kv = cdiv(n_q, b), cdiv(n_kv, b)
    qp = np.zeros((l_q * b, c), dtype=np.float64)
    kp = np.zeros((l_kv * b, c), dtype=np.float64)
    qp[:n_q] = q_p
    kp[:n_kv] = k_h
    phi_q = qp.reshape(l_q * G, g * c)            # rows (i, u), eq7
    phi_k = kp.reshape(l_kv * G, g * c)           # rows (j, v), eq7
    s_groups = phi_q @ phi_k.T                    # eq9, float64
    q_real = (np.arange(l_q * G) * g) < n_q       # group holds >= 1 real query
    k_real = (np.arange(l_kv * G) * g) < n_kv
    s_groups[~q_real, :] = -np.inf
    s_groups[:, ~k_real] = -np.inf
    s = s_groups.reshape(l_q, G, l_kv, G).max(axis=(1, 3))   # eq10
    s[~causal_block_mask(n_q, n_kv, b)] = -np.inf             # eq14
    return s


def block_probs(s32: np.ndarray, alpha: float) -> np.ndarray:
    """Block softmax mass (eq15), in float32, row-wise over the last axis.

    A_j = exp(alpha S_j) / sum_j' exp(alpha S_j'), evaluated as
    exp(alpha (S_j - max S)); -inf (non-causal) entries get 0.
    """
    s32 = np.asarray(s32, dtype=np.float32)
    a32 = np.float32(alpha)
    mx = s32.max(axis=-1, keepdims=True)
    e = np.exp(a32 * (s32 - mx)).astype(np.float32)
    return (e / e.sum(axis=-1, keepdims=True, dtype=np.float32)).astype(np.float32)


def keep_mass(s32: np.ndarray, gamma: float, alpha: float):
    """Keep-mass selection (eq16-eq18) for a batch of rows, in float32.

    s32: float32 [R, L] block scores, -inf where not causal.  Every row must
    hold at least one causal block.

    Sort the causal blocks by descending probability (ties: higher score
    first, then lower block index); accumulate the mass in that order in
    float32; keep the shortest prefix whose mass reaches gamma (gamma is
    taken as float32).  gamma >= 1 keeps every causal block (in exact
    arithmetic only the full set reaches 1); a row whose float32 prefix
    never reaches gamma also keeps every causal block.

    Returns (keep bool [R, L], tie bool [R, L], r_star int [R]).  A block is
    a near-tie if (a) it is the t-th in order and the mass before it lies
    within TIE_REL * gamma of gamma (its inclusion flips under a tiny
    perturbation), or (b) its probability lies within TIE_REL relative of
    the last kept block's (it can swap places across the cut).
    """
    s32 = np.asarray(s32, dtype=np.float32)
    R, L = s32.shape
    causal = np.isfinite(s32)
    n_causal = causal.sum(axis=1)
    if np.any(n_causal == 0):
        raise ValueError("row without causal blocks")
    a = block_probs(s32, alpha)
    idx = np.broadcast_to(np.arange(L), (R, L))
    # lexsort: last key is primary -> (-S) ascending, then index ascending.
    order = np.lexsort((idx, -np.where(causal, s32, -np.inf)), axis=-1)
    a_sorted = np.take_along_axis(a, order, axis=1)
    csum = np.cumsum(a_sorted, axis=1, dtype=np.float32)        # sequential
    g32 = np.float32(gamma)
    reached = (csum >= g32) & (np.arange(L)[None, :] < n_causal[:, None])
    first = np.where(reached.any(axis=1), reached.argmax(axis=1) + 1, n_causal)
    r_star = n_causal.copy() if gamma >= 1.0 else first
    pos = np.arange(L)[None, :]
    keep_sorted = pos < r_star[:, None]
    keep = np.zeros((R, L), dtype=bool)
    np.put_along_axis(keep, order, keep_sorted, axis=1)

    # Near-tie flags.
    prev = np.concatenate([np.zeros((R, 1), np.float32), csum[:, :-1]], axis=1)
    band = np.float64(TIE_REL) * np.float64(g32)
    thr_tie_sorted = (np.abs(prev.astype(np.float64) - np.float64(g32)) <= band) \
        & (pos < n_causal[:, None])
    if gamma >= 1.0:
        thr_tie_sorted[:] = False
    tie = np.zeros((R, L), dtype=bool)
    np.put_along_axis(tie, order, thr_tie_sorted, axis=1)
    # Order ties: the smallest kept mass a_in and the largest dropped mass
    # a_out are within TIE_REL of each other -> every block whose mass lies
    # in [a_in (1 - TIE_REL), a_out / (1 - TIE_REL)] may land on either side.
    a64 = a.astype(np.float64)
    a_in = np.take_along_axis(a_sorted, (r_star - 1)[:, None], axis=1).astype(np.float64)
    has_out = r_star < n_causal
    nxt = np.minimum(r_star, L - 1)[:, None]
    a_out = np.where(has_out[:, None],
                     np.take_along_axis(a_sorted, nxt, axis=1).astype(np.float64), -1.0)
    order_tie_row = has_out & (a_out[:, 0] >= (1.0 - TIE_REL) * a_in[:, 0])
    in_band = causal & (a64 >= (1.0 - TIE_REL) * a_in) & (a64 <= a_out / (1.0 - TIE_REL))
    tie |= in_band & order_tie_row[:, None]
    return keep, tie, r_star


def estimate_mask(q: np.ndarray, k: np.ndarray, b: int, g: int, gamma: float,
                  alpha: float) -> Dict[str, np.ndarray]:
    """Stage 1 for one request.

    q: [H_q, N_q, C], k: [H_kv, N_kv, C].  Returns
      scores    float32 [H_q, L_q, L_kv]  (eq10/eq14, float64 rounded once)
      head_keep bool    [H_q, L_q, L_kv]  (eq18, per query head)
      head_tie  bool    [H_q, L_q, L_kv]
      mask      uint8   [H_kv, L_q, L_kv] (GQA union of head_keep)
      status    uint8   [H_kv, L_q, L_kv] (DROP_SURE / KEEP_SURE / TIE)
    The per-KV-head mask is the OR of the masks of the query heads of its
    group (eq18 is per query head, the tile mask of eq20 per KV head).
    """
    h_q, n_q, _ = q.shape
    h_kv, n_kv, _ = k.shape
    if h_q % h_kv:
        raise ValueError("H_q must be a multiple of H_kv")
    m = h_q // h_kv
    l_q, l_kv = cdiv(n_q, b), cdiv(n_kv, b)
    scores = np.empty((h_q, l_q, l_kv), dtype=np.float32)
    keep = np.empty((h_q, l_q, l_kv), dtype=bool)
    tie = np.empty((h_q, l_q, l_kv), dtype=bool)
    for p in range(h_q):
        h = kv_head_of(p, m)
        s = block_scores(q[p], k[h], b, g)
        scores[p] = s.astype(np.float32)
        keep[p], tie[p], _ = keep_mass(scores[p], gamma, alpha)
    kg = keep.reshape(h_kv, m, l_q, l_kv)
    tg = tie.reshape(h_kv, m, l_q, l_kv)
    mask = kg.any(axis=1).astype(np.uint8)
    keep_sure = (kg & ~tg).any(axis=1)
    any_tie = tg.any(axis=1)
    status = np.where(keep_sure, KEEP_SURE, np.where(any_tie, TIE, DROP_SURE))
    return dict(scores=scores, head_keep=keep, head_tie=tie, mask=mask,
                status=status.astype(np.uint8))


# ---------------------------------------------------------------------------
# Stage 2a: tile expansion and rescue (Sec. 3.2 end, Sec. 3.3)
# ---------------------------------------------------------------------------

_M64 = np.uint64(0xFFFFFFFFFFFFFFFF)


def mix64(z):
    """SplitMix64 output mix (Steele, Lea and Flood, OOPSLA 2014):
    z ^= z >> 30; z *= 0xbf58476d1ce4e5b9; z ^= z >> 27;
    z *= 0x94d049bb133111eb; z ^= z >> 31  (all modulo 2^64)."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    return z


def splitmix64_stream(seed: int, n: int) -> List[int]:
    """The SplitMix64 generator: state += 0x9e3779b97f4a7c15, output mix64(state)."""
    out = []
    state = seed & 0xFFFFFFFFFFFFFFFF
    for _ in range(n):
        state = (state + 0x9E3779B97F4A7C15) & 0xFFFFFFFFFFFFFFFF
        out.append(int(mix64(np.uint64(state))))
    return out


def _pack(a, i, j):
    """Key a * 2^42 + i * 2^21 + j (i, j < 2^21)."""
    a = np.asarray(a, dtype=np.uint64)
    i = np.asarray(i, dtype=np.uint64)
    j = np.asarray(j, dtype=np.uint64)
    return (a << np.uint64(42)) | (i << np.uint64(21)) | j


def chi(i, j, seed: int):
    """Stride-rescue mixing function chi(i, j; s) of eq24 (no head index, as
    printed): mix64(mix64(s) xor pack(0, i, j))."""
    s = mix64(np.uint64(seed & 0xFFFFFFFFFFFFFFFF))
    return mix64(s ^ _pack(0, i, j))


def psi24(h, i, j, seed: int):
    """Random-rescue variate of eq25 as a 24-bit integer: psi = psi24 / 2^24
    in [0, 1), from mix64(mix64(s + 1) xor pack(h + 1, i, j)) >> 40."""
    s = mix64(np.uint64((seed + 1) & 0xFFFFFFFFFFFFFFFF))
    return mix64(s ^ _pack(np.asarray(h, dtype=np.uint64) + np.uint64(1), i, j)) \
        >> np.uint64(40)


def rho_threshold(rho: float) -> int:
    """psi < rho  <=>  psi24 < floor(rho * 2^24) (exact: rho * 2^24 is exact)."""
    return int(math.floor(rho * 16777216.0))


def tile_mask(block_mask_h: np.ndarray, n_q: int, n_kv: int, b: int, T: int,
              n_local: int, n_sink: int, eta: int, rho: float, seed: int,
              h: int) -> np.ndarray:
    """Final tile mask of one (request, KV head): bool [T_q, T_kv].

    * expansion (eq19-eq20): tile (qt, kt) inherits block
      (qt // rho_b, kt // rho_b), rho_b = b / T, clipped to causal tiles
      (kt T <= min(N_c + (qt+1) T - 1, N_kv - 1));
    * local band (eq21): the diagonal tile kt_diag(qt) and the n_local tiles
      before it (n_local < 0 switches the band off, diagonal included);
    * sink (eq22): KV tiles kt < n_sink (causal ones);
    * dropped set (eq23): causal and not kept;
    * stride rescue (eq24): dropped tiles with chi(qt, kt; s) mod eta == 0
      (eta = 0: off);
    * random rescue (eq25): dropped tiles with psi(h, qt, kt; s) < rho;
    * final mask (eq26): kept OR stride-rescued OR random-rescued.
    """
    if b % T:
        raise ValueError("b must be a multiple of T")
    rb = b // T
    n_c = n_kv - n_q
    t_q, t_kv = cdiv(n_q, T), cdiv(n_kv, T)
    qt = np.arange(t_q)[:, None]
    kt = np.arange(t_kv)[None, :]
    last_key = np.minimum(n_c + (qt + 1) * T - 1, n_kv - 1)
    causal = (kt * T) <= last_key
    kept = block_mask_h[qt // rb, kt // rb].astype(bool) & causal
    kt_diag = last_key // T
    band = (kt >= kt_diag - n_local) & (kt <= kt_diag) & (n_local >= 0)
    sink = (kt < n_sink) & causal
    kept = kept | band | sink
    dropped = causal & ~kept
    final = kept.copy()
    if eta > 0:
        final |= dropped & ((chi(qt, kt, seed) % np.uint64(eta)) == 0)
    if rho > 0.0:
        final |= dropped & (psi24(h, qt, kt, seed) < np.uint64(rho_threshold(rho)))
    return final


def expand_rescue(block_masks: Sequence[np.ndarray], n_q: Sequence[int],
                  n_kv: Sequence[int], b: int, T: int, n_local: int,
                  n_sink: int, eta: int, rho: float, seed: int):
    """Tile masks of a batch as compacted lists.

    block_masks[r]: uint8 [H_kv, L_q(r), L_kv(r)].  Rows are ordered
    (request, KV head, q-tile); each row lists its kept KV tiles in
    ascending order.  Returns (row_ptr int32 [rows+1], cols int32,
    tile_masks list of bool [H_kv, T_q, T_kv]).
    """
    counts, cols, masks = [], [], []
    for r, bm in enumerate(block_masks):
        h_kv = bm.shape[0]
        per = []
        for h in range(h_kv):
            tm = tile_mask(bm[h], n_q[r], n_kv[r], b, T, n_local, n_sink, eta,
                           rho, seed, h)
            per.append(tm)
            for qt in range(tm.shape[0]):
                nz = np.flatnonzero(tm[qt])
                counts.append(nz.size)
                cols.append(nz.astype(np.int32))
        masks.append(np.stack(per))
    row_ptr = np.zeros(len(counts) + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum(counts)
    if row_ptr[-1] > np.iinfo(np.int32).max:
        raise ValueError("too many kept tiles for int32 lists")
    flat = np.concatenate(cols) if cols else np.zeros(0, np.int32)
    return row_ptr.astype(np.int32), flat.astype(np.int32), masks


# ---------------------------------------------------------------------------
# Stage 2b: exact attention over the retained tiles (eq27) and dense (eq:vsa)
# ---------------------------------------------------------------------------

def attention_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray, p: int, qt: int,
                   T: int, scale: float, kv_tiles: Optional[np.ndarray]):
    """Exact softmax attention for the queries of tile qt of query head p.

    q [H_q, N_q, C], k/v [H_kv, N_kv, C].  Query t sits at absolute position
    N_c + t and may attend key k iff k <= N_c + t, k < N_kv, and (sparse
    case) the tile of k is in ``kv_tiles`` (eq27: dropped tiles carry -inf,
    token-level causal masking inside kept tiles).  kv_tiles=None means
    dense causal attention (eq:vsa with a causal mask).  Float64 throughout.
    Returns (O [rows, C], lse [rows]) with the natural-log LSE of the scaled
    logits; a query with no admissible key gets O = 0 and LSE = -inf.
    """
    h_q, n_q, c = q.shape
    h_kv, n_kv, _ = k.shape
    m = h_q // h_kv
    h = kv_head_of(p, m)
    n_c = n_kv - n_q
    t0, t1 = qt * T, min(n_q, (qt + 1) * T)
    pos = n_c + np.arange(t0, t1)
    last = min(n_kv - 1, int(pos[-1]))
    if kv_tiles is None:
        keys = np.arange(0, last + 1)
    else:
        tiles = np.asarray(kv_tiles, dtype=np.int64)
        keys = (tiles[:, None] * T + np.arange(T)[None, :]).reshape(-1)
        keys = keys[keys <= last]
    qf = q[p, t0:t1].astype(np.float64)
    kf = k[h, keys].astype(np.float64)
    vf = v[h, keys].astype(np.float64)
    logits = scale * (qf @ kf.T)
    allowed = keys[None, :] <= pos[:, None]
    logits = np.where(allowed, logits, -np.inf)
    mx = logits.max(axis=1, keepdims=True) if keys.size else \
        np.full((t1 - t0, 1), -np.inf)
    empty = ~np.isfinite(mx[:, 0])
    mx_safe = np.where(np.isfinite(mx), mx, 0.0)
    w = np.exp(logits - mx_safe)
    denom = w.sum(axis=1, keepdims=True)
    with np.errstate(invalid="ignore", divide="ignore"):
        o = np.where(empty[:, None], 0.0, (w @ vf) / np.where(denom > 0, denom, 1.0))
        lse = np.where(empty, -np.inf, mx_safe[:, 0] + np.log(np.where(denom[:, 0] > 0,
                                                                      denom[:, 0], 1.0)))
    return o, lse


def row_tiles(row_ptr: np.ndarray, cols: np.ndarray, row: int) -> np.ndarray:
    return cols[row_ptr[row]:row_ptr[row + 1]]


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, T: int, scale: float,
              row_ptr: Optional[np.ndarray] = None, cols: Optional[np.ndarray] = None,
              row_base: int = 0):
    """Sparse (lists given) or dense (lists None) attention of one request.

    Rows of this request start at ``row_base`` in (row_ptr, cols), ordered
    (KV head, q-tile).  Returns (O float64 [H_q, N_q, C], lse [H_q, N_q]).
    """
    h_q, n_q, c = q.shape
    h_kv = k.shape[0]
    m = h_q // h_kv
    t_q = cdiv(n_q, T)
    o = np.zeros((h_q, n_q, c), dtype=np.float64)
    lse = np.zeros((h_q, n_q), dtype=np.float64)
    for p in range(h_q):
        h = kv_head_of(p, m)
        for qt in range(t_q):
            tiles = None
            if row_ptr is not None:
                tiles = row_tiles(row_ptr, cols, row_base + h * t_q + qt)
            t0, t1 = qt * T, min(n_q, (qt + 1) * T)
            o[p, t0:t1], lse[p, t0:t1] = attention_rows(q, k, v, p, qt, T, scale, tiles)
    return o, lse


def default_scale(head_dim: int) -> float:
    """alpha = 1/sqrt(C) (eq15, eq27)."""
    return 1.0 / math.sqrt(head_dim)
