"""The C-ABI library: it loads, exports every declared symbol, and rejects bad
arguments before touching the GPU (these calls launch nothing)."""
import ctypes as C
import os
import re

import pytest

from paper_2605_12193_amd import bfla

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bfla.h")

pytestmark = pytest.mark.skipif(not os.path.exists(bfla._LIB_PATH),
                                reason="libbfla.so not built")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|const char\*)\s+(bfla_\w+)\(", text, re.M)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert set(names) == set(bfla.EXPORTS)
    lib = C.CDLL(bfla._LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def declared_parameters():
    """Parameter lists of the declared entry points, as written in the header."""
    text = re.sub(r"/\*.*?\*/", " ", open(HEADER).read(), flags=re.S)
    out = {}
    for name, params in re.findall(r"^(?:int|const char\*)\s+(bfla_\w+)\(([^)]*)\);", text,
                                   re.M):
        params = " ".join(params.split())
        out[name] = [] if params in ("", "void") else [x.strip() for x in params.split(",")]
    return out


def test_binding_signatures_match_the_header():
    decl = declared_parameters()
    assert set(decl) == set(bfla.EXPORTS)
    for name, params in decl.items():
        assert len(params) == len(bfla._SIGS[name]), (name, params)
    # the per-query-head keep sets (eq18) are an optional output of Stage 1
    est = decl["bfla_estimate_mask"]
    assert est[5] == "float* dbg_scores" and est[6] == "uint8_t* dbg_head_mask"


def test_version_and_status_strings():
    assert bfla.bfla_version() == "0.2.0"
    assert bfla.bfla_status_string(0) == "ok"
    assert bfla.bfla_status_string(4) == "list capacity too small"


def _prob(n=(256,), h_q=4, h_kv=2, c=64):
    return bfla.Problem(n, n, h_q, h_kv, c)


def test_capacity_and_workspace_sizes():
    p = _prob((256, 300))
    prm = bfla.params()
    cap = bfla.bfla_list_capacity(p, prm)
    # rows: H_kv * T_q per request; causal tiles: T(T+1)/2 per head
    assert cap.n_rows == 2 * 4 + 2 * 5
    assert cap.max_cols == 2 * (4 * 5 // 2) + 2 * (5 * 6 // 2)
    assert cap.mask_bytes == 2 * 2 * 2 + 2 * 3 * 3
    assert cap.score_elems == 4 * 2 * 2 + 4 * 3 * 3
    assert bfla.bfla_workspace_size(p, prm, bfla.BFLA_WS_ESTIMATE) >= cap.score_elems * 4
    assert bfla.bfla_workspace_size(p, prm, bfla.BFLA_WS_EXPAND) >= cap.n_rows * 4
    chunk = bfla.Problem([64], [320], 4, 2, 64)
    cap2 = bfla.bfla_list_capacity(chunk, prm)
    assert cap2.max_cols == 2 * 5          # one q-tile sees all 5 KV tiles


@pytest.mark.parametrize("mut,status", [
    (lambda p, q: setattr(p.c, "h_q", 5), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(p.c, "head_dim", 96), bfla.BFLA_ERR_UNSUPPORTED),
    (lambda p, q: setattr(p.c, "batch", 0), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(p.c, "batch", 65537), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(q, "gamma", 0.0), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(q, "gamma", 1.5), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(q, "gamma", float("nan")), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(q, "n_local", -2), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(q, "n_sink", -1), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(q, "eta", -1), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(q, "rho", 1.5), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(q, "tile", 32), bfla.BFLA_ERR_UNSUPPORTED),
    (lambda p, q: setattr(q, "block", 96), bfla.BFLA_ERR_UNSUPPORTED),
    (lambda p, q: setattr(q, "group", 48), bfla.BFLA_ERR_INVALID_ARG),
    (lambda p, q: setattr(q, "scale", -1.0), bfla.BFLA_ERR_INVALID_ARG),
])
def test_problem_and_param_errors(mut, status):
    p, prm = _prob(), bfla.params()
    mut(p, prm)
    with pytest.raises(bfla.BflaError) as e:
        bfla.bfla_list_capacity(p, prm)
    assert e.value.status == status
    assert bfla.lib().bfla_last_error().decode() != ""


def test_bad_request_lengths():
    prm = bfla.params()
    with pytest.raises(bfla.BflaError) as e:
        bfla.bfla_list_capacity(bfla.Problem([300], [200], 4, 2, 64), prm)
    assert e.value.status == bfla.BFLA_ERR_INVALID_ARG
    with pytest.raises(bfla.BflaError):
        bfla.bfla_list_capacity(bfla.Problem([0], [10], 4, 2, 64), prm)


def _fake_views():
    """Views over fake (never dereferenced) aligned addresses: every call
    below fails validation before any launch."""
    addr = 1 << 20
    v = bfla.bfla_view(addr, None, 0, 256 * 64, 64)
    kv = bfla.bfla_kv(bfla.BFLA_KV_CONTIGUOUS, addr, addr, None, 0, 256 * 64, 64, 0, 0, 0, None,
                      0)
    return v, kv


def test_entry_points_reject_before_launch():
    L = bfla.lib()
    p, prm = _prob(), bfla.params()
    v, kv = _fake_views()
    addr = C.c_void_p(1 << 20)
    # null block mask
    st = L.bfla_estimate_mask(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(kv), None, None,
                              None, addr, 1 << 30, None)
    assert st == bfla.BFLA_ERR_INVALID_ARG
    # workspace too small and no dbg output
    st = L.bfla_estimate_mask(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(kv), addr, None,
                              None, addr, 4, None)
    assert st == bfla.BFLA_ERR_WORKSPACE
    # list capacity too small
    st = L.bfla_expand_rescue(C.byref(p.c), C.byref(prm), addr, addr, addr, 3, addr, 1 << 20,
                              None)
    assert st == bfla.BFLA_ERR_CAPACITY
    # expand workspace too small
    st = L.bfla_expand_rescue(C.byref(p.c), C.byref(prm), addr, addr, addr, 1 << 20, addr, 0,
                              None)
    assert st == bfla.BFLA_ERR_WORKSPACE
    # expand workspace not 8-byte aligned
    st = L.bfla_expand_rescue(C.byref(p.c), C.byref(prm), addr, addr, addr, 1 << 20,
                              C.c_void_p((1 << 20) + 4), 1 << 30, None)
    assert st == bfla.BFLA_ERR_INVALID_ARG
    # misaligned q
    bad = bfla.bfla_view((1 << 20) + 2, None, 0, 256 * 64, 64)
    st = L.bfla_sparse_prefill(C.byref(p.c), C.byref(prm), C.byref(bad), C.byref(kv), addr,
                               addr, C.byref(v), None, None)
    assert st == bfla.BFLA_ERR_INVALID_ARG
    # null lists
    st = L.bfla_sparse_prefill(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(kv), None,
                               None, C.byref(v), None, None)
    assert st == bfla.BFLA_ERR_INVALID_ARG
    # unsupported GQA group size 9
    p3 = bfla.Problem([256], [256], 18, 2, 64)
    st = L.bfla_dense_prefill(C.byref(p3.c), C.byref(prm), C.byref(v), C.byref(kv),
                              C.byref(v), None, None)
    assert st == bfla.BFLA_ERR_UNSUPPORTED
    # paged K/V with too few pages in the table
    pk = bfla.bfla_kv(bfla.BFLA_KV_PAGED, 1 << 20, 1 << 20, None, 0, 64, 128, 16, 8, 16 * 128,
                      1 << 20, 64)
    st = L.bfla_dense_prefill(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(pk), C.byref(v),
                              None, None)
    assert st == bfla.BFLA_ERR_INVALID_ARG
    # page size not a power of two >= 16
    pk.max_pages = 64
    pk.page_size = 24
    st = L.bfla_dense_prefill(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(pk), C.byref(v),
                              None, None)
    assert st == bfla.BFLA_ERR_UNSUPPORTED
    # token rows narrower than a head (overlapping), or a 64-token tile of 2 GiB
    pk.page_size = 16
    pk.stride_tok = 32
    st = L.bfla_dense_prefill(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(pk), C.byref(v),
                              None, None)
    assert st == bfla.BFLA_ERR_INVALID_ARG
    pk.stride_tok = 1 << 24
    pk.page_stride = 16 << 24
    pk.n_pages = 1  # a pool of one page stays under 2 GiB
    st = L.bfla_dense_prefill(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(pk), C.byref(v),
                              None, None)
    assert st == bfla.BFLA_ERR_UNSUPPORTED
    assert b"2^24" in L.bfla_last_error()
    pk.stride_tok = 128
    pk.page_stride = 16 * 128
    # pool of 2 GiB or more
    pk.n_pages = 1 << 20
    st = L.bfla_dense_prefill(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(pk), C.byref(v),
                              None, None)
    assert st == bfla.BFLA_ERR_UNSUPPORTED


def test_estimate_address_limits():
    L = bfla.lib()
    addr = C.c_void_p(1 << 20)
    p, prm = _prob(), bfla.params()
    _, kv = _fake_views()
    # q rows of one score tile (256 groups of 64 tokens) spanning >= 2 GiB
    wide = bfla.bfla_view(1 << 20, None, 0, 64, 1 << 18)
    st = L.bfla_estimate_mask(C.byref(p.c), C.byref(prm), C.byref(wide), C.byref(kv), addr,
                              addr, None, None, 0, None)
    assert st == bfla.BFLA_ERR_UNSUPPORTED
    # paged K: 128 groups of 512 tokens cover 4097 16-token pages
    big = bfla.params(block=1024, group=512)
    pk = bfla.bfla_kv(bfla.BFLA_KV_PAGED, 1 << 20, 1 << 20, None, 0, 64, 128, 16, 64, 16 * 128,
                      1 << 20, 64)
    q = bfla.bfla_view(1 << 20, None, 0, 256 * 64, 64)
    st = L.bfla_estimate_mask(C.byref(p.c), C.byref(big), C.byref(q), C.byref(pk), addr, addr,
                              None, None, 0, None)
    assert st == bfla.BFLA_ERR_UNSUPPORTED
    assert "pages" in L.bfla_last_error().decode()


def test_expand_workspace_holds_counts_and_ballots():
    # per-row counts and scan partials (int32), then one 64-bit keep ballot per
    # 64 KV tiles of the longest request for every list row
    prm = bfla.params()
    for n_q, n_kv in (([4096], [4096]), ([300, 5000], [1000, 5000]), ([64], [64])):
        p = bfla.Problem(n_q, n_kv, 8, 2, 128)
        cap = bfla.bfla_list_capacity(p, prm)
        words = -(-max(-(-n // 64) for n in n_kv) // 64)
        want = (-(-cap.n_rows // 64) * 64 + 64) * 4 + cap.n_rows * words * 8
        assert bfla.bfla_workspace_size(p, prm, bfla.BFLA_WS_EXPAND) == want


def test_noalloc_tile_stage_rejects_problems_beyond_its_scratch():
    # the workspace of 8 KV heads x 4096 q-tiles x 64 ballot words is 16 MiB
    # plus the row counts: one row past the fixed scratch; rejected before any
    # device call (no GPU is touched here)
    L = bfla.lib()
    prm = bfla.params()
    big = bfla.Problem([262144], [262144], 8, 8, 128)
    need = bfla.bfla_workspace_size(big, prm, bfla.BFLA_WS_EXPAND)
    assert need > bfla.EXPAND_SCRATCH_BYTES
    cap = bfla.bfla_list_capacity(big, prm)
    addr = C.c_void_p(1 << 20)
    st = L.bfla_expand_rescue_noalloc(C.byref(big.c), C.byref(prm), addr, addr, addr,
                                      cap.max_cols, None)
    assert st == bfla.BFLA_ERR_WORKSPACE
    assert b"scratch" in L.bfla_last_error()
    # the other argument checks come first, as in bfla_expand_rescue
    st = L.bfla_expand_rescue_noalloc(C.byref(big.c), C.byref(prm), addr, addr, addr, 3, None)
    assert st == bfla.BFLA_ERR_CAPACITY
    st = L.bfla_expand_rescue_noalloc(C.byref(big.c), C.byref(prm), None, addr, addr,
                                      cap.max_cols, None)
    assert st == bfla.BFLA_ERR_INVALID_ARG
    # the largest workloads here fit: 128K x 8 KV heads, and the 4-request
    # paged batch of 16K-128K tokens
    for n in ([131072], [16384, 32768, 65536, 131072]):
        p = bfla.Problem(n, n, 40, 8, 128)
        assert bfla.bfla_workspace_size(p, prm, bfla.BFLA_WS_EXPAND) <= bfla.EXPAND_SCRATCH_BYTES


def _split_of(n, h_q, h_kv, c, **kw):
    """The split of the Stage-1 score GEMM, read off the workspace size:
    align256(split x tiles x 256 x 128 x 4 B) of partial sums + the scores."""
    p = bfla.Problem(n, n, h_q, h_kv, c)
    prm = bfla.params(**kw)
    ws = bfla.bfla_workspace_size(p, prm, bfla.BFLA_WS_ESTIMATE)
    part = ws - bfla.bfla_list_capacity(p, prm).score_elems * 4
    g = kw.get("group", 64)
    tiles = sum(h_q * -(-(-(-x // g)) // 256) * -(-(-(-x // g)) // 128) for x in n)
    if part == 0:
        return 1
    split = part // (tiles * 256 * 128 * 4)
    assert part == split * tiles * 256 * 128 * 4, (part, tiles)
    return split


def test_stage1_split_follows_the_tile_count():
    # 128K x 32 heads: 2304 causal score tiles, nine full rounds of 256
    # workgroups -> no split, the workspace is just the scores
    assert _split_of([131072], 32, 8, 128) == 1
    # 32K x 32 heads: 192 causal tiles; four parts would run three rounds of
    # quarter length, but their partial sums eat the gain -> no split
    assert _split_of([32768], 32, 8, 128) == 1
    # 64K x 16 heads at head dim 256: 320 causal tiles -> four parts (five rounds)
    assert _split_of([65536], 16, 8, 256) == 4
    # a 2K request: 4 tiles -> eight parts, the most whole 8-stage chains allow
    assert _split_of([2048], 4, 2, 64) == 8
    # 16 stages (g C = 1024) hold two chains: at most two parts
    assert _split_of([2048], 4, 2, 64, block=128, group=16) == 2
    # the paged batch (4 requests, 40 heads) fills the GPU unsplit
    assert _split_of([16384, 32768, 65536, 131072], 40, 8, 128) == 1


def test_estimate_workspace_is_checked():
    L = bfla.lib()
    p, prm = _prob(), bfla.params()   # small: split, so partial sums are needed
    v, kv = _fake_views()
    addr = C.c_void_p(1 << 20)
    ws = bfla.bfla_workspace_size(p, prm, bfla.BFLA_WS_ESTIMATE)
    scores = bfla.bfla_list_capacity(p, prm).score_elems * 4
    # with dbg_scores the partial sums still need the workspace
    st = L.bfla_estimate_mask(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(kv), addr, addr,
                              None, None, 0, None)
    assert st == bfla.BFLA_ERR_WORKSPACE
    st = L.bfla_estimate_mask(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(kv), addr, addr,
                              None, addr, ws - scores - 1, None)
    assert st == bfla.BFLA_ERR_WORKSPACE
    # misaligned workspace
    st = L.bfla_estimate_mask(C.byref(p.c), C.byref(prm), C.byref(v), C.byref(kv), addr, addr,
                              None, C.c_void_p((1 << 20) + 16), ws, None)
    assert st == bfla.BFLA_ERR_INVALID_ARG


def test_batches_beyond_one_launch_group_are_sized():
    # 70 requests (three launch groups of up to 32): sizes are the sums over
    # requests, and the Stage-1 workspace covers the largest group's split
    prm = bfla.params()
    n = [64 * (1 + i % 7) + i for i in range(70)]
    p = bfla.Problem(n, n, 4, 2, 64)
    cap = bfla.bfla_list_capacity(p, prm)
    assert cap.n_rows == sum(2 * -(-x // 64) for x in n)
    assert cap.mask_bytes == sum(2 * (-(-x // 128)) ** 2 for x in n)
    ws = bfla.bfla_workspace_size(p, prm, bfla.BFLA_WS_ESTIMATE)
    assert ws >= cap.score_elems * 4
