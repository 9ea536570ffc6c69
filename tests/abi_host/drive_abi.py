"""Drive a host-only build of the C ABI layer (real api.cpp and shapes.cpp,
stub launchers that touch no memory) through every entry point: the error
paths, and every entry point on seeded random problems (batches of up to 32
requests, chunked and ragged lengths, contiguous and paged K/V, valid and
invalid hyper-parameters).  Meant to run in a process with the
AddressSanitizer / UndefinedBehaviorSanitizer runtime preloaded, so that any
out-of-bounds access or undefined behaviour in the host code aborts it.

usage: python drive_abi.py <path to the sanitizer build> [cases]
Prints one summary line and exits 0 when every check passed.
"""
import ctypes as C
import os
import random
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
from paper_2605_12193_amd import abi  # noqa: E402  (ctypes only, no torch)

A = 1 << 20          # a fake, 16-byte aligned device address (never dereferenced)
OK, INVALID, UNSUP, WS, CAP, HIP = range(6)


def problem(n_q, n_kv, h_q, h_kv, c):
    nq = (C.c_int32 * len(n_q))(*n_q)
    nkv = (C.c_int32 * len(n_kv))(*n_kv)
    p = abi.bfla_problem(len(n_q), h_q, h_kv, c, nq, nkv)
    p._keep = (nq, nkv)
    return p


def params(**kw):
    base = dict(block=128, group=64, tile=64, gamma=0.9, n_local=2, n_sink=1, eta=16,
                rho=0.1, seed=7, scale=0.0)
    base.update(kw)
    return abi.bfla_params(*[base[k] for k in ("block", "group", "tile", "gamma", "n_local",
                                               "n_sink", "eta", "rho", "seed", "scale")])


def sizes(L, p, prm):
    vals = [C.c_size_t() for _ in range(4)]
    st = L.bfla_list_capacity(C.byref(p), C.byref(prm), *[C.byref(v) for v in vals])
    ws = [C.c_size_t(), C.c_size_t()]
    if st == OK:
        assert L.bfla_workspace_size(C.byref(p), C.byref(prm), abi.BFLA_WS_ESTIMATE,
                                     C.byref(ws[0])) == OK
        assert L.bfla_workspace_size(C.byref(p), C.byref(prm), abi.BFLA_WS_EXPAND,
                                     C.byref(ws[1])) == OK
    return st, [v.value for v in vals], [w.value for w in ws]


def error_paths(L):
    p, prm = problem([256], [256], 4, 2, 64), params()
    v = abi.bfla_view(A, None, 0, 256 * 64, 64)
    kv = abi.bfla_kv(abi.BFLA_KV_CONTIGUOUS, A, A, None, 0, 256 * 64, 64, 0, 0, 0, None, 0)
    a = C.c_void_p(A)
    checks = [
        (L.bfla_estimate_mask(C.byref(p), C.byref(prm), C.byref(v), C.byref(kv), None, None,
                              None, a, 1 << 30, None), INVALID),
        (L.bfla_estimate_mask(C.byref(p), C.byref(prm), C.byref(v), C.byref(kv), a, None, None,
                              a, 4, None), WS),
        (L.bfla_estimate_mask(None, C.byref(prm), C.byref(v), C.byref(kv), a, a, None, None, 0,
                              None), INVALID),
        (L.bfla_estimate_mask(C.byref(p), C.byref(prm), None, C.byref(kv), a, a, None, None, 0,
                              None), INVALID),
        (L.bfla_expand_rescue(C.byref(p), C.byref(prm), a, a, a, 3, a, 1 << 20, None), CAP),
        (L.bfla_expand_rescue(C.byref(p), C.byref(prm), a, a, a, 1 << 20, a, 0, None), WS),
        (L.bfla_expand_rescue(C.byref(p), C.byref(prm), a, a, a, 1 << 20, C.c_void_p(A + 4),
                              1 << 30, None), INVALID),
        (L.bfla_expand_rescue(C.byref(p), None, a, a, a, 1 << 20, a, 1 << 30, None), INVALID),
        (L.bfla_sparse_prefill(C.byref(p), C.byref(prm), C.byref(v), C.byref(kv), None, None,
                               C.byref(v), None, None), INVALID),
        (L.bfla_sparse_prefill(C.byref(p), C.byref(prm), C.byref(v), None, a, a, C.byref(v),
                               None, None), INVALID),
        (L.bfla_dense_prefill(C.byref(p), C.byref(prm), C.byref(v), C.byref(kv), None, None,
                              None), INVALID),
        (L.bfla_workspace_size(C.byref(p), C.byref(prm), 9, C.byref(C.c_size_t())), INVALID),
        (L.bfla_workspace_size(C.byref(p), C.byref(prm), 1, None), INVALID),
        (L.bfla_list_capacity(None, C.byref(prm), None, None, None, None), INVALID),
    ]
    for got, want in checks:
        assert got == want, (got, want)
        assert len(L.bfla_last_error()) > 0
    for s in range(-2, 8):
        assert len(L.bfla_status_string(s)) > 0
    assert L.bfla_version().decode().count(".") == 2
    return len(checks)


def random_case(rng, L):
    def pick(valid, invalid=(), p_bad=0.03):
        """A valid choice, or now and then an invalid one."""
        return rng.choice(invalid) if invalid and rng.random() < p_bad else rng.choice(valid)

    batch = pick([1, 1, 2, 3, 7, 32, 33, 70], [0, 65537])
    c = pick([64, 128, 256], [96])
    h_kv = rng.choice([1, 2, 8])
    m = pick([1, 2, 4, 5, 8], [9])
    n_kv = [rng.choice([1, 63, 64, 65, 1000, 4096, 131072, 1 << 20, rng.randint(1, 300000)])
            for _ in range(max(batch, 1))]
    n_q = [x if rng.random() < 0.6 else pick([rng.randint(1, x)], [0]) for x in n_kv]
    p = problem(n_q[:max(batch, 1)], n_kv[:max(batch, 1)], h_kv * m, h_kv, c)
    p.batch = batch
    block = pick([64, 128, 256, 1024], [96])
    prm = params(block=block, group=pick([block, block // 2, block // 16], [48, 0]),
                 gamma=pick([0.5, 0.9, 1.0], [0.0, 1.5]),
                 n_local=pick([-1, 0, 2, 8], [-2]), n_sink=pick([0, 1, 3], [-1]),
                 eta=pick([0, 1, 16], [-1]), rho=pick([0.0, 0.1, 1.0], [1.5]),
                 seed=rng.randint(0, 2 ** 64 - 1), scale=pick([0.0, 0.125], [-1.0]))
    st, (n_rows, max_cols, mask_bytes, score_elems), (ws_est, ws_exp) = sizes(L, p, prm)
    if st != OK:
        return "rejected"
    tok = c * rng.choice([1, h_kv * m])
    paged = rng.random() < 0.4
    if paged:
        ps = pick([16, 32, 256], [24])
        max_pages = max(-(-n // ps) for n in n_kv[:batch]) + pick([0], [-1])
        kv = abi.bfla_kv(abi.BFLA_KV_PAGED, A, A, None, 0, c, c * h_kv, ps, max_pages,
                         ps * c * h_kv, A, rng.choice([1, 64, 1 << 12]))
    else:
        offs = (C.c_int64 * batch)(*[8 * rng.randint(0, 1 << 20) for _ in range(batch)])
        kv = abi.bfla_kv(abi.BFLA_KV_CONTIGUOUS, A, A, offs if rng.random() < 0.5 else None,
                         8 * rng.randint(0, 1 << 22), tok * max(n_kv[:batch]), c, 0, 0, 0,
                         None, 0)
        kv._keep = offs
    q = abi.bfla_view(A, None, 8 * rng.randint(0, 1 << 22), c * max(n_q[:batch] + [1]), c)
    a = C.c_void_p(A)
    n_ok = 0
    st = L.bfla_estimate_mask(C.byref(p), C.byref(prm), C.byref(q), C.byref(kv), a,
                              a if rng.random() < 0.5 else None,
                              a if rng.random() < 0.5 else None, a, ws_est, None)
    assert st in (OK, INVALID, UNSUP), st
    n_ok += st == OK
    st = L.bfla_expand_rescue(C.byref(p), C.byref(prm), a, a, a, max_cols, a, ws_exp, None)
    assert st in (OK, INVALID, UNSUP), st
    n_ok += st == OK
    st = L.bfla_expand_rescue_noalloc(C.byref(p), C.byref(prm), a, a, a, max_cols, None)
    assert st in (OK, INVALID, UNSUP, WS), st
    # accepted only when its workspace fits the scratch; too large -> WORKSPACE
    # (unless an earlier check already refused the problem)
    assert st != OK or ws_exp <= abi.EXPAND_SCRATCH_BYTES, (st, ws_exp)
    assert st != WS or ws_exp > abi.EXPAND_SCRATCH_BYTES, (st, ws_exp)
    st = L.bfla_sparse_prefill(C.byref(p), C.byref(prm), C.byref(q), C.byref(kv), a, a,
                               C.byref(q), a, None)
    assert st in (OK, INVALID, UNSUP), st
    n_ok += st == OK
    st = L.bfla_dense_prefill(C.byref(p), C.byref(prm), C.byref(q), C.byref(kv), C.byref(q),
                              None, None)
    assert st in (OK, INVALID, UNSUP), st
    n_ok += st == OK
    return f"launched {n_ok}"


def main():
    L = abi.bind(sys.argv[1])
    cases = int(sys.argv[2]) if len(sys.argv) > 2 else 2000
    n_err = error_paths(L)
    rng = random.Random(20260)
    outcome = {}
    for _ in range(cases):
        r = random_case(rng, L)
        outcome[r] = outcome.get(r, 0) + 1
    launches = [L.stub_launches(i) for i in range(3)]
    bad = L.stub_bad_descriptors()
    assert bad == 0, f"{bad} inconsistent launch descriptors"
    assert min(launches) > 0, f"an entry point never launched: {launches}"
    print(f"abi driver ok: {n_err} error paths, {cases} random problems {sorted(outcome.items())}, "
          f"launches prefill/expand/estimate {launches}", flush=True)


if __name__ == "__main__":
    main()
