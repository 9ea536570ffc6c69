"""The oracle's pins catch planted mistakes (mutation check, CPU only).

Each mutant is a one-line change to the oracle's source -- a dropped term, a
flipped comparison, a transposed index, a wrong constant -- executed into a
module of its own.  The pin battery (the tests of test_oracle_stage1,
test_oracle_tiles, test_oracle_attention and the fast ones of
test_oracle_precision) runs against it, and at least one pin must fail.  An
unmutated copy built the same way must pass every pin, so the check says
something about the pins and not about the harness.  Mutations that leave
the method's result unchanged (equivalent rewrites) are not listed, nor are
changes to the key packing or seeding of the rescue hashes: any fixed hash is
a valid reading of eq24-eq25, and the one chosen is checked against the GPU
by the parity tests rather than pinned to the paper.
"""
import inspect
import os
import types

import pytest

import test_oracle_attention
import test_oracle_precision
import test_oracle_stage1
import test_oracle_tiles

ORACLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "oracle", "bfla_oracle.py")

# (name, text in the oracle, replacement): each text occurs exactly once
MUTANTS = [
    ("kv head p % m instead of p // m (eq8)",
     "return p // m", "return p % m"),
    ("padded query groups enter the max pool",
     "s_groups[~q_real, :] = -np.inf", "pass"),
    ("groups flattened across tokens (eq7)",
     "phi_k = kp.reshape(l_kv * G, g * c)", "phi_k = kp.reshape(g * c, l_kv * G).T"),
    ("sum instead of max over group pairs (eq10)",
     ".max(axis=(1, 3))   # eq10", ".sum(axis=(1, 3))   # eq10"),
    ("causal block end one past (eq11)",
     "e = np.minimum(n_c + (i + 1) * b - 1, n_kv - 1)",
     "e = np.minimum(n_c + (i + 1) * b, n_kv - 1)"),
    ("block softmax without the scale (eq15)",
     "e = np.exp(a32 * (s32 - mx))", "e = np.exp(s32 - mx)"),
    ("ties ranked by descending block index",
     "order = np.lexsort((idx, -np.where(causal, s32, -np.inf)), axis=-1)",
     "order = np.lexsort((-idx, -np.where(causal, s32, -np.inf)), axis=-1)"),
    ("mass must exceed gamma instead of reach it (eq17)",
     "reached = (csum >= g32)", "reached = (csum > g32)"),
    ("gamma = 1 left to the float sum",
     "r_star = n_causal.copy() if gamma >= 1.0 else first", "r_star = first"),
    ("AND instead of OR over the GQA group",
     "mask = kg.any(axis=1).astype(np.uint8)", "mask = kg.all(axis=1).astype(np.uint8)"),
    ("tile expansion indices swapped (eq20)",
     "kept = block_mask_h[qt // rb, kt // rb].astype(bool) & causal",
     "kept = block_mask_h[kt // rb, qt // rb].astype(bool) & causal"),
    ("local band one tile short (eq21)",
     "band = (kt >= kt_diag - n_local) & (kt <= kt_diag) & (n_local >= 0)",
     "band = (kt > kt_diag - n_local) & (kt <= kt_diag) & (n_local >= 0)"),
    ("one sink tile too many (eq22)",
     "sink = (kt < n_sink) & causal", "sink = (kt <= n_sink) & causal"),
    ("SplitMix64 multiplier off by two",
     "np.uint64(0xBF58476D1CE4E5B9)", "np.uint64(0xBF58476D1CE4E5BB)"),
    ("random-rescue variate from bit 41",
     ">> np.uint64(40)", ">> np.uint64(41)"),
    ("stride rescue keyed by the head (eq24 has none)",
     "final |= dropped & ((chi(qt, kt, seed) % np.uint64(eta)) == 0)",
     "final |= dropped & ((chi(qt + h, kt, seed) % np.uint64(eta)) == 0)"),
    ("random rescue ignores rho's threshold (eq25)",
     "final |= dropped & (psi24(h, qt, kt, seed) < np.uint64(rho_threshold(rho)))",
     "final |= dropped & (psi24(h, qt, kt, seed) <= np.uint64(rho_threshold(rho)))"),
    ("a query may not see itself (eq27)",
     "allowed = keys[None, :] <= pos[:, None]", "allowed = keys[None, :] < pos[:, None]"),
    ("attention logits without the scale",
     "logits = scale * (qf @ kf.T)", "logits = (qf @ kf.T)"),
    ("last admissible key one short",
     "last = min(n_kv - 1, int(pos[-1]))", "last = min(n_kv - 2, int(pos[-1]))"),
    ("LSE without the max it was shifted by",
     "lse = np.where(empty, -np.inf, mx_safe[:, 0] + np.log(",
     "lse = np.where(empty, -np.inf, 0.0 * mx_safe[:, 0] + np.log("),
    ("causal block pair needs a key strictly before the block end (eq13)",
     "return (j * b) <= e", "return (j * b) < e"),
    ("a key group starting at N_kv counted as real",
     "k_real = (np.arange(l_kv * G) * g) < n_kv", "k_real = (np.arange(l_kv * G) * g) <= n_kv"),
    ("padded key groups enter the max pool",
     "s_groups[:, ~k_real] = -np.inf", "pass"),
    ("block softmax without the max shift (overflows)",
     "e = np.exp(a32 * (s32 - mx)).astype(np.float32)", "e = np.exp(a32 * s32).astype(np.float32)"),
    ("r* one block short (eq17)",
     "first = np.where(reached.any(axis=1), reached.argmax(axis=1) + 1, n_causal)",
     "first = np.where(reached.any(axis=1), reached.argmax(axis=1), n_causal)"),
    ("a row that never reaches gamma keeps one block",
     "first = np.where(reached.any(axis=1), reached.argmax(axis=1) + 1, n_causal)",
     "first = np.where(reached.any(axis=1), reached.argmax(axis=1) + 1, 1)"),
    ("gamma compared in float64",
     "reached = (csum >= g32)", "reached = (csum.astype(np.float64) >= gamma)"),
    ("near-tie band 100 times wider",
     "TIE_REL = 1e-5", "TIE_REL = 1e-3"),
    ("a cell kept only as a near-tie counted as sure",
     "keep_sure = (kg & ~tg).any(axis=1)", "keep_sure = kg.any(axis=1)"),
    ("query block end without the prefix N_c (eq11)",
     "e = np.minimum(n_c + (i + 1) * b - 1, n_kv - 1)", "e = np.minimum((i + 1) * b - 1, n_kv - 1)"),
    ("tile causality without the prefix N_c (eq20)",
     "last_key = np.minimum(n_c + (qt + 1) * T - 1, n_kv - 1)",
     "last_key = np.minimum((qt + 1) * T - 1, n_kv - 1)"),
    ("expansion ratio b / T off by one (eq19)",
     "rb = b // T", "rb = b // T + 1"),
    ("local band without the diagonal tile (eq21)",
     "band = (kt >= kt_diag - n_local) & (kt <= kt_diag) & (n_local >= 0)",
     "band = (kt >= kt_diag - n_local) & (kt < kt_diag) & (n_local >= 0)"),
    ("stride rescue outside the causal triangle (eq23-eq24)",
     "final |= dropped & ((chi(qt, kt, seed) % np.uint64(eta)) == 0)",
     "final |= ~kept & ((chi(qt, kt, seed) % np.uint64(eta)) == 0)"),
    ("rho threshold rounded up (eq25)",
     "return int(math.floor(rho * 16777216.0))", "return int(math.ceil(rho * 16777216.0))"),
    ("SplitMix64 increment off by two",
     "state = (state + 0x9E3779B97F4A7C15) & 0xFFFFFFFFFFFFFFFF",
     "state = (state + 0x9E3779B97F4A7C17) & 0xFFFFFFFFFFFFFFFF"),
    ("last admissible key excluded",
     "keys = keys[keys <= last]", "keys = keys[keys < last]"),
    ("sparse rows looked up q-tile major",
     "tiles = row_tiles(row_ptr, cols, row_base + h * t_q + qt)",
     "tiles = row_tiles(row_ptr, cols, row_base + qt * h_kv + h)"),
    ("empty query row with LSE 0 instead of -inf",
     "lse = np.where(empty, -np.inf,", "lse = np.where(empty, 0.0,"),
    ("default scale 1/C instead of 1/sqrt(C) (eq15)",
     "return 1.0 / math.sqrt(head_dim)", "return 1.0 / head_dim"),
]

PIN_MODULES = [test_oracle_stage1, test_oracle_tiles, test_oracle_attention,
               test_oracle_precision]
# pins that need fixtures or take seconds run elsewhere, not in the battery
SKIP = {"test_llama_32k_sampled_rows", "test_long_rows_with_hundreds_of_kept_blocks"}


def _build(replace=None):
    src = open(ORACLE).read()
    if replace is not None:
        old, new = replace
        assert src.count(old) == 1, f"mutation site not unique: {old!r}"
        src = src.replace(old, new)
    mod = types.ModuleType("bfla_oracle_mutant")
    mod.__file__ = ORACLE
    exec(compile(src, ORACLE, "exec"), mod.__dict__)
    return mod


def _cases():
    """Every pin as a zero-argument call (parametrized pins expanded)."""
    out = []
    for m in PIN_MODULES:
        for name, fn in inspect.getmembers(m, inspect.isfunction):
            if not name.startswith("test_") or name in SKIP or fn.__module__ != m.__name__:
                continue
            marks = [mk for mk in getattr(fn, "pytestmark", []) if mk.name == "parametrize"]
            if not marks:
                out.append((f"{m.__name__}::{name}", fn, {}))
                continue
            (argnames, values), = [mk.args[:2] for mk in marks]
            names = [a.strip() for a in argnames.split(",")]
            for v in values:
                v = v if isinstance(v, (tuple, list)) else (v,)
                out.append((f"{m.__name__}::{name}{list(v)}", fn, dict(zip(names, v))))
    return out


def _run_battery(oracle_module, stop_at_first=True):
    """Run every pin against `oracle_module`; returns the pins that failed."""
    saved = [m.O for m in PIN_MODULES]
    failed = []
    try:
        for m in PIN_MODULES:
            m.O = oracle_module
        for label, fn, kw in _cases():
            try:
                fn(**kw)
            except Exception as e:   # an assertion, or the mutant breaking a shape / a lookup
                failed.append((label, type(e).__name__))
                if stop_at_first:
                    break
    finally:
        for m, o in zip(PIN_MODULES, saved):
            m.O = o
    return failed


def test_unmutated_copy_passes_every_pin():
    assert len(_cases()) >= 45
    assert _run_battery(_build(), stop_at_first=False) == []


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_the_mutant(name, old, new):
    failed = _run_battery(_build((old, new)))
    assert failed, f"no pin fails on the mutant: {name}"
    print(f"{name}: caught by {failed[0][0]} ({failed[0][1]})")
