"""Host-side logic of bench.py (no GPU): the dense-equivalent FLOP count, the
committed traffic profiles it reads, and the one-GPU guard."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_dense_equiv_flop_closed_form():
    # full prefill: query t attends t + 1 keys -> 4 C H_q N (N + 1) / 2
    n, h_q, c = 1000, 3, 64
    assert bench.dense_equiv_flop([n], [n], h_q, c) == 4.0 * c * h_q * n * (n + 1) / 2
    # chunked: the last n_q of n_kv tokens, query t attends n_c + t + 1 keys
    n_kv, n_q = 900, 100
    want = 4.0 * c * h_q * sum(n_kv - n_q + t + 1 for t in range(n_q))
    assert bench.dense_equiv_flop([n_kv], [n_q], h_q, c) == want
    # a batch is the sum of its requests
    assert bench.dense_equiv_flop([n, n_kv], [n, n_q], h_q, c) == pytest.approx(
        bench.dense_equiv_flop([n], [n], h_q, c) + want)


def test_committed_traffic_profiles_match_the_kernel_source():
    # every committed prefill traffic summary names the current source hash, so
    # the bench line reports measured HBM bytes for the kernel it times
    for wl in ("llama_128k", "llama_32k", "wide_64k", "paged_4x"):
        path = os.path.join(ROOT, "profiles", "prefill_" + wl.replace("_", "") + "_traffic.md")
        if not os.path.exists(path):
            continue
        traffic = bench.measured_traffic(wl)
        assert traffic is not None and traffic > 0, f"{wl}: stale or unreadable traffic profile"
    assert bench.measured_traffic("no_such_workload") is None


def test_source_hash_ignores_comments(tmp_path, monkeypatch):
    src = tmp_path / "paper_2605_12193_amd" / "csrc"
    src.mkdir(parents=True)
    (src / "bfla_device.h").write_text("int x;\n")
    (src / "prefill.hip").write_text("int f() { return 1; }  // one\n/* block */\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h1 = bench.prefill_source_hash()
    (src / "prefill.hip").write_text("// header\nint f() {\n  return 1;\n}\n")
    assert bench.prefill_source_hash() == h1
    (src / "prefill.hip").write_text("int f() { return 2; }\n")
    assert bench.prefill_source_hash() != h1


def test_more_than_one_gpu_is_refused():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert out.returncode == 2
    msg = json.loads(out.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_stage1_work_closed_form():
    # N_c = 0, N a multiple of b: L (L + 1) / 2 causal block pairs per query
    # head, G^2 group pairs each, 2 g C FLOP per group pair
    n, b, g, c, h_q, h_kv = 128 * 10, 128, 64, 128, 8, 2
    L, G = n // b, b // g
    flop, nbytes = bench.stage1_work([n], [n], h_q, h_kv, c, b, g)
    assert flop == 2.0 * g * c * G * G * h_q * L * (L + 1) // 2
    assert nbytes == 2.0 * c * (h_q + h_kv) * n


def test_stage1_work_counts_causal_pairs_by_brute_force():
    # chunked prefill and a ragged tail: a block pair is causal when the KV
    # block's first key is at or before the query block's last position
    b, g = 128, 64
    for n_kv, n_q in ((1000, 1000), (1000, 300), (777, 1)):
        n_c = n_kv - n_q
        pairs = 0
        for i in range(-(-n_q // b)):
            last = min(n_c + (i + 1) * b - 1, n_kv - 1)
            pairs += sum(1 for j in range(-(-n_kv // b)) if j * b <= last)
        flop, _ = bench.stage1_work([n_kv], [n_q], 1, 1, 64, b, g)
        assert flop == 2.0 * g * 64 * (b // g) ** 2 * pairs


def test_committed_score_traffic_matches_the_score_kernel_source():
    for wl in ("llama_128k", "llama_32k", "wide_64k", "paged_4x"):
        path = os.path.join(ROOT, "profiles", "prefill_" + wl.replace("_", "") + "_traffic.md")
        if not os.path.exists(path):
            continue
        t = bench.measured_traffic(wl, "traffic_bytes_scores")
        assert t is not None and t > 0, f"{wl}: stale or unreadable score-kernel traffic"


def _tiny_oracle_pass():
    import numpy as np
    import torch
    from oracle import bfla_oracle as O
    from paper_2605_12193_amd import synth
    wl = synth.workload("tiny_2k")
    seqs = synth.make_inputs(wl)
    n = seqs[0].q.shape[1]
    q, k, v = (t.double().numpy() for t in (seqs[0].q, seqs[0].k, seqs[0].v))
    alpha = O.default_scale(wl.head_dim)
    st = O.estimate_mask(q, k, wl.block, wl.group, wl.gamma, alpha)
    rp, cols, _ = O.expand_rescue([st["mask"]], [n], [n], wl.block, wl.tile, wl.n_local,
                                  wl.n_sink, wl.eta, wl.rho, wl.seed)
    o, _ = O.attention(q, k, v, wl.tile, alpha, rp, cols)

    class Inp:
        pass
    inp = Inp()
    inp.seqs, inp.n = seqs, [n]
    inp.out_rows = lambda oo, r, p, t0, t1: oo[p, t0:t1].numpy()
    return wl, inp, torch.from_numpy(o), st["mask"].reshape(-1).astype(np.uint8), rp, cols


def test_cpu_baseline_checks_masks_lists_and_outputs():
    # fed the oracle's own mask, lists and outputs as the "GPU" results, the
    # bench's oracle leg finds no mismatch; a flipped mask is a sure mismatch
    # on every sure cell, and a changed list is counted
    import numpy as np
    wl, inp, out, mask, rp, cols = _tiny_oracle_pass()
    cpu, err, m, lst = bench.cpu_baseline(wl, inp, out, mask, rp, cols, rows=16)
    assert m["cells"] == mask.size and m["sure_mismatch"] == 0 and m["tie_mismatch"] == 0
    assert lst["rows"] == len(rp) - 1 and lst["rows_differ"] == 0
    assert err["max_abs"] < 1e-12 and err["rows"] >= 16
    assert cpu["kind"] == "oracle" and cpu["extrapolated"] and cpu["value"] > 0
    assert cpu["attention_sample"]["of_kept_tiles"] == int(rp[-1])
    assert cpu["cores"] >= 1 and cpu["nproc"] >= 1 and cpu["cpu_model"]
    _, _, m2, _ = bench.cpu_baseline(wl, inp, out, 1 - mask, rp, cols, rows=4)
    assert m2["sure_mismatch"] == m2["cells"] - m2["tie_cells"] > 0
    cols2 = cols.copy()
    cols2[0] += 1
    _, _, _, lst2 = bench.cpu_baseline(wl, inp, out, mask, rp, cols2, rows=4)
    assert lst2["rows_differ"] == 1


def test_stratified_rows_cover_every_head_and_range():
    import numpy as np
    rng = np.random.default_rng(0)
    rows = bench.stratified_rows([131072], 8, 64, 256, rng)
    assert len(rows) == 256
    for h in range(8):
        qts = sorted(qt for r, hh, qt in rows if hh == h)
        assert len(qts) == 32
        # one q-tile in each of 32 equal ranges of the 2048 q-tiles
        assert [qt // 64 for qt in qts] == list(range(32))
    # a batch of requests of different lengths: every (request, head) pair
    rows = bench.stratified_rows([300, 5000], 2, 64, 20, rng)
    assert {(r, h) for r, h, _ in rows} == {(0, 0), (0, 1), (1, 0), (1, 1)}
    assert all(0 <= qt < -(-[300, 5000][r] // 64) for r, _, qt in rows)
