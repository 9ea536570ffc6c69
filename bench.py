"""Benchmark of the block-filtered sparse prefill hot path on one MI355X.

A step is one full pass of the path over one batch: Stage 1 (block scores,
keep-mass selection, GQA union) -> tile lists (expansion + rescue) -> fused
sparse prefill.  Inputs are seeded synthetic bf16 tensors already resident in
HBM.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload llama_128k|llama_32k|wide_64k|paged_4x|tiny_2k]

`value` is the dense-equivalent throughput 4 * C * H_q * sum_r N_r (N_r + 1) / 2
FLOP per step divided by the step time (the causal FlashAttention convention).
The roofline object reports the sparse prefill kernel (the dominant one):
4 * T^2 * C * m FLOP per kept (KV head, q-tile, kv-tile) tile over its average
launch time from HIP events on the launch stream, against the bf16 dense MFMA
peak.  cpu_baseline is the CPU oracle timed on a bounded random sample of
(request, KV head, q-tile) rows of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "sparse prefill ms + dense-equiv TFLOP/s at 32K/128K; speedup vs dense; rel-err"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama_128k")
    ap.add_argument("--gamma", type=float, default=None)
    ap.add_argument("--rho", type=float, default=None)
    ap.add_argument("--block", type=int, default=None, help="coarse block b")
    ap.add_argument("--group", type=int, default=None, help="flattening group g")
    ap.add_argument("--n-local", type=int, default=None)
    ap.add_argument("--eta", type=int, default=None)
    ap.add_argument("--dense-steps", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="time budget of the oracle sample")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, copy a buffer of this many MiB once (a dispatch "
                         "of known HBM traffic for scaling FETCH_SIZE / WRITE_SIZE)")
    return ap.parse_args()


PREFILL_SOURCES = ("paper_2605_12193_amd/csrc/prefill.hip", "paper_2605_12193_amd/csrc/bfla_device.h")
SCORES_SOURCES = ("paper_2605_12193_amd/csrc/estimate.hip", "paper_2605_12193_amd/csrc/bfla_device.h")


def prefill_source_hash(files=PREFILL_SOURCES) -> str:
    """Hash of a kernel's code (by default prefill.hip and the device header)
    with comments and whitespace removed, so only code changes invalidate a
    committed traffic profile."""
    m = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        m.update(" ".join(text.split()).encode())
    return m.hexdigest()[:16]


def measured_traffic(workload: str, key: str = "traffic_bytes_prefill_sparse"):
    """HBM bytes per launch of a kernel (the sparse prefill by default, or
    key="traffic_bytes_scores" for the Stage-1 score kernel) from the
    committed rocprofv3 counter summary, or None if there is none for this
    workload or that kernel's source changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "prefill_" + workload.replace("_", "") + "_traffic.md")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        parts = line.split()
        if len(parts) == 2:
            kv[parts[0]] = parts[1]
    if kv.get("workload") != workload:
        return None
    if key == "traffic_bytes_scores":
        if kv.get("scores_source_hash") != prefill_source_hash(SCORES_SOURCES):
            return None
    elif kv.get("source_hash") != prefill_source_hash():
        return None
    v = kv.get(key)
    return float(v) if v else None


def dense_equiv_flop(n_kv, n_q, h_q, c):
    """Causal: query t of a request attends N_c + t + 1 keys; 4 C FLOP per
    (query, key, head)."""
    tot = 0
    for nk, nq in zip(n_kv, n_q):
        tot += nq * (nk - nq) + nq * (nq + 1) // 2
    return 4.0 * c * h_q * tot


def stage1_work(n_kv, n_q, h_q, h_kv, c, b, g):
    """Algorithmic work of the Stage-1 score GEMM: 2 g C FLOP for each of the
    G^2 group pairs (G = b / g) of every causal (query block, KV block) pair
    of every query head (eq9-eq14), and Q and K read once (2 B per element)."""
    G = b // g
    pairs = 0
    for nk, nq in zip(n_kv, n_q):
        nc = nk - nq
        for i in range(-(-nq // b)):
            e = min(nc + (i + 1) * b - 1, nk - 1)
            pairs += e // b + 1
    flop = 2.0 * g * c * G * G * h_q * pairs
    nbytes = 2.0 * c * sum(h_q * nq + h_kv * nk for nk, nq in zip(n_kv, n_q))
    return flop, nbytes


class Inputs:
    """Device tensors and ABI views of one workload (contiguous head-first for a
    single request; vLLM-style pages and packed token-major Q/O for a batch)."""

    def __init__(self, wl, torch, bfla, synth):
        self.seqs = synth.make_inputs(wl)
        self.n = [s.q.shape[1] for s in self.seqs]
        dev = torch.device("cuda:0")
        self.paged = wl.page_size is not None
        self.prob = bfla.Problem(self.n, self.n, wl.h_q, wl.h_kv, wl.head_dim)
        if not self.paged:
            s = self.seqs[0]
            self.q = s.q.to(dev).contiguous()
            self.k = s.k.to(dev).contiguous()
            self.v = s.v.to(dev).contiguous()
            self.o = torch.empty_like(self.q)
            self.od = torch.empty_like(self.q)
            self.qv, self.ov, self.odv = (bfla.view_hnc(t) for t in (self.q, self.o, self.od))
            self.kv = bfla.KV(self.k, self.v)
        else:
            self.q = torch.cat([s.q.transpose(0, 1) for s in self.seqs], 0).contiguous().to(dev)
            self.o = torch.empty_like(self.q)
            self.od = torch.empty_like(self.q)
            self.starts = np.concatenate([[0], np.cumsum(self.n)[:-1]]).astype(int)
            table, total = synth.page_table(wl.seed, self.n, wl.page_size)
            kp, vp = synth.to_paged(self.seqs, table, total, wl.page_size)
            self.k, self.v = kp.to(dev), vp.to(dev)
            self.table = torch.from_numpy(table).to(dev)
            self.qv, self.ov, self.odv = (bfla.view_packed(t, self.starts)
                                          for t in (self.q, self.o, self.od))
            self.kv = bfla.KV(self.k, self.v, paged=True, block_table=self.table)

    def out_rows(self, o, r, p, t0, t1):
        """Rows [t0, t1) of query head p of request r of an output tensor (host float)."""
        if not self.paged:
            return o[p, t0:t1].float().cpu().numpy()
        a = int(self.starts[r])
        return o[a + t0:a + t1, p].float().cpu().numpy()


def cpu_baseline(wl, inp, gpu_o, budget_s, gpu_mask=None, seed=0):
    """Time the oracle on random (request, KV head, q-tile) rows: Stage 1 of
    the query block holding the q-tile (all m query heads of the KV head), the
    tile stage of that block row, and the sparse attention of the q-tile.
    Also returns the GPU-vs-oracle error on the sampled outputs and, given the
    GPU block mask (host uint8, the library's packed layout), its agreement
    with the oracle's mask on the sampled block rows: every sure cell must
    match; near-tie cells are counted, and so are the ones that differ."""
    from oracle import bfla_oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    T, b = wl.tile, wl.block
    m = wl.h_q // wl.h_kv
    alpha = O.default_scale(wl.head_dim)
    rng = np.random.default_rng(seed)
    rows = [(r, qt) for r, n in enumerate(inp.n) for qt in range(-(-n // T))]
    order = rng.permutation(len(rows))
    heads = rng.integers(0, wl.h_kv, len(rows))
    host = {}
    L = [-(-n // b) for n in inp.n]
    mask_off = np.concatenate([[0], np.cumsum([wl.h_kv * x * x for x in L])]).astype(np.int64)
    mchk = {"block_rows": 0, "blocks": 0, "sure_mismatch": 0, "tie_blocks": 0, "tie_mismatch": 0}
    seen = set()
    flop = 0.0
    max_abs, num, den = 0.0, 0.0, 0.0
    t0 = time.perf_counter()
    done = 0
    for idx in order:
        if time.perf_counter() - t0 >= budget_s:
            break
        r, qt = rows[idx]
        h = int(heads[idx])
        if r not in host:
            s = inp.seqs[r]
            host[r] = tuple(x.float().numpy() for x in (s.q, s.k, s.v))
        q, k, v = host[r]
        n = q.shape[1]
        done += 1
        i = qt // (b // T)
        st = O.estimate_mask(q[h * m:(h + 1) * m, i * b:(i + 1) * b].astype(np.float64),
                             k[h:h + 1, :min(n, (i + 1) * b)].astype(np.float64), b,
                             wl.group, wl.gamma, alpha)
        bm = np.zeros((-(-n // b), -(-n // b)), np.uint8)
        bm[i, :st["mask"].shape[2]] = st["mask"][0, 0]
        if gpu_mask is not None and (r, h, i) not in seen:
            seen.add((r, h, i))
            lr = L[r]
            row0 = int(mask_off[r]) + (h * lr + i) * lr
            got = gpu_mask[row0:row0 + st["mask"].shape[2]]
            want, status = st["mask"][0, 0], st["status"][0, 0]
            tie = status == O.TIE
            mchk["block_rows"] += 1
            mchk["blocks"] += int(want.size)
            mchk["sure_mismatch"] += int(np.sum((got != want) & ~tie))
            mchk["tie_blocks"] += int(np.sum(tie))
            mchk["tie_mismatch"] += int(np.sum((got != want) & tie))
        tm = O.tile_mask(bm, n, n, b, T, wl.n_local, wl.n_sink, wl.eta, wl.rho, wl.seed, h)
        tiles = np.flatnonzero(tm[qt])
        for pp in range(m):
            o, _ = O.attention_rows(q, k, v, h * m + pp, qt, T, alpha, tiles)
            g = inp.out_rows(gpu_o, r, h * m + pp, qt * T, qt * T + o.shape[0])
            max_abs = max(max_abs, float(np.abs(g - o).max()))
            num += float(((g - o) ** 2).sum())
            den += float((o ** 2).sum())
        t_rows = np.arange(qt * T, min(n, (qt + 1) * T))
        flop += 4.0 * wl.head_dim * m * float((t_rows + 1).sum())
    dt = time.perf_counter() - t0
    return {
        "value": flop / dt / 1e12, "unit": "TFLOP/s (dense-equivalent)", "cores": int(cores),
        "kind": "oracle",
        "sample": (f"{done} random (request, KV head, q-tile) rows of {len(rows) * wl.h_kv}: "
                   f"oracle Stage 1 of each row's query block (m={m} heads), its tile stage "
                   f"and the row's sparse attention; {dt:.1f} s; value = dense-equivalent "
                   f"FLOP of the sampled rows / oracle time"),
        "seconds": dt,
    }, {"max_abs": max_abs, "rel_l2": math.sqrt(num / max(den, 1e-30))}, mchk


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this library runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch
    from paper_2605_12193_amd import bfla, synth

    over = {}
    if args.gamma is not None:
        over["gamma"] = args.gamma
    if args.rho is not None:
        over["rho"] = args.rho
    for key, val in (("block", args.block), ("group", args.group), ("n_local", args.n_local),
                     ("eta", args.eta)):
        if val is not None:
            over[key] = val
    wl = synth.workload(args.workload, **over)
    t_gen = time.perf_counter()
    torch.cuda.set_device(0)
    inp = Inputs(wl, torch, bfla, synth)
    t_gen = time.perf_counter() - t_gen
    log(f"{wl.name}: inputs ready in {t_gen:.1f} s")
    prob = inp.prob
    prm = bfla.params(block=wl.block, group=wl.group, tile=wl.tile, gamma=wl.gamma,
                      n_local=wl.n_local, n_sink=wl.n_sink, eta=wl.eta, rho=wl.rho,
                      seed=wl.seed)
    buf = bfla.Buffers(prob, prm)
    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def step(marks=None):
        if marks:
            marks[0].record(stream)
        bfla.bfla_estimate_mask(prob, prm, inp.qv, inp.kv, buf.block_mask, dbg_scores=buf.scores)
        if marks:
            marks[1].record(stream)
        bfla.bfla_expand_rescue(prob, prm, buf.block_mask, buf.row_ptr, buf.cols, buf.ws_expand)
        if marks:
            marks[2].record(stream)
        bfla.bfla_sparse_prefill(prob, prm, inp.qv, inp.kv, buf.row_ptr, buf.cols, inp.ov,
                                 buf.lse)
        if marks:
            marks[3].record(stream)

    # first pass: validate the lists on the host before timing anything
    bfla.bfla_estimate_mask(prob, prm, inp.qv, inp.kv, buf.block_mask, dbg_scores=buf.scores)
    bfla.bfla_expand_rescue(prob, prm, buf.block_mask, buf.row_ptr, buf.cols, buf.ws_expand)
    torch.cuda.synchronize()
    rp = buf.row_ptr.cpu().numpy()
    cols_h = buf.cols[:int(rp[-1])].cpu().numpy()
    assert rp[0] == 0 and np.all(np.diff(rp) >= 0)
    row = 0
    for n in inp.n:
        rows = wl.h_kv * -(-n // wl.tile)
        seg = cols_h[rp[row]:rp[row + rows]]
        assert np.all((seg >= 0) & (seg < -(-n // wl.tile)))
        row += rows
    log(f"lists valid: {int(rp[-1])} kept tiles")

    for _ in range(args.warmup):
        step()
    marks = [[ev() for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start, end = ev(), ev()
    start.record(stream)
    for i in range(args.steps):
        step(marks[i])
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(end) / args.steps
    per_step = {name: [m[i].elapsed_time(m[i + 1]) for m in marks]
                for i, name in enumerate(("estimate_mask", "expand_rescue", "sparse_prefill"))}
    st1 = float(np.mean(per_step["estimate_mask"]))
    exp_ms = float(np.mean(per_step["expand_rescue"]))
    pre_ms = float(np.mean(per_step["sparse_prefill"]))
    log(f"timed {args.steps} steps: {ms_step:.3f} ms/step")

    # dense baseline (same kernel family, every causal tile)
    bfla.bfla_dense_prefill(prob, prm, inp.qv, inp.kv, inp.odv)
    torch.cuda.synchronize()
    dm = [(ev(), ev()) for _ in range(args.dense_steps)]
    for a, b in dm:
        a.record(stream)
        bfla.bfla_dense_prefill(prob, prm, inp.qv, inp.kv, inp.odv)
        b.record(stream)
    torch.cuda.synchronize()
    dense_ms = float(np.mean([a.elapsed_time(b) for a, b in dm]))
    log(f"dense {dense_ms:.3f} ms")
    if args.calib_copy_mib > 0:
        nbytes = args.calib_copy_mib << 20
        src = torch.ones(nbytes, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {args.calib_copy_mib} MiB done")
        del src, dst

    kept = int(rp[-1])
    causal_tiles = sum(wl.h_kv * t * (t + 1) // 2 for t in (-(-n // wl.tile) for n in inp.n))
    m = wl.h_q // wl.h_kv
    flop_dense = dense_equiv_flop(inp.n, inp.n, wl.h_q, wl.head_dim)
    flop_kept = 4.0 * wl.tile * wl.tile * wl.head_dim * m * kept
    achieved = flop_kept / (pre_ms * 1e-3) / 1e12
    num = den = 0.0
    for x in range(0, inp.q.shape[0], 4096):   # chunked to bound temporaries
        a = inp.o[x:x + 4096].float()
        b = inp.od[x:x + 4096].float()
        num += float(torch.sum((a - b) ** 2))
        den += float(torch.sum(b ** 2))
    sd_err = math.sqrt(num / max(den, 1e-30))

    # Stage 1 (estimate_mask: score GEMM + selection) against both rooflines:
    # algorithmic FLOP over its time vs the MFMA peak, and the score kernel's
    # measured HBM bytes (committed rocprofv3 counters) over the same time vs
    # the HBM peak (a lower bound on the kernel's own rate, since the stage
    # time also holds the selection kernel)
    f1, b1 = stage1_work(inp.n, inp.n, wl.h_q, wl.h_kv, wl.head_dim, wl.block, wl.group)
    t1 = measured_traffic(wl.name, "traffic_bytes_scores")
    hbm_bytes = t1 if t1 is not None else b1
    stage1 = {"kernels": "scores_kernel + select_kernel (bfla_estimate_mask)",
              "ms": round(st1, 4), "flop": f1,
              "achieved_tflops": round(f1 / (st1 * 1e-3) / 1e12, 2),
              "mfma_frac": round(f1 / (st1 * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
              "algorithmic_bytes": b1, "traffic": t1,
              "hbm_gbs": round(hbm_bytes / (st1 * 1e-3) / 1e9, 1),
              "hbm_bytes_source": "rocprofv3 FETCH+WRITE (profiles/)" if t1 is not None
              else "algorithmic (Q and K once)",
              "hbm_frac": round(hbm_bytes / (st1 * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
              "arithmetic_intensity": round(f1 / b1, 1),
              "bound": "mfma" if f1 / b1 > PEAK_BF16_TFLOPS / PEAK_HBM_GBS * 1e3 else "hbm"}

    traffic = measured_traffic(wl.name)

    config = {"workload": wl.name, "seq_lens": inp.n, "h_q": wl.h_q, "h_kv": wl.h_kv,
              "head_dim": wl.head_dim, "block": wl.block, "group": wl.group,
              "tile": wl.tile, "gamma": wl.gamma, "n_local": wl.n_local,
              "n_sink": wl.n_sink, "eta": wl.eta, "rho": wl.rho, "seed": wl.seed}
    if inp.paged:
        config["kv_layout"] = f"paged, {wl.page_size}-token pages, seeded block table"
    result = {
        "metric": METRIC,
        "value": round(flop_dense / (ms_step * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s (dense-equivalent)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) with planted sinks and heavy hitters)",
        "config": config,
        "stage_ms": {"estimate_mask": round(st1, 3), "expand_rescue": round(exp_ms, 3),
                     "sparse_prefill": round(pre_ms, 3)},
        "stage_ms_min_median_max": {k: [round(float(np.min(v)), 3), round(float(np.median(v)), 3),
                                        round(float(np.max(v)), 3)] for k, v in per_step.items()},
        "dense_ms": round(dense_ms, 3),
        "dense_tflops": round(flop_dense / (dense_ms * 1e-3) / 1e12, 2),
        "speedup_vs_dense": round(dense_ms / ms_step, 3),
        "keep_ratio": round(kept / causal_tiles, 5),
        "kept_tiles": kept,
        "sparse_vs_dense_rel_l2": round(sd_err, 5),
        "roofline": {"bound": "mfma", "kernel": "prefill_kernel (sparse)",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic,
                     "flop_per_launch": flop_kept,
                     "launch_ms": round(pre_ms, 3),
                     # the other roofline: measured HBM bytes over the same launch time
                     "hbm_gbs": None if traffic is None else round(traffic / (pre_ms * 1e-3) / 1e9, 1),
                     "hbm_frac": None if traffic is None else
                     round(traffic / (pre_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)},
        "stage1_roofline": stage1,
        "wall_s_timed": round(wall, 3),
        "input_gen_s": round(t_gen, 1),
    }
    if not args.no_cpu:
        cpu, err, mchk = cpu_baseline(wl, inp, inp.o, args.cpu_seconds,
                                      gpu_mask=buf.block_mask.cpu().numpy())
        log(f"cpu baseline {cpu['seconds']:.1f} s")
        result["cpu_baseline"] = {kk: vv for kk, vv in cpu.items() if kk != "seconds"}
        result["rel_err_vs_oracle_sampled"] = {kk: round(vv, 6) for kk, vv in err.items()}
        result["mask_vs_oracle_sampled"] = mchk
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
