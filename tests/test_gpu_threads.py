"""The library keeps no shared mutable state beyond a once-per-device launch
attribute, so host threads may drive it concurrently: two threads, each
with its own stream and buffers, run whole sparse passes (Stage 1, tile
lists, sparse prefill) and dense prefills at the same time, with different
kernel shapes; every result equals the single-threaded pass bit for bit."""
import threading

import pytest
import torch

from paper_2605_12193_amd import bfla, synth

pytestmark = pytest.mark.gpu

CASES = [(8, 2, 128, 4096 + 19, 5), (4, 2, 256, 2048 + 64, 6), (10, 2, 128, 3072 + 1, 7)]


class Job:
    def __init__(self, h_q, h_kv, c, n, seed):
        wl = synth.workload("tiny_2k", h_q=h_q, h_kv=h_kv, head_dim=c, seed=seed)
        s = synth.make_inputs(wl, seqlens=[n])[0]
        self.q, self.k, self.v = (t.cuda().contiguous() for t in (s.q, s.k, s.v))
        self.o = torch.empty_like(self.q)
        self.od = torch.empty_like(self.q)
        self.prob = bfla.Problem([n], [n], h_q, h_kv, c)
        self.prm = bfla.params(block=128, group=64, tile=64, gamma=0.9, n_local=2, n_sink=1,
                               eta=16, rho=0.1, seed=seed)
        self.buf = bfla.Buffers(self.prob, self.prm)
        self.qv, self.ov, self.odv = (bfla.view_hnc(t) for t in (self.q, self.o, self.od))
        self.kv = bfla.KV(self.k, self.v)

    def run(self, stream, reps=1):
        with torch.cuda.stream(stream):
            for _ in range(reps):
                bfla.sparse_pass(self.prob, self.prm, self.qv, self.kv, self.ov, self.buf,
                                 stream=stream)
                bfla.bfla_dense_prefill(self.prob, self.prm, self.qv, self.kv, self.odv,
                                        stream=stream)
        stream.synchronize()

    def result(self):
        rp = self.buf.row_ptr.clone()
        return (self.o.clone(), self.od.clone(), self.buf.lse.clone(), rp,
                self.buf.cols[:int(rp[-1])].clone())


def test_concurrent_threads_match_single_threaded():
    jobs = [Job(*c) for c in CASES]
    want = []
    for j in jobs:
        j.run(torch.cuda.current_stream())
        want.append(j.result())
    for j in jobs:
        j.o.fill_(float("nan"))
        j.od.fill_(float("nan"))
        j.buf.lse.fill_(float("nan"))
    torch.cuda.synchronize()

    errors = []

    def worker(j):
        try:
            j.run(torch.cuda.Stream(), reps=3)
        except Exception as e:  # reported below
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(j,)) for j in jobs]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    for i, (j, w) in enumerate(zip(jobs, want)):
        got = j.result()
        for name, a, b in zip(("O", "dense O", "LSE", "row_ptr", "cols"), got, w):
            assert torch.equal(a, b), f"case {i}: {name} differs from the single-threaded pass"
