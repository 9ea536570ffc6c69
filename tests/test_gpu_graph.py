"""The three entry points only launch kernels on the caller's stream (no
allocation, memset, copy or synchronisation), so a whole sparse pass can be
captured into a HIP graph and replayed.  Each replay runs on fresh input
contents with eager work and synchronisations in between, and must equal an
eager pass on the same inputs bit for bit (the kernels are deterministic)."""
import pytest
import torch

from paper_2605_12193_amd import bfla, synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("h_q,h_kv,c", [(8, 2, 128), (4, 2, 256), (10, 2, 128), (6, 2, 256)],
                         ids=["pingpong_gqa4", "wide_c256", "half_tile_gqa5", "q16_c256_gqa3"])
def test_sparse_pass_graph_replays_match_eager(h_q, h_kv, c):
    n = 4608 + 37
    prob = bfla.Problem([n], [n], h_q, h_kv, c)
    prm = bfla.params(block=128, group=64, tile=64, gamma=0.9, n_local=2, n_sink=1, eta=16,
                      rho=0.1, seed=3)
    q = torch.empty(h_q, n, c, dtype=torch.bfloat16, device="cuda")
    k = torch.empty(h_kv, n, c, dtype=torch.bfloat16, device="cuda")
    v = torch.empty_like(k)
    o = torch.empty_like(q)
    qv, ov, kv = bfla.view_hnc(q), bfla.view_hnc(o), bfla.KV(k, v)
    buf = bfla.Buffers(prob, prm)

    def fill(seed):
        wl = synth.workload("tiny_2k", h_q=h_q, h_kv=h_kv, head_dim=c, seed=seed)
        s = synth.make_inputs(wl, seqlens=[n])[0]
        q.copy_(s.q)
        k.copy_(s.k)
        v.copy_(s.v)

    def eager(seed):
        fill(seed)
        bfla.sparse_pass(prob, prm, qv, kv, ov, buf)
        torch.cuda.synchronize()
        rp = buf.row_ptr.clone()
        return o.clone(), buf.lse.clone(), rp, buf.cols[:int(rp[-1])].clone()

    want = {s: eager(s) for s in (31, 32, 33)}

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        bfla.sparse_pass(prob, prm, qv, kv, ov, buf)
    torch.cuda.synchronize()

    for rep, s in enumerate((31, 32, 33)):
        fill(s)
        o.fill_(float("nan"))
        buf.lse.fill_(float("nan"))
        junk = torch.randn(1 << 20, device="cuda") * 2  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        w_o, w_lse, w_rp, w_cols = want[s]
        assert torch.equal(o, w_o), f"replay {rep}: O differs from the eager pass"
        assert torch.equal(buf.lse, w_lse), f"replay {rep}: LSE differs"
        assert torch.equal(buf.row_ptr, w_rp), f"replay {rep}: row_ptr differs"
        assert torch.equal(buf.cols[:int(w_rp[-1])], w_cols), f"replay {rep}: lists differ"
        del junk
