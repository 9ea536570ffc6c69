"""The whole path driven from a plain C program through include/bfla.h (no
Python binding, no torch in that process): its block mask against the
oracle on sure cells, its lists against the oracle's tile stage on that
mask, its sparse and dense outputs and LSE against the oracle's attention."""
import os
import subprocess

import numpy as np
import pytest
import torch

from oracle import bfla_oracle as O
from paper_2605_12193_amd import synth
from parity_util import compare_outputs, mask_compare
from test_c_abi import DRIVER, build_driver

pytestmark = pytest.mark.gpu


def _bf16_to_f64(raw: np.ndarray) -> np.ndarray:
    return (raw.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("n,h_q,h_kv,c", [(700, 8, 2, 128), (333, 4, 4, 64)])
def test_c_program_matches_oracle(n, h_q, h_kv, c, tmp_path):
    driver = DRIVER if os.path.exists(DRIVER) else build_driver()
    wl = synth.workload("tiny_2k", h_q=h_q, h_kv=h_kv, head_dim=c, seed=41 + n)
    s = synth.make_inputs(wl, seqlens=[n])[0]
    raw = [t.contiguous().view(torch.int16).numpy().view(np.uint16) for t in (s.q, s.k, s.v)]
    inp, out = tmp_path / "in.bin", tmp_path / "out.bin"
    inp.write_bytes(b"".join(x.tobytes() for x in raw))
    r = subprocess.run([driver, str(inp), str(out), str(n), str(h_q), str(h_kv), str(c)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert "c driver ok" in r.stdout

    buf = out.read_bytes()
    mask_bytes, n_rows, n_cols = np.frombuffer(buf[:24], np.int64)
    off = 24
    def take(dtype, count):
        nonlocal off
        a = np.frombuffer(buf, dtype, count=int(count), offset=off)
        off += a.nbytes
        return a
    mask = take(np.uint8, mask_bytes)
    row_ptr = take(np.int32, n_rows + 1)
    cols = take(np.int32, n_cols)
    o_sparse = _bf16_to_f64(take(np.uint16, h_q * n * c)).reshape(h_q, n, c)
    lse = take(np.float32, h_q * n).reshape(h_q, n)
    o_dense = _bf16_to_f64(take(np.uint16, h_q * n * c)).reshape(h_q, n, c)
    assert off == len(buf)

    q, k, v = (x.double().numpy() for x in (s.q, s.k, s.v))
    alpha = O.default_scale(c)
    st = O.estimate_mask(q, k, 128, 64, 0.9, alpha)
    gm = mask.reshape(st["mask"].shape)
    mask_compare(gm, st["mask"], st["status"])
    rp, cl, _ = O.expand_rescue([gm], [n], [n], 128, 64, 2, 1, 16, 0.1, 7)
    assert np.array_equal(row_ptr, rp) and np.array_equal(cols, cl)
    want, want_lse = O.attention(q, k, v, 64, alpha, rp, cl, 0)
    compare_outputs(o_sparse, want, "C program, sparse")
    np.testing.assert_allclose(lse, want_lse, rtol=0, atol=2e-4)
    want_d, _ = O.attention(q, k, v, 64, alpha)
    compare_outputs(o_dense, want_d, "C program, dense")
