"""bfla_expand_rescue_noalloc (the tile stage with the library's fixed
per-device scratch, no allocation) against bfla_expand_rescue with a caller
workspace: the lists must be identical, bit for bit, on two calls in a row,
the second on a smaller problem than the first (the scratch keeps the first
call's contents), with the canary bands around every output intact."""
import numpy as np
import pytest
import torch

from paper_2605_12193_amd import bfla, synth
from parity_util import Guarded

pytestmark = pytest.mark.gpu

KW = dict(block=128, group=64, tile=64, gamma=0.9, n_local=2, n_sink=1, eta=16, rho=0.1,
          seed=31)


def _mask(prob, block, seed, density):
    """Seeded random block masks of every request, packed as Stage 1 writes them."""
    parts = []
    for r, (nq, nkv) in enumerate(zip(prob.n_q, prob.n_kv)):
        parts.append(synth.random_block_mask(seed + r, prob.c.h_kv, nq, nkv, block,
                                             density).ravel())
    return torch.from_numpy(np.concatenate(parts)).cuda()


def _lists(prob, prm, mask, noalloc):
    cap = bfla.bfla_list_capacity(prob, prm)
    rp = Guarded(cap.n_rows + 1, torch.int32, fill=-5)
    cols = Guarded(cap.max_cols, torch.int32, fill=-7)
    ws = None
    if noalloc:
        bfla.bfla_expand_rescue_noalloc(prob, prm, mask, rp.t, cols.t)
    else:
        ws = Guarded(bfla.bfla_workspace_size(prob, prm, bfla.BFLA_WS_EXPAND), torch.uint8)
        bfla.bfla_expand_rescue(prob, prm, mask, rp.t, cols.t, ws.t)
    torch.cuda.synchronize()
    rp.check("row_ptr")
    cols.check("cols")
    if ws is not None:
        ws.check("workspace")
    out = rp.t.cpu().numpy()
    return out, cols.t[:int(out[-1])].cpu().numpy()


@pytest.mark.parametrize("first,second", [
    # (lengths n_q, n_kv, h_q, h_kv) of the first call, then of a smaller second call
    ((([131072], [131072]), 32, 8), (([3000, 700], [3000, 1500]), 4, 2)),
    ((([16384, 32768, 65536, 131072], [16384, 32768, 65536, 131072]), 40, 8),
     (([64], [64]), 1, 1)),
], ids=["128k_then_batch", "paged4x_shape_then_one_tile"])
def test_noalloc_equals_workspace_entry_point(first, second):
    for i, ((n_q, n_kv), h_q, h_kv) in enumerate((first, second)):
        prob = bfla.Problem(n_q, n_kv, h_q, h_kv, 128)
        prm = bfla.params(**KW)
        mask = _mask(prob, KW["block"], 100 + i, 0.05 if i == 0 else 0.3)
        want_rp, want_cols = _lists(prob, prm, mask, noalloc=False)
        got_rp, got_cols = _lists(prob, prm, mask, noalloc=True)
        print(f"call {i + 1}: {len(want_rp) - 1} rows, {want_rp[-1]} kept tiles", flush=True)
        assert np.array_equal(got_rp, want_rp), f"call {i + 1}: row_ptr differs"
        assert np.array_equal(got_cols, want_cols), f"call {i + 1}: cols differ"
