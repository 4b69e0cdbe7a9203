"""sjd_verify_noalloc (the verification entry point that allocates nothing,
for callers that cannot call hipMalloc) against sjd_verify through the C
ABI: bit-identical outputs on two calls in a row, the second with a smaller
input, and one call at the scratch's full size."""
import numpy as np
import pytest
import torch

import paper_2603_18599_amd as sjd
from paper_2603_18599_amd.sjd import SJD_VERIFY_NOALLOC_MAX_ROWS, verify_outputs
from synth_inputs import verify_inputs

pytestmark = pytest.mark.gpu


def _both(inp, K, D, top_k, seed, step):
    res = []
    for noalloc in (False, True):
        B, L, V = inp["cur"].shape
        out = verify_outputs(B, L, K, D)
        rows = torch.full((B, L, 2), -7, dtype=torch.int32, device="cuda")
        sjd.sjd_verify(inp["cur"], inp["draft"], inp["draft_tok"], inp["meta"], out, K=K, D=D, top_k=top_k,
                       seed=seed, step=step, sib=inp["sib"], out_rows=rows, noalloc=noalloc)
        torch.cuda.synchronize()
        res.append({**{k: v.cpu().numpy() for k, v in out.items()}, "rows": rows.cpu().numpy()})
    return res


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_verify_equals_verify(order):
    cases = [(64, 32, 16384, 2000, 0), (8, 16, 4096, 100, 2)]  # (B, L, V, top_k, D_in)
    for i, (B, L, V, top_k, D_in) in enumerate(cases):
        inp = verify_inputs(B, L, V, top_k=top_k, seed=40 + i, D_in=D_in, device="cuda")
        print(f"noalloc call {i}: B={B} L={L} V={V} top_k={top_k} D_in={D_in}", flush=True)
        a, b = _both(inp, 4, 3, top_k, seed=9 + i, step=i)
        for k in a:
            assert np.array_equal(a[k], b[k]), (i, k)
        assert (a["meta"][:, 0] >= 1).all()


def test_noalloc_verify_at_its_row_limit():
    L = 32
    B = SJD_VERIFY_NOALLOC_MAX_ROWS // L
    inp = verify_inputs(B, L, 64, top_k=0, seed=77, device="cuda")
    print(f"noalloc at the limit: B={B} L={L} V=64", flush=True)
    a, b = _both(inp, 4, 3, 0, seed=3, step=1)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
