"""Non-finite inputs through the C ABI: a NaN in one query row makes every
score and p~ of that row NaN. Only that row is flagged (non-finite) and only
its output changes: rows stay independent. In particular row i ^ 16, the
other 16-query half of the same 32-row block, keeps its flag clear and its
output bit for bit (its c / l sums must not see the NaN)."""
import numpy as np
import pytest
import torch

import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")

CASES = [W.Workload("nf_causal", 1, 2, 300, 300, 128, True, 128 ** -0.5, seed=31),
         W.Workload("nf_cross64", 1, 2, 130, 517, 64, False, 0.125, seed=32)]


def _bits(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy()


@pytest.mark.parametrize("w", CASES, ids=[c.name for c in CASES])
@pytest.mark.parametrize("row", [5, 100])
@pytest.mark.parametrize("check", [True, False, "twopass"])
def test_nan_query_row_stays_in_its_row(w, row, check):
    print(f"[nonfinite] {w.name} row {row} check {check}", flush=True)
    q, k, v = G.dev_inputs(W.make_inputs(w))
    qn = q.clone()
    qn[0, 1, row, 7] = float("nan")
    if check == "twopass":
        # the NaN row's first pass finds no finite max; its second pass stays NaN
        o0, r0, f0 = F.attn_fwd_twopass(q, k, v, causal=w.causal, scale=w.scale)
        o, r, f = F.attn_fwd_twopass(qn, k, v, causal=w.causal, scale=w.scale)
    elif check:
        o0, r0, f0 = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
        o, r, f = F.attn_fwd(qn, k, v, causal=w.causal, scale=w.scale)
    else:
        o0 = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale, check=False)
        o = F.attn_fwd(qn, k, v, causal=w.causal, scale=w.scale, check=False)
    torch.cuda.synchronize()
    if check:
        assert int(f0.sum()) == 0
        assert int(f[0, 1, row]) & F.FLAG_NONFINITE
        others = f.clone()
        others[0, 1, row] = 0
        assert int(others.sum()) == 0
        keep = np.ones(w.Lq, dtype=bool)
        keep[row] = False
        assert np.array_equal(r[0, 1].cpu().numpy()[keep].view(np.int32),
                              r0[0, 1].cpu().numpy()[keep].view(np.int32))
    keep = np.ones(w.Lq, dtype=bool)
    keep[row] = False
    assert np.array_equal(_bits(o[0, 1])[keep], _bits(o0[0, 1])[keep])
    assert np.array_equal(_bits(o[0, 0]), _bits(o0[0, 0]))
    assert torch.isnan(o[0, 1, row].float()).all()
