"""Recompute on flag through the C ABI: after a transient fault in one forward,
re-running the checked forward on the flagged heads alone restores O, the
residuals and the flags of a fault-free run bit for bit (the kernel is
deterministic for a given head), leaves unflagged heads untouched, and a head
that stays flagged is reported as persistent."""
import numpy as np
import pytest
import torch

import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")

CASES = [W.Workload("rc_causal", 2, 3, 300, 300, 128, True, 128 ** -0.5, seed=11),
         W.Workload("rc_cross", 1, 4, 130, 517, 64, False, 0.125, seed=12)]


def _bits(t):
    return t.detach().contiguous().view(torch.int16).cpu().numpy()


@pytest.mark.parametrize("w", CASES, ids=[c.name for c in CASES])
def test_recompute_restores_clean_run(w):
    print(f"[recompute] {w.name}", flush=True)
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    o0, r0, f0 = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
    torch.cuda.synchronize()
    assert int(f0.sum()) == 0
    # a P-site flip of the top exponent bit in head (b=0, h=1) is flagged in its row
    row = min(100, w.Lq - 1)
    fault = F.Fault("P", b=0, h=1, row=row, col=5, tile=0, bit=14)
    o, r, f, _, _ = F.attn_fwd_inject(q, k, v, causal=w.causal, scale=w.scale, fault=fault)
    torch.cuda.synchronize()
    assert int(f[0, 1, row]) & F.FLAG_RESID
    # plant a second, host-side corruption in the last head and flag it
    o[-1, -1, 3] = o[-1, -1, 3] * 2 + 1
    f[-1, -1, 3] = F.FLAG_RESID
    untouched = _bits(o[0, 0])
    nrec, npers = F.recompute_flagged(q, k, v, o, r, f, causal=w.causal, scale=w.scale)
    torch.cuda.synchronize()
    assert (nrec, npers) == (2, 0)
    assert np.array_equal(_bits(o), _bits(o0))
    assert np.array_equal(r.cpu().numpy().view(np.int32), r0.cpu().numpy().view(np.int32))
    assert int(f.sum()) == 0
    assert np.array_equal(_bits(o[0, 0]), untouched)


def test_recompute_nothing_flagged_is_a_noop():
    w = CASES[0]
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    o, r, f = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
    before = _bits(o)
    assert F.recompute_flagged(q, k, v, o, r, f, causal=w.causal, scale=w.scale) == (0, 0)
    assert np.array_equal(_bits(o), before)


def test_recompute_reports_persistent_heads():
    """With a zero threshold every row whose residual is not exactly zero
    flags on every run, so those heads never clear."""
    w = CASES[1]
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    old = F.get_threshold()
    try:
        F.set_threshold(0.0, 0.0)
        o, r, f = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
        torch.cuda.synchronize()
        heads = (f.view(w.B * w.H, -1).amax(dim=1) > 0).cpu().numpy()
        assert heads.sum() > 0
        nrec, npers = F.recompute_flagged(q, k, v, o, r, f, causal=w.causal, scale=w.scale,
                                          max_retries=3)
        assert (nrec, npers) == (0, int(heads.sum()))
    finally:
        F.set_threshold(*old)
    # O itself is still the fault-free result
    ref = G.oracle_rows(inp, w.causal, w.scale)
    G.compare(o, torch.zeros_like(r), {"O": ref["O"], "pred": np.zeros_like(ref["pred"])}, w.d)
