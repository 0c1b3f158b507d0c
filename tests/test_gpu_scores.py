"""The score check (an extension): fault-free runs flag nothing and leave O
bitwise unchanged; a flipped exponent bit of a score in a full key tile
sets FLAG_SCORES, which the output checksum alone cannot see; so does a q
register fault that lands after the first key tile. A q fault present from
the start, or a score fault in a masked diagonal tile, is not covered."""
import numpy as np
import pytest
import torch

import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")

CASES = [W.Workload("s_causal", 2, 3, 300, 300, 128, True, 128 ** -0.5, seed=21),
         W.Workload("s_rect64", 1, 2, 130, 517, 64, False, 0.125, seed=22),
         W.Workload("s_d96", 1, 2, 200, 333, 96, True, 96 ** -0.5, seed=23),
         W.Workload("s_ragged", 1, 2, 77, 77, 128, True, 128 ** -0.5, seed=24)]


@pytest.fixture
def score_check():
    ws = torch.empty(8 << 20, dtype=torch.uint8, device="cuda")
    F.set_score_check(ws)
    yield ws
    F.set_score_check(None)


@pytest.mark.parametrize("w", CASES, ids=[c.name for c in CASES])
def test_fault_free_and_output_unchanged(w, score_check):
    print(f"[scores] {w.name}", flush=True)
    q, k, v = G.dev_inputs(W.make_inputs(w))
    o, r, f = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
    oi, ri, fi, _, _ = F.attn_fwd_inject(q, k, v, causal=w.causal, scale=w.scale)
    F.set_score_check(None)
    o0, r0, f0 = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
    F.set_score_check(score_check)
    torch.cuda.synchronize()
    assert int(f.sum()) == 0 and int(fi.sum()) == 0
    assert torch.equal(o.view(torch.int16), o0.view(torch.int16))
    assert torch.equal(r.view(torch.int32), r0.view(torch.int32))
    assert torch.equal(oi.view(torch.int16), o0.view(torch.int16))


def test_score_faults_in_full_tiles_are_flagged(score_check):
    w = CASES[0]
    q, k, v = G.dev_inputs(W.make_inputs(w))
    # row 250, key 10 (tile 0: full for the wave of rows 224..255)
    caught, caught_off = 0, 0
    for bit in range(23, 31):
        f = F.Fault("S", b=1, h=2, row=250, col=10, bit=bit)
        o, r, fl, _, _ = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale, fault=f)
        torch.cuda.synchronize()
        caught += int((int(fl[1, 2, 250]) & F.FLAG_SCORES) != 0)
        others = fl.clone()
        others[1, 2, 250] = 0
        assert int(others.sum()) == 0
    assert caught == 8
    F.set_score_check(None)
    for bit in range(23, 31):
        f = F.Fault("S", b=1, h=2, row=250, col=10, bit=bit)
        o, r, fl, _, _ = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale, fault=f)
        torch.cuda.synchronize()
        caught_off += int((int(fl[1, 2, 250]) & F.FLAG_SCORES) != 0)
    F.set_score_check(score_check)
    assert caught_off == 0


def test_not_covered_q_and_diagonal(score_check):
    w = CASES[0]
    q, k, v = G.dev_inputs(W.make_inputs(w))
    # the score of key 250 for row 250 sits in the masked diagonal tile
    f = F.Fault("S", b=0, h=0, row=250, col=250, bit=24)
    o, r, fl, _, _ = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale, fault=f)
    torch.cuda.synchronize()
    assert (int(fl[0, 0, 250]) & F.FLAG_SCORES) == 0
    # a q register fault present from the first tile on changes both sides
    # of the score check alike ...
    f = F.Fault("Q", b=0, h=0, row=250, col=3, tile=0, bit=10)
    o, r, fl, _, _ = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale, fault=f)
    torch.cuda.synchronize()
    assert int(fl.sum()) == 0
    # ... but one that lands later is caught: the scores of the earlier full
    # tiles used the old q, the right-hand side uses the final one
    f = F.Fault("Q", b=0, h=0, row=250, col=3, tile=1, bit=10)
    o, r, fl, _, _ = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale, fault=f)
    torch.cuda.synchronize()
    assert int(fl[0, 0, 250]) == F.FLAG_SCORES
    assert int(fl.sum()) == F.FLAG_SCORES


def test_workspace_too_small_is_rejected():
    w = CASES[0]
    q, k, v = G.dev_inputs(W.make_inputs(w))
    need = F.score_check_workspace_bytes(w.B, w.H, w.Lk, w.d)
    ws = torch.empty(need - 16, dtype=torch.uint8, device="cuda")
    F.set_score_check(ws)
    try:
        with pytest.raises(F.FabftError):
            F.attn_fwd(q, k, v, causal=True, scale=w.scale)
    finally:
        F.set_score_check(None)
