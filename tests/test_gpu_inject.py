"""Fault-injection path on the GPU: single bit flips at the S, P, O and V
sites change O only where they should, and the per-row check flags the rows
whose output moved by more than the threshold (P, O, V); S-site flips before
the checksum tap change O and pred consistently."""
import numpy as np
import pytest
import torch

import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")

W_INJ = W.Workload("inject", 1, 2, 300, 300, 128, True, 128 ** -0.5, seed=7)


@pytest.fixture(scope="module")
def golden():
    inp = W.make_inputs(W_INJ)
    q, k, v = G.dev_inputs(inp)
    out = F.attn_fwd_inject(q, k, v, causal=True, scale=W_INJ.scale)
    torch.cuda.synchronize()
    assert int(out[2].sum()) == 0
    return (q, k, v), out


def _inject(golden, fault):
    (q, k, v), _ = golden
    print(f"[inject] {fault}", flush=True)
    out = F.attn_fwd_inject(q, k, v, causal=True, scale=W_INJ.scale, fault=fault)
    torch.cuda.synchronize()
    return out


def _changed_rows(a, b):
    d = (a.view(torch.int16) != b.view(torch.int16)).any(dim=-1)
    return set(map(tuple, d.nonzero().cpu().numpy().tolist()))


def test_no_fault_matches_production(golden):
    (q, k, v), (o, resid, flags, pred, actual) = golden
    o2, r2, f2 = F.attn_fwd(q, k, v, causal=True, scale=W_INJ.scale)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(resid.view(torch.int32), r2.view(torch.int32))
    # resid is pred - actual (the kernel may fuse c*(1/l) - actual into one FMA)
    diff = (resid - (pred - actual)).abs()
    assert bool((diff <= 2.0 ** -22 * (pred.abs() + actual.abs())).all())


@pytest.mark.parametrize("bit", [30, 27, 23])
def test_o_site_flip(golden, bit):
    f = F.Fault("O", b=0, h=1, row=200, col=37, tile=2, bit=bit)
    o, resid, flags, pred, actual = _inject(golden, f)
    (_, (o0, r0, f0, p0, a0)) = golden
    changed = _changed_rows(o, o0)
    assert changed <= {(0, 1, 200)}
    # pred does not see an output-accumulator fault
    assert torch.equal(pred, p0)
    others = flags.clone()
    others[0, 1, 200] = 0
    assert int(others.sum()) == 0
    if bit == 30:
        # the top exponent bit moves o_ij by a factor 2^128 (or from 0 to 2)
        assert changed == {(0, 1, 200)}
        assert int(flags[0, 1, 200]) != 0


def test_p_site_flip(golden):
    f = F.Fault("P", b=0, h=0, row=250, col=100, bit=14)
    o, resid, flags, pred, actual = _inject(golden, f)
    (_, (o0, r0, f0, p0, a0)) = golden
    assert _changed_rows(o, o0) == {(0, 0, 250)}
    assert int(flags[0, 0, 250]) != 0
    assert int(flags.sum()) == int(flags[0, 0, 250])


def test_p_exponent_msb_flips_on_short_rows_are_flagged(golden):
    """Flipping the top exponent bit of p~ in the first key tile of a short
    row scales it by 2^128: O stays finite in bf16 but sum_j |O_ij| overflows
    fp32, which would make the threshold infinite. Every such row must still
    be flagged."""
    (_, (o0, r0, f0, p0, a0)) = golden
    row = 20
    for key in range(0, row + 1, 3):
        f = F.Fault("P", b=0, h=1, row=row, col=key, bit=14)
        o, resid, flags, pred, actual = _inject(golden, f)
        assert _changed_rows(o, o0) == {(0, 1, row)}, key
        assert int(flags[0, 1, row]) & F.FLAG_RESID, (key, float(resid[0, 1, row]))


def test_v_site_flip(golden):
    # key 100, column 5, in the workgroup holding the second query tile
    qt = F.query_tile(W_INJ.d)
    lo, hi = qt, min(2 * qt, W_INJ.Lq)
    f = F.Fault("V", b=0, h=1, row=100, col=5, tile=1, bit=14)
    o, resid, flags, pred, actual = _inject(golden, f)
    (_, (o0, r0, f0, p0, a0)) = golden
    changed = _changed_rows(o, o0)
    assert changed and all(h == 1 and lo <= i < hi for _, h, i in changed)
    flagged = set(map(tuple, (flags != 0).nonzero().cpu().numpy().tolist()))
    assert flagged and flagged <= {(0, 1, i) for i in range(lo, hi)}
    # every row whose output moved by more than 2^-8 of its max is flagged
    O = G.from_dev_bf16(o)[0, 1]
    O0 = G.from_dev_bf16(o0)[0, 1]
    big = np.where(np.abs(O - O0).max(axis=1) > 2 ** -8 * np.abs(O0).max(axis=1))[0]
    assert set((0, 1, int(i)) for i in big) <= flagged


def test_s_site_flip_is_consistent(golden):
    # a score flip before the checksum tap moves O and pred together
    f = F.Fault("S", b=0, h=0, row=120, col=3, bit=26)
    o, resid, flags, pred, actual = _inject(golden, f)
    (_, (o0, r0, f0, p0, a0)) = golden
    assert _changed_rows(o, o0) <= {(0, 0, 120)}
    others = flags.clone()
    others[0, 0, 120] = 0
    assert int(others.sum()) == 0


# --------------------------------------------------------------------------
# checker-state sites: c, l and the running max
# --------------------------------------------------------------------------

def test_c_site_flip_is_a_false_alarm(golden):
    # the checksum accumulator is only read by the check: O is unchanged
    f = F.Fault("C", b=0, h=1, row=210, col=0, tile=1, bit=30)
    o, resid, flags, pred, actual = _inject(golden, f)
    (_, (o0, r0, f0, p0, a0)) = golden
    assert torch.equal(o.view(torch.int16), o0.view(torch.int16))
    assert torch.equal(actual, a0)
    assert int(flags[0, 1, 210]) != 0
    assert int(flags.sum()) == int(flags[0, 1, 210])


def test_l_site_flip_moves_o_and_pred_together(golden):
    # l divides both o and c: the ratio the check tests is unchanged
    f = F.Fault("L", b=0, h=0, row=150, col=0, tile=1, bit=26)
    o, resid, flags, pred, actual = _inject(golden, f)
    (_, (o0, r0, f0, p0, a0)) = golden
    assert _changed_rows(o, o0) == {(0, 0, 150)}
    assert int(flags.sum()) == 0


def test_m_site_flip_stays_in_its_row(golden):
    f = F.Fault("M", b=0, h=1, row=290, col=0, tile=2, bit=28)
    o, resid, flags, pred, actual = _inject(golden, f)
    (_, (o0, r0, f0, p0, a0)) = golden
    assert _changed_rows(o, o0) <= {(0, 1, 290)}
    others = flags.clone()
    others[0, 1, 290] = 0
    assert int(others.sum()) == 0


def test_q_site_is_upstream_of_the_checksum(golden):
    """A q register fault changes every later score of its row; o, l and c
    all use the resulting p~, so the row's output moves but its checksum
    still matches (the paper's check cannot see it)."""
    (_, (o0, r0, f0, p0, a0)) = golden
    f = F.Fault("Q", b=0, h=1, row=250, col=37, tile=1, bit=10)
    o, resid, flags, pred, actual = _inject(golden, f)
    assert _changed_rows(o, o0) == {(0, 1, 250)}
    assert int(flags.sum()) == 0
    tau, _ = F.get_threshold()
    O = G.from_dev_bf16(o)[0, 1, 250]
    M = np.abs(O).sum() + abs(float(pred[0, 1, 250]))
    assert abs(float(resid[0, 1, 250])) <= tau * M


def test_vs_site_is_a_false_positive(golden):
    """A flip in the sumrow record of one workgroup changes pred of its rows
    that weight the key, not O: an alarm with a correct result."""
    (_, (o0, r0, f0, p0, a0)) = golden
    qt = F.query_tile(W_INJ.d)
    f = F.Fault("VS", b=0, h=1, row=100, col=0, tile=1, bit=14)
    o, resid, flags, pred, actual = _inject(golden, f)
    assert torch.equal(o.view(torch.int16), o0.view(torch.int16))
    assert torch.equal(actual, a0)
    flagged = set(map(tuple, (flags != 0).nonzero().cpu().numpy().tolist()))
    assert flagged and flagged <= {(0, 1, i) for i in range(qt, W_INJ.Lq)}


def test_several_faults_in_one_launch(golden):
    (_, (o0, r0, f0, p0, a0)) = golden
    faults = [F.Fault("O", b=0, h=0, row=40, col=3, tile=0, bit=30),
              F.Fault("O", b=0, h=1, row=270, col=100, tile=2, bit=30),
              F.Fault("P", b=0, h=1, row=10, col=5, bit=14)]
    o, resid, flags, pred, actual = _inject(golden, faults)
    assert _changed_rows(o, o0) == {(0, 0, 40), (0, 1, 270), (0, 1, 10)}
    for b, h, i in ((0, 0, 40), (0, 1, 270), (0, 1, 10)):
        assert int(flags[b, h, i]) != 0, (b, h, i)
    # an empty list is the fault-free debug run
    o2, r2, f2, _, _ = _inject(golden, [])
    assert torch.equal(o2.view(torch.int16), o0.view(torch.int16))
    assert torch.equal(r2.view(torch.int32), r0.view(torch.int32))


def test_d96_faults_on_the_last_columns():
    """d = 96 runs the d = 128 kernel with zero columns 96..127 on chip: an
    O fault in column 95 and a V fault in column 90 behave as at d = 128,
    and nothing is written past column 95."""
    w = W.Workload("inj96", 1, 2, 300, 300, 96, True, 96 ** -0.5, seed=9)
    q, k, v = G.dev_inputs(W.make_inputs(w))
    o0, r0, f0, p0, a0 = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale)
    torch.cuda.synchronize()
    assert int(f0.sum()) == 0
    f = F.Fault("O", b=0, h=1, row=200, col=95, tile=2, bit=30)
    o, resid, flags, pred, actual = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale,
                                                      fault=f)
    torch.cuda.synchronize()
    assert _changed_rows(o, o0) == {(0, 1, 200)} and int(flags[0, 1, 200]) != 0
    f = F.Fault("V", b=0, h=0, row=40, col=90, tile=0, bit=14)
    o, resid, flags, pred, actual = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale,
                                                      fault=f)
    torch.cuda.synchronize()
    changed = _changed_rows(o, o0)
    assert changed and all(h == 0 and i >= 40 for _, h, i in changed)
    assert int(flags[0, 0].sum()) != 0
    # the output buffer holds exactly [B, H, L, 96]: a guard band after it
    # stays untouched
    buf = torch.full((o0.numel() + 64,), -7, dtype=torch.int16, device=q.device)
    ob = buf[:o0.numel()].view(torch.bfloat16).view(o0.shape)
    F.attn_fwd(q, k, v, causal=True, scale=w.scale, out=(ob, r0.clone(), f0.clone()))
    torch.cuda.synchronize()
    assert torch.all(buf[o0.numel():] == -7)
    assert torch.equal(ob.view(torch.int16), o0.view(torch.int16))


def test_d256_sites_follow_the_128_row_query_tile():
    """d = 256 runs 128 query rows per workgroup: a V fault in query tile 1
    reaches only rows 128..255, an O fault only its row; both are flagged."""
    w = W.Workload("inj256", 1, 2, 300, 300, 256, True, 1.0 / 16.0, seed=10)
    qt = F.query_tile(256)
    assert qt == 128
    q, k, v = G.dev_inputs(W.make_inputs(w))
    o0, r0, f0, p0, a0 = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale)
    torch.cuda.synchronize()
    assert int(f0.sum()) == 0
    f = F.Fault("O", b=0, h=0, row=290, col=255, tile=4, bit=30)
    o, resid, flags, pred, actual = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale,
                                                      fault=f)
    torch.cuda.synchronize()
    assert _changed_rows(o, o0) == {(0, 0, 290)} and int(flags[0, 0, 290]) != 0
    f = F.Fault("V", b=0, h=1, row=50, col=200, tile=1, bit=14)
    o, resid, flags, pred, actual = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale,
                                                      fault=f)
    torch.cuda.synchronize()
    changed = _changed_rows(o, o0)
    assert changed and all(h == 1 and qt <= i < 2 * qt for _, h, i in changed)
    flagged = set(map(tuple, (flags != 0).nonzero().cpu().numpy().tolist()))
    assert flagged and flagged <= {(0, 1, i) for i in range(qt, 2 * qt)}
