"""The checksum hosted by Algorithm 1 (fabft_attn_fwd_twopass): a first pass
over the keys takes each row's maximum score, a second accumulates o, l and c
with that fixed maximum (Section III-B: the per-query check needs only the
exponentials and their sum, so either algorithm can carry it).

Parity with the fp64 oracle on the same seeded bf16 inputs: O element by
element (max abs <= 2e-2, relative L1 <= 5e-3), no row flagged, and the
residual against the checked row sums inside the detection threshold. The
one-pass kernel must agree with it to rounding (the exponentials use another
reference maximum), and rows without a visible key give O = 0 and resid = 0.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")


def _rows_of(a, rows):
    return a if rows is None else a[:, :, rows]


def _twopass(w: W.Workload, rows=None, inp=None):
    print(f"[twopass] {w.name} B{w.B} H{w.H} Lq{w.Lq} Lk{w.Lk} d{w.d} causal={w.causal}",
          flush=True)
    inp = W.make_inputs(w) if inp is None else inp
    q, k, v = G.dev_inputs(inp)
    o, resid, flags = F.attn_fwd_twopass(q, k, v, causal=w.causal, scale=w.scale)
    o1, resid1, flags1 = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
    torch.cuda.synchronize()
    assert int((flags != 0).sum()) == 0, "fault-free rows flagged by the two-pass check"
    assert int((flags1 != 0).sum()) == 0
    ref = G.oracle_rows(inp, w.causal, w.scale, rows=rows)
    O = _rows_of(G.from_dev_bf16(o), rows)
    err = np.abs(O - ref["O"])
    rel = err.sum() / max(np.abs(ref["O"]).sum(), 1e-300)
    assert np.all(np.isfinite(O))
    assert err.max() <= G.O_MAX_ABS and rel <= G.O_REL_L1, (float(err.max()), float(rel))
    # pred = resid + actual, with actual taken here from the bf16 O (the
    # kernel's comes from fp32 O before rounding; the two differ by a sum of
    # d roundings, each at most half a bf16 unit of its element)
    R = _rows_of(resid.double().cpu().numpy(), rows)
    pred_est = R + O.sum(axis=-1)
    perr = np.abs(pred_est - ref["pred"])
    assert perr.max() <= G.O_MAX_ABS * np.sqrt(w.d), float(perr.max())
    # one pass and two passes: the same attention to rounding
    O1 = _rows_of(G.from_dev_bf16(o1), rows)
    d12 = float(np.abs(O - O1).max())
    assert d12 <= G.O_MAX_ABS, d12
    M = np.abs(O).sum(axis=-1) + np.abs(pred_est)
    live = M > 0
    rho = float((np.abs(R)[live] / M[live]).max()) if live.any() else 0.0
    print(f"[twopass] {w.name}: o_max_abs={err.max():.3e} o_rel_l1={rel:.3e} "
          f"pred_max_abs={perr.max():.3e} |O_2p - O_1p|max={d12:.3e} rho={rho:.3e}", flush=True)
    return o, resid, flags


@pytest.mark.parametrize("d", [64, 96, 128, 256])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("L", [1, 129, 1000])
def test_twopass_ragged_square(d, causal, L):
    _twopass(W.Workload(f"tp_L{L}", 1, 2, L, L, d, causal, d ** -0.5, seed=5 * L + d))


@pytest.mark.parametrize("d", [64, 128, 256])
@pytest.mark.parametrize("Lq,Lk", [(100, 333), (333, 100), (1, 4096)])
def test_twopass_rectangular(d, Lq, Lk):
    w = W.Workload(f"tp_rect_{Lq}x{Lk}", 2, 3, Lq, Lk, d, True, d ** -0.5, seed=Lq + 3 * Lk)
    o, resid, flags = _twopass(w)
    if Lq > Lk:
        # rows with no visible key: O = 0 and resid = 0, not flagged
        dead = Lq - Lk
        assert torch.all(o[:, :, :dead].float() == 0)
        assert torch.all(resid[:, :, :dead] == 0)


def test_twopass_bert_l512_full():
    _twopass(W.WORKLOADS["bert_l512"])


def test_twopass_dec_l4096_rows():
    w = W.WORKLOADS["dec_l4096"]
    rows = W.sample_rows(w.Lq, 256, 0, must=(0, 1, 255, 256, w.Lq - 1))
    _twopass(w, rows=rows)


def test_twopass_peaked_keys():
    """Keys scaled by 8 arriving late in a row (the case where the one-pass
    kernel rescales o, l and c): the two-pass kernel never rescales, and both
    agree with the oracle on the rows at and just after those keys."""
    w = W.WORKLOADS["long_l32768"].with_(B=1, H=4, Lq=4096, Lk=4096, peaked_frac=0.01)
    inp = W.make_inputs(w)
    must = []
    for h in range(w.H):
        must += [int(r) for r in inp.peaked_rows[0, h][:16]]
        must += [int(r) + 1 for r in inp.peaked_rows[0, h][:16]]
    rows = W.sample_rows(w.Lq, 256, 7, must=tuple(must))
    _twopass(w, rows=rows, inp=inp)


def test_twopass_weighted_check():
    """With the weighted second checksum on, O is unchanged bit for bit and
    no row is flagged by either check."""
    w = W.Workload("tp_weighted", 2, 4, 700, 700, 128, True, 128 ** -0.5, seed=11)
    q, k, v = G.dev_inputs(W.make_inputs(w))
    o0, r0, f0 = F.attn_fwd_twopass(q, k, v, causal=True, scale=w.scale)
    old = F.get_weighted_check()
    try:
        F.set_weighted_check(True)
        o1, r1, f1 = F.attn_fwd_twopass(q, k, v, causal=True, scale=w.scale)
    finally:
        F.set_weighted_check(old)
    torch.cuda.synchronize()
    assert torch.equal(o0.view(torch.int16), o1.view(torch.int16))
    assert torch.equal(r0.view(torch.int32), r1.view(torch.int32))
    assert int((f0 != 0).sum()) == 0 and int((f1 != 0).sum()) == 0


def test_twopass_algorithm1_oracle_form():
    """Against the oracle's Algorithm 1 restatement (first pass: the row max;
    second: o, l and c with it) on one small head."""
    w = W.Workload("tp_alg1", 1, 1, 150, 150, 64, True, 0.125, seed=21)
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    o, resid, flags = F.attn_fwd_twopass(q, k, v, causal=True, scale=w.scale)
    torch.cuda.synchronize()
    qf, kf, vf = inp.as_f32()
    ref = oracle.lazy_softmax_attention(qf[0, 0], kf[0, 0], vf[0, 0], True, w.scale)
    O = G.from_dev_bf16(o)[0, 0]
    assert np.abs(O - ref["O"]).max() <= G.O_MAX_ABS
    pred_est = resid.double().cpu().numpy()[0, 0] + O.sum(axis=-1)
    assert np.abs(pred_est - ref["pred"]).max() <= G.O_MAX_ABS * np.sqrt(w.d)
    assert int((flags != 0).sum()) == 0


def test_twopass_deterministic():
    w = W.WORKLOADS["dec_l4096"].with_(B=1, H=4)
    q, k, v = G.dev_inputs(W.make_inputs(w))
    a = F.attn_fwd_twopass(q, k, v, causal=True, scale=w.scale)
    b = F.attn_fwd_twopass(q, k, v, causal=True, scale=w.scale)
    torch.cuda.synchronize()
    assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16))
    assert torch.equal(a[1].view(torch.int32), b[1].view(torch.int32))


def test_algorithm_switch_selects_the_two_pass_forms():
    """With Algorithm 1 selected, attn_fwd and the debug path run the two-pass
    kernels: the same O, resid and flags as attn_fwd_twopass, bit for bit;
    the debug outputs give pred directly, which matches the oracle's
    Algorithm 1 restatement."""
    import oracle as O_
    w = W.Workload("tp_switch", 1, 2, 333, 333, 128, True, 128 ** -0.5, seed=31)
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    o2, r2, f2 = F.attn_fwd_twopass(q, k, v, causal=True, scale=w.scale)
    try:
        F.set_algorithm(1)
        o, r, f = F.attn_fwd(q, k, v, causal=True, scale=w.scale)
        od, rd, fd, pred, actual = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale)
        torch.cuda.synchronize()
    finally:
        F.set_algorithm(3)
    for a, b in ((o, o2), (od, o2)):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert torch.equal(r.view(torch.int32), r2.view(torch.int32))
    assert torch.equal(rd.view(torch.int32), r2.view(torch.int32))
    assert int((f != 0).sum()) == 0 and int((fd != 0).sum()) == 0
    qf, kf, vf = inp.as_f32()
    for h in range(w.H):
        ref = O_.lazy_softmax_attention(qf[0, h], kf[0, h], vf[0, h], True, w.scale)
        P = pred[0, h].double().cpu().numpy()
        assert np.abs(P - ref["pred"]).max() <= G.O_MAX_ABS * np.sqrt(w.d)
        assert np.abs(P - ref["pred"]).sum() <= G.O_REL_L1 * np.abs(ref["pred"]).sum()


@pytest.mark.parametrize("site,kw", [
    ("P", dict(b=0, h=0, row=250, col=100, bit=14)),
    ("O", dict(b=0, h=1, row=200, col=37, tile=2, bit=30)),
    ("V", dict(b=0, h=1, row=100, col=5, tile=0, bit=14)),
])
def test_algorithm1_flags_injected_faults(site, kw):
    """Exponent flips at P, O and V under Algorithm 1: only rows of the
    faulted head change, and the rows whose output moved by more than 2^-8
    of their largest value are flagged (the same bar as the one-pass
    campaign)."""
    w = W.Workload("tp_inject", 1, 2, 300, 300, 128, True, 128 ** -0.5, seed=7)
    q, k, v = G.dev_inputs(W.make_inputs(w))
    try:
        F.set_algorithm(1)
        o0, r0, f0, p0, a0 = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale)
        o, r, f, p, a = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale,
                                          fault=F.Fault(site, **kw))
        torch.cuda.synchronize()
    finally:
        F.set_algorithm(3)
    assert int((f0 != 0).sum()) == 0
    moved = (o.view(torch.int16) != o0.view(torch.int16)).any(dim=-1)
    assert bool(moved.any())
    assert not bool(moved[0, 1 - kw["h"]].any())
    O = G.from_dev_bf16(o)[0, kw["h"]]
    O0 = G.from_dev_bf16(o0)[0, kw["h"]]
    # a row whose output turned non-finite counts as moved (an exponent flip
    # of an fp32 accumulator in [1, 2) makes it NaN or infinite)
    dif = np.abs(O - O0)
    dif[~np.isfinite(dif)] = np.inf
    big = np.where(dif.max(axis=1) > 2 ** -8 * np.abs(O0).max(axis=1))[0]
    assert len(big) > 0
    flagged = set(int(i) for i in (f[0, kw["h"]] != 0).nonzero().flatten().cpu().numpy())
    assert set(int(i) for i in big) <= flagged
