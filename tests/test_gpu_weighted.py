"""The weighted second checksum (weights (-1)^j, next to the paper's plain
one) on the GPU, through the C ABI: pred_w and actual_w agree with the fp64
oracle, switching it on changes neither O nor the paper's residual, nothing
is flagged fault-free, and a p~ fault on a key whose V row sums to 0 -- a
blind spot of the paper's check -- is flagged by the weighted check."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")

CASES = [
    W.WORKLOADS["bert_l128"],
    W.Workload("w_ragged", 2, 3, 129, 129, 64, True, 0.125, seed=3),
    W.Workload("w_rect", 1, 2, 300, 1000, 128, False, 128 ** -0.5, seed=4),
    W.Workload("w_masked", 1, 2, 333, 100, 128, True, 128 ** -0.5, seed=5),
    W.Workload("w_d96", 1, 2, 200, 200, 96, True, 96 ** -0.5, seed=6),
    W.Workload("w_d256", 1, 2, 300, 300, 256, True, 256 ** -0.5, seed=8),
]


@pytest.fixture
def weighted():
    F.set_weighted_check(True)
    yield
    F.set_weighted_check(False)


@pytest.mark.parametrize("w", CASES, ids=[c.name for c in CASES])
def test_weighted_parity(weighted, w):
    print(f"[weighted] {w.name} B{w.B} H{w.H} Lq{w.Lq} Lk{w.Lk} d{w.d} causal={w.causal}",
          flush=True)
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    o, resid, flags, pred, actual, pw, aw = F.attn_fwd_inject(
        q, k, v, causal=w.causal, scale=w.scale, weighted_out=True)
    o1, r1, f1 = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
    F.set_weighted_check(False)
    o0, r0, f0 = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
    F.set_weighted_check(True)
    torch.cuda.synchronize()
    # the second checksum changes neither O nor the paper's residual
    for t in (o1, o0):
        assert torch.equal(t.view(torch.int16), o.view(torch.int16))
    for t in (r1, r0):
        assert torch.equal(t.view(torch.int32), resid.view(torch.int32))
    assert int((flags != 0).sum()) == 0 and int((f1 != 0).sum()) == 0
    qf, kf, vf = inp.as_f32()
    pw_h = pw.cpu().numpy().astype(np.float64)
    aw_h = aw.cpu().numpy().astype(np.float64)
    O = G.from_dev_bf16(o)
    tau = F.get_threshold()[0]
    for b in range(w.B):
        for h in range(w.H):
            ref = oracle.weighted_check_head(qf[b, h], kf[b, h], vf[b, h], w.causal, w.scale)
            err = np.abs(pw_h[b, h] - ref["pred_w"])
            assert err.max() <= G.O_MAX_ABS * np.sqrt(w.d), err.max()
            assert err.sum() <= G.O_REL_L1 * max(np.abs(ref["pred_w"]).sum(), 1e-30)
            M = np.abs(O[b, h]).sum(axis=-1) + np.abs(pw_h[b, h])
            live = M > 0
            rho = (np.abs(pw_h[b, h] - aw_h[b, h])[live] / M[live]).max() if live.any() else 0.0
            # same margin as the paper check keeps on these shapes (>= 4x)
            assert rho <= tau / 4, rho


def test_weighted_off_reports_zero(weighted):
    F.set_weighted_check(False)
    w = CASES[0]
    q, k, v = G.dev_inputs(W.make_inputs(w))
    out = F.attn_fwd_inject(q, k, v, causal=w.causal, scale=w.scale, weighted_out=True)
    F.set_weighted_check(True)
    torch.cuda.synchronize()
    assert float(out[5].abs().max()) == 0.0 and float(out[6].abs().max()) == 0.0


def test_zero_sum_value_row_p_fault(weighted):
    # key 40 of head (0, 0): V row of pairs (x, -x), so sumrow = 0 exactly;
    # a flip of p~ at that key moves O but not the paper's prediction/actual
    w = W.Workload("w_blind", 1, 2, 300, 300, 128, True, 128 ** -0.5, seed=7)
    inp = W.make_inputs(w)
    x = inp.v[0, 0, 40, 0::2].copy()
    inp.v[0, 0, 40, 1::2] = x ^ np.uint16(0x8000)     # exact negation in bf16
    assert W.bf16_bits_to_f32(inp.v[0, 0, 40]).astype(np.float64).sum() == 0.0
    q, k, v = G.dev_inputs(inp)
    o0 = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale)[0]
    torch.cuda.synchronize()
    O0 = G.from_dev_bf16(o0)[0, 0, 200]
    significant = 0
    for bit in (10, 11, 12, 13):
        f = F.Fault("P", b=0, h=0, row=200, col=40, bit=bit)
        print(f"[weighted] blind-spot P fault bit {bit}", flush=True)
        o, resid, flags, *_ = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale, fault=f)
        torch.cuda.synchronize()
        O = G.from_dev_bf16(o)[0, 0, 200]
        if np.abs(O - O0).max() > 2 ** -8 * np.abs(O0).max():
            significant += 1
            fl = int(flags[0, 0, 200])
            assert fl & F.FLAG_WEIGHTED, (bit, fl)
            assert not fl & F.FLAG_RESID, (bit, fl)      # the paper's check is blind here
    assert significant >= 1
