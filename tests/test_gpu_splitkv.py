"""Key-split forward (partial states per key range and a merge that carries
the checksum c like one more column of o) on the GPU through the C ABI:
decode-shaped inputs (few queries, many keys; up to four rows take the
vector-ALU decode kernel, more the MFMA split kernel), empty splits,
d = 64, 96, 128 and 256, causal and not; O against the fp64 oracle, no
flags fault-free, the residual as small as in the one-pass kernel."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")

CASES = [
    (W.Workload("dec1", 2, 3, 1, 5000, 128, False, 128 ** -0.5, seed=11), 8),
    (W.Workload("dec16c", 1, 4, 16, 3000, 128, True, 128 ** -0.5, seed=12), 13),
    (W.Workload("dec7c64", 2, 2, 7, 777, 64, True, 0.125, seed=13), 20),   # 13 tiles: empty splits
    (W.Workload("sq300", 1, 2, 300, 300, 128, True, 128 ** -0.5, seed=14), 3),
    (W.Workload("one", 1, 1, 5, 2000, 64, False, 0.125, seed=15), 1),
    (W.Workload("dec3d96", 2, 2, 3, 1500, 96, True, 96 ** -0.5, seed=16), 6),
    (W.Workload("dec5d256", 1, 3, 5, 2100, 256, True, 256 ** -0.5, seed=17), 7),
    # up to four query rows: the vector-ALU decode kernel (ragged key counts,
    # causal rows that see different key counts, splits with no key)
    (W.Workload("dec1d64", 2, 3, 1, 3001, 64, False, 0.125, seed=18), 5),
    (W.Workload("dec2c", 1, 4, 2, 2500, 128, True, 128 ** -0.5, seed=19), 7),
    (W.Workload("dec4c256", 1, 2, 4, 1111, 256, True, 256 ** -0.5, seed=20), 3),
    (W.Workload("dec4d96", 2, 2, 4, 700, 96, False, 96 ** -0.5, seed=21), 11),
    (W.Workload("dec1e", 1, 2, 1, 100, 128, False, 128 ** -0.5, seed=22), 8),
    (W.Workload("dec3c64", 1, 3, 3, 4099, 64, True, 0.125, seed=23), 2),
    # 1% of the keys scaled by 8: scores that jump past the lazily kept max
    # late in a wave's keys, so the decode kernel rescales l, c and o
    (W.Workload("dec2peak", 1, 4, 2, 6000, 128, True, 128 ** -0.5, peaked_frac=0.01,
                seed=24), 3),
    (W.Workload("dec1peak64", 2, 2, 1, 5000, 64, False, 0.125, peaked_frac=0.01, seed=25), 4),
]


@pytest.mark.parametrize("w,ns", CASES, ids=[f"{c.name}-s{n}" for c, n in CASES])
def test_splitkv_parity(w, ns):
    print(f"[splitkv] {w.name} B{w.B} H{w.H} Lq{w.Lq} Lk{w.Lk} d{w.d} causal={w.causal} "
          f"nsplit={ns}", flush=True)
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    o, resid, flags = F.attn_fwd_splitkv(q, k, v, causal=w.causal, scale=w.scale, nsplit=ns)
    o1, r1, f1 = F.attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
    torch.cuda.synchronize()
    ref = G.oracle_rows(inp, w.causal, w.scale)
    O = G.from_dev_bf16(o)
    err = np.abs(O - ref["O"])
    assert err.max() <= G.O_MAX_ABS, err.max()
    assert err.sum() <= G.O_REL_L1 * max(np.abs(ref["O"]).sum(), 1e-30)
    assert int((flags != 0).sum()) == 0
    # the residual stays at the one-pass kernel's level
    M = np.abs(O).sum(axis=-1) + np.abs(ref["pred"])
    rho = (np.abs(resid.cpu().numpy()) / np.maximum(M, 1e-30)).max()
    assert rho <= F.get_threshold()[0] / 4, rho
    # and O is within one bf16 rounding of the one-pass kernel's
    O1 = G.from_dev_bf16(o1)
    assert np.abs(O - O1).max() <= 2 ** -7 * max(np.abs(O1).max(), 1e-30)


def test_splitkv_weighted():
    w, ns = CASES[1]
    F.set_weighted_check(True)
    try:
        q, k, v = G.dev_inputs(W.make_inputs(w))
        o, resid, flags = F.attn_fwd_splitkv(q, k, v, causal=w.causal, scale=w.scale, nsplit=ns)
        torch.cuda.synchronize()
        assert int((flags != 0).sum()) == 0
    finally:
        F.set_weighted_check(False)


@pytest.mark.parametrize("d", [64, 128])
def test_decode_rows_without_keys(d):
    """Four causal rows over two keys: rows 0 and 1 see no key (bottom-right
    alignment), so their O, resid and flags are 0; rows 2 and 3 match the
    oracle."""
    w = W.Workload("dec4short", 1, 2, 4, 2, d, True, d ** -0.5, seed=26)
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    o, resid, flags = F.attn_fwd_splitkv(q, k, v, causal=True, scale=w.scale, nsplit=2)
    torch.cuda.synchronize()
    assert torch.all(o[:, :, :2].float() == 0)
    assert torch.all(resid[:, :, :2] == 0)
    assert int((flags != 0).sum()) == 0
    ref = G.oracle_rows(inp, True, w.scale)
    O = G.from_dev_bf16(o)
    assert np.abs(O - ref["O"]).max() <= G.O_MAX_ABS


def test_splitkv_weighted_decode():
    """The weighted check in the decode kernel (two rows, causal): no flag,
    and O is the same with the check on and off."""
    w, ns = CASES[8]
    assert w.Lq <= 4
    q, k, v = G.dev_inputs(W.make_inputs(w))
    o0, r0, f0 = F.attn_fwd_splitkv(q, k, v, causal=w.causal, scale=w.scale, nsplit=ns)
    F.set_weighted_check(True)
    try:
        o1, r1, f1 = F.attn_fwd_splitkv(q, k, v, causal=w.causal, scale=w.scale, nsplit=ns)
        torch.cuda.synchronize()
    finally:
        F.set_weighted_check(False)
    assert int((f0 != 0).sum()) == 0 and int((f1 != 0).sum()) == 0
    assert torch.equal(o0.view(torch.int16), o1.view(torch.int16))


def test_splitkv_workspace_reused():
    # the workspace holds no state between calls: a second, smaller call in
    # the same buffer gives the same result as a fresh one
    w1, _ = CASES[1]
    w2, _ = CASES[2]
    ws = torch.empty(F.splitkv_workspace_bytes(w1.B, w1.H, w1.Lq, w1.d, 13), dtype=torch.uint8,
                     device="cuda")
    q, k, v = G.dev_inputs(W.make_inputs(w1))
    F.attn_fwd_splitkv(q, k, v, causal=w1.causal, scale=w1.scale, nsplit=13, workspace=ws)
    q2, k2, v2 = G.dev_inputs(W.make_inputs(w2))
    need2 = F.splitkv_workspace_bytes(w2.B, w2.H, w2.Lq, w2.d, 5)
    assert need2 <= ws.numel()
    a = F.attn_fwd_splitkv(q2, k2, v2, causal=True, scale=w2.scale, nsplit=5, workspace=ws)
    b = F.attn_fwd_splitkv(q2, k2, v2, causal=True, scale=w2.scale, nsplit=5)
    torch.cuda.synchronize()
    assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16))
    assert torch.equal(a[1].view(torch.int32), b[1].view(torch.int32))
