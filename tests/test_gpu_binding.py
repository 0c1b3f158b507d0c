"""The Python binding refuses caller tensors that do not fit the call
(out=, workspaces) before the library sees a pointer, and the kernels never
read the key rows past Lk: K and V placed at the end of a larger buffer whose
tail is NaN give the same O as the oracle, with no flag."""
import numpy as np
import pytest
import torch

import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")


@pytest.fixture(scope="module")
def qkv():
    w = W.Workload("bind", 1, 2, 100, 130, 128, True, 128 ** -0.5, seed=71)
    return w, G.dev_inputs(W.make_inputs(w))


def _bad_outs(B, H, Lq, d, dev):
    good_o = torch.empty((B, H, Lq, d), dtype=torch.bfloat16, device=dev)
    good_r = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)
    good_f = torch.empty((B, H, Lq), dtype=torch.uint8, device=dev)
    return [
        (good_o[:, :, :-1], good_r, good_f),                                   # short o
        (good_o.float(), good_r, good_f),                                      # o dtype
        (good_o.transpose(2, 3).contiguous().transpose(2, 3), good_r, good_f),  # not contiguous
        (good_o.cpu(), good_r, good_f),                                        # device
        (good_o, good_r[:, :, :-1], good_f),                                   # short resid
        (good_o, good_r.half(), good_f),                                       # resid dtype
        (good_o, good_r, good_f.to(torch.int32)),                              # flags dtype
        (good_o, good_r, good_f[:, :1]),                                       # flags shape
    ]


def test_bad_out_tensors_are_refused(qkv):
    w, (q, k, v) = qkv
    for out in _bad_outs(w.B, w.H, w.Lq, w.d, q.device):
        with pytest.raises(ValueError):
            F.attn_fwd(q, k, v, causal=True, out=out)
        with pytest.raises(ValueError):
            F.attn_fwd_splitkv(q, k, v, causal=True, nsplit=2, out=out)
        with pytest.raises(ValueError):
            F.recompute_flagged(q, k, v, *out, causal=True)
    pred = torch.empty((w.B, w.H, w.Lq), dtype=torch.float32, device=q.device)
    with pytest.raises(ValueError):
        F.attn_fwd_inject(q, k, v, causal=True, out=_bad_outs(w.B, w.H, w.Lq, w.d,
                                                               q.device)[0] + (pred, pred))
    with pytest.raises(ValueError):
        F.attn_fwd_inject(q, k, v, causal=True,
                          out=_bad_outs(w.B, w.H, w.Lq, w.d, q.device)[0][:1] * 3 + (pred[:, :1], pred))
    with pytest.raises(ValueError):
        F.attn_fwd(q, k, v, causal=True, out=(torch.empty_like(q),))   # check=True needs 3
    need = F.splitkv_workspace_bytes(w.B, w.H, w.Lq, w.d, 2)
    with pytest.raises(ValueError):
        F.attn_fwd_splitkv(q, k, v, causal=True, nsplit=2,
                           workspace=torch.empty(need - 1, dtype=torch.uint8, device=q.device))
    with pytest.raises(ValueError):
        F.attn_fwd_splitkv(q, k, v, causal=True, nsplit=2,
                           workspace=torch.empty(need, dtype=torch.uint8))
    # a good out= still works and equals the allocating call
    o, r, f = F.attn_fwd(q, k, v, causal=True)
    outs = (torch.empty_like(q), torch.empty_like(r), torch.empty_like(f))
    F.attn_fwd(q, k, v, causal=True, out=outs)
    torch.cuda.synchronize()
    assert torch.equal(outs[0].view(torch.int16), o.view(torch.int16))


@pytest.mark.parametrize("d", [64, 96, 128, 256])
@pytest.mark.parametrize("Lk", [77, 1000])
@pytest.mark.parametrize("split", [False, True, "twopass", "decode"])
@pytest.mark.parametrize("causal", [False, True])
def test_rows_past_the_keys_are_never_read(d, Lk, split, causal):
    """K and V of one head at the very end of a buffer with 64 NaN rows after
    them (the last key tile reads up to 63 rows past Lk, which must come back
    as zeros): O matches the oracle and no row is flagged. Every read stays
    inside the buffer, so a wrong bound shows as NaN, not as a fault."""
    # "decode": two query rows, the key split's vector-ALU decode kernel
    Lq = 2 if split == "decode" else 150
    w = W.Workload(f"tail{Lk}", 1, 1, Lq, Lk, d, causal, d ** -0.5, seed=Lk + d)
    print(f"[tail] Lk={Lk} d={d} split={split} causal={causal}", flush=True)
    inp = W.make_inputs(w)
    q = G.to_dev(inp.q)

    def tailed(bits):
        n = bits.size
        buf = torch.full((n + 64 * d,), float("nan"), dtype=torch.bfloat16, device=q.device)
        buf[:n] = G.to_dev(bits).reshape(-1)
        return buf[:n].view(1, 1, Lk, d)

    k, v = tailed(inp.k), tailed(inp.v)
    assert torch.isnan(k.reshape(-1)[-1:]).sum() == 0
    if split == "twopass":
        # both passes, the first one loading K alone
        o, resid, flags = F.attn_fwd_twopass(q, k, v, causal=causal, scale=w.scale)
        pred = None
    elif split:   # the MFMA split kernel, or the decode kernel for two rows
        o, resid, flags = F.attn_fwd_splitkv(q, k, v, causal=causal, scale=w.scale, nsplit=3)
        pred = None
    else:
        o, resid, flags, pred, actual = F.attn_fwd_inject(q, k, v, causal=causal, scale=w.scale)
    torch.cuda.synchronize()
    ref = G.oracle_rows(inp, causal, w.scale)
    O = G.from_dev_bf16(o)
    assert np.all(np.isfinite(O))
    err = np.abs(O - ref["O"])
    assert err.max() <= G.O_MAX_ABS and err.sum() / np.abs(ref["O"]).sum() <= G.O_REL_L1
    if pred is not None:
        G.compare(o, pred, ref, d)
    assert int((flags != 0).sum()) == 0
