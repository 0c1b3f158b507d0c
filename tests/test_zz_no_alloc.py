"""The allocation-free key split (fabft_attn_fwd_splitkv_noalloc), called
through the C ABI: its results equal those of fabft_attn_fwd_splitkv with a
caller workspace, bit for bit (same kernels, same split count), on two calls
in a row whose second is smaller than the first, so that the second reuses
the library's buffer with the first call's partial states still in it."""
import pytest
import torch

import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")


def _call_noalloc(q, k, v, causal, scale, nsplit):
    B, H, Lq, d = q.shape
    Lk = k.shape[2]
    o = torch.empty_like(q)
    resid = torch.full((B, H, Lq), float("nan"), dtype=torch.float32, device=q.device)
    flags = torch.full((B, H, Lq), 0xEE, dtype=torch.uint8, device=q.device)
    F.lib().fabft_set_stream(torch.cuda.current_stream(q.device).cuda_stream)
    rc = F.lib().fabft_attn_fwd_splitkv_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                                o.data_ptr(), resid.data_ptr(), flags.data_ptr(),
                                                B, H, Lq, Lk, d, int(causal), scale, nsplit)
    assert rc == F.FABFT_OK, F.status_str(rc)
    return o, resid, flags


def _call_workspace(q, k, v, causal, scale, nsplit):
    B, H, Lq, d = q.shape
    Lk = k.shape[2]
    need = F.splitkv_workspace_bytes(B, H, Lq, d, nsplit)
    ws = torch.empty(need, dtype=torch.uint8, device=q.device)
    o = torch.empty_like(q)
    resid = torch.empty((B, H, Lq), dtype=torch.float32, device=q.device)
    flags = torch.empty((B, H, Lq), dtype=torch.uint8, device=q.device)
    F.lib().fabft_set_stream(torch.cuda.current_stream(q.device).cuda_stream)
    rc = F.lib().fabft_attn_fwd_splitkv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                        resid.data_ptr(), flags.data_ptr(), B, H, Lq, Lk, d,
                                        int(causal), scale, nsplit, ws.data_ptr(), need)
    assert rc == F.FABFT_OK, F.status_str(rc)
    return o, resid, flags


CASES = [
    # a decode-shaped first call (8.6 MB of partial states), then a smaller one
    (W.Workload("noalloc_big", 4, 32, 16, 3000, 128, False, 128 ** -0.5, seed=51), 8),
    (W.Workload("noalloc_small", 1, 3, 5, 700, 64, True, 0.125, seed=52), 3),
]


def test_noalloc_matches_workspace_form_on_two_calls():
    for w, ns in CASES:
        print(f"[noalloc] {w.name} B{w.B} H{w.H} Lq{w.Lq} Lk{w.Lk} d{w.d} "
              f"causal={w.causal} nsplit={ns}", flush=True)
        q, k, v = G.dev_inputs(W.make_inputs(w))
        a = _call_noalloc(q, k, v, w.causal, w.scale, ns)
        b = _call_workspace(q, k, v, w.causal, w.scale, ns)
        torch.cuda.synchronize()
        assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16)), w.name
        assert torch.equal(a[1].view(torch.int32), b[1].view(torch.int32)), w.name
        assert torch.equal(a[2], b[2]), w.name
        assert int(a[2].sum()) == 0, w.name
        # and the oracle agrees (the bar of every other parity test)
        ref = G.oracle_rows(W.make_inputs(w), w.causal, w.scale)
        o, resid, flags, pred, actual = F.attn_fwd_inject(q, k, v, causal=w.causal,
                                                          scale=w.scale)
        torch.cuda.synchronize()
        G.compare(a[0], pred, ref, w.d)
