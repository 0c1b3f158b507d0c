"""GPU tests of the campaign machinery: per-head recomputation is bitwise
identical to the full launch (what the campaign relies on), a short
campaign classifies top-exponent-bit output faults as detected, and a short
fault-free sweep flags nothing."""
import json

import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")
from paper_2507_16676_amd import campaign as C  # noqa: E402

W_SMALL = W.Workload("camp_small", 2, 3, 1000, 1000, 128, True, 128 ** -0.5, seed=5)


def test_head_slice_matches_full_launch():
    q, k, v = C.device_inputs(W_SMALL, 5)
    o, resid, flags = F.attn_fwd(q, k, v, causal=True, scale=W_SMALL.scale)
    for b in range(W_SMALL.B):
        for h in range(W_SMALL.H):
            oh, rh, fh = F.attn_fwd(q[b:b + 1, h:h + 1], k[b:b + 1, h:h + 1],
                                    v[b:b + 1, h:h + 1], causal=True, scale=W_SMALL.scale)
            torch.cuda.synchronize()
            assert torch.equal(oh[0, 0].view(torch.int16), o[b, h].view(torch.int16))
            assert torch.equal(rh[0, 0].view(torch.int32), resid[b, h].view(torch.int32))
            assert torch.equal(fh[0, 0], flags[b, h])


def test_short_campaign(tmp_path):
    out = tmp_path / "c.jsonl"
    summ = C.run_campaign(W_SMALL, 400, str(out), seed=5, log_every=0)
    print("[campaign-test]", json.dumps({"headline": summ["headline"],
                                         "per_site": summ["per_site"]}), flush=True)
    assert summ["runs"] == 400
    recs = [json.loads(l) for l in open(out)]
    for r in recs:
        # the top exponent bit of an output accumulator or of a value moves the
        # output by orders of magnitude: always detected
        if r["site"] in ("O", "V") and r["bit"] == (30 if r["site"] == "O" else 14):
            assert r["outcome"] == "detected", r
    # resumable: a second call adds nothing
    summ2 = C.run_campaign(W_SMALL, 400, str(out), seed=5, log_every=0)
    assert summ2["runs"] == 400


def test_short_sweep(tmp_path):
    res = C.run_sweep(W_SMALL, 20, str(tmp_path / "s.json"), seed0=100, rho_every=5,
                      log_every=0)
    print("[sweep-test]", json.dumps(res), flush=True)
    assert res["flagged_rows"] == 0
    assert 0 < res["rho_max"] < F.get_threshold()[0] / 8
