"""Persistent workgroups (a launch shape, not part of the method): with more
(head, query tile) items than the device holds at once, each workgroup runs a
list of items and passes its LDS ring from one item to the next. Every output
row must be bitwise the one-workgroup-per-item result (each row is computed
by the same instructions in the same order), on shapes where the ring is
passed on (items of a multiple of 4 key tiles) and where it is not (ragged
tile counts, items that see no key), with the mask and without, at d = 64, 96
and 128, checksum on, off and weighted; and the oracle agrees on sampled
rows."""
import numpy as np
import pytest
import torch

import workloads as W
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")

# name, B, H, Lq, Lk, d, causal: all have more items than one workgroup per
# CU can hold
CASES = [
    ("causal_d128", 2, 16, 4096, 4096, 128, True),      # every item passes its ring on
    ("causal_d96", 4, 8, 4000, 4000, 96, True),         # each head's last item is ragged
    ("causal_wide", 4, 16, 1500, 4000, 128, True),      # Lq < Lk
    ("causal_tall", 8, 8, 1200, 700, 128, True),        # Lq > Lk: items with no key
    ("full_ragged", 4, 24, 3000, 777, 128, False),      # 13 tiles: never passed on
    ("full_d128", 4, 24, 3000, 1024, 128, False),
    ("bert_d64", 32, 12, 512, 512, 64, False),
    ("causal_d64", 4, 16, 2048, 2048, 64, True),
    ("full_d64_ragged", 8, 16, 1000, 700, 64, False),   # 11 tiles: never passed on
    ("causal_odd_heads", 3, 7, 2048, 2048, 128, True),  # B*H not a multiple of 8
]


def _run(q, k, v, causal, scale, persistent, check=True):
    F.set_persistent(F.PERSIST_ALWAYS if persistent else F.PERSIST_OFF)
    try:
        o = torch.full_like(q, float("nan"))
        if not check:
            F.attn_fwd(q, k, v, causal=causal, scale=scale, check=False, out=(o,))
            torch.cuda.synchronize()
            return (o,)
        B, H, Lq = q.shape[:3]
        r = torch.full((B, H, Lq), float("nan"), dtype=torch.float32, device=q.device)
        f = torch.full((B, H, Lq), 0xAA, dtype=torch.uint8, device=q.device)
        F.attn_fwd(q, k, v, causal=causal, scale=scale, out=(o, r, f))
        torch.cuda.synchronize()
        return o, r, f
    finally:
        F.set_persistent(F.PERSIST_AUTO)


def _same(a, b):
    ai = a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32) \
        if a.dtype == torch.float32 else a
    bi = b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32) \
        if b.dtype == torch.float32 else b
    return bool(torch.equal(ai, bi))


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_persistent_matches_one_item_per_workgroup(case):
    name, B, H, Lq, Lk, d, causal = case
    print(f"[persistent] {name} B{B} H{H} Lq{Lq} Lk{Lk} d{d} causal={causal}", flush=True)
    w = W.Workload(name, B, H, Lq, Lk, d, causal, d ** -0.5, seed=91)
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    assert F.get_persistent() == F.PERSIST_AUTO
    one = _run(q, k, v, causal, w.scale, False)
    per = _run(q, k, v, causal, w.scale, True)
    for a, b, what in zip(one, per, ("o", "resid", "flags")):
        assert _same(a, b), f"{what} differs between the two launch shapes"
    o, r, f = per
    assert int((f != 0).sum()) == 0
    assert bool(torch.isfinite(o.float()).all()) and bool(torch.isfinite(r).all())
    # the oracle on sampled rows (both tile edges, the first and last rows)
    rng = np.random.default_rng(7)
    rows = np.unique(np.concatenate([[0, 255, 256, Lq - 1], rng.integers(0, Lq, 12)]))
    ref = G.oracle_rows(inp, causal, w.scale, rows=rows)
    O = G.from_dev_bf16(o)[:, :, rows]
    err = np.abs(O - ref["O"])
    assert err.max() <= G.O_MAX_ABS
    assert err.sum() / max(np.abs(ref["O"]).sum(), 1e-300) <= G.O_REL_L1


@pytest.mark.parametrize("check", ["off", "weighted"])
def test_persistent_other_modes(check):
    B, H, Lq, Lk, d = 2, 16, 4096, 4096, 128
    print(f"[persistent] mode {check} B{B} H{H} L{Lq} d{d} causal", flush=True)
    w = W.Workload("modes", B, H, Lq, Lk, d, True, d ** -0.5, seed=92)
    q, k, v = G.dev_inputs(W.make_inputs(w))
    if check == "weighted":
        F.set_weighted_check(True)
    try:
        one = _run(q, k, v, True, w.scale, False, check=check != "off")
        per = _run(q, k, v, True, w.scale, True, check=check != "off")
    finally:
        F.set_weighted_check(False)
    for a, b in zip(one, per):
        assert _same(a, b)
