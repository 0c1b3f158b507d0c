"""Host-side tests of the fault campaign logic: fault draws respect the
documented descriptor rules and cover every site and bit, classification
follows the outcome definitions, and the summary arithmetic is right."""
import json

import numpy as np
import pytest
import torch

import workloads as W
from paper_2507_16676_amd import campaign as C

W_C = W.WORKLOADS["dec_l4096"]


def _valid(f, w, bc, qt):
    off = w.Lk - w.Lq
    assert 0 <= f.b < w.B and 0 <= f.h < w.H
    if f.site in ("S", "P"):
        assert 0 <= f.row < w.Lq and 0 <= f.col < w.Lk
        assert not w.causal or f.col <= f.row + off
        assert 0 <= f.bit < (32 if f.site == "S" else 16)
    elif f.site in ("O", "C", "L", "M", "Q"):
        ncol = w.d if f.site in ("O", "Q") else 2 if f.site == "C" else 1
        assert 0 <= f.row < w.Lq and 0 <= f.col < ncol
        assert 0 <= f.bit < (16 if f.site == "Q" else 32)
        last = min(w.Lk - 1, f.row + off) if w.causal else w.Lk - 1
        assert 0 <= f.tile * bc <= last
    else:
        assert f.site in ("V", "VS")
        assert 0 <= f.row < w.Lk and 0 <= f.col < (w.d if f.site == "V" else 2)
        assert 0 <= f.bit < 16
        n_qt = (w.Lq + qt - 1) // qt
        assert 0 <= f.tile < n_qt
        # some row of the query tile sees the key
        last_row = min(w.Lq, (f.tile + 1) * qt) - 1
        assert not w.causal or f.row <= last_row + off


@pytest.mark.parametrize("w", [W_C, W.Workload("rect", 2, 3, 300, 77, 64, True, 0.125),
                               W.Workload("nc", 1, 2, 100, 333, 128, False, 0.1)])
def test_draws_are_valid_and_cover_sites_and_bits(w):
    bc, qt = 64, 128
    seen = set()
    for r in range(3000):
        f = C.draw_fault(r, w, bc, qt)
        _valid(f, w, bc, qt)
        seen.add((f.site, f.bit))
    assert {s for s, _ in seen} == set(C.SITES)
    for s in C.SITES:
        assert {b for site, b in seen if site == s} == set(range(C.SITE_BITS[s]))


@pytest.mark.parametrize("w", [W_C, W.Workload("rect", 2, 3, 300, 77, 64, True, 0.125)])
def test_checker_site_draws_are_valid(w):
    bc, qt = 64, 256
    seen = set()
    for r in range(1500):
        f = C.draw_fault(r, w, bc, qt, sites=C.CHECKER_SITES)
        _valid(f, w, bc, qt)
        seen.add(f.site)
    assert seen == set(C.CHECKER_SITES)


def test_draws_are_reproducible():
    a = [C.draw_fault(r, W_C, 64, 128) for r in range(50)]
    b = [C.draw_fault(r, W_C, 64, 128) for r in range(50)]
    assert a == b


def test_classify_outcomes():
    g = torch.randn(8, 16, generator=torch.Generator().manual_seed(3)).to(torch.bfloat16)
    none = torch.zeros(8, dtype=torch.uint8)
    assert C.classify(g.clone(), g, none)["outcome"] == "benign"
    o = g.clone()
    o[3, 5] = o[3, 5] * 4 + 1                        # significant change in row 3
    assert C.classify(o, g, none)["outcome"] == "silent"
    fl = none.clone()
    fl[3] = 1
    r = C.classify(o, g, fl)
    assert r["outcome"] == "detected" and r["rows_significant"] == 1
    assert C.classify(g.clone(), g, fl)["outcome"] == "false_positive"
    tiny = g.clone()
    j = int(tiny[2].float().abs().argmin())       # a small element: its bf16 step is fine
    tiny[2, j] = tiny[2, j] + tiny[2].float().abs().max() * 2 ** -6 * 0.05   # < 2^-8 of row max
    assert not torch.equal(tiny, g)
    res = C.classify(tiny, g, none)
    assert res["outcome"] == "benign"
    fl2 = none.clone()
    fl2[2] = 1
    assert C.classify(tiny, g, fl2)["outcome"] == "detected_minor"
    # one bf16 unit at the row's largest element exceeds 2^-8 of it: a
    # rounding step alone is not significant, two units past the level are
    big = g.clone()
    j = int(big[4].float().abs().argmax())
    one_up = (big[4, j].float() + C.bf16_unit(big[4, j:j + 1])[0] * torch.sign(big[4, j].float()))
    big[4, j] = one_up.to(torch.bfloat16)
    assert float((big[4, j].float() - g[4, j].float()).abs()) > 2 ** -8 * float(g[4].float().abs().max())
    assert C.classify(big, g, none)["outcome"] == "benign"
    big[4, j] = (g[4, j].float() * (1 + 2 ** -5)).to(torch.bfloat16)
    assert C.classify(big, g, none)["outcome"] == "silent"
    u = C.bf16_unit(torch.tensor([1.0, 1.5, -3.0, 0.0, 2.0 ** -126, 2.0 ** -130]).to(torch.bfloat16))
    assert u.tolist() == [2.0 ** -7, 2.0 ** -7, 2.0 ** -6, 0.0, 2.0 ** -133, 2.0 ** -133]
    nan = g.clone()
    nan[1, 1] = float("nan")
    res = C.classify(nan, g, none)
    assert res["outcome"] == "silent" and res["nonfinite"]


def test_summary_counts(tmp_path):
    recs = [
        {"run": 0, "site": "O", "bit": 30, "exponent_bit": True, "outcome": "detected"},
        {"run": 1, "site": "O", "bit": 2, "exponent_bit": False, "outcome": "benign"},
        {"run": 2, "site": "P", "bit": 14, "exponent_bit": True, "outcome": "silent"},
        {"run": 3, "site": "S", "bit": 30, "exponent_bit": True, "outcome": "silent"},
        {"run": 4, "site": "V", "bit": 9, "exponent_bit": True, "outcome": "detected"},
        {"run": 5, "site": "V", "bit": 15, "exponent_bit": False, "outcome": "false_positive"},
    ]
    p = tmp_path / "c.jsonl"
    p.write_text("".join(json.dumps(r) + "\n" for r in recs))
    s = C.summarize(str(p))
    assert s["runs"] == 6
    assert s["headline"]["detected"] == 2 and s["headline"]["silent"] == 1
    assert s["headline"]["rate"] == pytest.approx(2 / 3)
    lo, hi = s["headline"]["wilson95"]
    assert lo < 2 / 3 < hi
    assert s["false_positives"] == 1
    # with S counted: detected 2 of the 4 significant exponent flips
    assert s["headline_with_S"]["detected"] == 2 and s["headline_with_S"]["silent"] == 2
    assert s["S_exponent"]["silent"] == 1 and s["S_exponent"]["detected"] == 0
    assert s["per_site"]["S"]["silent"] == 1
    assert s["per_bit"]["O30"]["detected"] == 1


def test_storage_weights_follow_the_register_sizes():
    w = W.WORKLOADS["dec_l4096"]   # d = 128
    p = C.storage_weights(w, C.PAPER_SITES)
    bits = dict(zip(C.PAPER_SITES, p * (16 * 128 + 32 * 128 + 32 + 32 + 64)))
    assert bits == pytest.approx({"Q": 2048, "O": 4096, "M": 32, "L": 32, "C": 64})
    assert p.sum() == pytest.approx(1.0)
    # the checker's share shrinks as d grows (the paper's trend in Table I)
    w64 = W.Workload("d64", 1, 1, 256, 256, 64, False, 0.125)
    assert C.storage_weights(w64, C.PAPER_SITES)[-1] > p[-1]


def test_storage_weighted_draws_match_the_weights():
    w = W.Workload("t1", 1, 4, 256, 256, 64, True, 0.125)
    p = C.storage_weights(w, C.PAPER_SITES)
    n = 20000
    counts = {s: 0 for s in C.PAPER_SITES}
    for r in range(n):
        f = C.draw_fault(r, w, 64, 256, C.PAPER_SITES, p)
        _valid(f, w, 64, 256)
        counts[f.site] += 1
    for s, pi in zip(C.PAPER_SITES, p):
        sd = (n * pi * (1 - pi)) ** 0.5
        assert abs(counts[s] - n * pi) <= 5 * sd + 1, (s, counts[s], n * pi)


def test_multi_fault_draws_share_a_head_and_are_reproducible():
    w = W.Workload("t1", 2, 4, 256, 256, 128, True, 0.125)
    p = C.storage_weights(w, C.PAPER_SITES)
    ks = set()
    for r in range(500):
        fl = C.draw_faults(r, w, 64, 256, C.PAPER_SITES, p, 1, 5)
        assert 1 <= len(fl) <= 5
        ks.add(len(fl))
        assert len({(f.b, f.h) for f in fl}) == 1
        for f in fl:
            _valid(f, w, 64, 256)
        assert fl == C.draw_faults(r, w, 64, 256, C.PAPER_SITES, p, 1, 5)
    assert ks == {1, 2, 3, 4, 5}
    # one fault per run reproduces the single-fault draw
    assert C.draw_faults(7, w, 64, 256) == [C.draw_fault(7, w, 64, 256)]


def test_sweep_rejects_an_unknown_path():
    """The sweep's entry-point choice is checked before any device work."""
    with pytest.raises(ValueError):
        C.run_sweep(W.WORKLOADS["bert_l128"], 1, None, path="nonsense")
