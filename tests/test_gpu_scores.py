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


def test_q_faults_and_the_masked_tiles(score_check):
    w = CASES[0]
    q, k, v = G.dev_inputs(W.make_inputs(w))
    # the score of key 250 for row 250 sits in the masked diagonal tile: the
    # second product of that tile catches it, and only that row is flagged
    for col, bit in ((250, 24), (200, 29), (192, 30)):
        f = F.Fault("S", b=0, h=0, row=250, col=col, bit=bit)
        o, r, fl, _, _ = F.attn_fwd_inject(q, k, v, causal=True, scale=w.scale, fault=f)
        torch.cuda.synchronize()
        assert int(fl[0, 0, 250]) & F.FLAG_SCORES, (col, bit)
        others = fl.clone()
        others[0, 0, 250] = 0
        assert int(others.sum()) == 0
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


# --------------------------------------------------------------------------
# parity of the score check's sums with the oracle (Section II's row
# checksum of a matrix product, applied to S = Q K^T)
# --------------------------------------------------------------------------

from oracle import faults as FM  # noqa: E402

PARITY_CASES = CASES + [W.Workload("s_dec", 1, 4, 1024, 1024, 128, True, 128 ** -0.5, seed=25),
                        W.Workload("s_long_keys", 1, 2, 64, 3000, 128, True, 128 ** -0.5, seed=26),
                        W.Workload("s_more_q", 1, 2, 500, 130, 64, True, 0.125, seed=27)]


def _scores_debug(w, q, k, v, fault=None):
    r = F.attn_fwd_debug(q, k, v, causal=w.causal, scale=w.scale, fault=fault,
                         outputs=("score_lhs", "score_rhs", "score_bound"))
    torch.cuda.synchronize()
    return {x: r[x].double().cpu().numpy() for x in ("score_lhs", "score_rhs", "score_bound",
                                                        "flags")} | {"o": r["o"]}


@pytest.mark.parametrize("w", PARITY_CASES, ids=[c.name for c in PARITY_CASES])
def test_score_sums_match_the_oracle(w, score_check):
    """Every row's lhs (sum of its raw scores over the wave's unmasked key
    tiles), rhs (q_i . the sum of those keys) and bound (|q_i| . sum |K_k|)
    equal the oracle's within 2^-20 of the bound (fp32 sums of fp32 MFMA
    scores; the check's own threshold is 2^-22 of it and fault-free rows
    stay below 2^-25)."""
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    got = _scores_debug(w, q, k, v)
    qf, kf, _ = inp.as_f32()
    for b in range(w.B):
        for h in range(w.H):
            for i in range(w.Lq):
                ref = FM.score_check_row(qf[b, h], kf[b, h], i, w.Lq, w.causal)
                tol = 2.0 ** -20 * ref["ms"] + 1e-30
                assert abs(got["score_lhs"][b, h, i] - ref["lhs"]) <= tol, (b, h, i, ref)
                assert abs(got["score_rhs"][b, h, i] - ref["rhs"]) <= tol, (b, h, i, ref)
                assert abs(got["score_bound"][b, h, i] - ref["ms"]) <= tol, (b, h, i, ref)
    assert int(got["flags"].sum()) == 0


def test_score_outputs_are_zero_with_the_check_off():
    w = CASES[0]
    q, k, v = G.dev_inputs(W.make_inputs(w))
    got = _scores_debug(w, q, k, v)
    assert not got["score_lhs"].any() and not got["score_rhs"].any()
    assert not got["score_bound"].any()


def _fault_runs(w, n, seed):
    """Seeded S and Q flips (S: any visible key; Q: any column, from a key
    tile the row processes), exponent bits mostly."""
    rng = np.random.default_rng(seed)
    out = []
    off = w.Lk - w.Lq
    for r in range(n):
        site = "S" if r % 2 == 0 else "Q"
        b, h = int(rng.integers(w.B)), int(rng.integers(w.H))
        i = int(rng.integers(max(0, -off), w.Lq))
        last = min(w.Lk - 1, i + off) if w.causal else w.Lk - 1
        bit = (int(rng.integers(23, 31)) if site == "S" else int(rng.integers(7, 15))) \
            if r % 4 < 3 else int(rng.integers(32 if site == "S" else 16))
        if site == "S":
            out.append(F.Fault("S", b=b, h=h, row=i, col=int(rng.integers(last + 1)), bit=bit))
        else:
            out.append(F.Fault("Q", b=b, h=h, row=i, col=int(rng.integers(w.d)),
                               tile=int(rng.integers(last // 64 + 1)), bit=bit))
    return out


@pytest.mark.parametrize("w", [PARITY_CASES[4], CASES[1]], ids=["causal1024", "rect64"])
def test_score_faults_match_the_oracle(w, score_check):
    """120 seeded S and Q flips: the faulted row's lhs, rhs and bound as the
    oracle predicts (within 2^-20 of the bound plus the changed terms' own
    magnitude, which a flip scales with the score's fp32 rounding),
    and its score flag as predicted outside the band where |lhs - rhs| is
    within a factor 2 of the threshold; no other row is flagged."""
    inp = W.make_inputs(w)
    q, k, v = G.dev_inputs(inp)
    qf, kf, _ = inp.as_f32()
    tau_s = F.get_score_threshold()
    n_dec = agree = 0
    for f in _fault_runs(w, 120, seed=31 + w.d):
        got = _scores_debug(w, q, k, v, fault=f)
        pr = FM.score_check_fault(qf[f.b, f.h], kf[f.b, f.h], f.row, w.Lq, w.causal,
                                  FM.FaultSpec(f.site, f.row, f.col, f.tile, f.bit),
                                  tau_s=tau_s)
        i = f.row
        gl, gr, gb = (got[x][f.b, f.h, i] for x in ("score_lhs", "score_rhs", "score_bound"))
        fl = int(got["flags"][f.b, f.h, i])
        others = got["flags"].copy()
        others[f.b, f.h, i] = 0
        assert int(others.sum()) == 0, f
        if pr["nonfinite"]:
            # a non-finite score sum makes the row non-finite (flag bits 0, 1)
            assert fl & F.FLAG_NONFINITE, (f, pr, fl)
            continue
        if pr["undetermined"]:
            # sums near the fp32 range: a non-finite result is still flagged
            if not (np.isfinite(gl) and np.isfinite(gr)):
                assert fl & F.FLAG_NONFINITE, (f, pr, fl)
            continue
        tol = 2.0 ** -20 * (pr["ms"] + pr["term"])
        assert abs(gl - pr["lhs"]) <= tol, (f, gl, pr)
        assert abs(gr - pr["rhs"]) <= tol, (f, gr, pr)
        assert abs(gb - pr["ms"]) <= tol, (f, gb, pr)
        ratio = abs(pr["lhs"] - pr["rhs"]) / (tau_s * pr["ms"]) if pr["ms"] > 0 else 0.0
        if pr["dup_undetermined"] or (0.5 <= ratio <= 2.0 and not pr["dup_flag"]):
            continue
        n_dec += 1
        agree += bool(fl & F.FLAG_SCORES) == pr["flag"]
        assert bool(fl & F.FLAG_SCORES) == pr["flag"], (f, ratio, fl)
    print(f"[scores] {w.name}: score flag agreement {agree}/{n_dec}", flush=True)
    assert n_dec >= 100
