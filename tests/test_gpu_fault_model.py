"""Injected runs on the GPU against the oracle's fault-outcome model.

Each run flips one bit through the debug entry point and compares, element
by element, the change of O, pred and actual (GPU faulty run minus GPU
fault-free run) with the closed-form prediction of oracle/faults.py on the
same seeded bf16 inputs; the predicted flag must equal the GPU flag. Rows
whose predicted |r| lies within a factor of 2 of the threshold are left out
of the flag comparison (there the fp32 rounding of the kernel decides).

Tolerances, from the arithmetic: the kernel's weights p~ and l carry a bf16
rounding of at most 2^-9 each, so its change differs from the exact-weight
closed form by at most ~2^-8 of the bound the model states (dO_err,
dpred_err; checked with a 2x margin); O is stored in bf16, so each of the two
outputs adds half a unit (2^-9 relative); pred and actual are fp32 sums of
d terms (2^-18 of the row's M covers them).
"""
import dataclasses

import numpy as np
import pytest
import torch

import workloads as W
from oracle import faults as FM
from tests import gpu_helpers as G

pytestmark = pytest.mark.gpu

F = pytest.importorskip("paper_2507_16676_amd")
from paper_2507_16676_amd import campaign as C  # noqa: E402

SITES = ("P", "O", "V", "C", "VS", "L", "S", "Q")


def _head_inputs(inp, b, h):
    return (inp.q[b, h], inp.k[b, h], inp.v[b, h])


class _Head:
    """One head on the GPU with its fault-free debug run, and on the host."""

    def __init__(self, w, inp, b, h):
        self.w = w
        qb, kb, vb = _head_inputs(inp, b, h)
        self.q, self.k, self.v = (G.to_dev(x[None, None]) for x in (qb, kb, vb))
        self.qh = W.bf16_bits_to_f32(qb).astype(np.float64)
        self.kh = W.bf16_bits_to_f32(kb).astype(np.float64)
        self.vh = W.bf16_bits_to_f32(vb).astype(np.float64)
        self.gold = self.run(None)
        assert int(self.gold["flags"].sum()) == 0

    def run(self, fault):
        o, resid, flags, pred, actual = F.attn_fwd_inject(self.q, self.k, self.v,
                                                          causal=self.w.causal,
                                                          scale=self.w.scale, fault=fault)
        torch.cuda.synchronize()
        return {"O": G.from_dev_bf16(o)[0, 0], "bits": o.view(torch.int16)[0, 0].cpu().numpy(),
                "flags": flags[0, 0].cpu().numpy(), "pred": pred[0, 0].double().cpu().numpy(),
                "actual": actual[0, 0].double().cpu().numpy()}


def _run_flag(pr, got, tau):
    """The run's predicted flag (some row flagged) where the model decides
    it: True if a row is predicted non-finite or beyond twice the threshold,
    False if every row is below half of it; None (undetermined) otherwise.
    Rows that only may turn non-finite (0 * inf) count as the GPU left them."""
    clear_true, all_low = False, True
    for i, res in zip(pr["rows"], pr["per_row"]):
        if res["nonfinite"]:
            clear_true = True
            continue
        if res["undetermined"]:
            all_low = False
            continue
        if res["nonfinite_maybe"] and got["flags"][i]:
            clear_true = True
            continue
        ratio = abs(res["resid"]) / (tau * res["M"]) if res["M"] > 0 else 0.0
        if ratio > 2.0:
            clear_true = True
        elif ratio >= 0.5:
            all_low = False
    if clear_true:
        return True
    return False if all_low else None


def _compare_run(head, fault, tau):
    """Run one fault on the GPU and compare with the model, row by row
    (asserting the element-wise bounds and every row flag outside the
    band). Returns the run's record."""
    w = head.w
    bc, qt = F.key_tile(w.d), F.query_tile(w.d)
    local = dataclasses.replace(fault, b=0, h=0)
    got = head.run(local)
    gold = head.gold
    spec = FM.FaultSpec(fault.site, fault.row, fault.col, fault.tile, fault.bit)
    pr = FM.fault_effect(head.qh, head.kh, head.vh, w.causal, w.scale, spec, key_tile=bc,
                         query_tile=qt, tau_rel=tau)
    rows = set(pr["rows"])
    # rows outside the prediction: bitwise unchanged and unflagged
    changed = np.nonzero((got["bits"] != gold["bits"]).any(axis=1))[0]
    assert set(changed.tolist()) <= rows, (fault, sorted(set(changed.tolist()) - rows)[:5])
    flagged = np.nonzero(got["flags"])[0]
    assert set(flagged.tolist()) <= rows, (fault, sorted(set(flagged.tolist()) - rows)[:5])
    n_rows = n_rows_flag = 0
    for i, res in zip(pr["rows"], pr["per_row"]):
        O0, O1 = gold["O"][i], got["O"][i]
        gpu_nonfinite = (not np.all(np.isfinite(O1)) or not np.isfinite(got["pred"][i])
                         or not np.isfinite(got["actual"][i]))
        gpu_flag = bool(got["flags"][i])
        if res["nonfinite"]:
            assert gpu_flag and (got["flags"][i] & F.FLAG_NONFINITE), (fault, i)
            continue
        if (res["nonfinite_maybe"] or res["undetermined"]) and gpu_nonfinite:
            # a non-finite row is always flagged (the kernel's rule)
            assert gpu_flag and (got["flags"][i] & F.FLAG_NONFINITE), (fault, i)
            continue
        if res["undetermined"]:
            continue
        assert not gpu_nonfinite, (fault, i, res)
        n_rows += 1
        rowmax = np.abs(O0).max()
        tol_o = (2.0 ** -7 * res["dO_err"] + 2.0 ** -8 * (np.abs(O0) + np.abs(res["O_new"]))
                 + 2.0 ** -16 * rowmax)
        dO = O1 - O0
        assert np.all(np.abs(dO - res["dO"]) <= tol_o), \
            (fault, i, np.max(np.abs(dO - res["dO"]) - tol_o))
        M = res["M"]
        dpred = got["pred"][i] - gold["pred"][i]
        assert abs(dpred - res["dpred"]) <= 2.0 ** -7 * res["dpred_err"] + 2.0 ** -18 * M, \
            (fault, i, dpred, res["dpred"])
        dact = got["actual"][i] - gold["actual"][i]
        assert abs(dact - res["dactual"]) <= 2.0 ** -7 * res["dactual_err"] + 2.0 ** -18 * M, \
            (fault, i, dact, res["dactual"])
        ratio = abs(res["resid"]) / (tau * M) if M > 0 else 0.0
        if 0.5 <= ratio <= 2.0:
            continue
        n_rows_flag += 1
        assert gpu_flag == res["flag"], (fault, i, ratio, int(got["flags"][i]))
    run_flag = _run_flag(pr, got, tau)
    return {"site": fault.site, "decided": run_flag is not None,
            "agree": run_flag is None or run_flag == bool(len(flagged)),
            "flagged": pr["flagged"], "rows": n_rows, "rows_flag": n_rows_flag}


def _draw(w, n, seed0):
    bc, qt = F.key_tile(w.d), F.query_tile(w.d)
    rng = np.random.default_rng(seed0)
    out = []
    for r in range(n):
        f = C.draw_fault(seed0 + r, w, bc, qt, sites=SITES)
        if r % 4 != 3:   # mostly exponent bits (the headline's high-order bits)
            f = dataclasses.replace(f, bit=int(rng.choice(list(C.EXP_BITS[f.site]))))
        out.append(f)
    return out


W_FM = W.Workload("fm_gpu", 1, 2, 700, 700, 128, True, 128 ** -0.5, seed=61)


def test_injected_runs_match_the_fault_model():
    """320 seeded single flips at P, O, V, C, VS, L, S, Q on a ragged causal
    d = 128 head pair (three query tiles, eleven key tiles, the last one
    ragged): every change of O, pred and actual as predicted, and the run's
    flag as predicted in every run outside the threshold band."""
    tau, _ = F.get_threshold()
    inp = W.make_inputs(W_FM)
    heads = {}
    recs = []
    for f in _draw(W_FM, 320, 7000):
        if (f.b, f.h) not in heads:
            heads[(f.b, f.h)] = _Head(W_FM, inp, f.b, f.h)
        recs.append(_compare_run(heads[(f.b, f.h)], f, tau))
    n = sum(1 for r in recs if r["decided"])
    agree = sum(1 for r in recs if r["agree"] and r["decided"])
    by_site = {s: sum(1 for r in recs if r["site"] == s) for s in SITES}
    print(f"[fault model] {len(recs)} runs, {n} with the flag decided by the model, flag "
          f"agreement {agree}/{n}; rows compared {sum(r['rows'] for r in recs)}, row flags "
          f"compared {sum(r['rows_flag'] for r in recs)}; predicted flagged "
          f"{sum(r['flagged'] for r in recs)}; sites {by_site}", flush=True)
    assert n >= 300
    assert agree >= 0.999 * n


@pytest.mark.parametrize("d", [64, 96])
def test_injected_runs_match_the_fault_model_other_widths(d):
    """The same on d = 64 (the 64-wide kernel, 256-row query tiles) and
    d = 96 (the 128-wide kernel with zero columns), 80 runs each."""
    w = W.Workload(f"fm_gpu{d}", 1, 2, 333, 400, d, True, d ** -0.5, seed=62 + d)
    tau, _ = F.get_threshold()
    inp = W.make_inputs(w)
    heads = {}
    recs = []
    for f in _draw(w, 80, 9000 + d):
        if (f.b, f.h) not in heads:
            heads[(f.b, f.h)] = _Head(w, inp, f.b, f.h)
        recs.append(_compare_run(heads[(f.b, f.h)], f, tau))
    n = sum(1 for r in recs if r["decided"])
    agree = sum(1 for r in recs if r["agree"] and r["decided"])
    print(f"[fault model d={d}] {len(recs)} runs, flag agreement {agree}/{n}", flush=True)
    assert n >= 70 and agree >= 0.999 * n


def test_headline_campaign_runs_match_the_fault_model():
    """The first 300 runs of the headline campaign (the 4096-token causal
    d = 128 workload, its own inputs and draws: sites S, P, O, V, bits
    uniform): the campaign's classification (flagged, significant) of each
    run equals the model's, outside the bands where the residual is within a
    factor 2 of the threshold or an output change within a factor 2 of the
    significance level (widened by the bf16 unit of the element)."""
    w = W.WORKLOADS["dec_l4096"]
    tau, _ = F.get_threshold()
    inp = W.make_inputs(w)
    bc, qt = F.key_tile(w.d), F.query_tile(w.d)
    q, k, v = C.campaign_inputs(w, w.seed)
    # the campaign's device inputs are the host recipe's values
    assert torch.equal(q.view(torch.int16).cpu(), torch.from_numpy(inp.q.view(np.int16)))
    del q, k, v
    heads = {}
    n = agree = 0
    outcomes = {}
    for r in range(300):
        f = C.draw_fault(r, w, bc, qt)
        if (f.b, f.h) not in heads:
            heads[(f.b, f.h)] = _Head(w, inp, f.b, f.h)
        hd = heads[(f.b, f.h)]
        local = dataclasses.replace(f, b=0, h=0)
        o, resid, flags, pred, actual = F.attn_fwd_inject(hd.q, hd.k, hd.v, causal=True,
                                                          scale=w.scale, fault=local)
        if not hasattr(hd, "o_gold"):
            hd.o_gold = F.attn_fwd_inject(hd.q, hd.k, hd.v, causal=True, scale=w.scale)[0]
        res = C.classify(o[0, 0], hd.o_gold[0, 0], flags[0, 0])
        gpu_flag = res["rows_flagged"] > 0
        gpu_sig = res["rows_significant"] > 0
        spec = FM.FaultSpec(f.site, f.row, f.col, f.tile, f.bit)
        pr = FM.fault_effect(hd.qh, hd.kh, hd.vh, True, w.scale, spec, key_tile=bc,
                             query_tile=qt, tau_rel=tau)
        got = {"flags": flags[0, 0].cpu().numpy()}
        run_flag = _run_flag(pr, got, tau)
        # significance, decided the same way: the campaign's level for an
        # element is 2^-8 of the row's largest output plus one bf16 unit u of
        # the element; decided True when some element moves by more than
        # twice (level + 2u), False when every element moves by less than
        # half the level
        sig_true, sig_low = pr["nonfinite"], True
        for rr in pr["per_row"]:
            if rr["nonfinite"] or rr["nonfinite_maybe"] or rr["undetermined"]:
                sig_low = False
                continue
            lvl = FM.SIG_REL * np.abs(rr["O"]).max()
            _, e = np.frexp(rr["O"])
            u = np.where(rr["O"] == 0, 0.0, np.ldexp(1.0, e - 8))
            sig_true |= bool(np.any(np.abs(rr["dO"]) > 2.0 * (lvl + 2.0 * u)))
            sig_low &= bool(np.all(np.abs(rr["dO"]) < 0.5 * lvl))
        run_sig = True if sig_true else (False if sig_low else None)
        key = FM.classify_prediction(pr)
        outcomes[key] = outcomes.get(key, 0) + 1
        if run_flag is None or run_sig is None:
            continue
        n += 1
        ok = gpu_flag == run_flag and gpu_sig == run_sig
        agree += ok
        assert ok, (r, f, res, run_flag, run_sig)
    print(f"[fault model campaign] 300 runs, {n} outside the bands, agreement {agree}/{n}, "
          f"predicted {outcomes}", flush=True)
    assert n >= 200
