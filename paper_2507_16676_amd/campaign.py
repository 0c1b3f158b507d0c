"""Fault-injection campaign and fault-free sweep for the Flash-ABFT kernel.

Section IV-B of the paper flips one bit per run at a random time in a random
register and sorts each run into Detected / False positive / Silent. Here a
run flips one bit at one of the kernel's fault sites (S, P, O, V; see
include/fabft.h), chosen uniformly, at a uniformly drawn live element and
bit, and compares the faulty output with the fault-free output of the same
kernel (which is bitwise deterministic):

  significant   some |O_ij - O*_ij| > 2^-8 * max_j |O*_ij| + u_ij in a row,
                with u_ij one bf16 unit of O*_ij (the rounding of the stored
                value alone), or a non-finite O_ij (O* = fault-free output)
  flagged       some row of the head has a nonzero flag

  Detected = flagged and significant; Detected (minor) = flagged, output
  changed but not significantly; False positive = flagged while the output
  is bitwise unchanged (an alarm with a correct result, the paper's sense);
  Silent = not flagged and significant; Benign = none of these.

The rate reported is Detected / (Detected + Silent) over exponent-bit flips
(fp32 bits 23-30, bf16 bits 7-14), over all sites the campaign draws (S, P,
O, V: headline_with_S) and over P, O and V alone (headline): S-site flips
happen before the checksum tap and change O and pred consistently, so the
output checksum sees them only through non-finite values, and the optional
score check is what covers them.

Only the faulted head is recomputed per run (heads are independent, and the
per-head computation does not depend on the others). Runs are drawn from
numpy PCG64(run id), so a campaign is reproducible and resumable; its inputs
follow the host recipe of workloads.make_inputs, so that any run can be
replayed on the host.

    python -m paper_2507_16676_amd.campaign campaign --runs 10000 --out c.jsonl
    python -m paper_2507_16676_amd.campaign sweep --seeds 10000 --out s.json
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

SITES = ("S", "P", "O", "V")
# checker state (c, l, running max, sumrow record): the paper's false-positive
# sources
CHECKER_SITES = ("C", "L", "M", "VS")
# the storage the paper draws from (Section IV-B): the kernel's per-query
# registers q, o, m, l and the checker's per-query accumulator c
PAPER_SITES = ("Q", "O", "M", "L", "C")
SITE_BITS = {"S": 32, "P": 16, "O": 32, "V": 16, "C": 32, "L": 32, "M": 32, "Q": 16, "VS": 16}
EXP_BITS = {"S": range(23, 31), "P": range(7, 15), "O": range(23, 31), "V": range(7, 15),
            "C": range(23, 31), "L": range(23, 31), "M": range(23, 31), "Q": range(7, 15),
            "VS": range(7, 15)}


def storage_bits(w, site):
    """Bits one query row keeps in `site` for the whole pass: q (d bf16), the
    output accumulator o (d fp32), m and l (fp32 each) and c (an fp32 pair,
    c_hi + c_lo: 64 bits, like the paper's double-precision accumulator)."""
    return {"Q": 16 * w.d, "O": 32 * w.d, "M": 32, "L": 32, "C": 64}[site]


def storage_weights(w, sites):
    """Probability of each site when a flipped bit is drawn uniformly over
    the storage of all sites (each row holds the same storage)."""
    bits = np.array([storage_bits(w, s) for s in sites], dtype=np.float64)
    return bits / bits.sum()
SIG_REL = 2.0 ** -8


def _torch():
    import torch
    return torch


def campaign_inputs(w, seed, device="cuda"):
    """The campaign's inputs: the seeded host recipe of workloads.make_inputs
    (numpy PCG64, rounded to bf16), moved to the GPU, so that every run can
    be replayed on the host from the workload and seed alone."""
    import workloads as W
    torch = _torch()
    inp = W.make_inputs(w, seed=int(seed))

    def dev(bits):
        t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
        return t.view(torch.bfloat16).to(device).contiguous()

    return dev(inp.q), dev(inp.k), dev(inp.v)


def device_inputs(w, seed, device="cuda"):
    """Seeded N(0,1) bf16 inputs of workload w drawn on the GPU (same
    distribution as the host recipe, not the same values; for the fault-free
    sweeps, which need no host replay)."""
    torch = _torch()
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    q = torch.randn((w.B, w.H, w.Lq, w.d), generator=g, device=device)
    k = torch.randn((w.B, w.H, w.Lk, w.d), generator=g, device=device)
    v = torch.randn((w.B, w.H, w.Lk, w.d), generator=g, device=device)
    if w.qk_prescale != 1.0:
        q *= w.qk_prescale
        k *= w.qk_prescale
    if w.peaked_frac > 0:
        n = int(round(w.peaked_frac * w.Lk))
        gc = torch.Generator()
        gc.manual_seed(int(seed) + 1)
        for b in range(w.B):
            for h in range(w.H):
                idx = torch.randperm(w.Lk, generator=gc)[:n].to(device)
                k[b, h, idx] *= w.peaked_mult
    return (q.to(torch.bfloat16).contiguous(), k.to(torch.bfloat16).contiguous(),
            v.to(torch.bfloat16).contiguous())


def draw_fault(run: int, w, key_tile: int, query_tile: int, sites=SITES, weights=None):
    """The fault of run `run`: site, head, element and bit, uniform over live
    elements (visible keys for S/P, processed key tiles for O/Q/C/L/M, query
    tiles that can see the key for V/VS). Sites are equally likely, or drawn
    with probabilities `weights`."""
    return _draw_one(np.random.default_rng(int(run)), w, key_tile, query_tile, sites, weights)


def draw_faults(run: int, w, key_tile: int, query_tile: int, sites=SITES, weights=None,
                kmin=1, kmax=1):
    """The faults of run `run`: k in [kmin, kmax] drawn uniformly, then k
    independent faults as in draw_fault, all in the head of the first one
    (the campaign recomputes one head per run). With kmin = kmax = 1 this is
    [draw_fault(run, ...)]."""
    rng = np.random.default_rng(int(run))
    if kmin == kmax == 1:
        return [_draw_one(rng, w, key_tile, query_tile, sites, weights)]
    k = int(rng.integers(kmin, kmax + 1))
    out = []
    for i in range(k):
        f = _draw_one(rng, w, key_tile, query_tile, sites, weights)
        if i:
            f = type(f)(f.site, out[0].b, out[0].h, f.row, f.col, f.tile, f.bit)
        out.append(f)
    return out


def _draw_one(rng, w, key_tile, query_tile, sites, weights):
    from . import Fault
    if weights is None:
        site = sites[int(rng.integers(len(sites)))]
    else:
        site = sites[int(rng.choice(len(sites), p=np.asarray(weights, dtype=np.float64)))]
    b = int(rng.integers(w.B))
    h = int(rng.integers(w.H))
    off = w.Lk - w.Lq
    bit = int(rng.integers(SITE_BITS[site]))
    if site in ("S", "P", "O", "C", "L", "M", "Q"):
        while True:
            row = int(rng.integers(w.Lq))
            last = min(w.Lk - 1, row + off) if w.causal else w.Lk - 1
            if last >= 0:
                break
        if site in ("O", "C", "L", "M", "Q"):
            col = (int(rng.integers(w.d)) if site in ("O", "Q") else
                   int(rng.integers(2)) if site == "C" else 0)
            tile = int(rng.integers(last // key_tile + 1))
        else:
            col = int(rng.integers(last + 1))
            tile = 0
        return Fault(site, b, h, row, col, tile, bit)
    # V, VS: key k, column j (V) or part (VS), one query tile whose rows can
    # see key k
    n_qt = (w.Lq + query_tile - 1) // query_tile
    while True:
        key = int(rng.integers(w.Lk))
        first = 0
        if w.causal:
            lo_row = key - off          # first row that sees the key
            if lo_row >= w.Lq:
                continue
            first = max(0, lo_row) // query_tile
        break
    col = int(rng.integers(w.d)) if site == "V" else int(rng.integers(2))
    tile = int(rng.integers(first, n_qt))
    return Fault(site, b, h, key, col, tile, bit)


def bf16_unit(x):
    """One bf16 unit in the last place at each element of x (0 at zeros;
    2^-133 below the smallest normal bf16, 2^-126)."""
    torch = _torch()
    xf = x.float()
    _, e = torch.frexp(xf)
    e = torch.clamp(e - 8, min=-133)
    return torch.where(xf == 0, torch.zeros_like(xf), torch.ldexp(torch.ones_like(xf), e))


def classify(o, o_gold, flags):
    """Outcome of one run on one head: tensors [L, d] (bf16) and [L] (u8).
    An element is significantly changed when it moved by more than 2^-8 of
    the row's largest fault-free output plus one bf16 unit of the element:
    the stored bf16 value can move by one unit through rounding alone, and
    at the row's largest element one unit already exceeds 2^-8 of it."""
    torch = _torch()
    of = o.float()
    og = o_gold.float()
    diff = (of - og).abs()
    nonfinite_rows = ~torch.isfinite(of).all(dim=1)
    ref = og.abs().amax(dim=1)
    sig_rows = (diff > SIG_REL * ref[:, None] + bf16_unit(og)).any(dim=1) | nonfinite_rows
    flag_rows = flags != 0
    n_sig = int(sig_rows.sum())
    n_flag = int(flag_rows.sum())
    n_sig_unflagged = int((sig_rows & ~flag_rows).sum())
    changed = int((o.view(torch.int16) != o_gold.view(torch.int16)).any(dim=1).sum())
    sig, flg = n_sig > 0, n_flag > 0
    outcome = ("detected" if flg and sig else
               "detected_minor" if flg and changed else
               "false_positive" if flg else
               "silent" if sig else "benign")
    return {"outcome": outcome, "rows_changed": changed, "rows_significant": n_sig,
            "rows_flagged": n_flag, "rows_significant_unflagged": n_sig_unflagged,
            "nonfinite": bool(nonfinite_rows.any())}


def run_campaign(w, runs, out_path, seed=0, start=0, log_every=1000, sites=SITES, weights=None,
                 kmin=1, kmax=1):
    """Run faults start..runs-1 on workload w (inputs drawn with `seed`),
    appending one JSON line per run to out_path; runs already in the file
    are skipped. Each run injects k in [kmin, kmax] faults (draw_faults)."""
    torch = _torch()
    from . import attn_fwd_inject, global_check, key_tile, query_tile
    done = set()
    if os.path.exists(out_path):
        with open(out_path) as f:
            for line in f:
                try:
                    done.add(json.loads(line)["run"])
                except (ValueError, KeyError):
                    pass
    q, k, v = campaign_inputs(w, seed)
    bc, qt = key_tile(w.d), query_tile(w.d)
    gold = {}
    t0 = time.time()
    n_new = 0
    with open(out_path, "a") as out:
        for r in range(start, runs):
            if r in done:
                continue
            fl = draw_faults(r, w, bc, qt, sites, weights, kmin, kmax)
            f = fl[0]
            b, h = f.b, f.h
            qh, kh, vh = q[b:b + 1, h:h + 1], k[b:b + 1, h:h + 1], v[b:b + 1, h:h + 1]
            if (b, h) not in gold:
                og, _, fg, _, _ = attn_fwd_inject(qh, kh, vh, causal=w.causal, scale=w.scale)
                torch.cuda.synchronize()
                assert int(fg.sum()) == 0, f"fault-free head ({b},{h}) flagged"
                gold[(b, h)] = og
            f_local = [type(x)(x.site, 0, 0, x.row, x.col, x.tile, x.bit) for x in fl]
            o, resid, flags, pred, actual = attn_fwd_inject(qh, kh, vh, causal=w.causal,
                                                            scale=w.scale, fault=f_local)
            res = classify(o[0, 0], gold[(b, h)][0, 0], flags[0, 0])
            # the paper's single check per attention, on the same output
            _, gflag = global_check(o, resid)
            rec = {"run": r, "site": f.site if len(fl) == 1 else "multi", "b": b, "h": h,
                   "row": f.row, "col": f.col, "tile": f.tile, "bit": f.bit,
                   "exponent_bit": any(x.bit in EXP_BITS[x.site] for x in fl),
                   "nfaults": len(fl), **res, "global_flag": int(gflag[0, 0])}
            if len(fl) > 1:
                rec["faults"] = [[x.site, x.row, x.col, x.tile, x.bit] for x in fl]
            out.write(json.dumps(rec) + "\n")
            n_new += 1
            if log_every and n_new % log_every == 0:
                out.flush()
                print(f"[campaign] {n_new} runs, {time.time() - t0:.1f} s", flush=True)
    return summarize(out_path)


def summarize(path):
    recs = [json.loads(l) for l in open(path) if l.strip()]
    table = {}
    for r in recs:
        for key in (("all", r["site"]), ("bit", r["site"], r["bit"])):
            t = table.setdefault(key, {"detected": 0, "detected_minor": 0,
                                       "false_positive": 0, "silent": 0, "benign": 0})
            t[r["outcome"]] += 1

    def wilson(k, n, z=1.96):
        if n == 0:
            return (0.0, 0.0)
        p = k / n
        den = 1 + z * z / n
        c = (p + z * z / (2 * n)) / den
        hw = z * math.sqrt(p * (1 - p) / n + z * z / (4 * n * n)) / den
        return (max(0.0, c - hw), min(1.0, c + hw))

    def exp_rate(sites):
        c = {"detected": 0, "silent": 0}
        for r in recs:
            if r["site"] in sites and r["exponent_bit"] and r["outcome"] in c:
                c[r["outcome"]] += 1
        m = c["detected"] + c["silent"]
        return {"detected": c["detected"], "silent": c["silent"],
                "rate": c["detected"] / m if m else float("nan"),
                "wilson95": wilson(c["detected"], m)}

    head = {"detected": 0, "silent": 0}
    for r in recs:
        if r["site"] in ("P", "O", "V") and r["exponent_bit"]:
            if r["outcome"] in head:
                head[r["outcome"]] += 1
    n = head["detected"] + head["silent"]
    rate = head["detected"] / n if n else float("nan")
    # the same significant runs judged by the global per-head check alone
    gl = {"detected": 0, "silent": 0}
    for r in recs:
        if (r["site"] in ("P", "O", "V") and r["exponent_bit"] and "global_flag" in r
                and r["outcome"] in ("detected", "silent")):
            gl["detected" if r["global_flag"] else "silent"] += 1
    ng = gl["detected"] + gl["silent"]
    per_site = {}
    for s in SITES + CHECKER_SITES + ("Q", "multi"):
        if ("all", s) not in table:
            continue
        t = table.get(("all", s), {})
        tot = sum(t.values())
        per_site[s] = {**t, "runs": tot,
                       "raw_detect_rate": (t.get("detected", 0) / tot) if tot else None}
    per_bit = {f"{s}{b}": table[("bit", s, b)] for (_, s, b) in
               sorted(k for k in table if k[0] == "bit") if s != "multi"}

    # the paper's three classes (Table I): every run that changed something
    # or raised a flag is Detected (flagged, output changed), False positive
    # (flagged, output bitwise unchanged) or Silent (significant error, not
    # flagged); runs that changed the output only below the significance
    # level without a flag, or nothing at all, are counted apart as benign
    def paper_table(rs):
        c = {"detected": 0, "false_positive": 0, "silent": 0, "benign": 0}
        for r in rs:
            o = r["outcome"]
            c["detected" if o in ("detected", "detected_minor") else o] += 1
        nb = c["detected"] + c["false_positive"] + c["silent"]
        pct = {k: (100.0 * c[k] / nb if nb else float("nan"))
               for k in ("detected", "false_positive", "silent")}
        return {"runs": len(rs), **c, "pct_of_non_benign": pct}
    by_k = {}
    for r in recs:
        by_k.setdefault(int(r.get("nfaults", 1)), []).append(r)
    return {"runs": len(recs),
            "headline": {"what": "exponent-bit flips at P, O, V: detected / (detected + silent)",
                         "detected": head["detected"], "silent": head["silent"],
                         "rate": rate, "wilson95": wilson(head["detected"], n)},
            "headline_with_S": {"what": "exponent-bit flips at S, P, O, V (every site the "
                                        "campaign draws): detected / (detected + silent)",
                                **exp_rate(("S", "P", "O", "V"))},
            "S_exponent": {"what": "exponent-bit flips at S alone (before the checksum tap)",
                           **exp_rate(("S",))},
            "headline_global": {"what": "the same significant runs, flagged by the per-head "
                                        "global check (Alg. 3 single check)",
                                "detected": gl["detected"], "silent": gl["silent"],
                                "rate": gl["detected"] / ng if ng else float("nan"),
                                "wilson95": wilson(gl["detected"], ng)},
            "global_false_alarms": sum(1 for r in recs if r.get("global_flag")
                                       and r["outcome"] in ("false_positive", "benign")),
            "false_positives": sum(1 for r in recs if r["outcome"] == "false_positive"),
            "per_site": per_site, "per_bit": per_bit,
            "paper_table": paper_table(recs),
            "paper_table_by_nfaults": {k: paper_table(v) for k, v in sorted(by_k.items())}}


def run_sweep(w, seeds, out_path, seed0=1, rho_every=100, log_every=1000, score_check=False,
              path="forward"):
    """Fault-free runs on seeds seed0..seed0+seeds-1: count flagged rows
    (must be 0) and track rho = max |resid| / (sum_j |O_ij| + |pred|), and
    with the weighted check on, the same ratio for it (rho_w). score_check
    records that the caller switched the score check on (its flags count).
    path: "forward" (fabft_attn_fwd), "splitkv" (the key split with its
    default split count) or "twopass" (the checksum on Algorithm 1); the two
    latter have no debug outputs, so their rho takes pred = resid + sum_j O_ij
    from the bf16 O."""
    torch = _torch()
    from . import (attn_fwd, attn_fwd_inject, attn_fwd_splitkv, attn_fwd_twopass, get_threshold,
                   get_weighted_check)
    if path not in ("forward", "splitkv", "twopass"):
        raise ValueError(f"unknown path {path!r}")
    weighted = get_weighted_check()
    rho_w_max = 0.0
    o = resid = flags = None
    flagged_total = 0
    flagged_seeds = []
    rho_max, rho_seeds = 0.0, 0
    t0 = time.time()
    for i in range(seeds):
        s = seed0 + i
        q, k, v = device_inputs(w, s)
        if path == "splitkv":
            o, resid, flags = attn_fwd_splitkv(q, k, v, causal=w.causal, scale=w.scale)
        elif path == "twopass":
            o, resid, flags = attn_fwd_twopass(q, k, v, causal=w.causal, scale=w.scale)
        else:
            o, resid, flags = attn_fwd(q, k, v, causal=w.causal, scale=w.scale)
        nf = int((flags != 0).sum())
        if nf:
            flagged_total += nf
            flagged_seeds.append(s)
        if rho_every and i % rho_every == 0 and path != "forward":
            of = o.float()
            M = of.abs().sum(dim=-1) + (resid + of.sum(dim=-1)).abs()
            rho_max = max(rho_max, (resid.abs() / M.clamp_min(1e-30)).max().item())
            rho_seeds += 1
        elif rho_every and i % rho_every == 0:
            od, rd, fd, pred, actual, pw, aw = attn_fwd_inject(
                q, k, v, causal=w.causal, scale=w.scale, weighted_out=True)
            absO = od.float().abs().sum(dim=-1)
            M = absO + pred.abs()
            ratio = (rd.abs() / M.clamp_min(1e-30)).max().item()
            rho_max = max(rho_max, ratio)
            if weighted:
                Mw = absO + pw.abs()
                rho_w_max = max(rho_w_max, ((pw - aw).abs() / Mw.clamp_min(1e-30)).max().item())
            rho_seeds += 1
        if log_every and (i + 1) % log_every == 0:
            print(f"[sweep] {i + 1} seeds, flagged rows {flagged_total}, rho max {rho_max:.3e}, "
                  f"{time.time() - t0:.1f} s", flush=True)
    rows = seeds * w.B * w.H * w.Lq
    res = {"workload": w.name, "seeds": seeds, "seed0": seed0, "rows_checked": rows,
           "flagged_rows": flagged_total, "flagged_seeds": flagged_seeds[:100],
           "rho_max": rho_max, "rho_seeds": rho_seeds, "threshold": get_threshold(),
           "weighted_check": weighted, "score_check": bool(score_check), "path": path,
           "seconds": time.time() - t0}
    if weighted:
        res["rho_w_max"] = rho_w_max
    if out_path:
        with open(out_path, "w") as f:
            json.dump(res, f, indent=1)
    return res


def main(argv=None):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import workloads as W
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("campaign")
    c.add_argument("--workload", default="dec_l4096")
    c.add_argument("--runs", type=int, default=10000)
    c.add_argument("--start", type=int, default=0)
    c.add_argument("--seed", type=int, default=0)
    c.add_argument("--out", required=True)
    c.add_argument("--summary")
    c.add_argument("--weighted", action="store_true",
                   help="also run the weighted (alternating-sign) checksum")
    c.add_argument("--score-check", action="store_true",
                   help="also run the score check (row sums of Q K^T)")
    c.add_argument("--sites", default=None,
                   help="comma-separated fault sites to draw from (S,P,O,V,C,L,M,Q,VS); "
                        "default S,P,O,V, or Q,O,M,L,C with --storage-weighted")
    c.add_argument("--storage-weighted", action="store_true",
                   help="draw sites with probability proportional to their storage bits "
                        "(sites Q,O,M,L,C: the paper's per-query registers)")
    c.add_argument("--faults", default="1",
                   help="faults per run: K or KMIN-KMAX (drawn uniformly; one head per run)")
    c.add_argument("--algorithm", type=int, default=3, choices=(1, 3),
                   help="the algorithm hosting the checksum: 3 (one pass) or 1 (two passes)")
    s = sub.add_parser("sweep")
    s.add_argument("--workload", default="dec_l4096")
    s.add_argument("--seeds", type=int, default=10000)
    s.add_argument("--seed0", type=int, default=1)
    s.add_argument("--rho-every", type=int, default=100)
    s.add_argument("--out", required=True)
    s.add_argument("--weighted", action="store_true",
                   help="also run the weighted (alternating-sign) checksum")
    s.add_argument("--score-check", action="store_true",
                   help="also run the score check (row sums of Q K^T); its flags count too")
    s.add_argument("--path", default="forward", choices=("forward", "splitkv", "twopass"),
                   help="the entry point swept: the forward, the key split or the two-pass form")
    a = ap.parse_args(argv)
    w = W.WORKLOADS[a.workload]
    if getattr(a, "algorithm", 3) != 3:
        from . import set_algorithm
        set_algorithm(a.algorithm)
    if a.weighted:
        from . import set_weighted_check
        set_weighted_check(True)
    if a.cmd == "campaign":
        if a.score_check:
            import torch
            from . import score_check_workspace_bytes, set_score_check
            # the campaign recomputes one head per run
            ws = torch.empty(score_check_workspace_bytes(1, 1, w.Lk, w.d), dtype=torch.uint8,
                             device="cuda")
            set_score_check(ws)
        sites = tuple(a.sites.split(",")) if a.sites else (
            PAPER_SITES if a.storage_weighted else SITES)
        weights = storage_weights(w, sites) if a.storage_weighted else None
        kmin, _, kmax = a.faults.partition("-")
        kmin = int(kmin)
        kmax = int(kmax) if kmax else kmin
        summ = run_campaign(w, a.runs, a.out, seed=a.seed, start=a.start, sites=sites,
                            weights=weights, kmin=kmin, kmax=kmax)
        summ["sites"] = list(sites)
        summ["site_weights"] = None if weights is None else [float(x) for x in weights]
        summ["faults_per_run"] = [kmin, kmax]
        summ["weighted_check"] = bool(a.weighted)
        summ["score_check"] = bool(a.score_check)
        txt = json.dumps(summ, indent=1)
        if a.summary:
            with open(a.summary, "w") as f:
                f.write(txt)
        print(json.dumps({"runs": summ["runs"], "headline": summ["headline"],
                          "false_positives": summ["false_positives"],
                          "paper_table": summ["paper_table"]}))
    else:
        if a.score_check:
            import torch
            from . import score_check_workspace_bytes, set_score_check
            ws = torch.empty(score_check_workspace_bytes(w.B, w.H, w.Lk, w.d), dtype=torch.uint8,
                             device="cuda")
            set_score_check(ws)
        print(json.dumps(run_sweep(w, a.seeds, a.out, seed0=a.seed0, rho_every=a.rho_every,
                                   score_check=a.score_check, path=a.path)))


if __name__ == "__main__":
    main()
