"""Pins of the fault-outcome model (oracle/faults.py), on the CPU.

The closed forms predict what one bit flip does to O, pred and actual. They
are checked against a pure-Python brute force that runs the one-pass
recurrence of Algorithm 3 key tile by key tile, with the kernel's exponent
reference and bf16 weights, and flips the bit literally at the site while
it runs. Two brute-force modes:
  * rounded: the weights are bf16 as in the kernel; the closed forms (which
    use the exact softmax weights) must agree to the bf16 rounding of the
    weights (2^-7 relative, with an absolute floor);
  * exact: the weights keep fp64 and the flip multiplies the site value by
    the factor f that the rounded run saw; the closed forms must then agree
    to 1e-10 relative.
Plus the site values themselves (bit for bit), and special cases with a
known answer (sign flips, flips at the last tile, l flips that cancel).
"""
import math
import struct

import numpy as np
import pytest

import workloads as W
from oracle import faults as FM

LOG2E32 = struct.unpack("<f", struct.pack("<f", 1.4426950408889634))[0]


# ---- storage formats, written out again here with struct (pure Python) ----

def f32(x):
    return struct.unpack("<f", struct.pack("<f", x))[0]


def f32_flip(x, bit):
    (u,) = struct.unpack("<I", struct.pack("<f", x))
    return struct.unpack("<f", struct.pack("<I", u ^ (1 << bit)))[0]


def bf16(x):
    """Round to bf16 (nearest, ties to even) via the fp32 pattern."""
    (u,) = struct.unpack("<I", struct.pack("<f", x))
    keep, rest = u >> 16, u & 0xFFFF
    if rest > 0x8000 or (rest == 0x8000 and keep & 1):
        keep += 1
    return struct.unpack("<f", struct.pack("<I", (keep & 0xFFFF) << 16))[0]


def bf16_flip(x, bit):
    (u,) = struct.unpack("<I", struct.pack("<f", x))
    assert u & 0xFFFF == 0
    return struct.unpack("<f", struct.pack("<I", u ^ (1 << (16 + bit))))[0]


def brute(q, k, v, causal, scale, fault, key_tile, query_tile, exact=False, factor=None):
    """Run every row through the tiled recurrence, flip the fault's bit at
    its site, return per-row (O, pred, actual) lists and the site value x
    (before the flip) of the faulted row/key."""
    Lq, d = len(q), len(q[0])
    Lk = len(k)
    off = Lk - Lq
    # the kernel's fp32 exponent scale; fp64 in the exact mode, where the
    # weights are exp(scale * s) to fp64 rounding
    sl2 = scale / math.log(2.0) if exact else max(f32(f32(scale) * LOG2E32), 2.0 ** -126)
    vs = [f32(sum(v[kk][j] for j in range(d))) for kk in range(Lk)]
    hi = [bf16(x) for x in vs]
    lo = [bf16(vs[kk] - hi[kk]) for kk in range(Lk)]
    site = fault.site if fault is not None else None
    site_x = [None]
    out = []
    for i in range(Lq):
        w0 = 32 * (i // 32)
        last_t = (Lk - 1) // key_tile
        if causal:
            last_t = min(last_t, (w0 + 31 + off) // key_tile) if w0 + 31 + off >= 0 else -1
        in_wg = fault is not None and site in ("V", "VS") and \
            fault.tile * query_tile <= i < (fault.tile + 1) * query_tile
        qi = list(q[i])
        ref = -math.inf
        o = [0.0] * d
        # c and l in two partial sums: keys with k mod 16 < 8 (half 0) and
        # the rest (half 1); the C and L sites flip half 0
        l = [0.0, 0.0]
        chi = [0.0, 0.0]
        clo = [0.0, 0.0]
        for t in range(last_t + 1):
            if site == "Q" and i == fault.row and t == fault.tile:
                x = qi[fault.col]
                site_x[0] = x
                qi[fault.col] = x * factor if exact else bf16_flip(x, fault.bit)
            keys = range(t * key_tile, min(Lk, (t + 1) * key_tile))
            s = {}
            for kk in keys:
                if causal and kk > i + off:
                    continue
                sc = sum(qi[j] * k[kk][j] for j in range(d))
                if site == "S" and i == fault.row and kk == fault.col:
                    site_x[0] = sc
                    sc = sc * factor if exact else f32_flip(f32(sc), fault.bit)
                s[kk] = sc
            mt = max((s[kk] * sl2 for kk in s), default=-math.inf)
            if not exact and mt != -math.inf:
                mt = f32(mt)
            new = mt if mt > ref + FM.LAZY else ref
            if new != ref and ref != -math.inf:
                a = 2.0 ** (ref - new)
                o = [x * a for x in o]
                l, chi, clo = [x * a for x in l], [x * a for x in chi], [x * a for x in clo]
            ref = new
            p = {}
            for kk in keys:
                if kk in s:
                    w = 2.0 ** (s[kk] * sl2 - ref)
                    p[kk] = w if exact else bf16(w)
                else:
                    p[kk] = 0.0
            for kk in keys:
                h, lw = hi[kk], lo[kk]
                if site == "VS" and in_wg and kk == fault.row:
                    x = h if fault.col == 0 else lw
                    site_x[0] = x
                    xn = x * factor if exact else bf16_flip(x, fault.bit)
                    if fault.col == 0:
                        h = xn
                    else:
                        lw = xn
                hf = 0 if kk % 16 < 8 else 1
                l[hf] += p[kk]
                chi[hf] += p[kk] * h
                clo[hf] += p[kk] * lw
            for kk in keys:
                w = p[kk]
                if site == "P" and i == fault.row and kk == fault.col:
                    site_x[0] = w
                    w = w * factor if exact else bf16_flip(w, fault.bit)
                for j in range(d):
                    vv = v[kk][j]
                    if site == "V" and in_wg and kk == fault.row and j == fault.col:
                        site_x[0] = vv
                        vv = vv * factor if exact else bf16_flip(vv, fault.bit)
                    o[j] += w * vv
            if i == getattr(fault, "row", None) and t == getattr(fault, "tile", None):
                if site == "O":
                    x = o[fault.col]
                    site_x[0] = f32(x)
                    o[fault.col] = x * factor if exact else f32_flip(f32(x), fault.bit)
                elif site == "C":
                    x = chi[0] if fault.col == 0 else clo[0]
                    site_x[0] = f32(x)
                    xn = x * factor if exact else f32_flip(f32(x), fault.bit)
                    if fault.col == 0:
                        chi[0] = xn
                    else:
                        clo[0] = xn
                elif site == "L":
                    site_x[0] = f32(l[0])
                    l[0] = l[0] * factor if exact else f32_flip(f32(l[0]), fault.bit)
        lt = l[0] + l[1]
        inv = 1.0 / lt if lt > 0 else 0.0
        O = [x * inv for x in o]
        out.append((O, (chi[0] + chi[1] + clo[0] + clo[1]) * inv, sum(O)))
    return out, site_x[0]


def _inputs(Lq, Lk, d, seed):
    w = W.Workload("fm", 1, 1, Lq, Lk, d, True, 1.0, seed=seed)
    q, k, v = W.make_inputs(w).as_f32()
    return (q[0, 0].astype(np.float64), k[0, 0].astype(np.float64),
            v[0, 0].astype(np.float64))


def _lists(a):
    return [[float(x) for x in r] for r in a]


def _factor(site, x, bit):
    xn = FM.flip_bf16(x, bit) if site in ("P", "V", "VS", "Q") else FM.flip_f32(x, bit)
    return xn / x


SITE_BITS = {"P": 16, "V": 16, "VS": 16, "O": 32, "C": 32, "L": 32, "Q": 16, "S": 32}


def _cases():
    """Seeded faults on small shapes (Lq, Lk up to 70, two 32-row waves),
    key tiles of 4 keys, query tiles of 8 rows."""
    rng = np.random.default_rng(5)
    cases = []
    for n in range(140):
        causal = bool(n % 2)
        Lq = int(rng.integers(3, 41))
        Lk = int(rng.integers(3, 41)) if n % 3 else Lq
        if n % 7 == 0:
            Lq, Lk = 40 + int(rng.integers(0, 30)), 40 + int(rng.integers(0, 30))
        d = int(rng.integers(1, 5))
        site = ("P", "O", "V", "C", "VS", "L", "Q", "S")[n % 8]
        bit = int(rng.integers(SITE_BITS[site]))
        if n % 4 != 3:   # mostly exponent bits, as in the headline
            bit = int(rng.integers(7, 15)) if SITE_BITS[site] == 16 else int(rng.integers(23, 31))
        cases.append((n, causal, Lq, Lk, d, site, bit))
    return cases


def _draw_fault(rng, site, bit, Lq, Lk, causal, key_tile, query_tile):
    off = Lk - Lq
    while True:
        i = int(rng.integers(Lq))
        last = min(Lk - 1, i + off) if causal else Lk - 1
        if last >= 0:
            break
    if site in ("P", "S"):
        return FM.FaultSpec(site, i, int(rng.integers(last + 1)), 0, bit)
    if site in ("O", "C", "L", "Q"):
        col = {"O": None, "C": int(rng.integers(2)), "L": 0, "Q": None}[site]
        return FM.FaultSpec(site, i, col, int(rng.integers(last // key_tile + 1)), bit)
    kk = int(rng.integers(Lk))
    first = max(0, kk - off) // query_tile if causal else 0
    n_qt = (Lq + query_tile - 1) // query_tile
    if causal and kk - off >= Lq:
        kk = Lk - 1 - int(rng.integers(min(Lk, Lq)))
        first = max(0, kk - off) // query_tile
    qt = int(rng.integers(first, n_qt))
    return FM.FaultSpec(site, kk, 0, qt, bit)


KT, QT = 4, 8


@pytest.mark.parametrize("n,causal,Lq,Lk,d,site,bit", _cases())
def test_prediction_matches_brute_force(n, causal, Lq, Lk, d, site, bit):
    q, k, v = _inputs(Lq, Lk, d, seed=100 + n)
    rng = np.random.default_rng(200 + n)
    f = _draw_fault(rng, site, bit, Lq, Lk, causal, KT, QT)
    if f.col is None:
        f = FM.FaultSpec(f.site, f.row, int(rng.integers(d)), f.tile, f.bit)
    scale = 0.7
    pred = FM.fault_effect(q, k, v, causal, scale, f, key_tile=KT, query_tile=QT)
    clean, _ = brute(_lists(q), _lists(k), _lists(v), causal, scale, None, KT, QT)
    faulty, x = brute(_lists(q), _lists(k), _lists(v), causal, scale, f, KT, QT)
    rows = pred["rows"]
    # rows outside the prediction are untouched
    for i in range(Lq):
        if i not in rows:
            assert faulty[i] == clean[i], (i, rows)
    for i, res in zip(rows, pred["per_row"]):
        O0, p0, a0 = clean[i]
        O1, p1, a1 = faulty[i]
        bad = not (all(math.isfinite(z) for z in O1) and math.isfinite(p1) and math.isfinite(a1))
        if res["nonfinite"]:
            assert bad, (i, O1, p1)
            continue
        if res["nonfinite_maybe"] or res["undetermined"]:
            continue
        assert not bad, (i, res)
        dO_b = np.array(O1) - np.array(O0)
        # the brute force rounds the weights to bf16, the closed forms use
        # the exact softmax: they differ by at most ~2^-8 of the bound the
        # model states (checked with a 2x margin), plus fp64 rounding
        tiny = 1e-12 * (np.abs(np.array(O0)).sum() + abs(p0) + 1e-300)
        assert np.all(np.abs(dO_b - res["dO"]) <= 2.0 ** -7 * res["dO_err"] + tiny), \
            (i, dO_b, res["dO"], res["dO_err"])
        assert abs((p1 - p0) - res["dpred"]) <= 2.0 ** -7 * res["dpred_err"] + tiny, \
            (i, p1 - p0, res["dpred"], res["dpred_err"])
        assert abs((a1 - a0) - res["dactual"]) <= 2.0 ** -7 * res["dactual_err"] + d * tiny, \
            (i, a1 - a0, res["dactual"], res["dactual_err"])
    # exact weights, the same factor: the closed forms hold to rounding of fp64
    if x is None or not math.isfinite(x) or x == 0.0 or pred["nonfinite"] or pred["nonfinite_maybe"]:
        return
    fac = _factor(site, x, bit)
    if not math.isfinite(fac) or site in ("S", "Q"):
        return   # S, Q: the exact run differs in which keys set the reference only
    clean_e, _ = brute(_lists(q), _lists(k), _lists(v), causal, scale, None, KT, QT, exact=True)
    faulty_e, _ = brute(_lists(q), _lists(k), _lists(v), causal, scale, f, KT, QT, exact=True,
                        factor=fac)
    for i, res in zip(rows, pred["per_row"]):
        O0, p0, a0 = clean_e[i]
        O1, p1, a1 = faulty_e[i]
        if not all(math.isfinite(z) for z in O1):
            continue
        sc = np.abs(np.array(O0)).max() + np.abs(res["dO"]).max() + abs(p0) + 1e-300
        assert np.all(np.abs((np.array(O1) - np.array(O0)) - res["dO"]) <= 1e-10 * sc), i
        assert abs((p1 - p0) - res["dpred"]) <= 1e-10 * (sc + abs(res["dpred"]))
        assert abs((a1 - a0) - res["dactual"]) <= 1e-10 * (sc * d + abs(res["dactual"]))


@pytest.mark.parametrize("causal", [False, True])
def test_site_values_match_the_brute_force_bit_for_bit(causal):
    """The weights and accumulators the model flips are the ones the
    tiled recurrence holds (both in fp64, different code)."""
    q, k, v = _inputs(37, 45, 3, seed=9)
    scale = 0.9
    for i in (0, 5, 36):
        for kk in range(0, 45, 7):
            if causal and kk > i + 8:
                continue
            f = FM.FaultSpec("P", i, kk, 0, 0)
            _, x = brute(_lists(q), _lists(k), _lists(v), causal, scale, f, KT, QT)
            vis = FM._visible(i, 37, 45, causal)
            vs, hi, lo = FM._sumrow_parts(v)
            fr = FM.row_frame(k @ q[i], vis, FM.exp2_scale(scale), v, hi, lo, KT)
            assert fr["ptil"][kk] == x
        last = min(44, i + 8) if causal else 44
        for t in range(last // KT + 1):
            for site, col in (("O", 1), ("C", 0), ("C", 1), ("L", 0)):
                f = FM.FaultSpec(site, i, col, t, 0)
                _, x = brute(_lists(q), _lists(k), _lists(v), causal, scale, f, KT, QT)
                vis = FM._visible(i, 37, 45, causal)
                vs, hi, lo = FM._sumrow_parts(v)
                fr = FM.row_frame(k @ q[i], vis, FM.exp2_scale(scale), v, hi, lo, KT)
                mv = {"O": fr["o"][t][1],
                      "C": fr["c_hi_half"][t] if col == 0 else fr["c_lo_half"][t],
                      "L": fr["l_half"][t]}[site]
                assert float(np.float32(mv)) == x, (site, i, t)


def test_sign_flip_of_a_weight_reverses_its_term():
    """f = -1: dO_i = -2 P_ik V_k and dactual = -2 P_ik vs_k exactly in the
    closed form; pred does not move."""
    q, k, v = _inputs(20, 20, 4, seed=3)
    import oracle
    ref = oracle.attention_head(q, k, v, True, 0.5)
    f = FM.FaultSpec("P", 12, 5, 0, 15)
    r = FM.fault_effect(q, k, v, True, 0.5, f, key_tile=KT, query_tile=QT)["per_row"][0]
    s = 0.5 * (k @ q[12])
    s[13:] = -np.inf
    P = np.exp(s - s.max())
    P /= P.sum()
    assert np.allclose(r["dO"], -2 * P[5] * v[5], rtol=1e-12, atol=1e-15)
    assert r["dpred"] == 0.0
    assert np.isclose(r["dactual"], -2 * P[5] * v[5].sum(), rtol=1e-12)
    assert np.allclose(r["O"], ref["O"][12], rtol=1e-12)


def test_output_flip_at_the_last_tile_scales_the_output():
    """A flip of o_ij after the row's last key tile multiplies O_ij by f."""
    q, k, v = _inputs(30, 30, 3, seed=4)
    i, j = 29, 2
    last_t = 29 // KT
    for bit in (23, 26, 31):
        f = FM.FaultSpec("O", i, j, last_t, bit)
        r = FM.fault_effect(q, k, v, True, 0.6, f, key_tile=KT, query_tile=QT)["per_row"][0]
        vis = FM._visible(i, 30, 30, True)
        vs, hi, lo = FM._sumrow_parts(v)
        fr = FM.row_frame(k @ q[i], vis, FM.exp2_scale(0.6), v, hi, lo, KT)
        x = float(np.float32(fr["o"][last_t][j]))
        fac = FM.flip_f32(x, bit) / x
        assert math.isclose(r["dO"][j], (fac - 1) * r["O"][j], rel_tol=1e-12)
        assert np.count_nonzero(r["dO"]) == 1


def test_l_flip_cancels_in_the_check():
    """l divides o and c alike: the residual stays 0 and O, pred scale
    together."""
    q, k, v = _inputs(25, 25, 4, seed=6)
    for bit in (23, 25, 28, 31):
        r = FM.fault_effect(q, k, v, True, 0.5, FM.FaultSpec("L", 20, 0, 2, bit),
                            key_tile=KT, query_tile=QT)["per_row"][0]
        assert abs(r["resid"]) <= 1e-12 * (r["M"] + 1)
        if r["pred"] != 0 and r["pred_new"] != 0:
            assert math.isclose(r["pred_new"] / r["pred"], r["O_new"][0] / r["O"][0],
                                rel_tol=1e-9)


def test_value_flip_moves_one_column_of_the_rows_that_see_it():
    q, k, v = _inputs(20, 24, 4, seed=8)
    f = FM.FaultSpec("V", 10, 3, 1, 12)   # key 10, column 3, query tile 1 (rows 8..15)
    pr = FM.fault_effect(q, k, v, True, 0.5, f, key_tile=KT, query_tile=QT)
    assert pr["rows"] == list(range(8, 16))
    for i, r in zip(pr["rows"], pr["per_row"]):
        sees = 10 <= i + 4
        assert (np.count_nonzero(r["dO"]) == 1) == sees
        if sees:
            assert r["dO"][3] != 0 and math.isclose(r["dactual"], r["dO"][3], rel_tol=1e-12)
        assert r["dpred"] == 0.0


def test_score_check_row_brute_force():
    """lhs = sum of raw scores over the wave's full key tiles, rhs = q . sum
    of those keys; brute force on small shapes with 64-key tiles."""
    for Lq, Lk, causal in ((100, 200, True), (150, 150, True), (70, 300, False), (200, 100, True)):
        q, k, _ = _inputs(Lq, Lk, 3, seed=Lq + Lk)
        for i in (0, 31, 32, 63, 64, Lq - 1):
            r = FM.score_check_row(q, k, i, Lq, causal, key_tile=64)
            w0 = 32 * (i // 32)
            n = 0
            for t in range(Lk // 64):
                full = (t * 64 + 64 <= Lk) and (not causal or t * 64 + 63 <= w0 + (Lk - Lq))
                if not full:
                    break
                n = (t + 1) * 64
            assert r["n"] == n
            lhs = sum(sum(q[i][j] * k[kk][j] for j in range(3)) for kk in range(n))
            rhs = sum(q[i][j] * sum(k[kk][j] for kk in range(n)) for j in range(3))
            ms = sum(abs(q[i][j]) * sum(abs(k[kk][j]) for kk in range(n)) for j in range(3))
            assert math.isclose(r["lhs"], lhs, rel_tol=1e-12, abs_tol=1e-12)
            assert math.isclose(r["rhs"], rhs, rel_tol=1e-12, abs_tol=1e-12)
            assert math.isclose(r["ms"], ms, rel_tol=1e-12, abs_tol=1e-12)
            assert abs(r["lhs"] - r["rhs"]) <= 1e-12 * (r["ms"] + 1)


def test_a_planted_sign_error_is_caught():
    """A plausible mistake in the closed form (the factor as 1 - f instead of
    f - 1) disagrees with the brute force."""
    q, k, v = _inputs(16, 16, 3, seed=12)
    f = FM.FaultSpec("P", 9, 4, 0, 9)
    r = FM.fault_effect(q, k, v, True, 0.8, f, key_tile=KT, query_tile=QT)["per_row"][0]
    clean, _ = brute(_lists(q), _lists(k), _lists(v), True, 0.8, None, KT, QT)
    faulty, _ = brute(_lists(q), _lists(k), _lists(v), True, 0.8, f, KT, QT)
    dO_b = np.array(faulty[9][0]) - np.array(clean[9][0])
    assert np.allclose(dO_b, r["dO"], rtol=2 ** -7, atol=1e-9)
    assert not np.allclose(dO_b, -r["dO"], rtol=2 ** -7, atol=1e-9)


@pytest.mark.parametrize("site,bit", [("S", 24), ("S", 29), ("S", 31), ("Q", 9), ("Q", 13), ("Q", 15)])
def test_score_check_fault_brute_force(site, bit):
    """The score check after an S or Q flip, by brute force: lhs sums the
    scores as computed with the flipped value, rhs and the bound use the
    final q (64-key tiles, causal 150 x 200)."""
    Lq, Lk = 150, 200
    q, k, _ = _inputs(Lq, Lk, 3, seed=77)
    for i in (40, 100, 149):
        r0 = FM.score_check_row(q, k, i, Lq, True)
        n = r0["n"]
        col = 3 if site == "S" else 1
        tile = 0 if site == "S" else 1
        f = FM.FaultSpec(site, i, col, tile, bit)
        pr = FM.score_check_fault(q, k, i, Lq, True, f)
        qi = [float(x) for x in q[i]]
        lhs = 0.0
        for kk in range(n):
            if site == "Q" and kk == 64 * tile:
                qi[col] = bf16_flip(qi[col], bit)
            sc = sum(qi[j] * float(k[kk][j]) for j in range(3))
            if site == "S" and kk == col:
                sc = f32_flip(f32(sc), bit)
            lhs += sc
        if site == "Q" and n <= 64 * tile:
            qi[col] = bf16_flip(qi[col], bit)
        rhs = sum(qi[j] * sum(float(k[kk][j]) for kk in range(n)) for j in range(3))
        ms = sum(abs(qi[j]) * sum(abs(float(k[kk][j])) for kk in range(n)) for j in range(3))
        assert math.isclose(pr["lhs"], lhs, rel_tol=1e-12, abs_tol=1e-9 * (ms + 1))
        assert math.isclose(pr["rhs"], rhs, rel_tol=1e-12, abs_tol=1e-9 * (ms + 1))
        assert math.isclose(pr["ms"], ms, rel_tol=1e-12)
        assert pr["nonfinite"] == (not math.isfinite(lhs - rhs) or not math.isfinite(ms))
        if not pr["nonfinite"]:
            assert pr["row_flag"] == (abs(lhs - rhs) > 2.0 ** -22 * ms)
            assert not pr["dup_flag"] and pr["flag"] == pr["row_flag"]


@pytest.mark.parametrize("bit", [0, 5, 12, 20, 23, 24, 27, 29, 30, 31])
def test_masked_tile_duplicate_check_brute_force(bit):
    """An S flip on a key past the full tiles (the diagonal tile here): the
    row check does not see it, the duplicate product does. Brute force: the
    tile's visible scores summed in fp32 with the flipped value against the
    same sum without it (in two lane halves, as the kernel adds them); the
    prediction, where it is not left open, must match (causal 150 x 150)."""
    Lq = Lk = 150
    q, k, _ = _inputs(Lq, Lk, 3, seed=91)
    for i in (70, 100, 149):
        r0 = FM.score_check_row(q, k, i, Lq, True)
        t0 = (i // 64) * 64
        assert r0["n"] <= t0
        for col in sorted({t0, (t0 + i) // 2, i}):
            pr = FM.score_check_fault(q, k, i, Lq, True, FM.FaultSpec("S", i, col, 0, bit))
            assert pr["lhs"] == r0["lhs"] and pr["rhs"] == r0["rhs"] and not pr["row_flag"]
            def tile_sum(flip):
                halves = [np.float32(0.0), np.float32(0.0)]
                for kk in range(t0, i + 1):
                    sc = f32(sum(float(q[i][j]) * float(k[kk][j]) for j in range(3)))
                    if flip and kk == col:
                        sc = f32_flip(sc, bit)
                    h = ((kk - t0) >> 3) & 1
                    with np.errstate(over="ignore", invalid="ignore"):
                        halves[h] = np.float32(halves[h] + np.float32(sc))
                with np.errstate(over="ignore", invalid="ignore"):
                    return np.float32(halves[0] + halves[1])
            a, b = tile_sum(True), tile_sum(False)
            differ = a.tobytes() != b.tobytes()
            if not pr["dup_undetermined"]:
                assert pr["dup_flag"] == differ, (i, col, bit, a, b)
                assert pr["flag"] == pr["dup_flag"]
