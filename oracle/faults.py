"""Predicted effect of one bit flip on the Flash-ABFT forward (arXiv 2507.16676).

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports this module;
only the tests do. It shares no code with the HIP kernels or their host
library.

Section III of the paper argues that one checksum per query row (Eq. 8)
catches an error anywhere in the attention, because the predicted row sum
c/l and the actual row sum of O are built along separate paths from the
same softmax weights; Section IV-B measures this by flipping bits. This
module states, in closed form and in fp64, what a flip at each fault site
of the kernel does to the output row O_i, to pred_i = c_i / l_i and to
actual_i = sum_j O_ij, so that every injected run on the GPU can be checked
against an independent prediction instead of only against a fault-free run
of the same kernel.

With P_ik = exp(s_ik - m_i) / l_i the normalised softmax weights (Eq. 2) and
vs_k = sumrow_k(V) (Eq. 4), a flip that multiplies a stored value x by
f = x'/x gives:

  P  (weight p~_ik after the checksum read it):
       dO_ij = (f - 1) P_ik V_kj,   dpred_i = 0,  dactual_i = (f - 1) P_ik vs_k
  O  (accumulator o_ij after the P V product of key tile t):
       dO_ij = (f - 1) sum_{k <= end of tile t} P_ik V_kj,  dpred_i = 0
  V  (V_kj in one workgroup's copy, after its sumrow was taken; V' = V + dV):
       dO_ij = P_ik dV for every row i of that workgroup that sees key k
  C  (one part of the checksum accumulator c_i = c_hi + c_lo after tile t,
     as held for the row's first key half):
       dO = 0,  dpred_i = (f - 1) sum_{k <= end of tile t, k in H} P_ik part_k
  VS (one part of the sumrow record of key k in one workgroup):
       dO = 0,  dpred_i = P_ik (part'_k - part_k) for its rows that see k
  L  (the accumulator l_i after tile t, first key half): O and pred are both
       divided by 1 + (f - 1) F_t with F_t = sum_{k <= end of tile t, k in H} P_ik
  S  (the raw score q_i . k_k), Q (q_ij from key tile t on): the scores
       change upstream of the checksum tap; O follows the plain definition
       with the changed scores and pred moves with it (resid stays 0).

The factor f needs the stored value x, which the closed forms do not give:
x is the kernel's own state. The fault model fixes it (the same description
the library's header gives for each site):
  * scores in exp2 units u_k = s_k * sl2 with sl2 = scale * log2(e) in fp32;
  * keys come in tiles of `key_tile`; after the max of tile t the exponent
    reference moves to the tile max (rounded to fp32) only when it exceeds
    the reference by more than 8 (lazy rescaling), and the weights of tile t
    are p~_k = bf16(2^(u_k - ref_t)) (round to nearest even);
  * after tile t, o, l and c sit in the frame of ref_t:
    o_j(t) = sum_{k <= end of t} p~_k 2^(ref_{t(k)} - ref_t) V_kj, and l, c
    alike with 1 and the sumrow parts;
  * the sumrow record of key k is vs_k in fp32 split into bf16 hi = bf16(vs)
    and lo = bf16(vs - hi);
  * c and l of a row are held as two partial sums, one per key half: H, the
    keys k with k mod 16 < 8, and the rest (one register each, added at the
    end); the C and L sites flip the register of H;
  * a wave of 32 query rows computes every key tile up to the diagonal of
    its last row (causal), so a non-finite V_kj or sumrow part also reaches
    the rows of that wave that give key k the weight 0 (0 * inf is NaN).
The model is evaluated in fp64; the kernel's fp32 sums and hardware exp2
can differ from it only where a value sits within rounding of an exponent
boundary.

Readings: fp32 overflow of the output accumulator, of the weight times V,
or of sum_j |O_ij| makes the row non-finite (the kernel flags it);
a flipped l that is not positive (or not finite) gives O = 0 and pred = 0
(the kernel divides only by a positive l). The running-max site M is not
modelled here (it changes which weights underflow, not the checksum).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = ["FaultSpec", "LAZY", "SIG_REL", "bf16_round_bits", "bf16_bits_value",
           "flip_bf16", "flip_f32", "exp2_scale", "row_frame", "fault_effect",
           "score_check_row", "score_check_fault", "classify_prediction"]

LAZY = 8.0                 # reference moves when a tile max exceeds it by more than this
SIG_REL = 2.0 ** -8        # significance of an output change (campaign classification)
F32_MAX = float(np.finfo(np.float32).max)


@dataclasses.dataclass(frozen=True)
class FaultSpec:
    """One single-bit fault of one head, in the library's site vocabulary:
    site in S, P, O, V, C, L, Q, VS; row, col, tile, bit as documented for
    the library's fault descriptor (row = query for S, P, O, C, L, Q; row =
    key for V, VS; tile = key tile for O, C, L, Q and query tile for V, VS)."""
    site: str
    row: int
    col: int = 0
    tile: int = 0
    bit: int = 0


# --------------------------------------------------------------------------
# storage formats
# --------------------------------------------------------------------------

def bf16_round_bits(x) -> np.ndarray:
    """fp64/fp32 values -> bf16 bit patterns, via fp32 (round to nearest,
    ties to even; the fp32 step is exact for every value used here, which
    are already fp32 or are rounded to fp32 first)."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    keep = u >> 16
    rest = u & 0xFFFF
    up = (rest > 0x8000) | ((rest == 0x8000) & ((keep & 1) == 1))
    out = (keep + up.astype(np.uint64)) & 0xFFFF
    out = np.where(np.isnan(f), (keep | 0x40) & 0xFFFF, out)
    return out.astype(np.uint16)


def bf16_bits_value(b) -> np.ndarray:
    """bf16 bit patterns -> exact fp64 values (inf and NaN included)."""
    b = np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16
    with np.errstate(invalid="ignore"):
        return b.view(np.float32).astype(np.float64)


def flip_bf16(x: float, bit: int) -> float:
    """The bf16 value x (exactly representable) with bit `bit` flipped."""
    b = int(bf16_round_bits(np.float32(x)))
    assert float(bf16_bits_value(np.uint16(b))) == x or math.isnan(x), "x is not a bf16 value"
    return float(bf16_bits_value(np.uint16(b ^ (1 << bit))))


def flip_f32(x: float, bit: int) -> float:
    """The value x rounded to fp32, with bit `bit` of its pattern flipped."""
    u = np.array([x], dtype=np.float32).view(np.uint32)
    u ^= np.uint32(1 << bit)
    return float(u.view(np.float32)[0])


def exp2_scale(scale: float) -> float:
    """sl2 = scale * log2(e) as the kernel holds it: an fp32 product of the
    fp32 scale and fp32 log2(e), raised to 2^-126 if smaller."""
    s = np.float32(scale) * np.float32(1.4426950408889634)
    return float(max(np.float32(s), np.float32(2.0 ** -126)))


# --------------------------------------------------------------------------
# plain definition pieces (Eq. 1, 2, 4) for one row
# --------------------------------------------------------------------------

def _visible(i: int, Lq: int, Lk: int, causal: bool) -> np.ndarray:
    keys = np.arange(Lk)
    if not causal:
        return np.ones(Lk, dtype=bool)
    return keys <= i + (Lk - Lq)


def _softmax_row(s: np.ndarray, vis: np.ndarray, scale: float):
    """P_i (normalised weights, 0 where masked) from raw scores s (no
    scale): the plain definition of Eq. 2 with the max shift."""
    x = np.where(vis, scale * s, -np.inf)
    if not vis.any():
        return np.zeros_like(x)
    m = x.max()
    if not np.isfinite(m):
        return np.full_like(x, np.nan)
    e = np.where(vis, np.exp(x - m), 0.0)
    return e / e.sum()


# --------------------------------------------------------------------------
# the kernel state of one query row (the fault model's site values)
# --------------------------------------------------------------------------

def row_frame(s: np.ndarray, vis: np.ndarray, sl2: float, v: np.ndarray,
              hi: np.ndarray, lo: np.ndarray, key_tile: int) -> dict:
    """Site values of one row: per key tile t the exponent reference ref[t]
    (exp2 units, after tile t's max), the bf16 weights ptil[k], and the
    accumulators o(t) [d], l(t), c_hi(t), c_lo(t) in the frame of ref[t].
    s: raw scores (fp64), vis: visible keys, v: V [Lk, d], hi/lo: the
    sumrow parts [Lk]."""
    Lk, d = v.shape
    u = s * sl2
    nt = (Lk + key_tile - 1) // key_tile
    ref = -np.inf
    refs = np.full(nt, -np.inf)
    ptil = np.zeros(Lk)
    o = np.zeros((nt, d))
    l = np.zeros(nt)
    chi = np.zeros(nt)
    clo = np.zeros(nt)
    # the same sums over the first key half (keys k with k mod 16 < 8), the
    # part one lane of the row holds
    h0 = (np.arange(Lk) % 16) < 8
    l0 = np.zeros(nt)
    chi0 = np.zeros(nt)
    clo0 = np.zeros(nt)
    run_o, run_l, run_hi, run_lo = np.zeros(d), 0.0, 0.0, 0.0
    run_l0, run_hi0, run_lo0 = 0.0, 0.0, 0.0
    for t in range(nt):
        a, b = t * key_tile, min(Lk, (t + 1) * key_tile)
        vt = vis[a:b]
        # the tile max enters the reference as an fp32 product
        mt = float(np.float32(u[a:b][vt].max())) if vt.any() else -np.inf
        new = mt if mt > ref + LAZY else ref
        if np.isfinite(ref) and new != ref:
            alpha = 2.0 ** (ref - new)
            run_o, run_l = run_o * alpha, run_l * alpha
            run_hi, run_lo = run_hi * alpha, run_lo * alpha
            run_l0, run_hi0, run_lo0 = run_l0 * alpha, run_hi0 * alpha, run_lo0 * alpha
        ref = new
        refs[t] = ref
        if vt.any():
            w = np.zeros(b - a)
            w[vt] = bf16_bits_value(bf16_round_bits(2.0 ** (u[a:b][vt] - ref)))
            ptil[a:b] = w
            run_o = run_o + w @ v[a:b]
            run_l = run_l + w.sum()
            run_hi = run_hi + w @ hi[a:b]
            run_lo = run_lo + w @ lo[a:b]
            w0 = np.where(h0[a:b], w, 0.0)
            run_l0 = run_l0 + w0.sum()
            run_hi0 = run_hi0 + w0 @ hi[a:b]
            run_lo0 = run_lo0 + w0 @ lo[a:b]
        o[t], l[t], chi[t], clo[t] = run_o, run_l, run_hi, run_lo
        l0[t], chi0[t], clo0[t] = run_l0, run_hi0, run_lo0
    return {"ref": refs, "ptil": ptil, "o": o, "l": l, "c_hi": chi, "c_lo": clo,
            "l_half": l0, "c_hi_half": chi0, "c_lo_half": clo0}


def _sumrow_parts(v: np.ndarray):
    """vs_k in fp32 and its bf16 hi / lo parts (the sumrow record)."""
    vs32 = v.sum(axis=1).astype(np.float32)
    hi = bf16_bits_value(bf16_round_bits(vs32))
    lo = bf16_bits_value(bf16_round_bits(vs32.astype(np.float64) - hi))
    return vs32.astype(np.float64), hi, lo


def _tile_end(t: int, key_tile: int, Lk: int) -> int:
    return min(Lk, (t + 1) * key_tile)


def _wave_sees_tile(i: int, t: int, Lq: int, Lk: int, causal: bool, key_tile: int) -> bool:
    """Does the 32-row wave holding query row i compute key tile t?"""
    w0 = 32 * (i // 32)
    if w0 >= Lq:
        return False
    return (not causal) or t * key_tile <= w0 + 31 + (Lk - Lq)


# --------------------------------------------------------------------------
# prediction
# --------------------------------------------------------------------------

def _row_result(O, pred, dO, dpred, tau_rel, tau_abs, nonfinite=False, nonfinite_maybe=False,
                O_new=None, pred_new=None, err_o=None, err_p=0.0, undetermined=False):
    """Residual, threshold and flag of one row after a fault. err_o [d] and
    err_p bound what the bf16 rounding of the kernel's weights can move dO
    and dpred by, in units of 2^-8 (each weight and l carry a relative
    rounding of at most 2^-9): sum_k P_ik |x_k| over the terms a change
    consists of, times |f - 1| where a factor applies."""
    O_new = O + dO if O_new is None else O_new
    pred_new = pred + dpred if pred_new is None else pred_new
    with np.errstate(invalid="ignore", over="ignore"):
        actual = float(np.sum(O))
        actual_new = float(np.sum(O_new))
        absum = float(np.abs(O_new).sum())
        r = pred_new - actual_new
        M = absum + abs(pred_new)
        nonfinite = bool(nonfinite or not np.all(np.isfinite(O_new)) or not np.isfinite(r)
                         or absum > F32_MAX)
        flag = bool(nonfinite or not (abs(r) <= tau_rel * M + tau_abs))
        ref = float(np.abs(O).max()) if O.size else 0.0
        sig = bool(nonfinite or np.any(np.abs(O_new - O) > SIG_REL * ref)
                   or np.any(np.abs(O_new) > bf16_max()))
    err_o = np.zeros_like(O) if err_o is None else np.asarray(err_o, dtype=np.float64)
    return {"O": O, "O_new": O_new, "dO": O_new - O, "pred": pred, "pred_new": pred_new,
            "dpred": pred_new - pred, "actual": actual, "actual_new": actual_new,
            "dactual": actual_new - actual, "resid": r, "M": M, "flag": flag,
            "nonfinite": nonfinite, "nonfinite_maybe": bool(nonfinite_maybe),
            "significant": sig, "dO_err": err_o, "dpred_err": float(err_p),
            "dactual_err": float(err_o.sum()), "undetermined": bool(undetermined)}


def bf16_max() -> float:
    return float(bf16_bits_value(np.uint16(0x7F7F)))


def fault_effect(q, k, v, causal: bool, scale: float, fault: FaultSpec, key_tile: int = 64,
                 query_tile: int = 256, tau_rel: float = 2.0 ** -16,
                 tau_abs: float = 0.0) -> dict:
    """Predicted effect of `fault` on one head (q [Lq, d], k, v [Lk, d], the
    bf16 input values in any float dtype). Returns {"rows": [i, ...],
    "per_row": [dict per row], "flagged": any row flagged, "significant":
    any row significant}; each row dict holds O (fault-free, fp64), dO,
    pred, dpred, actual, dactual, the new residual r, M = sum_j |O'_ij| +
    |pred'_i|, flag, nonfinite, nonfinite_maybe (0 * inf) and significant."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    Lq, Lk = q.shape[0], k.shape[0]
    sl2 = exp2_scale(scale)
    site = fault.site
    vs, hi, lo = _sumrow_parts(v)
    half0 = (np.arange(Lk) % 16) < 8   # keys of the row's first key half

    def base(i):
        vis = _visible(i, Lq, Lk, causal)
        s = k @ q[i]
        P = _softmax_row(s, vis, scale)
        return vis, s, P, P @ v, float(P @ vs)

    if site in ("P", "O", "C", "L", "S", "Q"):
        i = fault.row
        vis, s, P, O, pred = base(i)
        if site == "P":
            fr = row_frame(s, vis, sl2, v, hi, lo, key_tile)
            kk = fault.col
            x = fr["ptil"][kk]
            xn = flip_bf16(x, fault.bit)
            if not np.isfinite(xn):
                res = _row_result(O, pred, np.full_like(O, np.nan), 0.0, tau_rel, tau_abs,
                                  nonfinite=True)
            else:
                t = kk // key_tile
                if x != 0.0:
                    dO = (xn / x - 1.0) * P[kk] * v[kk]
                else:   # a weight that underflowed to 0: the new weight, in the final frame
                    dO = xn * 2.0 ** (fr["ref"][t] - fr["ref"][-1]) * v[kk] / fr["l"][-1]
                # the kernel adds p~' V_k to o(t) in the frame of ref_t (fp32)
                over = bool(np.any(np.abs(xn * v[kk]) > F32_MAX)
                            or np.any(np.abs(fr["o"][t] + (xn - x) * v[kk]) > F32_MAX))
                res = _row_result(O, pred, dO, 0.0, tau_rel, tau_abs, nonfinite=over,
                                  err_o=np.abs(dO))
        elif site == "O":
            fr = row_frame(s, vis, sl2, v, hi, lo, key_tile)
            t, j = fault.tile, fault.col
            x = fr["o"][t][j]
            xn = flip_f32(x, fault.bit)
            x32 = float(np.float32(x))
            if not np.isfinite(xn):
                dO = np.zeros_like(O)
                dO[j] = np.nan
                res = _row_result(O, pred, dO, 0.0, tau_rel, tau_abs, nonfinite=True)
            else:
                dO = np.zeros_like(O)
                part = P[:_tile_end(t, key_tile, Lk)] @ v[:_tile_end(t, key_tile, Lk), j]
                e = _tile_end(t, key_tile, Lk)
                err = np.zeros_like(O)
                if x32 != 0.0:
                    dO[j] = (xn / x32 - 1.0) * part
                    err[j] = abs(xn / x32 - 1.0) * (P[:e] @ np.abs(v[:e, j]))
                else:   # an exact zero: the flipped value itself, moved to the final frame
                    dO[j] = xn * 2.0 ** (fr["ref"][t] - fr["ref"][-1]) / fr["l"][-1]
                    err[j] = abs(dO[j])
                res = _row_result(O, pred, dO, 0.0, tau_rel, tau_abs, err_o=err)
        elif site == "C":
            fr = row_frame(s, vis, sl2, v, hi, lo, key_tile)
            t = fault.tile
            key = "c_hi_half" if fault.col == 0 else "c_lo_half"
            # the flipped register holds the first key half only
            parts = np.where(half0, hi if fault.col == 0 else lo, 0.0)
            x = float(np.float32(fr[key][t]))
            xn = flip_f32(x, fault.bit)
            if not np.isfinite(xn):
                res = _row_result(O, pred, np.zeros_like(O), np.nan, tau_rel, tau_abs,
                                  nonfinite=True)
            else:
                e = _tile_end(t, key_tile, Lk)
                part = float(P[:e] @ parts[:e])
                if x != 0.0:
                    dpred = (xn / x - 1.0) * part
                    err = abs(xn / x - 1.0) * float(P[:e] @ np.abs(parts[:e]))
                else:
                    dpred = xn * 2.0 ** (fr["ref"][t] - fr["ref"][-1]) / fr["l"][-1]
                    err = abs(dpred)
                res = _row_result(O, pred, np.zeros_like(O), dpred, tau_rel, tau_abs,
                                  err_p=err)
        elif site == "L":
            fr = row_frame(s, vis, sl2, v, hi, lo, key_tile)
            t = fault.tile
            x = float(np.float32(fr["l_half"][t]))
            xn = flip_f32(x, fault.bit)
            e = _tile_end(t, key_tile, Lk)
            # l' / l = (weight outside the flipped sum) + f (weight in it),
            # summed apart so that nothing cancels when f is tiny
            inside = np.zeros(Lk, dtype=bool)
            inside[:e] = True
            inside &= half0
            den = (float(P[~inside].sum()) + (xn / x) * float(P[inside].sum())
                   if np.isfinite(xn) else np.inf)
            if not (den > 0.0) or not np.isfinite(den):
                # l' not positive or not finite: the kernel writes O = 0, pred = 0
                # (the change is -O: the rounding of O's own weights bounds it)
                res = _row_result(O, pred, None, None, tau_rel, tau_abs,
                                  O_new=np.zeros_like(O), pred_new=0.0,
                                  err_o=P @ np.abs(v), err_p=float(P @ np.abs(vs)))
            else:
                # O' = O / den: the rounding of every weight enters, scaled
                res = _row_result(O, pred, None, None, tau_rel, tau_abs, O_new=O / den,
                                  pred_new=pred / den,
                                  err_o=(P @ np.abs(v)) * (1.0 + 1.0 / den),
                                  err_p=float(P @ np.abs(vs)) * (1.0 + 1.0 / den))
        else:   # S, Q: the scores change upstream of the checksum tap
            s_new = s.copy()
            if site == "S":
                s_new[fault.col] = flip_f32(s[fault.col], fault.bit)
            else:
                qn = flip_bf16(q[i, fault.col], fault.bit)
                a = fault.tile * key_tile
                s_new[a:] = s[a:] + (qn - q[i, fault.col]) * k[a:, fault.col]
            bad = s_new[vis]
            if np.any(np.isnan(bad)) or np.any(bad == np.inf):
                res = _row_result(O, pred, np.full_like(O, np.nan), np.nan, tau_rel, tau_abs,
                                  nonfinite=True)
            else:
                Pn = _softmax_row(s_new, vis, scale)
                # a new row max beyond 2^30 in exp2 units: the kernel's weight
                # of that key is 2 to the fp32 rounding residual of its score
                # times sl2 (up to 2^6 and more), which depends on score bits
                # below fp64's view of them; the outcome is not determined here
                und = bool(np.max(s_new[vis]) * sl2 >= 2.0 ** 30)
                # every weight changes: both rows' rounding enters
                res = _row_result(O, pred, None, None, tau_rel, tau_abs, O_new=Pn @ v,
                                  pred_new=float(Pn @ vs), err_o=(P + Pn) @ np.abs(v),
                                  err_p=float((P + Pn) @ np.abs(vs)), undetermined=und)
        return _summary([i], [res])

    if site in ("V", "VS"):
        kk = fault.row
        t = kk // key_tile
        r0 = fault.tile * query_tile
        rows = [i for i in range(r0, min(Lq, r0 + query_tile))
                if _wave_sees_tile(i, t, Lq, Lk, causal, key_tile)]
        if site == "V":
            x = v[kk, fault.col]
            xn = flip_bf16(x, fault.bit)
        else:
            x = (hi if fault.col == 0 else lo)[kk]
            xn = flip_bf16(x, fault.bit)
        out = []
        for i in rows:
            vis, s, P, O, pred = base(i)
            if not np.isfinite(xn):
                # 0 * inf: rows of the wave that give key k no weight may turn
                # non-finite too; rows that weight it certainly do
                certain = bool(vis[kk] and P[kk] > 0.0)
                if site == "V":
                    dO = np.zeros_like(O)
                    if certain:
                        dO[fault.col] = np.nan
                    res = _row_result(O, pred, dO, 0.0, tau_rel, tau_abs, nonfinite=certain,
                                      nonfinite_maybe=not certain)
                else:
                    res = _row_result(O, pred, np.zeros_like(O), np.nan if certain else 0.0,
                                      tau_rel, tau_abs, nonfinite=certain,
                                      nonfinite_maybe=not certain)
            elif site == "V":
                dO = np.zeros_like(O)
                dO[fault.col] = P[kk] * (xn - x)
                res = _row_result(O, pred, dO, 0.0, tau_rel, tau_abs, err_o=np.abs(dO))
            else:
                dp = float(P[kk] * (xn - x))
                res = _row_result(O, pred, np.zeros_like(O), dp, tau_rel, tau_abs,
                                  err_p=abs(dp))
            out.append(res)
        return _summary(rows, out)
    raise ValueError(f"site {site!r} is not modelled")


def _summary(rows, res):
    return {"rows": list(rows), "per_row": res,
            "undetermined": any(r["undetermined"] for r in res),
            "flagged": any(r["flag"] for r in res),
            "significant": any(r["significant"] for r in res),
            "nonfinite": any(r["nonfinite"] for r in res),
            "nonfinite_maybe": any(r["nonfinite_maybe"] for r in res)}


def classify_prediction(pred: dict) -> str:
    """The campaign's outcome classes for a predicted run: detected (flagged,
    significant), false_positive_or_minor (flagged, not significant), silent
    (not flagged, significant), benign."""
    fl, sig = pred["flagged"], pred["significant"]
    if fl and sig:
        return "detected"
    if fl:
        return "flagged_not_significant"
    return "silent" if sig else "benign"


# --------------------------------------------------------------------------
# the score check (an extension: Section II's row checksum of a matrix
# product applied to S = Q K^T)
# --------------------------------------------------------------------------

def score_check_row(q, k, i: int, Lq: int, causal: bool, key_tile: int = 64) -> dict:
    """For query row i, over the key tiles that need no mask for the whole
    32-row wave holding i (tiles t < min(Lk // key_tile, (w0 + off + 1) //
    key_tile) with w0 the wave's first row and off = Lk - Lq; all
    Lk // key_tile tiles when not causal): lhs = sum_k q_i . k_k (raw
    scores), rhs = q_i . sum_k k_k, and the bound ms = |q_i| . sum_k |k_k|.
    Returns fp64 lhs, rhs, ms and the number of keys n."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    Lk = k.shape[0]
    tw = Lk // key_tile
    if causal:
        lim = 32 * (i // 32) + (Lk - Lq) + 1
        tw = min(tw, lim // key_tile if lim > 0 else 0)
    n = tw * key_tile
    ks = k[:n]
    return {"lhs": float((ks @ q[i]).sum()), "rhs": float(q[i] @ ks.sum(axis=0)),
            "ms": float(np.abs(q[i]) @ np.abs(ks).sum(axis=0)), "n": n}


def score_check_fault(q, k, i: int, Lq: int, causal: bool, fault: FaultSpec,
                      key_tile: int = 64, tau_s: float = 2.0 ** -22, tau_abs: float = 0.0) -> dict:
    """The score check of row i after an S or Q fault (other sites leave it
    as score_check_row gives it). S (row i, key k): the flipped fp32 score
    enters lhs if k lies in the full tiles; the right-hand side is unchanged.
    Q (row i, column j, from key tile t on): the scores of tiles >= t use the
    flipped q_ij, and rhs and the bound use it for every full tile (the q
    the row holds at the end). Returns lhs, rhs, ms, n, row_flag (|lhs - rhs|
    > tau_s * ms + tau_abs with finite sums), nonfinite (the sums are not
    finite: the row counts as non-finite instead), term (the magnitude of
    the changed terms, sum of |x_j y_j| scaled by the flip, which bounds what
    fp32 rounding of the kernel's scores can move) and undetermined (a sum
    beyond 2^100: fp32 overflow inside the kernel's sums decides the
    outcome).

    The keys past the full tiles that row i sees lie in masked tiles (the
    diagonal one, a ragged last one), which have no per-row prefix of the K
    sums; there the kernel sums the row's visible scores of each such tile
    twice, from the product as stored and from a second product of the same
    operands, and flags any difference. An S flip on such a key changes the
    first sum by dsum = s' - s (a Q flip changes both products alike): the
    two fp32 sums differ for certain when |dsum| exceeds their rounding
    (2^-17 of A, the tile's sum of |s_ik| over the row's visible keys plus
    |s'|), never when dsum = 0, and the outcome is left undetermined in
    between; a non-finite s' always differs. Returned as dup_flag and
    dup_undetermined; flag = row_flag or dup_flag."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    r = score_check_row(q, k, i, Lq, causal, key_tile)
    n = r["n"]
    lhs, rhs, ms = r["lhs"], r["rhs"], r["ms"]
    term = 0.0   # scale of the changed terms: the kernel's fp32 score carries
    # a rounding of order 2^-24 of sum_j |q_ij k_kj|, which a flip scales by f
    if fault.row == i and fault.site == "S" and fault.col < n:
        s = float(k[fault.col] @ q[i])
        sn = flip_f32(s, fault.bit)
        lhs = lhs + sn - float(np.float32(s))
        s32 = float(np.float32(s))
        f = abs(sn / s32) if s32 != 0.0 else abs(sn)
        term = f * float(np.abs(k[fault.col]) @ np.abs(q[i]))
    elif fault.row == i and fault.site == "Q":
        j = fault.col
        qn = q[i].copy()
        qn[j] = flip_bf16(q[i, j], fault.bit)
        a = min(n, fault.tile * key_tile)
        ks = k[:n]
        with np.errstate(invalid="ignore", over="ignore"):
            lhs = float((ks[:a] @ q[i]).sum() + (ks[a:] @ qn).sum())
            rhs = float(qn @ ks.sum(axis=0))
            ms = float(np.abs(qn) @ np.abs(ks).sum(axis=0))
            term = float(abs(qn[j] - q[i, j]) * np.abs(ks[:, j]).sum())
    dup_flag = dup_und = False
    Lk = k.shape[0]
    last = min(Lk - 1, i + Lk - Lq) if causal else Lk - 1
    if fault.row == i and fault.site == "S" and n <= fault.col <= last:
        s = float(k[fault.col] @ q[i])
        s32 = float(np.float32(s))
        sn = flip_f32(s, fault.bit)
        t0 = (fault.col // key_tile) * key_tile
        keys = np.arange(t0, min(t0 + key_tile, last + 1))
        a_sum = float(np.abs(k[keys] @ q[i]).sum())
        if not np.isfinite(sn):
            dup_flag = True
        else:
            dsum = sn - s32
            a_sum += abs(sn)
            if dsum == 0.0:
                dup_flag = False
            elif abs(dsum) > 2.0 ** -17 * a_sum:
                dup_flag = True
            else:
                dup_und = True
    with np.errstate(invalid="ignore"):
        d = lhs - rhs
        nonfinite = bool(not np.isfinite(d) or not np.isfinite(ms))
        row_flag = bool(not nonfinite and abs(d) > tau_s * ms + tau_abs)
        # sums near the fp32 range: whether the kernel's fp32 products and
        # sums overflow (and in which order) decides the outcome
        und = bool(not nonfinite and max(abs(lhs), abs(rhs), ms, term) > 2.0 ** 100)
    return {"lhs": lhs, "rhs": rhs, "ms": ms, "n": n, "row_flag": row_flag,
            "dup_flag": dup_flag, "dup_undetermined": dup_und, "flag": row_flag or dup_flag,
            "nonfinite": nonfinite, "term": term, "undetermined": und}
