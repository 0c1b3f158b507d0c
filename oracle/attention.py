"""fp64 CPU oracle for Flash-ABFT attention (arXiv 2507.16676).

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports this module;
only the tests, the smoke check and the benchmark's CPU-baseline leg do. It
shares no code with the HIP kernels or their host library.

What it computes, per head and per query row i (Section III-A):

  s_ik   = scale * q_i . k_k                      (Eq. 1, Eq. 2; scaling as
                                                   described in Section II)
  m_i    = max_k s_ik over visible keys            (the max shift that Eq. 2
                                                   omits for simplicity)
  p_ik   = exp(s_ik - m_i),  l_i = sum_k p_ik
  O_ij   = sum_k p_ik V_kj / l_i                   (Eq. 1)
  vs_k   = sum_j V_kj                              (Eq. 4, sumrow_k(V), the
                                                   sum running over the d
                                                   entries of a row of V)
  pred_i = sum_k p_ik vs_k / l_i                   (Eq. 8, check(q_i); built
                                                   without reading O)
  actual_i = sum_j O_ij,  resid_i = pred_i - actual_i

and, as an extension beyond the paper (a classic weighted ABFT checksum
next to the paper's plain one), for weights w_j (default (-1)^j):

  pred_w_i = sum_k p_ik (sum_j w_j V_kj) / l_i,   actual_w_i = sum_j w_j O_ij

plus the global check of Eq. 5 from the explicit column sums of the
normalised score matrix (Eq. 3), and fp64 restatements of Algorithm 1
(attention with lazy softmax division, two passes over the keys) and
Algorithm 3 (FlashAttention-2 with the online checksum, one pass, keys
consumed in blocks of any size).

Readings where the paper is silent or garbled:
  * Scale is an argument (Eq. 1 prints none; the text says the scores are
    scaled).
  * sumrow sums over the d columns of V (Eq. 4 prints N as the bound).
  * Lq queries and Lk keys need not be equal (the paper assumes N x N).
  * Causal masking keeps key k for query i iff k <= i + (Lk - Lq); masked
    pairs take no part in m, l, o or c. A query with no visible key gets
    O = 0, pred = actual = resid = 0.
  * Initial state of the one-pass recurrence: m = -inf, l = o = c = 0; the
    rescale factor is taken as 0 while the running max is still -inf.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "visible_mask", "sumrow", "attention_head", "attention",
    "global_check", "lazy_softmax_attention", "online_checksum_attention",
    "threshold_flags", "alternating_weights", "weighted_check_head",
]


def visible_mask(Lq: int, Lk: int, causal: bool, rows=None) -> np.ndarray:
    """Boolean [n_rows, Lk]: True where query row i may attend to key k."""
    rows = np.arange(Lq) if rows is None else np.asarray(rows)
    if not causal:
        return np.ones((rows.size, Lk), dtype=bool)
    keys = np.arange(Lk)
    return keys[None, :] <= (rows[:, None] + (Lk - Lq))


def sumrow(v: np.ndarray) -> np.ndarray:
    """sumrow_k(V) = sum over the d entries of row k of V (Eq. 4)."""
    return np.asarray(v, dtype=np.float64).sum(axis=-1)


def attention_head(q, k, v, causal: bool, scale: float, rows=None) -> dict:
    """Plain-definition attention and per-row checksum for one head.

    q: [Lq, d], k and v: [Lk, d] (any float dtype; computed in fp64).
    rows: optional query-row indices (default all rows).
    Returns fp64 arrays O [n, d], pred, actual, resid, l, m [n].
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    Lq, Lk = q.shape[0], k.shape[0]
    rows = np.arange(Lq) if rows is None else np.asarray(rows)
    s = scale * (q[rows] @ k.T)                       # Eq. 2, s_ik
    vis = visible_mask(Lq, Lk, causal, rows)
    s = np.where(vis, s, -np.inf)
    any_vis = vis.any(axis=1)
    m = np.where(any_vis, s.max(axis=1), -np.inf)
    m_safe = np.where(any_vis, m, 0.0)
    p = np.where(vis, np.exp(s - m_safe[:, None]), 0.0)
    l = p.sum(axis=1)
    l_safe = np.where(any_vis, l, 1.0)
    O = (p @ v) / l_safe[:, None]                     # Eq. 1
    vs = sumrow(v)                                    # Eq. 4
    pred = (p @ vs) / l_safe                          # Eq. 8 (no use of O)
    actual = O.sum(axis=1)
    return {"O": O, "pred": pred, "actual": actual, "resid": pred - actual,
            "l": l, "m": m}


def alternating_weights(d: int) -> np.ndarray:
    """w_j = (-1)^j, j = 0 .. d-1."""
    return np.where(np.arange(d) % 2 == 0, 1.0, -1.0)


def weighted_check_head(q, k, v, causal: bool, scale: float, w=None, rows=None) -> dict:
    """Weighted checksum of one head (not in the paper): the plain definition
    of pred_w = sum_k p_ik (sum_j w_j V_kj) / l_i, built without reading O,
    and of actual_w = sum_j w_j O_ij. w defaults to (-1)^j; w = 1 gives the
    paper's check (Eq. 8). Returns fp64 arrays pred_w, actual_w, resid_w.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    d = v.shape[1]
    w = alternating_weights(d) if w is None else np.asarray(w, dtype=np.float64)
    Lq, Lk = q.shape[0], k.shape[0]
    rows = np.arange(Lq) if rows is None else np.asarray(rows)
    s = scale * (q[rows] @ k.T)
    vis = visible_mask(Lq, Lk, causal, rows)
    s = np.where(vis, s, -np.inf)
    any_vis = vis.any(axis=1)
    m = np.where(any_vis, s.max(axis=1), 0.0)
    p = np.where(vis, np.exp(s - m[:, None]), 0.0)
    l_safe = np.where(any_vis, p.sum(axis=1), 1.0)
    vw = v @ w                                        # weighted row sums of V
    pred_w = (p @ vw) / l_safe
    O = (p @ v) / l_safe[:, None]
    actual_w = O @ w
    return {"pred_w": pred_w, "actual_w": actual_w, "resid_w": pred_w - actual_w}


def attention(q, k, v, causal: bool, scale: float, rows=None,
              row_chunk: int = 1024) -> dict:
    """Batched form over [B, H, L, d] inputs (fp32 or fp64 arrays).

    rows: optional query-row indices shared by every head; results are then
    [B, H, len(rows), ...]. Rows are processed in chunks of ``row_chunk`` to
    bound memory; chunking does not change any result (rows are independent).
    """
    B, H, Lq, d = q.shape
    rows = np.arange(Lq) if rows is None else np.asarray(rows)
    n = rows.size
    out = {"O": np.empty((B, H, n, d)), "pred": np.empty((B, H, n)),
           "actual": np.empty((B, H, n)), "resid": np.empty((B, H, n)),
           "l": np.empty((B, H, n)), "m": np.empty((B, H, n))}
    for b in range(B):
        for h in range(H):
            qh = np.asarray(q[b, h], dtype=np.float64)
            kh = np.asarray(k[b, h], dtype=np.float64)
            vh = np.asarray(v[b, h], dtype=np.float64)
            for c0 in range(0, n, row_chunk):
                r = rows[c0:c0 + row_chunk]
                res = attention_head(qh, kh, vh, causal, scale, rows=r)
                for key, val in res.items():
                    out[key][b, h, c0:c0 + r.size] = val
    return out


def global_check(q, k, v, causal: bool, scale: float) -> float:
    """Eq. 5 for one head: sum_k sumcol_k(S) * sumrow_k(V), where sumcol is
    the column sum of the explicit normalised score matrix (Eq. 3)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    Lq, Lk = q.shape[0], k.shape[0]
    s = scale * (q @ k.T)
    vis = visible_mask(Lq, Lk, causal)
    s = np.where(vis, s, -np.inf)
    any_vis = vis.any(axis=1)
    m = np.where(any_vis, s.max(axis=1), 0.0)
    e = np.where(vis, np.exp(s - m[:, None]), 0.0)
    denom = np.where(any_vis, e.sum(axis=1), 1.0)
    A = e / denom[:, None]                 # normalised softmax matrix
    sumcol = A.sum(axis=0)                 # Eq. 3
    return float(sumcol @ sumrow(v))       # Eq. 5


def lazy_softmax_attention(q, k, v, causal: bool, scale: float) -> dict:
    """Algorithm 1 for one head, with the checksum carried as the paper
    suggests for this algorithm (Section III-B): a first pass over the keys
    finds the row max m_N; a second pass accumulates o, l and c with the
    final max; then o_N / l_N and c_N / l_N."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    Lq, Lk = q.shape[0], k.shape[0]
    d = v.shape[1]
    vis = visible_mask(Lq, Lk, causal)
    vs = sumrow(v)
    # first pass: running maximum of the scores
    m = np.full(Lq, -np.inf)
    for i in range(Lk):
        s_i = scale * (q @ k[i])
        m = np.where(vis[:, i], np.maximum(m, s_i), m)
    # second pass with the final max
    o = np.zeros((Lq, d))
    l = np.zeros(Lq)
    c = np.zeros(Lq)
    m_use = np.where(np.isfinite(m), m, 0.0)
    for i in range(Lk):
        s_i = scale * (q @ k[i])
        e = np.where(vis[:, i], np.exp(s_i - m_use), 0.0)
        o = o + e[:, None] * v[i][None, :]
        l = l + e
        c = c + e * vs[i]
    l_div = np.where(l > 0, l, 1.0)
    return {"O": o / l_div[:, None], "pred": c / l_div, "l": l, "m": m}


def online_checksum_attention(q, k, v, causal: bool, scale: float,
                              block: int = 1) -> dict:
    """Algorithm 3 for one head: FlashAttention-2 with the online checksum.

    Every query is processed in parallel (the unrolled outer loop of
    Section II). The keys are consumed in blocks of ``block`` keys; block=1
    is the per-key recurrence exactly as printed, larger blocks apply the
    same updates with the block's max (a key block is one step of the
    recurrence with the block's scores). Running state per query: m, l,
    o[d], c; each step rescales the old state by exp(m_old - m_new).
    Returns O = o_N / l_N, pred = c_N / l_N and the global check, the sum of
    pred over the queries.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    Lq, Lk = q.shape[0], k.shape[0]
    d = v.shape[1]
    vis = visible_mask(Lq, Lk, causal)
    vs = sumrow(v)
    m = np.full(Lq, -np.inf)
    l = np.zeros(Lq)
    o = np.zeros((Lq, d))
    c = np.zeros(Lq)
    for k0 in range(0, Lk, block):
        k1 = min(Lk, k0 + block)
        s = scale * (q @ k[k0:k1].T)                       # scores
        s = np.where(vis[:, k0:k1], s, -np.inf)
        m_new = np.maximum(m, s.max(axis=1))               # running max
        live = np.isfinite(m_new)
        m_use = np.where(live, m_new, 0.0)
        alpha = np.where(np.isfinite(m), np.exp(m - m_use), 0.0)
        e = np.exp(s - m_use[:, None])                     # exp(-inf) = 0
        l = l * alpha + e.sum(axis=1)                      # sum of exps
        o = o * alpha[:, None] + e @ v[k0:k1]              # output
        c = c * alpha + e @ vs[k0:k1]                      # checksum
        m = m_new
    l_div = np.where(l > 0, l, 1.0)
    pred = c / l_div
    return {"O": o / l_div[:, None], "pred": pred, "l": l, "m": m,
            "check": float(pred.sum())}


def threshold_flags(resid, O_abs_sum, pred, tau_rel: float,
                    tau_abs: float) -> np.ndarray:
    """Per-row detection rule: bit0 set when NOT |r| <= tau_rel*M + tau_abs,
    with M = sum_j |O_ij| + |pred_i| (a NaN residual also fails the
    comparison); bit1 set when the residual is not finite."""
    resid = np.asarray(resid, dtype=np.float64)
    M = np.asarray(O_abs_sum, dtype=np.float64) + np.abs(pred)
    with np.errstate(invalid="ignore"):
        ok = np.abs(resid) <= tau_rel * M + tau_abs
    bit0 = (~ok).astype(np.uint8)
    bit1 = (~np.isfinite(resid)).astype(np.uint8) << 1
    return bit0 | bit1


def brute_force_head(q, k, v, causal: bool, scale: float):
    """Pure-Python triple loop (math.exp, fp64) for tiny shapes: O, pred."""
    Lq, d = len(q), len(q[0])
    Lk = len(k)
    O, pred = [], []
    for i in range(Lq):
        keys = [kk for kk in range(Lk) if (not causal) or kk <= i + (Lk - Lq)]
        if not keys:
            O.append([0.0] * d)
            pred.append(0.0)
            continue
        s = {kk: scale * sum(float(q[i][j]) * float(k[kk][j]) for j in range(d))
             for kk in keys}
        mx = max(s.values())
        w = {kk: math.exp(s[kk] - mx) for kk in keys}
        den = sum(w.values())
        O.append([sum(w[kk] * float(v[kk][j]) for kk in keys) / den
                  for j in range(d)])
        pred.append(sum(w[kk] * sum(float(x) for x in v[kk]) for kk in keys) / den)
    return O, pred
