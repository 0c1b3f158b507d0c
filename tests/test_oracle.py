"""Pins for the fp64 oracle, checked against things other than itself.

Each pin targets a plausible mistake: a transposed operand or a wrong scale
(library SDPA, brute force), a wrong sumrow axis or a dropped 1/l (checksum
identity, worked example), a missing rescale of c (online vs two-pass on
peaked rows), an off-by-one causal bound (brute force, causal row 0), and the
bf16 input rounding (torch's own conversion).
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


# --------------------------------------------------------------------------
# input format: bf16 round-to-nearest-even against torch's conversion
# --------------------------------------------------------------------------

def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(1)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-39).astype(np.float32),   # subnormals
        (rng.uniform(-3.4e38, 3.4e38, 2000)).astype(np.float32),  # near max
        np.array([0.0, -0.0, np.inf, -np.inf, 1.0, -1.0,
                  3.3895314e38, 3.4028235e38], dtype=np.float32),
        # exact ties: low 16 bits == 0x8000, both parities of bit 16
        np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x00018000,
                  0x7F7F8000], dtype=np.uint32).view(np.float32),
    ])
    ours = W.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = W.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy(),
                          equal_nan=True)


def test_bf16_nan_stays_nan():
    x = np.array([np.nan, -np.nan], dtype=np.float32)
    assert np.isnan(W.bf16_bits_to_f32(W.f32_to_bf16_bits(x))).all()


def test_inputs_seed_stable_and_recipe():
    w = W.WORKLOADS["bert_l128"]
    a = W.make_inputs(w)
    b = W.make_inputs(w)
    assert a.q.dtype == np.uint16 and a.q.shape == (1, 12, 128, 64)
    assert np.array_equal(a.q, b.q) and np.array_equal(a.v, b.v)
    qf, kf, vf = W.make_fp32_inputs(w)
    assert np.array_equal(W.f32_to_bf16_bits(qf), a.q)
    assert np.array_equal(W.f32_to_bf16_bits(vf), a.v)
    c = W.make_inputs(w, seed=1)
    assert not np.array_equal(a.q, c.q)


def test_peaked_rows_recipe():
    w = W.Workload("t", 1, 2, 64, 300, 8, True, 0.3, peaked_frac=0.01)
    inp = W.make_inputs(w)
    assert inp.peaked_rows.shape == (1, 2, 3)
    qf, kf, vf = W.make_fp32_inputs(w)
    k = W.bf16_bits_to_f32(inp.k)
    for h in range(2):
        rows = inp.peaked_rows[0, h]
        assert len(set(rows.tolist())) == 3
        assert np.array_equal(k[0, h, rows], W.bf16_bits_to_f32(W.f32_to_bf16_bits(kf[0, h, rows] * 8)))
        other = np.setdiff1d(np.arange(300), rows)
        assert np.array_equal(k[0, h, other], W.bf16_bits_to_f32(W.f32_to_bf16_bits(kf[0, h, other])))


def test_visible_pairs_closed_form():
    for L in (1, 2, 17, 128):
        assert W.visible_pairs_per_head(L, L, True) == L * (L + 1) // 2
        assert W.visible_pairs_per_head(L, L, False) == L * L
    assert W.visible_pairs_per_head(5, 3, True) == 0 + 0 + 1 + 2 + 3
    assert W.visible_pairs_per_head(3, 5, True) == 3 + 4 + 5


# --------------------------------------------------------------------------
# worked example (hand-derived exact values)
# --------------------------------------------------------------------------

def test_worked_example():
    with open(os.path.join(GOLDEN, "worked_example.json")) as f:
        g = json.load(f)
    q, k, v = (np.array(g[x]) for x in ("q", "k", "v"))
    assert np.allclose(oracle.sumrow(v), g["sumrow_v"], rtol=0, atol=0)
    for mode, causal in (("noncausal", False), ("causal", True)):
        r = oracle.attention_head(q, k, v, causal, g["scale"])
        assert np.allclose(r["O"], g[mode]["O"], rtol=0, atol=1e-14)
        assert np.allclose(r["pred"], g[mode]["pred"], rtol=0, atol=1e-14)
        for blk in (1, 2, 3):
            a3 = oracle.online_checksum_attention(q, k, v, causal, g["scale"], block=blk)
            assert np.allclose(a3["O"], g[mode]["O"], rtol=0, atol=1e-14)
            assert np.allclose(a3["pred"], g[mode]["pred"], rtol=0, atol=1e-14)
        a1 = oracle.lazy_softmax_attention(q, k, v, causal, g["scale"])
        assert np.allclose(a1["O"], g[mode]["O"], rtol=0, atol=1e-14)
        assert np.allclose(a1["pred"], g[mode]["pred"], rtol=0, atol=1e-14)
    assert abs(oracle.global_check(q, k, v, False, 1.0) - g["noncausal"]["global_check"]) < 1e-14


# --------------------------------------------------------------------------
# brute force on tiny shapes
# --------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("Lq,Lk", [(1, 1), (2, 3), (3, 2), (5, 5), (8, 3), (3, 8), (5, 8)])
@pytest.mark.parametrize("d", [1, 2, 4])
def test_brute_force(causal, Lq, Lk, d):
    seed = 100 * Lq + 10 * Lk + d + (7 if causal else 0)
    q, k, v = _rand((Lq, d), seed), _rand((Lk, d), seed + 1), _rand((Lk, d), seed + 2)
    scale = 0.7
    O_bf, pred_bf = oracle.brute_force_head(q.tolist(), k.tolist(), v.tolist(), causal, scale)
    r = oracle.attention_head(q, k, v, causal, scale)
    assert np.allclose(r["O"], O_bf, rtol=0, atol=1e-13)
    assert np.allclose(r["pred"], pred_bf, rtol=0, atol=1e-13)
    assert np.all(np.isfinite(r["O"]))


def test_fully_masked_rows_zero():
    # causal with Lq > Lk: the first Lq - Lk rows see no key
    q, k, v = _rand((6, 4), 1), _rand((3, 4), 2), _rand((3, 4), 3)
    r = oracle.attention_head(q, k, v, True, 0.5)
    assert np.all(r["O"][:3] == 0) and np.all(r["pred"][:3] == 0)
    assert np.all(r["resid"][:3] == 0)
    a3 = oracle.online_checksum_attention(q, k, v, True, 0.5, block=2)
    assert np.all(a3["O"][:3] == 0) and np.all(a3["pred"][:3] == 0)
    assert np.allclose(a3["O"][3:], r["O"][3:], atol=1e-14)


# --------------------------------------------------------------------------
# library routine: torch's scaled_dot_product_attention in fp64 on the CPU
# --------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [False, True])
def test_matches_torch_sdpa(causal):
    w = W.WORKLOADS["bert_l128"]
    inp = W.make_inputs(w)
    q, k, v = (x.astype(np.float64) for x in inp.as_f32())
    r = oracle.attention(q, k, v, causal, w.scale)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
        is_causal=causal, scale=w.scale).numpy()
    assert np.max(np.abs(r["O"] - ref)) < 1e-12


def test_matches_torch_sdpa_rect_mask():
    # Lq != Lk: torch's is_causal aligns top-left, so pass the bottom-right
    # mask as a boolean tensor built with torch.tril's diagonal offset
    Lq, Lk, d = 37, 90, 16
    q, k, v = _rand((1, 2, Lq, d), 5), _rand((1, 2, Lk, d), 6), _rand((1, 2, Lk, d), 7)
    mask = torch.ones(Lq, Lk, dtype=torch.bool).tril(diagonal=Lk - Lq)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
        attn_mask=mask, scale=0.25).numpy()
    r = oracle.attention(q, k, v, True, 0.25)
    assert np.max(np.abs(r["O"] - ref)) < 1e-12


def test_softmax_matrix_via_identity_values():
    # with V = I the output is the normalised score matrix itself
    Lq, Lk = 9, 13
    q, k = _rand((Lq, 5), 11), _rand((Lk, 5), 12)
    r = oracle.attention_head(q, k, np.eye(Lk), False, 0.9)
    ref = scipy.special.softmax(0.9 * (q @ k.T), axis=1)
    assert np.max(np.abs(r["O"] - ref)) < 1e-15
    assert np.max(np.abs(r["O"].sum(axis=1) - 1.0)) < 1e-14
    # and pred with V = I: sumrow(I) = 1, so pred is the row sum = 1
    assert np.max(np.abs(r["pred"] - 1.0)) < 1e-14


# --------------------------------------------------------------------------
# the checksum identity and the global form
# --------------------------------------------------------------------------

def _identity_check(w, rows=None, heads=None):
    inp = W.make_inputs(w)
    q, k, v = inp.as_f32()
    if heads is not None:
        q, k, v = q[:, heads], k[:, heads], v[:, heads]
    r = oracle.attention(q, k, v, w.causal, w.scale, rows=rows)
    M = np.abs(r["O"]).sum(axis=-1) + np.abs(r["pred"])
    assert np.all(np.abs(r["pred"] - r["actual"]) <= 1e-12 * M)
    # pred is not trivially zero: it tracks the row sums of O
    assert np.max(np.abs(r["pred"])) > 1e-3
    return r


def test_checksum_identity_bert_l128():
    _identity_check(W.WORKLOADS["bert_l128"])


def test_checksum_identity_bert_l512_sample():
    w = W.WORKLOADS["bert_l512"]
    _identity_check(w.with_(B=2))   # first two batch entries of the recipe


@pytest.mark.slow
def test_checksum_identity_dec_l4096_rows():
    w = W.WORKLOADS["dec_l4096"].with_(B=1, H=2)
    rows = W.sample_rows(w.Lq, 64, 0, must=(0, w.Lq - 1))
    _identity_check(w, rows=rows)


@pytest.mark.slow
def test_checksum_identity_long_peaked_rows():
    w = W.WORKLOADS["long_l32768"].with_(H=1)
    rows = W.sample_rows(w.Lq, 32, 0, must=(0, w.Lq - 1))
    _identity_check(w, rows=rows)


@pytest.mark.parametrize("causal", [False, True])
def test_global_check_equals_sum_of_per_query_checks(causal):
    q, k, v = _rand((40, 8), 21), _rand((40, 8), 22), _rand((40, 8), 23)
    g = oracle.global_check(q, k, v, causal, 0.4)
    r = oracle.attention_head(q, k, v, causal, 0.4)
    assert abs(g - r["pred"].sum()) <= 1e-12 * np.abs(r["pred"]).sum()
    a3 = oracle.online_checksum_attention(q, k, v, causal, 0.4, block=8)
    assert abs(a3["check"] - g) <= 1e-12 * np.abs(r["pred"]).sum()


# --------------------------------------------------------------------------
# Algorithm 3 (online, any block) == Algorithm 1 (two-pass) == definition
# --------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("Lq,Lk", [(64, 64), (33, 77), (77, 33)])
def test_online_equals_two_pass(causal, Lq, Lk):
    d = 16
    q, k, v = _rand((Lq, d), 31), _rand((Lk, d), 32), _rand((Lk, d), 33)
    # peaked rows: a few keys scaled up so the running max jumps late
    k[[5 % Lk, Lk - 2, Lk // 2]] *= 12.0
    scale = 1.0 / math.sqrt(d)
    ref = oracle.attention_head(q, k, v, causal, scale)
    a1 = oracle.lazy_softmax_attention(q, k, v, causal, scale)
    live = ref["l"] > 0
    for blk in (1, 7, 64, Lk):
        a3 = oracle.online_checksum_attention(q, k, v, causal, scale, block=blk)
        assert np.max(np.abs(a3["O"] - ref["O"])) < 1e-12
        assert np.max(np.abs(a3["pred"] - ref["pred"])) < 1e-12
        # running max ends at the row max; l agrees once both use that max
        # (same max up to the rounding of the blocked dot products)
        assert np.allclose(a3["m"][live], ref["m"][live], rtol=1e-14, atol=1e-14)
        assert np.max(np.abs(a3["l"][live] - ref["l"][live]) / ref["l"][live]) < 1e-12
    assert np.max(np.abs(a1["O"] - ref["O"])) < 1e-12
    assert np.max(np.abs(a1["pred"] - ref["pred"])) < 1e-12


def test_online_rescale_matters():
    """A recurrence that forgets to rescale c by exp(m_old - m_new) must
    disagree with the two-pass result on a row whose max grows late."""
    q = np.array([[1.0, 0.0]])
    k = np.array([[0.0, 0.0], [0.0, 1.0], [5.0, 0.0]])
    v = np.array([[1.0, 1.0], [2.0, 0.0], [-1.0, 3.0]])
    good = oracle.online_checksum_attention(q, k, v, False, 1.0, block=1)
    ref = oracle.attention_head(q, k, v, False, 1.0)
    assert abs(good["pred"][0] - ref["pred"][0]) < 1e-14
    # hand recurrence without rescaling c (the planted mistake)
    vs = v.sum(axis=1)
    s = (q @ k.T)[0]
    m, l, c = -np.inf, 0.0, 0.0
    for i in range(3):
        mn = max(m, s[i])
        a = 0.0 if m == -np.inf else math.exp(m - mn)
        l = l * a + math.exp(s[i] - mn)
        c = c + vs[i] * math.exp(s[i] - mn)      # missing "* a"
        m = mn
    assert abs(c / l - ref["pred"][0]) > 1e-3


# --------------------------------------------------------------------------
# closed forms
# --------------------------------------------------------------------------

def test_single_key():
    q, k, v = _rand((7, 6), 41), _rand((1, 6), 42), _rand((1, 6), 43)
    r = oracle.attention_head(q, k, v, False, 0.3)
    assert np.array_equal(r["O"], np.repeat(v, 7, axis=0))
    assert np.allclose(r["pred"], v.sum(), atol=1e-15, rtol=0)


@pytest.mark.parametrize("causal", [False, True])
def test_zero_scale_is_mean_of_visible_values(causal):
    q, k, v = _rand((10, 4), 51), _rand((10, 4), 52), _rand((10, 4), 53)
    r = oracle.attention_head(q, k, v, causal, 0.0)
    for i in range(10):
        n = i + 1 if causal else 10
        assert np.allclose(r["O"][i], v[:n].mean(axis=0), atol=1e-14, rtol=0)
        assert abs(r["pred"][i] - v[:n].sum(axis=1).mean()) < 1e-13
    rz = oracle.attention_head(np.zeros((10, 4)), k, v, causal, 0.7)
    assert np.allclose(rz["O"], r["O"], atol=1e-15, rtol=0)


def test_all_ones_values():
    d = 12
    q, k = _rand((9, d), 61), _rand((14, d), 62)
    for causal in (False, True):
        r = oracle.attention_head(q, k, np.ones((14, d)), causal, 0.5)
        assert np.allclose(r["O"], 1.0, atol=1e-14, rtol=0)
        assert np.allclose(r["pred"], d, atol=1e-12, rtol=0)
        assert np.allclose(r["actual"], d, atol=1e-12, rtol=0)


def test_dominant_score_selects_one_value_row():
    # one score above all others by > 750: exp underflows to exactly 0
    q = np.array([[1.0, 0.0, 0.0]])
    k = np.array([[0.0, 0.0, 0.0], [800.0, 0.0, 0.0], [1.0, 2.0, 3.0]])
    v = _rand((3, 3), 71)
    r = oracle.attention_head(q, k, v, False, 1.0)
    assert np.array_equal(r["O"][0], v[1])
    assert r["pred"][0] == v[1].sum()


def test_causal_row_zero_is_first_value_row():
    q, k, v = _rand((16, 8), 81), _rand((16, 8), 82), _rand((16, 8), 83)
    r = oracle.attention_head(q, k, v, True, 0.35)
    assert np.array_equal(r["O"][0], v[0])


# --------------------------------------------------------------------------
# invariances
# --------------------------------------------------------------------------

def test_joint_key_value_permutation_noncausal():
    q, k, v = _rand((12, 8), 91), _rand((20, 8), 92), _rand((20, 8), 93)
    perm = np.random.default_rng(0).permutation(20)
    a = oracle.attention_head(q, k, v, False, 0.4)
    b = oracle.attention_head(q, k[perm], v[perm], False, 0.4)
    assert np.max(np.abs(a["O"] - b["O"])) < 1e-13
    assert np.max(np.abs(a["pred"] - b["pred"])) < 1e-13


@pytest.mark.parametrize("causal", [False, True])
def test_value_scaling_and_shift(causal):
    d = 8
    q, k, v = _rand((12, d), 101), _rand((12, d), 102), _rand((12, d), 103)
    a = oracle.attention_head(q, k, v, causal, 0.4)
    s = oracle.attention_head(q, k, -2.5 * v, causal, 0.4)
    assert np.max(np.abs(s["O"] + 2.5 * a["O"])) < 1e-13
    assert np.max(np.abs(s["pred"] + 2.5 * a["pred"])) < 1e-13
    t = oracle.attention_head(q, k, v + 1.75, causal, 0.4)
    assert np.max(np.abs(t["O"] - (a["O"] + 1.75))) < 1e-13
    assert np.max(np.abs(t["pred"] - (a["pred"] + 1.75 * d))) < 1e-12


# --------------------------------------------------------------------------
# detection rule
# --------------------------------------------------------------------------

def test_threshold_flags_rule():
    resid = np.array([0.0, 1e-6, 1e-3, np.nan, np.inf, -2e-6])
    Oabs = np.array([1.0, 1.0, 1.0, 1.0, 1.0, 0.0])
    pred = np.array([0.0, 0.0, 0.0, 0.0, 0.0, 1.0])
    f = oracle.threshold_flags(resid, Oabs, pred, tau_rel=2e-6, tau_abs=0.0)
    assert f.tolist() == [0, 0, 1, 3, 3, 0]
    f = oracle.threshold_flags(resid, Oabs, pred, tau_rel=0.0, tau_abs=0.0)
    assert f.tolist() == [0, 1, 1, 3, 3, 1]


# --------------------------------------------------------------------------
# the weighted checksum (an extension next to the paper's check)
# --------------------------------------------------------------------------

def _brute_weighted(q, k, v, causal, scale, w):
    """Pure-Python loops: pred_w and actual_w row by row."""
    Lq, Lk, d = len(q), len(k), len(v[0])
    out = []
    for i in range(Lq):
        keys = [j for j in range(Lk) if not causal or j <= i + (Lk - Lq)]
        if not keys:
            out.append((0.0, 0.0))
            continue
        s = {j: scale * sum(q[i][t] * k[j][t] for t in range(len(q[0]))) for j in keys}
        mx = max(s.values())
        e = {j: math.exp(s[j] - mx) for j in keys}
        l = sum(e.values())
        pw = sum(e[j] * sum(w[c] * v[j][c] for c in range(d)) for j in keys) / l
        aw = sum(w[c] * sum(e[j] * v[j][c] for j in keys) / l for c in range(d))
        out.append((pw, aw))
    return np.array(out)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("Lq,Lk,d", [(1, 1, 2), (3, 5, 4), (5, 3, 3), (6, 6, 5)])
def test_weighted_brute_force(causal, Lq, Lk, d):
    seed = 7 * Lq + 3 * Lk + d + (1 if causal else 0)
    q, k, v = _rand((Lq, d), seed), _rand((Lk, d), seed + 1), _rand((Lk, d), seed + 2)
    w = [1.0 if j % 2 == 0 else -1.0 for j in range(d)]
    ref = _brute_weighted(q.tolist(), k.tolist(), v.tolist(), causal, 0.6, w)
    r = oracle.weighted_check_head(q, k, v, causal, 0.6)
    assert np.allclose(r["pred_w"], ref[:, 0], rtol=0, atol=1e-13)
    assert np.allclose(r["actual_w"], ref[:, 1], rtol=0, atol=1e-13)


def test_weighted_with_unit_weights_is_the_paper_check():
    q, k, v = _rand((17, 8), 31), _rand((23, 8), 32), _rand((23, 8), 33)
    r1 = oracle.weighted_check_head(q, k, v, True, 0.4, w=np.ones(8))
    r0 = oracle.attention_head(q, k, v, True, 0.4)
    assert np.allclose(r1["pred_w"], r0["pred"], rtol=0, atol=1e-14)
    assert np.allclose(r1["actual_w"], r0["actual"], rtol=0, atol=1e-14)


def test_weighted_identity_values_closed_form():
    # V = I: pred_w_i = sum_k softmax(s_i)_k w_k (scipy's softmax)
    Lq, Lk = 7, 10
    q, k = _rand((Lq, 4), 41), _rand((Lk, 4), 42)
    r = oracle.weighted_check_head(q, k, np.eye(Lk), False, 1.1)
    sm = scipy.special.softmax(1.1 * (q @ k.T), axis=1)
    w = np.where(np.arange(Lk) % 2 == 0, 1.0, -1.0)
    assert np.allclose(r["pred_w"], sm @ w, rtol=0, atol=1e-15)
    assert np.allclose(r["actual_w"], sm @ w, rtol=0, atol=1e-15)


def test_weighted_rows_along_the_weights():
    # V_kj = a_k w_j: both sides are d * (softmax-weighted mean of a)
    Lq, Lk, d = 5, 9, 6
    q, k = _rand((Lq, 3), 51), _rand((Lk, 3), 52)
    a = _rand((Lk,), 53)
    w = oracle.alternating_weights(d)
    v = a[:, None] * w[None, :]
    r = oracle.weighted_check_head(q, k, v, True, 0.8)
    s = 0.8 * (q @ k.T)
    s = np.where(oracle.visible_mask(Lq, Lk, True), s, -np.inf)
    sm = scipy.special.softmax(s, axis=1)
    assert np.allclose(r["pred_w"], d * (sm @ a), rtol=0, atol=1e-13)
    assert np.allclose(r["actual_w"], d * (sm @ a), rtol=0, atol=1e-13)


def test_weighted_sees_a_zero_sum_value_row():
    # a planted change of p~ at a key whose V row sums to 0 is invisible to
    # the paper's check but moves the weighted one (the reason for it)
    d = 8
    v = _rand((4, d), 61)
    v[2] = np.repeat(_rand((d // 2,), 62), 2) * np.tile([1.0, -1.0], d // 2)
    assert abs(v[2].sum()) < 1e-12
    w = oracle.alternating_weights(d)
    p = np.array([0.3, 0.2, 0.4, 0.1])
    dp = np.zeros(4)
    dp[2] = 0.05
    # sums of the output row before and after the change, divided by l
    plain = ((p + dp) @ v).sum() - (p @ v).sum()
    weighted = ((p + dp) @ v) @ w - (p @ v) @ w
    assert abs(plain) < 1e-12 and abs(weighted) > 1e-3
