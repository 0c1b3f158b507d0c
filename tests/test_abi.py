"""Host-side tests of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments before launching anything (these
calls never reach a kernel, so they run without a GPU)."""
import ctypes
import os
import re

import pytest

import paper_2507_16676_amd as F

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fabft.h")

# fake, 16-byte aligned, never dereferenced: validation fails before a launch
P = 4096


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fabft_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert "fabft_attn_fwd" in names and "fabft_attn_fwd_nocheck" in names
    lib = F.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert set(F.EXPORTS) == set(names)


def test_status_strings():
    for s in (0, -1, -2, -3, -4, -5, -6, -7, -8, -9, -10):
        assert F.status_str(s) and F.status_str(s) != "unknown status"
    assert F.status_str(12345) == "unknown status"


def test_key_and_query_tiles():
    assert F.key_tile(128) == 64
    assert F.key_tile(64) == 64
    assert F.query_tile(128) == 256 and F.query_tile(96) == 256
    assert F.query_tile(256) == 128 and F.query_tile(64) == 256
    assert F.lib().fabft_query_tile(80) == F.E_HEADDIM
    assert F.key_tile(96) == 64
    with pytest.raises(F.FabftError):
        F.key_tile(80)


def test_threshold_validation_and_roundtrip():
    old = F.get_threshold()
    try:
        F.set_threshold(1e-3, 2e-6)
        assert F.get_threshold() == pytest.approx((1e-3, 2e-6))
        lib = F.lib()
        assert lib.fabft_set_threshold(-1.0, 0.0) == F.E_THRESHOLD
        assert lib.fabft_set_threshold(float("nan"), 0.0) == F.E_THRESHOLD
        assert lib.fabft_set_threshold(0.0, -1.0) == F.E_THRESHOLD
        assert F.get_threshold() == pytest.approx((1e-3, 2e-6))
    finally:
        F.set_threshold(*old)


@pytest.mark.parametrize("args,code", [
    ((0, P, P, P, P, P, 1, 1, 8, 8, 128, 0, 1.0), F.E_NULL),
    ((P, P, P, P, 0, P, 1, 1, 8, 8, 128, 0, 1.0), F.E_NULL),
    ((P, P, P, P, P, 0, 1, 1, 8, 8, 128, 0, 1.0), F.E_NULL),
    ((P, P, P, P, P, P, 1, 1, 8, 8, 80, 0, 1.0), F.E_HEADDIM),
    ((P, P, P, P, P, P, 1, 1, 8, 8, 512, 0, 1.0), F.E_HEADDIM),
    ((P, P, P, P, P, P, 0, 1, 8, 8, 128, 0, 1.0), F.E_SHAPE),
    ((P, P, P, P, P, P, 1, 0, 8, 8, 128, 0, 1.0), F.E_SHAPE),
    ((P, P, P, P, P, P, 1, 1, 0, 8, 128, 0, 1.0), F.E_SHAPE),
    ((P, P, P, P, P, P, 1, 1, 8, -3, 128, 0, 1.0), F.E_SHAPE),
    ((P, P, P, P, P, P, 65536, 65536, 1024, 8, 128, 0, 1.0), F.E_SHAPE),
    # a head's K/V byte offsets must fit 32 bits: (Lk + 64) * d * 4 <= 2^32 - 1
    ((P, P, P, P, P, P, 1, 1, 1, 8388544, 128, 0, 1.0), F.E_SHAPE),   # first Lk past it
    ((P, P, P, P, P, P, 1, 1, 1, 16777152, 64, 0, 1.0), F.E_SHAPE),
    ((P, P, P, P, P, P, 1, 1, 1, 4194240, 256, 0, 1.0), F.E_SHAPE),
    ((P + 2, P, P, P, P, P, 1, 1, 8, 8, 128, 0, 1.0), F.E_ALIGN),
    ((P, P, P + 8, P, P, P, 1, 1, 8, 8, 64, 0, 1.0), F.E_ALIGN),
    ((P, P, P, P, P, P, 1, 1, 8, 8, 128, 0, -0.5), F.E_SCALE),
    ((P, P, P, P, P, P, 1, 1, 8, 8, 128, 0, float("nan")), F.E_SCALE),
    ((P, P, P, P, P, P, 1, 1, 8, 8, 128, 1, float("inf")), F.E_SCALE),
])
def test_fwd_rejects_bad_arguments(args, code):
    assert F.lib().fabft_attn_fwd(*args) == code


@pytest.mark.parametrize("args,code", [
    ((0, P, P, P, P, P, 1, 1, 8, 8, 128, 0, 1.0), F.E_NULL),
    ((P, P, P, P, 0, P, 1, 1, 8, 8, 128, 0, 1.0), F.E_NULL),
    ((P, P, P, P, P, 0, 1, 1, 8, 8, 128, 0, 1.0), F.E_NULL),
    ((P, P, P, P, P, P, 1, 1, 8, 8, 80, 0, 1.0), F.E_HEADDIM),
    ((P, P, P, P, P, P, 1, 1, 0, 8, 128, 0, 1.0), F.E_SHAPE),
    ((P, P, P, P, P, P, 1, 1, 1, 8388544, 128, 0, 1.0), F.E_SHAPE),
    ((P + 2, P, P, P, P, P, 1, 1, 8, 8, 128, 0, 1.0), F.E_ALIGN),
    ((P, P, P, P, P, P, 1, 1, 8, 8, 128, 0, -0.5), F.E_SCALE),
])
def test_twopass_rejects_bad_arguments(args, code):
    assert F.lib().fabft_attn_fwd_twopass(*args) == code


def test_twopass_rejects_the_score_check():
    """The score check runs in the one-pass kernels only: with it on, the
    two-pass entry point refuses the call before any launch."""
    L = F.lib()
    try:
        assert L.fabft_set_score_check(P, 1 << 20, 0.0) == F.FABFT_OK
        assert L.fabft_attn_fwd_twopass(P, P, P, P, P, P, 1, 2, 8, 8, 128, 1, 0.1) == F.E_MODE
    finally:
        assert L.fabft_set_score_check(None, 0, 0.0) == F.FABFT_OK


def test_algorithm_switch_validation():
    L = F.lib()
    assert L.fabft_get_algorithm() == 3
    for bad in (0, 2, 4, -1):
        assert L.fabft_set_algorithm(bad) == F.E_MODE
    assert L.fabft_get_algorithm() == 3
    try:
        assert L.fabft_set_algorithm(1) == F.FABFT_OK
        assert F.get_algorithm() == 1
        # with Algorithm 1 selected the score check is refused before a launch
        assert L.fabft_set_score_check(P, 1 << 20, 0.0) == F.FABFT_OK
        try:
            assert L.fabft_attn_fwd(P, P, P, P, P, P, 1, 2, 8, 8, 128, 1, 0.1) == F.E_MODE
        finally:
            assert L.fabft_set_score_check(None, 0, 0.0) == F.FABFT_OK
    finally:
        F.set_algorithm(3)
    assert F.get_algorithm() == 3


def test_nocheck_rejects_bad_arguments():
    lib = F.lib()
    assert lib.fabft_attn_fwd_nocheck(P, P, P, 0, 1, 1, 8, 8, 128, 0, 1.0) == F.E_NULL
    assert lib.fabft_attn_fwd_nocheck(P, P, P, P, 1, 1, 8, 8, 32, 0, 1.0) == F.E_HEADDIM
    assert lib.fabft_attn_fwd_nocheck(P, P, P, P, 1, 1, 8, 8, 64, 0, -1.0) == F.E_SCALE


@pytest.mark.parametrize("fault", [
    F.Fault("S", b=1, row=0, col=0),              # b out of range (B=1)
    F.Fault("S", h=2, row=0, col=0),              # h out of range (H=2)
    F.Fault("S", row=8, col=0),                   # row >= Lq
    F.Fault("S", row=3, col=5),                   # causal: key 5 not visible to query 3
    F.Fault("S", row=3, col=0, bit=32),
    F.Fault("P", row=3, col=0, bit=16),
    F.Fault("O", row=3, col=128, tile=0),         # col >= d
    F.Fault("O", row=3, col=0, tile=1),           # tile beyond the row's keys
    F.Fault("O", row=3, col=0, tile=-1),
    F.Fault("V", row=8, col=0, tile=0),           # key >= Lk
    F.Fault("V", row=0, col=0, tile=1),           # only one query tile
    F.Fault("V", row=0, col=0, tile=0, bit=16),
    F.Fault("C", row=0, col=2, tile=0),           # c has two parts (hi, lo)
    F.Fault("L", row=0, col=1, tile=0),           # l and m have one column
    F.Fault("L", row=8, col=0, tile=0),           # row >= Lq
    F.Fault("M", row=3, col=0, tile=1),           # tile past the row's keys
    F.Fault("C", row=0, col=0, tile=0, bit=32),
    F.Fault("Q", row=3, col=128, tile=0),         # col >= d
    F.Fault("Q", row=3, col=0, tile=0, bit=16),   # q is bf16
    F.Fault("Q", row=3, col=0, tile=1),           # tile past the row's keys
    F.Fault("VS", row=0, col=2, tile=0),          # two parts (hi, lo)
    F.Fault("VS", row=8, col=0, tile=0),          # key >= Lk
    F.Fault("VS", row=0, col=0, tile=1),          # only one query tile
    F.Fault("VS", row=0, col=1, tile=0, bit=16),
])
def test_inject_rejects_bad_faults(fault):
    f = fault.to_c()
    rc = F.lib().fabft_attn_fwd_inject(P, P, P, P, P, P, 1, 2, 8, 8, 128, 1, 0.1,
                                       ctypes.byref(f), None, None, None, None)
    assert rc == F.E_FAULT


def test_inject_rejects_unknown_site():
    for site in (10, 99, -1):
        f = F.FabftFault(site, 0, 0, 0, 0, 0, 0)
        rc = F.lib().fabft_attn_fwd_inject(P, P, P, P, P, P, 1, 1, 8, 8, 128, 0, 0.1,
                                           ctypes.byref(f), None, None, None, None)
        assert rc == F.E_FAULT


def test_inject_n_validates_the_list():
    L = F.lib()
    args = (P, P, P, P, P, P, 1, 2, 8, 8, 128, 1, 0.1)
    good = F.Fault("O", row=3, col=0, tile=0).to_c()
    bad = F.Fault("O", row=3, col=0, tile=1).to_c()
    arr = (F.FabftFault * 9)(*([good] * 9))
    assert L.fabft_attn_fwd_inject_n(*args, arr, F.MAX_FAULTS + 1, None, None, None, None) \
        == F.E_FAULT
    assert L.fabft_attn_fwd_inject_n(*args, arr, -1, None, None, None, None) == F.E_FAULT
    assert L.fabft_attn_fwd_inject_n(*args, None, 2, None, None, None, None) == F.E_NULL
    # one bad entry anywhere in the list rejects the call before any launch
    arr2 = (F.FabftFault * 3)(good, good, bad)
    assert L.fabft_attn_fwd_inject_n(*args, arr2, 3, None, None, None, None) == F.E_FAULT


def test_global_check_validation():
    L = F.lib()
    assert L.fabft_global_check(None, P, 1, 1, 8, 128, P, P) == F.E_NULL
    assert L.fabft_global_check(P, P, 1, 1, 8, 128, None, P) == F.E_NULL
    assert L.fabft_global_check(P, P, 1, 1, 8, 80, P, P) == F.E_HEADDIM
    assert L.fabft_global_check(P, P, 0, 1, 8, 128, P, P) == F.E_SHAPE
    assert L.fabft_global_check(P, P, 1, 1, 0, 128, P, P) == F.E_SHAPE
    assert L.fabft_global_check(P + 2, P, 1, 1, 8, 128, P, P) == F.E_ALIGN


def test_splitkv_workspace_size_and_validation():
    L = F.lib()
    assert L.fabft_splitkv_workspace_bytes(2, 3, 5, 128, 4) == 2 * 3 * 5 * 4 * (128 + 4) * 4
    assert L.fabft_splitkv_workspace_bytes(1, 1, 1, 64, 1) == (64 + 4) * 4
    assert L.fabft_splitkv_workspace_bytes(1, 1, 1, 80, 1) == F.E_HEADDIM
    # d = 96 keeps its partial outputs at the compute width 128
    assert L.fabft_splitkv_workspace_bytes(1, 1, 1, 96, 1) == (128 + 4) * 4
    assert L.fabft_splitkv_workspace_bytes(1, 1, 1, 128, 0) == F.E_SHAPE
    assert L.fabft_splitkv_workspace_bytes(1, 1, 1, 128, 65) == F.E_SHAPE
    need = L.fabft_splitkv_workspace_bytes(1, 2, 8, 128, 4)
    args = (P, P, P, P, P, P, 1, 2, 8, 8, 128, 1, 0.1)
    assert L.fabft_attn_fwd_splitkv(*args, 4, None, need) == F.E_NULL
    assert L.fabft_attn_fwd_splitkv(*args, 0, P, need) == F.E_SHAPE
    assert L.fabft_attn_fwd_splitkv(*args, 65, P, need) == F.E_SHAPE
    assert L.fabft_attn_fwd_splitkv(*args, 4, P + 8, need) == F.E_ALIGN
    assert L.fabft_attn_fwd_splitkv(*args, 4, P, need - 1) == F.E_WORKSPACE


def test_splitkv_noalloc_validation():
    """The allocation-free key split validates like the workspace form and
    rejects a problem whose partial states exceed its static buffer before
    anything touches the GPU."""
    L = F.lib()
    args = (P, P, P, P, P, P, 1, 2, 8, 8, 128, 1, 0.1)
    assert L.fabft_attn_fwd_splitkv_noalloc(*args[:4], None, P, *args[6:], 4) == F.E_NULL
    assert L.fabft_attn_fwd_splitkv_noalloc(*args[:5], None, *args[6:], 4) == F.E_NULL
    assert L.fabft_attn_fwd_splitkv_noalloc(*args, 0) == F.E_SHAPE
    assert L.fabft_attn_fwd_splitkv_noalloc(*args, 65) == F.E_SHAPE
    bad_d = args[:10] + (80,) + args[11:]
    assert L.fabft_attn_fwd_splitkv_noalloc(*bad_d, 4) == F.E_HEADDIM
    # 1 * 1024 heads * 1024 rows * (128 + 4) floats: 528 MiB > 64 MiB
    big = (P, P, P, P, P, P, 1, 1024, 1024, 64, 128, 0, 0.1)
    assert L.fabft_splitkv_workspace_bytes(1, 1024, 1024, 128, 1) > (64 << 20)
    assert L.fabft_attn_fwd_splitkv_noalloc(*big, 1) == F.E_WORKSPACE
    # the largest accepted problem fits exactly: (d + 4) * 4 bytes per row
    # and split, 64 MiB = 127100 rows at d = 128 with one split (not run)
    rows = (64 << 20) // ((128 + 4) * 4)
    assert L.fabft_splitkv_workspace_bytes(1, 1, rows, 128, 1) <= (64 << 20)
    assert L.fabft_splitkv_workspace_bytes(1, 1, rows + 1, 128, 1) > (64 << 20)


def test_splitkv_default_splits():
    """About 512 workgroups, at least 32 key tiles per split, 1..64 splits;
    on the measured decode shapes the fastest count (or one within 1%)."""
    assert F.splitkv_default_splits(4, 32, 1, 32768, 128) == 4
    assert F.splitkv_default_splits(4, 32, 16, 32768, 128) == 4
    assert F.splitkv_default_splits(1, 32, 1, 131072, 128) == 16
    assert F.splitkv_default_splits(8, 8, 64, 8192, 128) == 4
    for B, H, Lq, Lk, d in [(1, 1, 1, 64, 128), (1, 1, 1, 10 ** 6, 64), (64, 64, 4096, 4096, 128),
                            (2, 3, 7, 777, 64), (1, 8, 1, 2 ** 20, 256)]:
        ns = F.splitkv_default_splits(B, H, Lq, Lk, d)
        tiles = -(-Lk // F.key_tile(d))
        assert 1 <= ns <= 64
        assert ns == 1 or tiles // ns >= 32


def test_recompute_flagged_validation():
    L = F.lib()
    n1, n2 = ctypes.c_int(7), ctypes.c_int(7)
    base = (P, P, P, P, P, P, 1, 2, 8, 8, 128, 0, 0.1)
    ok = (P, P, 2, ctypes.byref(n1), ctypes.byref(n2))
    assert L.fabft_recompute_flagged(*base, *ok[:2], 0, *ok[3:]) == F.E_SHAPE
    assert L.fabft_recompute_flagged(*base, None, P, 2, *ok[3:]) == F.E_NULL
    assert L.fabft_recompute_flagged(*base, P, None, 2, *ok[3:]) == F.E_NULL
    assert L.fabft_recompute_flagged(*base, P, P, 2, None, ctypes.byref(n2)) == F.E_NULL
    bad_d = base[:10] + (80,) + base[11:]
    assert L.fabft_recompute_flagged(*bad_d, *ok) == F.E_HEADDIM
    no_flags = base[:5] + (None,) + base[6:]
    assert L.fabft_recompute_flagged(*no_flags, *ok) == F.E_NULL


def test_score_check_workspace_and_switch():
    L = F.lib()
    ntk = (4096 + 63) // 64
    assert F.score_check_workspace_bytes(2, 3, 4096, 128) == 2 * 2 * 3 * (ntk + 1) * 128 * 4
    assert F.score_check_workspace_bytes(1, 1, 100, 96) == 2 * (2 + 1) * 128 * 4
    assert L.fabft_score_check_workspace_bytes(1, 1, 100, 256) == F.E_HEADDIM
    assert L.fabft_score_check_workspace_bytes(0, 1, 100, 64) == F.E_SHAPE
    assert L.fabft_set_score_check(P + 8, 1024, 0.0) == F.E_ALIGN
    assert L.fabft_set_score_check(P, 0, 0.0) == F.E_WORKSPACE
    assert L.fabft_set_score_check(P, 1024, -1.0) == F.E_THRESHOLD
    assert L.fabft_set_score_check(P, 1024, float("nan")) == F.E_THRESHOLD
    try:
        assert L.fabft_set_score_check(P, 1024, 0.0) == F.FABFT_OK
        assert L.fabft_get_score_threshold() == pytest.approx(2.0 ** -22)
        # a call that needs more than the workspace is rejected before a launch
        assert L.fabft_attn_fwd(P, P, P, P, P, P, 1, 2, 8, 5000, 128, 1, 0.1) == F.E_WORKSPACE
        assert L.fabft_attn_fwd(P, P, P, P, P, P, 1, 2, 8, 8, 256, 1, 0.1) == F.E_HEADDIM
        assert L.fabft_set_score_check(P, 1024, 1e-3) == F.FABFT_OK
        assert L.fabft_get_score_threshold() == pytest.approx(1e-3)
    finally:
        assert L.fabft_set_score_check(None, 0, 0.0) == F.FABFT_OK


def test_caller_tensor_checks():
    """Every caller-supplied tensor is checked before its pointer reaches the
    library: shape, dtype, contiguity and device (here on CPU tensors; the
    GPU tests run the same checks through the entry points)."""
    import torch
    cpu = torch.device("cpu")
    t = torch.empty((2, 3, 5), dtype=torch.float32)
    assert F._check_out(t, "t", (2, 3, 5), torch.float32, cpu) is t
    with pytest.raises(ValueError, match="shape"):
        F._check_out(t, "t", (2, 3, 6), torch.float32, cpu)
    with pytest.raises(ValueError, match="float32"):
        F._check_out(t.to(torch.float16), "t", (2, 3, 5), torch.float32, cpu)
    with pytest.raises(ValueError, match="contiguous"):
        F._check_out(torch.empty((2, 5, 3)).transpose(1, 2), "t", (2, 3, 5), torch.float32, cpu)
    with pytest.raises(ValueError, match="on"):
        F._check_out(t, "t", (2, 3, 5), torch.float32, torch.device("meta"))
    with pytest.raises(ValueError, match="tensor"):
        F._check_out(None, "t", (2, 3, 5), torch.float32, cpu)
    ws = torch.empty(100, dtype=torch.float32)
    assert F._check_workspace(ws, "ws", 400, cpu) is ws
    with pytest.raises(ValueError, match="needed"):
        F._check_workspace(ws, "ws", 401, cpu)
    with pytest.raises(ValueError, match="contiguous"):
        F._check_workspace(torch.empty((10, 20))[:, ::2], "ws", 4, cpu)


def test_persistent_mode_validation():
    """The launch-shape switch takes off / automatic / always and refuses
    anything else (no device work: the setting is host state)."""
    L = F.lib()
    assert L.fabft_get_persistent() == F.PERSIST_AUTO
    for bad in (-1, 3, 99):
        assert L.fabft_set_persistent(bad) == F.E_MODE
        assert L.fabft_get_persistent() == F.PERSIST_AUTO
    for m in (F.PERSIST_OFF, F.PERSIST_ALWAYS, F.PERSIST_AUTO):
        assert L.fabft_set_persistent(m) == F.FABFT_OK and L.fabft_get_persistent() == m
    with pytest.raises(F.FabftError):
        F.set_persistent(5)
    assert F.get_persistent() == F.PERSIST_AUTO
