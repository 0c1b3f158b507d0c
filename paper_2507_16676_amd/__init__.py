"""Flash-ABFT attention forward on AMD MI355X (gfx950).

Thin Python binding over the C ABI of ``libfabft.so`` (declared in
``include/fabft.h``): argument marshalling only. Every step of the attention
and of the checksum runs in the library's HIP kernels; torch supplies device
memory and the current stream. There is no fallback: if the library is not
built, every call raises.

    o, resid, flags = attn_fwd(q, k, v, causal=True)       # checksum on
    o = attn_fwd(q, k, v, causal=True, check=False)         # checksum off

q: [B, H, Lq, d], k and v: [B, H, Lk, d], torch.bfloat16 on the GPU,
contiguous; d in {64, 96, 128, 256}. scale defaults to 1/sqrt(d). Every
caller-supplied tensor (out=, workspaces) is checked for shape, dtype,
contiguity and device before the library sees its pointer.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

_HERE = os.path.dirname(os.path.abspath(__file__))
# the in-tree build, or another build of the same library named by FABFT_LIB
# (the host-sanitized one of `python -m paper_2507_16676_amd.build
# --host-sanitize OUT`)
LIB_PATH = os.environ.get("FABFT_LIB") or os.path.join(_HERE, "libfabft.so")

_vp, _i, _f = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
_fp = ctypes.POINTER(ctypes.c_float)

FABFT_OK = 0
E_NULL, E_SHAPE, E_HEADDIM, E_ALIGN, E_LAUNCH, E_SCALE, E_FAULT, E_THRESHOLD, E_WORKSPACE, \
    E_MODE = -1, -2, -3, -4, -5, -6, -7, -8, -9, -10
PERSIST_OFF, PERSIST_AUTO, PERSIST_ALWAYS = 0, 1, 2
FLAG_RESID, FLAG_NONFINITE, FLAG_WEIGHTED, FLAG_SCORES = 1, 2, 4, 8
SITE_NONE, SITE_S, SITE_P, SITE_O, SITE_V, SITE_C, SITE_L, SITE_M, SITE_Q, SITE_VS = range(10)
SITES = {"none": SITE_NONE, "S": SITE_S, "P": SITE_P, "O": SITE_O, "V": SITE_V,
         "C": SITE_C, "L": SITE_L, "M": SITE_M, "Q": SITE_Q, "VS": SITE_VS}
MAX_FAULTS = 8


class FabftFault(ctypes.Structure):
    _fields_ = [("site", _i), ("b", _i), ("h", _i), ("row", _i), ("col", _i),
                ("tile", _i), ("bit", _i)]


class FabftDebugOut(ctypes.Structure):
    _fields_ = [("pred", _vp), ("actual", _vp), ("pred_w", _vp), ("actual_w", _vp),
                ("score_lhs", _vp), ("score_rhs", _vp), ("score_bound", _vp)]


_LIB = None


def _load() -> ctypes.CDLL:
    """Load libfabft.so once; raise if it is not built (no CPU fallback)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_2507_16676_amd.build` "
            "(hipcc, gfx950). There is no CPU fallback.")
    # torch first: it brings its own HIP runtime, and the library must bind to
    # that same runtime (the one that owns torch's memory and streams); loaded
    # before torch, it would pull in the system runtime instead and launches
    # on torch's streams fail
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    L.fabft_attn_fwd.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _f]
    L.fabft_attn_fwd.restype = _i
    L.fabft_attn_fwd_nocheck.argtypes = [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _f]
    L.fabft_attn_fwd_nocheck.restype = _i
    L.fabft_attn_fwd_twopass.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _f]
    L.fabft_attn_fwd_twopass.restype = _i
    L.fabft_set_algorithm.argtypes = [_i]
    L.fabft_set_algorithm.restype = _i
    L.fabft_get_algorithm.argtypes = []
    L.fabft_get_algorithm.restype = _i
    L.fabft_attn_fwd_inject.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i,
                                        _f, ctypes.POINTER(FabftFault), _vp, _vp, _vp, _vp]
    L.fabft_attn_fwd_inject.restype = _i
    L.fabft_attn_fwd_inject_n.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i,
                                          _f, ctypes.POINTER(FabftFault), _i, _vp, _vp, _vp,
                                          _vp]
    L.fabft_attn_fwd_inject_n.restype = _i
    L.fabft_attn_fwd_debug.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i,
                                       _f, ctypes.POINTER(FabftFault), _i,
                                       ctypes.POINTER(FabftDebugOut)]
    L.fabft_attn_fwd_debug.restype = _i
    L.fabft_score_check_workspace_bytes.argtypes = [_i, _i, _i, _i]
    L.fabft_score_check_workspace_bytes.restype = ctypes.c_longlong
    L.fabft_set_score_check.argtypes = [_vp, ctypes.c_longlong, _f]
    L.fabft_set_score_check.restype = _i
    L.fabft_get_score_threshold.argtypes = []
    L.fabft_get_score_threshold.restype = _f
    L.fabft_set_stream.argtypes = [_vp]
    L.fabft_set_stream.restype = None
    L.fabft_set_threshold.argtypes = [_f, _f]
    L.fabft_set_threshold.restype = _i
    L.fabft_get_threshold.argtypes = [_fp, _fp]
    L.fabft_get_threshold.restype = None
    L.fabft_splitkv_workspace_bytes.argtypes = [_i, _i, _i, _i, _i]
    L.fabft_splitkv_workspace_bytes.restype = ctypes.c_longlong
    L.fabft_attn_fwd_splitkv.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i,
                                         _f, _i, _vp, ctypes.c_longlong]
    L.fabft_attn_fwd_splitkv.restype = _i
    L.fabft_attn_fwd_splitkv_noalloc.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i,
                                                 _i, _i, _f, _i]
    L.fabft_attn_fwd_splitkv_noalloc.restype = _i
    L.fabft_recompute_flagged.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i,
                                          _f, _vp, _vp, _i, ctypes.POINTER(_i),
                                          ctypes.POINTER(_i)]
    L.fabft_recompute_flagged.restype = _i
    L.fabft_global_check.argtypes = [_vp, _vp, _i, _i, _i, _i, _vp, _vp]
    L.fabft_global_check.restype = _i
    L.fabft_set_weighted_check.argtypes = [_i]
    L.fabft_set_weighted_check.restype = None
    L.fabft_get_weighted_check.argtypes = []
    L.fabft_get_weighted_check.restype = _i
    L.fabft_set_persistent.argtypes = [_i]
    L.fabft_set_persistent.restype = _i
    L.fabft_get_persistent.argtypes = []
    L.fabft_get_persistent.restype = _i
    L.fabft_key_tile.argtypes = [_i]
    L.fabft_key_tile.restype = _i
    L.fabft_query_tile.argtypes = [_i]
    L.fabft_query_tile.restype = _i
    L.fabft_status_str.argtypes = [_i]
    L.fabft_status_str.restype = ctypes.c_char_p
    _LIB = L
    return L


EXPORTS = ("fabft_attn_fwd", "fabft_attn_fwd_nocheck", "fabft_attn_fwd_twopass",
           "fabft_attn_fwd_inject",
           "fabft_attn_fwd_inject_n", "fabft_attn_fwd_debug", "fabft_score_check_workspace_bytes",
           "fabft_set_score_check", "fabft_get_score_threshold",
           "fabft_attn_fwd_splitkv", "fabft_splitkv_workspace_bytes",
           "fabft_attn_fwd_splitkv_noalloc",
           "fabft_set_stream", "fabft_set_threshold", "fabft_get_threshold",
           "fabft_global_check", "fabft_recompute_flagged",
           "fabft_set_weighted_check", "fabft_get_weighted_check",
           "fabft_set_persistent", "fabft_get_persistent",
           "fabft_set_algorithm", "fabft_get_algorithm",
           "fabft_key_tile", "fabft_query_tile", "fabft_status_str")


class FabftError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} (status {status})")


def status_str(status: int) -> str:
    return _load().fabft_status_str(int(status)).decode()


def lib() -> ctypes.CDLL:
    """The loaded C library (for tests of the raw ABI)."""
    return _load()


def _check(rc: int, where: str):
    if rc != FABFT_OK:
        raise FabftError(rc, where)


def set_threshold(tau_rel: float, tau_abs: float = 0.0):
    _check(_load().fabft_set_threshold(float(tau_rel), float(tau_abs)), "fabft_set_threshold")


def get_threshold() -> tuple[float, float]:
    a, b = ctypes.c_float(), ctypes.c_float()
    _load().fabft_get_threshold(ctypes.byref(a), ctypes.byref(b))
    return a.value, b.value


def score_check_workspace_bytes(B: int, H: int, Lk: int, d: int) -> int:
    r = _load().fabft_score_check_workspace_bytes(B, H, Lk, d)
    _check(int(r) if r < 0 else 0, "fabft_score_check_workspace_bytes")
    return int(r)


_SCORE_WS = None   # keeps the workspace tensor alive while the check is on


def set_score_check(workspace=None, tau_s: float = 0.0):
    """Switch the score check on with a device workspace (a tensor of at
    least score_check_workspace_bytes bytes), or off with None."""
    global _SCORE_WS
    if workspace is None:
        _check(_load().fabft_set_score_check(None, 0, 0.0), "fabft_set_score_check")
        _SCORE_WS = None
        return
    import torch
    if not isinstance(workspace, torch.Tensor) or not workspace.is_cuda or \
            not workspace.is_contiguous():
        raise ValueError("the score-check workspace must be a contiguous GPU tensor")
    nbytes = workspace.numel() * workspace.element_size()
    _check(_load().fabft_set_score_check(workspace.data_ptr(), nbytes, float(tau_s)),
           "fabft_set_score_check")
    _SCORE_WS = workspace


def get_score_threshold() -> float:
    return float(_load().fabft_get_score_threshold())


def set_weighted_check(on: bool):
    """Switch the second, weighted checksum on or off (process-global)."""
    _load().fabft_set_weighted_check(int(bool(on)))


def get_weighted_check() -> bool:
    return bool(_load().fabft_get_weighted_check())


def set_persistent(mode: int):
    """Persistent workgroups for attn_fwd (process-global): PERSIST_OFF,
    PERSIST_AUTO (default) or PERSIST_ALWAYS. A launch shape only: the
    results are bitwise the same."""
    _check(_load().fabft_set_persistent(int(mode)), "fabft_set_persistent")


def get_persistent() -> int:
    return int(_load().fabft_get_persistent())


def set_algorithm(alg: int):
    """The algorithm hosting the checksum in attn_fwd, the injection and
    debug paths and recompute_flagged (process-global): 3 (one pass, the
    default) or 1 (two passes, as attn_fwd_twopass)."""
    _check(_load().fabft_set_algorithm(int(alg)), "fabft_set_algorithm")


def get_algorithm() -> int:
    return int(_load().fabft_get_algorithm())


def key_tile(d: int) -> int:
    r = _load().fabft_key_tile(int(d))
    _check(min(r, 0), "fabft_key_tile")
    return r


def query_tile(d: int = 128) -> int:
    """Query rows per workgroup for head dimension d (the V/VS fault tile unit)."""
    r = _load().fabft_query_tile(int(d))
    _check(r if r < 0 else 0, "fabft_query_tile")
    return r


def _shape(q, k, v):
    import torch
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dtype != torch.bfloat16:
            raise TypeError(f"{name} must be torch.bfloat16, got {t.dtype}")
        if not t.is_cuda:
            raise ValueError(f"{name} must be on the GPU")
        if t.dim() != 4 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous [B, H, L, d] tensor")
    B, H, Lq, d = q.shape
    if tuple(k.shape[:2]) != (B, H) or k.shape[3] != d or tuple(v.shape) != tuple(k.shape):
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)}")
    return B, H, Lq, k.shape[2], d


def _check_out(t, name: str, shape, dtype, device):
    """A caller-supplied tensor must have exactly this shape and dtype, be
    contiguous and sit on `device`: the library only sees its pointer and
    would write past the end of a short or mistyped buffer."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} of shape {tuple(shape)}, got {t.dtype} "
                         f"{tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")
    return t


def _check_workspace(t, name: str, need: int, device):
    """A workspace: a contiguous tensor on `device` of at least `need` bytes."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if not t.is_contiguous() or t.device != device:
        raise ValueError(f"{name} must be a contiguous tensor on {device}")
    if t.numel() * t.element_size() < need:
        raise ValueError(f"{name} holds {t.numel() * t.element_size()} bytes, {need} needed")
    return t


def _stream(dev):
    import torch
    _load().fabft_set_stream(ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))


def attn_fwd(q, k, v, causal: bool = False, scale: float | None = None, check: bool = True,
             out=None):
    """Flash-ABFT forward. Returns (o, resid, flags) with check=True, else o.

    out: optional preallocated (o[, resid, flags]) tensors to write into.
    """
    import torch
    B, H, Lq, Lk, d = _shape(q, k, v)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dev = q.device
    if out is not None:
        if len(out) not in (1, 3) or (check and len(out) != 3):
            raise ValueError("out must be (o,) with check=False, or (o, resid, flags)")
        o = _check_out(out[0], "out[0] (o)", q.shape, torch.bfloat16, dev)
    else:
        o = torch.empty_like(q)
    _stream(dev)
    if not check:
        _check(_load().fabft_attn_fwd_nocheck(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                           B, H, Lq, Lk, d, int(bool(causal)), scale),
               "fabft_attn_fwd_nocheck")
        return o
    if out is not None:
        resid = _check_out(out[1], "out[1] (resid)", (B, H, Lq), torch.float32, dev)
        flags = _check_out(out[2], "out[2] (flags)", (B, H, Lq), torch.uint8, dev)
    else:
        resid = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)
        flags = torch.empty((B, H, Lq), dtype=torch.uint8, device=dev)
    _check(_load().fabft_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                               resid.data_ptr(), flags.data_ptr(), B, H, Lq, Lk, d,
                               int(bool(causal)), scale), "fabft_attn_fwd")
    return o, resid, flags


def attn_fwd_twopass(q, k, v, causal: bool = False, scale: float | None = None, out=None):
    """Flash-ABFT checksum on Algorithm 1 (the row max in a first pass over
    the keys, then o, l and c with that fixed max). Returns (o, resid, flags)
    with the meaning of attn_fwd's. out: optional preallocated (o, resid,
    flags)."""
    import torch
    B, H, Lq, Lk, d = _shape(q, k, v)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dev = q.device
    if out is not None:
        if len(out) != 3:
            raise ValueError("out must be (o, resid, flags)")
        o = _check_out(out[0], "out[0] (o)", q.shape, torch.bfloat16, dev)
        resid = _check_out(out[1], "out[1] (resid)", (B, H, Lq), torch.float32, dev)
        flags = _check_out(out[2], "out[2] (flags)", (B, H, Lq), torch.uint8, dev)
    else:
        o = torch.empty_like(q)
        resid = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)
        flags = torch.empty((B, H, Lq), dtype=torch.uint8, device=dev)
    _stream(dev)
    _check(_load().fabft_attn_fwd_twopass(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                       resid.data_ptr(), flags.data_ptr(), B, H, Lq, Lk, d,
                                       int(bool(causal)), scale), "fabft_attn_fwd_twopass")
    return o, resid, flags


def splitkv_workspace_bytes(B: int, H: int, Lq: int, d: int, nsplit: int) -> int:
    r = _load().fabft_splitkv_workspace_bytes(int(B), int(H), int(Lq), int(d), int(nsplit))
    _check(min(int(r), 0), "fabft_splitkv_workspace_bytes")
    return int(r)


def splitkv_default_splits(B: int, H: int, Lq: int, Lk: int, d: int) -> int:
    """A split count that gives the launch about 512 workgroups (two per CU),
    with at least 32 key tiles per split (shorter splits pay their start-up
    and merge too often) and at most 64 splits. Measured on decode shapes,
    one to 64 queries over 8K-128K keys: it picks the fastest count or one
    within 1% of it."""
    n_qt = -(-Lq // query_tile(d))
    tiles = -(-Lk // key_tile(d))
    return max(1, min(64, -(-512 // (B * H * n_qt)), tiles // 32))


def attn_fwd_splitkv(q, k, v, causal: bool = False, scale: float | None = None,
                     nsplit: int | None = None, workspace=None, out=None):
    """Flash-ABFT forward with the keys split into nsplit ranges and a merge
    (for few queries over many keys). Returns (o, resid, flags). nsplit
    defaults to splitkv_default_splits(...). workspace: optional uint8 GPU
    tensor of at least splitkv_workspace_bytes(...) bytes."""
    import torch
    B, H, Lq, Lk, d = _shape(q, k, v)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dev = q.device
    if nsplit is None:
        nsplit = splitkv_default_splits(B, H, Lq, Lk, d)
    need = splitkv_workspace_bytes(B, H, Lq, d, nsplit)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    _check_workspace(workspace, "workspace", need, dev)
    if out is not None:
        o, resid, flags = out
        _check_out(o, "out[0] (o)", q.shape, torch.bfloat16, dev)
        _check_out(resid, "out[1] (resid)", (B, H, Lq), torch.float32, dev)
        _check_out(flags, "out[2] (flags)", (B, H, Lq), torch.uint8, dev)
    else:
        o = torch.empty_like(q)
        resid = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)
        flags = torch.empty((B, H, Lq), dtype=torch.uint8, device=dev)
    _stream(dev)
    _check(_load().fabft_attn_fwd_splitkv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                          resid.data_ptr(), flags.data_ptr(), B, H, Lq, Lk, d,
                                          int(bool(causal)), scale, int(nsplit),
                                          workspace.data_ptr(),
                                          workspace.numel() * workspace.element_size()),
           "fabft_attn_fwd_splitkv")
    return o, resid, flags


def recompute_flagged(q, k, v, o, resid, flags, causal: bool = False,
                      scale: float | None = None, max_retries: int = 2):
    """Re-run the checked forward on every head with a flagged row (in place,
    up to max_retries times each). Returns (n_recovered, n_persistent)."""
    import numpy as np
    import torch
    B, H, Lq, Lk, d = _shape(q, k, v)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    _check_out(o, "o", q.shape, torch.bfloat16, q.device)
    _check_out(resid, "resid", (B, H, Lq), torch.float32, q.device)
    _check_out(flags, "flags", (B, H, Lq), torch.uint8, q.device)
    hf = torch.empty(B * H, dtype=torch.uint8, device=q.device)
    hf_host = np.zeros(B * H, dtype=np.uint8)
    nr, npers = ctypes.c_int(), ctypes.c_int()
    _stream(q.device)
    _check(_load().fabft_recompute_flagged(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                           resid.data_ptr(), flags.data_ptr(), B, H, Lq, Lk, d,
                                           int(bool(causal)), scale, hf.data_ptr(),
                                           hf_host.ctypes.data_as(ctypes.c_void_p),
                                           int(max_retries), ctypes.byref(nr),
                                           ctypes.byref(npers)),
           "fabft_recompute_flagged")
    return nr.value, npers.value


def global_check(o, resid):
    """Per-head global check from attn_fwd's o and resid: returns (gsum [B, H]
    fp64 = sum of the row residuals, gflags [B, H] uint8)."""
    import torch
    if o.dtype != torch.bfloat16 or not o.is_cuda or not o.is_contiguous() or o.dim() != 4:
        raise ValueError("o must be a contiguous bf16 [B, H, Lq, d] GPU tensor")
    B, H, Lq, d = o.shape
    _check_out(resid, "resid", (B, H, Lq), torch.float32, o.device)
    gsum = torch.empty((B, H), dtype=torch.float64, device=o.device)
    gflags = torch.empty((B, H), dtype=torch.uint8, device=o.device)
    _stream(o.device)
    _check(_load().fabft_global_check(o.data_ptr(), resid.data_ptr(), B, H, Lq, d,
                                      gsum.data_ptr(), gflags.data_ptr()), "fabft_global_check")
    return gsum, gflags


@dataclass
class Fault:
    """One single-bit fault for attn_fwd_inject (fields as in fabft_fault)."""
    site: str          # "S", "P", "O", "V", "C", "L", "M", "Q", "VS" or "none"
    b: int = 0
    h: int = 0
    row: int = 0
    col: int = 0
    tile: int = 0
    bit: int = 0

    def to_c(self) -> FabftFault:
        return FabftFault(SITES[self.site], self.b, self.h, self.row, self.col, self.tile,
                          self.bit)


def _faults_array(fault):
    faults = [] if fault is None else ([fault] if isinstance(fault, Fault) else list(fault))
    if len(faults) > MAX_FAULTS:
        raise ValueError(f"at most {MAX_FAULTS} faults per launch")
    return (FabftFault * max(1, len(faults)))(*[f.to_c() for f in faults]), len(faults)


def attn_fwd_debug(q, k, v, causal: bool = False, scale: float | None = None, fault=None,
                   outputs=("pred", "actual", "pred_w", "actual_w", "score_lhs",
                            "score_rhs", "score_bound")):
    """Debug / fault-injection forward with the debug outputs named in
    `outputs` (see fabft_debug_out). Returns a dict with o, resid, flags and
    one fp32 [B, H, Lq] tensor per requested output."""
    import torch
    B, H, Lq, Lk, d = _shape(q, k, v)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dev = q.device
    res = {"o": torch.empty_like(q),
           "resid": torch.empty((B, H, Lq), dtype=torch.float32, device=dev),
           "flags": torch.empty((B, H, Lq), dtype=torch.uint8, device=dev)}
    dbg = FabftDebugOut()
    for name in outputs:
        if name not in dict(FabftDebugOut._fields_):
            raise ValueError(f"unknown debug output {name!r}")
        res[name] = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)
        setattr(dbg, name, res[name].data_ptr())
    arr, n = _faults_array(fault)
    _stream(dev)
    _check(_load().fabft_attn_fwd_debug(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                        res["o"].data_ptr(), res["resid"].data_ptr(),
                                        res["flags"].data_ptr(), B, H, Lq, Lk, d,
                                        int(bool(causal)), scale, arr, n, ctypes.byref(dbg)),
           "fabft_attn_fwd_debug")
    return res


def attn_fwd_inject(q, k, v, causal: bool = False, scale: float | None = None,
                    fault=None, out=None, weighted_out: bool = False):
    """Debug / fault-injection forward. fault: None, one Fault, or a list of
    up to MAX_FAULTS Faults applied in the same launch. Returns (o, resid,
    flags, pred, actual), followed by (pred_w, actual_w) with weighted_out=True.
    out: optional preallocated (o, resid, flags, pred, actual)."""
    import torch
    B, H, Lq, Lk, d = _shape(q, k, v)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dev = q.device
    if out is None:
        o = torch.empty_like(q)
        resid = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)
        flags = torch.empty((B, H, Lq), dtype=torch.uint8, device=dev)
        pred = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)
        actual = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)
    else:
        if len(out) != 5:
            raise ValueError("out must be (o, resid, flags, pred, actual)")
        o, resid, flags, pred, actual = out
        _check_out(o, "out[0] (o)", q.shape, torch.bfloat16, dev)
        _check_out(resid, "out[1] (resid)", (B, H, Lq), torch.float32, dev)
        _check_out(flags, "out[2] (flags)", (B, H, Lq), torch.uint8, dev)
        _check_out(pred, "out[3] (pred)", (B, H, Lq), torch.float32, dev)
        _check_out(actual, "out[4] (actual)", (B, H, Lq), torch.float32, dev)
    pw = aw = None
    if weighted_out:
        pw = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)
        aw = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)
    arr, n = _faults_array(fault)
    _stream(dev)
    _check(_load().fabft_attn_fwd_inject_n(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                        resid.data_ptr(), flags.data_ptr(), B, H, Lq, Lk, d,
                                        int(bool(causal)), scale, arr, n,
                                        pred.data_ptr(), actual.data_ptr(),
                                        pw.data_ptr() if pw is not None else None,
                                        aw.data_ptr() if aw is not None else None),
           "fabft_attn_fwd_inject_n")
    if weighted_out:
        return o, resid, flags, pred, actual, pw, aw
    return o, resid, flags, pred, actual


__all__ = ["attn_fwd", "attn_fwd_twopass", "attn_fwd_inject", "attn_fwd_debug", "attn_fwd_splitkv", "splitkv_workspace_bytes",
           "splitkv_default_splits",
           "global_check", "recompute_flagged", "Fault", "FabftError", "set_threshold",
           "set_score_check", "score_check_workspace_bytes", "get_score_threshold",
           "get_threshold", "set_weighted_check", "get_weighted_check", "set_persistent",
           "get_persistent", "set_algorithm", "get_algorithm", "key_tile",
           "query_tile", "status_str", "lib", "LIB_PATH", "EXPORTS", "MAX_FAULTS", "FLAG_RESID",
           "FLAG_NONFINITE", "FLAG_WEIGHTED", "FLAG_SCORES", "PERSIST_OFF", "PERSIST_AUTO",
           "PERSIST_ALWAYS"]
