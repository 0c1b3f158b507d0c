"""Shared helpers for the GPU tests: moving the seeded bf16 inputs to the
device and comparing the HIP path's results with the fp64 oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import workloads as W

# O tolerances (bf16 inputs, fp32 accumulation): max abs and relative L1
O_MAX_ABS = 2e-2
O_REL_L1 = 5e-3


def to_dev(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 bf16 patterns -> contiguous torch.bfloat16 tensor on the GPU."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).to(device).contiguous()


def from_dev_bf16(t: torch.Tensor) -> np.ndarray:
    """torch.bfloat16 tensor -> fp64 numpy (exact)."""
    bits = t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return W.bf16_bits_to_f32(bits).astype(np.float64)


def dev_inputs(inp: W.Inputs):
    return to_dev(inp.q), to_dev(inp.k), to_dev(inp.v)


def compare(o_gpu, pred_gpu, ref, d, rows=None):
    """Element-wise comparison of O and pred with the oracle on `rows`."""
    O = from_dev_bf16(o_gpu)
    pred = pred_gpu.detach().cpu().numpy().astype(np.float64)
    if rows is not None:
        O = O[:, :, rows]
        pred = pred[:, :, rows]
    err = np.abs(O - ref["O"])
    stats = {
        "o_max_abs": float(err.max()),
        "o_rel_l1": float(err.sum() / max(np.abs(ref["O"]).sum(), 1e-300)),
        "pred_max_abs": float(np.abs(pred - ref["pred"]).max()),
        "pred_rel_l1": float(np.abs(pred - ref["pred"]).sum()
                             / max(np.abs(ref["pred"]).sum(), 1e-300)),
    }
    assert np.all(np.isfinite(O)), "non-finite output"
    assert stats["o_max_abs"] <= O_MAX_ABS, stats
    assert stats["o_rel_l1"] <= O_REL_L1, stats
    assert stats["pred_max_abs"] <= O_MAX_ABS * np.sqrt(d), stats
    assert stats["pred_rel_l1"] <= O_REL_L1, stats
    return stats


def resid_ratio(o_gpu, resid, pred):
    """max_i |r_i| / (sum_j |O_ij| + |pred_i|) over all rows (O from bf16)."""
    O = from_dev_bf16(o_gpu)
    M = np.abs(O).sum(axis=-1) + np.abs(pred.detach().cpu().numpy())
    r = np.abs(resid.detach().cpu().numpy())
    live = M > 0
    return float((r[live] / M[live]).max()) if live.any() else 0.0


def oracle_rows(inp: W.Inputs, causal, scale, rows=None):
    q, k, v = inp.as_f32()
    return oracle.attention(q, k, v, causal, scale, rows=rows)
