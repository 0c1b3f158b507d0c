"""Seeded synthetic inputs for the Flash-ABFT attention workloads.

This module only draws random numbers and stores them in bfloat16; it holds
none of the attention or checksum arithmetic. Both the fp64 oracle and the
HIP path take their inputs from here, so that they see the same bf16 values.

Workloads (attention in the paper is softmax(Q K^T) V over one head, Eq. 1;
heads run in parallel, Section II). The paper measures the first attention
layer of four language models on one 256-token prompt (Section IV-B); those
weights and prompts are not available, so these seeded N(0,1) tensors with
the same head dimensions and attention shapes stand in for them:

  bert_l128   B=1,  H=12, L=128,   d=64,  non-causal, scale 1/8
  bert_l512   B=32, H=12, L=512,   d=64,  non-causal, Q and K pre-scaled by
              d**-0.25, kernel scale 1.0
  dec_l4096   B=4,  H=32, L=4096,  d=128, causal, scale 1/sqrt(128)
  long_l32768 B=1,  H=32, L=32768, d=128, causal, scale 1/sqrt(128); 1% of
              the K rows of every head multiplied by 8 (peaked softmax rows)

Recipe: numpy PCG64 ``default_rng(seed)``; draw order Q, K, V, each
``standard_normal((B, H, L, d), float32)``; then, for the peaked workload,
``round(frac * Lk)`` distinct K rows per (b, h) in (b, h) order, chosen without
replacement, multiplied by the factor in fp32; then round to bf16 with
round-to-nearest-even.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np


# --------------------------------------------------------------------------
# bfloat16 storage format (1 sign, 8 exponent, 7 mantissa bits)
# --------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even).

    Returns the 16-bit patterns as uint16. NaN stays NaN (quiet bit set);
    infinities and signed zeros are kept; values that round past the largest
    finite bf16 become infinity, as IEEE rounding requires.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    rounded = ((u + 0x7FFF + lsb) >> 16) & 0xFFFF
    nan = np.isnan(x)
    quiet = ((u >> 16) | 0x0040) & 0xFFFF
    out = np.where(nan, quiet, rounded)
    return out.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to fp32 exactly."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# Workload shapes
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    Lq: int
    Lk: int
    d: int
    causal: bool
    scale: float
    qk_prescale: float = 1.0    # multiplies Q and K in fp32 before rounding
    peaked_frac: float = 0.0    # fraction of K rows per head multiplied
    peaked_mult: float = 8.0
    seed: int = 0

    @property
    def visible_pairs(self) -> int:
        """Number of (query, key) pairs that take part in the softmax."""
        return self.B * self.H * visible_pairs_per_head(self.Lq, self.Lk, self.causal)

    @property
    def flops(self) -> float:
        """Attention flop count: 2d for Q K^T plus 2d for P V per visible pair."""
        return 4.0 * self.d * self.visible_pairs

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def visible_pairs_per_head(Lq: int, Lk: int, causal: bool) -> int:
    """Visible pairs of one head; causal keeps key k for query i iff
    k <= i + (Lk - Lq) (bottom-right alignment)."""
    if not causal:
        return Lq * Lk
    total = 0
    off = Lk - Lq
    # rows i with i + off >= Lk - 1 see all Lk keys; others see i + off + 1
    for i in range(Lq):
        total += max(0, min(Lk, i + off + 1))
    return total


WORKLOADS = {
    "bert_l128": Workload("bert_l128", 1, 12, 128, 128, 64, False, 1.0 / 8.0),
    "bert_l512": Workload("bert_l512", 32, 12, 512, 512, 64, False, 1.0,
                          qk_prescale=64 ** -0.25),
    "dec_l4096": Workload("dec_l4096", 4, 32, 4096, 4096, 128, True,
                          1.0 / math.sqrt(128.0)),
    "long_l32768": Workload("long_l32768", 1, 32, 32768, 32768, 128, True,
                            1.0 / math.sqrt(128.0), peaked_frac=0.01),
    # the fault-detection setting of Table I (one attention layer, sequence
    # length 256): an encoder head shape with d = 64 (non-causal) and a
    # decoder head shape with d = 128 (causal); synthetic stand-ins
    "t1_enc_d64": Workload("t1_enc_d64", 1, 12, 256, 256, 64, False, 1.0 / 8.0),
    "t1_dec_d96": Workload("t1_dec_d96", 1, 32, 256, 256, 96, True, 1.0 / math.sqrt(96.0)),
    "t1_dec_d128": Workload("t1_dec_d128", 1, 32, 256, 256, 128, True,
                            1.0 / math.sqrt(128.0)),
    "t1_dec_d256": Workload("t1_dec_d256", 1, 16, 256, 256, 256, True, 1.0 / 16.0),
    # decode: one new query per head over a 32768-key cache (the key split's shape)
    "decode_l32768": Workload("decode_l32768", 4, 32, 1, 32768, 128, False,
                              1.0 / math.sqrt(128.0)),
}


@dataclasses.dataclass
class Inputs:
    """bf16 bit patterns, shape [B, H, L, d], C-contiguous, uint16."""
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    peaked_rows: np.ndarray | None = None   # [B, H, n] indices of scaled K rows

    def as_f32(self):
        return (bf16_bits_to_f32(self.q), bf16_bits_to_f32(self.k),
                bf16_bits_to_f32(self.v))


def make_inputs(w: Workload, seed: int | None = None) -> Inputs:
    """Draw the seeded bf16 inputs of workload ``w`` (recipe in the module
    docstring)."""
    rng = np.random.default_rng(w.seed if seed is None else seed)
    qf = rng.standard_normal((w.B, w.H, w.Lq, w.d), dtype=np.float32)
    kf = rng.standard_normal((w.B, w.H, w.Lk, w.d), dtype=np.float32)
    vf = rng.standard_normal((w.B, w.H, w.Lk, w.d), dtype=np.float32)
    if w.qk_prescale != 1.0:
        f = np.float32(w.qk_prescale)
        qf *= f
        kf *= f
    rows = None
    if w.peaked_frac > 0.0:
        n = int(round(w.peaked_frac * w.Lk))
        rows = np.empty((w.B, w.H, n), dtype=np.int64)
        for b in range(w.B):
            for h in range(w.H):
                rows[b, h] = rng.choice(w.Lk, size=n, replace=False)
                kf[b, h, rows[b, h], :] *= np.float32(w.peaked_mult)
    return Inputs(f32_to_bf16_bits(qf), f32_to_bf16_bits(kf),
                  f32_to_bf16_bits(vf), rows)


def make_fp32_inputs(w: Workload, seed: int | None = None):
    """The same draws as ``make_inputs`` before bf16 rounding (fp32)."""
    rng = np.random.default_rng(w.seed if seed is None else seed)
    qf = rng.standard_normal((w.B, w.H, w.Lq, w.d), dtype=np.float32)
    kf = rng.standard_normal((w.B, w.H, w.Lk, w.d), dtype=np.float32)
    vf = rng.standard_normal((w.B, w.H, w.Lk, w.d), dtype=np.float32)
    if w.qk_prescale != 1.0:
        f = np.float32(w.qk_prescale)
        qf *= f
        kf *= f
    return qf, kf, vf


def sample_rows(Lq: int, n: int, seed: int, must: tuple[int, ...] = ()) -> np.ndarray:
    """Seeded sorted sample of ``n`` distinct query rows (plus ``must``)."""
    rng = np.random.default_rng(10_000 + seed)
    n = min(n, Lq)
    pick = set(int(r) for r in rng.choice(Lq, size=n, replace=False))
    pick.update(int(r) for r in must if 0 <= r < Lq)
    return np.array(sorted(pick), dtype=np.int64)
