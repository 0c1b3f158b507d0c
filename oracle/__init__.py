"""fp64 CPU oracle for Flash-ABFT attention.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.
"""
from .attention import (visible_mask, sumrow, attention_head, attention,
                        global_check, lazy_softmax_attention,
                        online_checksum_attention, threshold_flags,
                        brute_force_head, alternating_weights,
                        weighted_check_head)

__all__ = ["visible_mask", "sumrow", "attention_head", "attention",
           "global_check", "lazy_softmax_attention",
           "online_checksum_attention", "threshold_flags", "brute_force_head",
           "alternating_weights", "weighted_check_head"]
