"""fp64 CPU oracle for verifier-side window scoring.

Test infrastructure only: the test suite, the smoke check and the benchmark's
CPU-baseline leg are its only users.  It shares no code with the HIP library.
"""
from .ipdv_oracle import (  # noqa: F401
    DRIVER_S, DRIVER_T, SRC_S, SRC_T, SRC_DISCARDED, REPLACEMENT,
    TAKE_COVERAGE, TAKE_ENTROPY, HAND_COVERAGE, HAND_FIXED_ONE, HAND_ENTROPY,
    append_window, gather_sequence, attention_rows, verify_attention,
    verify_attn_paged, logits_fp64, lmhead_logsoftmax, accept_scan, eq9_stepper,
    sample_categorical, sample_takeover,
    SUPPORT_UNION, SUPPORT_STUDENT, SUPPORT_TEACHER, SUPPORT_INTERSECTION,
    LOSS_IPD_SPLIT, LOSS_PURE_REVERSE, LOSS_PURE_FORWARD, LOSS_INVERSE_SPLIT,
    logp_gather, source_split_kl, source_split_kl_lists, propose_decode,
)
