"""Test-side helpers: host copies of a batch and the synthetic proposer.

The synthetic proposer turns a verifier's fp64 logits (from the oracle) and
the batch's per-row uniforms into proposed tokens: the argmax with
probability p_argmax, otherwise a uniform token or a sample of
softmax(l / T_alt) drawn by inverse CDF.  It is workload synthesis, not part
of the scored path.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle


def to_np(t: torch.Tensor) -> np.ndarray:
    """Exact host copy (bf16 -> fp32 is exact)."""
    t = t.detach().cpu()
    if t.dtype in (torch.bfloat16, torch.float16):
        t = t.float()
    return t.numpy()


def compose_proposals(logits: np.ndarray, u_mode, u_tok, p_argmax: float, mode: str,
                      temperature: float = 1.0) -> np.ndarray:
    M, V = logits.shape
    out = np.zeros(M, np.int64)
    for m in range(M):
        if u_mode[m] < p_argmax:
            out[m] = int(np.argmax(logits[m]))
        elif mode == "uniform":
            out[m] = min(int(u_tok[m] * V), V - 1)
        else:
            z = (logits[m] - logits[m].max()) / temperature
            cdf = np.cumsum(np.exp(z))
            out[m] = min(int(np.searchsorted(cdf, u_tok[m] * cdf[-1], side="right")), V - 1)
    return out


def model_logits(batch, mi: int) -> np.ndarray:
    mdl = batch.models[mi]
    return oracle.logits_fp64(to_np(mdl.hidden), to_np(mdl.W))


def batch_proposals(batch, logits_per_model=None) -> np.ndarray:
    """Proposed token for every batch row, from each row's verifier logits."""
    T = batch.T
    prop = np.zeros(T, np.int64)
    cfg = batch.cfg
    for mi, mdl in enumerate(batch.models):
        rows = to_np(mdl.rows).astype(np.int64)
        if len(rows) == 0:
            continue
        lg = model_logits(batch, mi) if logits_per_model is None else logits_per_model[mi]
        prop[rows] = compose_proposals(lg, batch.u_mode[rows], batch.u_tok[rows],
                                       cfg.p_argmax, cfg.alt_mode, cfg.alt_temperature)
    return prop
