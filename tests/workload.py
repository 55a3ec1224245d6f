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


def gpu_proposals(batch, mdl) -> torch.Tensor:
    """The synthetic proposer for full-size batches, on the GPU: per row of
    ``mdl``, the verifier's argmax with probability p_argmax, else a uniform
    token or an inverse-CDF sample of softmax(l / T_alt), from fp32 logits of
    a torch matmul.  Workload synthesis only: both the GPU path and the
    oracle score the tokens it returns (int32 [M], on the GPU)."""
    cfg = batch.cfg
    dev = mdl.hidden.device
    rows = to_np(mdl.rows).astype(np.int64)
    M = len(rows)
    um = torch.from_numpy(batch.u_mode[rows]).to(dev)
    ut = torch.from_numpy(batch.u_tok[rows]).to(dev)
    Wf = mdl.W.float()
    out = torch.empty(M, dtype=torch.int64, device=dev)
    for r0 in range(0, M, 64):
        l = mdl.hidden[r0:r0 + 64].float() @ Wf.T
        am = l.argmax(1)
        if cfg.alt_mode == "uniform":
            alt = torch.clamp((ut[r0:r0 + 64] * l.shape[1]).long(), max=l.shape[1] - 1)
        else:
            cdf = torch.softmax(l.double() / cfg.alt_temperature, 1).cumsum(1)
            alt = torch.searchsorted(cdf, (ut[r0:r0 + 64] * cdf[:, -1]).unsqueeze(1)).squeeze(1)
            alt = torch.clamp(alt, max=l.shape[1] - 1)
        out[r0:r0 + 64] = torch.where(um[r0:r0 + 64] < cfg.p_argmax, am, alt)
    return out.int()
