"""GPU parity of sample_takeover (the teacher's replacement draw at a takeover,
Eq. (9) second case) against the fp64 oracle, through the C ABI.

The draw is an inverse CDF: it is unique wherever the uniform lies farther
than the numerical error of the cumulative probabilities from an interval
end.  parity.DRAW_TOL is that error bound for the GPU's fp32 arithmetic:
group masses summed over up to 2048 groups and 128 entries (relative rounding
below 2048 * 6e-8 = 1.2e-4 of the total in the worst case, about 2e-6
typically) plus the difference between fp32 and fp64 logits (about 1e-6
relative per probability).  Draws with a larger oracle margin must equal the
oracle's.  Every draw must also put u within parity.CDF_TOL = 1e-5 of the
drawn token's interval in the oracle's CDF (the expected error of the GPU's
cumulative sums, about 1e-6 of the mass, times ten).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36546_amd import ops
from tests import parity
from tests.workload import to_np

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _setup(M, Hd, V, dtype, seed, std=0.02, K=16):
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    h = torch.randn(M, Hd, generator=gen, device="cuda")
    h = (h / h.pow(2).mean(1, keepdim=True).sqrt()).to(dtype)
    W = (torch.randn(V, Hd, generator=gen, device="cuda") * std).to(dtype)
    return h, W


def _lmhead(h, W, K):
    M = h.shape[0]
    ws = torch.empty(ops.lmhead_workspace_size(M, h.shape[1], W.shape[0], K), dtype=torch.uint8,
                     device="cuda")
    prop = torch.zeros(M, dtype=torch.int32, device="cuda")
    ops.lmhead_logsoftmax_verify(h, W, prop, K, workspace=ws)
    return ws


def _check(h, W, K, cu_q, driver, event_row, u, eos_id, row_local=None, finished0=None):
    ws = _lmhead(h, W, K)
    dev = h.device
    B = len(driver)
    fin = torch.from_numpy(np.zeros(B, np.uint8) if finished0 is None else finished0.copy()).to(dev)
    tok = ops.sample_takeover(
        h, W, K, ws, torch.from_numpy(np.asarray(cu_q, np.int32)).to(dev),
        torch.from_numpy(np.asarray(driver, np.uint8)).to(dev),
        torch.from_numpy(np.asarray(event_row, np.int32)).to(dev),
        torch.from_numpy(np.asarray(u, np.float32)).to(dev), eos_id, fin,
        row_local=None if row_local is None else torch.from_numpy(np.asarray(row_local, np.int32)).to(dev))
    torch.cuda.synchronize()
    tok, fin = to_np(tok), to_np(fin)
    logits_local = oracle.logits_fp64(to_np(h), to_np(W))
    T = int(cu_q[-1])
    if row_local is None:
        logits = logits_local
    else:
        logits = np.full((T, W.shape[0]), -np.inf)
        for r in range(T):
            if row_local[r] >= 0:
                logits[r] = logits_local[row_local[r]]
    # the oracle draws with the same float32 uniform
    u64 = np.asarray(u, np.float32).astype(np.float64)
    ref = oracle.sample_takeover(cu_q, driver, event_row, logits, u64, eos_id)
    fin0 = np.zeros(B, np.uint8) if finished0 is None else finished0
    lrow = lambda r: None if (row_local is not None and row_local[r] < 0) else logits[r]
    exact = parity.check_takeover_draws(tok, fin, fin0, ref, lrow, cu_q, driver, event_row, u64,
                                        eos_id)
    return tok, exact


def test_small_vocab_many_uniforms():
    """One takeover row per sequence, 64 sequences sharing four rows' logits,
    uniforms spread over [0, 1)."""
    _say("[sample] V=1000 Hd=256 B=64")
    M, Hd, V, K = 4, 256, 1000, 16
    h, W = _setup(M, Hd, V, torch.bfloat16, 1, std=0.2)
    B = 64
    # sequence b: one-row window on hidden row b % 4 -- cu_q maps sequence
    # b to global row b; row_local maps global rows onto the 4 hidden rows
    cu_q = np.arange(B + 1)
    row_local = np.arange(B) % M
    driver = np.full(B, oracle.DRIVER_S, np.uint8)
    event_row = np.zeros(B, np.int32)
    u = (np.arange(B) + 0.37) / B
    tok, exact = _check(h, W, K, cu_q, driver, event_row, u, eos_id=V - 1, row_local=row_local)
    _say(f"  exact={exact}/{B}")
    assert exact >= B // 2


def test_peaked_rows_exact():
    """Scaled W: a few tokens carry the mass, so every draw is far from an
    interval end and must equal the oracle's."""
    _say("[sample] peaked V=5003")
    M, Hd, V, K = 12, 128, 5003, 8
    h, W = _setup(M, Hd, V, torch.bfloat16, 2, std=0.6)
    cu_q = np.arange(M + 1)
    driver = np.full(M, oracle.DRIVER_S, np.uint8)
    event_row = np.zeros(M, np.int32)
    u = np.random.default_rng(3).random(M).astype(np.float32)
    tok, exact = _check(h, W, K, cu_q, driver, event_row, u, eos_id=V - 1)
    _say(f"  exact={exact}/{M}")
    assert exact >= M - 2


def test_full_vocab_teacher_shape_and_windows():
    """V = 151936, Hd = 2048; 8-row windows with takeovers at various rows,
    a window without event and teacher-driven windows (no draw).  At the
    workload's W scale every probability is below DRAW_TOL, so those draws
    are checked against CDF_TOL only; the windows of the last four sequences
    sit on rows whose distribution is made peaked (16 boosted W rows aligned
    with the hidden row, spread over the vocabulary and the group records),
    and at least one of their draws must equal the oracle's exactly."""
    _say("[sample] V=151936 Hd=2048 B=16 k=8")
    B, k = 16, 8
    M, Hd, V, K = B * k, 2048, 151936, 16
    h, W = _setup(M, Hd, V, torch.bfloat16, 4)
    rng = np.random.default_rng(5)
    # peaked rows: the takeover rows of sequences 12..15 share one hidden row
    # h0; 16 W rows get 0.008 * h0 added (logit gain about 0.008 * Hd = 16, so
    # they carry all but about 1e-3 of the mass)
    peaked_rows = [12 * k + 3, 13 * k + 0, 14 * k + 7, 15 * k + 5]
    h0 = h[peaked_rows[0]].float()
    for r in peaked_rows[1:]:
        h[r] = h[peaked_rows[0]]
    boosted = np.sort(rng.choice(V, 16, replace=False))
    W[torch.from_numpy(boosted).cuda()] = (W[torch.from_numpy(boosted).cuda()].float()
                                             + 0.008 * h0).to(W.dtype)
    cu_q = np.arange(B + 1) * k
    driver = np.where(np.arange(B) % 4 == 3, oracle.DRIVER_T, oracle.DRIVER_S).astype(np.uint8)
    driver[12:] = oracle.DRIVER_S
    event_row = rng.integers(0, k, size=B).astype(np.int32)
    event_row[1] = -1
    event_row[12:] = [3, 0, 7, 5]
    u = rng.random(B).astype(np.float32)
    fin0 = (np.arange(B) % 5 == 0).astype(np.uint8)
    tok, exact = _check(h, W, K, cu_q, driver, event_row, u, eos_id=V - 1, finished0=fin0)
    _say(f"  exact={exact}; peaked-row draws {tok[12:].tolist()}")
    assert exact >= 1
    assert all(int(t) in set(boosted.tolist()) for t in tok[12:])


def test_eos_replacement_finishes_and_fp32():
    """A row whose mass sits on EOS: the draw is EOS and finished is set;
    fp32 inputs; u close to 1 exercises the top end of the CDF."""
    _say("[sample] EOS path fp32")
    M, Hd, V, K = 3, 64, 300, 4
    h, W = _setup(M, Hd, V, torch.float32, 6, std=0.05)
    W[V - 1] = h[0] * 0.5           # logit of EOS on row 0: 0.5 * Hd = 32
    cu_q = np.array([0, 1, 2, 3])
    driver = np.full(3, oracle.DRIVER_S, np.uint8)
    event_row = np.zeros(3, np.int32)
    u = np.array([0.5, 0.9999999, 0.0], np.float32)
    tok, _ = _check(h, W, K, cu_q, driver, event_row, u, eos_id=V - 1)
    assert tok[0] == V - 1


def test_two_verifiers_compose_with_seq_ids():
    """Two LM heads over disjoint row sets (two models): each call handles its
    own sequences (seq_ids) and rows (row_local); the other call's outputs
    stay untouched."""
    _say("[sample] two verifiers")
    Hd, V, K = 128, 2000, 8
    cu_q = np.array([0, 2, 5, 6, 9])           # 4 sequences, 9 rows
    seqs = [np.array([0, 2], np.int32), np.array([1, 3], np.int32)]
    rows = [np.array([0, 1, 5], np.int32), np.array([2, 3, 4, 6, 7, 8], np.int32)]
    driver = np.full(4, oracle.DRIVER_S, np.uint8)
    event_row = np.array([1, 2, 0, 0], np.int32)
    u = np.array([0.3, 0.6, 0.9, 0.05], np.float32)
    dev = torch.device("cuda")
    tok = torch.full((4,), -7, dtype=torch.int32, device=dev)
    fin = torch.zeros(4, dtype=torch.uint8, device=dev)
    logits_rows = np.zeros((9, V))
    for mi in range(2):
        h, W = _setup(len(rows[mi]), Hd, V, torch.bfloat16, 10 + mi, std=0.1)
        ws = _lmhead(h, W, K)
        row_local = np.full(9, -1, np.int32)
        row_local[rows[mi]] = np.arange(len(rows[mi]))
        ops.sample_takeover(h, W, K, ws, torch.from_numpy(cu_q.astype(np.int32)).to(dev),
                            torch.from_numpy(driver).to(dev), torch.from_numpy(event_row).to(dev),
                            torch.from_numpy(u).to(dev), V - 1, fin,
                            row_local=torch.from_numpy(row_local).to(dev),
                            seq_ids=torch.from_numpy(seqs[mi]).to(dev), token=tok)
        logits_rows[rows[mi]] = oracle.logits_fp64(to_np(h), to_np(W))
    torch.cuda.synchronize()
    ref = oracle.sample_takeover(cu_q, driver, event_row, logits_rows, u.astype(np.float64), V - 1)
    exact = parity.check_takeover_draws(to_np(tok), to_np(fin), np.zeros(4, np.uint8), ref,
                                        lambda r: logits_rows[r], cu_q, driver, event_row,
                                        u.astype(np.float64), V - 1)
    _say(f"  exact={exact}/4")
