"""End-to-end verify step on the GPU (attention -> LM head -> accept scan ->
takeover draw) against the oracle pipeline, per workload (scaled where the
oracle needs it)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36546_amd import inputs, ops
from tests import parity
from tests.workload import batch_proposals, to_np

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _pipeline(cfg, seed):
    _say(f"[pipeline] cfg={cfg.name} B={cfg.B} seed={seed}")
    b = inputs.make_batch(cfg, seed=seed, device="cuda")
    K = cfg.K
    T = b.T
    dev = torch.device("cuda")
    logits = [oracle.logits_fp64(to_np(m.hidden), to_np(m.W)) for m in b.models]
    prop = batch_proposals(b, logits)
    prop_t = torch.from_numpy(prop.astype(np.int32)).to(dev)
    topk_gpu = torch.empty(T, K, dtype=torch.int32, device=dev)
    topk_ref = np.zeros((T, K), np.int64)
    cover_margin = np.zeros(T)
    for mi, m in enumerate(b.models):
        seqs = to_np(m.seq_ids).astype(np.int64)
        if len(seqs) == 0:
            continue
        out, _, _ = parity.run_gpu_attention(m, b, seq_ids=m.seq_ids)
        ref, _, _ = parity.oracle_attention(m, b, seqs, m.shape.D)
        rows = to_np(m.rows).astype(np.int64)
        parity.check_attention_rows(out, ref, rows, m.q.dtype)
        outs = {"lse": torch.empty(T, device=dev), "logp_prop": torch.empty(T, device=dev),
                "argmax": torch.empty(T, dtype=torch.int32, device=dev), "topk_idx": topk_gpu,
                "topk_logp": torch.empty(T, K, device=dev), "entropy": torch.empty(T, device=dev)}
        ops.lmhead_logsoftmax_verify(m.hidden, m.W, prop_t[m.rows.long()].contiguous(), K,
                                     out_rows=m.rows, n_out_rows=T, outs=outs)
        torch.cuda.synchronize()
        r = oracle.lmhead_logsoftmax(None, None, prop[rows], K, logits=logits[mi])
        sub = {k: v[m.rows.long()] for k, v in outs.items()}
        c = parity.check_lmhead(sub, r, logits[mi], K)
        topk_ref[rows] = r["topk_idx"]
        cover_margin[rows] = r["cover_margin"]
        _say(f"  model {mi}: rows={len(rows)} excluded={c['excluded']}")
    g = parity.run_gpu_scan(b, prop, topk_gpu, K, dev)
    torch.cuda.synchronize()
    ref = parity.oracle_scan(b, prop, topk_ref, K)
    # the scan of the GPU's own top-K lists equals the oracle scan wherever
    # every coverage decision up to the verdict row has margin > 1e-3
    n_cmp = 0
    for s in range(cfg.B):
        r0, r1 = int(b.cu_q[s]), int(b.cu_q[s + 1])
        stop = r1 if ref["n_acc"][s] == r1 - r0 else r0 + ref["n_acc"][s] + 1
        if np.all(cover_margin[r0:min(stop, r1)] > parity.MARGIN):
            n_cmp += 1
            parity.compare_scan(g, ref, [s])
    # and the GPU scan fed the oracle's top-K equals the oracle bit-exactly
    g2 = parity.run_gpu_scan(b, prop, torch.from_numpy(topk_ref.astype(np.int32)).to(dev), K, dev)
    torch.cuda.synchronize()
    parity.compare_scan(g2, ref)
    np.testing.assert_array_equal(to_np(g2["src"]).astype(np.int64), ref["src"])
    # the teacher's replacement at each takeover (from the scan above, whose
    # event rows equal the oracle's), drawn by each verifier for its sequences
    u = b.u_repl
    fin0 = to_np(g2["finished"]).copy()
    tok = torch.full((cfg.B,), -1, dtype=torch.int32, device=dev)
    cu_dev = torch.from_numpy(b.cu_q.astype(np.int32)).to(dev)
    logits_of = {}
    for mi, m in enumerate(b.models):
        if m.seq_ids.shape[0] == 0:
            continue
        rows = to_np(m.rows).astype(np.int64)
        row_local = np.full(T, -1, np.int32)
        row_local[rows] = np.arange(len(rows))
        ws = torch.empty(ops.lmhead_workspace_size(m.hidden.shape[0], m.shape.hidden, m.shape.vocab, K),
                         dtype=torch.uint8, device=dev)
        ops.lmhead_logsoftmax_verify(m.hidden, m.W, prop_t[m.rows.long()].contiguous(), K,
                                     workspace=ws)
        ops.sample_takeover(m.hidden, m.W, K, ws, cu_dev,
                            torch.from_numpy(b.driver.astype(np.uint8)).to(dev), g2["event_row"],
                            torch.from_numpy(u).to(dev), b.eos_id, g2["finished"],
                            row_local=torch.from_numpy(row_local).to(dev), seq_ids=m.seq_ids, token=tok)
        for j, r in enumerate(rows):
            logits_of[int(r)] = logits[mi][j]
    torch.cuda.synchronize()
    glog = np.stack([logits_of[r] for r in range(T)])
    ref_d = oracle.sample_takeover(b.cu_q, b.driver, ref["event_row"], glog, u.astype(np.float64), b.eos_id)
    n_draw = int((ref_d["token"] >= 0).sum())
    exact = parity.check_takeover_draws(to_np(tok), to_np(g2["finished"]), fin0, ref_d,
                                        lambda r: glog[r], b.cu_q, b.driver, ref["event_row"],
                                        u.astype(np.float64), b.eos_id)
    _say(f"  takeover draws: {n_draw}, {exact} above the margin compared exactly")
    _say(f"  scan: {n_cmp}/{cfg.B} sequences above the margin compared bit-exactly; "
         f"accepted {int(ref['n_acc'].sum())}/{T} drafts")


def test_tiny_fp32_config():
    _pipeline(inputs.WORKLOADS["tiny-f32"], 0)


def test_student_config_scaled():
    _pipeline(inputs.scaled(inputs.WORKLOADS["student-bf16"], B=6, ctx_lo=64, ctx_hi=1200), 2)


def test_teacher_config_scaled():
    _pipeline(inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=5, ctx_lo=300, ctx_hi=2000), 3)


def test_dual_cache_config_scaled():
    _pipeline(inputs.scaled(inputs.WORKLOADS["dual-cache-bf16"], B=8, ctx_lo=20, ctx_hi=1000), 5)


def test_rule_variants_on_verifier_outputs():
    """The rule variants fed by the verifier itself: the LM head's entropy at
    each row drives the entropy takeover (and, for teacher-driven windows, the
    entropy handback), and its top-K drives SKD's coverage takeover.  Both
    sides take the same float32 entropies and the same top-K lists, so the
    verdicts must be bit-exact."""
    cfg = inputs.scaled(inputs.WORKLOADS["dual-cache-bf16"], B=10, ctx_lo=20, ctx_hi=900)
    _say(f"[pipeline] rule variants on {cfg.name} B={cfg.B}")
    b = inputs.make_batch(cfg, seed=8, device="cuda")
    K, T, dev = cfg.K, b.T, torch.device("cuda")
    prop = batch_proposals(b)
    prop_t = torch.from_numpy(prop.astype(np.int32)).to(dev)
    outs = {"lse": torch.empty(T, device=dev), "logp_prop": torch.empty(T, device=dev),
            "argmax": torch.empty(T, dtype=torch.int32, device=dev),
            "topk_idx": torch.empty(T, K, dtype=torch.int32, device=dev),
            "topk_logp": torch.empty(T, K, device=dev), "entropy": torch.empty(T, device=dev)}
    for m in b.models:
        if m.hidden.shape[0] == 0:
            continue
        ops.lmhead_logsoftmax_verify(m.hidden, m.W, prop_t[m.rows.long()].contiguous(), K,
                                     out_rows=m.rows, n_out_rows=T, outs=outs)
    torch.cuda.synchronize()
    ent = to_np(outs["entropy"]).astype(np.float32)
    topk = to_np(outs["topk_idx"]).astype(np.int64)
    tau = np.float32(np.median(ent))          # about half the rows on each side
    t = lambda a, dt: torch.from_numpy(np.asarray(a, dt)).to(dev)
    for take, hand in [(oracle.TAKE_ENTROPY, oracle.HAND_ENTROPY),
                       (oracle.TAKE_COVERAGE, oracle.HAND_FIXED_ONE),
                       (oracle.TAKE_ENTROPY, oracle.HAND_COVERAGE)]:
        g = ops.accept_scan_rule(t(b.cu_q, np.int32), prop_t, outs["topk_idx"], K,
                                 t(b.driver, np.uint8), t(b.ctx_lens, np.int32),
                                 t(b.seq_lens, np.int32), b.eos_id, b.max_len, take_rule=take,
                                 hand_rule=hand, ent=outs["entropy"], tau_take=float(tau),
                                 tau_hand=float(tau))
        torch.cuda.synchronize()
        ref = oracle.accept_scan(b.cu_q, prop, topk, K, b.driver, b.ctx_lens, b.seq_lens,
                                 b.eos_id, b.max_len, take_rule=take, hand_rule=hand,
                                 ent=ent.astype(np.float64), tau_take=float(tau),
                                 tau_hand=float(tau))
        parity.compare_scan(g, ref)
        np.testing.assert_array_equal(to_np(g["src"]).astype(np.int64), ref["src"])
        _say(f"  take={take} hand={hand}: events {int((ref['event_row'] >= 0).sum())}/{cfg.B}, "
             f"accepted {int(ref['n_acc'].sum())}/{T}")
