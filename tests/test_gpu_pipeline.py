"""End-to-end verify step on the GPU (attention -> LM head -> accept scan)
against the oracle pipeline, per workload (scaled where the oracle needs it)."""
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
    _say(f"  scan: {n_cmp}/{cfg.B} sequences above the margin compared bit-exactly; "
         f"accepted {int(ref['n_acc'].sum())}/{T} drafts")


def test_tiny_fp32_config():
    _pipeline(inputs.CONFIGS[1], 0)


def test_student_config_scaled():
    _pipeline(inputs.scaled(inputs.CONFIGS[2], B=6, ctx_lo=64, ctx_hi=1200), 2)


def test_teacher_config_scaled():
    _pipeline(inputs.scaled(inputs.CONFIGS[3], B=5, ctx_lo=300, ctx_hi=2000), 3)


def test_dual_cache_config_scaled():
    _pipeline(inputs.scaled(inputs.CONFIGS[5], B=8, ctx_lo=20, ctx_hi=1000), 5)
