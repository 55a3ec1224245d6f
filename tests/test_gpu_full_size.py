"""Full-size parity of every bf16 workload (student, teacher, long-trajectory
teacher, interleaved dual cache) in the launch configuration the benchmark
times: per verifier model, verify_attn_paged over all its sequences, then
lmhead_logsoftmax_verify over all its rows with the packed W, scattering into
batch-wide outputs; one accept_scan over the whole batch; each model's
sample_takeover for its sequences.  The oracle recomputes sampled sequences of
each model (the longest, the shortest, one at the median context and, for
mixed windows, one per window length): their attention rows, their LM-head
rows, their verdicts and their takeover draws, at the bounds of the other
parity tests.

The proposals come from the synthetic proposer run on the GPU (fp32 logits;
tests.workload.gpu_proposals); both sides score the same tokens.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36546_amd import inputs, ops
from tests import parity
from tests.workload import gpu_proposals, to_np

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _sampled(b, seqs):
    """The sampled sequences of one model's sequence list."""
    ctx = b.ctx_lens[seqs]
    pick = {int(seqs[np.argmax(ctx)]), int(seqs[np.argmin(ctx)]),
            int(seqs[np.argsort(ctx, kind="stable")[len(seqs) // 2]])}
    if len(b.cfg.k_choices) > 1:
        for k in b.cfg.k_choices:
            with_k = seqs[b.k[seqs] == k]
            if len(with_k):
                pick.add(int(with_k[0]))
    return sorted(pick)


def _run(name):
    cfg = inputs.WORKLOADS[name]
    _say(f"[full-size] {name}: B={cfg.B} ctx=[{cfg.ctx_lo},{cfg.ctx_hi}] k={list(cfg.k_choices)}")
    b = inputs.make_batch(cfg, seed=0, device="cuda", poison=False)
    dev = torch.device("cuda")
    K, T = cfg.K, b.T
    t = lambda a, dt: torch.from_numpy(np.asarray(a, dt)).to(dev)
    prop_t = torch.zeros(T, dtype=torch.int32, device=dev)
    for m in b.models:
        if m.hidden.shape[0]:
            prop_t[m.rows.long()] = gpu_proposals(b, m)
    prop = to_np(prop_t).astype(np.int64)
    outs = {"lse": torch.empty(T, device=dev), "logp_prop": torch.empty(T, device=dev),
            "argmax": torch.empty(T, dtype=torch.int32, device=dev),
            "topk_idx": torch.empty(T, K, dtype=torch.int32, device=dev),
            "topk_logp": torch.empty(T, K, device=dev), "entropy": torch.empty(T, device=dev)}
    attn, ws_l, packed = {}, {}, {}
    for mi, m in enumerate(b.models):
        if m.hidden.shape[0] == 0:
            continue
        attn[mi] = parity.run_gpu_attention(m, b, seq_ids=m.seq_ids)[0]
        packed[mi] = ops.lmhead_pack_w(m.W)
        ws_l[mi] = torch.empty(ops.lmhead_workspace_size(m.hidden.shape[0], m.shape.hidden,
                                                         m.shape.vocab, K), dtype=torch.uint8,
                               device=dev)
        ops.lmhead_logsoftmax_verify(m.hidden, packed[mi], prop_t[m.rows.long()].contiguous(), K,
                                     out_rows=m.rows, n_out_rows=T, outs=outs, workspace=ws_l[mi])
    scan = parity.run_gpu_scan(b, prop, outs["topk_idx"], K, dev)
    torch.cuda.synchronize()

    # the oracle on the sampled sequences of each model
    S, logits_of, topk_ref, margin = [], {}, {}, {}
    for mi, m in enumerate(b.models):
        mine = to_np(m.seq_ids).astype(np.int64)
        if len(mine) == 0:
            continue
        seqs = _sampled(b, mine)
        S += seqs
        ref, rows = parity.oracle_attention_subset(m, b, seqs, m.shape.D)
        worst = parity.check_attention_rows(attn[mi], ref, rows, m.q.dtype)
        # LM-head rows: hidden row j of model mi is batch row m.rows[j]
        local = {int(r): j for j, r in enumerate(to_np(m.rows).astype(np.int64))}
        lrows = np.array([local[int(r)] for r in rows])
        lg = oracle.logits_fp64(to_np(m.hidden[torch.from_numpy(lrows).to(dev)]), to_np(m.W))
        r = oracle.lmhead_logsoftmax(None, None, prop[rows], K, logits=lg)
        sub = {k: v[torch.from_numpy(rows).to(dev)] for k, v in outs.items()}
        c = parity.check_lmhead(sub, r, lg, K)
        for j, row in enumerate(rows):
            logits_of[int(row)] = lg[j]
            topk_ref[int(row)] = r["topk_idx"][j]
            margin[int(row)] = r["cover_margin"][j]
        _say(f"  model {mi} sequences {seqs}: {len(rows)} rows, attention worst rel {worst:.2e}, "
             f"LM-head rows excluded {c['excluded']}")
    S = sorted(S)

    # verdicts of the sampled sequences: the oracle scan over a sub-batch of them
    ks = b.k[S]
    cu_s = np.concatenate([[0], np.cumsum(ks)])
    grow = np.concatenate([np.arange(b.cu_q[s], b.cu_q[s + 1]) for s in S])
    ref_s = oracle.accept_scan(cu_s, prop[grow], np.stack([topk_ref[int(r)] for r in grow]), K,
                               b.driver[S], b.ctx_lens[S], b.seq_lens[S], b.eos_id, b.max_len)
    # the GPU's verdict from its own top-K, where every coverage decision up
    # to the verdict row has margin > 1e-3
    n_cmp = 0
    for j, s in enumerate(S):
        r0, r1 = int(b.cu_q[s]), int(b.cu_q[s + 1])
        stop = r1 if ref_s["n_acc"][j] == r1 - r0 else r0 + ref_s["n_acc"][j] + 1
        if all(margin[r] > parity.MARGIN for r in range(r0, min(stop, r1))):
            n_cmp += 1
            for key in ("n_acc", "event_row", "next_driver", "finished", "new_cache_len"):
                assert int(to_np(scan[key])[s]) == int(ref_s[key][j]), (s, key)
    # the GPU scan with the oracle's top-K at the sampled rows: bit-exact there
    topk_mix = outs["topk_idx"].clone()
    topk_mix[torch.from_numpy(grow).to(dev)] = t(np.stack([topk_ref[int(r)] for r in grow]), np.int32)
    scan2 = parity.run_gpu_scan(b, prop, topk_mix, K, dev)
    torch.cuda.synchronize()
    for key in ("n_acc", "event_row", "next_driver", "finished", "new_cache_len"):
        np.testing.assert_array_equal(to_np(scan2[key]).astype(np.int64)[S], ref_s[key], err_msg=key)
    np.testing.assert_array_equal(to_np(scan2["src"]).astype(np.int64)[grow], ref_s["src"])

    # the teacher's replacement at each sampled takeover, drawn by the verifier
    fin0 = to_np(scan2["finished"]).copy()
    tok = torch.full((cfg.B,), -1, dtype=torch.int32, device=dev)
    for mi, m in enumerate(b.models):
        if m.hidden.shape[0] == 0:
            continue
        row_local = torch.full((T,), -1, dtype=torch.int32, device=dev)
        row_local[m.rows.long()] = torch.arange(m.rows.shape[0], dtype=torch.int32, device=dev)
        ops.sample_takeover(m.hidden, packed[mi], K, ws_l[mi], t(b.cu_q, np.int32),
                            t(b.driver, np.uint8), scan2["event_row"], t(b.u_repl, np.float32),
                            b.eos_id, scan2["finished"], row_local=row_local, seq_ids=m.seq_ids,
                            token=tok)
    torch.cuda.synchronize()
    sub_logits = np.stack([logits_of[int(r)] for r in grow])
    d = oracle.sample_takeover(cu_s, b.driver[S], ref_s["event_row"], sub_logits,
                               b.u_repl[S].astype(np.float64), b.eos_id)
    ref_d = {"token": np.full(cfg.B, -1, np.int64), "margin": np.zeros(cfg.B)}
    ref_d["token"][S] = d["token"]
    ref_d["margin"][S] = d["margin"]
    ev = to_np(scan2["event_row"]).astype(np.int64)
    exact = parity.check_takeover_draws(to_np(tok), to_np(scan2["finished"]), fin0, ref_d,
                                        lambda r: logits_of.get(int(r)), b.cu_q, b.driver, ev,
                                        b.u_repl.astype(np.float64), b.eos_id, handled=set(S))
    _say(f"  verdicts: {n_cmp}/{len(S)} sampled sequences compared from the GPU's own top-K; "
         f"draws {int((d['token'] >= 0).sum())} ({exact} above the margin)")


@pytest.mark.parametrize("name", ["student-bf16", "teacher-bf16", "long-teacher-bf16",
                                  "dual-cache-bf16"])
def test_full_size_workload_sampled(name):
    _run(name)
