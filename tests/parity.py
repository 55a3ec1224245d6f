"""Parity helpers shared by the GPU tests: run the HIP path through the C ABI,
run the oracle on the same inputs, and compare at the stated tolerances.

Tolerances (bf16 inputs, fp32 accumulation):
* attention: per (row, head) relative L2 error <= 1e-2 (fp32 inputs: 1e-4);
  every element within 2^-8 |o_ref| + 1e-2 x the row's rms (bf16; fp32:
  2^-24 |o_ref| + 1e-4 x rms).  The first term is the worst case of rounding
  the output to bf16 (unit roundoff 2^-8); the second covers rounding the
  softmax weights P to bf16 for the P.V product, whose element error measured
  by emulating that rounding on 2900 rows of N(0, 1) data (contexts 2..5000,
  D = 128) stays below 7.3e-3 x rms;
* log-probs (lse, logp_prop, topk_logp matched by index, entropy): 2e-3 abs;
* argmax, top-K sets and accept positions: bit-exact wherever the oracle's
  decision margin exceeds 1e-3; rows under the margin are checked for
  validity (each GPU pick is within 1e-3 of the oracle's K-th logit) and
  counted.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2609_36546_amd import ops
from tests.workload import to_np

MARGIN = 1e-3
LOGP_TOL = 2e-3


def attn_tol(dtype):
    return 1e-2 if dtype == torch.bfloat16 else 1e-4


def attn_elem_bound(ref, rms, dtype):
    """Per-element bound: output rounding (unit roundoff of the output type)
    times |o_ref|, plus the P-rounding allowance times the row's rms."""
    if dtype == torch.bfloat16:
        return 2.0 ** -8 * np.abs(ref) + 1e-2 * rms[..., None]
    return 2.0 ** -24 * np.abs(ref) + 1e-4 * rms[..., None]


def run_gpu_attention(mdl, batch, seq_ids=None, max_q=None, page_table=None, ctx=None, cu=None):
    """One model's verify_attn_paged on fresh copies of its pools."""
    dev = mdl.q.device
    kc = mdl.k_pool.clone()
    vc = mdl.v_pool.clone()
    ctx_t = torch.from_numpy(np.asarray(batch.ctx_lens if ctx is None else ctx, np.int32)).to(dev)
    cu_t = torch.from_numpy(np.asarray(batch.cu_q if cu is None else cu, np.int32)).to(dev)
    pt = mdl.page_table if page_table is None else page_table
    kmax = int(np.max(np.diff(np.asarray(batch.cu_q if cu is None else cu)))) if max_q is None else max_q
    out = ops.verify_attn_paged(mdl.q, mdl.k_new, mdl.v_new, kc, vc, pt, ctx_t, cu_t,
                                max_q=max(kmax, 1), seq_ids=seq_ids)
    torch.cuda.synchronize()
    return out, kc, vc


def oracle_attention(mdl, batch, seqs, D):
    """Oracle attention rows of the given sequences (host copies, fp64)."""
    out, kc, vc = oracle.verify_attn_paged(
        to_np(mdl.q), to_np(mdl.k_new), to_np(mdl.v_new), to_np(mdl.k_pool), to_np(mdl.v_pool),
        to_np(mdl.page_table), batch.ctx_lens, batch.cu_q, 1.0 / np.sqrt(D), seq_ids=seqs)
    return out, kc, vc


def check_attention_rows(gpu_out, ref_out, rows, dtype):
    """Per (row, head) relative L2 and max-abs checks; returns worst rel err."""
    tol = attn_tol(dtype)
    g = to_np(gpu_out[torch.as_tensor(rows, device=gpu_out.device)]).astype(np.float64)
    r = ref_out[rows]
    assert np.all(np.isfinite(g)), "non-finite attention output"
    num = np.linalg.norm(g - r, axis=-1)
    den = np.linalg.norm(r, axis=-1)
    rel = num / np.maximum(den, 1e-30)
    rms = den / np.sqrt(r.shape[-1])
    worst = float(rel.max()) if rel.size else 0.0
    assert worst <= tol, f"attention rel err {worst:.3e} > {tol}"
    bound = attn_elem_bound(r, rms, dtype) + 1e-30
    ratio = np.abs(g - r) / bound
    worst_elem = float(ratio.max()) if ratio.size else 0.0
    elem_rms = float((np.abs(g - r) / np.maximum(rms, 1e-30)[..., None]).max()) if ratio.size else 0.0
    print(f"  attention: worst rel L2 {worst:.3e}; worst element error {elem_rms:.3e} x rms, "
          f"{worst_elem:.3f} of its bound", flush=True)
    assert worst_elem <= 1.0, f"attention element error {worst_elem:.3f} x its bound"
    return worst


def check_lmhead(gpu, ref, logits, K, rows=None):
    """Compare GPU LM-head outputs with the oracle's; returns counts."""
    M = logits.shape[0]
    rows = np.arange(M) if rows is None else np.asarray(rows)
    lse = to_np(gpu["lse"]).astype(np.float64)[rows]
    np.testing.assert_allclose(lse, ref["lse"], atol=LOGP_TOL, rtol=0)
    lp = to_np(gpu["logp_prop"]).astype(np.float64)[rows]
    np.testing.assert_allclose(lp, ref["logp_prop"], atol=LOGP_TOL, rtol=0)
    if gpu.get("entropy") is not None:
        ent = to_np(gpu["entropy"]).astype(np.float64)[rows]
        np.testing.assert_allclose(ent, ref["entropy"], atol=LOGP_TOL, rtol=0)
    gi = to_np(gpu["topk_idx"]).astype(np.int64)[rows]
    gl = to_np(gpu["topk_logp"]).astype(np.float64)[rows]
    am = to_np(gpu["argmax"]).astype(np.int64)[rows]
    excluded = 0
    for n in range(len(rows)):
        l = logits[n]
        # log-probs of whatever the GPU picked, matched by index
        np.testing.assert_allclose(gl[n], l[gi[n]] - ref["lse"][n], atol=LOGP_TOL, rtol=0)
        assert am[n] == gi[n][0]
        assert len(set(gi[n].tolist())) == K, "duplicate top-K index"
        if ref["argmax_margin"][n] > MARGIN:
            assert am[n] == ref["argmax"][n], f"row {n}: argmax {am[n]} != {ref['argmax'][n]}"
        if ref["set_margin"][n] > MARGIN:
            assert set(gi[n].tolist()) == set(ref["topk_idx"][n].tolist()), f"row {n}: top-K set differs"
        else:
            excluded += 1
            kth = np.sort(l)[::-1][K - 1]
            assert np.all(l[gi[n]] >= kth - MARGIN), f"row {n}: invalid top-K pick"
        # the order: logits non-increasing (up to rounding) along the list
        assert np.all(np.diff(l[gi[n]]) <= 1e-4)
    return {"rows": len(rows), "excluded": excluded}


def oracle_scan(batch, prop, topk_idx, K):
    return oracle.accept_scan(batch.cu_q, prop, topk_idx, K, batch.driver, batch.ctx_lens,
                              batch.seq_lens, batch.eos_id, batch.max_len)


def run_gpu_scan(batch, prop, topk_idx_dev, K, dev):
    t = lambda a, dt: torch.from_numpy(np.asarray(a, dt)).to(dev)
    return ops.accept_scan(t(batch.cu_q, np.int32), t(prop, np.int32), topk_idx_dev, K,
                           t(batch.driver, np.uint8), t(batch.ctx_lens, np.int32),
                           t(batch.seq_lens, np.int32), batch.eos_id, batch.max_len)


def compare_scan(gpu, ref, seqs=None):
    B = len(ref["n_acc"])
    seqs = np.arange(B) if seqs is None else np.asarray(seqs)
    for key in ("n_acc", "event_row", "next_driver", "finished", "new_cache_len"):
        g = to_np(gpu[key]).astype(np.int64)[seqs]
        np.testing.assert_array_equal(g, ref[key][seqs], err_msg=key)


def oracle_attention_subset(mdl, batch, seqs, D):
    """Oracle attention for a few sequences of a large batch: only their pages
    are copied to the host (page table remapped), then the oracle runs on them."""
    ps = mdl.k_pool.shape[3]
    pt = to_np(mdl.page_table).astype(np.int64)
    need = {int(b): -(-(int(batch.ctx_lens[b]) + int(batch.k[b])) // ps) for b in seqs}
    pages = sorted({int(p) for b in seqs for p in pt[b, :need[b]]})
    remap = {p: i for i, p in enumerate(pages)}
    idx = torch.tensor(pages, dtype=torch.long, device=mdl.k_pool.device)
    kc = to_np(mdl.k_pool.index_select(0, idx))
    vc = to_np(mdl.v_pool.index_select(0, idx))
    sub_pt = np.zeros_like(pt)
    for b in seqs:
        sub_pt[b, :need[int(b)]] = [remap[int(p)] for p in pt[b, :need[int(b)]]]
    rows = np.concatenate([np.arange(batch.cu_q[b], batch.cu_q[b + 1]) for b in seqs])
    q = np.zeros(tuple(mdl.q.shape), np.float32)
    kn = np.zeros(tuple(mdl.k_new.shape), np.float32)
    vn = np.zeros(tuple(mdl.v_new.shape), np.float32)
    r = torch.from_numpy(rows).to(mdl.q.device)
    q[rows] = to_np(mdl.q.index_select(0, r))
    kn[rows] = to_np(mdl.k_new.index_select(0, r))
    vn[rows] = to_np(mdl.v_new.index_select(0, r))
    out, _, _ = oracle.verify_attn_paged(q, kn, vn, kc, vc, sub_pt, batch.ctx_lens, batch.cu_q,
                                         1.0 / np.sqrt(D), seq_ids=list(seqs))
    return out, rows


# Takeover draws: the numerical error bound of the GPU's cumulative
# probabilities (fp32 group masses over up to 2048 groups and 128 entries,
# relative rounding below 2048 * 6e-8 of the total, plus fp32-vs-fp64 logits).
DRAW_TOL = 1.2e-4
# The expected error of the same cumulative sums: fp32 logits within about
# 1e-6 relative, sums blocked over at most 16 levels of 2^-24; ten times that.
# Every draw, decided or not, must put u within CDF_TOL of the drawn token's
# interval in the oracle's CDF.
CDF_TOL = 1e-5


def check_takeover_draws(tok, fin, fin0, ref, logits_of_row, cu_q, driver, event_row, u, eos_id,
                         handled=None):
    """GPU draws against the oracle's: equal where the oracle margin exceeds
    DRAW_TOL, otherwise valid (u within DRAW_TOL of the drawn token's
    cumulative interval); finished set exactly when the draw is EOS.
    logits_of_row(r) returns the fp64 logits of global row r, or None when the
    row is not the handling verifier's.  Returns the number of exact draws."""
    exact = 0
    B = len(driver)
    for b in range(B):
        if handled is not None and b not in handled:
            continue
        r = int(cu_q[b]) + int(event_row[b]) if event_row[b] >= 0 else -1
        l = logits_of_row(r) if r >= 0 else None
        drawn = int(driver[b]) == oracle.DRIVER_S and l is not None
        if not drawn:
            assert tok[b] == -1, b
            assert fin[b] == fin0[b], b
            continue
        if ref["margin"][b] > DRAW_TOL:
            assert tok[b] == ref["token"][b], (b, tok[b], ref["token"][b], ref["margin"][b])
            exact += 1
        p = np.exp(l - l.max())
        p /= p.sum()
        c = np.cumsum(p)
        t = int(tok[b])
        assert 0 <= t < len(l), (b, t)
        lo = c[t - 1] if t > 0 else 0.0
        assert p[t] > 0 and lo - CDF_TOL <= u[b] < c[t] + CDF_TOL, (b, t, u[b], lo, c[t])
        assert fin[b] == (1 if tok[b] == eos_id else fin0[b]), b
    return exact


def check_row_draws(tok, logits, u, ref_tok, ref_margin):
    """Per-row draws against the oracle's: equal where the oracle margin
    exceeds DRAW_TOL, otherwise valid (u within DRAW_TOL of the drawn token's
    cumulative interval).  Returns (exact draws, the largest distance of u
    from the GPU token's interval in the oracle's CDF, as a fraction of the
    total mass; 0 for a draw inside its interval)."""
    exact = 0
    worst = 0.0
    for m in range(len(tok)):
        l = logits[m]
        p = np.exp(l - l.max())
        p /= p.sum()
        c = np.cumsum(p)
        t = int(tok[m])
        lo = c[t - 1] if t > 0 else 0.0
        worst = max(worst, lo - u[m], u[m] - c[t])
        if ref_margin[m] > DRAW_TOL:
            assert tok[m] == ref_tok[m], (m, tok[m], ref_tok[m], ref_margin[m])
            exact += 1
        else:
            assert p[t] > 0 and lo - DRAW_TOL <= u[m] < c[t] + DRAW_TOL, (m, t, u[m], lo, c[t])
    return exact, worst
