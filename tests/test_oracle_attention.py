"""Pins of the oracle's verification-stage attention (append + causal attention).

Each test checks the oracle against something other than itself: closed
forms, a library routine (torch fp64 scaled_dot_product_attention), or an
equivalence the method fixes (a k-token window equals k decode steps with
append; paged equals contiguous; eviction recompute equals the cached pass,
Section 3.2.3).
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

RNG = np.random.default_rng(1234)


def build_paged(Kseq, Vseq, ps, num_pages, pages):
    """Test-side writer of the documented layouts from contiguous K/V [n, Hkv, D]."""
    n, Hkv, D = Kseq.shape
    kc = np.full((num_pages, Hkv, D // 32, ps, 32), np.nan)
    vc = np.full((num_pages, Hkv, D, ps), np.nan)
    for p in range(n):
        for d in range(D):
            kc[pages[p // ps], :, d // 32, p % ps, d % 32] = Kseq[p, :, d]
        vc[pages[p // ps], :, :, p % ps] = Vseq[p]
    return kc, vc


def one_seq_case(L, k, Hq, Hkv, D, ps, rng=RNG, permute=True):
    """One sequence: cached prefix of L tokens + a k-row window."""
    n = L + k
    Kall = rng.standard_normal((n, Hkv, D))
    Vall = rng.standard_normal((n, Hkv, D))
    q = rng.standard_normal((k, Hq, D))
    need = -(-n // ps)
    num_pages = 2 * need + 1
    pages = rng.permutation(num_pages - 1)[:need] if permute else np.arange(need)
    pt = np.full((1, need + 2), num_pages - 1, np.int64)
    pt[0, :need] = pages
    kc, vc = build_paged(Kall[:L], Vall[:L], ps, num_pages, pages)
    return dict(q=q, k_new=Kall[L:], v_new=Vall[L:], kc=kc, vc=vc, pt=pt,
                ctx=np.array([L]), cu=np.array([0, k]), Kall=Kall, Vall=Vall)


def run(c, scale):
    return oracle.verify_attn_paged(c["q"], c["k_new"], c["v_new"], c["kc"], c["vc"],
                                    c["pt"], c["ctx"], c["cu"], scale)


def sdpa_reference(q, Kall, Vall, L, scale):
    """torch fp64 SDPA with an explicit causal mask on contiguous K/V, KV heads
    repeated per group."""
    k, Hq, D = q.shape
    Hkv = Kall.shape[1]
    G = Hq // Hkv
    Kr = torch.from_numpy(np.repeat(Kall, G, axis=1)).permute(1, 0, 2)   # [Hq, n, D]
    Vr = torch.from_numpy(np.repeat(Vall, G, axis=1)).permute(1, 0, 2)
    Q = torch.from_numpy(q).permute(1, 0, 2)                               # [Hq, k, D]
    n = Kall.shape[0]
    mask = torch.zeros(k, n, dtype=torch.bool)
    for i in range(k):
        mask[i, : L + i + 1] = True
    o = F.scaled_dot_product_attention(Q, Kr, Vr, attn_mask=mask, scale=scale)
    return o.permute(1, 0, 2).numpy()


@pytest.mark.parametrize("L,k,Hq,Hkv,D,ps", [
    (37, 4, 4, 2, 32, 16), (0, 5, 4, 4, 32, 16), (64, 1, 8, 2, 64, 16),
    (100, 8, 6, 3, 32, 32), (15, 3, 2, 1, 64, 8)])
def test_matches_torch_sdpa_fp64(L, k, Hq, Hkv, D, ps):
    c = one_seq_case(L, k, Hq, Hkv, D, ps)
    scale = 1.0 / np.sqrt(D)
    out, _, _ = run(c, scale)
    ref = sdpa_reference(c["q"], c["Kall"], c["Vall"], L, scale)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


def test_window_rows_appended_into_pages():
    c = one_seq_case(20, 6, 4, 2, 32, 16)
    _, kc, vc = run(c, 0.3)
    K, V = oracle.gather_sequence(kc, vc, c["pt"], 0, 26)
    np.testing.assert_array_equal(K, c["Kall"])
    np.testing.assert_array_equal(V, c["Vall"])


def test_constant_values_give_constant_output():
    c = one_seq_case(33, 4, 4, 2, 32, 16)
    c["vc"][:] = 2.5
    c["v_new"][:] = 2.5
    out, _, _ = run(c, 0.25)
    np.testing.assert_allclose(out, 2.5, rtol=0, atol=1e-13)


def test_zero_query_gives_mean_of_visible_values():
    L, k = 29, 5
    c = one_seq_case(L, k, 4, 2, 32, 16)
    c["q"][:] = 0.0
    out, _, _ = run(c, 0.25)
    G = 2
    for i in range(k):
        for h in range(4):
            np.testing.assert_allclose(out[i, h], c["Vall"][: L + i + 1, h // G].mean(axis=0),
                                       rtol=1e-12, atol=1e-12)


def test_dominant_key_selects_its_value():
    L, k, D = 40, 3, 32
    c = one_seq_case(L, k, 2, 1, D, 16)
    j = 17
    c["q"][:] = 0.0
    c["q"][:, :, 0] = 1.0
    Kd = np.zeros((L + k, 1, D))
    Kd[j, 0, 0] = 200.0
    c["kc"], c["vc"] = build_paged(Kd[:L], c["Vall"][:L], 16, c["kc"].shape[0],
                                   c["pt"][0][: -(-(L + k) // 16)])
    c["k_new"] = Kd[L:]
    out, _, _ = run(c, 1.0)
    np.testing.assert_allclose(out[:, 0, :], np.broadcast_to(c["Vall"][j, 0], (k, D)),
                               rtol=0, atol=1e-12)


def test_k_window_equals_sequential_decode_with_append():
    L, k, Hq, Hkv, D, ps = 45, 6, 4, 2, 32, 16
    c = one_seq_case(L, k, Hq, Hkv, D, ps)
    scale = 0.2
    win, _, _ = run(c, scale)
    kc, vc = c["kc"].copy(), c["vc"].copy()
    for i in range(k):
        out, kc, vc = oracle.verify_attn_paged(
            c["q"][i:i + 1], c["k_new"][i:i + 1], c["v_new"][i:i + 1], kc, vc, c["pt"],
            np.array([L + i]), np.array([0, 1]), scale)
        np.testing.assert_allclose(win[i], out[0], rtol=1e-12, atol=1e-13)


def test_k1_verify_equals_single_token_decode():
    """k = 1: one query over L cached keys plus its own, written directly."""
    L, Hq, Hkv, D = 50, 4, 4, 32
    c = one_seq_case(L, 1, Hq, Hkv, D, 16)
    out, _, _ = run(c, 0.5)
    for h in range(Hq):
        s = np.array([0.5 * np.dot(c["q"][0, h], c["Kall"][j, h]) for j in range(L + 1)])
        w = np.exp(s - s.max())
        w = w / w.sum()
        ref = sum(w[j] * c["Vall"][j, h] for j in range(L + 1))
        np.testing.assert_allclose(out[0, h], ref, rtol=1e-12, atol=1e-13)


def test_paged_equals_contiguous_and_page_permutation_invariant():
    rng1 = np.random.default_rng(7)
    rng2 = np.random.default_rng(7)
    a = one_seq_case(70, 5, 4, 2, 32, 16, rng=rng1, permute=False)
    b = one_seq_case(70, 5, 4, 2, 32, 16, rng=rng2, permute=True)
    assert not np.array_equal(a["pt"], b["pt"])
    oa, _, _ = run(a, 0.25)
    ob, _, _ = run(b, 0.25)
    np.testing.assert_array_equal(oa, ob)


def test_gqa_equals_mha_with_repeated_kv_heads():
    L, k, Hq, Hkv, D = 31, 4, 8, 2, 32
    c = one_seq_case(L, k, Hq, Hkv, D, 16)
    out, _, _ = run(c, 0.25)
    G = Hq // Hkv
    m = dict(c)
    m["Kall"] = np.repeat(c["Kall"], G, axis=1)
    m["Vall"] = np.repeat(c["Vall"], G, axis=1)
    need = -(-(L + k) // 16)
    m["kc"], m["vc"] = build_paged(m["Kall"][:L], m["Vall"][:L], 16, c["kc"].shape[0],
                                   c["pt"][0][:need])
    m["k_new"], m["v_new"] = m["Kall"][L:], m["Vall"][L:]
    out_mha, _, _ = run(m, 0.25)
    np.testing.assert_allclose(out, out_mha, rtol=1e-12, atol=1e-13)


def test_eviction_recompute_equals_cached_verify():
    """A preempted request recomputes its whole prefix (Section 3.2.3): a
    from-scratch pass with no cached tokens over all L+k rows must give the
    cached verify's k rows as its last k rows."""
    L, k, Hq, Hkv, D, ps = 23, 4, 4, 2, 32, 16
    c = one_seq_case(L, k, Hq, Hkv, D, ps)
    rng = np.random.default_rng(99)
    q_prefix = rng.standard_normal((L, Hq, D))
    cached, _, _ = run(c, 0.25)
    full_q = np.concatenate([q_prefix, c["q"]])
    kc = np.full_like(c["kc"], np.nan)
    vc = np.full_like(c["vc"], np.nan)
    out, _, _ = oracle.verify_attn_paged(full_q, c["Kall"], c["Vall"], kc, vc, c["pt"],
                                         np.array([0]), np.array([0, L + k]), 0.25)
    np.testing.assert_allclose(out[L:], cached, rtol=1e-12, atol=1e-13)


def test_seq_ids_subset_and_multi_sequence_rows():
    rng = np.random.default_rng(5)
    Hq, Hkv, D, ps = 4, 2, 32, 16
    Ls, ks = [10, 0, 33], [3, 2, 1]
    cu = np.concatenate([[0], np.cumsum(ks)])
    T = cu[-1]
    q = rng.standard_normal((T, Hq, D))
    kn = rng.standard_normal((T, Hkv, D))
    vn = rng.standard_normal((T, Hkv, D))
    npg = 20
    kc = rng.standard_normal((npg, Hkv, D // 32, ps, 32))
    vc = rng.standard_normal((npg, Hkv, D, ps))
    pt = np.array([[3, 4, 19], [5, 19, 19], [6, 7, 8]])
    full, _, _ = oracle.verify_attn_paged(q, kn, vn, kc, vc, pt, np.array(Ls), cu, 0.3)
    sub, kc2, _ = oracle.verify_attn_paged(q, kn, vn, kc, vc, pt, np.array(Ls), cu, 0.3,
                                           seq_ids=[2, 0])
    np.testing.assert_array_equal(sub[cu[0]:cu[1]], full[cu[0]:cu[1]])
    np.testing.assert_array_equal(sub[cu[2]:cu[3]], full[cu[2]:cu[3]])
    assert np.all(sub[cu[1]:cu[2]] == 0)
    # sequence 1 was not in the subset: its window was not appended
    np.testing.assert_array_equal(kc2[5], kc[5])
    for b in range(3):
        K, V = oracle.gather_sequence(*oracle.verify_attn_paged(
            q, kn, vn, kc, vc, pt, np.array(Ls), cu, 0.3)[1:], pt, b, Ls[b] + ks[b])
        ref = sdpa_reference(q[cu[b]:cu[b + 1]], K, V, Ls[b], 0.3)
        np.testing.assert_allclose(full[cu[b]:cu[b + 1]], ref, rtol=1e-12, atol=1e-12)


def test_large_scores_stay_finite_and_match_shifted_case():
    """Softmax is shift-invariant: adding a constant to every score of a row
    (here via a shared key component the query projects onto strongly) must
    not change the output, even when exp of the raw scores would overflow."""
    L, k, D = 12, 2, 32
    c = one_seq_case(L, k, 1, 1, D, 16)
    c["q"][:] = 0.0
    c["q"][:, :, 0] = 1.0
    base, _, _ = run(c, 1.0)
    shifted = dict(c)
    shifted["kc"] = c["kc"].copy()
    shifted["kc"][:, :, 0, :, 0] += 5000.0
    shifted["k_new"] = c["k_new"].copy()
    shifted["k_new"][:, :, 0] += 5000.0
    out, _, _ = run(shifted, 1.0)
    assert np.all(np.isfinite(out))
    np.testing.assert_allclose(out, base, rtol=1e-9, atol=1e-9)
