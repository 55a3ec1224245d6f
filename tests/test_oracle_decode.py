"""Pins of the oracle's proposer decode steps (Section 3.2.3, propose stage).

* gamma one-row decode steps give the same attention outputs and caches as
  one gamma-row verification window over the same positions (the engine's
  verifier scores, in one prefill pass, exactly the positions the proposer
  decoded one at a time);
* each step's LM-head outputs are those of the step's hidden rows;
* the draw is the inverse CDF of the step's distribution: a peaked
  distribution gives its mode for every u, and tokens are non-decreasing in
  u for fixed logits;
* handled sequences only: others' caches stay untouched.
"""
import numpy as np
import pytest

import oracle
from tests.test_oracle_attention import build_paged


def _batch(rng, B, Hq, Hkv, D, ps, lens, gamma, Hd, V):
    need = [-(-(L + gamma) // ps) for L in lens]
    num_pages = sum(need) + 3
    perm = rng.permutation(num_pages - 1)
    pt = np.full((B, max(need) + 1), num_pages - 1, np.int64)
    kc = np.full((num_pages, Hkv, D // 32, ps, 32), np.nan)
    vc = np.full((num_pages, Hkv, D, ps), np.nan)
    o = 0
    for b in range(B):
        pt[b, :need[b]] = perm[o:o + need[b]]
        o += need[b]
        Kb = rng.standard_normal((lens[b], Hkv, D))
        Vb = rng.standard_normal((lens[b], Hkv, D))
        k1, v1 = build_paged(Kb, Vb, ps, num_pages, pt[b])
        mask = ~np.isnan(k1)
        kc[mask] = k1[mask]
        mask = ~np.isnan(v1)
        vc[mask] = v1[mask]
    W = rng.standard_normal((V, Hd)) * 0.3
    steps = [dict(q=rng.standard_normal((B, Hq, D)), k_new=rng.standard_normal((B, Hkv, D)),
                  v_new=rng.standard_normal((B, Hkv, D)), hidden=rng.standard_normal((B, Hd)),
                  u=rng.random(B)) for _ in range(gamma)]
    return kc, vc, pt, W, steps


def test_decode_steps_equal_one_verification_window():
    rng = np.random.default_rng(0)
    B, Hq, Hkv, D, ps, gamma, Hd, V = 3, 4, 2, 32, 16, 5, 16, 50
    lens = np.array([13, 40, 1])
    kc, vc, pt, W, steps = _batch(rng, B, Hq, Hkv, D, ps, lens, gamma, Hd, V)
    res, kd, vd = oracle.propose_decode(steps, kc, vc, pt, lens, 0.3, W, 4)
    # the same positions as one gamma-row window per sequence
    q = np.stack([steps[i]["q"][b] for b in range(B) for i in range(gamma)])
    kn = np.stack([steps[i]["k_new"][b] for b in range(B) for i in range(gamma)])
    vn = np.stack([steps[i]["v_new"][b] for b in range(B) for i in range(gamma)])
    cu = np.arange(B + 1) * gamma
    win, kw, vw = oracle.verify_attn_paged(q, kn, vn, kc, vc, pt, lens, cu, 0.3)
    np.testing.assert_array_equal(np.isnan(kd), np.isnan(kw))
    np.testing.assert_array_equal(kd[~np.isnan(kd)], kw[~np.isnan(kw)])
    np.testing.assert_array_equal(vd[~np.isnan(vd)], vw[~np.isnan(vw)])
    for i in range(gamma):
        for b in range(B):
            np.testing.assert_allclose(res[i]["out"][b], win[b * gamma + i], rtol=1e-12, atol=1e-13)


def test_steps_score_their_hidden_rows_and_draw_by_inverse_cdf():
    rng = np.random.default_rng(1)
    B, Hq, Hkv, D, ps, gamma, Hd, V = 4, 2, 2, 32, 16, 3, 8, 30
    lens = np.array([5, 17, 33, 2])
    kc, vc, pt, W, steps = _batch(rng, B, Hq, Hkv, D, ps, lens, gamma, Hd, V)
    # step 1: a peaked distribution per row (mode = 7 + b) -> the mode for any u
    for b in range(B):
        W[7 + b] = 60.0 * steps[1]["hidden"][b] / np.dot(steps[1]["hidden"][b], steps[1]["hidden"][b])
    res, _, _ = oracle.propose_decode(steps, kc, vc, pt, lens, 0.2, W, 5)
    for j in range(gamma):
        l = steps[j]["hidden"] @ W.T
        ref = oracle.lmhead_logsoftmax(steps[j]["hidden"], W, np.zeros(B, np.int64), 5)
        np.testing.assert_allclose(res[j]["lm"]["lse"], ref["lse"], rtol=1e-13)
        np.testing.assert_array_equal(res[j]["lm"]["topk_idx"], ref["topk_idx"])
        np.testing.assert_allclose(res[j]["logits"], l, rtol=1e-12, atol=1e-12)
    # hidden[b] . W[7+b] = 60 while every other logit of that row is far lower
    assert list(res[1]["token"]) == [7, 8, 9, 10]
    # inverse CDF: tokens are non-decreasing in u for fixed logits
    l0 = res[0]["logits"][0]
    toks = [oracle.sample_categorical(l0, u)[0] for u in np.linspace(0, 0.999, 200)]
    assert toks == sorted(toks)


def test_only_handled_sequences_are_touched():
    rng = np.random.default_rng(2)
    B, Hq, Hkv, D, ps, gamma, Hd, V = 4, 2, 1, 32, 16, 2, 8, 20
    lens = np.array([9, 10, 11, 12])
    kc, vc, pt, W, steps = _batch(rng, B, Hq, Hkv, D, ps, lens, gamma, Hd, V)
    sub = [dict((k, v[[1, 3]]) for k, v in st.items()) for st in steps]
    res, kd, vd = oracle.propose_decode(sub, kc, vc, pt, lens, 0.2, W, 3, seq_ids=[1, 3])
    for b in (0, 2):                       # untouched pages
        for p in pt[b]:
            if p != pt.max():
                np.testing.assert_array_equal(np.isnan(kd[p]), np.isnan(kc[p]))
    with pytest.raises(ValueError):
        oracle.propose_decode(sub, kc, vc, pt, lens, 0.2, W, 3, seq_ids=[3, 1])
