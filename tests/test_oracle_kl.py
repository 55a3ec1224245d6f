"""Pins of the oracle's source-split KL values (Eqs. (5), (6), (10), (11)).

* hand-worked values for every support (tests/golden/kl_worked.txt);
* the two-token closed form (Bernoulli KL);
* K = V: every support is the whole vocabulary, renormalisation is the
  identity, and both directions equal scipy's full-vocabulary KL;
* zero for identical models, non-negativity, invariance to logit shifts;
* the loss variants and the bridges of Section 3.2.2 (all student tokens:
  reverse KL everywhere; all teacher tokens: forward KL);
* the list form (top-K lists plus gathered log-probs) equals the full form;
* the per-trajectory mean of Eq. (11) and the intervention ratio.
"""
import math
import os
import re
from fractions import Fraction

import numpy as np
import pytest
from scipy.stats import entropy as scipy_kl

import oracle
from oracle import SRC_DISCARDED, SRC_S, SRC_T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "kl_worked.txt")
SUPPORTS = {"union": oracle.SUPPORT_UNION, "student": oracle.SUPPORT_STUDENT,
            "teacher": oracle.SUPPORT_TEACHER, "intersection": oracle.SUPPORT_INTERSECTION}


def _value(expr):
    """Sum of terms a/b*ln(c/d)."""
    if expr == "0":
        return 0.0
    total = 0.0
    for term in expr.split("+"):
        m = re.fullmatch(r"(\d+)/(\d+)\*ln\((\d+)/(\d+)\)", term)
        assert m, term
        a, b, c, d = (int(x) for x in m.groups())
        total += a / b * math.log(c / d)
    return total


def load_golden():
    cases, cur = [], None
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        f = line.split()
        if f[0] == "case":
            kv = dict(x.split("=") for x in f[2:])
            cur = dict(name=f[1], pi=[float(x) for x in kv["pi"].split(",")],
                       q=[float(x) for x in kv["q"].split(",")], K=int(kv["K"]),
                       overlap=float(Fraction(kv["overlap"])), rows={})
            cases.append(cur)
        else:
            kv = dict(x.split("=") for x in f[1:])
            cur["rows"][f[0]] = (_value(kv["rev"]), _value(kv["fwd"]))
    return cases


GOLDEN_CASES = load_golden()


@pytest.mark.parametrize("case", GOLDEN_CASES, ids=[c["name"] for c in GOLDEN_CASES])
def test_hand_worked_values(case):
    lps = np.log(np.array([case["pi"]]))
    lpt = np.log(np.array([case["q"]]))
    for name, (rev, fwd) in case["rows"].items():
        r = oracle.source_split_kl(lps, lpt, case["K"], [SRC_S], support=SUPPORTS[name])
        assert r["kl_rev"][0] == pytest.approx(rev, abs=1e-12), name
        assert r["kl_fwd"][0] == pytest.approx(fwd, abs=1e-12), name
        assert r["overlap"][0] == pytest.approx(case["overlap"])
    assert set(case["rows"]) == set(SUPPORTS)


def test_two_token_closed_form():
    # V = 2, K = 1, distinct argmaxes: the union is both tokens
    p, q = 0.7, 0.35                     # P(token 0) under pi and q
    lps = np.log([[p, 1 - p]])
    lpt = np.log([[q, 1 - q]])
    rev = p * math.log(p / q) + (1 - p) * math.log((1 - p) / (1 - q))
    fwd = q * math.log(q / p) + (1 - q) * math.log((1 - q) / (1 - p))
    r = oracle.source_split_kl(lps, lpt, 1, [SRC_T])
    assert r["kl_rev"][0] == pytest.approx(rev, abs=1e-13)
    assert r["kl_fwd"][0] == pytest.approx(fwd, abs=1e-13)
    assert r["loss"][0] == pytest.approx(fwd, abs=1e-13)     # z = T: forward KL


def _logsoftmax(x):
    x = np.asarray(x, np.float64)
    m = x.max(axis=-1, keepdims=True)
    return x - m - np.log(np.exp(x - m).sum(axis=-1, keepdims=True))


def test_full_vocabulary_support_equals_scipy_kl():
    rng = np.random.default_rng(0)
    M, V = 6, 11
    lps = _logsoftmax(rng.normal(size=(M, V)) * 1.3)
    lpt = _logsoftmax(rng.normal(size=(M, V)) * 0.8)
    for support in SUPPORTS.values():
        r = oracle.source_split_kl(lps, lpt, V, [SRC_S] * M, support=support)
        for m in range(M):
            p, q = np.exp(lps[m]), np.exp(lpt[m])
            assert r["kl_rev"][m] == pytest.approx(scipy_kl(p, q), abs=1e-12)
            assert r["kl_fwd"][m] == pytest.approx(scipy_kl(q, p), abs=1e-12)
            assert r["overlap"][m] == 1.0


def test_identical_models_give_zero_and_values_are_nonnegative():
    rng = np.random.default_rng(1)
    M, V, K = 20, 50, 8
    lps = _logsoftmax(rng.normal(size=(M, V)) * 2)
    r = oracle.source_split_kl(lps, lps, K, [SRC_S] * M)
    assert np.all(np.abs(r["kl_rev"]) < 1e-14) and np.all(np.abs(r["kl_fwd"]) < 1e-14)
    assert np.all(r["overlap"] == 1.0)
    lpt = _logsoftmax(rng.normal(size=(M, V)) * 2)
    for support in SUPPORTS.values():
        r = oracle.source_split_kl(lps, lpt, K, [SRC_S] * M, support=support)
        assert np.all(r["kl_rev"] >= -1e-15) and np.all(r["kl_fwd"] >= -1e-15)


def test_shift_invariance():
    """Eq. (6) renormalises: adding a constant per row to either model's
    log-probs (unnormalised logits) changes nothing."""
    rng = np.random.default_rng(2)
    M, V, K = 10, 40, 5
    ls, lt = rng.normal(size=(M, V)), rng.normal(size=(M, V))
    a = oracle.source_split_kl(_logsoftmax(ls), _logsoftmax(lt), K, [SRC_T] * M)
    b = oracle.source_split_kl(ls + 7.25, lt - 3.5, K, [SRC_T] * M)
    for key in ("kl_rev", "kl_fwd", "loss", "overlap"):
        np.testing.assert_allclose(a[key], b[key], atol=1e-12)


def test_loss_modes_and_bridges():
    rng = np.random.default_rng(3)
    M, V, K = 12, 30, 4
    lps = _logsoftmax(rng.normal(size=(M, V)))
    lpt = _logsoftmax(rng.normal(size=(M, V)))
    src = np.array([SRC_S, SRC_T, SRC_DISCARDED] * 4)
    base = oracle.source_split_kl(lps, lpt, K, src)
    rev, fwd = base["kl_rev"], base["kl_fwd"]
    want = {oracle.LOSS_IPD_SPLIT: np.where(src == SRC_S, rev, fwd),
            oracle.LOSS_PURE_REVERSE: rev, oracle.LOSS_PURE_FORWARD: fwd,
            oracle.LOSS_INVERSE_SPLIT: np.where(src == SRC_S, fwd, rev)}
    for mode, w in want.items():
        r = oracle.source_split_kl(lps, lpt, K, src, loss_mode=mode)
        np.testing.assert_allclose(r["loss"], np.where(src == SRC_DISCARDED, 0.0, w), atol=0)
    # bridges: a pure student trajectory gets reverse KL (top-K on-policy
    # distillation), a pure teacher trajectory forward KL (off-policy)
    cu = np.array([0, M])
    on = oracle.source_split_kl(lps, lpt, K, [SRC_S] * M, cu=cu)
    assert on["seq_loss"][0] == pytest.approx(rev.mean()) and on["t_ratio"][0] == 0.0
    off = oracle.source_split_kl(lps, lpt, K, [SRC_T] * M, cu=cu)
    assert off["seq_loss"][0] == pytest.approx(fwd.mean()) and off["t_ratio"][0] == 1.0


def test_length_normalised_segments():
    rng = np.random.default_rng(4)
    V, K = 20, 3
    src = np.array([SRC_S, SRC_T, SRC_DISCARDED, SRC_S, SRC_DISCARDED, SRC_DISCARDED, SRC_T])
    M = len(src)
    lps = _logsoftmax(rng.normal(size=(M, V)))
    lpt = _logsoftmax(rng.normal(size=(M, V)))
    cu = np.array([0, 4, 6, 7, 7])          # segments of 4, 2 (all discarded), 1, 0 rows
    r = oracle.source_split_kl(lps, lpt, K, src, cu=cu)
    rev, fwd = r["kl_rev"], r["kl_fwd"]
    assert r["seq_loss"][0] == pytest.approx((rev[0] + fwd[1] + rev[3]) / 3)
    assert r["t_ratio"][0] == pytest.approx(1 / 3)
    assert r["seq_loss"][1] == 0.0 and r["t_ratio"][1] == 0.0
    assert r["seq_loss"][2] == pytest.approx(fwd[6]) and r["t_ratio"][2] == 1.0
    assert r["seq_loss"][3] == 0.0


@pytest.mark.parametrize("support", list(SUPPORTS.values()))
def test_list_form_equals_full_form(support):
    """The GPU path sees each model's top-K lists and gathered log-probs, not
    full rows; built from full rows, the list form must agree exactly."""
    rng = np.random.default_rng(10 + support)
    M, V, K = 25, 60, 6
    ls = rng.normal(size=(M, V)) * 1.5
    lt = ls * 0.6 + rng.normal(size=(M, V))     # correlated: partial overlaps
    lps, lpt = _logsoftmax(ls), _logsoftmax(lt)
    src = rng.choice([SRC_S, SRC_T, SRC_DISCARDED], size=M)
    s_idx = np.array([np.argsort(-lps[m], kind="stable")[:K] for m in range(M)])
    t_idx = np.array([np.argsort(-lpt[m], kind="stable")[:K] for m in range(M)])
    take = lambda lp, idx: np.take_along_axis(lp, idx, axis=1)
    cu = np.array([0, 10, 25])
    a = oracle.source_split_kl(lps, lpt, K, src, support=support, cu=cu)
    b = oracle.source_split_kl_lists(s_idx, take(lps, s_idx), take(lps, t_idx), t_idx,
                                     take(lpt, t_idx), take(lpt, s_idx), src, support=support,
                                     cu=cu)
    for key in a:
        np.testing.assert_allclose(a[key], b[key], atol=1e-13, err_msg=key)
    assert 0 < np.mean(a["overlap"]) < 1


def test_logp_gather_matches_log_softmax():
    rng = np.random.default_rng(5)
    h = rng.normal(size=(3, 16))
    W = rng.normal(size=(40, 16)) * 0.3
    l = h @ W.T
    ref = _logsoftmax(l)
    idx = np.array([[0, 39, 5], [7, 7, -1], [40, 2, 3]])
    g = oracle.logp_gather(h, W, idx)
    for m in range(3):
        for j in range(3):
            v = idx[m, j]
            if 0 <= v < 40:
                assert g[m, j] == pytest.approx(ref[m, v], abs=1e-12)
            else:
                assert g[m, j] == -np.inf
