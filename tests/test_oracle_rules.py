"""Pins of the oracle's rule variants (Section 3.2.1, after Eq. (9)):
entropy-threshold takeover and handback, asymmetric rules, and SKD's fixed
one-token handback (Section 2).

* hand-derived golden windows (tests/golden/rule_variants.txt);
* the entropy rules reduce to the coverage rules when the entropy is the
  indicator of an uncovered draft and the threshold lies between 0 and 1;
* under SKD the teacher never drives a window, and each of its tokens sits
  where a student draft was rejected;
* brute force over tiny windows: the windowed scan equals the token-by-token
  Eq. (9) stepper under every rule pair.
"""
import itertools
import math
import os

import numpy as np
import pytest

import oracle
from oracle import DRIVER_S, DRIVER_T, SRC_DISCARDED, SRC_S, SRC_T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "rule_variants.txt")
EOS = 7
OTHER = 5


def _rule(tok):
    """'C' / 'F' / 'E<tau>' -> (kind, tau)."""
    if tok == "C":
        return "C", 0.0
    if tok == "F":
        return "F", 0.0
    return "E", float(tok[1:])


def load_golden():
    cases = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        f = line.split()
        tk, tt = _rule(f[0])
        hk, ht = _rule(f[1])
        cases.append(dict(
            take=oracle.TAKE_COVERAGE if tk == "C" else oracle.TAKE_ENTROPY, tau_take=tt,
            hand={"C": oracle.HAND_COVERAGE, "F": oracle.HAND_FIXED_ONE,
                  "E": oracle.HAND_ENTROPY}[hk], tau_hand=ht,
            drv=DRIVER_S if f[2] == "S" else DRIVER_T,
            covered=[c == "1" for c in f[3]], ent=[float(x) for x in f[4].split(",")],
            eos=int(f[5]), room=int(f[6]), n_acc=int(f[7]), event=int(f[8]),
            next=DRIVER_S if f[9] == "S" else DRIVER_T, fin=int(f[10]), cache=int(f[11]),
            src=[{"S": SRC_S, "T": SRC_T, "-": SRC_DISCARDED}[c] for c in f[12]]))
    return cases


GOLDEN_CASES = load_golden()


def window_case(covered, eos_row):
    k = len(covered)
    drafts = [10 + i for i in range(k)]
    if eos_row >= 0:
        drafts[eos_row] = EOS
    topk = [[drafts[i], OTHER] if covered[i] else [OTHER, 99] for i in range(k)]
    return drafts, topk


@pytest.mark.parametrize("case", GOLDEN_CASES, ids=[str(i) for i in range(len(GOLDEN_CASES))])
def test_golden_rule_windows(case):
    drafts, topk = window_case(case["covered"], case["eos"])
    k = len(drafts)
    assert len(case["ent"]) == k and len(case["src"]) == k
    r = oracle.accept_scan(np.array([0, k]), np.array(drafts), np.array(topk), 2,
                           np.array([case["drv"]]), np.array([100]), np.array([1000]), EOS,
                           1000 + case["room"], take_rule=case["take"], hand_rule=case["hand"],
                           ent=np.array(case["ent"]), tau_take=case["tau_take"],
                           tau_hand=case["tau_hand"])
    assert r["n_acc"][0] == case["n_acc"]
    assert r["event_row"][0] == case["event"]
    assert r["next_driver"][0] == case["next"]
    assert r["finished"][0] == case["fin"]
    assert r["new_cache_len"][0] == case["cache"]
    assert list(r["src"]) == case["src"]


def test_golden_file_covers_every_rule():
    kinds = {(c["take"], c["hand"]) for c in GOLDEN_CASES}
    assert {t for t, _ in kinds} == {oracle.TAKE_COVERAGE, oracle.TAKE_ENTROPY}
    assert {h for _, h in kinds} == {oracle.HAND_COVERAGE, oracle.HAND_FIXED_ONE,
                                     oracle.HAND_ENTROPY}


def _random_batch(rng, B, V, K):
    ks = rng.integers(1, 12, size=B)
    cu = np.concatenate([[0], np.cumsum(ks)])
    T = int(cu[-1])
    prop = rng.integers(0, V, size=T)
    topk = np.array([rng.permutation(V)[:K] for _ in range(T)])
    drv = rng.integers(0, 2, size=B)
    ctx = rng.integers(0, 500, size=B)
    sl = ctx + 1
    maxl = sl + rng.integers(0, 14, size=B)
    return cu, prop, topk, drv, ctx, sl, maxl


def test_entropy_rules_reduce_to_coverage():
    """ent = 1 for an uncovered draft, 0 for a covered one, thresholds in
    (0, 1): 'ent > tau' is 'uncovered' and 'ent <= tau' is 'covered', so every
    entropy/coverage rule pair gives the coverage verdict."""
    rng = np.random.default_rng(21)
    B, V, K = 300, 9, 3
    cu, prop, topk, drv, ctx, sl, maxl = _random_batch(rng, B, V, K)
    unc = np.array([0.0 if prop[r] in topk[r] else 1.0 for r in range(len(prop))])
    ref = oracle.accept_scan(cu, prop, topk, K, drv, ctx, sl, 3, maxl.max())
    for take, hand in [(oracle.TAKE_ENTROPY, oracle.HAND_COVERAGE),
                       (oracle.TAKE_COVERAGE, oracle.HAND_ENTROPY),
                       (oracle.TAKE_ENTROPY, oracle.HAND_ENTROPY)]:
        for tau in (0.25, 0.5, 0.999):
            r = oracle.accept_scan(cu, prop, topk, K, drv, ctx, sl, 3, maxl.max(),
                                   take_rule=take, hand_rule=hand, ent=unc, tau_take=tau,
                                   tau_hand=tau)
            for key in ref:
                assert np.array_equal(r[key], ref[key]), (take, hand, tau, key)
    # a threshold outside (0, 1) breaks the equivalence in a known direction:
    # tau_take = 1 never takes over
    r = oracle.accept_scan(cu, prop, topk, K, drv, ctx, sl, 3, 10**9,
                           take_rule=oracle.TAKE_ENTROPY, ent=unc, tau_take=1.0)
    s_rows = drv == DRIVER_S
    assert np.all(r["event_row"][s_rows] == -1)


def test_skd_teacher_never_drives_and_only_replaces_rejected_drafts():
    """A long rollout, window by window, under coverage takeover and fixed
    one-token handback (SKD).  From m_1 = S the driver stays S, and every
    teacher token is a replacement at a rejected student draft: one teacher
    token per takeover, each followed by the student's own proposal (two
    teacher tokens are adjacent only when that next draft is rejected too)."""
    rng = np.random.default_rng(5)
    V, K = 6, 2
    z = []
    rejected_positions = []
    drv = DRIVER_S
    pos = 0
    for _ in range(400):
        k = int(rng.integers(1, 7))
        prop = rng.integers(0, V, size=k)
        topk = np.array([rng.permutation(V)[:K] for _ in range(k)])
        r = oracle.accept_scan(np.array([0, k]), prop, topk, K, np.array([drv]),
                               np.array([pos]), np.array([pos]), -1, 10**9,
                               hand_rule=oracle.HAND_FIXED_ONE)
        assert drv == DRIVER_S
        n = int(r["n_acc"][0])
        z += [SRC_S] * n
        pos += n
        if r["event_row"][0] >= 0:
            rejected_positions.append(pos)
            z.append(SRC_T)
            pos += 1
        drv = int(r["next_driver"][0])
    zs = "".join("S" if x == SRC_S else "T" for x in z)
    assert "T" in zs and "S" in zs
    assert [i for i, c in enumerate(zs) if c == "T"] == rejected_positions


def test_fixed_one_handback_from_a_teacher_window_keeps_exactly_one_token():
    rng = np.random.default_rng(6)
    for k in range(1, 9):
        prop = rng.integers(0, 9, size=k)
        topk = np.array([rng.permutation(9)[:3] for _ in range(k)])
        r = oracle.accept_scan(np.array([0, k]), prop, topk, 3, np.array([DRIVER_T]),
                               np.array([10]), np.array([10]), -1, 10**9,
                               hand_rule=oracle.HAND_FIXED_ONE)
        assert r["n_acc"][0] == 1 and r["event_row"][0] == 0
        assert r["next_driver"][0] == DRIVER_S and r["new_cache_len"][0] == 11
        assert list(r["src"]) == [SRC_T] + [SRC_DISCARDED] * (k - 1)


RULES = [(oracle.TAKE_COVERAGE, oracle.HAND_COVERAGE), (oracle.TAKE_COVERAGE, oracle.HAND_FIXED_ONE),
         (oracle.TAKE_ENTROPY, oracle.HAND_COVERAGE), (oracle.TAKE_COVERAGE, oracle.HAND_ENTROPY),
         (oracle.TAKE_ENTROPY, oracle.HAND_ENTROPY), (oracle.TAKE_ENTROPY, oracle.HAND_FIXED_ONE)]


@pytest.mark.parametrize("take,hand", RULES)
def test_brute_force_scan_equals_stepper_under_every_rule(take, hand):
    """Every window of length <= 3 over V = 4 (EOS = 0), K in {0, 1, 4}, both
    drivers, several rooms, and entropies drawn from {0.2, 0.5, 0.9, nan}
    (0.5 is the threshold, so ties are exercised)."""
    V, eos = 4, 0
    rng = np.random.default_rng(7)
    n = 0
    for k in range(1, 4):
        for drafts in itertools.product(range(V), repeat=k):
            for K in (0, 1, V):
                topk = [list(rng.permutation(V)[: max(K, 1)]) for _ in range(k)]
                ent = rng.choice([0.2, 0.5, 0.9, math.nan], size=k)
                for drv in (DRIVER_S, DRIVER_T):
                    for room in (0, 1, k, 99):
                        r = oracle.accept_scan(np.array([0, k]), np.array(drafts), np.array(topk),
                                               K, np.array([drv]), np.array([50]),
                                               np.array([10]), eos, 10 + room, take_rule=take,
                                               hand_rule=hand, ent=ent, tau_take=0.5,
                                               tau_hand=0.5)
                        xs, zs, m, fin = oracle.eq9_stepper(list(drafts), topk, K, drv, eos, room,
                                                            take_rule=take, hand_rule=hand,
                                                            ent=ent, tau_take=0.5, tau_hand=0.5)
                        takeover = len(xs) > 0 and xs[-1] == oracle.REPLACEMENT
                        n_acc = len(xs) - (1 if takeover else 0)
                        event = len(xs) - 1 if (takeover or m != drv) else -1
                        assert r["n_acc"][0] == n_acc
                        assert r["next_driver"][0] == m
                        assert r["finished"][0] == int(fin)
                        assert r["event_row"][0] == event
                        assert r["new_cache_len"][0] == 50 + n_acc + (1 if takeover else 0)
                        assert list(r["src"][:n_acc]) == zs[:n_acc]
                        assert all(s == SRC_DISCARDED for s in r["src"][n_acc:])
                        n += 1
    assert n > 1000


def test_entropy_rule_needs_entropies():
    with pytest.raises(ValueError):
        oracle.accept_scan(np.array([0, 1]), np.array([1]), np.array([[1]]), 1,
                           np.array([DRIVER_S]), np.array([0]), np.array([0]), 0, 10,
                           take_rule=oracle.TAKE_ENTROPY)
