"""Pins of the oracle's verdict stage (Eq. (9) over a window).

* hand-derived golden windows (tests/golden/eq9_windows.txt);
* brute force over every window, driver, coverage pattern and EOS position on
  tiny vocabularies: the windowed scan equals the token-by-token Eq. (9)
  stepper, a separate writing of the rule;
* the bridge special cases of Section 3.2.2 (pure on-policy / off-policy);
* invariants over random batches.
"""
import itertools
import os

import numpy as np
import pytest

import oracle
from oracle import DRIVER_S, DRIVER_T, SRC_DISCARDED, SRC_S, SRC_T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "eq9_windows.txt")
EOS = 7
OTHER = 5     # a token that is never a draft below


def window_case(covered, eos_row, drv):
    """Drafts 1..k (EOS at eos_row) and top-K lists realising ``covered``."""
    k = len(covered)
    drafts = [10 + i for i in range(k)]
    if eos_row >= 0:
        drafts[eos_row] = EOS
    topk = [[drafts[i], OTHER] if covered[i] else [OTHER, 99] for i in range(k)]
    return drafts, topk


def scan_one(drafts, topk, K, drv, L, seq_len, max_len):
    k = len(drafts)
    return oracle.accept_scan(np.array([0, k]), np.array(drafts, np.int64),
                              np.array(topk, np.int64).reshape(k, -1), K,
                              np.array([drv]), np.array([L]), np.array([seq_len]),
                              EOS, max_len)


def load_golden():
    cases = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        f = line.split()
        cases.append(dict(drv=DRIVER_S if f[0] == "S" else DRIVER_T,
                          covered=[c == "1" for c in f[1]], eos=int(f[2]), room=int(f[3]),
                          n_acc=int(f[4]), event=int(f[5]),
                          next=DRIVER_S if f[6] == "S" else DRIVER_T, fin=int(f[7]),
                          cache=int(f[8]),
                          src=[{"S": SRC_S, "T": SRC_T, "-": SRC_DISCARDED}[c] for c in f[9]]))
    return cases


GOLDEN_CASES = load_golden()


@pytest.mark.parametrize("case", GOLDEN_CASES, ids=[str(i) for i in range(len(GOLDEN_CASES))])
def test_golden_windows(case):
    drafts, topk = window_case(case["covered"], case["eos"], case["drv"])
    seq_len = 1000
    r = scan_one(drafts, topk, 2, case["drv"], 100, seq_len, seq_len + case["room"])
    assert r["n_acc"][0] == case["n_acc"]
    assert r["event_row"][0] == case["event"]
    assert r["next_driver"][0] == case["next"]
    assert r["finished"][0] == case["fin"]
    assert r["new_cache_len"][0] == case["cache"]
    assert list(r["src"]) == case["src"]


def test_golden_file_covers_all_four_transition_cases():
    seen = set()
    for c in GOLDEN_CASES:
        for i, cov in enumerate(c["covered"]):
            if c["src"][i] == SRC_DISCARDED and not (c["drv"] == DRIVER_S and not cov):
                continue
            seen.add((c["drv"], cov))
    assert seen == {(DRIVER_S, True), (DRIVER_S, False), (DRIVER_T, True), (DRIVER_T, False)}


def stepper_verdict(drafts, topk, K, drv, L, room):
    xs, zs, m, fin = oracle.eq9_stepper(drafts, topk, K, drv, EOS, room)
    takeover = len(xs) > 0 and xs[-1] == oracle.REPLACEMENT
    n_acc = len(xs) - (1 if takeover else 0)
    event = len(xs) - 1 if m != drv else -1
    src = [SRC_DISCARDED] * len(drafts)
    for i in range(n_acc):
        src[i] = zs[i]
    return dict(n_acc=n_acc, event=event, next=m, fin=int(fin),
                cache=L + n_acc + (1 if takeover else 0), src=src)


@pytest.mark.parametrize("V", [3, 5])
def test_brute_force_tiny_vocab_scan_equals_eq9_stepper(V):
    """Every window of length <= 3 over a V-token vocabulary, every top-K set
    family (K in {0, 1, 2, V}), both drivers, EOS = token 0, several rooms."""
    eos = 0
    rng = np.random.default_rng(3)
    n = 0
    for k in range(1, 4):
        for drafts in itertools.product(range(V), repeat=k):
            for K in (0, 1, 2, V):
                # a random top-K list per row (distinct tokens)
                topk = [list(rng.permutation(V)[: max(K, 1)]) for _ in range(k)]
                for drv in (DRIVER_S, DRIVER_T):
                    for room in (0, 1, k, 99):
                        r = oracle.accept_scan(np.array([0, k]), np.array(drafts),
                                               np.array(topk), K, np.array([drv]),
                                               np.array([50]), np.array([10]), eos, 10 + room)
                        xs, zs, m, fin = oracle.eq9_stepper(list(drafts), topk, K, drv, eos, room)
                        takeover = len(xs) > 0 and xs[-1] == oracle.REPLACEMENT
                        n_acc = len(xs) - (1 if takeover else 0)
                        assert r["n_acc"][0] == n_acc
                        assert r["next_driver"][0] == m
                        assert r["finished"][0] == int(fin)
                        assert r["event_row"][0] == (len(xs) - 1 if m != drv else -1)
                        assert r["new_cache_len"][0] == 50 + n_acc + (1 if takeover else 0)
                        assert list(r["src"][:n_acc]) == zs[:n_acc]
                        assert all(s == SRC_DISCARDED for s in r["src"][n_acc:])
                        n += 1
    assert n > 1000


def test_bridge_pure_on_policy_when_control_never_transfers():
    """K >= V: every student draft is covered, the teacher never takes over:
    a purely student-generated trajectory (on-policy distillation)."""
    k, V = 6, 4
    drafts = [1, 3, 2, 2, 1, 3]
    topk = [list(range(V))] * k
    r = scan_one(drafts, topk, V, DRIVER_S, 40, 1, 10**6)
    assert r["n_acc"][0] == k and r["event_row"][0] == -1
    assert r["next_driver"][0] == DRIVER_S
    assert all(s == SRC_S for s in r["src"])


def test_bridge_off_policy_when_first_student_draft_rejected_and_never_handed_back():
    """K = 0: nothing is covered.  Driver S: the first student draft is
    rejected (takeover at row 0).  Driver T then never hands back: the teacher
    keeps every draft (off-policy distillation on teacher trajectories)."""
    drafts = [1, 2, 3, 4]
    topk = [[0]] * 4
    r = scan_one(drafts, topk, 0, DRIVER_S, 40, 1, 10**6)
    assert r["n_acc"][0] == 0 and r["event_row"][0] == 0 and r["next_driver"][0] == DRIVER_T
    r = scan_one(drafts, topk, 0, DRIVER_T, 40, 1, 10**6)
    assert r["n_acc"][0] == 4 and r["event_row"][0] == -1 and r["next_driver"][0] == DRIVER_T
    assert all(s == SRC_T for s in r["src"])


def test_random_batch_invariants():
    rng = np.random.default_rng(11)
    B, V, K = 200, 12, 3
    ks = rng.integers(1, 9, size=B)
    cu = np.concatenate([[0], np.cumsum(ks)])
    T = cu[-1]
    prop = rng.integers(0, V, size=T)
    topk = np.array([rng.permutation(V)[:K] for _ in range(T)])
    drv = rng.integers(0, 2, size=B)
    ctx = rng.integers(0, 500, size=B)
    sl = ctx + 1
    maxl = sl + rng.integers(0, 10, size=B)
    r = oracle.accept_scan(cu, prop, topk, K, drv, ctx, sl, 0, 0)  # max_len 0: all finished
    assert np.all(r["n_acc"] == 0) and np.all(r["finished"] == 1)
    for b in range(B):
        rb = oracle.accept_scan(cu[b:b + 2] - cu[b], prop[cu[b]:cu[b + 1]],
                                topk[cu[b]:cu[b + 1]], K, drv[b:b + 1], ctx[b:b + 1],
                                sl[b:b + 1], 0, int(maxl[b]))
        n = rb["n_acc"][0]
        assert 0 <= n <= ks[b]
        assert ctx[b] <= rb["new_cache_len"][0] <= ctx[b] + ks[b]
        src = rb["src"]
        want = SRC_S if drv[b] == DRIVER_S else SRC_T
        assert np.all(src[:n] == want) and np.all(src[n:] == SRC_DISCARDED)
        if rb["event_row"][0] >= 0:
            assert rb["next_driver"][0] != drv[b]
            e = rb["event_row"][0]
            assert n == (e if drv[b] == DRIVER_S else e + 1)
