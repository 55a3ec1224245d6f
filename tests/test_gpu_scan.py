"""GPU parity of accept_scan (integer work: bit-exact) against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36546_amd import ops
from tests import parity
from tests.test_oracle_scan import GOLDEN_CASES, EOS, window_case
from tests.workload import to_np

pytestmark = pytest.mark.gpu


def _t(a, dt):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dt))).cuda()


def _scan(cu, prop, topk, K, drv, ctx, sl, eos, max_len):
    g = ops.accept_scan(_t(cu, np.int32), _t(prop, np.int32), _t(topk, np.int32) if K > 0 else None,
                        K, _t(drv, np.uint8), _t(ctx, np.int32), _t(sl, np.int32), eos, max_len)
    torch.cuda.synchronize()
    return g


def _compare(g, r):
    for key in ("n_acc", "event_row", "next_driver", "finished", "new_cache_len", "src"):
        np.testing.assert_array_equal(to_np(g[key]).astype(np.int64), r[key], err_msg=key)


def test_golden_windows_on_gpu():
    for case in GOLDEN_CASES:
        drafts, topk = window_case(case["covered"], case["eos"], case["drv"])
        k = len(drafts)
        g = _scan([0, k], drafts, np.array(topk).reshape(k, 2), 2, [case["drv"]], [100], [1000],
                  EOS, 1000 + case["room"])
        assert int(to_np(g["n_acc"])[0]) == case["n_acc"]
        assert int(to_np(g["event_row"])[0]) == case["event"]
        assert int(to_np(g["new_cache_len"])[0]) == case["cache"]
        assert int(to_np(g["finished"])[0]) == case["fin"]
        assert to_np(g["src"]).tolist() == case["src"]


@pytest.mark.parametrize("K,V,kmax", [(16, 40, 16), (0, 10, 8), (32, 33, 4), (1, 3, 80), (4, 6, 130)])
def test_random_batches_bit_exact(K, V, kmax):
    rng = np.random.default_rng(K * 100 + V)
    B = 300
    ks = rng.integers(0, kmax + 1, size=B)
    cu = np.concatenate([[0], np.cumsum(ks)]).astype(np.int64)
    T = int(cu[-1])
    prop = rng.integers(0, V, size=T)
    topk = np.array([rng.permutation(V)[:max(K, 1)] for _ in range(T)])[:, :K] if K > 0 \
        else np.zeros((T, 0), np.int64)
    drv = rng.integers(0, 2, size=B)
    ctx = rng.integers(0, 5000, size=B)
    sl = ctx + 1
    max_len = 2000
    r = oracle.accept_scan(cu, prop, topk, K, drv, ctx, sl, 0, max_len)
    g = _scan(cu, prop, topk, K, drv, ctx, sl, 0, max_len)
    _compare(g, r)


# ---- rule variants (accept_scan_rule) ----

from tests.test_oracle_rules import GOLDEN_CASES as RULE_CASES  # noqa: E402
from tests.test_oracle_rules import window_case as rule_window  # noqa: E402


def _scan_rule(cu, prop, topk, K, drv, ctx, sl, eos, max_len, take, hand, ent, tt, th):
    g = ops.accept_scan_rule(_t(cu, np.int32), _t(prop, np.int32),
                             _t(topk, np.int32) if K > 0 else None, K, _t(drv, np.uint8),
                             _t(ctx, np.int32), _t(sl, np.int32), eos, max_len, take_rule=take,
                             hand_rule=hand, ent=_t(ent, np.float32) if ent is not None else None,
                             tau_take=tt, tau_hand=th)
    torch.cuda.synchronize()
    return g


def test_rule_golden_windows_on_gpu():
    print(f"[scan] {len(RULE_CASES)} rule-variant golden windows", flush=True)
    for case in RULE_CASES:
        drafts, topk = rule_window(case["covered"], case["eos"])
        k = len(drafts)
        g = _scan_rule([0, k], drafts, np.array(topk).reshape(k, 2), 2, [case["drv"]], [100],
                       [1000], EOS, 1000 + case["room"], case["take"], case["hand"], case["ent"],
                       case["tau_take"], case["tau_hand"])
        assert int(to_np(g["n_acc"])[0]) == case["n_acc"], case
        assert int(to_np(g["event_row"])[0]) == case["event"], case
        assert int(to_np(g["next_driver"])[0]) == case["next"], case
        assert int(to_np(g["new_cache_len"])[0]) == case["cache"], case
        assert int(to_np(g["finished"])[0]) == case["fin"], case
        assert to_np(g["src"]).tolist() == case["src"], case


RULE_PAIRS = [(oracle.TAKE_COVERAGE, oracle.HAND_FIXED_ONE), (oracle.TAKE_ENTROPY, oracle.HAND_COVERAGE),
              (oracle.TAKE_COVERAGE, oracle.HAND_ENTROPY), (oracle.TAKE_ENTROPY, oracle.HAND_ENTROPY),
              (oracle.TAKE_ENTROPY, oracle.HAND_FIXED_ONE), (oracle.TAKE_COVERAGE, oracle.HAND_COVERAGE)]


@pytest.mark.parametrize("take,hand", RULE_PAIRS)
@pytest.mark.parametrize("K,kmax", [(16, 16), (4, 130)])
def test_rule_random_batches_bit_exact(take, hand, K, kmax):
    """Random windows up to 130 rows (several 64-row chunks); entropies drawn
    from a few float32 values that include the thresholds themselves (ties)
    and NaN."""
    print(f"[scan] rules take={take} hand={hand} K={K} kmax={kmax}", flush=True)
    rng = np.random.default_rng(1000 + 10 * take + hand + K)
    B, V = 300, 40
    ks = rng.integers(0, kmax + 1, size=B)
    cu = np.concatenate([[0], np.cumsum(ks)]).astype(np.int64)
    T = int(cu[-1])
    prop = rng.integers(0, V, size=T)
    topk = np.array([rng.permutation(V)[:K] for _ in range(T)])
    drv = rng.integers(0, 2, size=B)
    ctx = rng.integers(0, 4100, size=B)     # a few windows cross the length cap
    sl = ctx + 1
    vals = np.array([0.25, 1.5, 2.0, 3.75, np.nan], np.float32)
    # mostly below both thresholds, so windows run long before an event
    ent = np.where(rng.random(T) < 0.9, np.float32(0.25), rng.choice(vals, size=T)).astype(np.float32)
    tt, th = 2.0, 0.25
    r = oracle.accept_scan(cu, prop, topk, K, drv, ctx, sl, 0, 4000, take_rule=take, hand_rule=hand,
                           ent=ent.astype(np.float64), tau_take=tt, tau_hand=th)
    g = _scan_rule(cu, prop, topk, K, drv, ctx, sl, 0, 4000, take, hand, ent, tt, th)
    _compare(g, r)
