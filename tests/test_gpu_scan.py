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
