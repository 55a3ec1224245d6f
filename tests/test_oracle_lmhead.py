"""Pins of the oracle's LM head + vocabulary log-softmax + top-K support.

Checked against closed forms (uniform and worked small examples), a library
routine on tie-free data (torch fp64 log_softmax / topk), the rank form of
top-K coverage, and invariants (normalisation, LSE and entropy bounds).
"""
import math

import numpy as np
import pytest
import torch

import oracle


def rand_case(M, Hd, V, seed=0):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((M, Hd))
    W = 0.3 * rng.standard_normal((V, Hd))
    prop = rng.integers(0, V, size=M)
    return h, W, prop


def test_worked_example_closed_form():
    """hidden (1, 0.5); W rows (2,0), (0,2), (1,1), (-1,0) -> logits
    (2, 1, 1.5, -1) by hand."""
    h = np.array([[1.0, 0.5]])
    W = np.array([[2.0, 0.0], [0.0, 2.0], [1.0, 1.0], [-1.0, 0.0]])
    r = oracle.lmhead_logsoftmax(h, W, np.array([2]), K=2)
    Z = math.exp(2) + math.exp(1) + math.exp(1.5) + math.exp(-1)
    assert r["lse"][0] == pytest.approx(math.log(Z), abs=1e-14)
    assert r["logp_prop"][0] == pytest.approx(1.5 - math.log(Z), abs=1e-14)
    assert r["argmax"][0] == 0
    assert list(r["topk_idx"][0]) == [0, 2]
    np.testing.assert_allclose(r["topk_logp"][0], [2 - math.log(Z), 1.5 - math.log(Z)], atol=1e-14)
    p = np.array([math.exp(2), math.exp(1), math.exp(1.5), math.exp(-1)]) / Z
    assert r["entropy"][0] == pytest.approx(-(p * np.log(p)).sum(), abs=1e-14)
    assert r["covered"][0]
    assert r["argmax_margin"][0] == pytest.approx(0.5)
    assert r["set_margin"][0] == pytest.approx(0.5)
    assert r["cover_margin"][0] == pytest.approx(0.5)


def test_against_torch_fp64_on_tie_free_data():
    h, W, prop = rand_case(6, 32, 300)
    r = oracle.lmhead_logsoftmax(h, W, prop, K=16)
    lt = torch.from_numpy(h) @ torch.from_numpy(W).T
    ls = torch.log_softmax(lt, dim=1)
    np.testing.assert_allclose(r["logp_prop"], ls[torch.arange(6), torch.from_numpy(prop)].numpy(),
                               atol=1e-12)
    np.testing.assert_allclose(r["lse"], torch.logsumexp(lt, dim=1).numpy(), atol=1e-12)
    vals, idx = torch.topk(lt, 16, dim=1)
    np.testing.assert_array_equal(r["topk_idx"], idx.numpy())
    np.testing.assert_allclose(r["topk_logp"], (vals - torch.logsumexp(lt, 1, keepdim=True)).numpy(),
                               atol=1e-12)
    np.testing.assert_array_equal(r["argmax"], lt.argmax(dim=1).numpy())
    ent = -(ls.exp() * ls).sum(dim=1)
    np.testing.assert_allclose(r["entropy"], ent.numpy(), atol=1e-12)


def test_normalisation_and_bounds():
    h, W, prop = rand_case(5, 16, 777, seed=2)
    r = oracle.lmhead_logsoftmax(h, W, prop, K=8)
    l = h @ W.T
    assert np.allclose(np.exp(l - r["lse"][:, None]).sum(axis=1), 1.0, atol=1e-13)
    assert np.all(l.max(axis=1) <= r["lse"] + 1e-15)
    assert np.all(r["lse"] <= l.max(axis=1) + math.log(777) + 1e-12)
    assert np.all(r["entropy"] >= -1e-12) and np.all(r["entropy"] <= math.log(777) + 1e-12)


def test_uniform_logits_pin_tie_break_and_entropy():
    V, K = 50, 5
    h = np.ones((3, 4))
    W = np.zeros((V, 4))
    r = oracle.lmhead_logsoftmax(h, W, np.array([0, 4, 5]), K=K)
    np.testing.assert_allclose(r["logp_prop"], -math.log(V), atol=1e-14)
    np.testing.assert_allclose(r["lse"], math.log(V), atol=1e-14)
    assert np.all(r["argmax"] == 0)
    np.testing.assert_array_equal(r["topk_idx"], np.tile(np.arange(K), (3, 1)))
    np.testing.assert_allclose(r["entropy"], math.log(V), atol=1e-13)
    assert list(r["covered"]) == [True, True, False]


def test_duplicated_rows_keep_index_order():
    rng = np.random.default_rng(4)
    W = rng.standard_normal((40, 8))
    W[30] = W[7]
    W[12] = W[7]
    h = np.zeros((1, 8))
    h[0] = W[7] * 10          # rows 7, 12, 30 share the largest logit
    r = oracle.lmhead_logsoftmax(h, W, np.array([30]), K=2)
    assert list(r["topk_idx"][0]) == [7, 12]
    assert r["argmax"][0] == 7
    assert not r["covered"][0]
    assert r["cover_margin"][0] == 0.0


@pytest.mark.parametrize("K", [0, 1, 4, 16, 64])
def test_coverage_rank_form(K):
    """covered <=> #{v : l_v > l_p or (l_v == l_p and v < p)} < K."""
    rng = np.random.default_rng(K)
    V = 64
    h = rng.standard_normal((20, 6))
    W = np.round(rng.standard_normal((V, 6)), 1)   # coarse values create ties
    prop = rng.integers(0, V, size=20)
    r = oracle.lmhead_logsoftmax(h, W, prop, K=K)
    l = h @ W.T
    for m in range(20):
        p = prop[m]
        rank = sum(1 for v in range(V) if l[m, v] > l[m, p] or (l[m, v] == l[m, p] and v < p))
        assert r["covered"][m] == (rank < K)
        assert (p in set(r["topk_idx"][m])) == (rank < K)


def test_brute_force_full_sort_small_vocab():
    """Top-K equals the first K of an explicit selection sort with index tie-break."""
    rng = np.random.default_rng(8)
    V = 24
    h = rng.standard_normal((4, 3))
    W = np.round(rng.standard_normal((V, 3)), 0)
    r = oracle.lmhead_logsoftmax(h, W, np.zeros(4, np.int64), K=V)
    l = h @ W.T
    for m in range(4):
        remaining = list(range(V))
        order = []
        while remaining:
            best = remaining[0]
            for v in remaining[1:]:
                if l[m, v] > l[m, best]:
                    best = v
            order.append(best)
            remaining.remove(best)
        assert list(r["topk_idx"][m]) == order


def test_large_logits_stay_finite():
    h = np.array([[1.0]])
    W = np.array([[900.0], [899.0], [0.0]])
    r = oracle.lmhead_logsoftmax(h, W, np.array([1]), K=1)
    Z = 1 + math.exp(-1) + math.exp(-900)
    assert r["lse"][0] == pytest.approx(900 + math.log(Z), abs=1e-12)
    assert r["logp_prop"][0] == pytest.approx(-1 - math.log(Z), abs=1e-12)
    assert np.isfinite(r["entropy"][0])
