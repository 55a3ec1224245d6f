"""Pins of the oracle's takeover draw (Eq. (9), second case) on the CPU.

The draw is the inverse CDF of softmax(logits) in index order.  Pins use
distributions whose cumulative probabilities are known exactly (logits that
are logs of integer weights), the two-token closed form, the measure of each
token's interval over a fine grid of uniforms, and invariances.
"""
import math

import numpy as np
import pytest

import oracle


def test_integer_weight_boundaries():
    # weights 1, 2, 3, 4: p = 0.1, 0.2, 0.3, 0.4; CDF 0.1, 0.3, 0.6, 1.0
    logits = np.log([1.0, 2.0, 3.0, 4.0])
    cases = [(0.0, 0), (0.05, 0), (0.0999, 0), (0.1001, 1), (0.2999, 1), (0.3001, 2),
             (0.5999, 2), (0.6001, 3), (0.99999, 3)]
    for u, want in cases:
        tok, margin = oracle.sample_categorical(logits, u)
        assert tok == want, (u, tok, want)
        assert margin >= 0.0
    # margins: distance to the nearer interval end
    assert oracle.sample_categorical(logits, 0.05)[1] == pytest.approx(0.05)
    assert oracle.sample_categorical(logits, 0.45)[1] == pytest.approx(0.15)


def test_two_token_closed_form():
    a, b = 0.3, -1.2
    p0 = 1.0 / (1.0 + math.exp(b - a))
    assert oracle.sample_categorical([a, b], p0 - 1e-9)[0] == 0
    assert oracle.sample_categorical([a, b], p0 + 1e-9)[0] == 1


def test_interval_measure_matches_probabilities():
    # over N equally spaced uniforms, token v is drawn for ~N p_v of them
    rng = np.random.default_rng(0)
    logits = rng.normal(size=23) * 1.5
    p = np.exp(logits - logits.max())
    p /= p.sum()
    N = 20000
    counts = np.zeros(23)
    for i in range(N):
        counts[oracle.sample_categorical(logits, (i + 0.5) / N)[0]] += 1
    assert np.all(np.abs(counts / N - p) <= 1.0 / N + 1e-12)


def test_shift_invariance_and_zero_probability_head():
    rng = np.random.default_rng(1)
    logits = rng.normal(size=50)
    for u in rng.random(20):
        assert oracle.sample_categorical(logits, u)[0] == oracle.sample_categorical(logits + 37.5, u)[0]
    # tokens of probability zero are never drawn, even for u = 0
    assert oracle.sample_categorical([-np.inf, -np.inf, 0.0, 0.0], 0.0)[0] == 2


def test_takeover_bookkeeping():
    # three sequences: a student-driven takeover at row 1, a student-driven
    # window without event, a teacher-driven handback (no draw)
    cu_q = np.array([0, 3, 5, 8])
    driver = np.array([oracle.DRIVER_S, oracle.DRIVER_S, oracle.DRIVER_T])
    event_row = np.array([1, -1, 0])
    V = 6
    logits = np.full((8, V), -np.inf)
    logits[:, 0] = 0.0
    logits[1] = np.log([1.0, 1.0, 1.0, 1.0, 1.0, 3.0])   # row of the takeover
    u = np.array([0.75, 0.1, 0.1])
    r = oracle.sample_takeover(cu_q, driver, event_row, logits, u, eos_id=V - 1)
    # CDF of row 1: 1/8, 2/8, 3/8, 4/8, 5/8, 1 -> u = 0.75 draws token 5 = EOS
    assert list(r["token"]) == [5, -1, -1]
    assert list(r["eos"]) == [True, False, False]
    assert r["margin"][0] == pytest.approx(0.125)
    assert np.isinf(r["margin"][1]) and np.isinf(r["margin"][2])
