"""Pins for the oracle's LM head, argmax, entropy and acceptance.

Entropy (Sec. 3.3.1, H = -sum p log p over the vocabulary) is pinned by
closed forms (uniform, one-hot, two-level logits), shift invariance and
scipy's entropy routine; argmax by numpy; acceptance by brute force on
constructed drafts; the route by the threshold rule at tau = H +- eps.
"""
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle


@pytest.mark.parametrize("vocab,expected", [
    (4096, 12 * math.log(2)),                      # 2^12
    (151936, 7 * math.log(2) + math.log(1187)),    # 2^7 * 1187
])
def test_uniform_logits_entropy_is_log_vocab(vocab, expected):
    z = np.full((2, vocab), 3.25, np.float32)
    am, ent, margin = oracle.lmhead_rows(logits=z)
    # a sequential fp64 sum of V positive terms is exact to ~V * 2^-53
    np.testing.assert_allclose(ent, expected, rtol=vocab * 2.0 ** -53)
    assert list(am) == [0, 0]          # ties resolve to the lowest index
    assert list(margin) == [0.0, 0.0]


def test_one_hot_entropy_is_zero():
    z = np.full((3, 1000), -np.inf, np.float32)
    z[0, 17] = 0.0
    z[1, 999] = 5.0
    z[2, 0] = -3.0
    am, ent, _ = oracle.lmhead_rows(logits=z)
    assert list(am) == [17, 999, 0]
    np.testing.assert_array_equal(ent, 0.0)
    z = np.zeros((1, 1000), np.float32)
    z[0, 5] = 1e4                      # finite but overwhelming gap
    am, ent, margin = oracle.lmhead_rows(logits=z)
    assert am[0] == 5 and ent[0] == 0.0 and margin[0] == 1e4


@pytest.mark.parametrize("k,a,b", [(1, 2.0, 0.0), (7, 0.5, -1.0),
                                   (300, 1.0, 0.9)])
def test_two_level_logits_closed_form(k, a, b):
    vocab = 1000
    z = np.full((1, vocab), b, np.float32)
    idx = np.random.default_rng(k).choice(vocab, k, replace=False)
    z[0, idx] = a
    a64, b64 = float(np.float32(a)), float(np.float32(b))
    zsum = k * math.exp(a64) + (vocab - k) * math.exp(b64)
    pa, pb = math.exp(a64) / zsum, math.exp(b64) / zsum
    expected = -(k * pa * math.log(pa) + (vocab - k) * pb * math.log(pb))
    am, ent, _ = oracle.lmhead_rows(logits=z)
    assert am[0] == idx.min()
    np.testing.assert_allclose(ent[0], expected, rtol=1e-12)


def test_entropy_matches_scipy_and_is_shift_invariant():
    rng = np.random.default_rng(1)
    z = (rng.standard_normal((4, 5000)) * np.array([[0.5], [2], [8], [30]])
         ).astype(np.float32)
    am, ent, margin = oracle.lmhead_rows(logits=z)
    z64 = z.astype(np.float64)
    ref = scipy.stats.entropy(scipy.special.softmax(z64, axis=1), axis=1)
    np.testing.assert_allclose(ent, ref, rtol=1e-10)
    np.testing.assert_array_equal(am, np.argmax(z, axis=1))
    srt = np.sort(z64, axis=1)
    np.testing.assert_array_equal(margin, srt[:, -1] - srt[:, -2])
    am2, ent2, _ = oracle.lmhead_rows(logits=z + np.float32(64.0))
    np.testing.assert_array_equal(am2, am)
    np.testing.assert_allclose(ent2, ent, rtol=1e-5)   # shift is fp32-rounded


def test_hidden_times_weight_matches_matmul():
    rng = np.random.default_rng(2)
    gamma, d, vocab = 5, 64, 3000
    h = rng.standard_normal((gamma, d)).astype(np.float32)
    w = (rng.standard_normal((vocab, d)) * 0.1).astype(np.float32)
    am, ent, margin, z = oracle.lmhead_rows(h, w, want_logits=True)
    ref = h.astype(np.float64) @ w.astype(np.float64).T
    np.testing.assert_allclose(z, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(am, np.argmax(ref, axis=1))
    ref_ent = scipy.stats.entropy(scipy.special.softmax(ref, axis=1), axis=1)
    np.testing.assert_allclose(ent, ref_ent, rtol=1e-10)


def test_accept_constructed_prefixes():
    rng = np.random.default_rng(3)
    gamma = 8
    argmax = rng.integers(0, 100, gamma).astype(np.int32)
    ent = rng.random(gamma) * 5
    for k in range(gamma):
        draft = rng.integers(0, 100, gamma - 1).astype(np.int32)
        draft[:k] = argmax[:k]
        if k < gamma - 1:
            draft[k] = (argmax[k] + 1) % 100
        n, bonus, route, ht = oracle.accept(argmax, ent, draft, tau=2.5)
        assert n == k
        assert bonus == argmax[k]
        assert ht == ent[k]
        assert route == int(ent[k] > 2.5)


def test_accept_gamma_one_is_plain_decode():
    n, bonus, route, ht = oracle.accept(np.array([42], np.int32),
                                        np.array([1.5]), None, tau=1.0)
    assert (n, bonus, route, ht) == (0, 42, 1, 1.5)


def test_route_threshold_is_strict():
    argmax = np.array([3, 4, 5], np.int32)
    ent = np.array([0.1, 2.0, 0.3])
    draft = np.array([3, 9], np.int32)          # n = 1, H_t = 2.0
    assert oracle.accept(argmax, ent, draft, 2.0 - 1e-9)[2] == 1
    assert oracle.accept(argmax, ent, draft, 2.0)[2] == 0
    assert oracle.accept(argmax, ent, draft, 2.0 + 1e-9)[2] == 0


@settings(max_examples=200, deadline=None)
@given(st.lists(st.integers(0, 3), min_size=1, max_size=20), st.data())
def test_accept_is_longest_matching_prefix(argmax, data):
    gamma = len(argmax)
    draft = data.draw(st.lists(st.integers(0, 3), min_size=gamma - 1,
                               max_size=gamma - 1))
    am = np.array(argmax, np.int32)
    ent = np.arange(gamma, dtype=np.float64)
    n, bonus, _, ht = oracle.accept(am, ent, np.array(draft, np.int32), 0.0)
    brute = 0
    for j in range(gamma - 1):
        if all(draft[t] == argmax[t] for t in range(j + 1)):
            brute = j + 1
    assert n == brute and bonus == argmax[n] and ht == float(n)
