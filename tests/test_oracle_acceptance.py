"""Pins of the acceptance-rate oracle (Sec. 3.1, Eq. 1) and of its per-bin tail
statistic against things the oracle's own code does not decide: the identities
of Eq. 1, total-variation distance, closed forms, invariances, and numpy's
percentile."""
import math

import numpy as np
import pytest
import scipy.special

import oracle


def rows(T, V, seed, scale=2.0):
    return (np.random.default_rng(seed).standard_normal((T, V)) * scale).astype(np.float32)


def softmax64(z, tau=1.0):
    return scipy.special.softmax(tau * z.astype(np.float64), axis=-1)


def test_identical_rows_accept_everything():
    z = rows(4, 3000, 0)
    np.testing.assert_allclose(oracle.acceptance(z, z), 1.0, rtol=0, atol=1e-12)


def test_symmetric():
    a, b = rows(5, 2000, 1), rows(5, 2000, 2)
    np.testing.assert_array_equal(oracle.acceptance(a, b), oracle.acceptance(b, a))


def test_equals_one_minus_total_variation():
    a = rows(6, 5000, 3)
    b = a + rows(6, 5000, 4, scale=0.7)
    p, q = softmax64(a), softmax64(b)
    tv = 0.5 * np.array([math.fsum(np.abs(p[t] - q[t])) for t in range(6)])
    np.testing.assert_allclose(oracle.acceptance(a, b), 1.0 - tv, rtol=0, atol=1e-12)


def test_equals_expectation_under_the_draft():
    # Eq. 1, left form: E_{x ~ q} [min(p(x) / q(x), 1)]
    a = rows(4, 3000, 5)
    b = a + rows(4, 3000, 6, scale=1.5)
    p, q = softmax64(a), softmax64(b)
    lhs = np.array([math.fsum(q[t] * np.minimum(p[t] / q[t], 1.0)) for t in range(4)])
    np.testing.assert_allclose(oracle.acceptance(a, b), lhs, rtol=0, atol=1e-12)


def test_two_token_closed_form():
    # p = (1 - s(a), s(a)), q = (1 - s(b), s(b)) with s the logistic function:
    # alpha = 1 - |s(a) - s(b)|
    for a_, b_ in [(0.0, 1.0), (2.5, -1.0), (7.0, 7.0), (-3.0, 4.0)]:
        t = np.array([[0.0, a_]], np.float32)
        d = np.array([[0.0, b_]], np.float32)
        s = lambda x: 1.0 / (1.0 + math.exp(-x))   # noqa: E731
        assert abs(oracle.acceptance(t, d)[0] - (1.0 - abs(s(a_) - s(b_)))) < 1e-14


def test_masked_entries_drop_out():
    # a logit of -inf is a token of probability 0 in both rows: the rate equals the rate over
    # the rest of the vocabulary (runs at the start, in the middle and at the end of the row)
    a = rows(3, 3000, 21)
    b = a + rows(3, 3000, 22, scale=0.8)
    keep = np.ones(3000, bool)
    keep[:700] = keep[1500:1503] = keep[-129:] = False
    am, bm = a.copy(), b.copy()
    am[:, ~keep] = -np.inf
    bm[:, ~keep] = -np.inf
    for tau in (1.0, 0.6):
        want = oracle.acceptance(np.ascontiguousarray(a[:, keep]),
                                 np.ascontiguousarray(b[:, keep]), tau)
        np.testing.assert_allclose(oracle.acceptance(am, bm, tau), want, rtol=0, atol=1e-14)
    # and against the definition on the masked distributions
    p, q = softmax64(a[:, keep]), softmax64(b[:, keep])
    np.testing.assert_allclose(oracle.acceptance(am, bm),
                               [math.fsum(np.minimum(p[t], q[t])) for t in range(3)],
                               rtol=0, atol=1e-12)


def test_shift_and_temperature():
    a, b = rows(3, 4000, 7), rows(3, 4000, 8)
    a, b = np.round(a * 1024) / 1024, np.round(b * 1024) / 1024   # so that shifts are exact
    base = oracle.acceptance(a, b)
    # a constant added to a row does not change its distribution
    np.testing.assert_allclose(oracle.acceptance(a + 3.0, b - 5.0), base, rtol=0, atol=1e-12)
    # inverse temperature tau on logits z is the same as temperature 1 on tau * z
    tau = 0.6
    np.testing.assert_allclose(oracle.acceptance(a, b, inv_temp=tau),
                               oracle.acceptance((tau * a.astype(np.float64)).astype(np.float32),
                                                 (tau * b.astype(np.float64)).astype(np.float32)),
                               rtol=0, atol=1e-6)
    # tau = 0: both distributions uniform
    np.testing.assert_allclose(oracle.acceptance(a, b, inv_temp=0.0), 1.0, rtol=0, atol=1e-12)


def test_disjoint_peaks_accept_almost_nothing():
    V = 1000
    t = np.zeros((1, V), np.float32)
    d = np.zeros((1, V), np.float32)
    t[0, 3] = 60.0
    d[0, 700] = 60.0
    # each distribution puts 1 - (V-1) e^-60 on its own peak
    assert oracle.acceptance(t, d)[0] < 1e-20


def test_bf16_input_equals_fp32_of_the_same_values():
    a = rows(3, 2048, 9)
    b = rows(3, 2048, 10)
    ab = (a.view(np.uint32) >> 16).astype(np.uint16)        # truncate to bf16 patterns
    bb = (b.view(np.uint32) >> 16).astype(np.uint16)
    af = (ab.astype(np.uint32) << 16).view(np.float32)
    bf = (bb.astype(np.uint32) << 16).view(np.float32)
    np.testing.assert_array_equal(oracle.acceptance(ab, bb), oracle.acceptance(af, bf))


def test_topk_approximation():
    a = rows(5, 600, 11)
    b = a + rows(5, 600, 12, scale=0.8)
    lp = np.log(softmax64(a)).astype(np.float32)
    lq = np.log(softmax64(b)).astype(np.float32)
    exact = oracle.acceptance(a, b)
    # all tokens listed: the approximation is exact (up to fp32 log-probabilities)
    np.testing.assert_allclose(oracle.acceptance_topk(lp, lq), exact, rtol=0, atol=1e-5)
    # the top-K of the draft: a lower bound that grows with K
    order = np.argsort(-lq, axis=1)
    prev = np.zeros(5)
    for K in (1, 5, 20, 100):
        sel = order[:, :K]
        approx = oracle.acceptance_topk(np.take_along_axis(lp, sel, 1),
                                        np.take_along_axis(lq, sel, 1))
        assert (approx <= exact + 1e-6).all() and (approx >= prev - 1e-12).all()
        prev = approx


def test_tail_stats_match_numpy_percentile():
    rng = np.random.default_rng(13)
    T = 5000
    alpha = (1.0 - rng.beta(0.3, 4.0, size=T) * 0.6).astype(np.float32)
    pos = rng.integers(-5, 45000, size=T).astype(np.int32)
    n_bins = 20
    for pct in (0.0, 5.0, 37.5, 50.0, 100.0):
        q, m, c = oracle.tail_stats(alpha, pos, 2048, n_bins, pct)
        for b in range(n_bins):
            sel = pos >= 0
            bins = np.minimum(pos[sel] // 2048, n_bins - 1)
            vals = alpha[sel][bins == b].astype(np.float64)
            assert c[b] == len(vals)
            assert q[b] == np.percentile(vals, pct, method="linear")
            assert abs(m[b] - math.fsum(vals) / len(vals)) < 1e-12


def test_tail_stats_small_cases():
    a = np.array([0.9, 0.2, 0.7], np.float32)
    q, m, c = oracle.tail_stats(a, np.array([1, 2, 3], np.int32), 2048, 3, 5.0)
    # sorted (0.2, 0.7, 0.9): h = 2 * 0.05 = 0.1 -> 0.2 + 0.1 * (0.7 - 0.2)
    assert c.tolist() == [3, 0, 0]
    assert q[0] == np.float64(np.float32(0.2)) + 0.1 * (np.float64(np.float32(0.7))
                                                        - np.float64(np.float32(0.2)))
    assert math.isnan(q[1]) and math.isnan(m[2])
    q1, _, c1 = oracle.tail_stats(np.array([0.5], np.float32), np.array([99999], np.int32),
                                  2048, 4, 5.0)
    assert c1.tolist() == [0, 0, 0, 1] and q1[3] == np.float64(np.float32(0.5))
