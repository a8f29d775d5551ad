"""Pins of the distillation oracle (oracle/luna_distill.py) to what the mathematics
fixes: a student equal to the teacher costs exactly the teacher's entropy (scipy's
softmax and entropy, not the oracle's), Gibbs' inequality, uniform rows, values by
hand, the smoothed student being a distribution, finite differences of the loss for
the feature and parameter gradients, causal rows blind to later keys, and the scale
invariance of the normalised weights.  Each pin takes the distillation module."""

from __future__ import annotations

import math

import numpy as np
import scipy.special
import scipy.stats

from oracle import luna_oracle as base


def _params(rng, M=3, L=2, d=4, hidden=5):
    s = 1.0 / math.sqrt(d)
    return {"W": rng.standard_normal((M, d)) * s, "b": rng.standard_normal(M) * s,
            "fc1_w": rng.standard_normal((L, hidden)), "fc1_b": rng.standard_normal((L, hidden)),
            "fc2_w": rng.standard_normal((L, hidden)) * 0.5, "fc2_b": rng.standard_normal(L) * 0.3 + 0.6,
            "M": M, "L": L, "hidden": hidden, "nonneg": True, "shared_channels": False, "per_head": False}


def _masked_logits(Q, K, causal):
    n, d = Q.shape[-2], Q.shape[-1]
    logits = Q @ K.T / np.sqrt(d)
    if causal:
        logits = np.where(np.tril(np.ones((n, n), bool)), logits, -np.inf)
    return logits


def pin_student_equal_to_teacher_costs_the_entropy(v):
    """With phi(k_s) = e_s and phi(q_t) = the teacher's row t (computed here by scipy),
    P = A and den = 1, so with eps = 0 the loss of every row is the teacher row's
    Shannon entropy (scipy.stats.entropy)."""
    rng = np.random.default_rng(51)
    n, d = 7, 5
    Q, K = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    for causal in (False, True):
        A = scipy.special.softmax(_masked_logits(Q, K, causal), axis=-1)
        ce = v.distill_rows_features(Q, K, A, np.eye(n), causal=causal, eps=0.0)
        ent = np.array([scipy.stats.entropy(A[t][A[t] > 0]) for t in range(n)])
        assert np.max(np.abs(ce - ent)) < 1e-12, (causal, ce, ent)


def pin_gibbs_inequality(v):
    """CE_t >= H(A_t), with equality only for Ahat_t = A_t: random positive features
    cost strictly more than the entropy."""
    rng = np.random.default_rng(52)
    n, d, D = 9, 4, 6
    Q, K = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    fq, fk = rng.uniform(0.1, 1.0, (n, D)), rng.uniform(0.1, 1.0, (n, D))
    for causal in (False, True):
        A = scipy.special.softmax(_masked_logits(Q, K, causal), axis=-1)
        ent = np.array([scipy.stats.entropy(A[t][A[t] > 0]) for t in range(n)])
        ce = v.distill_rows_features(Q, K, fq, fk, causal=causal, eps=0.0)
        gap = ce - ent
        first = 1 if causal else 0  # a causal row 0 sees one key: both distributions are [1]
        assert np.all(gap[first:] > 1e-6), gap
        assert abs(gap[0]) < 1e-12 or not causal


def pin_uniform_rows(v):
    """Q = 0 makes the teacher uniform over the visible keys and constant features make
    the smoothed student exactly uniform too ((c + eps/n_t) / (n_t c + eps) = 1/n_t), so
    CE_t = log n_t: log n, or log(t + 1) when causal, for any eps."""
    n, d, D = 6, 3, 4
    rng = np.random.default_rng(53)
    Q, K = np.zeros((n, d)), rng.standard_normal((n, d))
    fq, fk = np.full((n, D), 0.3), np.full((n, D), 0.7)
    for eps in (0.0, 0.5):
        ce = v.distill_rows_features(Q, K, fq, fk, causal=False, eps=eps)
        assert np.allclose(ce, math.log(n), rtol=0, atol=1e-13), ce
        ce = v.distill_rows_features(Q, K, fq, fk, causal=True, eps=eps)
        assert np.allclose(ce, np.log(np.arange(1, n + 1)), rtol=0, atol=1e-13), ce


def pin_hand_example(v):
    """d = 1, Q = [1, 1], K = [0, ln 3]: teacher rows (1/4, 3/4).  phi(K) = [1, 3] with any
    positive phi(q) reproduces them: CE = ln 4 - (3/4) ln 3 on both rows; phi(K) = [1, 1]
    gives the uniform student: CE = ln 2.  Causal row 0 sees one key: CE = 0."""
    Q = np.array([[1.0], [1.0]])
    K = np.array([[0.0], [math.log(3.0)]])
    fq = np.array([[1.0], [2.0]])
    h = math.log(4.0) - 0.75 * math.log(3.0)
    ce = v.distill_rows_features(Q, K, fq, np.array([[1.0], [3.0]]), eps=0.0)
    assert np.allclose(ce, [h, h], rtol=0, atol=1e-14), ce
    ce = v.distill_rows_features(Q, K, fq, np.array([[1.0], [1.0]]), eps=0.0)
    assert np.allclose(ce, [math.log(2.0)] * 2, rtol=0, atol=1e-14), ce
    ce = v.distill_rows_features(Q, K, fq, np.array([[1.0], [3.0]]), causal=True, eps=0.0)
    assert np.allclose(ce, [0.0, h], rtol=0, atol=1e-14), ce


def pin_smoothed_student_is_a_distribution(v):
    """Every student row sums to 1 over its visible keys; a key whose P is 0 gets
    exactly (eps / n_t) / (den_t + eps)."""
    rng = np.random.default_rng(54)
    n, D, eps = 5, 3, 0.25
    fq = rng.uniform(0.0, 1.0, (n, D))
    fk = rng.uniform(0.0, 1.0, (n, D))
    fk[2] = 0.0  # key 2 has P = 0 for every query
    for causal in (False, True):
        Ah = v.student(fq, fk, causal=causal, eps=eps)
        assert np.allclose(Ah.sum(axis=-1), 1.0, rtol=0, atol=1e-14)
        P = fq @ fk.T
        for t in range(2 if causal else 0, n):
            nt = t + 1 if causal else n
            den = P[t, :nt].sum()
            assert abs(Ah[t, 2] - (eps / nt) / (den + eps)) < 1e-15


def _fd(f, x, idx, h=1e-6):
    xp, xm = x.copy(), x.copy()
    xp[idx] += h
    xm[idx] -= h
    return (f(xp) - f(xm)) / (2 * h)


def pin_feature_gradients_by_finite_differences(v):
    """dphi(Q), dphi(K) of mean(CE) against central differences, both forms, eps > 0."""
    rng = np.random.default_rng(55)
    B, n, d, D, eps = 2, 6, 3, 4, 1e-2
    Q, K = rng.standard_normal((B, n, d)), rng.standard_normal((B, n, d))
    fq, fk = rng.uniform(0.05, 1.0, (B, n, D)), rng.uniform(0.05, 1.0, (B, n, D))
    for causal in (False, True):
        gq, gk = v.distill_feature_grads(Q, K, fq, fk, causal=causal, eps=eps)
        for _ in range(6):
            idx = tuple(int(rng.integers(s)) for s in fq.shape)
            num = _fd(lambda x: v.distill_rows_features(Q, K, x, fk, causal, eps).mean(), fq, idx)
            assert abs(num - gq[idx]) < 1e-7 * max(1.0, abs(num)), ("q", causal, num, gq[idx])
            num = _fd(lambda x: v.distill_rows_features(Q, K, fq, x, causal, eps).mean(), fk, idx)
            assert abs(num - gk[idx]) < 1e-7 * max(1.0, abs(num)), ("k", causal, num, gk[idx])


def pin_parameter_gradients_by_finite_differences(v):
    """The feature-map parameter gradients of mean(CE) (through phi of the queries and of
    the keys) against central differences of the loss in each parameter."""
    rng = np.random.default_rng(56)
    n, d = 5, 4
    p = _params(rng, d=d)
    Q, K = rng.standard_normal((2, n, d)), rng.standard_normal((2, n, d))
    for causal in (False, True):
        _, grads = v.distill_backward(Q, K, p, causal=causal, eps=1e-3)
        for name in base.PARAM_NAMES:
            arr = np.asarray(p[name], float)
            for _ in range(2):
                idx = tuple(int(rng.integers(s)) for s in arr.shape)

                def loss(x, name=name):
                    q = dict(p)
                    q[name] = x
                    return v.distill_rows(Q, K, q, causal, 1e-3).mean()

                num = _fd(loss, arr, idx, h=1e-6)
                assert abs(num - grads[name][idx]) < 1e-6 * max(1.0, abs(num)), (name, causal, num, grads[name][idx])


def pin_causal_rows_ignore_later_keys(v):
    """Changing the keys after position t (teacher logits and student features alike)
    leaves the causal losses of rows 0..t unchanged."""
    rng = np.random.default_rng(57)
    n, d, t = 8, 4, 4
    p = _params(rng, d=d)
    Q, K = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    K2 = K.copy()
    K2[t + 1:] = rng.standard_normal((n - t - 1, d)) * 3.0
    a = v.distill_rows(Q, K, p, causal=True)
    b = v.distill_rows(Q, K2, p, causal=True)
    assert np.max(np.abs(a[:t + 1] - b[:t + 1])) < 1e-13
    assert np.max(np.abs(a[t + 1:] - b[t + 1:])) > 1e-6


def pin_scale_invariance(v):
    """With eps = 0 the student is P_ts / den_t: scaling phi(Q) or phi(K) by positive
    constants changes no loss."""
    rng = np.random.default_rng(58)
    n, d, D = 6, 3, 5
    Q, K = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    fq, fk = rng.uniform(0.1, 1.0, (n, D)), rng.uniform(0.1, 1.0, (n, D))
    for causal in (False, True):
        a = v.distill_rows_features(Q, K, fq, fk, causal, 0.0)
        b = v.distill_rows_features(Q, K, 3.7 * fq, 0.2 * fk, causal, 0.0)
        assert np.max(np.abs(a - b)) < 1e-13


ALL_PINS = [
    pin_student_equal_to_teacher_costs_the_entropy,
    pin_gibbs_inequality,
    pin_uniform_rows,
    pin_hand_example,
    pin_smoothed_student_is_a_distribution,
    pin_feature_gradients_by_finite_differences,
    pin_parameter_gradients_by_finite_differences,
    pin_causal_rows_ignore_later_keys,
    pin_scale_invariance,
]


def pin_sampled_rows_match_the_whole_head(v):
    """distill_rows_at (row by row, for long sequences) equals the pinned whole-head
    losses at every row, both forms."""
    rng = np.random.default_rng(59)
    n, d, D = 11, 4, 5
    Q, K = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    fq, fk = rng.uniform(0.0, 1.0, (n, D)), rng.uniform(0.0, 1.0, (n, D))
    for causal in (False, True):
        whole = v.distill_rows_features(Q, K, fq, fk, causal, 1e-3)
        rows = v.distill_rows_at(Q, K, fq, fk, list(range(n)), causal, 1e-3)
        assert np.max(np.abs(whole - rows)) < 1e-13


ALL_PINS.append(pin_sampled_rows_match_the_whole_head)
