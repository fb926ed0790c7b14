"""Pins for the oracle's SEM loss (selective entropy minimization, Sec. 4.2)
and its gradient (CPU only): closed forms (uniform and one-hot distributions),
scipy's log-softmax and entropy, numpy's percentile, and central finite
differences of an independently written FP64 loss."""
import numpy as np
import pytest
import scipy.special
import scipy.stats

import oracle
from tests import indep


def _bits(v):
    return indep.to_bf16_bits(np.asarray(v, np.float64))


def test_uniform_and_one_hot_rows():
    V = 1000
    z = np.zeros((2, V))
    z[1, 17] = 1000.0                                  # every other probability underflows
    H, nll, lse = oracle.sem_row_stats(_bits(z), np.array([3, 17]))
    assert abs(H[0] - np.log(V)) < 1e-12 and abs(nll[0] - np.log(V)) < 1e-12
    assert H[1] == 0.0 and nll[1] == 0.0 and lse[1] == 1000.0


def test_rows_match_scipy():
    rng = np.random.default_rng(4)
    z = indep.bf16_values(_bits(rng.normal(0, 3, (6, 513))))
    t = rng.integers(0, 513, 6)
    H, nll, lse = oracle.sem_row_stats(_bits(z), t)
    ls = scipy.special.log_softmax(z, axis=1)
    assert np.allclose(H, scipy.stats.entropy(np.exp(ls), axis=1), rtol=1e-12, atol=1e-12)
    assert np.allclose(nll, -ls[np.arange(6), t], rtol=1e-12, atol=1e-12)
    assert np.allclose(lse, scipy.special.logsumexp(z, axis=1), rtol=1e-13)


def test_weights_use_the_75th_percentile_and_the_minimum():
    rng = np.random.default_rng(5)
    for T in (1, 2, 5, 8, 101):
        H = rng.uniform(0, 4, T)
        w, tau, hmin = oracle.sem_weights(H, 1e-6)
        assert tau == pytest.approx(np.percentile(H, 75), abs=1e-15)
        assert hmin == H.min()
        assert w[np.argmin(H)] == 1.0
        expect = np.clip(1.0 - (H - H.min()) / (np.percentile(H, 75) - H.min() + 1e-6), 0.0, None)
        assert np.allclose(w, expect, atol=1e-15)
        assert np.all(w[H >= tau + 1e-6] == 0.0)


def test_loss_closed_form():
    H = np.array([0.5, 1.0, 2.0, 4.0])
    nll = np.array([1.0, 2.0, 3.0, 4.0])
    L, l_sft, l_ent, w = oracle.sem_loss(H, nll, lam=0.3, eps=0.0)
    tau = 2.0 + 0.25 * 2.0                               # position 2.25 between 2.0 and 4.0
    wexp = np.maximum(0, 1 - (H - 0.5) / (tau - 0.5))
    assert np.allclose(w, wexp)
    assert l_sft == 2.5
    assert l_ent == pytest.approx(np.sum(wexp * H) / 4)
    assert L == pytest.approx(2.5 + 0.3 * np.sum(wexp * H) / 4)


def _loss_fixed_weights(z, t, w, lam):
    ls = scipy.special.log_softmax(z, axis=1)
    p = np.exp(ls)
    H = -(p * ls).sum(axis=1)
    return (np.sum(-ls[np.arange(len(t)), t]) + lam * np.sum(w * H)) / len(t)


def test_gradient_matches_finite_differences():
    rng = np.random.default_rng(6)
    T, V, lam = 5, 9, 0.7
    z = np.round(rng.normal(0, 2, (T, V)) * 8) / 8      # exact in bfloat16
    t = rng.integers(0, V, T)
    bits = _bits(z)
    assert np.array_equal(indep.bf16_values(bits), z)
    H, nll, lse = oracle.sem_row_stats(bits, t)
    _, _, _, w = oracle.sem_loss(H, nll, lam, 1e-6)
    g = oracle.sem_grad(bits, t, H, lse, w, lam)
    h = 1e-6
    num = np.zeros_like(z)
    for i in range(T):
        for j in range(V):
            zp, zm = z.copy(), z.copy()
            zp[i, j] += h
            zm[i, j] -= h
            num[i, j] = (_loss_fixed_weights(zp, t, w, lam) - _loss_fixed_weights(zm, t, w, lam)) / (2 * h)
    assert np.allclose(g, num, atol=1e-8)
