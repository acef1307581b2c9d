"""Seeded input generators: time-rescaling checks of the history processes and
basic properties of the weight generator.

Time-rescaling theorem (App. A.4): the compensator increments between events of
a correctly simulated process are i.i.d. Exp(1); a one-sample KS statistic
below 1.36/sqrt(n) passes at the 5 % level (App. C.3.1).
"""
import numpy as np
import pytest
import scipy.stats

from paper_2507_09252_amd import workloads as W

KS = 1.36


def _ks_exp(z):
    return scipy.stats.kstest(z, "expon").statistic < KS / np.sqrt(len(z))


def test_hpp_rescaled():
    t, _ = W.hpp(4000, 2.5, np.random.default_rng(0))
    assert _ks_exp(np.diff(np.concatenate([[0.0], t])) * 2.5)


def test_ipp_sin_rescaled():
    t, _ = W.ipp_sin(4000, np.random.default_rng(1))
    tt = np.concatenate([[0.0], t])
    z = np.array([W.ipp_sin_compensator(a, b) for a, b in zip(tt[:-1], tt[1:])])
    assert _ks_exp(z)


@pytest.mark.parametrize("kind", ["hawkes1", "hawkes22", "hawkes5"])
def test_hawkes_rescaled(kind):
    rng = np.random.default_rng(2)
    mu, alpha, beta = W.hawkes_params(kind, rng)
    t, k = W.hawkes(3000, mu, alpha, beta, rng)
    assert np.all(np.diff(t) > 0)
    z = W.hawkes_compensator_intervals(t, k, mu, alpha, beta)
    assert _ks_exp(z)
    if kind != "hawkes1":
        rho = np.max(np.abs(np.linalg.eigvals(alpha / beta)))
        assert abs(rho - (0.7 if kind == "hawkes22" else 0.5)) < 1e-9


def test_hawkes_type_mix():
    # with alpha = 0 the types follow mu / sum(mu)
    rng = np.random.default_rng(3)
    mu = np.array([0.5, 0.3, 0.2])
    t, k = W.hawkes(20000, mu, np.zeros((3, 3)), np.ones((3, 3)), rng)
    assert scipy.stats.chisquare(np.bincount(k, minlength=3), mu * 20000).pvalue > 1e-3


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_weights_and_histories(name):
    wl = W.WORKLOADS[name]
    wt, wd = W.workload_weights(wl)
    for cfg, w in ((wl.target, wt), (wl.draft, wd)):
        names = W.weight_names(cfg)
        assert set(w) == {n for n, _, _ in names}
        for n, shape, kind in names:
            assert w[n].shape == shape and w[n].dtype == np.float32
            if cfg.prec == "bf16" and kind == "mat":
                assert np.array_equal(W.to_bf16_values(w[n]), w[n])
    wt2, _ = W.workload_weights(wl)
    assert all(np.array_equal(wt[n], wt2[n]) for n in wt)
    B = min(wl.batch, 8)
    t, k = W.make_histories(wl, batch=B)
    assert t.shape == (B, wl.n_hist) and t.dtype == np.float32 and k.dtype == np.int32
    assert np.all(np.diff(t, axis=1) > 0) and np.all(t > 0)
    assert k.min() >= 0 and k.max() < wl.target.n_types
