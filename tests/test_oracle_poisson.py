"""Pins for the oracle's homogeneous-Poisson draft (App. D.3).

The draft intervals are Exp(rate) and the marks categorical(p), with rate and
p the maximum-likelihood estimates n / T and n_m / n. Pinned here:

- the fit on a hand-computed example;
- one drafted block: intervals against the exponential CDF (KS), marks
  against p (chi-square), the recorded log-densities against scipy's
  exponential log-density (an independent implementation of the closed form);
- Theorem 1 with the exponential draft density: the acceptance rate of the
  residual loop equals the integral of max(0, g_T - g_D) (quadrature) and the
  accepted intervals follow norm(max(0, g_T - g_D));
- the whole sampler: TPP-SD with the Poisson draft has the law of AR sampling
  (two-sample KS per position and chi-square on types, Bonferroni 1 %), while
  redrawing from the target instead of the adjusted distribution fails.
"""
import concurrent.futures as cf
import multiprocessing as mp
import os

import numpy as np
import scipy.integrate
import scipy.stats

from oracle import sampler as S
from oracle.numerics import log_softmax
from test_oracle_sampling import KS_C, _log_grid_cdf
from test_oracle_sd_law import GAMMA, N_GEN, _history, _models, _pvalues


def test_poisson_fit_hand_example():
    ht = np.array([[0.0, 1.0, 3.0], [2.0, 4.0, 8.0]])
    hk = np.array([[0, 2, 2], [1, 2, 0]])
    rate, logp = S.poisson_fit(ht, hk, K=4)
    # 2 x 2 intervals over spans 3 + 6
    assert rate == 4.0 / 9.0
    np.testing.assert_allclose(np.exp(logp), [2 / 6, 1 / 6, 3 / 6, 0.0])
    assert logp[3] == -np.inf


def test_poisson_draft_block():
    B, gamma, rate = 4000, 5, 0.7
    logp = np.log([0.5, 0.3, 0.2])
    T, _ = _models()
    HT, HK = _history(B)
    st = S.prefill(T, None, HT, HK, 10)
    dr = S.draft_poisson(st, gamma, rate, logp, seed=9, rows=np.arange(B))
    for l in range(gamma):
        assert scipy.stats.kstest(dr.tau[:, l], scipy.stats.expon(scale=1 / rate).cdf).statistic < KS_C / np.sqrt(B)
        counts = np.bincount(dr.k[:, l], minlength=3)
        assert scipy.stats.chisquare(counts, B * np.exp(logp)).pvalue > 1e-3
    np.testing.assert_allclose(dr.logg, scipy.stats.expon(scale=1 / rate).logpdf(dr.tau), rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(dr.logf, logp[dr.k])
    # event times: running float32 sums of the intervals after the pending event
    t0 = HT[:, -1].astype(np.float64)
    np.testing.assert_allclose(dr.t[:, 0], (t0 + dr.tau[:, 0]).astype(np.float32), rtol=0)
    np.testing.assert_allclose(dr.t[:, 1], (dr.t[:, 0] + dr.tau[:, 1]).astype(np.float32), rtol=0)


def test_theorem1_with_exponential_draft():
    Tw, Tmu, Ts = log_softmax(np.array([0.2, -0.5, 0.1])), np.array([0.3, -0.8, 1.0]), np.log([0.5, 0.7, 0.4])
    rate = 0.8

    def gT(x):
        return np.exp(S.mixture_logpdf(Tw, Tmu, Ts, x))

    def gD(x):
        return rate * np.exp(-rate * x)

    Z = scipy.integrate.quad(lambda y: max(0.0, gT(np.exp(y)) - gD(np.exp(y))) * np.exp(y), -30, 30,
                             limit=500, points=[-2, -1, 0, 1, 2])[0]
    assert 0.1 < Z < 0.9
    n = 3000
    taus, iters = np.zeros(n), np.zeros(n)
    for b in range(n):
        tau, j, _, _ = S.resid_time(Tw, Tmu, Ts, None, None, None, seed=5, b=b, r=0, draft_rate=rate)
        taus[b], iters[b] = tau, j
    zhat = n / np.sum(iters + 1)
    assert abs(zhat - Z) < 4 * np.sqrt(Z * Z * (1 - Z) / n)
    x, c = _log_grid_cdf(lambda t: np.maximum(0, gT(t) - gD(t)))
    cdf_res = lambda t: np.interp(np.log(t), x, c / c[-1])
    assert scipy.stats.kstest(taus, cdf_res).statistic < KS_C / np.sqrt(n)


def _chunk(args):
    kind, seq0, B, opts = args
    T, _ = _models()
    HT, HK = _history(B)
    if kind == "ar":
        st = S.sample_ar(T, HT, HK, N_GEN, seed=11, seq0=seq0)
    else:
        rate, logp = S.poisson_fit(HT[:1], HK[:1], K=3)
        st = S.sample_sd_poisson(T, HT, HK, N_GEN, GAMMA, rate, logp, seed=11, seq0=seq0, **opts)
    n0 = HT.shape[1]
    tau = np.diff(st.t[:, n0 - 1:n0 + N_GEN], axis=1)
    return tau, st.k[:, n0:n0 + N_GEN], st.accepted_drafts, st.drafted


def _run(kind, n, opts=None, chunk=2500):
    jobs = [(kind, s, min(chunk, n - s), opts or {}) for s in range(0, n, chunk)]
    workers = max(1, min(8, os.cpu_count() or 1))
    with cf.ProcessPoolExecutor(workers, mp_context=mp.get_context("fork")) as ex:
        parts = list(ex.map(_chunk, jobs))
    tau = np.concatenate([p[0] for p in parts])
    k = np.concatenate([p[1] for p in parts])
    acc = sum(p[2] for p in parts) / max(1, sum(p[3] for p in parts))
    return tau, k, acc


def test_sd_poisson_law_equals_ar():
    ar = _run("ar", 20000)
    sd = _run("sdp", 20000)
    assert 0.1 < sd[2] < 0.9, sd[2]
    ps = _pvalues(ar, sd)
    assert ps.min() > 0.01 / len(ps), ps
    bad = _run("sdp", 20000, {"resample_from_target": True})
    assert _pvalues(ar, bad).min() < 1e-4
