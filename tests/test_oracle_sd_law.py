"""Whole-sampler pins for the oracle: TPP-SD output law equals AR sampling's.

TPP-SD is exact (§4.3, App. A.2): sequences it generates have the law of
autoregressive sampling from the target. On a small model pair with K = 3
types and a deliberately mismatched draft (acceptance rate about 0.5), both
samplers generate 2*gamma + 2 events after one fixed history; per output
position we compare inter-event times (two-sample KS) and types (chi-square
contingency), Bonferroni-corrected at 1 %.

Negative controls must FAIL the same tests: Algorithm 1 read literally
(redraw both components at the first rejection) and redrawing from the target
instead of the adjusted distributions (the incorrect scheme of App. A.2).

Special cases: draft == target accepts every draft (alpha = 1); K = 1 never
rejects a type.
"""
import concurrent.futures as cf
import multiprocessing as mp
import os

import numpy as np
import pytest
import scipy.stats

from oracle import sampler as S
from oracle.model import Model
from paper_2507_09252_amd import workloads as W

GAMMA = 3
N_GEN = 2 * GAMMA + 2
TCFG = W.ModelCfg(2, 32, 2, 64, 4, 3, "fp32")
DCFG = W.ModelCfg(1, 16, 1, 32, 4, 3, "fp32")


def _models():
    wt = W.make_weights(TCFG, np.random.SeedSequence([5, 1]), "paper")
    wd = W.make_weights(DCFG, np.random.SeedSequence([5, 2]), "paper")
    wd = W.mismatch_draft(wd, DCFG, np.random.SeedSequence([5, 3]))
    return Model(TCFG, wt), Model(DCFG, wd)


def _history(B):
    rng = np.random.default_rng(0)
    ht, _ = W.hpp(20, 1.0, rng)
    hk = rng.integers(0, 3, 20)
    return np.tile(ht.astype(np.float32), (B, 1)), np.tile(hk.astype(np.int32), (B, 1))


def _chunk(args):
    kind, seq0, B, opts = args
    T, D = _models()
    HT, HK = _history(B)
    if kind == "ar":
        st = S.sample_ar(T, HT, HK, N_GEN, seed=11, seq0=seq0)
    else:
        st = S.sample_sd(T, D, HT, HK, N_GEN, GAMMA, seed=11, seq0=seq0, **opts)
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


def _pvalues(a, b):
    ps = []
    for j in range(N_GEN):
        ps.append(scipy.stats.ks_2samp(a[0][:, j], b[0][:, j]).pvalue)
        tab = np.stack([np.bincount(a[1][:, j], minlength=3), np.bincount(b[1][:, j], minlength=3)])
        ps.append(scipy.stats.chi2_contingency(tab)[1])
    # pooled intervals as well
    ps.append(scipy.stats.ks_2samp(a[0].ravel(), b[0].ravel()).pvalue)
    return np.array(ps)


def _law_check(n):
    ar = _run("ar", n)
    sd = _run("sd", n)
    assert 0.3 < sd[2] < 0.8                 # the mismatched draft keeps alpha away from 1
    ps = _pvalues(ar, sd)
    assert ps.min() > 0.01 / len(ps), ps
    return ar


def test_sd_law_equals_ar():
    ar = _law_check(20000)
    # negative controls fail the same tests
    for opts in ({"literal_alg1": True}, {"resample_from_target": True}):
        bad = _run("sd", 20000, opts)
        ps = _pvalues(ar, bad)
        assert ps.min() < 1e-4, (opts, ps.min())


@pytest.mark.slow
def test_sd_law_equals_ar_1e5():
    _law_check(100000)


def test_draft_equal_target_accepts_all():
    T, _ = _models()
    HT, HK = _history(64)
    st = S.sample_sd(T, T, HT, HK, 20, 4, seed=3)
    assert st.accepted_drafts == st.drafted
    assert np.all(st.rounds_run == 4)          # 5 events per round with the bonus, 20 events


def test_single_type_never_rejects_type():
    tc = W.ModelCfg(1, 16, 2, 32, 3, 1, "fp32")
    T = Model(tc, W.make_weights(tc, np.random.SeedSequence([8, 1]), "stress"))
    D = Model(tc, W.make_weights(tc, np.random.SeedSequence([8, 2]), "stress"))
    HT, HK = _history(200)
    HK[:] = 0
    st = S.prefill(T, D, HT, HK, 30)
    while not np.all(st.done):
        out = S.sd_round(T, D, st, 3, seed=4)
        assert not np.any(out[2]["flags"] & 2)
    assert np.all(st.k[:, 20:50] == 0)
