"""Pins for oracle.sampler: draws, the accept rule and the adjusted distributions.

* mixture sampler (App. A.1): one-sample KS of 10^6 draws against the closed-form
  mixture CDF sum_m w_m Phi((ln tau - mu_m) / sigma_m); M = 1 against scipy's lognorm;
* categorical draws: chi-square against the pmf; the "first index with
  u * C_total < C_m" tie rule on exact boundaries;
* accept rule (§4.3, Algorithm 1): every accept/reject path for gamma <= 3 by
  enumeration of forced test outcomes; P(L = l) = prod_{j<l} a_j (1 - a_l);
* Eq. (4) / App. A.2: the residual type draw makes the output pmf equal to f_T,
  by exhaustive enumeration of the uniform grid;
* Theorem 1 / App. A.2-A.3: acceptance rate per candidate equals
  Z = int max(0, g_T - g_D) (quadrature), the residual draw follows g', and one
  position's combined output follows g_T; redrawing from g_T instead (the
  incorrect scheme of App. A.2) fails the same test.
"""
import numpy as np
import pytest
import scipy.integrate
import scipy.stats

from oracle.numerics import log_softmax
from oracle.philox import word_to_uniform
from oracle import sampler as S

KS_C = 1.36   # 5 % critical constant of the KS statistic


def mixture_cdf(logw, mu, s, tau):
    z = (np.log(tau)[..., None] - mu) / np.exp(s)
    return np.sum(np.exp(logw) * scipy.stats.norm.cdf(z), -1)


def _rand_mix(rng, M, scale=1.0):
    return log_softmax(rng.normal(0, scale, M)), rng.normal(0, 0.8, M), rng.normal(-0.3, 0.3, M)


def test_mixture_sampler_ks():
    rng = np.random.default_rng(0)
    logw, mu, s = _rand_mix(rng, 5)
    n = 10 ** 6
    U = rng.uniform(size=(n, 4))
    logf = np.zeros((n, 1))
    tau, k, _ = S.sample_event(np.broadcast_to(logw, (n, 5)), np.broadcast_to(mu, (n, 5)),
                               np.broadcast_to(s, (n, 5)), logf, U)
    assert np.all(k == 0)
    D = scipy.stats.kstest(tau, lambda x: mixture_cdf(logw, mu, s, x)).statistic
    assert D < KS_C / np.sqrt(n)


def test_single_component_is_lognormal():
    rng = np.random.default_rng(1)
    n = 200000
    U = rng.uniform(size=(n, 4))
    tau, _, _ = S.sample_event(np.zeros((n, 1)), np.full((n, 1), 0.4), np.full((n, 1), np.log(0.7)),
                               np.zeros((n, 1)), U)
    D = scipy.stats.kstest(tau, scipy.stats.lognorm(s=0.7, scale=np.exp(0.4)).cdf).statistic
    assert D < KS_C / np.sqrt(n)


def test_box_muller_normal():
    rng = np.random.default_rng(2)
    u = rng.uniform(size=(2, 200000))
    eps = S.box_muller(u[0], u[1])
    assert scipy.stats.kstest(eps, "norm").statistic < KS_C / np.sqrt(u.shape[1])


def test_categorical_chi2_and_ties():
    rng = np.random.default_rng(3)
    p = rng.dirichlet(np.ones(6))
    n = 200000
    idx, _ = S.categorical(np.broadcast_to(np.log(p), (n, 6)), rng.uniform(size=n))
    obs = np.bincount(idx, minlength=6)
    assert scipy.stats.chisquare(obs, p * n).pvalue > 1e-3
    # exact boundaries: u * C_total == C_m selects m + 1
    q = np.array([0.25, 0.25, 0.5])
    idx, _ = S.categorical(np.broadcast_to(np.log(q), (4, 3)), np.array([0.25, 0.5, 0.2499999, 1e-12]))
    assert list(idx) == [1, 2, 0, 0]


def test_uniform_grid_mean():
    # odd multiples of 2^-24: symmetric grid, mean exactly 1/2
    x = np.arange(0, 1 << 23, dtype=np.uint64) << np.uint64(41)
    u = word_to_uniform(x)
    assert u.min() == 2.0 ** -24 and u.max() == 1 - 2.0 ** -24 and u.mean() == 0.5


# ---------------------------------------------------------------------------
# accept rule
# ---------------------------------------------------------------------------

def _fake_round(rng, B, gamma, M=3, K=3, same=False):
    """State + draft/verify outputs with random (independent per row) mixtures."""
    cap = 8 + gamma + 4
    t = np.zeros((B, cap))
    t[:, :4] = [1.0, 2.0, 3.0, 4.0]
    st = S.State(t=t, k=np.zeros((B, cap), np.int64), n=np.full(B, 4), gen=np.zeros(B, np.int64),
                 n_gen=10 ** 6, tcache=None, dcache=None,
                 log_margin=np.full((B, 10 ** 3), np.inf), cat_margin=np.full((B, 10 ** 3), np.inf),
                 rounds_run=np.zeros(B, np.int64))

    def mix(shape):
        return (log_softmax(rng.normal(0, 0.5, shape + (M,))), rng.normal(0, 0.5, shape + (M,)),
                rng.normal(-0.2, 0.2, shape + (M,)), log_softmax(rng.normal(0, 0.7, shape + (K,))))
    dw, dmu, ds, dlf = mix((B, gamma))
    tw, tmu, ts, tlf = mix((B, gamma + 1))
    if same:
        tw[:, :gamma], tmu[:, :gamma], ts[:, :gamma], tlf[:, :gamma] = dw, dmu, ds, dlf
    tau = rng.lognormal(0, 1, (B, gamma))
    kk = rng.integers(0, K, (B, gamma))
    dr = S.DraftOut(tau=tau, t=4 + np.cumsum(tau, 1), k=kk,
                    logg=S.mixture_logpdf(dw, dmu, ds, tau),
                    logf=np.take_along_axis(dlf, kk[..., None], -1)[..., 0],
                    logw=dw, mu=dmu, s=ds, logtype=dlf, cat_margin=np.full((B, gamma), np.inf))
    vf = S.VerifyOut(logg=S.mixture_logpdf(tw[:, :gamma], tmu[:, :gamma], ts[:, :gamma], tau),
                     logf=np.take_along_axis(tlf[:, :gamma], kk[..., None], -1)[..., 0],
                     logw=tw, mu=tmu, s=ts, logtype=tlf)
    return st, dr, vf


@pytest.mark.parametrize("gamma", [1, 2, 3])
def test_accept_paths_enumerated(gamma):
    """Force every pass/fail pattern of the 2*gamma tests and check L, flags, events."""
    rng = np.random.default_rng(10 + gamma)
    n_pat = 4 ** gamma
    st, dr, vf = _fake_round(rng, n_pat, gamma)
    # every ratio strictly below 1 so both outcomes are reachable
    vf.logg = dr.logg + np.log(rng.uniform(0.2, 0.9, dr.logg.shape))
    vf.logf = dr.logf + np.log(rng.uniform(0.2, 0.9, dr.logf.shape))
    ratio_t, ratio_k = np.exp(vf.logg - dr.logg), np.exp(vf.logf - dr.logf)
    pats = np.array([[(p >> (2 * l + c)) & 1 for l in range(gamma) for c in range(2)]
                     for p in range(n_pat)]).reshape(n_pat, gamma, 2)   # 1 = pass
    u = np.where(pats == 1, 0.5 * np.stack([ratio_t, ratio_k], -1),
                 np.stack([ratio_t, ratio_k], -1) + 0.5 * (1 - np.stack([ratio_t, ratio_k], -1)))
    t_before = st.t[:, 3].copy()
    res = S.accept(st, gamma, dr, vf, seed=7, rows=np.arange(n_pat), ext_uniforms=u)
    for i in range(n_pat):
        ok = pats[i].all(axis=1)
        L = int(np.argmin(ok)) + 1 if not ok.all() else gamma + 1
        assert res["L"][i] == L
        if L <= gamma:
            want_flags = (0 if pats[i, L - 1, 0] else 1) | (0 if pats[i, L - 1, 1] else 2)
            assert res["flags"][i] == want_flags
            assert np.array_equal(res["k_new"][i, :L - 1], dr.k[i, :L - 1])
            assert np.allclose(res["tau_new"][i, :L - 1], dr.tau[i, :L - 1])
            if pats[i, L - 1, 0]:
                assert res["tau_new"][i, L - 1] == dr.tau[i, L - 1]
            if pats[i, L - 1, 1]:
                assert res["k_new"][i, L - 1] == dr.k[i, L - 1]
            assert res["n_new"][i] == L
        else:
            assert res["flags"][i] == 4 and res["n_new"][i] == gamma + 1
        # times are the float32 running sums of the intervals
        tt = t_before[i]
        for j in range(res["n_new"][i]):
            tt = float(np.float32(tt + res["tau_new"][i, j]))
            assert res["t_new"][i, j] == tt


def test_first_rejection_law():
    """P(L = l) = prod_{j<l} a_j (1 - a_l), a_j = min(1, r^tau_j) min(1, r^k_j)."""
    rng = np.random.default_rng(20)
    d_tau = np.array([-0.3, 0.2, -1.0, -0.05])
    d_k = np.array([-0.1, -0.5, 0.0, 0.3])
    a = np.minimum(1, np.exp(d_tau)) * np.minimum(1, np.exp(d_k))
    want = np.array([np.prod(a[:l]) * (1 - a[l]) for l in range(4)] + [np.prod(a)])
    n = 200000
    lu = np.log(rng.uniform(size=(n, 2, 4)))
    Ls = np.array([S.first_rejection(d_tau, d_k, lu[i, 0], lu[i, 1])[0] for i in range(n)])
    obs = np.bincount(Ls, minlength=6)[1:]
    assert scipy.stats.chisquare(obs, want * n).pvalue > 1e-3
    # expected events per round with the bonus: E[L] = sum_{l=0}^{gamma} prod_{j<l} a_j
    assert abs(Ls.mean() - sum(np.prod(a[:l]) for l in range(5))) < 4 * Ls.std() / np.sqrt(n)


def test_residual_type_law_exact():
    """App. A.2: P(out = k) = f_D(k) min(1, f_T/f_D) + (1 - beta_k) f'(k) = f_T(k), on the u grid."""
    rng = np.random.default_rng(30)
    K = 5
    fT, fD = rng.dirichlet(np.ones(K)), rng.dirichlet(np.ones(K))
    grid = word_to_uniform(np.arange(0, 1 << 23, dtype=np.uint64) << np.uint64(41))
    # the residual draw as a function of u, enumerated over every grid value
    k_res, _ = S.resid_type(np.broadcast_to(np.log(fT), (len(grid), K)),
                            np.broadcast_to(np.log(fD), (len(grid), K)), grid)
    p_res = np.bincount(k_res, minlength=K) / len(grid)
    # the accept test for a drafted type k: ln u < log f_T(k) - log f_D(k)
    lg = np.log(grid)
    p_acc = np.array([np.mean(lg < np.log(fT[k]) - np.log(fD[k])) for k in range(K)])
    assert np.allclose(p_acc, np.minimum(1, fT / fD), atol=2.0 ** -22)
    beta = np.sum(fD * p_acc)
    p_out = fD * p_acc + (1 - beta) * p_res
    assert np.allclose(p_out, fT, atol=1e-6)
    # and the residual pmf itself is norm(max(0, f_T - f_D)) (Eq. 4)
    fprime = np.maximum(0, fT - fD) / np.maximum(0, fT - fD).sum()
    assert np.allclose(p_res, fprime, atol=2.0 ** -21)


def _log_grid_cdf(f, lo=-25, hi=25, n=200001):
    x = np.linspace(lo, hi, n)
    dens = f(np.exp(x)) * np.exp(x)
    c = scipy.integrate.cumulative_trapezoid(dens, x, initial=0.0)
    return x, c


def test_theorem1_residual_time():
    rng = np.random.default_rng(40)
    Tw, Tmu, Ts = log_softmax(np.array([0.2, -0.5, 0.1])), np.array([0.3, -0.8, 1.0]), np.log([0.5, 0.7, 0.4])
    Dw, Dmu, Ds = log_softmax(np.array([0.0, 0.3])), np.array([0.9, -1.3]), np.log([0.6, 0.9])

    def gT(x):
        return np.exp(S.mixture_logpdf(Tw, Tmu, Ts, x))

    def gD(x):
        return np.exp(S.mixture_logpdf(Dw, Dmu, Ds, x))

    Z = scipy.integrate.quad(lambda y: max(0.0, gT(np.exp(y)) - gD(np.exp(y))) * np.exp(y), -30, 30,
                             limit=500, points=[-2, -1, 0, 1, 2])[0]
    assert 0.1 < Z < 0.9
    n = 3000
    taus, iters = np.zeros(n), np.zeros(n)
    for b in range(n):
        tau, j, _, _ = S.resid_time(Tw, Tmu, Ts, Dw, Dmu, Ds, seed=5, b=b, r=0)
        taus[b], iters[b] = tau, j
    # candidates per accepted sample ~ Geometric(Z)
    zhat = n / np.sum(iters + 1)
    assert abs(zhat - Z) < 4 * np.sqrt(Z * Z * (1 - Z) / n)
    # accepted candidates ~ g' = norm(max(0, g_T - g_D))
    x, c = _log_grid_cdf(lambda t: np.maximum(0, gT(t) - gD(t)))
    cdf_res = lambda t: np.interp(np.log(t), x, c / c[-1])
    assert scipy.stats.kstest(taus, cdf_res).statistic < KS_C / np.sqrt(n)

    # one position: draft tau ~ g_D accepted w.p. min(1, g_T/g_D), else residual -> g_T
    def one_position(resample_from_target):
        out = np.zeros(n)
        U = rng.uniform(size=(n, 4))
        tau_d, _, _ = S.sample_event(np.broadcast_to(Dw, (n, 2)), np.broadcast_to(Dmu, (n, 2)),
                                     np.broadcast_to(Ds, (n, 2)), np.zeros((n, 1)), U)
        d = S.mixture_logpdf(Tw, Tmu, Ts, tau_d) - S.mixture_logpdf(Dw, Dmu, Ds, tau_d)
        acc = np.log(rng.uniform(size=n)) < d
        for i in range(n):
            if acc[i]:
                out[i] = tau_d[i]
            else:
                out[i] = S.resid_time(Tw, Tmu, Ts, Dw, Dmu, Ds, seed=6, b=i, r=1,
                                      literal_target=resample_from_target)[0]
        return scipy.stats.kstest(out, lambda t: mixture_cdf(Tw, Tmu, Ts, t)).statistic

    assert one_position(False) < KS_C / np.sqrt(n)
    # negative control: redrawing from g_T after a rejection is biased (App. A.2)
    assert one_position(True) > 2 * KS_C / np.sqrt(n)
