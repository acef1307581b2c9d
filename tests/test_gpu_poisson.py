"""GPU parity of the homogeneous-Poisson draft (App. D.3) against the oracle.

- fit: rate and log p from the device fit against the oracle's float64 fit;
- drafting: same prefilled state, Philox counters and (float32) parameters;
  intervals, times and log-densities within a few float32 ulps, types
  bit-exact outside the categorical near-tie window;
- accept, teacher-forced on the oracle's Poisson draft and verify outputs
  (rounded to float32): decisions, L, flags and Theorem-1 candidate indices
  bit-exact outside the near-tie windows (the Theorem-1 loop runs with the
  exponential draft density here);
- end to end: TPP-SD rounds with the Poisson draft against the oracle's
  sampler, event by event up to each sequence's first near-tie decision.
The parameters handed to both sides come from the oracle's fit, rounded to
float32.
"""
import numpy as np
import pytest
import torch

from gpu_common import (CAT_TIE, NEAR_TIE, compare_events, first_fragile, gpu_state, histories, tol_of,
                        oracle_models, small, to_dev, verify_buffers_from_oracle, weights)
from oracle import sampler as S
from paper_2507_09252_amd import tppsd as tp

pytestmark = pytest.mark.gpu

RTOL_T = {"fp32": 2e-4, "bf16": 1e-2}


def _params(ht, hk, K):
    """Oracle fit rounded to float32: (rate, log p) as float64 values and the device tensor."""
    rate, logp = S.poisson_fit(ht, hk, K)
    rate32 = float(np.float32(rate))
    logp32 = logp.astype(np.float32).astype(np.float64)
    dev = to_dev(np.concatenate([[rate32], logp32]).astype(np.float32))
    return rate32, logp32, dev


FIT_CASES = [(small("c1", 8), False), (small("c3", 64, n_hist=40), False), (small("c5", 300), False),
             (small("c3", 64, n_hist=40), True), (small("c5", 300), True)]


@pytest.mark.parametrize("case,unseen", FIT_CASES,
                         ids=[c.name + ("-unseen-type" if u else "") for c, u in FIT_CASES])
def test_poisson_fit(case, unseen):
    K = case.wl.target.n_types
    ht, hk = histories(case)
    if unseen:
        hk = np.where(hk == K - 1, 0, hk)   # type K - 1 never occurs: log p = -inf
    got = tp.tppsd_poisson_fit(to_dev(ht), to_dev(hk.astype(np.int32)), K).cpu().numpy()
    rate, logp = S.poisson_fit(ht.astype(np.float64), hk, K)
    np.testing.assert_allclose(got[0], rate, rtol=1e-6)
    fin = np.isfinite(logp)
    assert np.array_equal(np.isfinite(got[1:]), fin)
    np.testing.assert_allclose(got[1:][fin], logp[fin], rtol=1e-6, atol=1e-7)
    if unseen:
        assert got[K] == -np.inf


DRAFT_CASES = [small("c1", 16), small("c3", 48, n_hist=40, init="bias"), small("c5", 64, init="bias")]


@pytest.mark.parametrize("case", DRAFT_CASES, ids=[c.name for c in DRAFT_CASES])
def test_draft_poisson_parity(case):
    gamma, n_gen, seed = min(case.wl.gamma, 10), 64, 31
    wt, wd = weights(case)
    T, _ = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    K, M = case.wl.target.n_types, case.wl.target.n_mix
    rate, logp, params = _params(ht, hk, K)
    st_o = S.prefill(T, None, ht, hk, n_gen)
    rows = np.arange(case.B)
    dr = S.draft_poisson(st_o, gamma, rate, logp, seed, rows)
    st = gpu_state(case, wt, wd, gamma, n_gen, seed, draft=False)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    dbuf = tp.DraftBuffers(case.B, gamma, M, K, poisson=True)
    st.tppsd_draft_poisson(gamma, params, dbuf)
    torch.cuda.synchronize()
    assert st.tppsd_state_status()["bits"] == 0
    g = {f: getattr(dbuf, f).cpu().numpy() for f in ("tau", "t", "k", "logg", "logf", "logtype", "rate")}
    # positions are independent draws: every position is compared, types
    # outside the categorical near-tie window
    sure = dr.cat_margin >= CAT_TIE
    assert sure.mean() > 0.99
    assert np.array_equal(g["k"][sure], dr.k[sure])
    np.testing.assert_allclose(g["tau"], dr.tau, rtol=4e-7)
    np.testing.assert_allclose(g["t"], dr.t, rtol=1e-6)
    np.testing.assert_allclose(g["logg"], dr.logg, rtol=1e-6, atol=1e-5)
    np.testing.assert_array_equal(g["logf"][sure], dr.logf[sure].astype(np.float32))
    np.testing.assert_array_equal(g["logtype"], np.broadcast_to(logp.astype(np.float32), g["logtype"].shape))
    np.testing.assert_array_equal(g["rate"], np.full(case.B, np.float32(rate)))


ACCEPT_CASES = [small("c1", 64), small("c3", 48, n_hist=30, init="bias"), small("c5", 96, init="bias")]


@pytest.mark.parametrize("case", ACCEPT_CASES, ids=[c.name for c in ACCEPT_CASES])
def test_accept_poisson_teacher_forced(case):
    gamma, n_gen, seed = min(case.wl.gamma, 10), 64, 7
    wt, wd = weights(case)
    T, _ = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    K, M = case.wl.target.n_types, case.wl.target.n_mix
    rate, logp, params = _params(ht, hk, K)
    st_o = S.prefill(T, None, ht, hk, n_gen)
    rows = np.arange(case.B)
    dr = S.draft_poisson(st_o, gamma, rate, logp, seed, rows)
    vf = S.verify(T, st_o, dr, rows)
    # the GPU receives exactly the values the oracle decides on (rounded to float32)
    r32 = lambda a: a.astype(np.float32).astype(np.float64) if a.dtype.kind == "f" else a
    dr32 = S.DraftOut(**{f: (r32(getattr(dr, f)) if isinstance(getattr(dr, f), np.ndarray) else getattr(dr, f))
                         for f in dr.__dataclass_fields__})
    vf32 = S.VerifyOut(**{f: r32(getattr(vf, f)) for f in vf.__dataclass_fields__})
    res = S.accept(st_o, gamma, dr32, vf32, seed, rows)
    st = gpu_state(case, wt, wd, gamma, n_gen, seed, draft=False)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    dbuf = tp.DraftBuffers(case.B, gamma, M, K, poisson=True)
    for f in ("tau", "t", "logg", "logf", "logtype"):
        getattr(dbuf, f).copy_(to_dev(getattr(dr32, f).astype(np.float32)))
    dbuf.k.copy_(to_dev(dr32.k.astype(np.int32)))
    dbuf.rate.fill_(rate)
    vbuf = verify_buffers_from_oracle(vf32, case.B, gamma, M, K)
    abuf = tp.AcceptBuffers(case.B, gamma)
    st.tppsd_accept(gamma, dbuf, vbuf, abuf)
    t, k, n = st.tppsd_read_events()
    torch.cuda.synchronize()
    assert st.tppsd_state_status()["bits"] == 0
    got = {f: getattr(abuf, f).cpu().numpy() for f in ("L", "flags", "ar_iter", "n_new", "k_new", "tau_new")}
    n0 = case.n_hist
    fragile = (st_o.log_margin[:, 0:gamma + 1].min(1) < NEAR_TIE) | (st_o.cat_margin[:, 0:gamma + 1].min(1) < CAT_TIE)
    checked = 0
    for b in range(case.B):
        if fragile[b]:
            continue
        checked += 1
        assert got["L"][b] == res["L"][b], (b, got["L"][b], res["L"][b])
        assert got["flags"][b] & 7 == res["flags"][b], b
        assert got["ar_iter"][b] == res["ar_iter"][b], b
        m = got["n_new"][b]
        assert m == res["n_new"][b], b
        assert np.array_equal(got["k_new"][b, :m], res["k_new"][b, :m]), b
        np.testing.assert_allclose(got["tau_new"][b, :m], res["tau_new"][b, :m], rtol=2e-6)
        assert np.array_equal(k.cpu().numpy()[b, n0:n0 + m], res["k_new"][b, :m])
    assert checked >= 0.9 * case.B
    assert np.any(res["flags"] & 1), "no interval was redrawn: the exponential g_D path was not exercised"
    print(f"{case.name}: checked {checked}/{case.B}; L histogram {np.bincount(res['L'])}; "
          f"A-R candidates {np.sum(res['ar_iter'] + 1)}")


E2E_CASES = [small("c1", 4, init="bias"), small("c2", 8, init="bias"), small("c3", 4, n_hist=30, init="bias"),
             small("c5", 16, init="bias")]


@pytest.mark.parametrize("bonus", [True, False])
@pytest.mark.parametrize("case", E2E_CASES, ids=[c.name for c in E2E_CASES])
def test_sd_poisson_end_to_end(case, bonus):
    gamma, n_gen, seed = min(case.wl.gamma, 10), 48, 19
    wt, wd = weights(case)
    T, _ = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    K = case.wl.target.n_types
    rate, logp, params = _params(ht, hk, K)
    ref = S.sample_sd_poisson(T, ht, hk, n_gen, gamma, rate, logp, seed, bonus=bonus)
    st = gpu_state(case, wt, wd, gamma, n_gen, seed, bonus=bonus, draft=False)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    rounds = st.tppsd_sample_sd_poisson(gamma, params)
    t, k, n = st.tppsd_read_events()
    status = st.tppsd_state_status()
    assert status["bits"] == 0 and status["n_done"] == case.B, status
    assert np.all(n.cpu().numpy() == case.n_hist + n_gen)
    tol = tol_of(case.wl)
    n0 = case.n_hist
    upto = first_fragile(ref.log_margin, ref.cat_margin, tol + NEAR_TIE, max(CAT_TIE, tol))
    frac = compare_events(t.cpu().numpy()[:, n0:n0 + n_gen], k.cpu().numpy()[:, n0:n0 + n_gen],
                          ref.t[:, n0:n0 + n_gen], ref.k[:, n0:n0 + n_gen], upto, rtol=RTOL_T[case.wl.prec])
    if frac == 1.0:
        assert status["accepted"] == ref.accepted_drafts and status["drafted"] == ref.drafted
    print(f"{case.name} bonus={bonus}: rounds {rounds}, fully matched {frac:.2f}, "
          f"alpha {status['accepted'] / max(1, status['drafted']):.3f}")


def test_poisson_buffer_checks():
    case = small("c1", 4)
    wt, wd = weights(case)
    K, M = case.wl.target.n_types, case.wl.target.n_mix
    st = gpu_state(case, wt, wd, 4, 8, 1)
    ht, hk = histories(case)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), 8)
    params = tp.tppsd_poisson_fit(to_dev(ht), to_dev(hk.astype(np.int32)), K)
    with pytest.raises(tp.TppsdError, match="E_ARG"):
        st.tppsd_draft(4, tp.DraftBuffers(4, 4, M, K, poisson=True))      # a Poisson record to the model draft
    with pytest.raises(tp.TppsdError, match="E_ARG"):
        st.tppsd_draft_poisson(4, params, tp.DraftBuffers(4, 4, M, K))    # no rate array
    with pytest.raises(tp.TppsdError, match="E_ARG"):
        tp.tppsd_poisson_fit(to_dev(ht[:, :1]), to_dev(hk[:, :1].astype(np.int32)), K)   # n0 < 2
    # after Poisson rounds the draft model's cache is stale
    st.tppsd_sample_sd_poisson(4, params, max_rounds=1)
    with pytest.raises(tp.TppsdError, match="E_ORDER"):
        st.tppsd_sample_sd(4)
