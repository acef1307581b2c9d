"""GPU parity of the AttNHP encoder (App. D.4) against the oracle, through the
same C ABI as the THP models (the encoder is a field of the model
configuration): teacher-forced verify (decoder outputs and log-densities at
the oracle's drafts), drafting with an AttNHP draft model (per-step kernels),
end-to-end AR and TPP-SD sampling. Tolerances and the near-tie protocol are
those of test_gpu_parity.py; bf16 uses max(2e-3, twice the drift of a float32
evaluation with the same rounding points).
"""
import numpy as np
import pytest
import torch

from gpu_common import (CAT_TIE, NEAR_TIE, TOL, Case, compare_events, first_fragile, gpu_state, histories,
                        oracle_models, to_dev, weights)
from fp32_emulation import emulated_verify
from oracle import sampler as S
from paper_2507_09252_amd import tppsd as tp
from paper_2507_09252_amd import workloads as W

pytestmark = pytest.mark.gpu

# a small fp32 AttNHP pair beside the bf16 workload a3
A1 = W.Workload("a1", 6, W.ModelCfg(2, 32, 2, 0, 4, 3, "fp32", W.ENC_ATTNHP, 0.5, 20.0),
                W.ModelCfg(1, 16, 1, 0, 4, 3, "fp32", W.ENC_ATTNHP, 0.5, 20.0),
                batch=8, n_gen=64, gammas=(4,), n_hist=20, history="ipp_sin", description="small fp32 AttNHP")
A3 = W.WORKLOADS["a3"]


def case(wl, B, n_hist=None, init="stress", mismatch=True):
    return Case(f"{wl.name}-B{B}-{init}", wl, B, n_hist or wl.n_hist, init, mismatch)


VERIFY_CASES = [case(A1, 6), case(A1, 4, init="bias"), case(A3, 4, n_hist=40, init="bias"), case(A3, 3, n_hist=40)]
RTOL_T = {"fp32": 2e-4, "bf16": 1e-2}


def _gamma(c):
    return min(c.wl.gamma, 10)


@pytest.mark.parametrize("c", VERIFY_CASES, ids=[c.name for c in VERIFY_CASES])
def test_attnhp_verify_teacher_forced(c):
    gamma, n_gen, seed = _gamma(c), 64, 3
    wt, wd = weights(c)
    T, D = oracle_models(c, wt, wd)
    ht, hk = histories(c)
    st_o = S.prefill(T, D, ht, hk, n_gen)
    rows = np.arange(c.B)
    dr = S.draft(D, st_o, gamma, seed, rows)
    vf = S.verify(T, st_o, dr, rows)
    M, K = c.wl.target.n_mix, c.wl.target.n_types
    st = gpu_state(c, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    dbuf = tp.DraftBuffers(c.B, gamma, M, K)
    for f in ("tau", "t", "logg", "logf", "logtype"):
        getattr(dbuf, f).copy_(to_dev(getattr(dr, f).astype(np.float32)))
    dbuf.k.copy_(to_dev(dr.k.astype(np.int32)))
    dbuf.mix.copy_(to_dev(np.stack([dr.logw, dr.mu, dr.s], 2).astype(np.float32)))
    vbuf = tp.VerifyBuffers(c.B, gamma, M, K)
    st.tppsd_verify(gamma, dbuf, vbuf)
    torch.cuda.synchronize()
    assert st.tppsd_state_status()["bits"] == 0
    tol = TOL[c.wl.prec]
    if c.wl.prec == "bf16":
        dr32 = S.DraftOut(**{f: (getattr(dr, f).astype(np.float32).astype(np.float64)
                                 if isinstance(getattr(dr, f), np.ndarray) and getattr(dr, f).dtype.kind == "f"
                                 else getattr(dr, f)) for f in dr.__dataclass_fields__})
        em = emulated_verify(c.wl.target, wt, ht.astype(np.float32), hk, dr32)
        want = (vf.logg, vf.logf, np.stack([vf.logw, vf.mu, vf.s], 2), vf.logtype)
        drift = max(np.abs(a - w).max() for a, w in zip(em, want))
        tol = max(tol, 2 * drift)
    got = (vbuf.logg, vbuf.logf, vbuf.mix, vbuf.logtype)
    want = (vf.logg, vf.logf, np.stack([vf.logw, vf.mu, vf.s], 2), vf.logtype)
    errs = []
    for what, g_, w_ in zip(("log g_T", "log f_T", "mixture", "log f"), got, want):
        g_ = g_.cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(g_)), what
        err = np.abs(g_ - w_).max()
        errs.append(err)
        assert err <= tol, f"{c.name} {what}: err {err:.3g} tol {tol:.3g}"
    print(f"{c.name}: max abs err {max(errs):.2e} (tol {tol:.2e})")


DRAFT_CASES = [case(A1, 8), case(A3, 8, n_hist=40, init="bias")]


@pytest.mark.parametrize("c", DRAFT_CASES, ids=[c.name for c in DRAFT_CASES])
def test_attnhp_draft_parity(c):
    gamma, n_gen, seed = _gamma(c), 64, 13
    wt, wd = weights(c)
    T, D = oracle_models(c, wt, wd)
    ht, hk = histories(c)
    st_o = S.prefill(T, D, ht, hk, n_gen)
    dr = S.draft(D, st_o, gamma, seed, np.arange(c.B))
    st = gpu_state(c, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    M, K = c.wl.target.n_mix, c.wl.target.n_types
    dbuf = tp.DraftBuffers(c.B, gamma, M, K)
    st.tppsd_draft(gamma, dbuf)
    torch.cuda.synchronize()
    tol = TOL[c.wl.prec]
    upto = first_fragile(np.zeros_like(dr.cat_margin) + np.inf, dr.cat_margin, 0.0, max(CAT_TIE, tol))
    g = {f: getattr(dbuf, f).cpu().numpy() for f in ("tau", "t", "k", "logg", "logf")}
    for b in range(c.B):
        u = upto[b]
        assert np.array_equal(g["k"][b, :u], dr.k[b, :u]), b
        np.testing.assert_allclose(g["tau"][b, :u], dr.tau[b, :u], rtol=20 * tol)
        np.testing.assert_allclose(g["logg"][b, :u], dr.logg[b, :u], atol=20 * tol, rtol=tol)
    assert upto.mean() > 0.25 * gamma, upto


E2E_CASES = [case(A1, 4, init="bias"), case(A3, 4, n_hist=30, init="bias")]


@pytest.mark.parametrize("kind", ["ar", "sd"])
@pytest.mark.parametrize("c", E2E_CASES, ids=[c.name for c in E2E_CASES])
def test_attnhp_end_to_end(c, kind):
    gamma, n_gen, seed = _gamma(c), 40, 29
    wt, wd = weights(c)
    T, D = oracle_models(c, wt, wd)
    ht, hk = histories(c)
    n0 = c.n_hist
    if kind == "ar":
        ref = S.sample_ar(T, ht, hk, n_gen, seed)
        st = gpu_state(c, wt, wd, gamma, n_gen, seed, draft=False)
        st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
        st.tppsd_sample_ar(n_gen)
    else:
        ref = S.sample_sd(T, D, ht, hk, n_gen, gamma, seed)
        st = gpu_state(c, wt, wd, gamma, n_gen, seed)
        st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
        st.tppsd_sample_sd(gamma)
    t, k, n = (a.cpu().numpy() for a in st.tppsd_read_events())
    status = st.tppsd_state_status()
    assert status["bits"] == 0 and status["n_done"] == c.B, status
    tol = TOL[c.wl.prec]
    upto = first_fragile(ref.log_margin, ref.cat_margin, tol + NEAR_TIE, max(CAT_TIE, tol))
    frac = compare_events(t[:, n0:n0 + n_gen], k[:, n0:n0 + n_gen], ref.t[:, n0:n0 + n_gen],
                          ref.k[:, n0:n0 + n_gen], upto, rtol=RTOL_T[c.wl.prec])
    print(f"{c.name} {kind}: fully matched {frac:.2f}")
