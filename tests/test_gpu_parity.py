"""GPU parity: HIP path through the C ABI vs the CPU oracle, same weights,
histories and Philox seed.

Teacher-forced per call (primary): verify on the oracle's drafts; accept on the
oracle's draft and verify outputs; draft from the same prefilled state.
End to end (secondary): AR and SD sampling, compared event by event up to each
sequence's first decision inside the near-tie window.

Tolerances: log-densities and decoder outputs within 1e-5 (fp32) or 2e-3
(bf16) absolute (plus the same relative amount for the large-activation
"stress" weights); accept decisions, L, flags and A-R indices bit-exact except
at near-ties |ln u - (log p_T - log p_D)| < 1e-4 (categorical: within 1e-5 of
the total mass); residual and bonus intervals within 2e-6 relative.
"""
import numpy as np
import pytest
import torch

from gpu_common import (CAT_TIE, NEAR_TIE, TOL, compare_events, draft_buffers_from_oracle, first_fragile,
                        gpu_state, histories, oracle_models, small, to_dev, verify_buffers_from_oracle, weights)
from fp32_emulation import emulated_verify
from oracle import sampler as S
from paper_2507_09252_amd import tppsd as tp

pytestmark = pytest.mark.gpu

VERIFY_CASES = [
    small("c1", 3, init="paper", mismatch=False),
    small("c1", 5),
    small("c2", 6),
    small("c2", 4, init="paper", mismatch=False),
    # 517 rows: the fp32 d = 64 / F = 256 target takes the row-block kernel
    # (packed weights) from 512 rows; 33 tiles of 16, the last ragged
    small("c2", 47, init="bias"),
    small("c3", 5, n_hist=40, init="bias"),
    small("c3", 3, n_hist=40, init="paper", mismatch=False),
    small("c3", 3, n_hist=40),
    small("c4", 2, n_hist=70, init="bias"),
    small("c4", 2, n_hist=70, init="paper", mismatch=False),
    small("c5", 9, init="bias"),
    small("c5", 5),
    # long histories over few (sequence, head) pairs: the key range is split
    # across workgroups and the partials merged
    small("c1", 2, n_hist=1100),
    small("c2", 2, n_hist=1100),
    small("c3", 1, n_hist=1100, init="bias"),
]

# bf16 with the large-activation "stress" weights: a float32-accumulating
# implementation with the oracle's bf16 rounding points drifts from the
# float64 oracle by up to ~2e-2 on decoder outputs (rounding flips); this
# bound still catches a wrong bias, gain, index or layout (O(0.1-1) errors).
BF16_STRESS_TOL = 0.1


def _ids(cases):
    return [c.name for c in cases]


def _gamma(case):
    return min(case.wl.gamma, 10)


def _oracle_round(case, wt, wd, gamma, n_gen, seed):
    T, D = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    st = S.prefill(T, D, ht, hk, n_gen)
    rows = np.arange(case.B)
    dr = S.draft(D, st, gamma, seed, rows)
    vf = S.verify(T, st, dr, rows)
    return T, D, ht, hk, st, dr, vf


def _close(got, want, tol, stress, what):
    got = got.detach().cpu().numpy().astype(np.float64)
    rtol = tol if stress else 0.0
    err = np.abs(got - want) - rtol * np.abs(want)
    assert np.all(np.isfinite(got)), what
    assert err.max() <= tol, f"{what}: max abs err {np.abs(got - want).max():.3g} (tol {tol})"
    return np.abs(got - want).max()


@pytest.mark.parametrize("case", VERIFY_CASES, ids=_ids(VERIFY_CASES))
def test_verify_teacher_forced(case):
    gamma, n_gen, seed = _gamma(case), 64, 11
    wt, wd = weights(case)
    T, D, ht, hk, st_o, dr, vf = _oracle_round(case, wt, wd, gamma, n_gen, seed)
    M, K = case.wl.target.n_mix, case.wl.target.n_types
    st = gpu_state(case, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    dbuf = draft_buffers_from_oracle(dr, case.B, gamma, M, K)
    vbuf = tp.VerifyBuffers(case.B, gamma, M, K)
    st.tppsd_verify(gamma, dbuf, vbuf)
    torch.cuda.synchronize()
    tol = TOL[case.wl.prec]
    stress = case.init == "stress"
    if stress and case.wl.prec == "bf16":
        tol = BF16_STRESS_TOL
    elif case.wl.prec == "bf16":
        # floor 2e-3; above it, twice the drift of an exact float32 evaluation
        em = emulated_verify(case.wl.target, wt, ht, hk, dr)
        drift = max(np.abs(a - b).max() for a, b in
                    zip(em, (vf.logg, vf.logf, np.stack([vf.logw, vf.mu, vf.s], 2), vf.logtype)))
        tol = max(tol, 2 * drift)
        print(f"{case.name}: float32-emulation drift {drift:.2e}, tolerance {tol:.2e}")
    e1 = _close(vbuf.logg, vf.logg, tol, stress, "log g_T")
    e2 = _close(vbuf.logf, vf.logf, tol, stress, "log f_T")
    e3 = _close(vbuf.mix, np.stack([vf.logw, vf.mu, vf.s], 2), tol, stress, "mixture params")
    e4 = _close(vbuf.logtype, vf.logtype, tol, stress, "log f")
    assert st.tppsd_state_status()["bits"] == 0
    print(f"{case.name}: max abs err logg {e1:.2e} logf {e2:.2e} mix {e3:.2e} logtype {e4:.2e}")


# the row-local part of each layer as one launch (output projection, FFN
# with its hidden activations on chip, next layer's q, k, v), forced at these
# small sizes: several row tiles with a ragged last one
FFN_FUSED_CASES = [small("c3", 5, n_hist=40, init="bias"), small("c3", 3, n_hist=40, init="paper", mismatch=False),
                   small("c5", 9, init="bias"), small("c5", 5)]


@pytest.mark.parametrize("case", FFN_FUSED_CASES, ids=_ids(FFN_FUSED_CASES))
def test_verify_fused_layer(case, monkeypatch):
    monkeypatch.setenv("TPPSD_FFN_FUSED", "1")
    test_verify_teacher_forced(case)


# the row-block kernel with four waves instead of its default eight (the
# 517-row fp32 pass runs it; the d = 32 drafts' per-step kernels too)
BLOCK_NT_CASES = [small("c2", 47, init="bias")]


@pytest.mark.parametrize("case", BLOCK_NT_CASES, ids=_ids(BLOCK_NT_CASES))
def test_verify_block_four_waves(case, monkeypatch):
    monkeypatch.setenv("TPPSD_BLOCK_NT", "256")
    test_verify_teacher_forced(case)


ACCEPT_CASES = [small("c1", 64), small("c3", 48, n_hist=30, init="bias"), small("c5", 96, init="bias")]


@pytest.mark.parametrize("external", [False, True])
@pytest.mark.parametrize("case", ACCEPT_CASES, ids=_ids(ACCEPT_CASES))
def test_accept_teacher_forced(case, external):
    gamma, n_gen, seed = _gamma(case), 64, 5
    wt, wd = weights(case)
    T, D, ht, hk, st_o, dr, vf = _oracle_round(case, wt, wd, gamma, n_gen, seed)
    # the GPU receives exactly the values the oracle decides on (rounded to float32)
    r32 = lambda a: a.astype(np.float32).astype(np.float64) if isinstance(a, np.ndarray) and a.dtype.kind == "f" else a
    dr32 = S.DraftOut(**{f: r32(getattr(dr, f)) for f in dr.__dataclass_fields__})
    vf32 = S.VerifyOut(**{f: getattr(vf, f).astype(np.float32).astype(np.float64) for f in vf.__dataclass_fields__})
    rows = np.arange(case.B)
    ext = None
    if external:
        ext = np.random.default_rng(3).integers(1, 1 << 23, size=(case.B, gamma, 2)) * 2.0 ** -23
    res = S.accept(st_o, gamma, dr32, vf32, seed, rows, ext_uniforms=ext)
    M, K = case.wl.target.n_mix, case.wl.target.n_types
    st = gpu_state(case, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    dbuf = draft_buffers_from_oracle(dr32, case.B, gamma, M, K)
    vbuf = verify_buffers_from_oracle(vf32, case.B, gamma, M, K)
    abuf = tp.AcceptBuffers(case.B, gamma)
    ub = to_dev(ext.astype(np.float32)) if external else None
    st.tppsd_accept(gamma, dbuf, vbuf, abuf, uniforms=ub)
    t, k, n = st.tppsd_read_events()
    torch.cuda.synchronize()
    L = abuf.L.cpu().numpy()
    flags = abuf.flags.cpu().numpy()
    ar = abuf.ar_iter.cpu().numpy()
    nn = abuf.n_new.cpu().numpy()
    kn = abuf.k_new.cpu().numpy()
    taun = abuf.tau_new.cpu().numpy()
    n0 = case.n_hist
    fragile = (st_o.log_margin[:, 0:gamma + 1].min(1) < NEAR_TIE) | (st_o.cat_margin[:, 0:gamma + 1].min(1) < CAT_TIE)
    checked = 0
    for b in range(case.B):
        if fragile[b]:
            continue
        checked += 1
        assert L[b] == res["L"][b], (b, L[b], res["L"][b])
        assert flags[b] & 7 == res["flags"][b], b
        assert ar[b] == res["ar_iter"][b], b
        assert nn[b] == res["n_new"][b], b
        m = nn[b]
        assert np.array_equal(kn[b, :m], res["k_new"][b, :m]), b
        np.testing.assert_allclose(taun[b, :m], res["tau_new"][b, :m], rtol=2e-6)
        assert np.array_equal(k.cpu().numpy()[b, n0:n0 + m], res["k_new"][b, :m])
        assert int(n.cpu()[b]) == n0 + m
    assert checked >= 0.9 * case.B
    # the batch exercises both residual draws
    assert np.any(res["flags"] & 1)
    assert np.any(res["flags"] & 2) or case.wl.target.n_types == 1
    print(f"{case.name}: checked {checked}/{case.B}; L histogram {np.bincount(res['L'])}")


DRAFT_CASES = [small("c1", 8), small("c2", 8), small("c3", 16, n_hist=40, init="bias"), small("c5", 16, init="bias"),
               small("c4", 4, n_hist=40, init="bias")]


# both drafting paths: one workgroup per sequence for all gamma steps (where
# the draft model fits it), and per-step batched kernels
@pytest.mark.parametrize("layered", [False, True], ids=["fused", "layered"])
@pytest.mark.parametrize("case", DRAFT_CASES, ids=_ids(DRAFT_CASES))
def test_draft_parity(case, layered, monkeypatch):
    monkeypatch.setenv("TPPSD_LAYERED_DRAFT", "1" if layered else "0")
    _draft_parity(case)


def _draft_parity(case):
    gamma, n_gen, seed = _gamma(case), 64, 13
    wt, wd = weights(case)
    T, D, ht, hk, st_o, dr, vf = _oracle_round(case, wt, wd, gamma, n_gen, seed)
    M, K = case.wl.target.n_mix, case.wl.target.n_types
    st = gpu_state(case, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    dbuf = tp.DraftBuffers(case.B, gamma, M, K)
    st.tppsd_draft(gamma, dbuf)
    torch.cuda.synchronize()
    tol = TOL[case.wl.prec]
    upto = first_fragile(np.zeros_like(dr.cat_margin) + np.inf, dr.cat_margin, 0.0, max(CAT_TIE, tol))
    g = {f: getattr(dbuf, f).cpu().numpy() for f in ("tau", "t", "k", "logg", "logf")}
    for b in range(case.B):
        u = upto[b]
        assert np.array_equal(g["k"][b, :u], dr.k[b, :u]), b
        np.testing.assert_allclose(g["tau"][b, :u], dr.tau[b, :u], rtol=20 * tol)
        np.testing.assert_allclose(g["t"][b, :u], dr.t[b, :u], rtol=20 * tol)
        np.testing.assert_allclose(g["logg"][b, :u], dr.logg[b, :u], atol=20 * tol, rtol=tol)
        np.testing.assert_allclose(g["logf"][b, :u], dr.logf[b, :u], atol=tol, rtol=tol)
    # categorical near-ties cut the comparison; most draft positions are still compared
    assert upto.mean() > 0.25 * gamma, upto


# the per-step draft's row-block kernel with four waves (4096-sequence drafts
# run it at d = 32)
@pytest.mark.parametrize("case", [DRAFT_CASES[3]], ids=_ids(DRAFT_CASES[3:4]))
def test_draft_block_four_waves(case, monkeypatch):
    monkeypatch.setenv("TPPSD_BLOCK_NT", "256")
    monkeypatch.setenv("TPPSD_LAYERED_DRAFT", "1")
    _draft_parity(case)


# end to end on paper-scale weights: the sampled times feed back through the
# time encoding, and large weights would amplify float32-vs-float64 time
# differences into decision flips long before any defect shows
# event times: the interval error is about (1 + |sigma eps|) times the
# parameter error, and times are running sums of intervals
RTOL_T = {"fp32": 2e-4, "bf16": 1e-2}
E2E_CASES = [small("c1", 4, init="bias"), small("c2", 8, init="bias"), small("c3", 4, n_hist=30, init="bias"),
             small("c5", 16, init="bias")]


@pytest.mark.parametrize("case", E2E_CASES, ids=_ids(E2E_CASES))
def test_ar_end_to_end(case):
    n_gen, seed = 40, 21
    wt, wd = weights(case)
    T, D = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    ref = S.sample_ar(T, ht, hk, n_gen, seed)
    st = gpu_state(case, wt, wd, 1, n_gen, seed, draft=False)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    t_out = torch.zeros(case.B, n_gen, dtype=torch.float32, device="cuda")
    k_out = torch.zeros(case.B, n_gen, dtype=torch.int32, device="cuda")
    st.tppsd_sample_ar(n_gen, t_out, k_out)
    status = st.tppsd_state_status()
    assert status["bits"] == 0 and status["n_done"] == case.B
    tol = TOL[case.wl.prec]
    n0 = case.n_hist
    upto = first_fragile(ref.log_margin, ref.cat_margin, NEAR_TIE, max(CAT_TIE, tol))
    frac = compare_events(t_out.cpu().numpy(), k_out.cpu().numpy(), ref.t[:, n0:n0 + n_gen], ref.k[:, n0:n0 + n_gen],
                          upto, rtol=RTOL_T[case.wl.prec])
    print(f"{case.name}: fully matched sequences {frac:.2f}")


@pytest.mark.parametrize("bonus", [True, False])
@pytest.mark.parametrize("case", E2E_CASES, ids=_ids(E2E_CASES))
def test_sd_end_to_end(case, bonus):
    gamma, n_gen, seed = _gamma(case), 48, 17
    wt, wd = weights(case)
    T, D = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    ref = S.sample_sd(T, D, ht, hk, n_gen, gamma, seed, bonus=bonus)
    st = gpu_state(case, wt, wd, gamma, n_gen, seed, bonus=bonus)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    rounds = st.tppsd_sample_sd(gamma)
    t, k, n = st.tppsd_read_events()
    status = st.tppsd_state_status()
    assert status["bits"] == 0 and status["n_done"] == case.B, status
    assert np.all(n.cpu().numpy() == case.n_hist + n_gen)
    tol = TOL[case.wl.prec]
    n0 = case.n_hist
    upto = first_fragile(ref.log_margin, ref.cat_margin, tol + NEAR_TIE, max(CAT_TIE, tol))
    frac = compare_events(t.cpu().numpy()[:, n0:n0 + n_gen], k.cpu().numpy()[:, n0:n0 + n_gen],
                          ref.t[:, n0:n0 + n_gen], ref.k[:, n0:n0 + n_gen], upto, rtol=RTOL_T[case.wl.prec])
    # accounting agrees with the oracle when every sequence matched fully
    if frac == 1.0:
        assert status["accepted"] == ref.accepted_drafts and status["drafted"] == ref.drafted
    print(f"{case.name} bonus={bonus}: rounds {rounds}, fully matched {frac:.2f}, "
          f"alpha {status['accepted'] / max(1, status['drafted']):.3f}")
