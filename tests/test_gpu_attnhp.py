"""GPU parity of the AttNHP encoder (App. D.4) against the oracle, through the
same C ABI as the THP models (the encoder is a field of the model
configuration): teacher-forced verify (decoder outputs and log-densities at
the oracle's drafts), drafting with an AttNHP draft model (per-step kernels),
end-to-end AR and TPP-SD sampling replayed step by step / round by round.
Tolerances and the near-tie protocol are those of test_gpu_parity.py (fixed
per workload: 1e-5 fp32, 2e-3 for the bf16 workload).
"""
import numpy as np
import pytest
import torch

from gpu_common import (EMU_DRIFT_MAX, STRESS_BF16_TOL, Case, check_draft_record, check_verify, draft_buffers_from_oracle,
                        draft_out, f32_round, gpu_state, histories, oracle_models, replay_ar_steps, replay_sd_rounds,
                        to_dev, tol_of, verify_out, weights)
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


@pytest.mark.parametrize("c", VERIFY_CASES, ids=[c.name for c in VERIFY_CASES])
def test_attnhp_verify_teacher_forced(c):
    gamma, n_gen, seed = c.g, 64, 3
    wt, wd = weights(c)
    T, D = oracle_models(c, wt, wd)
    ht, hk = histories(c)
    st_o = S.prefill(T, D, ht, hk, n_gen)
    rows = np.arange(c.B)
    dr = S.draft(D, st_o, gamma, seed, rows)
    vf = S.verify(T, st_o, dr, rows)
    M, K = c.wl.target.n_mix, c.wl.target.n_types
    print(f"{c.name}: gamma {gamma}", flush=True)
    st = gpu_state(c, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    dbuf = draft_buffers_from_oracle(dr, c.B, gamma, M, K)
    vbuf = tp.VerifyBuffers(c.B, gamma, M, K)
    st.tppsd_verify(gamma, dbuf, vbuf)
    torch.cuda.synchronize()
    assert st.tppsd_state_status()["bits"] == 0
    tol = tol_of(c.wl)
    stress = c.init == "stress" and c.wl.prec == "bf16"
    dr32 = S.DraftOut(**{f: f32_round(getattr(dr, f)) for f in dr.__dataclass_fields__})
    err = check_verify(verify_out(vbuf, rows, gamma), vf, tol, c.name, stress, dr32)
    msg = f"{c.name}: max abs err {err:.2e} (tol {STRESS_BF16_TOL if stress else tol:.1e})"
    if c.wl.prec == "bf16":
        em = emulated_verify(c.wl.target, wt, ht.astype(np.float32), hk, dr32)
        pairs = list(zip(em, (vf.logg, vf.logf, np.stack([vf.logw, vf.mu, vf.s], 2), vf.logtype)))
        drift = max(np.abs(a - w).max() for a, w in (pairs[2:] if stress else pairs))
        assert drift <= (STRESS_BF16_TOL if stress else EMU_DRIFT_MAX[c.wl.name]), drift
        msg += f"; float32-emulation drift {drift:.2e}"
    print(msg)


DRAFT_CASES = [case(A1, 8), case(A3, 8, n_hist=40, init="bias")]


@pytest.mark.parametrize("c", DRAFT_CASES, ids=[c.name for c in DRAFT_CASES])
def test_attnhp_draft_parity(c):
    gamma, n_gen, seed = c.g, 64, 13
    wt, wd = weights(c)
    T, D = oracle_models(c, wt, wd)
    ht, hk = histories(c)
    print(f"{c.name}: gamma {gamma}", flush=True)
    st = gpu_state(c, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    M, K = c.wl.target.n_mix, c.wl.target.n_types
    dbuf = tp.DraftBuffers(c.B, gamma, M, K)
    st.tppsd_draft(gamma, dbuf)
    torch.cuda.synchronize()
    rows = np.arange(c.B)
    ost = S.prefill(T, D, ht, hk, n_gen)
    compared = check_draft_record(D, ost, draft_out(dbuf, rows, gamma), gamma, seed, 0, rows, tol_of(c.wl), c.name)
    assert compared >= 0.9 * c.B * gamma, compared
    print(f"{c.name}: {compared} of {c.B * gamma} draws compared")


E2E_CASES = [case(A1, 4, init="bias"), case(A3, 4, n_hist=30, init="bias")]
E2E_FLOOR = 0.5


@pytest.mark.parametrize("kind", ["ar", "sd"])
@pytest.mark.parametrize("c", E2E_CASES, ids=[c.name for c in E2E_CASES])
def test_attnhp_end_to_end(c, kind):
    """GPU AR (step by step) and TPP-SD (round by round), each step or round
    replayed into the oracle from the events the GPU had committed."""
    gamma, n_gen, seed = c.g, 32, 29
    wt, wd = weights(c)
    T, D = oracle_models(c, wt, wd)
    ht, hk = histories(c)
    print(f"{c.name}: {kind}, {n_gen} events", flush=True)
    if kind == "ar":
        st = gpu_state(c, wt, wd, gamma, n_gen, seed, draft=False)
        st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
        compared, generated = replay_ar_steps(c, T, st, seed, n_gen)
    else:
        st = gpu_state(c, wt, wd, gamma, n_gen, seed)
        st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
        compared, generated, _, _, _ = replay_sd_rounds(c, T, D, st, gamma, seed, n_gen)
    status = st.tppsd_state_status()
    assert status["bits"] == 0 and status["n_done"] == c.B, status
    assert generated == c.B * n_gen
    assert compared >= E2E_FLOOR * generated, (compared, generated)
    print(f"{c.name} {kind}: events compared {compared}/{generated}")
