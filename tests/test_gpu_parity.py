"""GPU parity: HIP path through the C ABI vs the CPU oracle, same weights,
histories and Philox seed.

Teacher-forced per call (primary): verify on the oracle's drafts; accept on the
oracle's draft and verify outputs; drafting checked against the oracle's draft
model on the GPU's own drafted prefix. Every case runs at its workload's draft
length (c3 also over its whole sweep, and one case at the largest supported
draft length, 32, whose 33 verify positions take three query tiles).
End to end (secondary): AR and TPP-SD sampling run on the GPU step by step /
round by round, and every step or round is replayed into the oracle from the
events the GPU had committed before it (draft record, verify outputs and
accept decisions compared), with a floor on the share of events compared.

Tolerances (fixed per workload, tests/gpu_common.py): decoder outputs and
log-densities within 1e-5 (fp32), 2e-3 (bf16) or 4e-3 (the 8-layer d = 512
workload); accept decisions, L, flags and A-R indices bit-exact except at
near-ties |ln u - (log p_T - log p_D)| < 1e-4 (categorical: within 1e-5 of the
total mass); residual and bonus intervals within 2e-6 relative.
"""
import numpy as np
import pytest
import torch

from gpu_common import (CAT_TIE, EMU_DRIFT_MAX, NEAR_TIE, STRESS_BF16_TOL, Case, check_close, check_draft_record, check_verify,
                        draft_buffers_from_oracle, draft_out, f32_round, gpu_state, histories, oracle_models,
                        replay_ar_steps, replay_sd_rounds, small, to_dev, tol_of, verify_buffers_from_oracle,
                        verify_out, weights)
from fp32_emulation import emulated_verify
from oracle import sampler as S
from paper_2507_09252_amd import tppsd as tp
from paper_2507_09252_amd import workloads as W

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
    # 32 x 17 = 544 rows of width 512: LayerNorm runs as its own launch ahead
    # of the direct-to-LDS GEMMs
    small("c4", 32, n_hist=40, init="bias"),
    small("c5", 9, init="bias"),
    small("c5", 5),
    # 256 x 9 = 2304 rows of width 128: LayerNorm-operand products over many
    # 64 x 64 tiles, below the fused layer kernel's row threshold
    small("c5", 256, init="bias"),
    # long histories over few (sequence, head) pairs: the key range is split
    # across workgroups and the partials merged (fp32; bf16 with four or more
    # splits), or, where two bf16 splits would do, one workgroup of eight
    # waves merges in LDS (c3: one query tile of d_head 32; c4: two of 64)
    small("c1", 2, n_hist=1100),
    small("c2", 2, n_hist=1100),
    small("c3", 1, n_hist=1100, init="bias"),
    small("c4", 2, n_hist=1100, init="bias"),
    small("c3", 1, n_hist=2100, init="bias"),
    # the c3 draft-length sweep (P = gamma + 1 = 2, 3, 6, 16, 21 verify positions)
] + [small("c3", 4, n_hist=40, init="bias", gamma=g) for g in (1, 2, 5, 15, 20)] + [
    # the largest draft length: 33 positions, three query tiles per (sequence, head)
    small("c3", 2, n_hist=40, init="bias", gamma=32),
    small("c2", 3, n_hist=60, init="bias", gamma=32),
]


def _ids(cases):
    return [c.name for c in cases]


def _oracle_round(case, wt, wd, gamma, n_gen, seed):
    T, D = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    st = S.prefill(T, D, ht, hk, n_gen)
    rows = np.arange(case.B)
    dr = S.draft(D, st, gamma, seed, rows)
    vf = S.verify(T, st, dr, rows)
    return T, D, ht, hk, st, dr, vf


@pytest.mark.parametrize("case", VERIFY_CASES, ids=_ids(VERIFY_CASES))
def test_verify_teacher_forced(case):
    gamma, n_gen, seed = case.g, 64, 11
    wt, wd = weights(case)
    T, D, ht, hk, st_o, dr, vf = _oracle_round(case, wt, wd, gamma, n_gen, seed)
    M, K = case.wl.target.n_mix, case.wl.target.n_types
    print(f"{case.name}: gamma {gamma}, B {case.B}, history {case.n_hist}", flush=True)
    st = gpu_state(case, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    dbuf = draft_buffers_from_oracle(dr, case.B, gamma, M, K)
    vbuf = tp.VerifyBuffers(case.B, gamma, M, K)
    st.tppsd_verify(gamma, dbuf, vbuf)
    torch.cuda.synchronize()
    tol = tol_of(case.wl)
    stress = case.init == "stress" and case.wl.prec == "bf16"
    dr32 = S.DraftOut(**{f: f32_round(getattr(dr, f)) for f in dr.__dataclass_fields__})
    err = check_verify(verify_out(vbuf, np.arange(case.B), gamma), vf, tol, case.name, stress, dr32)
    assert st.tppsd_state_status()["bits"] == 0
    msg = f"{case.name}: max abs err {err:.2e} (tol {STRESS_BF16_TOL if stress else tol:.1e})"
    if case.wl.prec == "bf16":
        # the float32 evaluation with the same rounding points stays within its stated drift
        em = emulated_verify(case.wl.target, wt, ht, hk, dr)
        pairs = list(zip(em, (vf.logg, vf.logf, np.stack([vf.logw, vf.mu, vf.s], 2), vf.logtype)))
        drift = max(np.abs(a - b).max() for a, b in (pairs[2:] if stress else pairs))
        assert drift <= (STRESS_BF16_TOL if stress else EMU_DRIFT_MAX[case.wl.name]), drift
        msg += f"; float32-emulation drift {drift:.2e}"
    print(msg)


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


ACCEPT_CASES = [small("c1", 64), small("c3", 48, n_hist=30, init="bias"), small("c5", 96, init="bias"),
                small("c4", 24, n_hist=40, init="bias"), small("c3", 48, n_hist=30, init="bias", gamma=1),
                small("c3", 48, n_hist=30, init="bias", gamma=20)]


@pytest.mark.parametrize("external", [False, True])
@pytest.mark.parametrize("case", ACCEPT_CASES, ids=_ids(ACCEPT_CASES))
def test_accept_teacher_forced(case, external):
    gamma, n_gen, seed = case.g, 64, 5
    wt, wd = weights(case)
    T, D, ht, hk, st_o, dr, vf = _oracle_round(case, wt, wd, gamma, n_gen, seed)
    print(f"{case.name}: gamma {gamma}, external uniforms {external}", flush=True)
    # the GPU receives exactly the values the oracle decides on (rounded to float32)
    dr32 = S.DraftOut(**{f: f32_round(getattr(dr, f)) for f in dr.__dataclass_fields__})
    vf32 = S.VerifyOut(**{f: f32_round(getattr(vf, f)) for f in vf.__dataclass_fields__})
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


# a draft with eight heads of width 16: the one-launch draft's attention runs
# on MFMA (the vector-ALU form serves up to four heads)
H8 = W.Workload("h8", 7, W.ModelCfg(2, 64, 4, 256, 16, 22, "bf16"), W.ModelCfg(1, 128, 8, 256, 16, 22, "bf16"),
                batch=8, n_gen=64, gammas=(6,), n_hist=30, history="hawkes22", description="8-head bf16 draft")
# a three-layer row-drafting draft (d 128, four heads of 32, F 512): its middle
# layer runs the FFN in four slices and takes its rows as the residual plus the
# first layer's slices, a form the two-layer c4 draft does not reach
R3 = W.Workload("r3", 8, W.ModelCfg(2, 64, 4, 256, 16, 5, "bf16"), W.ModelCfg(3, 128, 4, 512, 16, 5, "bf16"),
                batch=4, n_gen=64, gammas=(6,), n_hist=600, history="hawkes5", description="3-layer row draft")
DRAFT_CASES = [small("c1", 8), small("c2", 8), small("c3", 16, n_hist=40, init="bias"), small("c5", 16, init="bias"),
               small("c4", 4, n_hist=40, init="bias"), small("c3", 8, n_hist=40, init="bias", gamma=20),
               small("c2", 4, n_hist=40, init="bias", gamma=32), Case("h8-B6-bias", H8, 6, 30, "bias", True),
               # d = 128 drafts over a long history: four key splits of 384 per (sequence, head)
               small("c4", 3, n_hist=1100, init="bias"), Case("r3-B4-h600-bias", R3, 4, 600, "bias", True)]


# both drafting paths: one workgroup per sequence for all gamma steps (where
# the draft model fits it), and per-step batched kernels
@pytest.mark.parametrize("layered", [False, True], ids=["fused", "layered"])
@pytest.mark.parametrize("case", DRAFT_CASES, ids=_ids(DRAFT_CASES))
def test_draft_parity(case, layered, monkeypatch):
    monkeypatch.setenv("TPPSD_LAYERED_DRAFT", "1" if layered else "0")
    _draft_parity(case)


def _draft_parity(case):
    gamma, n_gen, seed = case.g, 64, 13
    wt, wd = weights(case)
    T, D = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    M, K = case.wl.target.n_mix, case.wl.target.n_types
    print(f"{case.name}: gamma {gamma}", flush=True)
    st = gpu_state(case, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    dbuf = tp.DraftBuffers(case.B, gamma, M, K)
    st.tppsd_draft(gamma, dbuf)
    torch.cuda.synchronize()
    ost = S.prefill(T, D, ht, hk, n_gen)
    rows = np.arange(case.B)
    stress = case.init == "stress" and case.wl.prec == "bf16"
    compared = check_draft_record(D, ost, draft_out(dbuf, rows, gamma), gamma, seed, 0, rows, tol_of(case.wl),
                                  case.name, stress)
    # categorical near-ties skip a few draws; almost all are compared
    assert compared >= 0.9 * case.B * gamma, compared
    # the first draft position sees only committed events: the oracle's own
    # free-running draft draws the same type there unless it is a near-tie
    odr = S.draft(D, S.prefill(T, D, ht, hk, n_gen), gamma, seed, rows)
    g_k = dbuf.k.cpu().numpy()
    sure = odr.cat_margin[:, 0] >= CAT_TIE
    assert np.array_equal(g_k[sure, 0], odr.k[sure, 0])
    print(f"{case.name}: {compared} of {case.B * gamma} draws compared")


# the per-step draft's row-block kernel with four waves (4096-sequence drafts
# run it at d = 32)
@pytest.mark.parametrize("case", [DRAFT_CASES[3]], ids=_ids(DRAFT_CASES[3:4]))
def test_draft_block_four_waves(case, monkeypatch):
    monkeypatch.setenv("TPPSD_BLOCK_NT", "256")
    monkeypatch.setenv("TPPSD_LAYERED_DRAFT", "1")
    _draft_parity(case)


# end to end on paper-scale weights with non-zero biases
E2E_CASES = [small("c1", 4, init="bias"), small("c2", 8, init="bias"), small("c3", 4, n_hist=30, init="bias"),
             small("c4", 2, n_hist=40, init="bias"), small("c5", 16, init="bias")]
# share of generated events whose decisions must have been compared
E2E_FLOOR = 0.5


@pytest.mark.parametrize("case", E2E_CASES, ids=_ids(E2E_CASES))
def test_ar_end_to_end(case):
    n_gen, seed = 24, 21
    wt, wd = weights(case)
    T, _ = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    print(f"{case.name}: AR, {n_gen} events", flush=True)
    st = gpu_state(case, wt, wd, 1, n_gen, seed, draft=False)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    compared, generated = replay_ar_steps(case, T, st, seed, n_gen)
    status = st.tppsd_state_status()
    assert status["bits"] == 0 and status["n_done"] == case.B, status
    assert generated == case.B * n_gen
    assert compared >= E2E_FLOOR * generated, (compared, generated)
    print(f"{case.name}: AR events compared {compared}/{generated}")


# the kernel-timing mode launches the AR steps one by one instead of replaying
# graphs: the same kernels in the same order, so the same events bit for bit
AR_DIRECT_CASES = [small("c4", 2, n_hist=40, init="bias"), small("c5", 16, init="bias")]


@pytest.mark.parametrize("case", AR_DIRECT_CASES, ids=_ids(AR_DIRECT_CASES))
def test_ar_direct_launch_matches_graphs(case):
    n_gen, seed = 20, 5
    wt, wd = weights(case)
    ht, hk = histories(case)
    st = gpu_state(case, wt, wd, 1, n_gen, seed, draft=False)
    runs = []
    for direct in (False, True):
        st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
        st.tppsd_timing_enable(tp.TIME_KERNELS if direct else 0)
        st.tppsd_sample_ar(n_gen)
        st.tppsd_timing_enable(0)
        t, k, n = st.tppsd_read_events()
        status = st.tppsd_state_status()
        assert status["bits"] == 0 and status["n_done"] == case.B, status
        runs.append((t.cpu().numpy(), k.cpu().numpy(), n.cpu().numpy()))
    (t0, k0, n0), (t1, k1, n1) = runs
    assert np.array_equal(n0, n1)
    for b in range(case.B):
        assert np.array_equal(t0[b, :n0[b]].view(np.uint32), t1[b, :n1[b]].view(np.uint32)), b
        assert np.array_equal(k0[b, :n0[b]], k1[b, :n1[b]]), b


# a job run in pieces (SD rounds a few at a time, AR in two calls) continues
# from the device state exactly: the same events and counters as one call
RESUME_CASES = [small("c4", 2, n_hist=40, init="bias"), small("c3", 4, n_hist=30, init="bias"),
                small("c5", 16, init="bias")]


def _job_result(st):
    t, k, n = st.tppsd_read_events()
    status = st.tppsd_state_status()
    return t.cpu().numpy(), k.cpu().numpy(), n.cpu().numpy(), status


def _same_events(a, b, B):
    (t0, k0, n0, s0), (t1, k1, n1, s1) = a, b
    assert np.array_equal(n0, n1)
    for i in range(B):
        assert np.array_equal(t0[i, :n0[i]].view(np.uint32), t1[i, :n1[i]].view(np.uint32)), i
        assert np.array_equal(k0[i, :n0[i]], k1[i, :n1[i]]), i
    assert s0 == s1, (s0, s1)


@pytest.mark.parametrize("case", RESUME_CASES, ids=_ids(RESUME_CASES))
def test_resumed_jobs_match_one_call(case):
    gamma, n_gen, seed = case.g, 40, 9
    wt, wd = weights(case)
    ht, hk = histories(case)
    st = gpu_state(case, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    st.tppsd_sample_sd(gamma)
    whole = _job_result(st)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    pieces = 0
    while st.tppsd_state_status()["n_done"] < case.B:
        st.tppsd_sample_sd(gamma, max_rounds=3)
        pieces += 1
        assert pieces < 1000
    assert pieces > 1
    _same_events(whole, _job_result(st), case.B)
    assert whole[3]["bits"] == 0 and whole[3]["n_done"] == case.B
    # AR: n_gen steps at once, then as 7 + (n_gen - 7)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    st.tppsd_sample_ar(n_gen)
    whole = _job_result(st)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    st.tppsd_sample_ar(7)
    st.tppsd_sample_ar(n_gen - 7)
    _same_events(whole, _job_result(st), case.B)
    assert whole[3]["n_done"] == case.B


@pytest.mark.parametrize("bonus", [True, False])
@pytest.mark.parametrize("case", E2E_CASES, ids=_ids(E2E_CASES))
def test_sd_end_to_end(case, bonus):
    gamma, n_gen, seed = case.g, 48, 17
    wt, wd = weights(case)
    T, D = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    print(f"{case.name}: SD bonus={bonus}, gamma {gamma}, {n_gen} events", flush=True)
    st = gpu_state(case, wt, wd, gamma, n_gen, seed, bonus=bonus)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    compared, generated, rounds, type_redraws, vmax = replay_sd_rounds(case, T, D, st, gamma, seed, n_gen,
                                                                       bonus=bonus)
    status = st.tppsd_state_status()
    assert status["bits"] == 0 and status["n_done"] == case.B, status
    _, _, n = st.tppsd_read_events()
    assert np.all(n.cpu().numpy() == case.n_hist + n_gen)
    assert generated == case.B * n_gen
    assert compared >= E2E_FLOOR * generated, (compared, generated)
    if case.wl.target.n_types == 1:
        assert type_redraws == 0      # K = 1: log f = 0 on both sides, the type test always passes
    print(f"{case.name} bonus={bonus}: rounds {rounds}, events compared {compared}/{generated}, "
          f"max verify err {vmax:.2e}, alpha {status['accepted'] / max(1, status['drafted']):.3f}")


@pytest.mark.parametrize("case", [small("c2", 8, init="bias", mismatch=False), small("c1", 4, init="stress",
                                                                                  mismatch=False)],
                         ids=["c2-B8", "c1-B4"])
def test_draft_equal_target_accepts_all(case):
    """With the target as its own draft the accept ratio is 1 up to float32
    rounding: a position fails only if ln u > (a rounding-sized difference),
    i.e. for u within ~1e-6 of 1, so alpha stays above 1 - 1e-4."""
    gamma, n_gen, seed = case.g, 120, 3
    wt, _ = weights(case)
    tm = tp.Model(case.wl.target, wt)
    st = tp.State(tm, tm, case.B, case.n_hist + n_gen + gamma + 1, gamma, seed=seed)
    ht, hk = histories(case)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    rounds = st.tppsd_sample_sd(gamma)
    s = st.tppsd_state_status()
    assert s["bits"] == 0 and s["n_done"] == case.B, s
    alpha = s["accepted"] / s["drafted"]
    assert alpha > 1 - 1e-4, alpha
    # with the bonus every round yields gamma + 1 events
    assert rounds <= -(-n_gen // (gamma + 1)) + 1, rounds
    print(f"{case.name}: alpha {alpha}, {rounds} rounds")


def test_nonfinite_status_bit():
    """A NaN in the target's weights makes the verify outputs non-finite; the
    sticky NONFINITE bit reports it (and nothing else is set)."""
    case = small("c2", 4, init="bias")
    gamma, n_gen, seed = case.g, 32, 9
    wt, wd = weights(case)
    st = gpu_state(case, wt, wd, gamma, n_gen, seed)
    ht, hk = histories(case)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    M, K = case.wl.target.n_mix, case.wl.target.n_types
    dbuf, vbuf = tp.DraftBuffers(case.B, gamma, M, K), tp.VerifyBuffers(case.B, gamma, M, K)
    st.tppsd_draft(gamma, dbuf)
    st.tppsd_verify(gamma, dbuf, vbuf)
    assert st.tppsd_state_status()["bits"] == 0
    bad = {k: v.copy() for k, v in wt.items()}
    bad["head.mu.b"][0] = np.nan
    st2 = gpu_state(case, bad, wd, gamma, n_gen, seed)
    st2.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    st2.tppsd_draft(gamma, dbuf)
    st2.tppsd_verify(gamma, dbuf, vbuf)
    bits = st2.tppsd_state_status()["bits"]
    assert bits == tp.STATUS_NONFINITE, bits
