"""GPU parity at the workloads' full sizes, in the configuration bench.py times.

Each workload runs at its full batch, with the bench's weights, histories and
seed, through graph-replayed TPP-SD rounds until about half of its events are
generated (so the KV caches hold long contexts and every launch has the
bench's shape), then one explicit draft / verify / accept round through the
C ABI. A few sampled sequences are replayed by the oracle from the events the
GPU committed (teacher-forced history; sequences are independent, so each
sample is an oracle state of its own keyed by its global sequence id) and
compared:

- draft records: the oracle drafts from the same state and Philox counters;
  compared up to each sequence's first categorical near-tie;
- verify outputs, teacher-forced on the GPU's drafts: within 1e-5 (fp32), or
  max(2e-3, twice the drift of a float32 evaluation with the same rounding
  points) (bf16);
- accept decisions, teacher-forced on the GPU's draft and verify outputs:
  bit-exact unless a decision is inside the near-tie window.
"""
import numpy as np
import pytest
import torch

from gpu_common import CAT_TIE, NEAR_TIE, TOL, first_fragile
from fp32_emulation import emulated_verify
from oracle import sampler as S
from oracle.model import Model as OModel
from paper_2507_09252_amd import tppsd as tp
from paper_2507_09252_amd import workloads as W

pytestmark = pytest.mark.gpu

SEED = 1234           # bench.py's sampler seed
# workload -> (sampled sequences, fraction of n_gen generated before the checked round)
CASES = {"c2": ([0, 17, 63], 0.5), "c3": ([0, 37, 101, 200, 255], 0.5), "c4": ([0, 31], 0.25),
         "c5": ([0, 1234, 4095], 0.5), "a3": ([0, 101, 255], 0.5)}


def _gpu_run(wl, gamma, frac):
    B, n_gen = wl.batch, wl.n_gen
    wt, wd = W.workload_weights(wl)
    ht, hk = W.make_histories(wl)
    dev = torch.device("cuda:0")
    tm, dm = tp.Model(wl.target, wt, dev), tp.Model(wl.draft, wd, dev)
    cap = wl.n_hist + n_gen + gamma + 1
    st = tp.State(tm, dm, B, cap, gamma, seed=SEED)
    st._models = (tm, dm)
    st.tppsd_prefill(torch.from_numpy(ht).to(dev), torch.from_numpy(hk).to(dev), n_gen)
    rounds = 0
    while True:
        _, _, n = st.tppsd_read_events()
        gen = n.cpu().numpy() - wl.n_hist
        if gen.max() >= frac * n_gen:
            break
        rounds += st.tppsd_sample_sd(gamma, max_rounds=5)
    assert gen.max() + gamma + 1 <= n_gen, "a sequence would be truncated in the checked round"
    return wt, wd, st, rounds


def _draft_out(dbuf, rows):
    g = {f: getattr(dbuf, f).cpu().numpy()[rows] for f in ("tau", "t", "k", "logg", "logf", "mix", "logtype")}
    mix = g["mix"].astype(np.float64)
    return S.DraftOut(tau=g["tau"].astype(np.float64), t=g["t"].astype(np.float64), k=g["k"].astype(np.int64),
                      logg=g["logg"].astype(np.float64), logf=g["logf"].astype(np.float64),
                      logw=mix[:, :, 0], mu=mix[:, :, 1], s=mix[:, :, 2],
                      logtype=g["logtype"].astype(np.float64), cat_margin=np.full(g["tau"].shape, np.inf))


def _verify_out(vbuf, rows):
    g = {f: getattr(vbuf, f).cpu().numpy()[rows].astype(np.float64) for f in ("logg", "logf", "mix", "logtype")}
    return S.VerifyOut(logg=g["logg"], logf=g["logf"], logw=g["mix"][:, :, 0], mu=g["mix"][:, :, 1],
                       s=g["mix"][:, :, 2], logtype=g["logtype"])


@pytest.mark.parametrize("name", list(CASES))
def test_fullsize_round(name):
    wl = W.WORKLOADS[name]
    gamma = wl.gamma
    samples, frac = CASES[name]
    wt, wd, st, rounds = _gpu_run(wl, gamma, frac)
    M, K = wl.target.n_mix, wl.target.n_types
    B = wl.batch
    dbuf = tp.DraftBuffers(B, gamma, M, K)
    vbuf = tp.VerifyBuffers(B, gamma, M, K)
    abuf = tp.AcceptBuffers(B, gamma)
    ev_t, ev_k, ev_n = (a.cpu().numpy() for a in st.tppsd_read_events())
    st.tppsd_draft(gamma, dbuf)
    st.tppsd_verify(gamma, dbuf, vbuf)
    st.tppsd_accept(gamma, dbuf, vbuf, abuf)
    torch.cuda.synchronize()
    assert st.tppsd_state_status()["bits"] == 0
    T, D = OModel(wl.target, wt), OModel(wl.draft, wd)
    tol0 = TOL[wl.prec]
    drafts_checked = 0
    for b in samples:
        n_b = int(ev_n[b])
        gen_b = n_b - wl.n_hist
        ht = ev_t[b:b + 1, :n_b]
        hk = ev_k[b:b + 1, :n_b].astype(np.int64)
        print(f"{name} seq {b}: {n_b} events after {rounds} rounds")
        # --- draft: same state, same counters
        ost = S.prefill(T, D, ht, hk, wl.n_gen - gen_b, seq0=b)
        ost.round = rounds
        odr = S.draft(D, ost, gamma, SEED, np.array([0]))
        gdr = _draft_out(dbuf, [b])
        upto = int(first_fragile(np.full((1, gamma), np.inf), odr.cat_margin, 0.0, max(CAT_TIE, tol0))[0])
        assert np.array_equal(gdr.k[0, :upto], odr.k[0, :upto]), (b, gdr.k[0], odr.k[0])
        np.testing.assert_allclose(gdr.tau[0, :upto], odr.tau[0, :upto], rtol=20 * tol0)
        np.testing.assert_allclose(gdr.logg[0, :upto], odr.logg[0, :upto], atol=20 * tol0, rtol=tol0)
        drafts_checked += upto
        print(f"{name} seq {b}: draft compared at {upto} of {gamma} positions")
        # --- verify, teacher-forced on the GPU's drafts
        ovf = S.verify(T, ost, gdr, np.array([0]))
        gvf = _verify_out(vbuf, [b])
        want = (ovf.logg, ovf.logf, np.stack([ovf.logw, ovf.mu, ovf.s], 2), ovf.logtype)
        got = (gvf.logg, gvf.logf, np.stack([gvf.logw, gvf.mu, gvf.s], 2), gvf.logtype)
        drift, tol = 0.0, tol0
        if wl.prec == "bf16":
            # bf16 operands: floor 2e-3, above it twice the drift of an exact
            # float32 evaluation with the same rounding points
            em = emulated_verify(wl.target, wt, ht.astype(np.float32), hk, gdr)
            drift = max(np.abs(a - w).max() for a, w in zip(em, want))
            tol = max(tol0, 2 * drift)
        for what, g_, w_ in zip(("log g_T", "log f_T", "mixture", "log f"), got, want):
            err = np.abs(g_ - w_).max()
            assert np.all(np.isfinite(g_)) and err <= tol, f"{name} seq {b} {what}: err {err:.3g} tol {tol:.3g}"
        print(f"{name} seq {b}: verify max err {max(np.abs(g_ - w_).max() for g_, w_ in zip(got, want)):.2e}"
              f" (float32 drift {drift:.2e}, tol {tol:.2e})")
        # --- accept, teacher-forced on the GPU's draft and verify outputs
        res = S.accept(ost, gamma, gdr, gvf, SEED, np.array([0]))
        fragile = (ost.log_margin[0, :gamma + 1].min() < NEAR_TIE) or (ost.cat_margin[0, :gamma + 1].min() < CAT_TIE)
        if fragile:
            print(f"{name} seq {b}: accept decision inside the near-tie window, not compared")
            continue
        assert int(abuf.L[b]) == res["L"][0]
        assert int(abuf.flags[b]) & 7 == res["flags"][0]
        assert int(abuf.ar_iter[b]) == res["ar_iter"][0]
        m = int(abuf.n_new[b])
        assert m == res["n_new"][0]
        assert np.array_equal(abuf.k_new[b, :m].cpu().numpy(), res["k_new"][0, :m])
        np.testing.assert_allclose(abuf.tau_new[b, :m].cpu().numpy(), res["tau_new"][0, :m], rtol=2e-6)
    assert drafts_checked >= len(samples), "categorical near-ties cut the draft comparisons"
