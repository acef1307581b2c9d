"""Shared helpers of the GPU parity tests (HIP path through the C ABI vs the oracle)."""
import dataclasses

import numpy as np
import torch

from oracle import sampler as S
from oracle.model import Model as OModel
from paper_2507_09252_amd import tppsd as tp
from paper_2507_09252_amd import workloads as W

# spec tolerances on log-densities
TOL = {"fp32": 1e-5, "bf16": 2e-3}
NEAR_TIE = 1e-4          # decision window on identical inputs (log space)
CAT_TIE = 1e-5           # categorical window (relative probability mass)


@dataclasses.dataclass
class Case:
    name: str
    wl: W.Workload
    B: int
    n_hist: int
    init: str
    mismatch: bool


def small(name, B, n_hist=None, init="stress", mismatch=True):
    wl = W.WORKLOADS[name]
    return Case(f"{name}-B{B}-{init}{'-mm' if mismatch else ''}", wl, B, n_hist or wl.n_hist, init, mismatch)


def weights(case: Case):
    wt, wd = W.workload_weights(case.wl, init=case.init)
    if case.mismatch:
        wd = W.mismatch_draft(wd, case.wl.draft, W.seed_sequence(case.wl.index, 4))
    return wt, wd


def histories(case: Case):
    return W.make_histories(case.wl, batch=case.B, n_hist=case.n_hist)


def oracle_models(case: Case, wt, wd):
    return OModel(case.wl.target, wt), OModel(case.wl.draft, wd)


def gpu_state(case: Case, wt, wd, gamma, n_gen, seed, bonus=True, draft=True):
    tm = tp.Model(case.wl.target, wt)
    dm = tp.Model(case.wl.draft, wd) if draft else None
    cap = case.n_hist + n_gen + gamma + 1
    st = tp.State(tm, dm, case.B, cap, gamma, seed=seed, bonus=bonus)
    st._models = (tm, dm)
    return st


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def draft_buffers_from_oracle(dr: S.DraftOut, B, gamma, M, K):
    buf = tp.DraftBuffers(B, gamma, M, K)
    buf.tau.copy_(to_dev(dr.tau.astype(np.float32)))
    buf.t.copy_(to_dev(dr.t.astype(np.float32)))
    buf.k.copy_(to_dev(dr.k.astype(np.int32)))
    buf.logg.copy_(to_dev(dr.logg.astype(np.float32)))
    buf.logf.copy_(to_dev(dr.logf.astype(np.float32)))
    mix = np.stack([dr.logw, dr.mu, dr.s], axis=2).astype(np.float32)
    buf.mix.copy_(to_dev(mix))
    buf.logtype.copy_(to_dev(dr.logtype.astype(np.float32)))
    return buf


def verify_buffers_from_oracle(vf: S.VerifyOut, B, gamma, M, K):
    buf = tp.VerifyBuffers(B, gamma, M, K)
    buf.logg.copy_(to_dev(vf.logg.astype(np.float32)))
    buf.logf.copy_(to_dev(vf.logf.astype(np.float32)))
    buf.mix.copy_(to_dev(np.stack([vf.logw, vf.mu, vf.s], axis=2).astype(np.float32)))
    buf.logtype.copy_(to_dev(vf.logtype.astype(np.float32)))
    return buf


def first_fragile(log_margin, cat_margin, log_win, cat_win):
    """Per row: index of the first event whose decisions were within the windows (n if none)."""
    frag = (log_margin < log_win) | (cat_margin < cat_win)
    n = frag.shape[1]
    return np.where(frag.any(axis=1), np.argmax(frag, axis=1), n)


def compare_events(g_t, g_k, o_t, o_k, upto, rtol):
    """Events must match before each row's first fragile decision."""
    rows_full = 0
    for b in range(g_t.shape[0]):
        u = upto[b]
        assert np.array_equal(g_k[b, :u], o_k[b, :u]), (b, u, g_k[b, :u], o_k[b, :u])
        np.testing.assert_allclose(g_t[b, :u], o_t[b, :u], rtol=rtol, atol=rtol, err_msg=f"row {b}")
        rows_full += int(u == g_t.shape[1])
    return rows_full / g_t.shape[0]
