"""Naive AR sampling and TPP-SD sampling, float64 oracle.

ORACLE / TEST INFRASTRUCTURE (see oracle/__init__.py).

Follows §4.2 ("Naive autoregressive sampling"), App. A.1 (sampling a
log-normal mixture), §4.3 (drafting, verification, adjusted distributions
Eq. (3)-(4), Theorem 1) and Algorithm 1 (App. C.1), with these readings of
points the paper leaves open:

  * Joint (tau, k) proposals: at the first rejected position L each
    component is tested with its own uniform; a component that passed is
    kept and one that failed is redrawn from its own adjusted distribution
    (Eq. (3) via Theorem 1 for tau, Eq. (4) for k). The decoder's type
    distribution does not depend on the new interval, so App. A.2's two
    identities hold per component. Algorithm 1's literal "redraw both"
    is available as a negative control (``literal_alg1=True``).
  * L is the first rejected position, or gamma + 1 when all gamma drafts pass;
    with ``bonus`` on, a full acceptance adds one event drawn from the
    target's distribution after the last draft (the extra distribution of
    §2.3), otherwise the round yields the gamma drafts.
  * Uniforms lie in (0, 1); a test accepts iff ln u < log p_T - log p_D.
  * The acceptance-rejection loop of Theorem 1 draws its candidates from a
    counter-indexed stream and returns the first accepted one.
  * Categorical draws take the first index m with u * C_total < C_m, C the
    ascending cumulative sum of the probabilities.
  * Generation stops after n_gen new events per sequence (the last round is
    truncated) or, when an end time T is given, at the first event past T
    (Algorithm 1 samples while t < T and then drops events with t > T, so
    events are committed in order while t <= T), whichever comes first.
  * The model log-likelihood (Eq. (2)) of the generated events is the sum of
    the target's log g(tau_i) + log f(k_i) at each committed event, tau_i the
    interval as drawn (event times are its float32 running sum), plus, for a
    sequence ended by its end time T, the survival term log(1 - G(T - t_N))
    under the distribution that followed the last committed event.
  * A seed history is prefilled; its last event is the pending one whose
    history embedding gives the next distribution.

Every discrete decision also reports its margin (distance of the compared
quantities) so that GPU parity tests can recognise near-ties.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

import scipy.special

from .model import Model
from .numerics import f32, logsumexp
from .philox import (TAG_ACCEPT, TAG_AR, TAG_BONUS, TAG_DRAFT, TAG_RES_K,
                     TAG_RES_T, uniforms)

HALF_LOG_2PI = 0.5 * np.log(2.0 * np.pi)
AR_ITER_CAP = 1 << 20


# ---------------------------------------------------------------------------
# decoder densities and draws
# ---------------------------------------------------------------------------

def mixture_logpdf(logw, mu, s, tau):
    """log g(tau) for the log-normal mixture of §4.2 (density as in App. A.1).

    logw, mu, s: [..., M] with s = log sigma; tau: [...] > 0.
    """
    lt = np.log(np.asarray(tau, dtype=np.float64))[..., None]
    comp = logw - s - HALF_LOG_2PI - lt - (lt - mu) ** 2 / (2.0 * np.exp(2.0 * s))
    return logsumexp(comp, axis=-1)


def mixture_log_survival(logw, mu, s, x):
    """log(1 - G(x)) for the log-normal mixture (the survival term of Eq. (2)).

    1 - G(x) = sum_m w_m P(LogNormal(mu_m, sigma_m) > x) = sum_m w_m Phi(-(ln x - mu_m) / sigma_m),
    evaluated as a log-sum-exp of log w_m + log Phi(.) (scipy's log_ndtr). x <= 0 gives 0.
    """
    x = float(x)
    if x <= 0.0:
        return 0.0
    z = (np.log(x) - np.asarray(mu, dtype=np.float64)) / np.exp(np.asarray(s, dtype=np.float64))
    return float(logsumexp(np.asarray(logw, dtype=np.float64) + scipy.special.log_ndtr(-z)))


def categorical(logp, u):
    """First index m with u * C_total < C_m; returns (index, relative margin)."""
    p = np.exp(np.asarray(logp, dtype=np.float64))
    C = np.cumsum(p, axis=-1)
    tot = C[..., -1]
    x = np.asarray(u) * tot
    idx = np.minimum(np.sum(C <= x[..., None], axis=-1), p.shape[-1] - 1)
    upper = np.take_along_axis(C, idx[..., None], -1)[..., 0]
    lower = np.where(idx > 0, np.take_along_axis(C, np.maximum(idx - 1, 0)[..., None], -1)[..., 0], 0.0)
    margin = np.minimum(x - lower, upper - x) / tot
    if p.shape[-1] == 1:
        margin = np.full_like(margin, np.inf)
    return idx, margin


def box_muller(u1, u2):
    """Standard normal from two uniforms (Box and Muller, 1958), cosine branch."""
    return np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)


def sample_event(logw, mu, s, logf, U):
    """Draw (tau, k) from one decoder output with U[..., 4] = (u_c, u_1, u_2, u_k).

    App. A.1 / §4.2: z ~ Categorical(w), eps ~ N(0, 1), tau = exp(mu_z + sigma_z eps);
    k ~ f(k | h). tau is returned rounded to float32 (times are float32).
    Returns (tau, k, categorical margin).
    """
    z, mz = categorical(logw, U[..., 0])
    eps = box_muller(U[..., 1], U[..., 2])
    mz_ = np.take_along_axis(mu, z[..., None], -1)[..., 0]
    sz_ = np.take_along_axis(s, z[..., None], -1)[..., 0]
    tau = f32(np.exp(mz_ + np.exp(sz_) * eps))
    k, mk = categorical(logf, U[..., 3])
    return tau, k, np.minimum(mz, mk)


# ---------------------------------------------------------------------------
# sampler state
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class State:
    t: np.ndarray          # [B, cap] float64 holding float32 times
    k: np.ndarray          # [B, cap] int64
    n: np.ndarray          # [B] committed events (history + generated)
    gen: np.ndarray        # [B] generated events
    n_gen: int
    tcache: object
    dcache: Optional[object]
    round: int = 0
    seq0: int = 0          # global id of row 0 (Philox counter word 0 is seq0 + row)
    # margins for the near-tie protocol, per generated event
    log_margin: Optional[np.ndarray] = None   # [B, n_gen]
    cat_margin: Optional[np.ndarray] = None   # [B, n_gen]
    # accounting (O-7)
    rounds_run: Optional[np.ndarray] = None
    drafted: int = 0
    accepted_drafts: int = 0
    ar_iters_total: int = 0
    # end-time stop and model log-likelihood (Eq. (2))
    t_end: Optional[np.ndarray] = None        # [B] float32 end times, or None (count stop only)
    stopped: Optional[np.ndarray] = None      # [B] ended by the end time
    stop_margin: Optional[np.ndarray] = None  # [B] min |t - T| over the end-time decisions taken
    ll: Optional[np.ndarray] = None           # [B] log-likelihood of the generated events
    tau: Optional[np.ndarray] = None          # [B, cap] drawn interval of each generated event

    def __post_init__(self):
        B = len(self.n)
        if self.stopped is None:
            self.stopped = np.zeros(B, dtype=bool)
        if self.stop_margin is None:
            self.stop_margin = np.full(B, np.inf)
        if self.ll is None:
            self.ll = np.zeros(B)
        if self.tau is None:
            self.tau = np.zeros_like(self.t)

    @property
    def done(self):
        return (self.gen >= self.n_gen) | self.stopped


def prefill(T: Model, D: Optional[Model], hist_t, hist_k, n_gen: int, extra: int = 64,
            seq0: int = 0, t_end=None) -> State:
    """Store the seed histories and cache every event except the pending (last) one.

    The draft cache holds all but the last two events: each round's first
    draft step re-encodes the last two committed events. t_end (scalar or
    [B], rounded to float32): per-sequence end time; a sequence whose pending
    event is already at or past it generates nothing.
    """
    hist_t = np.asarray(hist_t, dtype=np.float32).astype(np.float64)
    hist_k = np.asarray(hist_k, dtype=np.int64)
    B, n0 = hist_t.shape
    assert n0 >= 2
    cap = n0 + n_gen + extra
    t = np.zeros((B, cap))
    k = np.zeros((B, cap), dtype=np.int64)
    t[:, :n0], k[:, :n0] = hist_t, hist_k
    st = State(t=t, k=k, n=np.full(B, n0, dtype=np.int64), gen=np.zeros(B, dtype=np.int64),
               n_gen=n_gen, tcache=T.new_cache(B, cap), dcache=None,
               log_margin=np.full((B, n_gen), np.inf), cat_margin=np.full((B, n_gen), np.inf),
               rounds_run=np.zeros(B, dtype=np.int64), seq0=seq0)
    if t_end is not None:
        st.t_end = f32(np.broadcast_to(np.asarray(t_end, dtype=np.float64), (B,))).copy()
        st.stopped = hist_t[:, -1] >= st.t_end
        st.stop_margin = np.abs(hist_t[:, -1] - st.t_end)
    if n0 > 1:
        T.forward_block(st.tcache, hist_t[:, :n0 - 1], hist_k[:, :n0 - 1], np.zeros(B, dtype=np.int64))
    if D is not None:
        st.dcache = D.new_cache(B, cap)
        if n0 > 2:
            D.forward_block(st.dcache, hist_t[:, :n0 - 2], hist_k[:, :n0 - 2], np.zeros(B, dtype=np.int64))
    return st


def _commit(st: State, b: int, times, types, taus, log_margins, cat_margins, logdens, dists):
    """Append new events to sequence b in order until it has n_gen generated
    events or, with an end time T, until the first event past T (which is
    dropped; an event exactly at T is kept and ends the sequence).

    logdens[j]: the target's log g(tau_j) + log f(k_j) for event j, added to
    the log-likelihood when the event is committed; dists[j] = (log w, mu, s)
    of the distribution event j was drawn from, whose survival at T - t_N ends
    the log-likelihood of a sequence stopped by its end time."""
    room = st.n_gen - st.gen[b]
    T_end = None if st.t_end is None else st.t_end[b]
    m = 0
    for j in range(len(times)):
        if m >= room:
            break
        if T_end is not None:
            st.stop_margin[b] = min(st.stop_margin[b], abs(times[j] - T_end))
            if times[j] > T_end:
                st.stopped[b] = True
                st.ll[b] += mixture_log_survival(*dists[j], T_end - st.t[b, st.n[b] - 1])
                break
        n, g = st.n[b], st.gen[b]
        st.t[b, n] = times[j]
        st.k[b, n] = types[j]
        st.tau[b, n] = taus[j]
        st.log_margin[b, g] = log_margins[j]
        st.cat_margin[b, g] = cat_margins[j]
        st.ll[b] += logdens[j]
        st.n[b] += 1
        st.gen[b] += 1
        m += 1
        if T_end is not None and times[j] >= T_end:
            st.stopped[b] = True      # survival at T - t_N = 0 adds log 1
            break
    return m


# ---------------------------------------------------------------------------
# naive AR sampling (§4.2)
# ---------------------------------------------------------------------------

def ar_step(T: Model, st: State, seed: int):
    """One autoregressive event for every unfinished sequence."""
    rows = np.nonzero(~st.done)[0]
    if len(rows) == 0:
        return
    n = st.n[rows]
    h = T.forward_block(st.tcache, st.t[rows, n - 1][:, None], st.k[rows, n - 1][:, None],
                        n - 1, rows=rows)[:, 0]
    logw, mu, s, logf = T.head(h)
    U = uniforms(seed, st.seq0 + rows, st.gen[rows], 0, TAG_AR)
    tau, k, cm = sample_event(logw, mu, s, logf, U)
    for i, b in enumerate(rows):
        t_new = f32(st.t[b, st.n[b] - 1] + tau[i])
        ld = mixture_logpdf(logw[i], mu[i], s[i], tau[i]) + logf[i, k[i]]
        _commit(st, b, [t_new], [k[i]], [tau[i]], [np.inf], [cm[i]], [ld], [(logw[i], mu[i], s[i])])


def sample_ar(T: Model, hist_t, hist_k, n_gen: int, seed: int, seq0: int = 0, t_end=None) -> State:
    st = prefill(T, None, hist_t, hist_k, n_gen, seq0=seq0, t_end=t_end)
    while not np.all(st.done):
        ar_step(T, st, seed)
    return st


# ---------------------------------------------------------------------------
# TPP-SD (§4.3, Algorithm 1)
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class DraftOut:
    tau: np.ndarray       # [B, g]
    t: np.ndarray         # [B, g]
    k: np.ndarray         # [B, g]
    logg: np.ndarray      # [B, g]  log g_D(tau_hat)
    logf: np.ndarray      # [B, g]  log f_D(k_hat)
    logw: np.ndarray      # [B, g, M]
    mu: np.ndarray
    s: np.ndarray
    logtype: np.ndarray   # [B, g, K]
    cat_margin: np.ndarray  # [B, g]
    rate: Optional[float] = None   # homogeneous-Poisson draft: its rate (mixture fields unused)


@dataclasses.dataclass
class VerifyOut:
    logg: np.ndarray      # [B, g]   log g_T(tau_hat_l) from row l-1
    logf: np.ndarray      # [B, g]   log f_T(k_hat_l)
    logw: np.ndarray      # [B, g+1, M]
    mu: np.ndarray
    s: np.ndarray
    logtype: np.ndarray   # [B, g+1, K]


def draft(D: Model, st: State, gamma: int, seed: int, rows) -> DraftOut:
    """Drafting (§4.3): gamma sequential draws from the draft model, recording its
    full decoder outputs at every position (Theorem 1 needs g_D at fresh points
    and Eq. (4) needs all of f_D)."""
    rows = np.asarray(rows)
    B = len(rows)
    n = st.n[rows]
    r = st.round
    out = {key: [] for key in ("tau", "t", "k", "logg", "logf", "logw", "mu", "s", "logtype", "cm")}
    t_prev = st.t[rows, n - 1]
    h = D.forward_block(st.dcache, np.stack([st.t[rows, n - 2], st.t[rows, n - 1]], 1),
                        np.stack([st.k[rows, n - 2], st.k[rows, n - 1]], 1), n - 2, rows=rows)[:, -1]
    for l in range(1, gamma + 1):
        if l > 1:
            h = D.forward_block(st.dcache, out["t"][-1][:, None], out["k"][-1][:, None],
                                n + l - 2, rows=rows)[:, 0]
        logw, mu, s, logf = D.head(h)
        U = uniforms(seed, st.seq0 + rows, r, l, TAG_DRAFT)
        tau, k, cm = sample_event(logw, mu, s, logf, U)
        t_hat = f32(t_prev + tau)
        out["tau"].append(tau)
        out["t"].append(t_hat)
        out["k"].append(k)
        out["logg"].append(mixture_logpdf(logw, mu, s, tau))
        out["logf"].append(np.take_along_axis(logf, k[:, None], -1)[:, 0])
        out["logw"].append(logw)
        out["mu"].append(mu)
        out["s"].append(s)
        out["logtype"].append(logf)
        out["cm"].append(cm)
        t_prev = t_hat
    st2 = {key: np.stack(v, axis=1) for key, v in out.items()}
    return DraftOut(tau=st2["tau"], t=st2["t"], k=st2["k"], logg=st2["logg"], logf=st2["logf"],
                    logw=st2["logw"], mu=st2["mu"], s=st2["s"], logtype=st2["logtype"],
                    cat_margin=st2["cm"])


def poisson_fit(hist_t, hist_k, K: int):
    """App. D.3: maximum-likelihood homogeneous Poisson draft from the data,
    rate = n / T and mark probabilities p_m = n_m / n. Here the data are the
    seed histories: n counts their inter-event intervals and T sums their time
    spans (first to last event); the marks count every history event.
    Returns (rate, log p [K]) with log 0 = -inf for unseen marks."""
    hist_t = np.asarray(hist_t, dtype=np.float64)
    hist_k = np.asarray(hist_k, dtype=np.int64)
    n = hist_t.shape[0] * (hist_t.shape[1] - 1)
    span = float(np.sum(hist_t[:, -1] - hist_t[:, 0]))
    counts = np.bincount(hist_k.ravel(), minlength=K)[:K].astype(np.float64)
    with np.errstate(divide="ignore"):
        logp = np.log(counts / counts.sum())
    return n / span, logp


def draft_poisson(st: State, gamma: int, rate: float, logp, seed: int, rows) -> DraftOut:
    """Homogeneous-Poisson drafting (App. D.3): the gamma intervals are
    independent Exp(rate) draws and the marks independent draws from p, so
    the whole block is drawn at once. Draft position l uses the counter
    (sequence, round, l, DRAFT): tau = -ln(u_1) / rate by inversion of the
    exponential CDF, k from p with u_3. The draft densities are
    log g_D(tau) = log rate - rate tau and log f_D(k) = log p_k."""
    rows = np.asarray(rows)
    B = len(rows)
    logp = np.asarray(logp, dtype=np.float64)
    K = len(logp)
    r = st.round
    n = st.n[rows]
    t_prev = st.t[rows, n - 1]
    taus, ts, ks, lgs, lfs, cms = [], [], [], [], [], []
    for l in range(1, gamma + 1):
        U = uniforms(seed, st.seq0 + rows, r, l, TAG_DRAFT)
        tau = f32(-np.log(U[:, 1]) / rate)
        k, cm = categorical(np.broadcast_to(logp, (B, K)), U[:, 3])
        t_hat = f32(t_prev + tau)
        taus.append(tau)
        ts.append(t_hat)
        ks.append(k)
        lgs.append(np.log(rate) - rate * tau)
        lfs.append(logp[k])
        cms.append(cm)
        t_prev = t_hat
    st2 = {key: np.stack(v, axis=1) for key, v in
           (("tau", taus), ("t", ts), ("k", ks), ("logg", lgs), ("logf", lfs), ("cm", cms))}
    zeros = np.zeros((B, gamma, 1))
    return DraftOut(tau=st2["tau"], t=st2["t"], k=st2["k"], logg=st2["logg"], logf=st2["logf"],
                    logw=zeros, mu=zeros, s=zeros,
                    logtype=np.broadcast_to(logp, (B, gamma, K)).copy(), cat_margin=st2["cm"], rate=rate)


def verify(T: Model, st: State, dr: DraftOut, rows) -> VerifyOut:
    """Verification (§4.3): one target pass over the pending event and the gamma
    drafts gives gamma + 1 decoder outputs; row l - 1 scores draft l."""
    rows = np.asarray(rows)
    n = st.n[rows]
    tt = np.concatenate([st.t[rows, n - 1][:, None], dr.t], axis=1)
    kk = np.concatenate([st.k[rows, n - 1][:, None], dr.k], axis=1)
    h = T.forward_block(st.tcache, tt, kk, n - 1, rows=rows)
    logw, mu, s, logf = T.head(h)
    g = dr.t.shape[1]
    logg = mixture_logpdf(logw[:, :g], mu[:, :g], s[:, :g], dr.tau)
    logft = np.take_along_axis(logf[:, :g], dr.k[..., None], -1)[..., 0]
    return VerifyOut(logg=logg, logf=logft, logw=logw, mu=mu, s=s, logtype=logf)


def resid_time(Tw, Tmu, Ts, Dw, Dmu, Ds, seed: int, b: int, r: int, literal_target=False,
               first_chunk=None, draft_rate=None):
    """Theorem 1: draw from g' = norm(max(0, g_T - g_D)) by acceptance-rejection.

    g_D is the draft's log-normal mixture (Dw, Dmu, Ds), or the exponential
    density of a homogeneous-Poisson draft when ``draft_rate`` is given.

    Candidates tau ~ g_T; accept iff u_a < max(0, g_T - g_D) / g_T = 1 - exp(-delta)
    with delta = log g_T(tau) - log g_D(tau) > 0. Candidate j uses the counter
    (b, r, j, RES_T) with uniforms (u_c, u_1, u_2, u_a). Returns
    (tau, j, log margin, categorical margin), margins taken over the candidates
    tested up to the accepted one. ``literal_target=True`` is the negative
    control that keeps the first candidate, i.e. redraws from g_T itself.
    ``first_chunk`` may carry the uniforms of candidates 0..63, drawn beforehand.
    """
    log_m, cat_m = np.inf, np.inf
    for base in range(0, AR_ITER_CAP, 64):
        j = np.arange(base, base + 64)
        U = first_chunk if (base == 0 and first_chunk is not None) else uniforms(seed, b, r, j, TAG_RES_T)
        z, zm = categorical(np.broadcast_to(Tw, (64,) + Tw.shape), U[:, 0])
        eps = box_muller(U[:, 1], U[:, 2])
        tau = f32(np.exp(Tmu[z] + np.exp(Ts[z]) * eps))
        if literal_target:
            return tau[0], base, np.inf, float(zm[0])
        log_gd = (np.log(draft_rate) - draft_rate * tau) if draft_rate is not None \
            else mixture_logpdf(Dw, Dmu, Ds, tau)
        delta = mixture_logpdf(Tw, Tmu, Ts, tau) - log_gd
        with np.errstate(divide="ignore"):
            thresh = np.where(delta > 0, np.log(-np.expm1(-np.maximum(delta, 1e-300))), -np.inf)
        lu = np.log(U[:, 3])
        acc = lu < thresh
        m = np.abs(lu - thresh)
        last = int(np.argmax(acc)) if np.any(acc) else 63
        log_m = min(log_m, float(np.min(m[:last + 1])))
        cat_m = min(cat_m, float(np.min(zm[:last + 1])))
        if np.any(acc):
            return tau[last], base + last, log_m, cat_m
    return tau[-1], AR_ITER_CAP, log_m, cat_m


def resid_type(logfT, logfD, u):
    """Eq. (4): draw from f' = norm(max(0, f_T - f_D)); returns (k, relative margin)."""
    q = np.maximum(0.0, np.exp(logfT) - np.exp(logfD))
    with np.errstate(divide="ignore"):
        return categorical(np.log(q), u)


def first_rejection(d_tau, d_k, lu_tau, lu_k):
    """Verification tests of §4.3 along the draft block.

    Position l passes iff ln u^tau_l < log g_T - log g_D and ln u^k_l < log f_T - log f_D
    (u < ratio, a ratio >= 1 always passes). Returns (L, tau passed at L,
    k passed at L) with L the 1-based first failing position, gamma + 1 if none.
    """
    gamma = len(d_tau)
    for l in range(gamma):
        a_tau = bool(lu_tau[l] < d_tau[l])
        a_k = bool(lu_k[l] < d_k[l])
        if not (a_tau and a_k):
            return l + 1, a_tau, a_k
    return gamma + 1, True, True


def accept(st: State, gamma: int, dr: DraftOut, vf: VerifyOut, seed: int, rows, bonus=True,
           ext_uniforms=None, literal_alg1=False, resample_from_target=False):
    """Accept/reject of §4.3 + adjusted-distribution replacement + commit, per sequence.

    ext_uniforms: optional [B, gamma, 2] (u_tau, u_k) per draft position; default
    is the counter stream (b, r, l, ACCEPT). Negative controls: literal_alg1
    redraws both components at L whatever their tests said (Algorithm 1 read
    literally); resample_from_target redraws from g_T / f_T instead of the
    adjusted distributions (shown wrong in App. A.2).

    Returns a dict of per-row arrays: L, n_new, flags, ar_iter, and the new events.
    flags: bit0 tau redrawn at L, bit1 k redrawn at L, bit2 bonus event.
    """
    rows = np.asarray(rows)
    r = st.round
    if ext_uniforms is None:
        U = uniforms(seed, st.seq0 + rows[:, None], r, np.arange(1, gamma + 1)[None, :], TAG_ACCEPT)
        u_tau, u_k = U[..., 0], U[..., 1]
    else:
        u_tau, u_k = ext_uniforms[..., 0], ext_uniforms[..., 1]
    nb = len(rows)
    # the round's residual and bonus uniforms for every row, drawn in one batch
    gid = st.seq0 + rows
    U_rest = uniforms(seed, gid[:, None], r, np.arange(64)[None, :], TAG_RES_T)
    U_resk = uniforms(seed, gid, r, 0, TAG_RES_K)
    U_bonus = uniforms(seed, gid, r, 0, TAG_BONUS)
    res = dict(L=np.zeros(nb, np.int64), n_new=np.zeros(nb, np.int64),
               flags=np.zeros(nb, np.int64), ar_iter=np.full(nb, -1, np.int64),
               t_new=np.zeros((nb, gamma + 1)), k_new=np.zeros((nb, gamma + 1), np.int64),
               tau_new=np.zeros((nb, gamma + 1)))
    single_type = dr.logtype.shape[-1] == 1
    for i, b in enumerate(rows):
        d_tau = vf.logg[i] - dr.logg[i]
        d_k = vf.logf[i] - dr.logf[i]
        lu_tau, lu_k = np.log(u_tau[i]), np.log(u_k[i])
        # margins of the decisions taken at each output position
        log_m = np.full(gamma + 1, np.inf)
        cat_m = np.concatenate([dr.cat_margin[i], [np.inf]])
        L, a_tau, a_k = first_rejection(d_tau, d_k, lu_tau, lu_k)
        for l in range(min(L, gamma)):
            mk = np.inf if single_type else abs(lu_k[l] - d_k[l])
            log_m[l] = min(abs(lu_tau[l] - d_tau[l]), mk)
        taus = list(dr.tau[i, :L - 1])
        ks = [int(x) for x in dr.k[i, :L - 1]]
        flags = 0
        if L <= gamma:
            li = L - 1
            redraw_tau = (not a_tau) or literal_alg1
            redraw_k = (not a_k) or literal_alg1
            if redraw_tau:
                tau_L, j, lm, cm = resid_time(vf.logw[i, li], vf.mu[i, li], vf.s[i, li],
                                              dr.logw[i, li], dr.mu[i, li], dr.s[i, li], seed,
                                              st.seq0 + b, r,
                                              literal_target=resample_from_target,
                                              first_chunk=U_rest[i], draft_rate=dr.rate)
                res["ar_iter"][i] = j
                st.ar_iters_total += j + 1
                log_m[li] = min(log_m[li], lm)
                cat_m[li] = min(cat_m[li], cm)
                flags |= 1
            else:
                tau_L = dr.tau[i, li]
            if redraw_k:
                uk = U_resk[i, 0]
                if resample_from_target:
                    k_L, km = categorical(vf.logtype[i, li], uk)
                else:
                    k_L, km = resid_type(vf.logtype[i, li], dr.logtype[i, li], uk)
                cat_m[li] = min(cat_m[li], float(km))
                flags |= 2
            else:
                k_L = dr.k[i, li]
            taus.append(float(tau_L))
            ks.append(int(k_L))
        elif bonus:
            Ub = U_bonus[i]
            tau_b, k_b, cm = sample_event(vf.logw[i, gamma], vf.mu[i, gamma], vf.s[i, gamma],
                                          vf.logtype[i, gamma], Ub)
            taus.append(float(tau_b))
            ks.append(int(k_b))
            cat_m[gamma] = float(cm)
            flags |= 4
        # event times from the intervals, accumulated in float32
        t_prev = st.t[b, st.n[b] - 1]
        times = []
        for tau in taus:
            t_prev = float(f32(t_prev + tau))
            times.append(t_prev)
        # target log-densities of the round's events: verify row j scores event j
        # (the accepted drafts at their recorded values, the event at L or the
        # bonus event at its interval and type)
        logdens = [vf.logg[i, j] + vf.logf[i, j] for j in range(min(L - 1, len(taus)))]
        if len(taus) > L - 1:
            j = len(taus) - 1
            logdens.append(mixture_logpdf(vf.logw[i, j], vf.mu[i, j], vf.s[i, j], taus[j]) + vf.logtype[i, j, ks[j]])
        dists = [(vf.logw[i, j], vf.mu[i, j], vf.s[i, j]) for j in range(len(taus))]
        # a decision at position l can change every event from l on
        lmc = np.minimum.accumulate(log_m[:len(times)])
        cmc = np.minimum.accumulate(cat_m[:len(times)])
        st.drafted += gamma
        st.accepted_drafts += L - 1
        m = _commit(st, b, times, ks, taus, lmc, cmc, logdens, dists)
        res["L"][i] = L
        res["n_new"][i] = m
        res["flags"][i] = flags
        res["t_new"][i, :len(times)] = times
        res["tau_new"][i, :len(taus)] = taus
        res["k_new"][i, :len(ks)] = ks
        st.rounds_run[b] += 1
    return res


def sd_round(T: Model, D: Model, st: State, gamma: int, seed: int, bonus=True, **kw):
    rows = np.nonzero(~st.done)[0]
    if len(rows) == 0:
        return None
    dr = draft(D, st, gamma, seed, rows)
    vf = verify(T, st, dr, rows)
    res = accept(st, gamma, dr, vf, seed, rows, bonus=bonus, **kw)
    st.round += 1
    return dr, vf, res


def sd_round_poisson(T: Model, st: State, gamma: int, rate: float, logp, seed: int, bonus=True, **kw):
    rows = np.nonzero(~st.done)[0]
    if len(rows) == 0:
        return None
    dr = draft_poisson(st, gamma, rate, logp, seed, rows)
    vf = verify(T, st, dr, rows)
    res = accept(st, gamma, dr, vf, seed, rows, bonus=bonus, **kw)
    st.round += 1
    return dr, vf, res


def sample_sd_poisson(T: Model, hist_t, hist_k, n_gen: int, gamma: int, rate: float, logp, seed: int,
                      bonus=True, seq0: int = 0, t_end=None, **kw) -> State:
    st = prefill(T, None, hist_t, hist_k, n_gen, seq0=seq0, t_end=t_end)
    while not np.all(st.done):
        sd_round_poisson(T, st, gamma, rate, logp, seed, bonus=bonus, **kw)
    return st


def sample_sd(T: Model, D: Model, hist_t, hist_k, n_gen: int, gamma: int, seed: int,
              bonus=True, seq0: int = 0, t_end=None, **kw) -> State:
    st = prefill(T, D, hist_t, hist_k, n_gen, seq0=seq0, t_end=t_end)
    while not np.all(st.done):
        sd_round(T, D, st, gamma, seed, bonus=bonus, **kw)
    return st


# ---------------------------------------------------------------------------
# model log-likelihood of sampled sequences (Eq. (2))
# ---------------------------------------------------------------------------

def loglik(T: Model, t, k, tau, n, first: int, t_end=None, stopped=None):
    """Eq. (2) for each sequence b, from one cache-free forward pass over its
    committed events 0 .. n[b] - 1: the sum over i = first .. n[b] - 1 of
    log g(tau_i | h_{i-1}) + log f(k_i | h_{i-1}), tau_i = tau[b, i] (the
    drawn interval), plus log(1 - G(T_b - t_{n-1} | h_{n-1})) when stopped[b]
    (a sequence ended by its end time T_b = t_end[b]). Returns [B] totals and
    the per-event terms [B, max n] (0 outside first .. n[b] - 1)."""
    t = np.asarray(t, dtype=np.float64)
    k = np.asarray(k, dtype=np.int64)
    n = np.asarray(n, dtype=np.int64)
    B = len(n)
    total = np.zeros(B)
    terms = np.zeros((B, int(n.max())))
    for b in range(B):
        N = int(n[b])
        h = T.forward_full(t[b:b + 1, :N], k[b:b + 1, :N])[0]
        logw, mu, s, logf = T.head(h)
        for i in range(first, N):
            terms[b, i] = mixture_logpdf(logw[i - 1], mu[i - 1], s[i - 1], tau[b, i]) + logf[i - 1, k[b, i]]
        total[b] = terms[b].sum()
        if stopped is not None and stopped[b]:
            total[b] += mixture_log_survival(logw[N - 1], mu[N - 1], s[N - 1], float(t_end[b]) - t[b, N - 1])
    return total, terms
