"""Seeded synthetic inputs: model configurations, weights and seed histories.

This module holds input generation only. It contains none of the sampling
method's arithmetic (no encoder, no decoder, no accept rule), so the CPU oracle
and the HIP path can both consume its outputs without sharing any of the
method's code.

The five workloads follow the synthetic settings used for TPP-SD sampling
(CDF-based Transformer TPP of §4.2, sampled by Algorithm 1): a tiny
univariate case, a univariate Hawkes-shaped case, a 22-type case swept over
the draft length, a long-history KV-cache stress case and a throughput batch.
Seed histories come from the processes named for each workload, simulated by
thinning (Lewis-Shedler for Poisson processes, Ogata for Hawkes processes,
the proposal/accept scheme of §2.2).

Weights: every Linear matrix and the type-embedding matrix are drawn
N(0, 0.02^2); biases are 0; LayerNorm gains 1 and offsets 0. For bf16
workloads the matrices are rounded to bf16 here, so both implementations read
identical values. Two extra initialisations serve the tests: ``"stress"``
(larger weights and non-zero biases, so that a wrong bias, gain or index shows
up in the outputs) and a ``"mismatch"`` draft perturbation that lowers the
acceptance rate.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Tuple

import numpy as np
import torch

PREC_FP32 = "fp32"
PREC_BF16 = "bf16"


ENC_THP = "thp"          # THP encoder: summed encoding, pre-LN softmax-attention blocks with FFN
ENC_ATTNHP = "attnhp"    # AttNHP encoder (App. D.4): q, k, v from [1; z(t); h], h += tanh(attention)


@dataclasses.dataclass(frozen=True)
class ModelCfg:
    n_layers: int
    d_model: int
    n_heads: int
    d_ffn: int
    n_mix: int
    n_types: int
    prec: str = PREC_FP32
    encoder: str = ENC_THP
    time_m: float = 1.0      # AttNHP time encoding: shortest wavelength scale m
    time_M: float = 100.0    # ... and M (longest wavelength 5 M)

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_heads


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int
    target: ModelCfg
    draft: ModelCfg
    batch: int
    n_gen: int
    gammas: Tuple[int, ...]
    n_hist: int
    history: str          # generator name, see make_histories
    description: str

    @property
    def gamma(self) -> int:
        return self.gammas[0] if len(self.gammas) == 1 else 10

    @property
    def prec(self) -> str:
        return self.target.prec


def _cfg(L, d, H, F, M, K, prec, enc=ENC_THP, tm=1.0, tM=100.0):
    return ModelCfg(L, d, H, F, M, K, prec, enc, tm, tM)


# Draft FFN width keeps the target's F/d ratio; draft M equals the target's.
WORKLOADS: Dict[str, Workload] = {
    "c1": Workload(
        "c1", 0, _cfg(2, 32, 2, 64, 4, 1, PREC_FP32), _cfg(1, 16, 1, 32, 4, 1, PREC_FP32),
        batch=1, n_gen=200, gammas=(4,), n_hist=20, history="hpp",
        description="tiny univariate fp32, B=1 x 200 events, gamma=4"),
    "c2": Workload(
        "c2", 1, _cfg(4, 64, 4, 256, 8, 1, PREC_FP32), _cfg(1, 32, 2, 128, 8, 1, PREC_FP32),
        batch=64, n_gen=500, gammas=(10,), n_hist=50, history="hawkes1",
        description="univariate Hawkes-shaped fp32, B=64 x 500 events, gamma=10"),
    "c3": Workload(
        "c3", 2, _cfg(6, 256, 8, 1024, 16, 22, PREC_BF16), _cfg(2, 64, 4, 256, 16, 22, PREC_BF16),
        batch=256, n_gen=1024, gammas=(1, 2, 5, 10, 15, 20), n_hist=64, history="hawkes22",
        description="22-type bf16, B=256 x 1024 events, gamma in {1,2,5,10,15,20}"),
    "c4": Workload(
        "c4", 3, _cfg(8, 512, 8, 2048, 16, 5, PREC_BF16), _cfg(2, 128, 4, 512, 16, 5, PREC_BF16),
        batch=32, n_gen=4096, gammas=(16,), n_hist=512, history="hawkes5",
        description="long-history bf16, B=32 x 4096 events, gamma=16"),
    "c5": Workload(
        "c5", 4, _cfg(6, 128, 4, 512, 8, 3, PREC_BF16), _cfg(1, 32, 2, 128, 8, 3, PREC_BF16),
        batch=4096, n_gen=256, gammas=(8,), n_hist=32, history="ipp_sin",
        description="throughput bf16, B=4096 x 256 events, gamma=8"),
    # c3's data and sizes with the AttNHP encoder (App. D.4) for target and draft
    "a3": Workload(
        "a3", 5, _cfg(6, 256, 8, 0, 16, 22, PREC_BF16, ENC_ATTNHP, 0.01, 100.0),
        _cfg(2, 64, 4, 0, 16, 22, PREC_BF16, ENC_ATTNHP, 0.01, 100.0),
        batch=256, n_gen=1024, gammas=(10,), n_hist=64, history="hawkes22",
        description="c3 with the AttNHP encoder, bf16, B=256 x 1024 events, gamma=10"),
}


def seed_sequence(workload_index: int, stream: int) -> np.random.SeedSequence:
    """Streams: 1 = target weights, 2 = draft weights, 3 = histories."""
    return np.random.SeedSequence([0, workload_index, stream])


# ---------------------------------------------------------------------------
# weights
# ---------------------------------------------------------------------------

def weight_names(cfg: ModelCfg) -> List[Tuple[str, Tuple[int, ...], str]]:
    """(name, shape, kind) for every parameter; kind in {mat, bias, ln_g, ln_b}.

    Linear matrices are stored [out, in]. The fused QKV matrix stacks the
    query, key and value projections along its output rows (in that order);
    head h owns columns h*d_head .. (h+1)*d_head-1 of each.
    """
    d, F, M, K = cfg.d_model, cfg.d_ffn, cfg.n_mix, cfg.n_types
    out = [("type_emb", (K, d), "mat")]
    if cfg.encoder == ENC_ATTNHP:
        # q, k, v = W [z(t); h] + b, W in R^{3d x 2d}: the constant input 1 of
        # the concatenation is the bias column
        for l in range(cfg.n_layers):
            p = f"layers.{l}."
            out += [(p + "qkv.w", (3 * d, 2 * d), "mat"), (p + "qkv.b", (3 * d,), "bias")]
        return out + _decoder_names(d, M, K)
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        out += [
            (p + "ln1.g", (d,), "ln_g"), (p + "ln1.b", (d,), "ln_b"),
            (p + "qkv.w", (3 * d, d), "mat"), (p + "qkv.b", (3 * d,), "bias"),
            (p + "out.w", (d, d), "mat"), (p + "out.b", (d,), "bias"),
            (p + "ln2.g", (d,), "ln_g"), (p + "ln2.b", (d,), "ln_b"),
            (p + "ffn1.w", (F, d), "mat"), (p + "ffn1.b", (F,), "bias"),
            (p + "ffn2.w", (d, F), "mat"), (p + "ffn2.b", (d,), "bias"),
        ]
    out += [("lnf.g", (d,), "ln_g"), ("lnf.b", (d,), "ln_b")]
    return out + _decoder_names(d, M, K)


def _decoder_names(d, M, K):
    return [
        ("head.E", (3 * d, d), "mat"),
        ("head.w.w", (M, d), "mat"), ("head.w.b", (M,), "bias"),
        ("head.mu.w", (M, d), "mat"), ("head.mu.b", (M,), "bias"),
        ("head.sigma.w", (M, d), "mat"), ("head.sigma.b", (M,), "bias"),
        ("head.k1.w", (d, d), "mat"), ("head.k1.b", (d,), "bias"),
        ("head.k2.w", (K, d), "mat"), ("head.k2.b", (K,), "bias"),
    ]


def to_bf16_values(a: np.ndarray) -> np.ndarray:
    """Round float values to the nearest bf16 (torch's RNE conversion)."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def make_weights(cfg: ModelCfg, ss: np.random.SeedSequence, init: str = "paper") -> Dict[str, np.ndarray]:
    """Seeded parameters as float32 arrays (bf16-representable when cfg.prec is bf16).

    init = "paper": matrices N(0, 0.02^2), biases 0, LN (1, 0).
    init = "bias": as "paper" but biases N(0, 0.1^2), LN gains 1 + N(0, 0.1^2), offsets N(0, 0.1^2).
    init = "stress": matrices N(0, s^2) with s = 1/sqrt(fan_in), biases N(0, 0.1^2),
                     LN gains 1 + N(0, 0.1^2), offsets N(0, 0.1^2).
    """
    rng = np.random.default_rng(ss)
    out: Dict[str, np.ndarray] = {}
    for name, shape, kind in weight_names(cfg):
        if init == "paper":
            if kind == "mat":
                v = rng.normal(0.0, 0.02, size=shape)
            elif kind == "ln_g":
                v = np.ones(shape)
            else:
                v = np.zeros(shape)
        elif init == "bias":
            # paper-scale matrices, non-zero biases and LayerNorm parameters
            if kind == "mat":
                v = rng.normal(0.0, 0.02, size=shape)
            elif kind == "ln_g":
                v = 1.0 + rng.normal(0.0, 0.1, size=shape)
            else:
                v = rng.normal(0.0, 0.1, size=shape)
        elif init == "stress":
            if kind == "mat":
                fan_in = shape[1]
                scale = 1.0 if name == "type_emb" else 1.0 / np.sqrt(fan_in)
                v = rng.normal(0.0, scale, size=shape)
            elif kind == "ln_g":
                v = 1.0 + rng.normal(0.0, 0.1, size=shape)
            else:
                v = rng.normal(0.0, 0.1, size=shape)
        else:
            raise ValueError(init)
        v = v.astype(np.float32)
        if cfg.prec == PREC_BF16 and kind == "mat":
            v = to_bf16_values(v)
        out[name] = v
    return out


def mismatch_draft(weights: Dict[str, np.ndarray], cfg: ModelCfg, ss: np.random.SeedSequence) -> Dict[str, np.ndarray]:
    """Shift the draft's decoder biases so that it disagrees with the target.

    b_mu += 0.5, b_sigma += 0.3 and b_k2 += N(0, 0.5^2): lowers the acceptance
    rate to the range reported for trained models, which gives the
    distribution tests power.
    """
    rng = np.random.default_rng(ss)
    w = {k: v.copy() for k, v in weights.items()}
    w["head.mu.b"] = (w["head.mu.b"] + 0.5).astype(np.float32)
    w["head.sigma.b"] = (w["head.sigma.b"] + 0.3).astype(np.float32)
    w["head.k2.b"] = (w["head.k2.b"] + rng.normal(0, 0.5, size=w["head.k2.b"].shape)).astype(np.float32)
    return w


def workload_weights(wl: Workload, init: str = "paper"):
    wt = make_weights(wl.target, seed_sequence(wl.index, 1), init)
    wd = make_weights(wl.draft, seed_sequence(wl.index, 2), init)
    return wt, wd


# ---------------------------------------------------------------------------
# seed histories (thinning, §2.2)
# ---------------------------------------------------------------------------

def hpp(n: int, rate: float, rng: np.random.Generator):
    tau = rng.exponential(1.0 / rate, size=n)
    return np.cumsum(tau), np.zeros(n, dtype=np.int64)


def ipp_sin(n: int, rng: np.random.Generator, n_types: int = 1):
    """lambda(t) = 1 + 0.5 sin(2 pi t / 10), Lewis-Shedler thinning with bound 1.5."""
    lam_bar = 1.5
    t, out = 0.0, []
    while len(out) < n:
        t += rng.exponential(1.0 / lam_bar)
        if rng.uniform() * lam_bar < 1.0 + 0.5 * np.sin(2 * np.pi * t / 10.0):
            out.append(t)
    ts = np.asarray(out)
    ks = rng.integers(0, n_types, size=n) if n_types > 1 else np.zeros(n, dtype=np.int64)
    return ts, ks


def ipp_sin_compensator(t0: float, t1: float) -> float:
    """Integral of 1 + 0.5 sin(2 pi t / 10) over [t0, t1]."""
    c = 10.0 / (2 * np.pi)
    return (t1 - t0) - 0.5 * c * (np.cos(t1 / c) - np.cos(t0 / c))


def hawkes(n: int, mu: np.ndarray, alpha: np.ndarray, beta: np.ndarray, rng: np.random.Generator):
    """Multivariate Hawkes process with exponential kernels, Ogata thinning from t = 0.

    lambda_i(t) = mu_i + sum_j sum_{t_e of type j, t_e < t} alpha[i, j] exp(-beta[i, j] (t - t_e)).
    Between events every intensity decays, so the total intensity just after
    the current time bounds it until the next accepted event.
    """
    K = len(mu)
    S = np.zeros((K, K))          # S[i, j] = sum over type-j events of exp(-beta_ij (t - t_e))
    t = 0.0
    ts, ks = [], []
    while len(ts) < n:
        lam_bar = float(np.sum(mu + np.sum(alpha * S, axis=1)))
        dt = rng.exponential(1.0 / lam_bar)
        S_new = S * np.exp(-beta * dt)
        lam = mu + np.sum(alpha * S_new, axis=1)
        t += dt
        S = S_new
        if rng.uniform() * lam_bar < lam.sum():
            k = int(np.searchsorted(np.cumsum(lam), rng.uniform() * lam.sum(), side="right"))
            k = min(k, K - 1)
            ts.append(t)
            ks.append(k)
            S[:, k] += 1.0
    return np.asarray(ts), np.asarray(ks, dtype=np.int64)


def hawkes_compensator_intervals(ts, ks, mu, alpha, beta) -> np.ndarray:
    """Total compensator over each inter-event interval (time-rescaling theorem)."""
    K = len(mu)
    S = np.zeros((K, K))
    prev = 0.0
    out = []
    for t, k in zip(ts, ks):
        dt = t - prev
        decay = np.exp(-beta * dt)
        # integral of alpha S exp(-beta s) ds over [0, dt] for each (i, j)
        integ = np.sum(alpha * S * (1.0 - decay) / beta)
        out.append(np.sum(mu) * dt + integ)
        S = S * decay
        S[:, k] += 1.0
        prev = t
    return np.asarray(out)


def _spectral_scale(A: np.ndarray, target: float) -> np.ndarray:
    rho = float(np.max(np.abs(np.linalg.eigvals(A))))
    return A * (target / rho) if rho > 0 else A


def hawkes_params(kind: str, rng: np.random.Generator):
    if kind == "hawkes1":
        return np.array([0.2]), np.array([[0.8]]), np.array([[1.0]])
    if kind == "hawkes22":
        K = 22
        mu = (np.arange(1, K + 1) ** -1.2)
        mu = mu / mu.sum()
        mask = rng.uniform(size=(K, K)) < 0.15
        alpha = np.where(mask, rng.uniform(size=(K, K)), 0.0)
        beta = np.ones((K, K))
        alpha = _spectral_scale(alpha / beta, 0.7) * beta
        return mu, alpha, beta
    if kind == "hawkes5":
        K = 5
        mu = np.full(K, 0.1)
        beta = rng.uniform(0.5, 2.0, size=(K, K))
        alpha = rng.uniform(size=(K, K))
        alpha = _spectral_scale(alpha / beta, 0.5) * beta
        return mu, alpha, beta
    raise ValueError(kind)


def make_histories(wl: Workload, batch: int | None = None, n_hist: int | None = None):
    """Seed histories t[B, n0] (float32, strictly increasing) and k[B, n0] (int32)."""
    B = wl.batch if batch is None else batch
    n = wl.n_hist if n_hist is None else n_hist
    rng = np.random.default_rng(seed_sequence(wl.index, 3))
    K = wl.target.n_types
    T = np.zeros((B, n), dtype=np.float64)
    Kk = np.zeros((B, n), dtype=np.int64)
    if wl.history.startswith("hawkes"):
        mu, alpha, beta = hawkes_params(wl.history, rng)
    for b in range(B):
        if wl.history == "hpp":
            t, k = hpp(n, 1.0, rng)
        elif wl.history == "ipp_sin":
            t, k = ipp_sin(n, rng, K)
        else:
            t, k = hawkes(n, mu, alpha, beta, rng)
            if wl.history == "hawkes22":
                # per-sequence inter-event scale, log-uniform on [1e-2, 1e2]
                t = t * float(np.exp(rng.uniform(np.log(1e-2), np.log(1e2))))
        T[b], Kk[b] = t, k
    t32 = T.astype(np.float32)
    # keep times strictly increasing after the float32 cast
    for b in range(B):
        for i in range(1, n):
            if t32[b, i] <= t32[b, i - 1]:
                t32[b, i] = np.nextafter(t32[b, i - 1], np.float32(np.inf))
    return t32, Kk.astype(np.int32)
