"""Pins for the oracle's AttNHP encoder (App. D.4).

* temporal encoding: closed form for D = 4 (wavelengths m and m (5M/m)^(1/2));
* one layer against an independent torch formulation: the 1 in the
  denominator of the AttNHP attention is an extra key with score 0 and value
  0, so torch's scaled_dot_product_attention over the keys with a zero key and
  a zero value prepended (visible to every query) must give the same output;
* the whole stack against the same torch formulation, layer by layer;
* cached block forward == cache-free forward (ragged chunks), causality;
* TPP-SD with AttNHP target and draft has the law of AR sampling.
"""
import concurrent.futures as cf
import multiprocessing as mp
import os

import numpy as np
import torch
import torch.nn.functional as Fn

from oracle import sampler as S
from oracle.model import Model
from paper_2507_09252_amd import workloads as W
from test_oracle_sd_law import _pvalues


def _model(prec="fp32", L=2, d=32, H=2, M=4, K=3, init="stress", seed=0, m=0.5, Mx=50.0):
    cfg = W.ModelCfg(L, d, H, 0, M, K, prec, W.ENC_ATTNHP, m, Mx)
    return Model(cfg, W.make_weights(cfg, np.random.SeedSequence([77, seed]), init))


def test_attnhp_encoding_closed_form_d4():
    # D = 4: wavelengths m for j = 0, 1 and m (5M/m)^(2/4) for j = 2, 3
    mo = _model(d=4, H=1, m=0.5, Mx=50.0)
    t = np.array([1.3, 0.0, 40.0], dtype=np.float32)
    w0 = np.float32(1.0 / 0.5)
    w2 = np.float32(1.0 / (0.5 * np.sqrt(500.0)))
    z = mo.time_encoding(t)
    a0, a2 = (t * w0).astype(np.float32), (t * w2).astype(np.float32)
    want = np.stack([np.sin(a0), np.cos(a0), np.sin(a2), np.cos(a2)], -1)
    np.testing.assert_allclose(z, want, atol=1e-7)
    assert np.array_equal(z[1], [0.0, 1.0, 0.0, 1.0])


def _torch_attnhp(mo: Model, t, k):
    """The AttNHP stack with torch primitives: Linear on cat(z, h), causal
    scaled_dot_product_attention over [zero key; keys] / [zero value; values]."""
    z = torch.from_numpy(mo.time_encoding(t))
    h = torch.from_numpy(mo.w["type_emb"][k])
    B, N, D = h.shape
    H, dh = mo.H, mo.dh
    allow = torch.ones(N, N + 1, dtype=torch.bool).tril(diagonal=1)   # column 0: the zero key
    for l in range(mo.L):
        W_ = torch.from_numpy(mo.w[f"layers.{l}.qkv.w"])
        b_ = torch.from_numpy(mo.w[f"layers.{l}.qkv.b"])
        qkv = Fn.linear(torch.cat([z, h], -1), W_, b_)
        q, kk, v = (qkv[..., i * D:(i + 1) * D].reshape(B, N, H, dh).transpose(1, 2) for i in range(3))
        zero = torch.zeros(B, H, 1, dh, dtype=torch.float64)
        o = Fn.scaled_dot_product_attention(q, torch.cat([zero, kk], 2), torch.cat([zero, v], 2),
                                            attn_mask=allow)
        h = h + torch.tanh(o.transpose(1, 2).reshape(B, N, D))
    return h.numpy()


def test_attnhp_stack_matches_torch():
    rng = np.random.default_rng(3)
    for L, d, H in [(1, 16, 1), (2, 32, 2), (3, 64, 4)]:
        mo = _model(L=L, d=d, H=H, seed=L)
        t = np.cumsum(rng.exponential(1.0, (2, 15)), axis=1).astype(np.float32)
        k = rng.integers(0, 3, (2, 15))
        np.testing.assert_allclose(mo.forward_full(t, k), _torch_attnhp(mo, t, k), rtol=1e-11, atol=1e-11)


def test_attnhp_sink_limits():
    # one event: its own key only, weight f = exp(q.k / sqrt(d_h)), output v f / (1 + f)
    mo = _model(L=1, d=16, H=1, seed=5)
    t = np.array([[0.7]], dtype=np.float32)
    k = np.array([[1]])
    z = mo.time_encoding(t)[0, 0]
    h0 = mo.w["type_emb"][1]
    qkv = mo.w["layers.0.qkv.w"] @ np.concatenate([z, h0]) + mo.w["layers.0.qkv.b"]
    q, kk, v = qkv[:16], qkv[16:32], qkv[32:]
    f = np.exp(q @ kk / 4.0)
    np.testing.assert_allclose(mo.forward_full(t, k)[0, 0], h0 + np.tanh(v * f / (1.0 + f)), rtol=1e-12)


def test_attnhp_block_equals_full_ragged():
    for prec in ("fp32", "bf16"):
        mo = _model(prec=prec, L=2, d=32, H=2, seed=7)
        rng = np.random.default_rng(11)
        t = np.cumsum(rng.exponential(1.0, (3, 17)), axis=1).astype(np.float32)
        k = rng.integers(0, 3, (3, 17))
        full = mo.forward_full(t, k)
        cache = mo.new_cache(3, 24)
        outs, p0 = [], 0
        for P in (5, 1, 7, 4):
            outs.append(mo.forward_block(cache, t[:, p0:p0 + P], k[:, p0:p0 + P], np.full(3, p0)))
            p0 += P
        np.testing.assert_allclose(np.concatenate(outs, 1), full, rtol=1e-12, atol=1e-12)
        # causality: changing a later event leaves earlier outputs unchanged
        t2 = t.copy()
        t2[:, 10] += np.float32(0.5)
        np.testing.assert_array_equal(mo.forward_full(t2, k)[:, :10], full[:, :10])


GAMMA, N_GEN = 3, 8
TCFG = W.ModelCfg(2, 32, 2, 0, 4, 3, "fp32", W.ENC_ATTNHP, 0.5, 20.0)
DCFG = W.ModelCfg(1, 16, 1, 0, 4, 3, "fp32", W.ENC_ATTNHP, 0.5, 20.0)


def _models():
    wt = W.make_weights(TCFG, np.random.SeedSequence([6, 1]), "stress")
    wd = W.mismatch_draft(W.make_weights(DCFG, np.random.SeedSequence([6, 2]), "stress"), DCFG,
                          np.random.SeedSequence([6, 3]))
    return Model(TCFG, wt), Model(DCFG, wd)


def _history(B):
    rng = np.random.default_rng(1)
    ht = np.cumsum(rng.exponential(1.0, 20))
    hk = rng.integers(0, 3, 20)
    return np.tile(ht.astype(np.float32), (B, 1)), np.tile(hk.astype(np.int32), (B, 1))


def _chunk(args):
    kind, seq0, B = args
    T, D = _models()
    HT, HK = _history(B)
    if kind == "ar":
        st = S.sample_ar(T, HT, HK, N_GEN, seed=13, seq0=seq0)
    else:
        st = S.sample_sd(T, D, HT, HK, N_GEN, GAMMA, seed=13, seq0=seq0)
    n0 = HT.shape[1]
    return (np.diff(st.t[:, n0 - 1:n0 + N_GEN], axis=1), st.k[:, n0:n0 + N_GEN], st.accepted_drafts, st.drafted)


def _run(kind, n, chunk=1500):
    jobs = [(kind, s, min(chunk, n - s)) for s in range(0, n, chunk)]
    with cf.ProcessPoolExecutor(max(1, min(8, os.cpu_count() or 1)), mp_context=mp.get_context("fork")) as ex:
        parts = list(ex.map(_chunk, jobs))
    return (np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts]),
            sum(p[2] for p in parts) / max(1, sum(p[3] for p in parts)))


def test_attnhp_sd_law_equals_ar():
    ar = _run("ar", 12000)
    sd = _run("sd", 12000)
    assert 0.2 < sd[2] < 0.9, sd[2]
    ps = _pvalues(ar, sd)
    assert ps.min() > 0.01 / len(ps), ps


# ---------------------------------------------------------------------------
# bf16 rounding points, pinned by an independent formulation
# ---------------------------------------------------------------------------

def _bf(x):
    """float64 -> bfloat16 -> float64 by integer arithmetic on the IEEE bits
    (round to nearest, ties to even: keep 7 of the 52 stored mantissa bits)."""
    bits = x.contiguous().view(torch.int64)
    lsb = (bits >> 45) & 1
    return ((bits + ((1 << 44) - 1) + lsb) & ~((1 << 45) - 1)).view(torch.float64)


ATTNHP_BF16_POINTS = ("z", "h", "qkv", "attn", "dec_h", "e", "tanh")


def _torch_attnhp_bf16(mo: Model, t, k, skip=None):
    """bf16 AttNHP stack + decoder with torch primitives in float64: both
    halves of the layer input [z; h], q, k, v after the bias, the attention
    output before tanh, and the decoder's Linear inputs (h, e, the tanh
    output) are rounded to bfloat16; the rest stays float64. The time
    encoding is computed here from its definition (float32 wavelength table,
    float32 product t * omega). Returns (log w, mu, s, log f)."""
    W_ = {n: torch.from_numpy(v) for n, v in mo.w.items()}

    def rb(x, point):
        return x if point == skip else _bf(x)

    D, H, dh = mo.d, mo.H, mo.dh
    j = torch.arange(D, dtype=torch.float64)
    m_, M_ = float(mo.cfg.time_m), float(mo.cfg.time_M)
    omega = (1.0 / (m_ * torch.pow(torch.tensor(5.0 * M_ / m_, dtype=torch.float64),
                                   (j - torch.remainder(j, 2)) / D))).float()
    arg = (torch.from_numpy(np.asarray(t, np.float32))[..., None] * omega).double()
    z = torch.where(torch.remainder(torch.arange(D), 2) == 0, torch.sin(arg), torch.cos(arg))
    h = W_["type_emb"][torch.from_numpy(np.asarray(k))]
    B, N, _ = h.shape
    allow = torch.ones(N, N + 1, dtype=torch.bool).tril(diagonal=1)   # column 0: the zero key
    for l in range(mo.L):
        u = torch.cat([rb(z, "z"), rb(h, "h")], -1)
        qkv = rb(Fn.linear(u, W_[f"layers.{l}.qkv.w"], W_[f"layers.{l}.qkv.b"]), "qkv")
        q, kk, v = (qkv[..., i * D:(i + 1) * D].reshape(B, N, H, dh).transpose(1, 2) for i in range(3))
        zero = torch.zeros(B, H, 1, dh, dtype=torch.float64)
        o = Fn.scaled_dot_product_attention(q, torch.cat([zero, kk], 2), torch.cat([zero, v], 2), attn_mask=allow)
        h = h + torch.tanh(rb(o.transpose(1, 2).reshape(B, N, D), "attn"))
    hb = rb(h, "dec_h")
    e = rb(Fn.linear(hb, W_["head.E"]), "e")
    logw = torch.log_softmax(Fn.linear(e[..., :D], W_["head.w.w"], W_["head.w.b"]), -1)
    mu = Fn.linear(e[..., D:2 * D], W_["head.mu.w"], W_["head.mu.b"])
    s = Fn.linear(e[..., 2 * D:], W_["head.sigma.w"], W_["head.sigma.b"])
    th = rb(torch.tanh(Fn.linear(hb, W_["head.k1.w"], W_["head.k1.b"])), "tanh")
    logf = torch.log_softmax(Fn.linear(th, W_["head.k2.w"], W_["head.k2.b"]), -1)
    return tuple(a.numpy() for a in (logw, mu, s, logf))


def test_attnhp_bf16_rounding_points_match_torch():
    """The oracle's bf16 AttNHP (cache-free and cached block forward, decoder)
    against the independent formulation to 1e-12; leaving out any single
    rounding point moves the outputs far beyond that."""
    rng = np.random.default_rng(12)
    for L, d, H, init in [(2, 32, 2, "stress"), (2, 64, 4, "paper")]:
        cfg = W.ModelCfg(L, d, H, 0, 5, 4, "bf16", W.ENC_ATTNHP, 0.01, 100.0)
        mo = Model(cfg, W.make_weights(cfg, np.random.SeedSequence([78, L, d]), init))
        t = np.cumsum(rng.exponential(1.0, (3, 19)), axis=1).astype(np.float32)
        k = rng.integers(0, 4, (3, 19))
        want = _torch_attnhp_bf16(mo, t, k)
        for g, w in zip(mo.head(mo.forward_full(t, k)), want):
            np.testing.assert_allclose(g, w, rtol=0, atol=1e-12)
        cache = mo.new_cache(3, 24)
        mo.forward_block(cache, t[:, :11], k[:, :11], np.zeros(3, np.int64))
        for g, w in zip(mo.head(mo.forward_block(cache, t[:, 11:], k[:, 11:], np.full(3, 11))), want):
            np.testing.assert_allclose(g, w[:, 11:], rtol=0, atol=1e-12)
        for point in ATTNHP_BF16_POINTS:
            alt = _torch_attnhp_bf16(mo, t, k, skip=point)
            assert max(np.abs(a - w).max() for a, w in zip(alt, want)) > 1e-7, point
