"""Pins for oracle.model (CDF-based Transformer TPP, §4.2 and App. D.4).

* temporal encoding: closed form of the THP encoding for D = 4 and general
  identities (z(0), shared frequency per sin/cos pair);
* LayerNorm and the pre-LN causal block stack: torch's LayerNorm and
  TransformerEncoderLayer(norm_first=True) in float64 with copied weights;
* decoder: torch.distributions MixtureSameFamily(LogNormal) log-density,
  scipy's lognorm, and a torch Linear/Tanh type head with copied weights;
* cached block forward == cache-free forward (causality invariant).
"""
import math

import numpy as np
import pytest
import scipy.stats
import torch
import torch.nn.functional as Fn

from oracle.model import Model
from oracle.sampler import mixture_logpdf
from paper_2507_09252_amd.workloads import ModelCfg, make_weights


def _model(prec="fp32", L=2, d=32, H=2, F=64, M=4, K=3, init="stress", seed=0):
    cfg = ModelCfg(L, d, H, F, M, K, prec)
    return Model(cfg, make_weights(cfg, np.random.SeedSequence([99, seed]), init))


def test_time_encoding_closed_form_d4():
    # D = 4: frequencies 10000^0 = 1 for j = 0, 1 and 10000^(-2/4) = 0.01 for j = 2, 3
    m = _model(d=4, H=1)
    t = np.array([2.0, 0.0, 7.25], dtype=np.float32)
    z = m.time_encoding(t)
    want = np.stack([np.sin(t), np.cos(t), np.sin(np.float32(t * np.float32(0.01))),
                     np.cos(np.float32(t * np.float32(0.01)))], -1)
    assert np.allclose(z, want, atol=1e-7)
    assert np.array_equal(z[1], [0.0, 1.0, 0.0, 1.0])


def test_time_encoding_identities():
    m = _model(d=64, H=4)
    t = np.random.default_rng(0).uniform(0, 500, 50).astype(np.float32)
    z = m.time_encoding(t)
    # sin/cos pairs share a frequency: z_2i^2 + z_2i+1^2 = 1
    assert np.allclose(z[:, 0::2] ** 2 + z[:, 1::2] ** 2, 1.0, atol=1e-12)
    assert np.allclose(m.time_encoding(np.zeros(1, np.float32))[0], np.tile([0.0, 1.0], 32))
    # pair frequencies decrease geometrically with ratio 10000^(-2/D)
    w = m.frequencies().astype(np.float64)
    assert np.allclose(w[2::2] / w[0:-2:2], 10000.0 ** (-2 / 64), rtol=1e-6)
    assert np.array_equal(w[0::2], w[1::2]) and w[0] == 1.0


def test_layer_norm_matches_torch():
    rng = np.random.default_rng(2)
    x, g, b = rng.normal(0, 3, (5, 48)), rng.normal(1, 0.1, 48), rng.normal(0, 0.1, 48)
    want = torch.nn.functional.layer_norm(torch.from_numpy(x), (48,), torch.from_numpy(g),
                                          torch.from_numpy(b), eps=1e-5).numpy()
    assert np.allclose(Model.layer_norm(x, g, b), want, atol=1e-12)


def _torch_stack(m: Model):
    layers = []
    for l in range(m.L):
        p = f"layers.{l}."
        enc = torch.nn.TransformerEncoderLayer(m.d, m.H, m.F, dropout=0.0, activation="relu",
                                               batch_first=True, norm_first=True).double()
        with torch.no_grad():
            enc.self_attn.in_proj_weight.copy_(torch.from_numpy(m.w[p + "qkv.w"]))
            enc.self_attn.in_proj_bias.copy_(torch.from_numpy(m.w[p + "qkv.b"]))
            enc.self_attn.out_proj.weight.copy_(torch.from_numpy(m.w[p + "out.w"]))
            enc.self_attn.out_proj.bias.copy_(torch.from_numpy(m.w[p + "out.b"]))
            enc.linear1.weight.copy_(torch.from_numpy(m.w[p + "ffn1.w"]))
            enc.linear1.bias.copy_(torch.from_numpy(m.w[p + "ffn1.b"]))
            enc.linear2.weight.copy_(torch.from_numpy(m.w[p + "ffn2.w"]))
            enc.linear2.bias.copy_(torch.from_numpy(m.w[p + "ffn2.b"]))
            enc.norm1.weight.copy_(torch.from_numpy(m.w[p + "ln1.g"]))
            enc.norm1.bias.copy_(torch.from_numpy(m.w[p + "ln1.b"]))
            enc.norm2.weight.copy_(torch.from_numpy(m.w[p + "ln2.g"]))
            enc.norm2.bias.copy_(torch.from_numpy(m.w[p + "ln2.b"]))
        enc.eval()
        layers.append(enc)
    lnf = torch.nn.LayerNorm(m.d, eps=1e-5).double()
    with torch.no_grad():
        lnf.weight.copy_(torch.from_numpy(m.w["lnf.g"]))
        lnf.bias.copy_(torch.from_numpy(m.w["lnf.b"]))
    return layers, lnf


@pytest.mark.parametrize("L,d,H,F", [(2, 32, 2, 64), (3, 64, 4, 128)])
def test_forward_full_matches_torch_encoder(L, d, H, F):
    m = _model(L=L, d=d, H=H, F=F)
    rng = np.random.default_rng(3)
    B, N = 3, 25
    t = np.cumsum(rng.exponential(1.0, (B, N)), 1).astype(np.float32)
    k = rng.integers(0, m.K, (B, N))
    got = m.forward_full(t, k)
    layers, lnf = _torch_stack(m)
    x = torch.from_numpy(m.embed(t, k))
    mask = torch.nn.Transformer.generate_square_subsequent_mask(N, dtype=torch.float64)
    with torch.no_grad():
        for enc in layers:
            x = enc(x, src_mask=mask, is_causal=True)
        want = lnf(x).numpy()
    assert np.allclose(got, want, atol=1e-10)


def test_decoder_matches_torch():
    m = _model(M=5, K=4)
    rng = np.random.default_rng(4)
    h = rng.normal(0, 1, (7, m.d))
    logw, mu, s, logf = m.head(h)
    d = m.d
    E = torch.nn.Linear(d, 3 * d, bias=False).double()
    heads = {n: torch.nn.Linear(d, m.M).double() for n in ("w", "mu", "sigma")}
    k1, k2 = torch.nn.Linear(d, d).double(), torch.nn.Linear(d, m.K).double()
    with torch.no_grad():
        E.weight.copy_(torch.from_numpy(m.w["head.E"]))
        for n, lin in heads.items():
            lin.weight.copy_(torch.from_numpy(m.w[f"head.{n}.w"]))
            lin.bias.copy_(torch.from_numpy(m.w[f"head.{n}.b"]))
        k1.weight.copy_(torch.from_numpy(m.w["head.k1.w"]))
        k1.bias.copy_(torch.from_numpy(m.w["head.k1.b"]))
        k2.weight.copy_(torch.from_numpy(m.w["head.k2.w"]))
        k2.bias.copy_(torch.from_numpy(m.w["head.k2.b"]))
        th = torch.from_numpy(h)
        e1, e2, e3 = E(th).chunk(3, dim=-1)
        w_t = torch.softmax(heads["w"](e1), -1)
        mu_t = heads["mu"](e2)
        sig_t = torch.exp(heads["sigma"](e3))
        f_t = torch.softmax(k2(torch.tanh(k1(th))), -1)
    assert np.allclose(np.exp(logw), w_t.numpy(), atol=1e-13)
    assert np.allclose(mu, mu_t.numpy(), atol=1e-13)
    assert np.allclose(np.exp(s), sig_t.numpy(), atol=1e-13)
    assert np.allclose(np.exp(logf), f_t.numpy(), atol=1e-13)
    # mixture log-density against torch.distributions and scipy
    tau = rng.lognormal(0, 1.5, 7)
    mix = torch.distributions.MixtureSameFamily(
        torch.distributions.Categorical(probs=w_t),
        torch.distributions.LogNormal(mu_t, sig_t))
    want = mix.log_prob(torch.from_numpy(tau)).numpy()
    got = mixture_logpdf(logw, mu, s, tau)
    assert np.allclose(got, want, atol=1e-12)
    want2 = np.log(np.sum(np.exp(logw) * scipy.stats.lognorm.pdf(tau[:, None], s=np.exp(s),
                                                                scale=np.exp(mu)), -1))
    assert np.allclose(got, want2, atol=1e-10)


def test_single_key_attention_returns_value():
    # one event: attention weight is 1 on itself, so the block output equals
    # x + W_o v + b_o with v the value of that event
    m = _model(L=1)
    t = np.array([[1.5]], np.float32)
    k = np.array([[2]])
    x = m.embed(t, k)
    a = Model.layer_norm(x, m.w["layers.0.ln1.g"], m.w["layers.0.ln1.b"])
    v = a @ m.w["layers.0.qkv.w"][2 * m.d:].T + m.w["layers.0.qkv.b"][2 * m.d:]
    x1 = x + v @ m.w["layers.0.out.w"].T + m.w["layers.0.out.b"]
    a2 = Model.layer_norm(x1, m.w["layers.0.ln2.g"], m.w["layers.0.ln2.b"])
    x2 = x1 + np.maximum(a2 @ m.w["layers.0.ffn1.w"].T + m.w["layers.0.ffn1.b"], 0) @ m.w["layers.0.ffn2.w"].T \
        + m.w["layers.0.ffn2.b"]
    want = Model.layer_norm(x2, m.w["lnf.g"], m.w["lnf.b"])
    assert np.allclose(m.forward_full(t, k), want, atol=1e-12)


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_block_equals_full_ragged(prec):
    m = _model(prec=prec, L=2, d=32, H=4)
    rng = np.random.default_rng(5)
    B, N = 4, 40
    t = np.cumsum(rng.exponential(1.0, (B, N)), 1).astype(np.float32)
    k = rng.integers(0, m.K, (B, N))
    full = m.forward_full(t, k)
    cache = m.new_cache(B, N + 8)
    # different cached lengths per sequence, then blocks of P = 1, 5, 3 events
    pos = np.array([10, 3, 17, 22])
    for b in range(B):
        m.forward_block(cache, t[b:b + 1, :pos[b]], k[b:b + 1, :pos[b]], np.array([0]), rows=[b])
    for P in (1, 5, 3):
        idx = pos[:, None] + np.arange(P)
        h = m.forward_block(cache, np.take_along_axis(t, idx, 1), np.take_along_axis(k, idx, 1), pos)
        want = np.stack([full[b, idx[b]] for b in range(B)])
        assert np.allclose(h, want, atol=1e-12)
        pos = pos + P


def test_causality():
    m = _model()
    rng = np.random.default_rng(6)
    t = np.cumsum(rng.exponential(1.0, (1, 20)), 1).astype(np.float32)
    k = rng.integers(0, m.K, (1, 20))
    h1 = m.forward_full(t, k)
    t2, k2 = t.copy(), k.copy()
    t2[0, 15] += 0.5
    k2[0, 17] = (k2[0, 17] + 1) % m.K
    h2 = m.forward_full(t2, k2)
    assert np.array_equal(h1[0, :15], h2[0, :15])
    assert not np.allclose(h1[0, 15:], h2[0, 15:])


def test_bf16_mode_rounds():
    mf = _model(prec="fp32", init="paper")
    cfg = ModelCfg(mf.L, mf.d, mf.H, mf.F, mf.M, mf.K, "bf16")
    mb = Model(cfg, {k: v for k, v in mf.w.items()})
    rng = np.random.default_rng(7)
    t = np.cumsum(rng.exponential(1.0, (2, 12)), 1).astype(np.float32)
    k = rng.integers(0, mf.K, (2, 12))
    hf, hb = mf.forward_full(t, k), mb.forward_full(t, k)
    rel = np.abs(hb - hf).max() / np.abs(hf).max()
    assert 1e-5 < rel < 3e-2          # bf16-sized perturbation, nothing larger
    lf = mf.head(hf)
    lb = mb.head(hb)
    assert np.abs(lf[0] - lb[0]).max() < 5e-2


# ---------------------------------------------------------------------------
# bf16 rounding points, pinned by an independent formulation
# ---------------------------------------------------------------------------

def _bf(x):
    """Round float64 values to bfloat16 (8 significant bits, round to nearest,
    ties to even) by integer arithmetic on the IEEE bits: of the 52 stored
    mantissa bits keep 7, adding 2^44 - 1 plus the lowest kept bit before
    truncating. (torch's own float64 -> bfloat16 cast goes through float32,
    a double rounding that differs at ties.)"""
    bits = x.contiguous().view(torch.int64)
    lsb = (bits >> 45) & 1
    bits = (bits + ((1 << 44) - 1) + lsb) & ~((1 << 45) - 1)
    return bits.view(torch.float64)


def test_bf_helper_matches_torch_on_float32_values():
    # on float32 inputs torch's cast rounds once, so the two must agree exactly (ties included)
    g = torch.Generator().manual_seed(0)
    x = (torch.randn(200000, generator=g) * 10).float()
    ties = (x.view(torch.int32) & ~0xFFFF) | 0x8000          # exact midpoints between bf16 values
    for v in (x, ties.view(torch.float32)):
        assert torch.equal(_bf(v.double()), v.to(torch.bfloat16).double())


BF16_POINTS = ("ln1", "qkv", "attn", "ln2", "relu", "lnf", "e", "tanh")


def _torch_thp_bf16(m: Model, t, k, skip=None):
    """A bf16 THP encoder + decoder written with torch primitives in float64:
    Linear inputs (the LayerNorm outputs, the attention output, the ReLU
    output, the decoder's LN_f output, e and the tanh output) and q, k, v
    after the bias are cast to bfloat16 and back; everything else (residual
    stream, LayerNorm statistics, softmax, decoder arithmetic) stays float64.
    Returns (log w, mu, s, log f) for every event. skip names one rounding
    point to leave out (the test's power check)."""
    W_ = {n: torch.from_numpy(v) for n, v in m.w.items()}

    def rb(x, point):
        return x if point == skip else _bf(x)
    d, H, dh = m.d, m.H, m.dh
    j = torch.arange(d, dtype=torch.float64)
    freq = torch.pow(torch.tensor(10000.0, dtype=torch.float64), -(j - torch.remainder(j, 2)) / d).float()
    arg = (torch.from_numpy(np.asarray(t, np.float32))[..., None] * freq).double()
    z = torch.where(torch.remainder(torch.arange(d), 2) == 0, torch.sin(arg), torch.cos(arg))
    x = z + W_["type_emb"][torch.from_numpy(np.asarray(k))]
    B, N, _ = x.shape
    for l in range(m.L):
        p = f"layers.{l}."
        a = rb(Fn.layer_norm(x, (d,), W_[p + "ln1.g"], W_[p + "ln1.b"], eps=1e-5), "ln1")
        qkv = rb(Fn.linear(a, W_[p + "qkv.w"], W_[p + "qkv.b"]), "qkv")
        q, kk, v = (qkv[..., i * d:(i + 1) * d].reshape(B, N, H, dh).transpose(1, 2) for i in range(3))
        o = Fn.scaled_dot_product_attention(q, kk, v, is_causal=True)
        x = x + Fn.linear(rb(o.transpose(1, 2).reshape(B, N, d), "attn"), W_[p + "out.w"], W_[p + "out.b"])
        a2 = rb(Fn.layer_norm(x, (d,), W_[p + "ln2.g"], W_[p + "ln2.b"], eps=1e-5), "ln2")
        hid = rb(torch.relu(Fn.linear(a2, W_[p + "ffn1.w"], W_[p + "ffn1.b"])), "relu")
        x = x + Fn.linear(hid, W_[p + "ffn2.w"], W_[p + "ffn2.b"])
    h = rb(Fn.layer_norm(x, (d,), W_["lnf.g"], W_["lnf.b"], eps=1e-5), "lnf")
    e = rb(Fn.linear(h, W_["head.E"]), "e")
    logw = torch.log_softmax(Fn.linear(e[..., :d], W_["head.w.w"], W_["head.w.b"]), -1)
    mu = Fn.linear(e[..., d:2 * d], W_["head.mu.w"], W_["head.mu.b"])
    s = Fn.linear(e[..., 2 * d:], W_["head.sigma.w"], W_["head.sigma.b"])
    th = rb(torch.tanh(Fn.linear(h, W_["head.k1.w"], W_["head.k1.b"])), "tanh")
    logf = torch.log_softmax(Fn.linear(th, W_["head.k2.w"], W_["head.k2.b"]), -1)
    return tuple(a.numpy() for a in (logw, mu, s, logf))


@pytest.mark.parametrize("init", ["paper", "stress"])
@pytest.mark.parametrize("L,d,H,F", [(2, 64, 4, 256), (1, 32, 2, 64)])
def test_bf16_rounding_points_match_torch(L, d, H, F, init):
    """The oracle's bf16 mode (forward_full, forward_block on a cache, head)
    against the independent torch formulation: agreement to 1e-12 means every
    rounding point is where the formulation puts it; a missing or extra
    rounding moves outputs by about a bf16 ulp (4e-3 relative) and fails."""
    cfg = ModelCfg(L, d, H, F, 6, 5, "bf16")
    m = Model(cfg, make_weights(cfg, np.random.SeedSequence([98, L]), init))
    rng = np.random.default_rng(8)
    B, N = 3, 21
    t = np.cumsum(rng.exponential(1.0, (B, N)), 1).astype(np.float32)
    k = rng.integers(0, m.K, (B, N))
    want = _torch_thp_bf16(m, t, k)
    got = m.head(m.forward_full(t, k))
    for g, w in zip(got, want):
        np.testing.assert_allclose(g, w, rtol=0, atol=1e-12)
    # the cached block pass (as verification runs it): ragged cached lengths, then a block of 6
    cache = m.new_cache(B, N + 4)
    pos = np.array([7, 12, 15])
    for b in range(B):
        m.forward_block(cache, t[b:b + 1, :pos[b]], k[b:b + 1, :pos[b]], np.array([0]), rows=[b])
    idx = pos[:, None] + np.arange(6)
    hb = m.forward_block(cache, np.take_along_axis(t, idx, 1), np.take_along_axis(k, idx, 1), pos)
    got_b = m.head(hb)
    for g, w in zip(got_b, want):
        np.testing.assert_allclose(g, np.stack([w[b, idx[b]] for b in range(B)]), rtol=0, atol=1e-12)
    # power: leaving out any single rounding point moves the outputs far beyond the bar
    for point in BF16_POINTS:
        alt = _torch_thp_bf16(m, t, k, skip=point)
        assert max(np.abs(a - w).max() for a, w in zip(alt, want)) > 1e-7, point
