"""CDF-based Transformer TPP (§4.2 "CDF-based Transformer TPPs"), float64 oracle.

ORACLE / TEST INFRASTRUCTURE (see oracle/__init__.py).

Encoder (§4.2 "Encoder", App. D.4 THP form):
  * temporal encoding z(t): component j uses frequency 10000^(-(j - j mod 2)/D),
    sine for even j and cosine for odd j, evaluated at the absolute time t;
  * type embedding: row k of W (K x D), fused with z(t) by summation;
  * Transformer T_theta: causal self-attention blocks (App. D.4 THP/SAHP form:
    softmax-normalised exp(q.k / sqrt(d)) weights over the event and its
    predecessors, residual connection, linear q, k, v).
Decoder (§4.2 "Decoder"):
  * e = E h with E in R^{3D x D}, sliced into e1, e2, e3;
  * w = softmax(V_w e1 + b_w), mu = V_mu e2 + b_mu, sigma = exp(V_sigma e3 + b_sigma);
  * f(k | h) = softmax(V_k2 tanh(V_k1 h + b_k1) + b_k2).
The head at event i gives the distribution of event i + 1.

Readings where the paper leaves the block unspecified (all listed in the
design notes): multi-head attention with scale 1/sqrt(d_head) per head,
pre-LayerNorm blocks x += Attn(LN1(x)); x += FFN(LN2(x)) with a ReLU FFN,
a final LayerNorm before the decoder, LayerNorm with biased variance and
eps = 1e-5, no dropout, V_k1 of size D x D, E without bias, sigma kept as
s = log(sigma). Times are float32; the encoding's argument is the float32
product of t and the float32 frequency.

AttNHP encoder (App. D.4, with cfg.encoder == "attnhp"): the temporal
encoding uses wavelengths between m and 5M, z_j(t) = sin(t / (m (5M/m)^{j/D}))
for even j and cos(t / (m (5M/m)^{(j-1)/D})) for odd j (the printed second
sine read as a cosine: the pair (j-1, j) would repeat a dimension otherwise);
h^(0) is the type embedding; each layer forms q, k, v = W [z(t); h] + b (the
constant 1 of [1; z; h] is the bias) and updates
h += tanh(sum_j f_ij v_j / (1 + sum_j f_ij)), f_ij = exp(q_i . k_j / sqrt(d_head))
over j <= i, per head, heads concatenated; no LayerNorm, feed-forward block
or output projection, and the decoder reads h^(L).

bf16 mode emulates the rounding points of a bf16 implementation: every
Linear input (LN outputs, attention output, ReLU output, the decoder's e and
tanh activations) and q, k, v are rounded to bf16; the residual stream,
statistics, softmax and all decoder arithmetic stay in float64.
"""
from __future__ import annotations

import math
from typing import Dict

import numpy as np

from .numerics import log_softmax, round_bf16

LN_EPS = 1e-5


def _ident(x):
    return x


class Model:
    """Weights + configuration of one CDF-based Transformer TPP."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray]):
        self.cfg = cfg
        self.L = cfg.n_layers
        self.d = cfg.d_model
        self.H = cfg.n_heads
        self.dh = cfg.d_model // cfg.n_heads
        self.F = cfg.d_ffn
        self.M = cfg.n_mix
        self.K = cfg.n_types
        self.w = {k: np.asarray(v, dtype=np.float64) for k, v in weights.items()}
        self.rb = round_bf16 if cfg.prec == "bf16" else _ident
        self.attnhp = getattr(cfg, "encoder", "thp") == "attnhp"

    # ---- encoder pieces -------------------------------------------------
    def frequencies(self) -> np.ndarray:
        """Float32 frequency table (App. D.4): THP 10000^(-(j - j mod 2)/D);
        AttNHP 1 / (m (5M/m)^((j - j mod 2)/D)), j = 0..D-1."""
        j = np.arange(self.d)
        if self.attnhp:
            m, M = float(self.cfg.time_m), float(self.cfg.time_M)
            return (1.0 / (m * np.power(5.0 * M / m, (j - j % 2) / self.d))).astype(np.float32)
        return np.power(10000.0, -(j - j % 2) / self.d).astype(np.float32)

    def time_encoding(self, t) -> np.ndarray:
        """z(t) for float32 times t[...] -> [..., D] float64."""
        t32 = np.asarray(t, dtype=np.float32)
        arg = (t32[..., None] * self.frequencies()).astype(np.float64)   # float32 product
        j = np.arange(self.d)
        return np.where(j % 2 == 0, np.sin(arg), np.cos(arg))

    def embed(self, t, k) -> np.ndarray:
        """X = z(t) + W^T onehot(k)  (§4.2 Encoder, summation fusion); for AttNHP
        h^(0) = W^T onehot(k), the time entering every layer through [z(t); h]."""
        if self.attnhp:
            return self.w["type_emb"][np.asarray(k)].copy()
        return self.time_encoding(t) + self.w["type_emb"][np.asarray(k)]

    def _attnhp_layer(self, l, x, z, kc_fn, mask):
        """One AttNHP layer: q, k, v from [z; h] (bias = the constant input), per
        head sum_j f v / (1 + sum_j f), h += tanh(.). kc_fn(k, v) returns the keys
        and values attended over (the new ones, or the cache holding them)."""
        rb = self.rb
        p = f"layers.{l}."
        u = np.concatenate([rb(z), rb(x)], axis=-1)
        qkv = rb(self._lin(u, p + "qkv"))
        q, kk, v = (self._split_heads(qkv[..., i * self.d:(i + 1) * self.d]) for i in range(3))
        Kc, Vc = kc_fn(kk, v)
        s = q @ np.swapaxes(Kc, -1, -2) / math.sqrt(self.dh)
        s = np.where(mask, s, -np.inf)
        smax = np.maximum(s.max(axis=-1, keepdims=True), 0.0)   # the 1 of the denominator is exp(0)
        pr = np.exp(s - smax)
        o = (pr @ Vc) / (np.exp(-smax) + pr.sum(axis=-1, keepdims=True))
        return x + np.tanh(rb(self._merge_heads(o)))

    @staticmethod
    def layer_norm(x, g, b):
        mu = x.mean(axis=-1, keepdims=True)
        var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
        return (x - mu) / np.sqrt(var + LN_EPS) * g + b

    def _lin(self, x, name):
        y = x @ self.w[name + ".w"].T
        bn = name + ".b"
        return y + self.w[bn] if bn in self.w else y

    def _split_heads(self, y):
        """[..., P, d] -> [..., H, P, dh]."""
        sh = y.shape[:-1] + (self.H, self.dh)
        return np.moveaxis(y.reshape(sh), -2, -3)

    def _merge_heads(self, y):
        """[..., H, P, dh] -> [..., P, d]."""
        y = np.moveaxis(y, -3, -2)
        return y.reshape(y.shape[:-2] + (self.d,))

    # ---- full (cache-free) forward --------------------------------------
    def forward_full(self, t, k) -> np.ndarray:
        """History embeddings for every event of t[B, N], k[B, N]; returns LN_f(x) [B, N, D].

        Position i attends to positions 0..i (the event itself and its past).
        """
        rb = self.rb
        x = self.embed(t, k)
        N = x.shape[-2]
        causal = np.tril(np.ones((N, N), dtype=bool))
        if self.attnhp:
            z = self.time_encoding(t)
            for l in range(self.L):
                x = self._attnhp_layer(l, x, z, lambda kk, v: (kk, v), causal)
            return x
        for l in range(self.L):
            p = f"layers.{l}."
            a = rb(self.layer_norm(x, self.w[p + "ln1.g"], self.w[p + "ln1.b"]))
            qkv = rb(self._lin(a, p + "qkv"))
            q, kk, v = (self._split_heads(qkv[..., i * self.d:(i + 1) * self.d]) for i in range(3))
            s = q @ np.swapaxes(kk, -1, -2) / math.sqrt(self.dh)
            s = np.where(causal, s, -np.inf)
            s = s - s.max(axis=-1, keepdims=True)
            pr = np.exp(s)
            pr = pr / pr.sum(axis=-1, keepdims=True)
            o = rb(self._merge_heads(pr @ v))
            x = x + self._lin(o, p + "out")
            a2 = rb(self.layer_norm(x, self.w[p + "ln2.g"], self.w[p + "ln2.b"]))
            hid = rb(np.maximum(self._lin(a2, p + "ffn1"), 0.0))
            x = x + self._lin(hid, p + "ffn2")
        return self.layer_norm(x, self.w["lnf.g"], self.w["lnf.b"])

    # ---- cached block forward --------------------------------------------
    def new_cache(self, B: int, cap: int) -> "KVCache":
        return KVCache(self.L, B, self.H, cap, self.dh)

    def forward_block(self, cache: "KVCache", t, k, pos0, rows=None) -> np.ndarray:
        """P new events per sequence on top of cached keys/values.

        t, k: [B, P]; pos0[b] = number of events of sequence b already cached;
        rows (optional) = the cache rows these B sequences occupy.
        Keys/values of the new events are stored at pos0[b] .. pos0[b] + P - 1,
        and query p of sequence b attends to cached positions 0 .. pos0[b] + p.
        Returns LN_f(x) for the new events, [B, P, D].
        """
        rb = self.rb
        t = np.asarray(t)
        B, P = t.shape
        pos0 = np.asarray(pos0, dtype=np.int64)
        x = self.embed(t, k)
        n_keys = int(pos0.max()) + P
        pos = pos0[:, None] + np.arange(P)[None, :]                  # [B, P]
        rows = np.arange(B) if rows is None else np.asarray(rows, dtype=np.int64)
        bidx = rows[:, None]
        keymask = np.arange(n_keys)[None, None, :] <= pos[:, :, None]  # [B, P, n_keys]
        if self.attnhp:
            z = self.time_encoding(t)
            for l in range(self.L):
                def kc_fn(kk, v, l=l):
                    cache.K[l][bidx, :, pos, :] = np.moveaxis(kk, 1, 2)
                    cache.V[l][bidx, :, pos, :] = np.moveaxis(v, 1, 2)
                    return cache.K[l][rows, :, :n_keys, :], cache.V[l][rows, :, :n_keys, :]
                x = self._attnhp_layer(l, x, z, kc_fn, keymask[:, None, :, :])
            return x
        for l in range(self.L):
            p = f"layers.{l}."
            a = rb(self.layer_norm(x, self.w[p + "ln1.g"], self.w[p + "ln1.b"]))
            qkv = rb(self._lin(a, p + "qkv"))
            q, kk, v = (self._split_heads(qkv[..., i * self.d:(i + 1) * self.d]) for i in range(3))
            # kk, v: [B, H, P, dh] -> cache[l][b, :, pos[b, p], :]
            cache.K[l][bidx, :, pos, :] = np.moveaxis(kk, 1, 2)
            cache.V[l][bidx, :, pos, :] = np.moveaxis(v, 1, 2)
            Kc = cache.K[l][rows, :, :n_keys, :]
            Vc = cache.V[l][rows, :, :n_keys, :]
            s = q @ np.swapaxes(Kc, -1, -2) / math.sqrt(self.dh)      # [B, H, P, n_keys]
            s = np.where(keymask[:, None, :, :], s, -np.inf)
            s = s - s.max(axis=-1, keepdims=True)
            pr = np.exp(s)
            pr = pr / pr.sum(axis=-1, keepdims=True)
            o = rb(self._merge_heads(pr @ Vc))
            x = x + self._lin(o, p + "out")
            a2 = rb(self.layer_norm(x, self.w[p + "ln2.g"], self.w[p + "ln2.b"]))
            hid = rb(np.maximum(self._lin(a2, p + "ffn1"), 0.0))
            x = x + self._lin(hid, p + "ffn2")
        return self.layer_norm(x, self.w["lnf.g"], self.w["lnf.b"])

    # ---- decoder ----------------------------------------------------------
    def head(self, h):
        """Decoder of §4.2: (log w, mu, s = log sigma, log f) for history embeddings h[..., D]."""
        rb = self.rb
        hb = rb(h)
        e = rb(hb @ self.w["head.E"].T)
        d = self.d
        e1, e2, e3 = e[..., :d], e[..., d:2 * d], e[..., 2 * d:]
        logw = log_softmax(self._lin(e1, "head.w"))
        mu = self._lin(e2, "head.mu")
        s = self._lin(e3, "head.sigma")
        th = rb(np.tanh(self._lin(hb, "head.k1")))
        logf = log_softmax(self._lin(th, "head.k2"))
        return logw, mu, s, logf


class KVCache:
    """Append-only per-layer key/value store, [B, H, cap, d_head] per layer."""

    def __init__(self, L, B, H, cap, dh):
        self.K = [np.zeros((B, H, cap, dh)) for _ in range(L)]
        self.V = [np.zeros((B, H, cap, dh)) for _ in range(L)]
