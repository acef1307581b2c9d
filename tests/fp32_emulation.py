"""Float32 emulation of a bf16 implementation, used to derive bf16 tolerances.

bf16 results depend on where float32-vs-float64 accumulation differences flip a
bf16 rounding: an implementation that accumulates in float32 cannot be closer
to the float64 oracle than an exact float32 evaluation of the same arithmetic
with the same rounding points. This class is that evaluation (NumPy float32,
oracle's rounding points); its distance to the oracle, times 2 for summation
order, is the bound used where it exceeds the stated 2e-3.
Test infrastructure only.
"""
import numpy as np

from oracle import numerics as N
from oracle import sampler as S
from oracle.model import Model


class Model32(Model):
    def __init__(self, cfg, weights):
        super().__init__(cfg, weights)
        self.w = {k: v.astype(np.float32) for k, v in self.w.items()}
        self.rb = lambda x: N.round_bf16(np.asarray(x, np.float32).astype(np.float64)).astype(np.float32)

    def embed(self, t, k):
        if self.attnhp:
            return self.w["type_emb"][np.asarray(k)].astype(np.float32)
        return (self.time_encoding(t).astype(np.float32) + self.w["type_emb"][np.asarray(k)]).astype(np.float32)

    @staticmethod
    def layer_norm(x, g, b):
        x = np.asarray(x, np.float32)
        mu = x.mean(-1, keepdims=True, dtype=np.float32)
        var = ((x - mu) ** 2).mean(-1, keepdims=True, dtype=np.float32)
        return ((x - mu) / np.sqrt(var + np.float32(1e-5)) * g + b).astype(np.float32)


def emulated_verify(cfg, weights, hist_t, hist_k, dr: S.DraftOut):
    """Verify outputs (log g, log f at the drafts, decoder rows) of the float32 emulation."""
    m = Model32(cfg, weights)
    t = np.concatenate([hist_t, dr.t.astype(np.float32)], 1)
    k = np.concatenate([hist_k, dr.k], 1)
    g = dr.t.shape[1]
    h = m.forward_full(t, k)[:, -(g + 1):].astype(np.float64)
    logw, mu, s, logf = m.head(h)
    logw, mu, s, logf = (np.asarray(a, np.float64) for a in (logw, mu, s, logf))
    logg = S.mixture_logpdf(logw[:, :g], mu[:, :g], s[:, :g], dr.tau)
    lf = np.take_along_axis(logf[:, :g], dr.k[..., None], -1)[..., 0]
    return logg, lf, np.stack([logw, mu, s], 2), logf
