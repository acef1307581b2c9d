"""Pins for oracle.numerics: bf16 rounding against torch's conversion."""
import numpy as np
import scipy.special
import torch

from oracle.numerics import log_softmax, logsumexp, round_bf16


def test_round_bf16_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.normal(0, 1, 100000), rng.normal(0, 1e-3, 1000), rng.normal(0, 300, 1000)])
    x = x.astype(np.float32)
    # exact halfway cases: bf16 value +- half an ulp
    base = torch.from_numpy(rng.normal(0, 1, 1000).astype(np.float32)).bfloat16().float().numpy()
    halfway = (base.view(np.uint32) + np.uint32(0x8000)).view(np.float32)
    x = np.concatenate([x, halfway, -halfway, np.zeros(1, np.float32)])
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = round_bf16(x.astype(np.float64))
    assert np.array_equal(got, want)


def test_log_softmax_logsumexp():
    rng = np.random.default_rng(1)
    z = rng.normal(0, 5, (20, 7))
    assert np.allclose(log_softmax(z), scipy.special.log_softmax(z, axis=-1), atol=1e-13)
    assert np.allclose(logsumexp(z), scipy.special.logsumexp(z, axis=-1), atol=1e-13)
