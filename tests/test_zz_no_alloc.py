"""tppsd_verify_noalloc (the verify pass with its activation scratch in the
library's static device array) against tppsd_verify (scratch in the state's
workspace): the same kernels, so the outputs must be identical, on two calls
in a row -- the second with a smaller input -- for a bf16 and an fp32 target,
and a pass too large for the array must be refused with TPPSD_E_WORKSPACE."""
import numpy as np
import pytest
import torch

from gpu_common import gpu_state, histories, small, to_dev, weights
from oracle import sampler as S
from gpu_common import draft_buffers_from_oracle, oracle_models
from paper_2507_09252_amd import tppsd as tp

pytestmark = pytest.mark.gpu


def _verify_pair(st, case, gamma, dbuf):
    M, K = case.wl.target.n_mix, case.wl.target.n_types
    B = st.B
    ref, got = tp.VerifyBuffers(B, st.max_gamma, M, K), tp.VerifyBuffers(B, st.max_gamma, M, K)
    for t in (got.logg, got.logf, got.mix, got.logtype):
        t.fill_(float("nan"))
    st.tppsd_verify(gamma, dbuf, ref)
    st.tppsd_verify_noalloc(gamma, dbuf, got)
    torch.cuda.synchronize()
    for name in ("logg", "logf", "mix", "logtype"):
        a = getattr(ref, name).cpu().numpy()
        b = getattr(got, name).cpu().numpy()
        if name in ("logg", "logf"):
            a, b = a[:, :gamma], b[:, :gamma]
        else:
            a, b = a[:, :gamma + 1], b[:, :gamma + 1]
        assert np.array_equal(a, b), (case.name, gamma, name, np.nanmax(np.abs(a - b)))
    assert st.tppsd_state_status()["bits"] == 0


@pytest.mark.parametrize("case", [small("c3", 6, n_hist=40, init="bias"), small("c2", 5, init="bias")],
                         ids=["c3-B6", "c2-B5"])
def test_noalloc_verify_matches_verify(case):
    gamma, n_gen, seed = case.g, 32, 7
    wt, wd = weights(case)
    T, D = oracle_models(case, wt, wd)
    ht, hk = histories(case)
    M, K = case.wl.target.n_mix, case.wl.target.n_types
    print(f"{case.name}: gamma {gamma}, then {gamma // 2}", flush=True)
    st = gpu_state(case, wt, wd, gamma, n_gen, seed)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), n_gen)
    dr = S.draft(D, S.prefill(T, D, ht, hk, n_gen), gamma, seed, np.arange(case.B))
    dbuf = draft_buffers_from_oracle(dr, case.B, gamma, M, K)
    _verify_pair(st, case, gamma, dbuf)
    # second call, smaller input: fewer positions per sequence
    _verify_pair(st, case, gamma // 2, dbuf)
    # and a state with fewer sequences (the array keeps the last call's contents)
    small_case = small(case.wl.name, 2, n_hist=case.n_hist, init=case.init)
    st2 = gpu_state(small_case, wt, wd, gamma, n_gen, seed)
    st2.tppsd_prefill(to_dev(ht[:2]), to_dev(hk[:2]), n_gen)
    dbuf2 = draft_buffers_from_oracle(S.DraftOut(**{f: getattr(dr, f)[:2] for f in dr.__dataclass_fields__
                                                    if f != "rate"}), 2, gamma, M, K)
    _verify_pair(st2, small_case, gamma, dbuf2)


def test_noalloc_refuses_an_oversized_pass():
    # 4096 sequences x 33 positions of a d = 128 / F = 512 target need more than the array holds
    case = small("c5", 4096, init="bias")
    wt, wd = weights(case)
    gamma = 32
    st = gpu_state(case, wt, wd, gamma, 8, 3, max_gamma=gamma)
    ht, hk = histories(case)
    st.tppsd_prefill(to_dev(ht), to_dev(hk), 8)
    M, K = case.wl.target.n_mix, case.wl.target.n_types
    dbuf, vbuf = tp.DraftBuffers(case.B, gamma, M, K), tp.VerifyBuffers(case.B, gamma, M, K)
    st.tppsd_draft(gamma, dbuf)
    with pytest.raises(tp.TppsdError, match="E_WORKSPACE"):
        st.tppsd_verify_noalloc(gamma, dbuf, vbuf)
