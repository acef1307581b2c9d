"""C-ABI library: loads, exports every declared symbol, and validates
arguments on the host (no GPU needed for these calls)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2507_09252_amd import tppsd as tp
from paper_2507_09252_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "tppsd.h")).read()
    return sorted(set(re.findall(r"\b(tppsd_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(tp.LIB_PATH):
        pytest.fail("libtppsd.so is not built (run __graft_entry__.build())")
    return tp.lib()


def test_exports_every_declared_symbol(lib):
    declared = _declared()
    assert set(declared) == set(tp.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_weight_layout_covers_parameters(lib, name):
    wl = W.WORKLOADS[name]
    for cfg in (wl.target, wl.draft):
        layout = tp.weights_layout(cfg)
        names = {n for n, *_ in layout}
        assert names == {n for n, _, _ in W.weight_names(cfg)}
        total = tp.tppsd_weights_bytes(cfg)
        ends = []
        for n, off, r, c, bf in layout:
            size = r * c * (2 if bf else 4)
            ends.append((off, off + size))
            assert off + size <= total
            assert bf == (1 if (cfg.prec == "bf16" and c > 1 or (cfg.prec == "bf16" and n == "type_emb")) else 0) \
                or c == 1
        ends.sort()
        assert all(a[1] <= b[0] for a, b in zip(ends, ends[1:]))     # no overlap
        d = cfg.d_model
        off = {n: o for n, o, *_ in layout}
        me = 2 if cfg.prec == "bf16" else 4
        # groups read as one matrix by the kernels
        assert off["head.k1.w"] == off["head.E"] + 3 * d * d * me
        assert off["head.mu.w"] == off["head.w.w"] + cfg.n_mix * d * me
        assert off["head.sigma.b"] == off["head.w.b"] + 2 * cfg.n_mix * 4


def test_config_validation(lib):
    bad = [
        W.ModelCfg(2, 48, 4, 64, 4, 1, "fp32"),        # d_head 12
        W.ModelCfg(2, 64, 4, 48, 4, 1, "bf16"),        # d_ffn not a multiple of 32
        W.ModelCfg(2, 64, 4, 64, 65, 1, "fp32"),       # too many components
        W.ModelCfg(0, 64, 4, 64, 4, 1, "fp32"),
        W.ModelCfg(2, 64, 4, 0, 4, 1, "fp32"),                          # THP without an FFN
        W.ModelCfg(2, 64, 4, 0, 4, 1, "fp32", W.ENC_ATTNHP, 0.0, 10.0),  # AttNHP time scale m = 0
        W.ModelCfg(2, 64, 4, 0, 4, 1, "fp32", W.ENC_ATTNHP, 5.0, 1.0),   # m > M
    ]
    for cfg in bad:
        with pytest.raises(tp.TppsdError) as e:
            tp.tppsd_weights_bytes(cfg)
        assert e.value.code == 2


def test_model_and_state_sizes(lib):
    wl = W.WORKLOADS["c3"]
    hT, hD = ctypes.c_void_p(), ctypes.c_void_p()
    fake = ctypes.c_void_p(1 << 20)        # aligned address; model_create only records offsets
    assert lib.tppsd_model_create(ctypes.byref(tp.cfg_c(wl.target)), fake, ctypes.byref(hT)) == 0
    assert lib.tppsd_model_create(ctypes.byref(tp.cfg_c(wl.draft)), fake, ctypes.byref(hD)) == 0
    n = ctypes.c_size_t()
    cap = wl.n_hist + wl.n_gen + 21
    assert lib.tppsd_state_bytes(hT, hD, wl.batch, cap, 20, ctypes.byref(n)) == 0
    # the KV caches dominate: 2 * layers * B * cap * d * 2 bytes per model
    kv = 2 * (6 * 256 + 2 * 64) * wl.batch * cap * 2
    assert kv < n.value < 2 * kv
    # argument errors
    assert lib.tppsd_state_bytes(hT, hD, 0, cap, 20, ctypes.byref(n)) == 1
    assert lib.tppsd_state_bytes(hT, hD, 4, cap, 33, ctypes.byref(n)) == 1
    assert lib.tppsd_model_create(ctypes.byref(tp.cfg_c(wl.target)), ctypes.c_void_p(1 << 20 | 8),
                                  ctypes.byref(hT)) == 1
    assert b"aligned" in lib.tppsd_last_error()
    ws = ctypes.c_void_p(1 << 30)
    st = ctypes.c_void_p()
    assert lib.tppsd_state_create(hT, hD, 4, cap, 20, 0, 0, ws, 16, ctypes.byref(st)) == 3   # too small
    assert lib.tppsd_state_create(hT, hD, 4, cap, 20, 0, 8, ws, 1 << 40, ctypes.byref(st)) == 1  # bad flag
    assert lib.tppsd_draft(None, 4, None, None) == 1
    lib.tppsd_model_destroy(hT)
    lib.tppsd_model_destroy(hD)


def test_pack_weights_roundtrip(lib):
    wl = W.WORKLOADS["c5"]
    wt, _ = W.workload_weights(wl, init="stress")
    buf = tp.pack_weights(wl.target, wt, device="cpu")
    import torch
    for name, off, r, c, bf in tp.weights_layout(wl.target):
        raw = buf[off:off + r * c * (2 if bf else 4)]
        vals = raw.view(torch.bfloat16 if bf else torch.float32).float().numpy()
        want = wt[name].reshape(-1)
        if bf:
            want = W.to_bf16_values(want)
        assert np.array_equal(vals, want), name
