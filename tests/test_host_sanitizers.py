"""The C-ABI library with its host code built under AddressSanitizer and
UndefinedBehaviorSanitizer (no GPU needed): the host-side paths -- every
workload's weight layout, configuration and argument validation, model and
state sizing, error reporting -- run without a sanitizer report."""
import os
import subprocess
import sys
import textwrap

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHECKS = textwrap.dedent("""
    import ctypes, sys
    sys.path.insert(0, sys.argv[2])
    from paper_2507_09252_amd import tppsd as tp
    from paper_2507_09252_amd import workloads as W
    tp.LIB_PATH = sys.argv[1]
    L = tp.lib()
    for wl in W.WORKLOADS.values():
        for cfg in (wl.target, wl.draft):
            layout = tp.weights_layout(cfg)
            assert layout and tp.tppsd_weights_bytes(cfg) > 0
    bad = [W.ModelCfg(2, 48, 4, 64, 4, 1, "fp32"), W.ModelCfg(2, 64, 4, 48, 4, 1, "bf16"),
           W.ModelCfg(2, 64, 4, 64, 65, 1, "fp32"), W.ModelCfg(0, 64, 4, 64, 4, 1, "fp32"),
           W.ModelCfg(2, 64, 4, 0, 4, 1, "fp32"),
           W.ModelCfg(2, 64, 4, 0, 4, 1, "fp32", W.ENC_ATTNHP, 0.0, 10.0)]
    for cfg in bad:
        try:
            tp.tppsd_weights_bytes(cfg)
            raise SystemExit("a bad configuration was accepted")
        except tp.TppsdError as e:
            assert e.code == 2 and len(L.tppsd_last_error()) > 0
    for name in ("c3", "c4", "c5", "a3"):
        wl = W.WORKLOADS[name]
        hT, hD = ctypes.c_void_p(), ctypes.c_void_p()
        fake = ctypes.c_void_p(1 << 20)   # aligned address: model creation only records offsets
        assert L.tppsd_model_create(ctypes.byref(tp.cfg_c(wl.target)), fake, ctypes.byref(hT)) == 0
        assert L.tppsd_model_create(ctypes.byref(tp.cfg_c(wl.draft)), fake, ctypes.byref(hD)) == 0
        n = ctypes.c_size_t()
        cap = wl.n_hist + wl.n_gen + 33
        assert L.tppsd_state_bytes(hT, hD, wl.batch, cap, 32, ctypes.byref(n)) == 0 and n.value > 0
        assert L.tppsd_state_bytes(hT, None, wl.batch, cap, 32, ctypes.byref(n)) == 0
        assert L.tppsd_state_bytes(hT, hD, 0, cap, 20, ctypes.byref(n)) == 1
        assert L.tppsd_state_bytes(hT, hD, 4, cap, 33, ctypes.byref(n)) == 1
        assert L.tppsd_model_create(ctypes.byref(tp.cfg_c(wl.target)), ctypes.c_void_p(1 << 20 | 8),
                                    ctypes.byref(ctypes.c_void_p())) == 1
        st = ctypes.c_void_p()
        ws = ctypes.c_void_p(1 << 30)
        assert L.tppsd_state_create(hT, hD, 4, cap, 20, 0, 0, ws, 16, ctypes.byref(st)) == 3
        assert L.tppsd_state_create(hT, hD, 4, cap, 20, 0, 8, ws, 1 << 40, ctypes.byref(st)) == 1
        L.tppsd_model_destroy(hT)
        L.tppsd_model_destroy(hD)
    assert L.tppsd_draft(None, 4, None, None) == 1
    assert L.tppsd_verify(None, 4, None, None, None) == 1
    assert L.tppsd_accept(None, 4, None, None, None, None, None) == 1
    assert L.tppsd_sample_sd(None, 4, 1, None, None) == 1
    assert L.tppsd_timing_enable(None, 1) == 1
    print("sanitized host checks passed")
""")


def test_host_library_under_sanitizers(tmp_path):
    from paper_2507_09252_amd import build as B
    lib = B.build_host_sanitized(str(tmp_path))
    env = dict(os.environ, LD_PRELOAD=B.sanitizer_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-c", CHECKS, lib, ROOT], env=env, capture_output=True, text=True,
                       timeout=900)
    assert r.returncode == 0 and "sanitized host checks passed" in r.stdout, (r.stdout[-2000:], r.stderr[-6000:])
