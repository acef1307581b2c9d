"""Python binding of libtppsd (the C ABI declared in include/tppsd.h).

Argument marshalling only: every step of the sampler runs in the HIP library.
torch provides device memory and the stream (its current HIP stream); torch
must be imported before the library is loaded so both use the same HIP
runtime. If the library has not been built, loading fails loudly: there is no
fallback.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_int, c_int32, c_int64, c_size_t, c_uint, c_uint32, c_uint64, c_void_p
from typing import Dict, Optional

import numpy as np
import torch  # noqa: F401  (loads torch's HIP runtime first)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtppsd.so")

TPPSD_OK = 0
PREC = {"fp32": 0, "bf16": 1}
FLAG_BONUS = 1
STATUS_CAPACITY, STATUS_NONFINITE, STATUS_AR_CAP = 1, 2, 4

ERRORS = {1: "TPPSD_E_ARG", 2: "TPPSD_E_CONFIG", 3: "TPPSD_E_WORKSPACE", 4: "TPPSD_E_ORDER", 5: "TPPSD_E_HIP"}

# every symbol the header declares
EXPORTS = [
    "tppsd_weights_bytes", "tppsd_weights_entry", "tppsd_model_create", "tppsd_model_destroy",
    "tppsd_state_bytes", "tppsd_state_create", "tppsd_state_destroy", "tppsd_prefill", "tppsd_draft",
    "tppsd_verify", "tppsd_accept", "tppsd_sample_ar", "tppsd_sample_sd", "tppsd_read_events",
    "tppsd_state_status", "tppsd_timing_enable", "tppsd_timing_read", "tppsd_last_error",
    "tppsd_poisson_fit", "tppsd_draft_poisson", "tppsd_sample_sd_poisson", "tppsd_prefill_window",
    "tppsd_read_loglik", "tppsd_verify_noalloc",
]


class TppsdError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


TIME_KERNELS = 1   # TPPSD_TIME_KERNELS
TIME_PHASES = 2    # TPPSD_TIME_PHASES


class TimingC(ctypes.Structure):
    _fields_ = [("attn_ms", c_double), ("attn_launches", c_int64), ("gemm_ms", c_double),
                ("gemm_launches", c_int64), ("gemm_flop", c_double), ("draft_ms", c_double),
                ("verify_ms", c_double), ("accept_ms", c_double), ("rounds", c_int64),
                ("draft_kernel_ms", c_double), ("draft_kernel_launches", c_int64),
                ("draft_attn_ms", c_double), ("draft_attn_launches", c_int64),
                ("draft_rows_ms", c_double), ("draft_rows_launches", c_int64)]


ENCODER = {"thp": 0, "attnhp": 1}   # TPPSD_ENC_*


class ModelCfgC(ctypes.Structure):
    _fields_ = [(n, c_int32) for n in ("n_layers", "d_model", "n_heads", "d_ffn", "n_mix", "n_types", "prec",
                                       "encoder")] + [("time_m", ctypes.c_float), ("time_M", ctypes.c_float)]


class DraftBufC(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("tau", "t", "k", "logg", "logf", "mix", "logtype", "rate")]


class VerifyBufC(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("logg", "logf", "mix", "logtype")]


class AcceptBufC(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("L", "n_new", "k_new", "t_new", "tau_new", "ar_iter", "flags")]


_lib = None


def lib():
    """Load libtppsd.so (built in-tree); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                           "(python paper_2507_09252_amd/build.py)")
    L = ctypes.CDLL(LIB_PATH)
    P = POINTER
    sig = {
        "tppsd_weights_bytes": (c_int, [P(ModelCfgC), P(c_size_t)]),
        "tppsd_weights_entry": (c_int, [P(ModelCfgC), c_int, P(c_char_p), P(c_size_t), P(c_int64), P(c_int64), P(c_int)]),
        "tppsd_model_create": (c_int, [P(ModelCfgC), c_void_p, P(c_void_p)]),
        "tppsd_model_destroy": (None, [c_void_p]),
        "tppsd_state_bytes": (c_int, [c_void_p, c_void_p, c_int, c_int, c_int, P(c_size_t)]),
        "tppsd_state_create": (c_int, [c_void_p, c_void_p, c_int, c_int, c_int, c_uint64, c_uint, c_void_p,
                                       c_size_t, P(c_void_p)]),
        "tppsd_state_destroy": (None, [c_void_p]),
        "tppsd_prefill": (c_int, [c_void_p, c_void_p, c_void_p, c_int, c_int, c_void_p]),
        "tppsd_draft": (c_int, [c_void_p, c_int, P(DraftBufC), c_void_p]),
        "tppsd_verify": (c_int, [c_void_p, c_int, P(DraftBufC), P(VerifyBufC), c_void_p]),
        "tppsd_verify_noalloc": (c_int, [c_void_p, c_int, P(DraftBufC), P(VerifyBufC), c_void_p]),
        "tppsd_accept": (c_int, [c_void_p, c_int, P(DraftBufC), P(VerifyBufC), c_void_p, P(AcceptBufC), c_void_p]),
        "tppsd_sample_ar": (c_int, [c_void_p, c_int, c_void_p, c_void_p, c_void_p]),
        "tppsd_sample_sd": (c_int, [c_void_p, c_int, c_int, P(c_int), c_void_p]),
        "tppsd_read_events": (c_int, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]),
        "tppsd_state_status": (c_int, [c_void_p, c_void_p, P(c_uint32), P(c_int32), P(c_int64), P(c_int64), P(c_int64)]),
        "tppsd_timing_enable": (c_int, [c_void_p, c_int]),
        "tppsd_timing_read": (c_int, [c_void_p, P(TimingC)]),
        "tppsd_last_error": (c_char_p, []),
        "tppsd_poisson_fit": (c_int, [c_void_p, c_void_p, c_int, c_int, c_int, c_void_p, c_void_p]),
        "tppsd_draft_poisson": (c_int, [c_void_p, c_int, c_void_p, P(DraftBufC), c_void_p]),
        "tppsd_sample_sd_poisson": (c_int, [c_void_p, c_int, c_void_p, c_int, P(c_int), c_void_p]),
        "tppsd_prefill_window": (c_int, [c_void_p, c_void_p, c_void_p, c_int, c_int, c_void_p, c_void_p]),
        "tppsd_read_loglik": (c_int, [c_void_p, c_void_p, c_void_p]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(rc):
    if rc != TPPSD_OK:
        raise TppsdError(rc, lib().tppsd_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else c_void_p(t.data_ptr())


def _stream():
    return c_void_p(torch.cuda.current_stream().cuda_stream)


def cfg_c(cfg) -> ModelCfgC:
    return ModelCfgC(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.d_ffn, cfg.n_mix, cfg.n_types, PREC[cfg.prec],
                     ENCODER[getattr(cfg, "encoder", "thp")], float(getattr(cfg, "time_m", 1.0)),
                     float(getattr(cfg, "time_M", 100.0)))


# ---------------------------------------------------------------------------
# weights
# ---------------------------------------------------------------------------

def tppsd_weights_bytes(cfg) -> int:
    n = c_size_t()
    _check(lib().tppsd_weights_bytes(ctypes.byref(cfg_c(cfg)), ctypes.byref(n)))
    return n.value


def weights_layout(cfg):
    """[(name, offset, rows, cols, is_bf16)] of the packed layout, from the library."""
    out, i = [], 0
    c = cfg_c(cfg)
    L = lib()
    while True:
        name, off, r, cl, bf = c_char_p(), c_size_t(), c_int64(), c_int64(), c_int()
        rc = L.tppsd_weights_entry(ctypes.byref(c), i, ctypes.byref(name), ctypes.byref(off), ctypes.byref(r),
                                   ctypes.byref(cl), ctypes.byref(bf))
        if rc != TPPSD_OK:
            break
        out.append((name.value.decode(), off.value, r.value, cl.value, bf.value))
        i += 1
    return out


def pack_weights(cfg, weights: Dict[str, np.ndarray], device="cuda") -> torch.Tensor:
    """Packs named parameters into the library's device layout (a uint8 tensor)."""
    total = tppsd_weights_bytes(cfg)
    buf = torch.zeros(total, dtype=torch.uint8)
    for name, off, r, cl, bf in weights_layout(cfg):
        a = np.asarray(weights[name], dtype=np.float32).reshape(r * cl)
        t = torch.from_numpy(a.copy())
        if bf:
            t = t.to(torch.bfloat16)
        raw = t.view(torch.uint8)
        buf[off:off + raw.numel()] = raw
    return buf.to(device)


class Model:
    """tppsd_model handle over packed device weights (kept alive here)."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray], device="cuda"):
        self.cfg = cfg
        self.wbuf = pack_weights(cfg, weights, device)
        h = c_void_p()
        _check(lib().tppsd_model_create(ctypes.byref(cfg_c(cfg)), _ptr(self.wbuf), ctypes.byref(h)))
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.tppsd_model_destroy(self.handle)
            self.handle = None


def tppsd_poisson_fit(t: torch.Tensor, k: torch.Tensor, K: int) -> torch.Tensor:
    """Homogeneous-Poisson draft parameters [1 + K] (rate, log p) fitted on the
    device from sequences t/k [B, n0]."""
    t = t.to(torch.float32).contiguous()
    k = k.to(torch.int32).contiguous()
    params = torch.empty(1 + K, dtype=torch.float32, device=t.device)
    _check(lib().tppsd_poisson_fit(_ptr(t), _ptr(k), t.shape[0], t.shape[1], K, _ptr(params), _stream()))
    return params


# ---------------------------------------------------------------------------
# round buffers
# ---------------------------------------------------------------------------

class DraftBuffers:
    """Draft record; poisson=True makes the record of a homogeneous-Poisson
    draft (a rate array, no mixture)."""

    def __init__(self, B, max_gamma, M, K, device="cuda", poisson=False):
        f = dict(dtype=torch.float32, device=device)
        self.tau = torch.zeros(B, max_gamma, **f)
        self.t = torch.zeros(B, max_gamma, **f)
        self.k = torch.zeros(B, max_gamma, dtype=torch.int32, device=device)
        self.logg = torch.zeros(B, max_gamma, **f)
        self.logf = torch.zeros(B, max_gamma, **f)
        self.mix = None if poisson else torch.zeros(B, max_gamma, 3, M, **f)
        self.logtype = torch.zeros(B, max_gamma, K, **f)
        self.rate = torch.zeros(B, **f) if poisson else None

    def c(self):
        return DraftBufC(*(None if t is None else t.data_ptr()
                           for t in (self.tau, self.t, self.k, self.logg, self.logf, self.mix, self.logtype,
                                     self.rate)))


class VerifyBuffers:
    def __init__(self, B, max_gamma, M, K, device="cuda"):
        f = dict(dtype=torch.float32, device=device)
        self.logg = torch.zeros(B, max_gamma, **f)
        self.logf = torch.zeros(B, max_gamma, **f)
        self.mix = torch.zeros(B, max_gamma + 1, 3, M, **f)
        self.logtype = torch.zeros(B, max_gamma + 1, K, **f)

    def c(self):
        return VerifyBufC(*(t.data_ptr() for t in (self.logg, self.logf, self.mix, self.logtype)))


class AcceptBuffers:
    def __init__(self, B, max_gamma, device="cuda"):
        i = dict(dtype=torch.int32, device=device)
        self.L = torch.zeros(B, **i)
        self.n_new = torch.zeros(B, **i)
        self.k_new = torch.zeros(B, max_gamma + 1, **i)
        self.t_new = torch.zeros(B, max_gamma + 1, dtype=torch.float32, device=device)
        self.tau_new = torch.zeros(B, max_gamma + 1, dtype=torch.float32, device=device)
        self.ar_iter = torch.zeros(B, **i)
        self.flags = torch.zeros(B, dtype=torch.uint8, device=device)

    def c(self):
        return AcceptBufC(*(t.data_ptr() for t in (self.L, self.n_new, self.k_new, self.t_new, self.tau_new,
                                                    self.ar_iter, self.flags)))


# ---------------------------------------------------------------------------
# sampler state
# ---------------------------------------------------------------------------

class State:
    """tppsd_state over a torch-allocated workspace; methods map 1:1 to the C ABI."""

    def __init__(self, target: Model, draft: Optional[Model], B: int, max_events: int, max_gamma: int,
                 seed: int = 0, bonus: bool = True, device="cuda"):
        self.target, self.draft = target, draft
        self.B, self.max_events, self.max_gamma = B, max_events, max_gamma
        n = c_size_t()
        dh = draft.handle if draft is not None else None
        _check(lib().tppsd_state_bytes(target.handle, dh, B, max_events, max_gamma, ctypes.byref(n)))
        self.ws = torch.empty(n.value, dtype=torch.uint8, device=device)
        h = c_void_p()
        _check(lib().tppsd_state_create(target.handle, dh, B, max_events, max_gamma, c_uint64(seed),
                                        FLAG_BONUS if bonus else 0, _ptr(self.ws), n.value, ctypes.byref(h)))
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.tppsd_state_destroy(self.handle)
            self.handle = None

    def tppsd_prefill(self, t: torch.Tensor, k: torch.Tensor, n_gen: int, t_end: Optional[torch.Tensor] = None):
        """t_end [B] (optional): per-sequence end time (tppsd_prefill_window)."""
        t = t.contiguous()
        k = k.to(torch.int32).contiguous()
        self._hist = (t, k)
        if t_end is None:
            _check(lib().tppsd_prefill(self.handle, _ptr(t), _ptr(k), t.shape[1], n_gen, _stream()))
        else:
            t_end = t_end.to(torch.float32).contiguous()
            self._t_end = t_end
            _check(lib().tppsd_prefill_window(self.handle, _ptr(t), _ptr(k), t.shape[1], n_gen, _ptr(t_end),
                                              _stream()))

    def tppsd_draft(self, gamma: int, out: DraftBuffers):
        _check(lib().tppsd_draft(self.handle, gamma, ctypes.byref(out.c()), _stream()))

    def tppsd_draft_poisson(self, gamma: int, params: torch.Tensor, out: DraftBuffers):
        _check(lib().tppsd_draft_poisson(self.handle, gamma, _ptr(params), ctypes.byref(out.c()), _stream()))

    def tppsd_verify(self, gamma: int, drafts: DraftBuffers, out: VerifyBuffers):
        _check(lib().tppsd_verify(self.handle, gamma, ctypes.byref(drafts.c()), ctypes.byref(out.c()), _stream()))

    def tppsd_verify_noalloc(self, gamma: int, drafts: DraftBuffers, out: VerifyBuffers):
        _check(lib().tppsd_verify_noalloc(self.handle, gamma, ctypes.byref(drafts.c()), ctypes.byref(out.c()),
                                          _stream()))

    def tppsd_accept(self, gamma: int, drafts: DraftBuffers, verify: VerifyBuffers, out: AcceptBuffers,
                     uniforms: Optional[torch.Tensor] = None):
        _check(lib().tppsd_accept(self.handle, gamma, ctypes.byref(drafts.c()), ctypes.byref(verify.c()),
                                  _ptr(uniforms), ctypes.byref(out.c()), _stream()))

    def tppsd_sample_ar(self, n_events: int, t_out: Optional[torch.Tensor] = None,
                        k_out: Optional[torch.Tensor] = None):
        _check(lib().tppsd_sample_ar(self.handle, n_events, _ptr(t_out), _ptr(k_out), _stream()))

    def tppsd_sample_sd(self, gamma: int, max_rounds: int = 1 << 30) -> int:
        r = c_int()
        _check(lib().tppsd_sample_sd(self.handle, gamma, max_rounds, ctypes.byref(r), _stream()))
        return r.value

    def tppsd_sample_sd_poisson(self, gamma: int, params: torch.Tensor, max_rounds: int = 1 << 30) -> int:
        r = c_int()
        _check(lib().tppsd_sample_sd_poisson(self.handle, gamma, _ptr(params), max_rounds, ctypes.byref(r),
                                             _stream()))
        return r.value

    def tppsd_read_events(self):
        t = torch.empty(self.B, self.max_events, dtype=torch.float32, device=self.ws.device)
        k = torch.empty(self.B, self.max_events, dtype=torch.int32, device=self.ws.device)
        n = torch.empty(self.B, dtype=torch.int32, device=self.ws.device)
        _check(lib().tppsd_read_events(self.handle, _ptr(t), _ptr(k), _ptr(n), _stream()))
        return t, k, n

    def tppsd_read_loglik(self) -> torch.Tensor:
        ll = torch.empty(self.B, dtype=torch.float64, device=self.ws.device)
        _check(lib().tppsd_read_loglik(self.handle, _ptr(ll), _stream()))
        return ll

    def tppsd_state_status(self):
        bits, nd, acc, dr, ar = c_uint32(), c_int32(), c_int64(), c_int64(), c_int64()
        _check(lib().tppsd_state_status(self.handle, _stream(), ctypes.byref(bits), ctypes.byref(nd),
                                        ctypes.byref(acc), ctypes.byref(dr), ctypes.byref(ar)))
        return dict(bits=bits.value, n_done=nd.value, accepted=acc.value, drafted=dr.value, ar_candidates=ar.value)

    def tppsd_timing_enable(self, modes: int):
        """modes: 0 (off), TIME_KERNELS or TIME_PHASES."""
        _check(lib().tppsd_timing_enable(self.handle, int(modes)))

    def tppsd_timing_read(self):
        t = TimingC()
        _check(lib().tppsd_timing_read(self.handle, ctypes.byref(t)))
        return {name: getattr(t, name) for name, _ in TimingC._fields_}
