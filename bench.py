"""Benchmark: accepted events/sec of TPP-SD sampling on one MI355X, vs the GPU
autoregressive sampler, with the round's dominant kernel against its
roofline, the events/s of both samplers as fractions of their rooflines, and
the CPU oracle's rate as a reported baseline.

A step is one generation job over the batch: TPP-SD rounds (draft, verify,
accept, commit) until every sequence has n_gen new events, starting from seed
histories already encoded into both KV caches (the prefill runs untimed
before each step and is reported separately). value = B * n_gen * steps /
(summed step times). The same job with naive AR sampling gives the speedup
denominator.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config c4] [--gamma G]
                    [--gamma-sweep 1,2,5,10,15,20]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "accepted events/sec (1 MI355X) SD vs AR; verify MFMA util %; KV-attn HBM GB/s"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}
ATTN_KERNEL = {"bf16": "k_attn_mfma<d_head, 1, QT> (verify attention)",
               "fp32": "k_attn_mfma_f32<d_head, 1, QT> (verify attention)"}
MAX_CPU_PROCS = 16   # host CPU cores available per GPU


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="c4")
    ap.add_argument("--gamma", type=int, default=None)
    ap.add_argument("--ar-steps", type=int, default=1)
    ap.add_argument("--ar-direct", action="store_true",
                    help="AR job with its steps launched directly (no graphs), for per-dispatch counters")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-poisson", action="store_true", help="skip the homogeneous-Poisson draft run")
    ap.add_argument("--no-window", action="store_true", help="skip the end-time (window) runs")
    ap.add_argument("--no-mismatch", action="store_true", help="skip the mismatched-draft run")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="oracle sample: target CPU seconds")
    ap.add_argument("--cpu-events", type=int, default=64, help="oracle sample: generated events per sequence")
    ap.add_argument("--gamma-sweep", default=None,
                    help="comma-separated draft lengths: the SD job at each, against the same AR job")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# algorithmic work (no kernel structure: what the method must move / compute)
# ---------------------------------------------------------------------------

def _elt(c):
    return 2 if c.prec == "bf16" else 4


def _is_attnhp(c):
    return getattr(c, "encoder", "thp") == "attnhp"


def _layer_matrix_elems(c):
    d, F = c.d_model, c.d_ffn
    return 6 * d * d if _is_attnhp(c) else 4 * d * d + 2 * d * F


def _decoder_elems(c):
    d, M, K = c.d_model, c.n_mix, c.n_types
    return 4 * d * d + (3 * M + K) * d


def model_weight_bytes(c):
    """The model's matrices, read once per pass."""
    return _elt(c) * (c.n_layers * _layer_matrix_elems(c) + _decoder_elems(c))


def pass_roofline(c, B, P, ctx):
    """One forward pass of P new positions per sequence over ctx cached
    positions (d.3): GEMM flops of every layer and the decoder plus QK and PV;
    bytes: the K/V cache read and the append, the weights once, the decoder
    outputs written. Returns (flop, bytes, bound seconds)."""
    T = B * P
    d, L = c.d_model, c.n_layers
    flop = 2.0 * T * (L * _layer_matrix_elems(c) + _decoder_elems(c)) + 4.0 * T * L * d * (ctx + P)
    byt = B * L * (ctx + P) * 2 * d * _elt(c) + model_weight_bytes(c) + T * 4 * (3 * c.n_mix + c.n_types)
    t = max(flop / (MFMA_PEAK_TFLOPS[c.prec] * 1e12), byt / (HBM_PEAK_GBS * 1e9))
    return flop, byt, t


def attention_bytes_per_launch(c, B, P, ctx):
    """Verify attention, one launch (one layer): every cached key and value
    of the run-average context plus the P new ones read once, queries read
    and outputs written."""
    return B * c.n_heads * (ctx + P) * c.d_head * 2 * _elt(c) + 2 * B * P * c.d_model * _elt(c)


def draft_kernel_bytes(wl, B, gamma, ctx):
    """The one-launch draft kernel (one launch per round): gamma draft steps,
    each reading every draft layer's cached keys and values (the context grows
    by one per step), the draft model's weights once, the draft record
    written."""
    c = wl.draft
    kv = sum(B * c.n_layers * (ctx + l) * 2 * c.d_model * _elt(c) for l in range(gamma))
    rec = B * gamma * (5 + 3 * c.n_mix + c.n_types) * 4
    return kv + model_weight_bytes(c) + rec


def draft_attn_bytes(wl, B, gamma, ctx):
    """Row drafting's split attention, one launch (one draft layer, one
    step): the layer's cached keys and values up to the step's position (the
    run-average context plus half a round's drafts), read once; the layer's
    q, k, v matrices; the step's LayerNorm'd rows in; the new keys and values
    appended; and each 384-key split's (max, sum, d_head sums) out. Token rows
    per step average (gamma + 1) / gamma (two in a round's first step)."""
    c = wl.draft
    keys = ctx + gamma / 2.0
    rows = (gamma + 1.0) / gamma
    splits = math.ceil(keys / 384.0)
    e = _elt(c)
    return float(B * c.n_heads * keys * c.d_head * 2 * e + 3 * c.d_model * c.d_model * e
                 + B * rows * c.d_model * e + B * rows * 2 * c.d_model * e
                 + B * c.n_heads * splits * rows * (c.d_head + 2) * 4)


def draft_rows_bytes(wl, B, gamma):
    """Row drafting's row launch, averaged over a round's 1 + L gamma
    launches: the matrices the round's row launches read, each launch's once
    (per step and layer the output projection and FFN; after the last layer
    also the decoder; the step-0 launch only embeds), the residual rows in
    and out, and a non-last layer's FFN output in its four hidden-unit slices
    (fp32, written, then read by the next row launch)."""
    c = wl.draft
    d, F, L = c.d_model, c.d_ffn, c.n_layers
    elems = gamma * (L * (d * d + 2 * d * F) + _decoder_elems(c))
    launches = 1 + L * gamma
    slices = (L - 1) * gamma * 2 * 4 * B * d * 4
    return float((elems * _elt(c) + slices) / launches + 2 * B * 2 * d * 4)


def run_context(wl):
    """Run-average context: contexts grow linearly over a job from n0 to n0 + n_gen."""
    return wl.n_hist + wl.n_gen / 2.0


def verify_gemm_bytes(c, B, gamma):
    """HBM bytes the verify pass's products must move at least: per THP layer
    its attention output in, the residual stream in and out, q, k, v out, the
    layer's matrices once; plus the decoder's first product. AttNHP layer: one
    product over the 2d-wide [z; h] in, q, k, v out."""
    elt, d, L = _elt(c), c.d_model, c.n_layers
    T = B * (gamma + 1)
    if _is_attnhp(c):
        layers = L * (T * 2 * d * elt + 6 * d * d * elt + T * 3 * d * elt)
    else:
        layers = L * (T * d * elt + T * d * 8 + T * 3 * d * elt + (4 * d * d + 2 * d * c.d_ffn) * elt) + T * d * 4
    return float(layers + T * d * 4 + 4 * d * d * elt + T * 4 * d * elt)


# ---------------------------------------------------------------------------
# CPU baseline (the oracle on the host cores); runs before the GPU is touched
# ---------------------------------------------------------------------------

def note(msg):
    """A progress line on stderr (the JSON result is the only stdout line)."""
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def _cpu_model_name():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_job(args):
    """One process's share of the oracle sample (BLAS limited to one thread)."""
    name, seq0, seq1, n_events, gamma = args
    from threadpoolctl import threadpool_limits

    from oracle import sampler as S
    from oracle.model import Model as OModel
    from paper_2507_09252_amd import workloads as W
    wl = W.WORKLOADS[name]
    wt, wd = W.workload_weights(wl)
    ht, hk = W.make_histories(wl)
    with threadpool_limits(1):
        t0 = time.perf_counter()
        st = S.sample_sd(OModel(wl.target, wt), OModel(wl.draft, wd), ht[seq0:seq1], hk[seq0:seq1], n_events,
                         gamma, seed=1234, seq0=seq0)
        dt = time.perf_counter() - t0
    return int(st.gen.sum()), dt


def cpu_baseline(wl, gamma, budget_s, n_events):
    """The float64 oracle on the host: the first n_events generated events of
    min(B, 8 P) sequences, P = the worker processes (one per available core,
    at most MAX_CPU_PROCS), as one process per core over a partition of the
    sequences (reported value) and as one process with one BLAS thread over a
    leading subset sized to about budget_s seconds."""
    import concurrent.futures as cf
    import multiprocessing as mp
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    P = max(1, min(MAX_CPU_PROCS, avail))
    n_events = min(n_events, wl.n_gen)
    n_seq = min(wl.batch, 8 * P)
    # single process: grow the sequence count until a run takes half the budget
    s1 = 1
    while True:
        ev1, dt1 = _oracle_job((wl.name, 0, s1, n_events, gamma))
        note(f"cpu baseline: {s1} sequences in one process, {dt1:.1f} s")
        if dt1 >= 0.5 * budget_s or s1 >= n_seq:
            break
        s1 = int(min(n_seq, max(s1 + 1, s1 * min(4.0, 0.75 * budget_s / max(dt1, 1e-3)))))
    # one process per core, sequences partitioned
    bounds = np.linspace(0, n_seq, P + 1).astype(int)
    jobs = [(wl.name, int(a), int(b), n_events, gamma) for a, b in zip(bounds[:-1], bounds[1:]) if b > a]
    # fresh interpreters (spawn): a fork would inherit the BLAS thread pool the
    # single-process leg left in this process
    t0 = time.perf_counter()
    with cf.ProcessPoolExecutor(len(jobs), mp_context=mp.get_context("spawn")) as ex:
        parts = list(ex.map(_oracle_job, jobs))
    dtp = time.perf_counter() - t0
    evp = sum(p[0] for p in parts)
    note(f"cpu baseline: {n_seq} sequences in {len(jobs)} processes, {dtp:.1f} s")
    return {"value": evp / dtp, "unit": "events/s", "cores": len(jobs), "kind": "oracle",
            "sample": f"first {n_events} generated events of {n_seq} sequences of {wl.name} (TPP-SD, gamma={gamma}), "
                      f"float64 NumPy, one process per core over a partition of the sequences, {dtp:.1f} s wall",
            "cpu_model": _cpu_model_name(), "cores_available": avail,
            "single_process": {"value": ev1 / dt1, "sequences": s1, "seconds": dt1, "blas_threads": 1}}


# ---------------------------------------------------------------------------
# GPU jobs
# ---------------------------------------------------------------------------

def timed_jobs(st, HT, HK, n_gen, steps, run, t_end=None):
    """steps jobs; each: prefill (untimed, synchronised), then the generation
    job bracketed by device synchronisation. Returns (generation seconds,
    prefill seconds, result of the last run)."""
    import torch
    gen_s = pre_s = 0.0
    out = None
    for _ in range(steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st.tppsd_prefill(HT, HK, n_gen, t_end=t_end)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        out = run()
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        pre_s += t1 - t0
        gen_s += t2 - t1
    return gen_s, pre_s, out


def sd_phases(st, tp, HT, HK, n_gen, gamma, mode):
    """One SD job with the library's measurement mode on; returns its timing record."""
    st.tppsd_prefill(HT, HK, n_gen)
    st.tppsd_timing_enable(mode)
    st.tppsd_sample_sd(gamma)
    t = st.tppsd_timing_read()
    st.tppsd_timing_enable(0)
    return t


def gamma_sweep(args, wl, tm, dm, HT, HK, ar_value, B, n_gen):
    """The SD job at each draft length of the sweep (one state per length,
    one warmup job, args.steps timed jobs), against the AR job's rate."""
    from paper_2507_09252_amd import tppsd as tp
    rows = []
    for g in [int(x) for x in args.gamma_sweep.split(",") if x.strip()]:
        st = tp.State(tm, dm, B, wl.n_hist + n_gen + g + 1, g, seed=1234)
        timed_jobs(st, HT, HK, n_gen, 1, lambda: st.tppsd_sample_sd(g))
        dt, _, _ = timed_jobs(st, HT, HK, n_gen, args.steps, lambda: st.tppsd_sample_sd(g))
        s = st.tppsd_state_status()
        assert s["bits"] == 0 and s["n_done"] == B, s
        ph = sd_phases(st, tp, HT, HK, n_gen, g, tp.TIME_PHASES)
        nr = max(1, ph["rounds"])
        value = B * n_gen * args.steps / dt
        rows.append({"gamma": g, "value": value, "speedup_vs_gpu_ar": value / ar_value if ar_value else None,
                     "alpha": s["accepted"] / max(1, s["drafted"]),
                     "round_us": {"draft": ph["draft_ms"] * 1e3 / nr, "verify": ph["verify_ms"] * 1e3 / nr,
                                  "accept": ph["accept_ms"] * 1e3 / nr}})
        note(f"gamma {g}: {value:.4g} events/s, alpha {rows[-1]['alpha']:.3f}")
        del st
    return rows


# the sources each kernel class's measured traffic depends on
TRAFFIC_SOURCES = {
    "verify_attention": ("tppsd_attention.hip", "tppsd_attention.h", "tppsd_device.h"),
    "draft_attention": ("tppsd_draft_rows.hip", "tppsd_internal.h", "tppsd_device.h"),
    "draft_rows": ("tppsd_draft_rows.hip", "tppsd_internal.h", "tppsd_device.h"),
    "ar_attention": ("tppsd_attention.hip", "tppsd_attention.h", "tppsd_device.h"),
}


def source_sha256(files):
    """SHA-256 over the given kernel sources (paper_2507_09252_amd/csrc)."""
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2507_09252_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(cls, wl_name):
    """HBM bytes per launch of a kernel class from the committed rocprofv3
    --pmc runs (FETCH_SIZE and WRITE_SIZE scaled by a copy of known size), if
    the class's sources are unchanged since they were taken; else None."""
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "hbm_traffic.json")))
    except OSError:
        return None
    k = rec["kernels"].get(cls)
    if k is None or source_sha256(TRAFFIC_SOURCES[cls]) != k["sources_sha256"]:
        return None
    w = k["workloads"].get(wl_name)
    return None if w is None else w["traffic_bytes_per_launch"]


def window_jobs(args, wl, gamma, sd, ar, HT, HK, ht, n_gen, B):
    """TPP-SD and AR with an end time per sequence (Algorithm 1's T): each
    sequence's window is 0.75 n_gen of its history's mean interval after its
    pending event, n_gen stays the cap. Reports generated events per second,
    how the sequences ended, and the model log-likelihood (Eq. (2)) both
    samplers accumulate: its batch means and their difference."""
    import torch
    mean_iv = (ht[:, -1] - ht[:, 0]) / (ht.shape[1] - 1)
    t_end = torch.from_numpy((ht[:, -1] + 0.75 * n_gen * mean_iv).astype(np.float32)).to(HT.device)
    res = {}
    for name, st, steps in (("sd", sd, args.steps), ("ar", ar, max(1, args.ar_steps))):
        run = (lambda: st.tppsd_sample_sd(gamma)) if name == "sd" else (lambda: st.tppsd_sample_ar(n_gen))
        timed_jobs(st, HT, HK, n_gen, 1, run, t_end=t_end)
        dt, _, _ = timed_jobs(st, HT, HK, n_gen, steps, run, t_end=t_end)
        dt /= steps
        s = st.tppsd_state_status()
        assert s["bits"] == 0 and s["n_done"] == B, s
        _, _, n = st.tppsd_read_events()
        ll = st.tppsd_read_loglik().cpu().numpy()
        gen = n.cpu().numpy() - wl.n_hist
        res[name] = {"events_per_s": float(gen.sum()) / dt, "mean_events": float(gen.mean()),
                     "ended_by_time": float(np.mean(gen < n_gen)), "loglik_mean": float(ll.mean()),
                     "loglik_per_event": float(ll.sum() / max(1, gen.sum()))}
    res["speedup_vs_gpu_ar"] = res["sd"]["events_per_s"] / res["ar"]["events_per_s"]
    res["delta_L"] = abs(res["sd"]["loglik_mean"] - res["ar"]["loglik_mean"])
    res["window"] = "0.75 n_gen mean history intervals after the pending event"
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the batch shards across GPUs with no exchange: one process per GPU over its own sequences)",
              file=sys.stderr)
        sys.exit(2)
    from paper_2507_09252_amd import workloads as W
    wl = W.WORKLOADS[args.config]
    gamma = args.gamma or wl.gamma
    B, n_gen = wl.batch, wl.n_gen
    # the oracle leg first, before anything initialises the GPU
    cpu = None if args.no_cpu_baseline else cpu_baseline(wl, gamma, args.cpu_seconds, args.cpu_events)

    import torch

    from paper_2507_09252_amd import tppsd as tp

    wt, wd = W.workload_weights(wl)
    ht, hk = W.make_histories(wl)
    dev = torch.device("cuda:0")
    tm, dm = tp.Model(wl.target, wt, dev), tp.Model(wl.draft, wd, dev)
    cap = wl.n_hist + n_gen + gamma + 1
    sd = tp.State(tm, dm, B, cap, gamma, seed=1234)
    ar = tp.State(tm, None, B, cap, gamma, seed=1234)
    HT, HK = torch.from_numpy(ht).to(dev), torch.from_numpy(hk).to(dev)
    sd_run = lambda: sd.tppsd_sample_sd(gamma)
    ar_run = lambda: ar.tppsd_sample_ar(n_gen)

    note(f"{wl.name}: models and states ready")
    if args.warmup > 0:
        timed_jobs(sd, HT, HK, n_gen, args.warmup, sd_run)
        if args.ar_steps > 0:
            timed_jobs(ar, HT, HK, n_gen, 1, ar_run)
    # timed SD jobs: every round replays one captured HIP graph
    rounds = 0
    t_sd = t_pre = 0.0
    for _ in range(args.steps):
        g, p, r = timed_jobs(sd, HT, HK, n_gen, 1, sd_run)
        t_sd, t_pre, rounds = t_sd + g, t_pre + p, rounds + r
    st = sd.tppsd_state_status()
    assert st["bits"] == 0 and st["n_done"] == B, st
    note(f"SD: {args.steps} timed jobs, {t_sd:.2f} s")
    # instrumented jobs (same kernels and data): single kernels bracketed by
    # HIP events (rounds launched directly), then events between the draft /
    # verify / accept graphs of each round
    tk = sd_phases(sd, tp, HT, HK, n_gen, gamma, tp.TIME_KERNELS)
    tph = sd_phases(sd, tp, HT, HK, n_gen, gamma, tp.TIME_PHASES)
    torch.cuda.synchronize()
    note("SD: kernel and phase timing jobs done")

    events = B * n_gen
    ar_value = None
    if args.ar_steps > 0:
        if args.ar_direct:
            ar.tppsd_timing_enable(tp.TIME_KERNELS)
        t_ar, _, _ = timed_jobs(ar, HT, HK, n_gen, args.ar_steps, ar_run)
        if args.ar_direct:
            ar.tppsd_timing_enable(0)
        sa = ar.tppsd_state_status()
        assert sa["bits"] == 0 and sa["n_done"] == B, sa
        ar_value = events * args.ar_steps / t_ar
        note(f"AR: {args.ar_steps} timed jobs, {t_ar:.2f} s")
    value = events * args.steps / t_sd
    alpha = st["accepted"] / max(1, st["drafted"])
    c = wl.target
    ctx = run_context(wl)
    P = gamma + 1
    nr_k = max(1, tk["rounds"])

    # --- the round's kernels as timed live: per-round time of each timed class
    classes = {}
    per_attn = attention_bytes_per_launch(c, B, P, ctx)
    if tk["attn_launches"]:
        classes["verify_attention"] = {
            "bound": "hbm", "kernel": ATTN_KERNEL[wl.prec], "ms": tk["attn_ms"], "launches": tk["attn_launches"],
            "per_launch": per_attn, "unit": "GB/s", "peak": HBM_PEAK_GBS,
            "traffic": measured_traffic("verify_attention", wl.name)}
    if tk["draft_attn_launches"]:
        classes["draft_attention"] = {
            "bound": "hbm", "kernel": "k_rd_attn<128, 32> (row drafting: split attention, one launch per step and layer)",
            "ms": tk["draft_attn_ms"], "launches": tk["draft_attn_launches"],
            "per_launch": draft_attn_bytes(wl, B, gamma, ctx), "unit": "GB/s", "peak": HBM_PEAK_GBS,
            "traffic": measured_traffic("draft_attention", wl.name)}
    if tk["draft_rows_launches"]:
        classes["draft_rows"] = {
            "bound": "hbm", "kernel": "k_rd_rows<128, 512, 32, split> (row drafting, per step and layer: four workgroups "
                                      "per sequence for a non-last layer, one for the last)",
            "ms": tk["draft_rows_ms"], "launches": tk["draft_rows_launches"],
            "per_launch": draft_rows_bytes(wl, B, gamma), "unit": "GB/s", "peak": HBM_PEAK_GBS,
            "traffic": measured_traffic("draft_rows", wl.name)}
    if tk["draft_kernel_launches"]:
        classes["draft"] = {
            "bound": "hbm", "kernel": "k_draft_fused / k_draft_wave (one launch per round: all gamma draft steps)",
            "ms": tk["draft_kernel_ms"], "launches": tk["draft_kernel_launches"],
            "per_launch": draft_kernel_bytes(wl, B, gamma, ctx), "unit": "GB/s", "peak": HBM_PEAK_GBS,
            "traffic": None}
    if tk["gemm_launches"] and tk["attn_launches"] == 0:
        # the whole verify pass is one launch (k_verify_seq, small targets)
        _, vbytes, _ = pass_roofline(c, B, P, ctx)
        classes["verify_pass"] = {
            "bound": "hbm", "kernel": "k_verify_seq (whole verify pass, one workgroup per sequence)",
            "ms": tk["gemm_ms"], "launches": tk["gemm_launches"], "per_launch": vbytes, "unit": "GB/s",
            "peak": HBM_PEAK_GBS, "traffic": None}
    gemm_tflops = tk["gemm_flop"] / (tk["gemm_ms"] * 1e-3) / 1e12 if tk["gemm_ms"] else 0.0
    dominant = max(classes, key=lambda k: classes[k]["ms"]) if classes else None

    def roof(k):
        x = classes[k]
        avg_ms = x["ms"] / max(1, x["launches"])
        ach = x["per_launch"] / (avg_ms * 1e-3) / 1e9
        return {"bound": x["bound"], "kernel": x["kernel"], "achieved": ach, "peak": x["peak"], "unit": x["unit"],
                "frac": ach / x["peak"], "traffic": x["traffic"], "avg_launch_us": avg_ms * 1e3,
                "launches": x["launches"], "algorithmic_bytes_per_launch": x["per_launch"],
                "us_per_round": x["ms"] * 1e3 / nr_k}

    # --- events/s as fractions of roofline (d.5)
    nr = max(1, tph["rounds"])
    events_per_round = events * args.steps / max(1, rounds)
    _, _, t_verify = pass_roofline(c, B, P, ctx)
    _, _, t_dstep = pass_roofline(wl.draft, B, 1, ctx + gamma / 2.0)
    t_accept = B * (2 * gamma + 1) * (3 * c.n_mix + c.n_types + 4) * 4 / (HBM_PEAK_GBS * 1e9)
    sd_roof = events_per_round / (t_verify + gamma * t_dstep + t_accept)
    _, _, t_ar = pass_roofline(c, B, 1, ctx)
    ar_roof = B / t_ar

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_sd * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.prec == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.description}", "batch": B, "n_gen": n_gen, "gamma": gamma,
                   "history_events": wl.n_hist, "weights": "random N(0, 0.02^2), seeded",
                   "target": f"{c.n_layers} layers, d {c.d_model}, {c.n_heads} heads, FFN {c.d_ffn}, "
                             f"{c.n_mix} components, {c.n_types} types",
                   "draft": f"{wl.draft.n_layers} layers, d {wl.draft.d_model}, {wl.draft.n_heads} heads"},
        "prefill_ms_per_step": t_pre * 1e3 / args.steps,
        "ar_value": ar_value,
        "ar_launch": "direct (per-dispatch counters; not a throughput figure)" if args.ar_direct else "graphs",
        "speedup_vs_gpu_ar": value / ar_value if ar_value else None,
        "alpha": alpha,
        "events_per_round": events_per_round,
        "rounds_per_job": rounds / args.steps,
        "ar_candidates_per_job": st["ar_candidates"],
        "roofline": roof(dominant) if dominant else None,
        "events_roofline": {
            "sd": {"roofline_events_per_s": sd_roof, "frac": value / sd_roof,
                   "round_bound_us": (t_verify + gamma * t_dstep + t_accept) * 1e6},
            "ar": {"roofline_events_per_s": ar_roof, "frac": ar_value / ar_roof if ar_value else None,
                   "step_bound_us": t_ar * 1e6},
            "context": ctx},
    }
    for k in classes:
        if k != dominant:
            out[k] = roof(k)
    layered = tk["attn_launches"] > 0
    gemm_gbs = (verify_gemm_bytes(c, B, gamma) * tk["rounds"] / (tk["gemm_ms"] * 1e-3) / 1e9
                if tk["gemm_ms"] and layered else None)
    gemm_peak = MFMA_PEAK_TFLOPS[c.prec]
    out["verify_gemm"] = {"bound": "mfma", "achieved": gemm_tflops, "peak": gemm_peak, "unit": "TFLOP/s",
                          "frac": gemm_tflops / gemm_peak, "launches": tk["gemm_launches"],
                          "avg_launch_us": tk["gemm_ms"] * 1e3 / max(1, tk["gemm_launches"]),
                          "us_per_round": tk["gemm_ms"] * 1e3 / nr_k,
                          "hbm_achieved_gbs": gemm_gbs,
                          "hbm_frac": gemm_gbs / HBM_PEAK_GBS if gemm_gbs is not None else None}
    out["round_us"] = {"draft": tph["draft_ms"] * 1e3 / nr, "verify": tph["verify_ms"] * 1e3 / nr,
                       "accept": tph["accept_ms"] * 1e3 / nr, "rounds": tph["rounds"]}
    vflop, vbytes, vt = pass_roofline(c, B, P, ctx)
    vms = tph["verify_ms"] / nr
    out["verify_pass"] = {"flop": vflop, "bytes": vbytes, "t_bound_us": vt * 1e6, "t_measured_us": vms * 1e3,
                          "frac": vt / (vms * 1e-3) if vms else None,
                          "tflops": vflop / (vms * 1e-3) / 1e12 if vms else None}

    if not args.no_poisson:
        # the same job with the homogeneous-Poisson draft (no draft model),
        # fitted once on the device from the seed histories
        params = tp.tppsd_poisson_fit(HT, HK, c.n_types)
        sp = tp.State(tm, None, B, cap, gamma, seed=1234)
        sp_run = lambda: sp.tppsd_sample_sd_poisson(gamma, params)
        timed_jobs(sp, HT, HK, n_gen, 1, sp_run)
        t_sp, _, _ = timed_jobs(sp, HT, HK, n_gen, args.steps, sp_run)
        sps = sp.tppsd_state_status()
        assert sps["bits"] == 0 and sps["n_done"] == B, sps
        p_value = events * args.steps / t_sp
        note("Poisson draft done")
        out["poisson_draft"] = {"value": p_value, "unit": "events/s", "alpha": sps["accepted"] / max(1, sps["drafted"]),
                                "speedup_vs_gpu_ar": p_value / ar_value if ar_value else None}
        del sp
    if not args.no_mismatch:
        # a draft whose decoder biases disagree with the target's (acceptance
        # in the range trained models reach): same target, histories and seed
        wdm = W.mismatch_draft(wd, wl.draft, W.seed_sequence(wl.index, 4))
        dmm = tp.Model(wl.draft, wdm, dev)
        sm = tp.State(tm, dmm, B, cap, gamma, seed=1234)
        sm_run = lambda: sm.tppsd_sample_sd(gamma)
        timed_jobs(sm, HT, HK, n_gen, 1, sm_run)
        t_sm, _, _ = timed_jobs(sm, HT, HK, n_gen, args.steps, sm_run)
        sms = sm.tppsd_state_status()
        assert sms["bits"] == 0 and sms["n_done"] == B, sms
        m_value = events * args.steps / t_sm
        note("mismatched draft done")
        out["mismatch_draft"] = {"value": m_value, "unit": "events/s",
                                 "alpha": sms["accepted"] / max(1, sms["drafted"]),
                                 "speedup_vs_gpu_ar": m_value / ar_value if ar_value else None,
                                 "draft": "decoder biases b_mu + 0.5, b_sigma + 0.3, b_k2 + N(0, 0.5^2)"}
        del sm, dmm
    if not args.no_window:
        out["window"] = window_jobs(args, wl, gamma, sd, ar, HT, HK, ht, n_gen, B)
        note("window jobs done")
    if args.gamma_sweep:
        out["gamma_sweep"] = gamma_sweep(args, wl, tm, dm, HT, HK, ar_value, B, n_gen)
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
