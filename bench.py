"""Benchmark: accepted events/sec of TPP-SD sampling on one MI355X, vs the GPU
autoregressive sampler, with the verify-attention kernel's roofline and the
CPU oracle's rate as a reported baseline.

A step is one complete sampling job over the batch: prefill of the seed
histories (encoding them into both KV caches) followed by TPP-SD rounds
(draft, verify, accept) until every sequence has n_gen new events.
value = B * n_gen * steps / (timed seconds). The same job with naive AR
sampling gives the speedup denominator.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config c2] [--gamma G]
                    [--gamma-sweep 1,2,5,10,15,20]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "accepted events/sec (1 MI355X) SD vs AR; verify MFMA util %; KV-attn HBM GB/s"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}
KERNEL_NAME = {"bf16": "k_attn_mfma<d_head, 1> (verify attention)",
               "fp32": "k_attn_mfma_f32<d_head, 1> (verify attention)"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="c2")
    ap.add_argument("--gamma", type=int, default=None)
    ap.add_argument("--ar-steps", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-poisson", action="store_true", help="skip the homogeneous-Poisson draft run")
    ap.add_argument("--no-window", action="store_true", help="skip the end-time (window) runs")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="oracle sample: target CPU seconds")
    ap.add_argument("--cpu-seqs", type=int, default=64, help="oracle sample: at most this many sequences")
    ap.add_argument("--gamma-sweep", default=None,
                    help="comma-separated draft lengths: the SD job at each, against the same AR job")
    return ap.parse_args()


def attention_bytes_per_launch(wl, gamma, B):
    """Algorithmic HBM bytes of one verify-attention launch (all layers counted
    per launch of one layer): keys and values of every cached position plus
    the P new ones, read once, at the run-average context n0 + n_gen / 2;
    plus the queries read and the outputs written."""
    c = wl.target
    elt = 2 if c.prec == "bf16" else 4
    P = gamma + 1
    ctx = wl.n_hist + wl.n_gen / 2.0
    kv = B * c.n_heads * (ctx + P) * c.d_head * 2 * elt
    qo = B * P * c.d_model * elt * 2
    return kv + qo


def verify_weight_bytes(wl):
    """Bytes of the target's weights read by one verify pass (once)."""
    c = wl.target
    elt = 2 if c.prec == "bf16" else 4
    d, F, M, K = c.d_model, c.d_ffn, c.n_mix, c.n_types
    layer = 6 * d * d if getattr(c, "encoder", "thp") == "attnhp" else 4 * d * d + 2 * d * F
    return elt * (c.n_layers * layer + 4 * d * d + (3 * M + K) * 4 * d)


def verify_pass_fraction(wl, gamma, B, verify_ms):
    """Roofline time of one verify pass, max(flop / MFMA peak, bytes / HBM
    peak), against its measured time (phase timing, graph-replayed). flop:
    the GEMMs of every layer and the decoder plus QK and PV over the run-average
    context; bytes: the K/V read and append, the weights once, the activations
    of the pass in and out."""
    c = wl.target
    elt = 2 if c.prec == "bf16" else 4
    L, d, F, M, K = c.n_layers, c.d_model, c.d_ffn, c.n_mix, c.n_types
    P = gamma + 1
    T = B * P
    ctx = wl.n_hist + wl.n_gen / 2.0
    # per layer: THP QKV, output and FFN matrices; AttNHP one 3d x 2d matrix over [z; h]
    layer = 6 * d * d if getattr(c, "encoder", "thp") == "attnhp" else 4 * d * d + 2 * d * F
    flop = 2.0 * T * (L * layer + 4 * d * d + 3 * M * d + K * d) + 4.0 * T * L * d * ctx
    w_bytes = elt * (L * layer + 4 * d * d + 3 * M * d + K * d)
    bytes_ = B * L * (ctx + P) * 2 * d * elt + w_bytes + T * 8 * (3 * M + K)
    t_bound = max(flop / (MFMA_PEAK_TFLOPS[c.prec] * 1e12), bytes_ / (HBM_PEAK_GBS * 1e9))
    return {"flop": flop, "bytes": bytes_, "t_bound_us": t_bound * 1e6, "t_measured_us": verify_ms * 1e3,
            "frac": t_bound / (verify_ms * 1e-3) if verify_ms else None,
            "tflops": flop / (verify_ms * 1e-3) / 1e12 if verify_ms else None}


def verify_gemm_bytes(wl, gamma, B):
    """Algorithmic HBM bytes of the GEMM part of one verify pass: what the
    products must move at least, whatever the kernels. THP layer: its
    attention output o in, the residual stream x in and out, its q, k, v out
    (once per layer), the layer's matrices once; plus the first layer's
    LayerNorm input and the decoder's first product (LN_f(x) in, [E; V_k1]
    out). The layered kernels move more (the FFN hidden activations out and
    back, x re-read per product); the fused layer kernel moves this. AttNHP
    layer: one product over the 2d-wide [z; h] in, q, k, v out."""
    c = wl.target
    elt = 2 if c.prec == "bf16" else 4
    d, F, L = c.d_model, c.d_ffn, c.n_layers
    T = B * (gamma + 1)
    if getattr(c, "encoder", "thp") == "attnhp":
        layers = L * (T * 2 * d * elt + 6 * d * d * elt + T * 3 * d * elt)
    else:
        layers = L * (T * d * elt + T * d * 8 + T * 3 * d * elt + (4 * d * d + 2 * d * F) * elt) + T * d * 4
    dec = T * d * 4 + 4 * d * d * elt + T * 4 * d * elt
    return float(layers + dec)


def gamma_sweep(args, wl, tm, dm, HT, HK, ar_value, B, n_gen):
    """The SD job at each draft length of the sweep (one state per length,
    one warmup job, args.steps timed jobs), against the AR job's rate."""
    import torch

    from paper_2507_09252_amd import tppsd as tp
    rows = []
    for g in [int(x) for x in args.gamma_sweep.split(",") if x.strip()]:
        st = tp.State(tm, dm, B, wl.n_hist + n_gen + g + 1, g, seed=1234)

        def job():
            st.tppsd_prefill(HT, HK, n_gen)
            return st.tppsd_sample_sd(g)

        job()
        torch.cuda.synchronize()
        rounds = 0
        t0 = time.perf_counter()
        for _ in range(args.steps):
            rounds += job()
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        s = st.tppsd_state_status()
        assert s["bits"] == 0 and s["n_done"] == B, s
        st.tppsd_timing_enable(tp.TIME_PHASES)
        job()
        ph = st.tppsd_timing_read()
        st.tppsd_timing_enable(0)
        nr = max(1, ph["rounds"])
        value = B * n_gen * args.steps / dt
        rows.append({"gamma": g, "value": value, "speedup_vs_gpu_ar": value / ar_value if ar_value else None,
                     "alpha": s["accepted"] / max(1, s["drafted"]), "rounds_per_job": rounds / args.steps,
                     "round_us": {"draft": ph["draft_ms"] * 1e3 / nr, "verify": ph["verify_ms"] * 1e3 / nr,
                                  "accept": ph["accept_ms"] * 1e3 / nr}})
        print(f"gamma {g}: {value:.4g} events/s, alpha {rows[-1]['alpha']:.3f}", file=sys.stderr, flush=True)
        del st
    return rows


def attention_source_sha256():
    """SHA-256 over the sources that define the attention kernels."""
    import hashlib
    h = hashlib.sha256()
    for f in ("tppsd_attention.hip", "tppsd_attention.h", "tppsd_device.h"):
        with open(os.path.join(ROOT, "paper_2507_09252_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(wl_name):
    """HBM bytes per verify-attention launch from the committed rocprofv3 --pmc
    runs, if the kernel source is unchanged since they were taken; else None."""
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "verify_attention_traffic.json")))
    except OSError:
        return None
    if attention_source_sha256() != rec["kernel_source_sha256"]:
        return None
    w = rec["workloads"].get(wl_name)
    return None if w is None else w["traffic_bytes_per_launch"]


def cpu_baseline(wl, gamma, wt, wd, ht, hk, budget_s, max_seqs):
    """The oracle (float64 NumPy, one thread) on a bounded sample of the same
    job, sized to about budget_s seconds of CPU work: starting from 8
    sequences x 16 events, the sample grows (events per sequence first, up to
    n_gen, then sequences, up to max_seqs) by the ratio of the budget to the
    last run's time, until a run takes at least half the budget or the sample
    is the whole allowed job; a whole job shorter than half the budget is
    repeated to about three quarters of it. The last run is reported."""
    from threadpoolctl import threadpool_limits

    from oracle import sampler as S
    from oracle.model import Model as OModel
    T, D = OModel(wl.target, wt), OModel(wl.draft, wd)
    top_seq = max(1, min(wl.batch, max_seqs))
    n_seq, n_events = min(top_seq, 8), min(wl.n_gen, 16)
    with threadpool_limits(1):
        for _ in range(6):
            t0 = time.perf_counter()
            st = S.sample_sd(T, D, ht[:n_seq], hk[:n_seq], n_events, gamma, seed=1234)
            dt = time.perf_counter() - t0
            if dt >= 0.5 * budget_s or (n_seq == top_seq and n_events == wl.n_gen):
                break
            grow = min(8.0, budget_s / max(dt, 1e-3))
            e2 = int(min(wl.n_gen, n_events * grow))
            n_seq = int(min(top_seq, max(n_seq, n_seq * grow * n_events / e2)))
            n_events = e2
        ev = int(st.gen.sum())
        reps = 1
        if dt < 0.5 * budget_s:
            # the whole allowed job is shorter than the budget: repeat it
            reps = int(min(20, np.ceil(0.75 * budget_s / max(dt, 1e-3))))
            t0 = time.perf_counter()
            for _ in range(reps):
                st = S.sample_sd(T, D, ht[:n_seq], hk[:n_seq], n_events, gamma, seed=1234)
            dt = time.perf_counter() - t0
            ev = int(st.gen.sum()) * reps
    return {"value": ev / dt, "unit": "events/s", "cores": 1, "kind": "oracle",
            "sample": f"{n_seq} sequences x first {n_events} generated events of {wl.name} "
                      f"(TPP-SD, gamma={gamma}){f', {reps} repetitions' if reps > 1 else ''}, "
                      f"float64 NumPy, {dt:.1f} s"}


def window_jobs(args, wl, gamma, sd, ar, HT, HK, ht, n_gen, B):
    """TPP-SD and AR with an end time per sequence (Algorithm 1's T): each
    sequence's window is 0.75 n_gen of its history's mean interval after its
    pending event, n_gen stays the cap. Reports generated events per second,
    how the sequences ended, and the model log-likelihood (Eq. (2)) both
    samplers accumulate: its batch means and their difference (the model-side
    likelihood discrepancy |L_ar - L_sd|)."""
    import torch
    mean_iv = (ht[:, -1] - ht[:, 0]) / (ht.shape[1] - 1)
    t_end = torch.from_numpy((ht[:, -1] + 0.75 * n_gen * mean_iv).astype(np.float32)).to(HT.device)
    res = {}
    for name, st, steps in (("sd", sd, args.steps), ("ar", ar, max(1, args.ar_steps))):
        def job():
            st.tppsd_prefill(HT, HK, n_gen, t_end=t_end)
            if name == "sd":
                st.tppsd_sample_sd(gamma)
            else:
                st.tppsd_sample_ar(n_gen)
        job()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            job()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / steps
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
              "(the batch shards across GPUs with no exchange, see DESIGN.md)", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2507_09252_amd import tppsd as tp
    from paper_2507_09252_amd import workloads as W

    wl = W.WORKLOADS[args.config]
    gamma = args.gamma or wl.gamma
    B, n_gen = wl.batch, wl.n_gen
    wt, wd = W.workload_weights(wl)
    ht, hk = W.make_histories(wl)
    dev = torch.device("cuda:0")
    tm, dm = tp.Model(wl.target, wt, dev), tp.Model(wl.draft, wd, dev)
    cap = wl.n_hist + n_gen + gamma + 1
    sd = tp.State(tm, dm, B, cap, gamma, seed=1234)
    ar = tp.State(tm, None, B, cap, gamma, seed=1234)
    HT, HK = torch.from_numpy(ht).to(dev), torch.from_numpy(hk).to(dev)

    def sd_job():
        sd.tppsd_prefill(HT, HK, n_gen)
        return sd.tppsd_sample_sd(gamma)

    def ar_job():
        ar.tppsd_prefill(HT, HK, n_gen)
        ar.tppsd_sample_ar(n_gen)

    for _ in range(args.warmup):
        sd_job()
        if args.ar_steps > 0:
            ar_job()
    torch.cuda.synchronize()
    # timed SD jobs: every round replays one captured HIP graph
    rounds = 0
    t0 = time.perf_counter()
    for _ in range(args.steps):
        rounds += sd_job()
    torch.cuda.synchronize()
    t_sd = time.perf_counter() - t0
    st = sd.tppsd_state_status()
    assert st["bits"] == 0 and st["n_done"] == B, st
    # one more job with the verify attention and GEMM launches bracketed by
    # HIP events (rounds launched directly on this stream, same kernels and
    # data), and one with events between the draft / verify / accept graphs
    sd.tppsd_timing_enable(tp.TIME_KERNELS)
    sd_job()
    tk = sd.tppsd_timing_read()
    sd.tppsd_timing_enable(tp.TIME_PHASES)
    sd_job()
    tph = sd.tppsd_timing_read()
    sd.tppsd_timing_enable(0)
    torch.cuda.synchronize()
    attn_ms, attn_launches = tk["attn_ms"], tk["attn_launches"]

    events = B * n_gen
    ar_value = None
    if args.ar_steps > 0:
        t0 = time.perf_counter()
        for _ in range(args.ar_steps):
            ar_job()
        torch.cuda.synchronize()
        t_ar = time.perf_counter() - t0
        sa = ar.tppsd_state_status()
        assert sa["bits"] == 0 and sa["n_done"] == B, sa
        ar_value = events * args.ar_steps / t_ar
    value = events * args.steps / t_sd
    alpha = st["accepted"] / max(1, st["drafted"])
    poisson = None
    if not args.no_poisson:
        # the same job with the homogeneous-Poisson draft (no draft model),
        # fitted once on the device from the seed histories
        params = tp.tppsd_poisson_fit(HT, HK, wl.target.n_types)
        sp = tp.State(tm, None, B, cap, gamma, seed=1234)

        def sp_job():
            sp.tppsd_prefill(HT, HK, n_gen)
            return sp.tppsd_sample_sd_poisson(gamma, params)

        sp_job()
        torch.cuda.synchronize()
        p_rounds = 0
        t0 = time.perf_counter()
        for _ in range(args.steps):
            p_rounds += sp_job()
        torch.cuda.synchronize()
        t_sp = time.perf_counter() - t0
        sps = sp.tppsd_state_status()
        assert sps["bits"] == 0 and sps["n_done"] == B, sps
        sp.tppsd_timing_enable(tp.TIME_PHASES)
        sp_job()
        pph = sp.tppsd_timing_read()
        sp.tppsd_timing_enable(0)
        p_nr = max(1, pph["rounds"])
        p_value = events * args.steps / t_sp
        poisson = {"value": p_value, "unit": "events/s", "alpha": sps["accepted"] / max(1, sps["drafted"]),
                   "speedup_vs_gpu_ar": None, "rounds_per_job": p_rounds / args.steps,
                   "ar_candidates_per_job": sps["ar_candidates"],
                   "round_us": {"draft": pph["draft_ms"] * 1e3 / p_nr, "verify": pph["verify_ms"] * 1e3 / p_nr,
                                "accept": pph["accept_ms"] * 1e3 / p_nr, "rounds": pph["rounds"]}}
        del sp
    per_launch = attention_bytes_per_launch(wl, gamma, B)
    kernel_name = KERNEL_NAME[wl.prec]
    if attn_launches == 0 and tk["gemm_launches"] > 0:
        # the whole verify pass is one launch (k_verify_seq, small targets): its
        # attention is inside it, so the pass's own algorithmic bytes (every
        # layer's K/V and queries / outputs, the weights once) over its duration
        attn_launches, attn_ms = tk["gemm_launches"], tk["gemm_ms"]
        per_launch = per_launch * wl.target.n_layers + verify_weight_bytes(wl)
        kernel_name = "k_verify_seq (whole verify pass, one workgroup per sequence)"
    avg_ms = attn_ms / max(1, attn_launches)
    achieved = per_launch / (avg_ms * 1e-3) / 1e9 if attn_launches else 0.0
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
                   "history_events": wl.n_hist, "weights": "random N(0, 0.02^2), seeded"},
        "ar_value": ar_value,
        "speedup_vs_gpu_ar": value / ar_value if ar_value else None,
        "alpha": alpha,
        "events_per_round": events * args.steps / max(1, rounds),
        "rounds_per_job": rounds / args.steps,
        "ar_candidates_per_job": st["ar_candidates"],
        "roofline": {"bound": "hbm", "kernel": kernel_name, "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(wl.name) if kernel_name == KERNEL_NAME[wl.prec] else None,
                     "avg_launch_us": avg_ms * 1e3, "launches": attn_launches,
                     "algorithmic_bytes_per_launch": per_launch},
    }
    if not args.no_window:
        out["window"] = window_jobs(args, wl, gamma, sd, ar, HT, HK, ht, n_gen, B)
    c = wl.target
    gemm_tflops = tk["gemm_flop"] / (tk["gemm_ms"] * 1e-3) / 1e12 if tk["gemm_ms"] else 0.0
    gemm_peak = MFMA_PEAK_TFLOPS[c.prec]
    # (a one-launch verify pass has no separate GEMM launches to price)
    layered = kernel_name == KERNEL_NAME[wl.prec]
    gemm_gbs = (verify_gemm_bytes(wl, gamma, B) * tk["rounds"] / (tk["gemm_ms"] * 1e-3) / 1e9
                if tk["gemm_ms"] and layered else None)
    out["verify_gemm"] = {"bound": "mfma", "achieved": gemm_tflops, "peak": gemm_peak, "unit": "TFLOP/s",
                          "frac": gemm_tflops / gemm_peak, "launches": tk["gemm_launches"],
                          "avg_launch_us": tk["gemm_ms"] * 1e3 / max(1, tk["gemm_launches"]),
                          "hbm_achieved_gbs": gemm_gbs,
                          "hbm_frac": gemm_gbs / HBM_PEAK_GBS if gemm_gbs is not None else None}
    nr = max(1, tph["rounds"])
    out["round_us"] = {"draft": tph["draft_ms"] * 1e3 / nr, "verify": tph["verify_ms"] * 1e3 / nr,
                       "accept": tph["accept_ms"] * 1e3 / nr, "rounds": tph["rounds"]}
    out["verify_pass"] = verify_pass_fraction(wl, gamma, B, tph["verify_ms"] / nr)
    if poisson is not None:
        poisson["speedup_vs_gpu_ar"] = poisson["value"] / ar_value if ar_value else None
        out["poisson_draft"] = poisson
    if args.gamma_sweep:
        out["gamma_sweep"] = gamma_sweep(args, wl, tm, dm, HT, HK, ar_value, B, n_gen)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, gamma, wt, wd, ht, hk, args.cpu_seconds, args.cpu_seqs)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
