"""Benchmark of the progressive approximate-LSTM hot path on one MI355X.

A step is one call of approx_lstm_run over one synthetic driving-shaped
sequence (D=2048 ReLU-like features, H=512, T=16, batch 1; gate matrices
2048x2560 per gate factorised to rank 512 with 75% magnitude pruning) at the
full refinement budget K=512 per gate.  The factorisation (prepare) is setup
and is not timed.  Inputs are resident in HBM before the timed region.

Prints one JSON line: timesteps/s at K=512, microseconds per timestep, a
sweep over K = 1..512, the roofline of the run kernel, and the float64 CPU
oracle timed on a bounded sample of the same workload.
"""

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0


def progress(msg):
    """One progress line on stderr (stdout carries only the JSON line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_bytes_per_timestep(G, Rg, NZ, C, K, D, H, B, L):
    """Bytes the method must move per timestep (Eq. (1) streamed once per
    timestep, as the paper's design streams u and v for every refinement):
    per term 4*R_g (u) + 6*NZ (fp32 value + 16-bit index; 4*C if v is dense)
    + 4 (sigma), plus x_t and the h outputs."""
    v_bytes = 4 * C if NZ == C else 6 * NZ
    return G * K * (4 * Rg + v_bytes + 4) + 4 * D * B + 4 * H * B * L


def algorithmic_flops_per_timestep(G, Rg, NZ, K, B):
    """N_steps * (2R + 2NZ + 1) per gate (Sec. III), per sequence."""
    return G * K * (2 * Rg + 2 * NZ + 1) * B


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--prune", type=float, default=0.75)
    ap.add_argument("--K", type=int, default=512)
    ap.add_argument("--blocks", type=int, default=0, help="workgroups of the run kernel (0 = automatic)")
    ap.add_argument("--sweep", default="0,1,2,4,8,16,32,64,128,256,512")
    ap.add_argument("--sweep-steps", type=int, default=50)
    ap.add_argument("--blocks-sweep", default="", help="comma list of workgroup counts to time at K (tuning)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-phases", action="store_true", help="skip the in-kernel phase stamps")
    ap.add_argument("--no-anytime", action="store_true", help="skip the error-vs-time comparison with the row-tile baseline")
    ap.add_argument("--no-batched", action="store_true",
                    help="skip the batched (256 sequences, bf16 MFMA) summary in the default line")
    ap.add_argument("--no-prune-sweep", action="store_true",
                    help="skip the pruning sweep (0, 50, 90%% at K=512) in the default line")
    ap.add_argument("--no-stack", action="store_true", help="skip the stacked-layer summary in the default line")
    ap.add_argument("--no-deadline", action="store_true", help="skip the deadline-workload summary in the default line")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only time a plain 256 MiB device copy (reference for HBM counters)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--batched-sweep", default="32,128,512", help="K values timed in the batched workload")
    ap.add_argument("--time-prepare", default="",
                    help="NAME:RANK:PRUNE -- only time the device factorisation of a named workload "
                         "(e.g. deadline:2048:0.9) and print one JSON line")
    ap.add_argument("--workload", default="driving", choices=["driving", "batched", "deadline", "stack"],
                    help="driving: batch 1, fp32 (default line); batched: 256 sequences, bf16 MFMA path; "
                         "deadline: D=H=2048, T=64, 8 sequences, rank 2048, both deadline modes; "
                         "stack: two layers D=4096 -> 1024 -> 1024, T=32, rank 1024, per-layer budgets")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): this build has no multi-GPU path; "
              "independent sequences or levels would shard across GPUs with no exchange.", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_calibration:
        copy_calibration(torch)
        return
    from paper_1905_00689_amd import synth
    from paper_1905_00689_amd import binding as B

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.time_prepare:
        time_prepare(args.time_prepare, torch, synth, B)
        return
    if args.workload == "batched":
        bench_batched(args, torch)
        return
    if args.workload == "deadline":
        bench_deadline(args, torch)
        return
    if args.workload == "stack":
        bench_stack(args, torch)
        return
    dev = torch.device("cuda")
    wl = synth.named("driving")
    D, H, T, Bn = wl.D, wl.H, wl.T, wl.B
    C = D + H
    rank = 512
    t0 = time.time()
    m = B.approx_lstm_prepare(wl.W[:, :D], wl.W[:, D:], wl.b, D, H, rank, prune_ratio=args.prune, groups=4)
    prep_s = time.time() - t0
    info = m.info
    NZ, G, Rg = info["nz"], info["groups"], info["rows_per_group"]
    if args.blocks:
        B.approx_lstm_set_launch(m, args.blocks, 0)
    B.approx_lstm_reserve(m, T, Bn, 1)
    x = torch.from_numpy(wl.x).to(dev)
    h_out = torch.empty((1, T, Bn, H), device=dev)
    stream = torch.cuda.current_stream()

    def timed(K, steps, warmup):
        for _ in range(warmup):
            B.approx_lstm_run(m, x, [K], h_out, stream=stream)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            B.approx_lstm_run(m, x, [K], h_out, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        B.approx_lstm_check(m)
        return e0.elapsed_time(e1) / steps   # ms per run

    K = args.K
    progress(f"driving prepared ({prep_s:.1f} s); timing K={K}")
    ms = timed(K, args.steps, args.warmup)
    us_per_ts = ms * 1e3 / T
    value = T * Bn / (ms * 1e-3)
    dist = step_distribution(torch, lambda: B.approx_lstm_run(m, x, [K], h_out, stream=stream), stream, args.steps)

    sweep = {"K": [], "us_per_timestep": [], "timesteps_per_s": [], "hbm_frac": []}
    for k in [int(s) for s in args.sweep.split(",") if s]:
        if k > rank:
            continue
        msk = timed(k, args.sweep_steps, 5)
        byts = T * algorithmic_bytes_per_timestep(G, Rg, NZ, C, k, D, H, Bn, 1)
        sweep["K"].append(k)
        sweep["us_per_timestep"].append(round(msk * 1e3 / T, 4))
        sweep["timesteps_per_s"].append(round(T * Bn / (msk * 1e-3), 1))
        sweep["hbm_frac"].append(round(byts / (msk * 1e-3) / 1e9 / HBM_PEAK_GBS, 4))

    progress("K sweep done")
    tune = None
    if args.blocks_sweep:
        tune = {"K": K, "blocks": [], "us_per_timestep": []}
        for P in [int(s) for s in args.blocks_sweep.split(",") if s]:
            B.approx_lstm_set_launch(m, P, 0)
            tune["blocks"].append(P)
            tune["us_per_timestep"].append(round(timed(K, args.sweep_steps, 5) * 1e3 / T, 4))
        B.approx_lstm_set_launch(m, args.blocks, 0)

    # in-kernel phase timing of one run per K (workgroup 0's stamps)
    phases = {}
    for k in ([] if args.no_phases else sorted({1, 64, K})):
        B.approx_lstm_set_timing(m, 1)
        B.approx_lstm_run(m, x, [k], h_out, stream=stream)
        st = B.approx_lstm_get_timing(m, T, stream=stream)
        B.approx_lstm_set_timing(m, 0)
        ph = np.array([[st[1 + 4 * t + i] for i in range(4)] + [st[1 + 4 * (t + 1)]] for t in range(T)])
        phases[str(k)] = {"phaseA_us": round(float(np.mean(ph[:, 1] - ph[:, 0])), 3),
                          "z_wait_us": round(float(np.mean(ph[:, 2] - ph[:, 1])), 3),
                          "phaseB_us": round(float(np.mean(ph[:, 3] - ph[:, 2])), 3),
                          "h_out_us": round(float(np.mean(ph[:, 4] - ph[:, 3])), 3),
                          "recurrence_us": round(float(st[1 + 4 * T] - st[1]), 3)}

    # One step launches input_proj_kernel (x-part projections, whole GPU) and
    # then the recurrence (pair_lstm_kernel for one level of one sequence,
    # else progressive_lstm_kernel); the roofline covers the step, timed with
    # events on the launch stream over the timed region.
    plan = B.approx_lstm_plan(m, T, Bn, [K])
    rec = "pair_lstm_kernel" if plan["pair_kernel"] else "progressive_lstm_kernel"
    bytes_launch = T * algorithmic_bytes_per_timestep(G, Rg, NZ, C, K, D, H, Bn, 1)
    achieved = bytes_launch / (ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic("driving") if (K == 512 and abs(args.prune - 0.75) < 1e-9) else None,
                "kernel": f"one step: input_proj_kernel + {rec} ({plan['blocks']} workgroups)",
                "bytes_per_launch": bytes_launch,
                "flops_per_launch": T * algorithmic_flops_per_timestep(G, Rg, NZ, K, Bn)}

    # the same step at the other pruning ratios of the driving configuration
    # (factorised on the device), K = 512 and 64
    progress("phases done")
    prune_sweep = None
    if not args.no_prune_sweep:
        prune_sweep = {"prune": [], "nz": [], "prepare_device_s": [], "us_per_timestep_K512": [],
                       "hbm_frac_K512": [], "us_per_timestep_K64": []}
        for p in (0.0, 0.5, 0.75, 0.9):
            t1 = time.time()
            mp = B.approx_lstm_prepare(wl.W[:, :D], wl.W[:, D:], wl.b, D, H, rank, prune_ratio=p, groups=4,
                                       flags=B.FLAG_DEVICE_FACTORISE)
            sec = round(time.time() - t1, 2)
            nzp = mp.info["nz"]
            row = {}
            for kk in (512, 64):
                for _ in range(5):
                    B.approx_lstm_run(mp, x, [kk], h_out, stream=stream)
                torch.cuda.synchronize()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for _ in range(args.sweep_steps):
                    B.approx_lstm_run(mp, x, [kk], h_out, stream=stream)
                e1.record(stream)
                torch.cuda.synchronize()
                B.approx_lstm_check(mp)
                row[kk] = e0.elapsed_time(e1) / args.sweep_steps
            byts = T * algorithmic_bytes_per_timestep(G, Rg, nzp, C, 512, D, H, Bn, 1)
            prune_sweep["prune"].append(p)
            prune_sweep["nz"].append(nzp)
            prune_sweep["prepare_device_s"].append(sec)
            prune_sweep["us_per_timestep_K512"].append(round(row[512] * 1e3 / T, 4))
            prune_sweep["hbm_frac_K512"].append(round(byts / (row[512] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4))
            prune_sweep["us_per_timestep_K64"].append(round(row[64] * 1e3 / T, 4))
            del mp
            progress(f"prune {p} done")

    # the exact (dense) LSTM on the same sequence, timed the same way: the
    # baseline the progressive approximation trades accuracy against
    me = B.approx_lstm_exact_prepare(wl.W[:, :D], wl.W[:, D:], wl.b, D, H)
    he = torch.empty((T, Bn, H), device=dev)

    def timed_exact(steps, warmup):
        for _ in range(warmup):
            B.approx_lstm_exact_run(me, x, he, stream=stream)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            B.approx_lstm_exact_run(me, x, he, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        B.approx_lstm_exact_check(me)
        return e0.elapsed_time(e1) / steps

    ms_exact = timed_exact(args.sweep_steps, 5)
    progress("exact baseline done")
    exact = {"us_per_timestep": round(ms_exact * 1e3 / T, 4), "timesteps_per_s": round(T * Bn / (ms_exact * 1e-3), 1),
             "weights_bytes": 4 * 4 * H * (D + H)}
    anytime = None if args.no_anytime else anytime_comparison(torch, B, stream)
    progress("anytime comparison done")
    batched = None if args.no_batched else batched_summary(args, torch)
    progress("batched summary done")
    stack = None if args.no_stack else stack_summary(args, torch)
    progress("stack summary done")
    deadline = None if args.no_deadline else deadline_summary(args, torch)
    progress("deadline summary done")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(m, wl, K, args.cpu_seconds)
        progress("cpu baseline done")

    out = {
        "metric": "LSTM timesteps/sec at refinement budget K (and us/timestep vs K)",
        "value": round(value, 1), "unit": "timesteps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "driving-shaped LSTM D=2048 H=512 T=16 B=1, per-gate rank 512, "
                               f"{int(args.prune * 100)}% pruning (NZ={NZ}), K={K}",
                   "D": D, "H": H, "T": T, "batch": Bn, "rank": rank, "nz": NZ, "K": K, "groups": G},
        "us_per_timestep": round(us_per_ts, 4), "step_ms": dist, "prepare_s": round(prep_s, 2),
        "phases": phases, "sweep": sweep, "prune_sweep": prune_sweep, "tune": tune, "exact_baseline": exact,
        "anytime": anytime, "batched": batched, "stack": stack, "deadline": deadline, "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def _qor(head, ref):
    """Error measures of an output sequence h [T, B, H] against the exact one:
    max over (t, b) of ||h - h_exact||_inf / ||h_exact||_inf, and the mean
    KL(p_exact || p) of the 4-way softmax of a fixed random read-out."""
    lref = ref @ head.T
    pref = np.exp(lref - lref.max(-1, keepdims=True))
    pref /= pref.sum(-1, keepdims=True)

    def quality(h):
        h = h.astype(np.float64)
        num = np.abs(h - ref).max(-1)
        den = np.maximum(np.abs(ref).max(-1), 1e-6)
        lg = h @ head.T
        lq = lg - lg.max(-1, keepdims=True)
        lq = lq - np.log(np.exp(lq).sum(-1, keepdims=True))
        kl = (pref * (np.log(np.maximum(pref, 1e-300)) - lq)).sum(-1)
        return float((num / den).max()), max(0.0, float(kl.mean()))
    return quality


def _sig(v):
    return float("%.3g" % v)


def anytime_curves(torch, B, wl, stream, configs, Ks, rows_list, steps=30):
    """Error against time per timestep for the two anytime schemes on the
    device (Sec. VI-B and its error-vs-time figure): the progressive scheme at
    budget K for each (rank, nz) in `configs`, and the dense baseline stopped
    after `rows` rows of every gate.  Errors are measured against the
    device's exact dense LSTM on the same input (see _qor); the read-out is a
    fixed random stand-in for the driving model's 4-way prediction layer.
    `time_to_kl` gives, per KL level, the fastest configuration of each scheme
    that reaches it and the ratio."""
    from paper_1905_00689_amd import synth
    D, H, T, Bn = wl.D, wl.H, wl.T, wl.B
    dev = torch.device("cuda")
    x = torch.from_numpy(wl.x).to(dev)
    head = synth.softmax_head(H).astype(np.float64)

    def us_per_timestep(fn):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps * 1e3 / T

    me = B.approx_lstm_exact_prepare(wl.W[:, :D], wl.W[:, D:], wl.b, D, H)
    hr = torch.empty((T, Bn, H), device=dev)
    B.approx_lstm_exact_run(me, x, hr, stream=stream)
    torch.cuda.synchronize()
    B.approx_lstm_exact_check(me)
    quality = _qor(head, hr.cpu().numpy().astype(np.float64))

    tiles = {"rows": [], "us_per_timestep": [], "rel_err": [], "kl": []}
    for r in rows_list:
        us = us_per_timestep(lambda: B.approx_lstm_exact_run_rows(me, x, r, hr, stream=stream))
        B.approx_lstm_exact_check(me)
        e, kl = quality(hr.cpu().numpy())
        tiles["rows"].append(r)
        tiles["us_per_timestep"].append(round(us, 3))
        tiles["rel_err"].append(_sig(e))
        tiles["kl"].append(_sig(kl))

    prog = {}
    hk = torch.empty((1, T, Bn, H), device=dev)
    for cfg in configs:
        rank, nz = cfg[0], cfg[1]
        residual = len(cfg) < 3 or cfg[2] != "non-residual"
        flags = 0 if residual else B.FLAG_NON_RESIDUAL
        m = B.approx_lstm_prepare(wl.W[:, :D], wl.W[:, D:], wl.b, D, H, rank, nz=nz, groups=4, flags=flags)
        c = {"nz": m.info["nz"], "rank": rank, "K": [], "us_per_timestep": [], "rel_err": [], "kl": []}
        for k in Ks:
            if k > rank:
                continue
            us = us_per_timestep(lambda: B.approx_lstm_run(m, x, [k], hk, stream=stream))
            B.approx_lstm_check(m)
            e, kl = quality(hk[0].cpu().numpy())
            c["K"].append(k)
            c["us_per_timestep"].append(round(us, 3))
            c["rel_err"].append(_sig(e))
            c["kl"].append(_sig(kl))
        prog[str(c["nz"]) + ("" if residual else "-nonres")] = c
        del m

    def fastest(us, err, level):
        ok = [u for u, v in zip(us, err) if v <= level]
        return min(ok) if ok else None

    tte = []
    for level in [1e-2, 1e-3, 1e-4, 1e-5, 1e-6]:
        row = {"kl": level, "row_tile_us": fastest(tiles["us_per_timestep"], tiles["kl"], level)}
        for name, c in prog.items():
            if not name.endswith("-nonres"):
                row["nz" + name + "_us"] = fastest(c["us_per_timestep"], c["kl"], level)
        best = [v for k, v in row.items() if k.startswith("nz") and v is not None]
        row["speedup"] = round(row["row_tile_us"] / min(best), 3) if best and row["row_tile_us"] else None
        tte.append(row)
    return {"workload": f"{wl.name} D={D} H={H} T={T} B={Bn}", "progressive": prog, "row_tile": tiles,
            "exact_us_per_timestep": tiles["us_per_timestep"][-1] if tiles["rows"] and tiles["rows"][-1] == H else None,
            "time_to_kl": tte}


def anytime_comparison(torch, B, stream):
    """The error-vs-time comparison on three workloads: the driving shape
    with Gaussian weights (the hard, flat-spectrum case) and with
    decaying-spectrum weights at 75% pruning, and the paper's own model shape
    (D=8256, H=64, T=100) with decaying-spectrum weights at its three
    non-zero counts (4160, 130 and 32 per v)."""
    from paper_1905_00689_amd import synth
    Kd = [0, 1, 2, 4, 8, 16, 32, 64, 128, 256, 384, 512]
    rows_d = [0, 16, 32, 64, 128, 256, 384, 448, 480, 496, 504, 512]
    out = {}
    for name in ("driving", "driving-decay"):
        out[name] = anytime_curves(torch, B, synth.named(name), stream, [(512, 640)], Kd, rows_d)
    Kp = [0, 1, 2, 4, 8, 16, 24, 32, 48, 64, 96, 128]
    rows_p = [0, 4, 8, 16, 24, 32, 40, 48, 56, 60, 62, 63, 64]
    # the non-residual alternative of Sec. III at NZ = 130 and 4160: same
    # cost per step, larger error at every budget
    out["paper"] = anytime_curves(torch, B, synth.named("paper"), stream,
                                  [(128, 4160), (128, 130), (128, 32), (64, 4160, "non-residual"),
                                   (64, 130, "non-residual")], Kp, rows_p)
    return out


def stack_summary(args, torch):
    """The stacked workload's budgets sweep, exact baseline and device
    factorisation time, for the default line (full record: --workload stack)."""
    out = bench_stack(args, torch, emit=False)
    return {"workload": out["config"]["workload"], "prepare_device_s": out["prepare_device_s"],
            "sweep": out["sweep"], "exact_baseline": out["exact_baseline"], "roofline": out["roofline"]}


def bench_stack(args, torch, emit=True):
    """The stacked workload: layer 1 D=4096 -> H=1024, layer 2 1024 -> 1024,
    T=32, one sequence, fp32, per-layer rank 1024, 75% pruning (NZ = 1280 and
    512), factorised on the device.  A step is one approx_lstm_run_stack at one
    pair of per-layer budgets; each layer is one input projection and one
    persistent recurrence.  The roofline counts both layers' algorithmic
    bytes (every term streamed once per timestep, the paper's accounting)."""
    from paper_1905_00689_amd import synth
    from paper_1905_00689_amd import binding as B
    dev = torch.device("cuda")
    wl = synth.named("stack")
    (W1, b1), (W2, b2) = wl.layers
    D, H, T, Bn = wl.D, wl.H, wl.T, wl.B
    rank = 1024
    t0 = time.time()
    m1 = B.approx_lstm_prepare(W1[:, :D], W1[:, D:], b1, D, H, rank, prune_ratio=0.75, groups=4,
                               flags=B.FLAG_DEVICE_FACTORISE)
    m2 = B.approx_lstm_prepare(W2[:, :H], W2[:, H:], b2, H, H, rank, prune_ratio=0.75, groups=4,
                               flags=B.FLAG_DEVICE_FACTORISE)
    prep_s = time.time() - t0
    progress(f"stack: both layers prepared on the device in {prep_s:.1f} s")
    nz1, nz2 = m1.info["nz"], m2.info["nz"]
    x = torch.from_numpy(wl.x).to(dev)
    stream = torch.cuda.current_stream()

    def timed(fn, steps, warmup):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps   # ms per step

    h = torch.empty((1, T, Bn, H), device=dev)
    sweep = {"K": [], "us_per_timestep": [], "timesteps_per_s": [], "hbm_frac": []}
    ms = bytes_step = None
    for k1, k2 in ((64, 64), (256, 256), (1024, 1024)):
        ms = timed(lambda: B.approx_lstm_run_stack([m1, m2], x, [(k1, k2)], h, stream=stream),
                   args.sweep_steps, 5)
        B.approx_lstm_check(m1)
        B.approx_lstm_check(m2)
        bytes_step = T * (algorithmic_bytes_per_timestep(4, H, nz1, D + H, k1, D, H, Bn, 1)
                          + algorithmic_bytes_per_timestep(4, H, nz2, 2 * H, k2, H, H, Bn, 1))
        sweep["K"].append([k1, k2])
        sweep["us_per_timestep"].append(round(ms * 1e3 / T, 4))
        sweep["timesteps_per_s"].append(round(T * Bn / (ms * 1e-3), 1))
        sweep["hbm_frac"].append(round(bytes_step / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4))
    achieved = bytes_step / (ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                "kernel": "one step at budgets (1024, 1024): per layer input_proj_kernel + progressive_lstm_kernel",
                "bytes_per_launch": bytes_step}
    # the exact (dense) two-layer LSTM on the same input, layer after layer
    e1 = B.approx_lstm_exact_prepare(W1[:, :D], W1[:, D:], b1, D, H)
    e2 = B.approx_lstm_exact_prepare(W2[:, :H], W2[:, H:], b2, H, H)
    h1 = torch.empty((T, Bn, H), device=dev)
    h2 = torch.empty((T, Bn, H), device=dev)

    def exact_step():
        B.approx_lstm_exact_run(e1, x, h1, stream=stream)
        B.approx_lstm_exact_run(e2, h1, h2, stream=stream)

    ms_exact = timed(exact_step, args.sweep_steps, 5)
    B.approx_lstm_exact_check(e1)
    B.approx_lstm_exact_check(e2)
    out = {
        "metric": "LSTM timesteps/sec at refinement budget K (and us/timestep vs K)",
        "value": round(T * Bn / (ms * 1e-3), 1), "unit": "timesteps/s", "n_gpus": 1, "steps": args.sweep_steps,
        "warmup": 5, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "stacked LSTM D=4096 -> H=1024 -> H=1024, T=32, B=1, per-layer rank 1024, "
                               f"75% pruning (NZ={nz1}, {nz2}), budgets (1024, 1024)",
                   "D": D, "H": H, "T": T, "batch": Bn, "rank": rank, "nz": [nz1, nz2], "K": [1024, 1024],
                   "groups": 4, "layers": 2},
        "us_per_timestep": round(ms * 1e3 / T, 4), "prepare_device_s": round(prep_s, 2), "sweep": sweep,
        "exact_baseline": {"us_per_timestep": round(ms_exact * 1e3 / T, 4),
                           "timesteps_per_s": round(T * Bn / (ms_exact * 1e-3), 1)},
        "roofline": roofline, "cpu_baseline": None,
    }
    if emit:
        print(json.dumps(out), flush=True)
    return out


def deadline_record(torch, name, steps=10):
    """One weights model of the deadline workload (D=2048, H=2048, T=64, 8
    sequences, per-gate rank 2048, 90% pruning, fp32), factorised on the
    device: fixed budgets timed, then both deadline modes at 5, 20 and 100 us
    per timestep, one K for the sequence (approx_lstm_run_deadline) and K_t
    chosen per timestep on the device (approx_lstm_run_anytime).  Each
    reports the budgets achieved, the measured step times and the output's
    error against the device's exact LSTM on the same input (see _qor)."""
    from paper_1905_00689_amd import synth
    from paper_1905_00689_amd import binding as B
    dev = torch.device("cuda")
    wl = synth.named(name)
    D, H, T, Bn = wl.D, wl.H, wl.T, wl.B
    rank = 2048
    t0 = time.time()
    m = B.approx_lstm_prepare(wl.W[:, :D], wl.W[:, D:], wl.b, D, H, rank, prune_ratio=0.9, groups=4,
                              flags=B.FLAG_DEVICE_FACTORISE)
    prep_s = time.time() - t0
    progress(f"{name}: prepared on the device in {prep_s:.1f} s")
    x = torch.from_numpy(wl.x).to(dev)
    stream = torch.cuda.current_stream()
    me = B.approx_lstm_exact_prepare(wl.W[:, :D], wl.W[:, D:], wl.b, D, H)
    href = torch.empty((T, Bn, H), device=dev)
    B.approx_lstm_exact_run(me, x, href, stream=stream)
    torch.cuda.synchronize()
    B.approx_lstm_exact_check(me)
    quality = _qor(synth.softmax_head(H).astype(np.float64), href.cpu().numpy().astype(np.float64))

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps   # ms per run

    h1 = torch.empty((1, T, Bn, H), device=dev)
    fixed = {"K": [], "us_per_timestep": [], "rel_err": [], "kl": []}
    for k in (0, 1, 16, 256, 1024, 2048):
        ms = timed(lambda: B.approx_lstm_run(m, x, [k], h1, stream=stream))
        B.approx_lstm_check(m)
        e, kl = quality(h1[0].cpu().numpy())
        fixed["K"].append(k)
        fixed["us_per_timestep"].append(round(ms * 1e3 / T, 3))
        fixed["rel_err"].append(_sig(e))
        fixed["kl"].append(_sig(kl))
    ms_exact = timed(lambda: B.approx_lstm_exact_run(me, x, href, stream=stream))

    modes = {}
    h = torch.empty((T, Bn, H), device=dev)
    for mode, fn in (("one_K", B.approx_lstm_run_deadline), ("anytime", B.approx_lstm_run_anytime)):
        rows = []
        for dl in (5.0, 20.0, 100.0):
            try:
                k, us = fn(m, x, dl, h, stream=stream)
            except B.ApproxLstmError as err:
                if err.status != B.ERR_DEADLINE_INFEASIBLE:
                    raise
                rows.append({"deadline_us": dl, "status": "infeasible", "detail": str(err).split(": ", 1)[-1]})
                continue
            e, kl = quality(h.cpu().numpy())
            rows.append({"deadline_us": dl, "status": "ok", "k_mean": round(float(np.mean(k)), 1),
                         "k_min": int(np.min(k)), "k_max": int(np.max(k)),
                         "step_us_mean": round(float(np.mean(us)), 3), "step_us_max": round(float(np.max(us)), 3),
                         "steps_within_deadline": round(float(np.mean(us <= dl)), 3),
                         "ends_within_schedule": round(float(np.mean(np.cumsum(us.astype(np.float64))
                                                                     <= dl * np.arange(1, len(us) + 1) + 1e-3)), 3),
                         "rel_err": _sig(e), "kl": _sig(kl)})
        modes[mode] = rows
    return {"weights": "gaussian" if name == "deadline" else "decaying spectrum", "nz": m.info["nz"],
            "prepare_device_s": round(prep_s, 2), "fixed_budgets": fixed,
            "exact_us_per_timestep": round(ms_exact * 1e3 / T, 3), "deadline_modes": modes}


NOTE_DEADLINE = ("errors against the device's exact LSTM; 'steps_within_deadline' is the share of timesteps "
                 "whose measured time met the deadline, 'ends_within_schedule' the share whose end came by "
                 "(t + 1) x deadline after the recurrence began (the anytime mode's target: a cheap step's "
                 "slack is spent on a later one)")


def deadline_summary(args, torch):
    """Both weights models of the deadline workload, for the default line."""
    return {"workload": "deadline: D=2048 H=2048 T=64 B=8, per-gate rank 2048, 90% pruning",
            "gaussian": deadline_record(torch, "deadline", steps=5),
            "decay": deadline_record(torch, "deadline-decay", steps=5),
            "note": NOTE_DEADLINE}


def bench_deadline(args, torch):
    """The deadline workload on Gaussian weights (flat spectrum: every budget
    short of full rank leaves a large error) and on decaying-spectrum weights
    (where the refinement order pays off)."""
    g = deadline_record(torch, "deadline")
    d = deadline_record(torch, "deadline-decay")
    T, Bn = 64, 8
    value = T * Bn / (g["fixed_budgets"]["us_per_timestep"][-1] * 1e-6 * T)
    out = {
        "metric": "deadline mode: achieved K, step time and error vs the exact LSTM at per-timestep deadlines",
        "value": round(value, 1), "unit": "timesteps/s at K=2048", "n_gpus": 1, "higher_is_better": True,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"deadline: D=2048 H=2048 T=64 B=8, per-gate rank 2048, 90% pruning (NZ={g['nz']})",
                   "D": 2048, "H": 2048, "T": T, "batch": Bn, "rank": 2048, "nz": g["nz"]},
        "gaussian": g, "decay": d,
        "note": NOTE_DEADLINE,
    }
    print(json.dumps(out), flush=True)


def time_prepare(spec, torch, synth, B):
    """Wall time of approx_lstm_prepare with the factorisation on the device
    (APPROX_LSTM_FLAG_DEVICE_FACTORISE) for a named synthetic workload."""
    name, rank, prune = spec.split(":")
    w = synth.named(name)
    torch.cuda.init()
    t0 = time.time()
    m = B.approx_lstm_prepare(w.W[:, :w.D], w.W[:, w.D:], w.b, w.D, w.H, int(rank), prune_ratio=float(prune),
                              flags=B.FLAG_DEVICE_FACTORISE)
    sec = time.time() - t0
    inf = m.info
    print(json.dumps({"prepare": f"device factorisation, {name} D={w.D} H={w.H} rank {rank} prune {prune}",
                      "seconds": round(sec, 3), "nz": inf["nz"], "eff_rank": inf["eff_rank"],
                      "unconverged_steps": inf["unconverged_steps"]}), flush=True)


def step_distribution(torch, step, stream, n):
    """Per-step times (ms) of n further steps, each between its own pair of
    events on the launch stream: median, p99 and max (the headline value
    comes from the bracketed total)."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    torch.cuda.synchronize()
    for e0, e1 in evs:
        e0.record(stream)
        step()
        e1.record(stream)
    torch.cuda.synchronize()
    t = np.sort([e0.elapsed_time(e1) for e0, e1 in evs])
    return {"steps": n, "median": round(float(np.median(t)), 5), "p99": round(float(t[min(n - 1, int(0.99 * n))]), 5),
            "max": round(float(t[-1]), 5)}


def mfma_flops_batched(G, D, H, T, Bp, K):
    """MFMA flops one batched run executes at budget K (dense zero-filled
    panels; rows, D, H padded to the 32-wide MFMA contraction, sequences to
    64): the x-projection once, then per timestep the h-projection and the U
    accumulation of all four gates."""
    r32 = lambda v: (v + 31) // 32 * 32
    rows = G * r32(K)
    xproj = 2 * rows * r32(D) * T * Bp
    hproj = 2 * rows * r32(H) * Bp
    accum = 2 * 4 * H * r32(K) * Bp
    return xproj + T * (hproj + accum)


def batched_summary(args, torch):
    """The batched workload's sweep (us per timestep and MFMA fraction at each
    budget) and its K=512 roofline, for the default line; the full record is
    `--workload batched`."""
    sub = argparse.Namespace(**vars(args))
    sub.K, sub.steps, sub.warmup, sub.prune, sub.no_cpu_baseline = 512, 30, 5, 0.75, True
    sub.sweep_steps = 30
    out = bench_batched(sub, torch, emit=False, step_dist=False)
    return {"workload": out["config"]["workload"], "us_per_timestep": out["us_per_timestep"],
            "timesteps_per_s": out["value"], "sweep": out["sweep"], "roofline": out["roofline"]}


def bench_batched(args, torch, emit=True, step_dist=True):
    """The batched workload: 256 independent driving-shaped sequences (D=2048,
    H=512, T=16), rank 512, 75% pruning, bf16 factors with fp32 accumulation
    on MFMA.  A step is one approx_lstm_run over the batch at budget K."""
    from paper_1905_00689_amd import synth
    from paper_1905_00689_amd import binding as B
    dev = torch.device("cuda")
    wl = synth.named("batched")
    D, H, T, Bn = wl.D, wl.H, wl.T, wl.B
    rank = 512
    t0 = time.time()
    m = B.approx_lstm_prepare(wl.W[:, :D], wl.W[:, D:], wl.b, D, H, rank, prune_ratio=args.prune, groups=4,
                              factor_dtype=1)
    prep_s = time.time() - t0
    info = m.info
    NZ, G, Rg = info["nz"], info["groups"], info["rows_per_group"]
    B.approx_lstm_reserve(m, T, Bn, 1)
    x = torch.from_numpy(wl.x).to(dev)
    h_out = torch.empty((1, T, Bn, H), device=dev)
    stream = torch.cuda.current_stream()
    Bp = (Bn + 63) // 64 * 64

    def timed(K, steps, warmup):
        for _ in range(warmup):
            B.approx_lstm_run(m, x, [K], h_out, stream=stream)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            B.approx_lstm_run(m, x, [K], h_out, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        B.approx_lstm_check(m)
        return e0.elapsed_time(e1) / steps

    K = args.K
    progress(f"driving prepared ({prep_s:.1f} s); timing K={K}")
    ms = timed(K, args.steps, args.warmup)
    dist = (step_distribution(torch, lambda: B.approx_lstm_run(m, x, [K], h_out, stream=stream), stream, args.steps)
            if step_dist else None)
    sweep = {"K": [], "us_per_timestep": [], "timesteps_per_s": [], "mfma_frac": []}
    for k in [int(v) for v in args.batched_sweep.split(",") if v]:
        msk = timed(k, args.sweep_steps, 5)
        sweep["K"].append(k)
        sweep["us_per_timestep"].append(round(msk * 1e3 / T, 4))
        sweep["timesteps_per_s"].append(round(T * Bn / (msk * 1e-3), 1))
        sweep["mfma_frac"].append(round(mfma_flops_batched(G, D, H, T, Bp, k) / (msk * 1e-3) / 1e12
                                        / MFMA_BF16_PEAK_TFLOPS, 4))
    flops = mfma_flops_batched(G, D, H, T, Bp, K)
    algo = T * algorithmic_flops_per_timestep(G, Rg, NZ, K, Bn)
    achieved = flops / (ms * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
                "traffic": measured_traffic("batched") if (K == 512 and abs(args.prune - 0.75) < 1e-9) else None,
                "kernel": "one step: batched_xproj_kernel + batched_persistent_kernel (T timesteps in one launch)",
                "flops_per_launch": flops, "algorithmic_flops_per_launch": algo,
                "algorithmic_tflops": round(algo / (ms * 1e-3) / 1e12, 2),
                "algorithmic_frac": round(algo / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)}
    cpu = None if args.no_cpu_baseline else cpu_baseline_batched(m, wl, K, args.cpu_seconds)
    out = {
        "metric": "LSTM timesteps/sec at refinement budget K (and us/timestep vs K)",
        "value": round(T * Bn / (ms * 1e-3), 1), "unit": "timesteps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"batched driving-shaped LSTM D=2048 H=512 T=16 B=256, per-gate rank 512, "
                               f"{int(args.prune * 100)}% pruning (NZ={NZ}), bf16 factors, fp32 accumulation, K={K}",
                   "D": D, "H": H, "T": T, "batch": Bn, "rank": rank, "nz": NZ, "K": K, "groups": G},
        "us_per_timestep": round(ms * 1e3 / T, 4), "step_ms": dist, "prepare_s": round(prep_s, 2),
        "sweep": sweep, "roofline": roofline, "cpu_baseline": cpu,
    }
    if emit:
        print(json.dumps(out), flush=True)
    return out


def cpu_baseline_batched(m, wl, K, seconds):
    """The float64 oracle (bf16 operand mode) on the library's exported terms,
    over the whole sequence for a sample of the batch, repeated for about
    `seconds`; the rate is timesteps of single sequences per second."""
    import oracle
    fac = exported_terms(m)
    threads = oracle_threads()
    sample = 8
    xs = wl.x[:, :sample]
    runs, t0 = 0, time.time()
    while True:
        oracle.run(fac, wl.b, xs, [K], operand_round="bf16")
        runs += 1
        el = time.time() - t0
        if el >= seconds or runs >= 10000:
            break
    ts = runs * wl.T * sample
    return {"value": round(ts / el, 2), "unit": "timesteps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"oracle.run (float64 NumPy, bf16 operand mode) over the full T={wl.T} sequence of "
                      f"{sample} of the {wl.B} sequences at K={K}, repeated {runs} times ({el:.1f} s), "
                      "on the library's exported terms"}


def exported_terms(m):
    """The library's stored terms as an oracle Factors object (timing only)."""
    from oracle.factorise import Factors
    from paper_1905_00689_amd import binding as B
    inf = m.info
    G, N, Rg, nz = inf["groups"], inf["rank"], inf["rows_per_group"], inf["nz"]
    sig = np.zeros((G, N)); U = np.zeros((G, N, Rg)); mask = np.zeros((G, N, nz), np.int64)
    vals = np.zeros((G, N, nz))
    for g in range(G):
        f = B.approx_lstm_get_factors(m, g)
        sig[g], U[g], mask[g], vals[g] = f["sigma"], f["u"], f["v_idx"], f["v_val"]
    return Factors(inf["input_size"], inf["hidden_size"], G, N, nz, sig, U, mask, vals,
                   np.zeros((G, N, 1)), np.array(inf["eff_rank"]), "bf16" if inf["factor_dtype"] else "f32")


def oracle_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:
        return os.cpu_count()


def blas_info():
    """The BLAS NumPy calls (library, version, threading layer, threads)."""
    try:
        from threadpoolctl import threadpool_info
        libs = [d for d in threadpool_info() if d.get("user_api") == "blas"]
        return [{"library": d.get("internal_api"), "version": d.get("version"),
                 "threading_layer": d.get("threading_layer"), "threads": d.get("num_threads"),
                 "file": os.path.basename(d.get("filepath", ""))} for d in libs]
    except Exception as exc:
        return [{"error": str(exc)}]


TRAFFIC_PROFILES = {
    "driving": ("driving_K512_p75_hbm_counters.md",
                ("kernels.hip", "kernels_pair.hip", "kernels.hpp", "device_common.hpp")),
    "batched": ("batched_K512_p75_hbm_counters.md", ("batched.hip", "kernels.hpp", "device_common.hpp")),
}


def kernel_sources_sha256(names):
    """sha256 over the named kernel sources, concatenated in order."""
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    h = hashlib.sha256()
    for n in names:
        h.update(open(os.path.join(root, "paper_1905_00689_amd", "csrc", n), "rb").read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per step from the committed rocprofv3 counter summary of the
    workload, if it was taken on the kernel sources as they are now (else
    None)."""
    root = os.path.dirname(os.path.abspath(__file__))
    prof_name, src_names = TRAFFIC_PROFILES[workload]
    prof = os.path.join(root, "profiles", prof_name)
    try:
        fields = dict(l.split(": ", 1) for l in open(prof).read().splitlines() if ": " in l and not l.startswith(" "))
        if fields.get("kernel_sources_sha256", "").strip() != kernel_sources_sha256(src_names):
            return None
        return int(fields["traffic_bytes_per_step"])
    except (OSError, KeyError, ValueError):
        return None


def copy_calibration(torch):
    """A plain device-to-device copy of 256 MiB, 5 times: its HBM counters per
    dispatch (read 256 MiB, write 256 MiB) calibrate FETCH_SIZE / WRITE_SIZE."""
    n = 64 << 20                                   # float32 elements = 256 MiB
    a = torch.ones(n, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 5
    print(json.dumps({"copy_bytes_each_way": 4 * n, "ms_per_copy": round(ms, 4),
                      "gbs_read_plus_write": round(8 * n / (ms * 1e-3) / 1e9, 1)}), flush=True)


def cpu_baseline(m, wl, K, seconds):
    """Time the float64 oracle's progressive run on the same workload: the
    whole T=16 sequence at budget K, repeated for about `seconds`.  The
    oracle runs on the library's exported terms (timing only: values do not
    change its cost)."""
    import oracle
    fac = exported_terms(m)
    threads = oracle_threads()
    def rate(fn, budget):
        runs, t0 = 0, time.time()
        while True:
            fn()
            runs += 1
            el = time.time() - t0
            if el >= budget or runs >= 10000:
                return runs * wl.T * wl.B / el, runs, el

    v, runs, el = rate(lambda: oracle.run(fac, wl.b, wl.x, [K]), seconds)
    single = exact = None
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            single, _, _ = rate(lambda: oracle.run(fac, wl.b, wl.x, [K]), seconds / 2)
    except Exception:
        pass
    exact, _, _ = rate(lambda: oracle.exact_lstm(wl.W, wl.b, wl.x), seconds / 2)
    return {"value": round(v, 2), "unit": "timesteps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"oracle.run (float64 NumPy) over the full T={wl.T} sequence at K={K}, "
                      f"repeated {runs} times ({el:.1f} s), on the library's exported terms",
            "single_thread_value": None if single is None else round(single, 2),
            "exact_lstm_value": round(exact, 2), "cpu_model": cpu_model(), "blas": blas_info(),
            "host_cpus": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0))}


def cpu_model():
    """The host CPU as /proc/cpuinfo names it: model name, vendor, family /
    model / stepping (the name alone can be a generic string in a VM)."""
    info = {}
    try:
        for line in open("/proc/cpuinfo"):
            if ":" not in line:
                continue
            k, v = (t.strip() for t in line.split(":", 1))
            if k in ("model name", "vendor_id", "cpu family", "model", "stepping", "cpu MHz", "cache size") \
                    and k not in info:
                info[k] = v
            if not line.strip():
                break
    except OSError:
        return None
    name = info.get("model name")
    return {"name": name, "vendor": info.get("vendor_id"), "family": info.get("cpu family"),
            "model": info.get("model"), "stepping": info.get("stepping"), "cache": info.get("cache size"),
            "mhz": info.get("cpu MHz")}


if __name__ == "__main__":
    main()
