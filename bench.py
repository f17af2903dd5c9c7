#!/usr/bin/env python3
"""Benchmark of the DSDE verification step on one MI355X.

One step = verification + KLD signal update + SL rule with the batch cap
(dsde_step, which is bit-identical to dsde_verify, dsde_kld_signal and
dsde_next_sl in sequence) over one batch of synthetic inputs already resident
in HBM (workload b256 by default: B=256, SL ~ U{1..8}, V=128256 bf16,
T = 0.7 / 1.0 alternating).  Input copies rotate between steps so that no
step finds its logits in the 256 MB last-level cache: two for b256 and the
larger workloads, as many as 512 MiB of logits need for the small ones (at
most 64).

Prints one JSON line: rows/s over all logit rows of the step (2N + B), the
algorithmic HBM rate, the roofline of the dominant kernel (the row-statistics
pass, timed with HIP events recorded by the library on the launch stream), and
the CPU oracle timed on the host as a baseline.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "verified logit rows/sec + achieved HBM GB/s (V=128256 bf16, B=256)"
PEAK_HBM_GBPS = 8000.0

# The paper's own numbers, quoted as context (not a target): it times no
# kernel of this path, only end-to-end serving latency (Table 3: mean
# completion time of 128 prompts, LLaMA-3.1-70B-Instruct target with
# LLaMA-3.2-1B-Instruct draft, on one server of 8x NVIDIA A100 80GB, vLLM 0.8.4
# in eager mode).
PAPER_CONTEXT = {
    "hardware": "8x NVIDIA A100 80GB, vLLM 0.8.4 (eager mode)",
    "workload": "LLaMA-3.1-70B-Instruct target, LLaMA-3.2-1B-Instruct draft, 128 prompts",
    "metric": "end-to-end mean latency, seconds (Table 3)",
    "temperature_0": {"autoregressive": 38.41, "static_opt": 13.44, "dsde": 13.97, "adaedl": 13.83},
    "temperature_1": {"autoregressive": 38.47, "static_opt": 18.02, "dsde": 19.19, "adaedl": 17.64},
    "note": "no kernel-level figure for the verification step exists in the paper; vs_baseline is null",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="b256")
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target CPU time of the oracle baseline")
    ap.add_argument("--settle-ms", type=float, default=300.0,
                    help="untimed steps run before the warm-up steps, in milliseconds of wall time")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-stream-ceiling", action="store_true")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM traffic of the row-statistics kernel (from rocprofv3 counters)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a streaming kernel of known size (for scaling the HBM counters)")
    return ap.parse_args()


def stats_kernel_name(esz, V):
    """The statistics kernel the library dispatches for this row layout (the
    bench's tensors are 16-byte aligned): the bf16 vector kernel in its form
    without the draft-entropy accumulator (the step asks for no entropy), else
    the generic one instantiated for the dtype and vector width."""
    if esz == 2:
        return "stats_kernel_bf16<false>" if V % 8 == 0 else "stats_kernel_generic<bf16, scalar>"
    return "stats_kernel_generic<fp32, vec4>" if V % 4 == 0 else "stats_kernel_generic<fp32, scalar>"


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(see the design notes on how the step would shard)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2509_01083_amd as dsde
    import workloads as W
    from paper_2509_01083_amd.profiling import kernel_source_hash, step_source_hash

    dsde.load()
    dev = torch.device("cuda:0")
    if args.workload == "shard8":
        print(json.dumps(run_shard(args, dev)), flush=True)
        return
    cfg = W.CONFIGS[args.workload]
    if args.workload == "loop":
        print(json.dumps(run_loop(args, cfg, dev)), flush=True)
        return
    sl = W.sample_sl(cfg, args.seed)
    copies = [W.make_step(cfg, seed=args.seed, device=dev, sl=sl)]
    step_bytes = (copies[0].target.numel() + copies[0].draft.numel()) * copies[0].target.element_size()
    n_copies = max(2, min(64, -(-(512 << 20) // step_bytes)))
    copies += [W.make_step(cfg, seed=args.seed + i, device=dev, sl=sl) for i in range(1, n_copies)]
    st = W.make_signal_state(cfg, seed=args.seed, device=dev)
    s0 = copies[0]
    B, N, V, k_max = s0.B, s0.N, s0.V, s0.k_max
    esz = 2 if s0.target.dtype == torch.bfloat16 else 4
    ws = dsde.new_workspace(B, N, V, k_max, device=dev)
    outs = [None] * n_copies

    def one_step(i):
        c = i % n_copies
        s = copies[c]
        outs[c] = dsde.step(s.target, s.draft, s.sl, s.cu_sl, s.draft_tokens, s.temperature, s.u_acc, s.u_res,
                            k_max, st.hist, st.head, st.count, st.sl_max, out=outs[c], workspace=ws)

    # settle: the GPU runs the step untimed for a fixed span of wall time
    # before the warm-up steps, so that the timed regions see the clocks of
    # sustained work (a fresh box started from idle ran the first few
    # milliseconds of steps measurably slower)
    settle_steps, t_settle = 0, time.perf_counter()
    while (time.perf_counter() - t_settle) * 1e3 < args.settle_ms:
        for _ in range(16):
            one_step(settle_steps)
            settle_steps += 1
        torch.cuda.synchronize()
    settle_s = time.perf_counter() - t_settle
    for i in range(args.warmup):
        one_step(settle_steps + i)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    base = settle_steps + args.warmup

    # timed region: K whole steps between two events on the launch stream
    step_ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    step_ev[0].record(stream)
    for i in range(args.steps):
        one_step(base + i)
    step_ev[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # second timed region of K steps in which the library attaches a pair of
    # HIP events to the completions of the set-up and row-statistics
    # dispatches (the interval is the statistics kernel alone); kept apart
    # from the headline region in case the events cost stream time.  The
    # events skip the system-scope fence of an ordinary event record.
    ev = [(HipEvent(), HipEvent()) for _ in range(args.steps)]
    ev_region = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    torch.cuda.synchronize()
    ev_region[0].record(stream)
    for i in range(args.steps):
        dsde.set_profile_events(ev[i][0].handle, ev[i][1].handle)
        one_step(base + args.steps + i)
    ev_region[1].record(stream)
    torch.cuda.synchronize()
    dsde.set_profile_events(None, None)

    gpu_ms = step_ev[0].elapsed_time(step_ev[1])
    ms_per_step = gpu_ms / args.steps
    k1_ms = float(np.mean([a.elapsed_ms(b) for a, b in ev]))
    for a_, b_ in ev:
        a_.destroy()
        b_.destroy()
    rows = 2 * N + B
    last = (base + 2 * args.steps - 1) % n_copies
    acc = outs[last]["accepted"].cpu().numpy()
    sls = s0.sl.cpu().numpy()
    b_full = int((acc == sls).sum())
    io_bytes = 4 * (3 * N + 2 * B + B * (k_max + 1)) + 8 * B * cfg["W"]
    alg_bytes = (2 * N + b_full) * V * esz + io_bytes
    k1_bytes = 2 * N * V * esz  # every drafted pair read once
    k1_gbps = k1_bytes / (k1_ms * 1e-3) / 1e9

    traffic, step_traffic = None, None
    if os.path.exists(args.traffic):
        with open(args.traffic) as f:
            tr = json.load(f)
        if tr.get("workload") == args.workload and tr.get("kernel_source_hash") == kernel_source_hash():
            traffic = tr.get("bytes_per_launch")
        if tr.get("workload") == args.workload and tr.get("step_source_hash") == step_source_hash() \
                and tr.get("step_bytes"):
            sb = tr["step_bytes"]
            step_traffic = {"bytes": sb, "gbps": sb / (ms_per_step * 1e-3) / 1e9,
                            "frac_of_peak": sb / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBPS,
                            "ratio_to_algorithmic": sb / alg_bytes,
                            "per_kernel": {k: v["fetch_bytes"] + v["write_bytes"]
                                           for k, v in tr["step_kernels"].items()},
                            "source": "rocprofv3 FETCH_SIZE + WRITE_SIZE per kernel, scaled by a streaming "
                                      "kernel of known size; one launch of each step kernel"}

    result = {
        "metric": METRIC,
        "value": rows / (ms_per_step * 1e-3),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if esz == 2 else "fp32",
        "data": "synthetic",
        "config": {"workload": args.workload, "B": B, "N": N, "V": V, "rows_per_step": rows, "k_max": k_max,
                   "logit_bytes_per_step": rows * V * esz, "seed": args.seed, "input_copies": n_copies},
        "positions_per_s": N / (ms_per_step * 1e-3),
        "hbm_gbps_algorithmic": alg_bytes / (ms_per_step * 1e-3) / 1e9,
        "hbm_frac_algorithmic": alg_bytes / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBPS,
        "wall_ms_per_step": wall * 1e3 / args.steps,
        "ms_per_step_kernel_events": ev_region[0].elapsed_time(ev_region[1]) / args.steps,
        "b_full": b_full,
        "algorithmic_bytes_per_step": alg_bytes,
        "step_traffic": step_traffic,
        "settle": {"steps": settle_steps, "seconds": settle_s,
                   "note": "untimed steps before the warm-up steps (fixed span of wall time)"},
        "roofline": {"bound": "hbm", "kernel": stats_kernel_name(esz, V), "achieved": k1_gbps, "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": k1_gbps / PEAK_HBM_GBPS, "traffic": traffic,
                     "kernel_ms": k1_ms, "algorithmic_bytes": k1_bytes},
        "cpu_baseline": None,
    }

    # streaming-read ceiling of this GPU: the library's read-reduce probe over
    # 4 GiB (16x the last-level cache), and over as many bytes as one launch of
    # the statistics kernel reads (the same launch-size ramp-up and tail), each
    # timed with the same fence-free events
    if not args.no_stream_ceiling:
        def probe(nbytes, reps):
            buf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
            acc = torch.empty(-(-nbytes // 32768), dtype=torch.int32, device=dev)
            for _ in range(2):
                dsde.stream_read(buf, acc)
            e0, e1 = HipEvent(), HipEvent()
            torch.cuda.synchronize()
            _record(e0, stream)
            for _ in range(reps):
                dsde.stream_read(buf, acc)
            _record(e1, stream)
            torch.cuda.synchronize()
            gbps = reps * nbytes / (e0.elapsed_ms(e1) * 1e-3) / 1e9
            e0.destroy()
            e1.destroy()
            del buf, acc
            return gbps
        ceil_gbps = probe(4 << 30, 10)
        same = k1_bytes // 32768 * 32768
        same_gbps = probe(same, 50)
        result["stream_read_ceiling"] = {"gbps": ceil_gbps, "bytes": 4 << 30, "launches": 10,
                                         "same_bytes_gbps": same_gbps, "same_bytes": same, "same_launches": 50}
        result["roofline"]["frac_of_stream_ceiling"] = k1_gbps / ceil_gbps
        result["roofline"]["frac_of_same_bytes_read"] = k1_gbps / same_gbps

    result["straggler"] = straggler_report(outs[last], k_max)

    if not args.no_cpu_baseline:
        result["cpu_baseline"], result["parity"] = cpu_baseline(copies[last], outs[last], st, args.cpu_seconds)
        result["cpu_baseline"]["gpu_speedup"] = result["value"] / result["cpu_baseline"]["value"]
    result["paper_context"] = PAPER_CONTEXT
    if args.copy_calibration:
        # a plain streaming kernel of known size for scaling the HBM counters:
        # bitwise_not over 2^28 int32 reads 1 GiB and writes 1 GiB
        n = 1 << 28
        src = torch.zeros(n, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.bitwise_not(src, out=dst)
        torch.cuda.synchronize()
        result["copy_calibration"] = {"kernel": "bitwise_not", "read_bytes": 4 * n, "write_bytes": 4 * n,
                                      "launches": 3}
    print(json.dumps(result), flush=True)


def _record(ev, stream):
    """hipEventRecord of a HipEvent on a torch stream."""
    import ctypes
    HipEvent._hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    if HipEvent._hip.hipEventRecord(ev.handle, ctypes.c_void_p(stream.cuda_stream)) != 0:
        raise RuntimeError("hipEventRecord failed")


def straggler_report(out, sl_hi, sl_min=2.0):
    """Next-step SLs with and without the batch cap (Sec. 3.3): the largest SL,
    the sum, and the padded-slot waste B * max - sum of a batch padded to its
    longest sequence (the quantity the cap shrinks)."""
    import numpy as np
    hat = out["sl_hat"].cpu().numpy().astype(np.float64)
    capped = out["sl_next"].cpu().numpy().astype(np.int64)
    ok = np.isfinite(hat)
    lo = int(np.ceil(sl_min))
    uncapped = np.where(ok, np.clip(np.floor(hat + 0.5), lo, sl_hi), lo).astype(np.int64)
    B = len(capped)
    rep = {"sl_cap": float(out["sl_cap"].cpu().numpy()[0])}
    for name, v in (("with_cap", capped), ("without_cap", uncapped)):
        rep[name] = {"max": int(v.max()), "sum": int(v.sum()), "mean": float(v.mean()),
                     "padded_waste": int(B * v.max() - v.sum())}
    return rep


def run_loop(args, cfg, dev):
    """The controller loop (B = 1024, V = 128256): every step's SLs are the
    previous step's decisions (dsde_step's sl_next), the ring starts empty and
    carries across steps, the per-sequence draft noise sigma follows its
    seeded reflected random walk, and every step gets fresh seeded logits,
    drafted tokens and uniforms, generated on the GPU before the step
    (untimed).  Each dsde_step is timed by its own pair of events, after a
    synchronisation, so the times are of the step alone."""
    import numpy as np
    import torch

    import paper_2509_01083_amd as dsde
    import workloads as W
    B, V, k_max = cfg["B"], cfg["V"], cfg["k_max"]
    steps = args.steps
    st = W.make_signal_state(cfg, seed=args.seed, device=dev)
    ws = dsde.new_workspace(B, B * k_max, V, k_max, device=dev)
    sl = W.sample_sl(cfg, args.seed)
    sigma = W.initial_sigma(cfg, args.seed)
    times, mean_sl, caps, min_branch, sigma_mean, rows_total, bytes_total = [], [], [], [], [], 0, 0
    evs = (HipEvent(), HipEvent())
    stream = torch.cuda.current_stream()
    esz = 2 if cfg["dtype"] == "bf16" else 4
    t_wall = time.perf_counter()
    for t in range(args.warmup + steps):
        step = W.make_step(cfg, seed=args.seed, device=dev, step=t, sl=sl, sigma=sigma)
        N = step.N
        torch.cuda.synchronize()
        _record(evs[0], stream)
        out = dsde.step(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                        step.u_acc, step.u_res, k_max, st.hist, st.head, st.count, st.sl_max, workspace=ws)
        _record(evs[1], stream)
        torch.cuda.synchronize()
        if t >= args.warmup:
            times.append(evs[0].elapsed_ms(evs[1]))
            mean_sl.append(float(sl.mean()))
            caps.append(float(out["sl_cap"].cpu().numpy()[0]))
            hat = out["sl_hat"].cpu().numpy()
            min_branch.append(float(np.mean(hat <= 2.0)))
            sigma_mean.append(float(sigma.mean()))
            rows_total += 2 * N + B
            bytes_total += 2 * N * V * esz
        sl = out["sl_next"].cpu().numpy().astype(np.int32)
        sigma = W.walk_sigma(sigma, cfg, args.seed, t)
        del step, out
        if t % 20 == 0:
            print(f"[loop] step {t}: N={N} next mean SL {sl.mean():.2f} ({time.perf_counter() - t_wall:.0f} s)",
                  file=sys.stderr, flush=True)
    evs[0].destroy()
    evs[1].destroy()
    tms = np.asarray(times)
    total_s = tms.sum() * 1e-3
    return {
        "metric": METRIC, "value": rows_total / total_s, "unit": "rows/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": float(tms.mean()), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if esz == 2 else "fp32", "data": "synthetic",
        "config": {"workload": "loop", "B": B, "V": V, "k_max": k_max, "W": cfg["W"], "seed": args.seed},
        "paper_context": PAPER_CONTEXT,
        "loop": {"ms_per_step": {"mean": float(tms.mean()), "median": float(np.median(tms)),
                                 "p95": float(np.percentile(tms, 95)), "min": float(tms.min()),
                                 "max": float(tms.max())},
                 "drafted_pair_gbps": bytes_total / total_s / 1e9,
                 "mean_sl": {"first": mean_sl[0], "last": mean_sl[-1], "mean": float(np.mean(mean_sl))},
                 "sl_cap": {"first": caps[0], "last": caps[-1], "mean": float(np.mean(caps)),
                            "min": float(np.min(caps)), "max": float(np.max(caps))},
                 "fraction_in_sl_min_branch": float(np.mean(min_branch)),
                 "sigma_mean": {"first": sigma_mean[0], "last": sigma_mean[-1]},
                 "trajectory_every_10_steps": {"mean_sl": [round(x, 3) for x in mean_sl[::10]],
                                               "sl_cap": [round(x, 3) for x in caps[::10]],
                                               "fraction_in_sl_min_branch": [round(x, 3)
                                                                             for x in min_branch[::10]],
                                               "ms": [round(float(x), 4) for x in tms[::10]]},
                 "inputs": "fresh seeded logits, drafted tokens and uniforms every step (generated on the GPU, "
                           "untimed), per-sequence draft noise sigma on a seeded reflected random walk in "
                           "[0.2, 4], SLs from the previous step's decisions, ring empty at the start",
                 "note": "each step timed alone between two events"},
    }


def run_shard(args, dev, G=8):
    """One GPU's share of the b256 step with the vocabulary split eight ways:
    shard 0's four calls on its 16,032-column slices (statistics, acceptance
    from the gathered partials with the signal update and the SL rule fused
    behind it, draw mass, draw).  The other shards'
    contributions to the two exchanges are computed before the timed region
    (on this GPU, with the same calls); the exchanges themselves (RCCL
    all-gathers) are not part of the measurement."""
    import numpy as np
    import torch

    import paper_2509_01083_amd as dsde
    import workloads as W
    dsde.load()
    cfg = W.CONFIGS["b256"]
    sl = W.sample_sl(cfg, args.seed)
    copies = [W.make_step(cfg, seed=args.seed + i, device=dev, sl=sl) for i in range(2)]
    st = W.make_signal_state(cfg, seed=args.seed, device=dev)
    s0 = copies[0]
    B, N, V, k_max = s0.B, s0.N, s0.V, s0.k_max
    esz = 2 if s0.target.dtype == torch.bfloat16 else 4
    slices = dsde.slice_bounds(V, G)
    v0, v1 = slices[0]
    Vs = v1 - v0
    ws = dsde.new_shard_workspace(B, N, Vs, k_max, device=dev)
    prep = []
    for s in copies:
        full = dsde.verify_sharded(s.target, s.draft, s.sl, s.cu_sl, s.draft_tokens, s.temperature, s.u_acc,
                                   s.u_res, k_max, slices)
        prep.append(dict(step=s, t=s.target[:, v0:v1].contiguous(), d=s.draft[:, v0:v1].contiguous(),
                         parts=full["parts"].clone(), masses=full["masses"].clone(),
                         err=torch.empty(B, dtype=torch.int32, device=dev), out=None,
                         drawn=torch.empty(B, dtype=torch.int32, device=dev), ref_tokens=full["tokens"].clone(),
                         ref_accepted=full["accepted"].clone()))
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]

    def one(i, timed=False):
        p = prep[i % 2]
        s = p["step"]
        if timed:
            ev[0].record()
        dsde.shard_stats(p["t"], p["d"], v0, V, s.sl, s.cu_sl, s.draft_tokens, s.temperature, k_max, ws,
                         part=p["parts"][0], seq_err=p["err"])
        if timed:
            ev[1].record()
        p["out"] = dsde.shard_accept_step(p["parts"], V, s.sl, s.cu_sl, s.draft_tokens, s.temperature, s.u_acc,
                                          s.u_res, k_max, p["err"], st.hist, st.head, st.count, st.sl_max,
                                          out=p["out"])
        if timed:
            ev[2].record()
        dsde.shard_draw_mass(p["t"], p["d"], v0, p["parts"][0], p["out"]["jobs"], k_max, ws, mass=p["masses"][0])
        if timed:
            ev[3].record()
        dsde.shard_draw_pick(0, p["masses"], p["t"], p["d"], v0, p["out"]["jobs"], k_max, p["out"]["accepted"],
                             p["out"]["tokens"], p["err"], ws, drawn=p["drawn"])
        if timed:
            ev[4].record()

    for i in range(args.warmup):
        one(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        one(args.warmup + i)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    # per-call split from a second region with events between the calls
    split = np.zeros(4)
    for i in range(args.steps):
        one(args.warmup + args.steps + i, timed=True)
        torch.cuda.synchronize()
        split += [ev[k].elapsed_time(ev[k + 1]) for k in range(4)]
    split /= args.steps
    # shard 0's decisions agree with the run of all shards: the accepted counts,
    # and the whole token rows of the sequences whose token shard 0 drew
    p = prep[(args.warmup + 2 * args.steps - 1) % 2]
    own = p["drawn"] >= 0
    agree = bool(torch.equal(p["out"]["accepted"], p["ref_accepted"]) and
                 torch.equal(p["out"]["tokens"][own], p["ref_tokens"][own]))
    rows = 2 * N + B
    return {
        "metric": METRIC, "value": rows / (ms * 1e-3), "unit": "rows/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if esz == 2 else "fp32", "data": "synthetic",
        "config": {"workload": "shard8", "B": B, "N": N, "V": V, "shard": 0, "shards": len(slices),
                   "V_shard": Vs, "k_max": k_max, "seed": args.seed},
        "note": "rows/s counts one shard's slices of the step's 2N+B rows; exchanges excluded",
        "shard_bytes_per_step": rows * Vs * esz,
        "shard_gbps_rows": rows * Vs * esz / (ms * 1e-3) / 1e9,
        "ms_per_call": {"stats": split[0], "accept_signal_sl": split[1], "draw_mass": split[2],
                        "draw_pick": split[3]},
        "draws_by_this_shard": int(own.sum()),
        "decisions_match_all_shards_run": agree,
    }


class HipEvent:
    """A timing HIP event without the system-scope fence (hipEventDisableSystemFence)."""
    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        import ctypes
        if HipEvent._hip is None:
            # the HIP runtime this process already uses (torch's), never a second copy
            paths = [ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64.so" in ln]
            if not paths:
                raise RuntimeError("the HIP runtime is not loaded")
            HipEvent._hip = ctypes.CDLL(paths[0])
            HipEvent._hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            HipEvent._hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                          ctypes.c_void_p]
            HipEvent._hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        h = ctypes.c_void_p()
        if HipEvent._hip.hipEventCreateWithFlags(ctypes.byref(h), self.DISABLE_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")
        self.handle = h.value

    def elapsed_ms(self, stop):
        import ctypes
        ms = ctypes.c_float()
        if HipEvent._hip.hipEventElapsedTime(ctypes.byref(ms), self.handle, stop.handle) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self):
        HipEvent._hip.hipEventDestroy(self.handle)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cgroup_cpu_limit():
    """CPUs the process's cgroup may use per period (cpu.max), None when unlimited or unknown."""
    try:
        with open("/sys/fs/cgroup/cpu.max") as f:
            quota, period = f.read().split()[:2]
        return None if quota == "max" else float(quota) / float(period)
    except (OSError, ValueError):
        return None


KLD_REL, KLD_ABS = 1e-4, 1e-7  # the KLD comparison rule of the parity tests


def cpu_baseline(step, out, st, seconds):
    """The oracle, as it stands, on the host: whole steps (verify, signal update,
    SL rule) with as many threads as the host has logical CPUs (what
    std::thread::hardware_concurrency reports), repeated until about
    ``seconds`` have passed; then one more verify on a single thread.  Also
    checks the GPU's last step against it."""
    import numpy as np

    import oracle
    import workloads as W
    host = W.host_arrays(step)
    hist = st.hist.cpu().numpy()
    head = st.head.cpu().numpy()
    count = st.count.cpu().numpy()
    smax = st.sl_max.cpu().numpy().astype(np.float64)
    hw = os.cpu_count() or 1
    usable = len(os.sched_getaffinity(0))
    threads = hw
    t0 = time.perf_counter()
    n = 0
    ref = None
    while True:
        ref = oracle.verify(**host, n_threads=threads)
        sig = oracle.kld_signal(host["sl"], host["cu_sl"], ref["kld"], hist, head, count)
        oracle.next_sl(sig["sf"], sig["wvir"], smax, 2.0, step.k_max)
        n += 1
        if time.perf_counter() - t0 >= seconds or n >= 20:
            break
    dt = (time.perf_counter() - t0) / n
    rows = 2 * int(host["cu_sl"][-1]) + len(host["sl"])
    # one more step of the oracle's verify on a single thread (the signal update
    # and SL rule are a few microseconds), for the per-core rate
    t1 = time.perf_counter()
    oracle.verify(**host, n_threads=1)
    dt1 = time.perf_counter() - t1
    # parity of the timed GPU step against the oracle (ties excluded)
    acc = out["accepted"].cpu().numpy()
    tok = out["tokens"].cpu().numpy()
    ok = (ref["seq_err"] == 0) & (ref["acc_tie"] == 0) & (ref["cdf_tie"] == 0)
    mism = int((ok & ((acc != ref["accepted"]) | (tok != ref["tokens"]).any(axis=1))).sum())
    kg = out["kld"].cpu().numpy().astype(np.float64)
    fine = np.repeat(ref["seq_err"] == 0, host["sl"])
    dk = np.abs(kg - ref["kld"])[fine]
    kr = np.abs(ref["kld"])[fine]
    cpu = {"value": rows / dt, "unit": "rows/s", "cores": threads, "kind": "oracle",
           "sample": f"the full step (verify + signal + SL rule; B={len(host['sl'])}, {rows} logit rows, "
                     f"V={host['V']}), {n} repetition(s), {threads} threads, fp64",
           "seconds_per_step": dt, "threads": threads, "host_logical_cpus": hw, "usable_cpus": usable,
           "cgroup_cpu_limit": cgroup_cpu_limit(), "cpu_model": cpu_model(),
           "single_thread": {"value": rows / dt1, "unit": "rows/s", "seconds_per_step": dt1, "threads": 1}}
    parity = {"compared": int(ok.sum()), "ties": int((ref["acc_tie"] | ref["cdf_tie"]).sum()),
              "mismatches": mism,
              "kld_max_abs_err": float(dk.max()) if dk.size else 0.0,
              "kld_max_rel_err": float((dk / np.maximum(kr, 1e-12)).max()) if dk.size else 0.0,
              "kld_err_over_tolerance": float((dk / (KLD_REL * kr + KLD_ABS)).max()) if dk.size else 0.0,
              "kld_tolerance": f"{KLD_REL:g} * |ref| + {KLD_ABS:g}"}
    return cpu, parity


if __name__ == "__main__":
    main()
