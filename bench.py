#!/usr/bin/env python3
"""Benchmark of the per-micro-step MoE expert layer on one MI355X.

Workload: the Qwen3-30B-A3B-shaped EP=8 rank share in the policy-update
stage (T=16384 tokens, d=2048, F=768, E=128, top-8, 16 hosted experts + 4
replica slots, 16 micro-steps with independently jittered routing). One
step = one micro-step through every step of the path:

  histogram + assign_replicas (one call) -> permute -> gate/up (+SwiGLU) -> down
  -> combine -> combine_bwd -> down dgrad (+SwiGLU') -> gate/up dgrad
  -> gate/up wgrad -> down wgrad -> permute_bwd

The weight-gradient GEMMs of every group of 8 micro-steps (--wgrad-group)
run as one launch pair over the group's rows after its last micro-step, on
a third stream, while the next group's micro-steps run: the fp32 gradients
are read and written once per group instead of once per micro-step (the
fp32 accumulation over micro-steps of App. A.4; the operands stay resident
in a ring of 17 buffer sets). The streams are not joined at the end of a
micro-step: the next micro-step's dispatch and forward start on the other
activation set. The combine and permute_bwd (whose outputs feed nothing
later in the micro-step) run on a second stream, and so does the next
micro-step's histogram + replica split, beside this micro-step's combine,
so that the next micro-step starts with its permute right after the gate/up
dgrad. --wgrad-group 1 gives every micro-step its own weight gradients on
the second stream, each beside the data-gradient GEMM that does not feed
it; --no-pipeline joins the streams after every micro-step; --no-overlap
runs all phases on one stream; --side-gathers 1 keeps the combine, 0 also
permute_bwd, on the main stream; --no-early-hist runs each histogram at
the start of its micro-step on the main stream.

All inputs are resident in HBM before timing. A first pass brackets every
ABI call with HIP events on the stream it runs on, one kernel after
another, for every phase's own duration; the largest single-launch phase is
the dominant kernel. In the timed region only that kernel's calls carry
events (events around every call would add about 80 us per step); their
average duration gives the roofline line. The fp64 CPU oracle is timed on
one micro-step as the CPU baseline.

    python bench.py [--gpus 1] [--steps 32] [--warmup 16] [--no-cpu-baseline] [--no-overlap] [--no-pipeline] [--no-split]
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

# The CPU baseline's BLAS threads, fixed before numpy is first imported: the
# host's thread budget (OMP_NUM_THREADS where the machine sets one, else
# every CPU this process may run on).
AFFINITY_CPUS = len(os.sched_getaffinity(0))
os.environ.setdefault("OPENBLAS_NUM_THREADS", os.environ.get("OMP_NUM_THREADS", str(AFFINITY_CPUS)))

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "grouped-FFN TFLOP/s & % bf16 MFMA peak; permute+combine GB/s; tokens/s per micro-step"

# phases that are exactly one kernel launch (candidates for the roofline line)
SINGLE_LAUNCH = {"gate_up_fwd", "down_fwd", "combine", "combine_bwd", "down_dgrad",
                 "gate_up_dgrad", "permute_bwd"}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--micro-steps", type=int, default=16, help="distinct micro-steps cycled through")
    ap.add_argument("--no-planner", action="store_true", help="skip the planner report")
    ap.add_argument("--no-cache-report", action="store_true",
                    help="skip the warm- vs cold-cache report (one micro-step at a time, one stream)")
    ap.add_argument("--no-transfer", action="store_true", help="skip the transfer-engine report")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the per-phase report of the Mixtral-8x7B and DeepSeek-V3 rank shares")
    ap.add_argument("--no-reference-peaks", action="store_true",
                    help="skip the measured square-GEMM and copy peaks reported beside the nominal ones")
    ap.add_argument("--no-split", action="store_true",
                    help="run the row GEMMs without the workspace (no K split of a partial last round of tiles)")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="join the two streams at the end of every micro-step instead of letting the next "
                         "micro-step's forward start while this one's weight gradients run")
    ap.add_argument("--fwd-after-side", action="store_true",
                    help="pipelined: the gate/up forward waits for the previous micro-step's second-stream work")
    ap.add_argument("--side-gathers", type=int, default=2, choices=(0, 1, 2),
                    help="with overlap: run permute_bwd (1), and also the combine (2, the default), on the second "
                         "stream; 0 keeps both on the main stream")
    ap.add_argument("--no-early-hist", action="store_true",
                    help="pipelined: run each micro-step's histogram + replica split at its start on the main "
                         "stream instead of on the second stream beside the previous micro-step's combine")
    ap.add_argument("--wgrad-group", type=int, default=8,
                    help="micro-steps per weight-gradient launch pair (their fp32 read-modify-write of dW "
                         "is shared; 1: every micro-step its own, beside its data-gradient GEMMs)")
    ap.add_argument("--no-overlap", action="store_true",
                    help="run the weight-gradient GEMMs on the main stream instead of beside the data gradients")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run three plain 1 GiB device copies (reference for HBM byte counters)")
    ap.add_argument("--counters-pass", action="store_true",
                    help="only run each micro-step twice in the benchmark's schedule (for rocprofv3 --pmc runs)")
    ap.add_argument("--summarize-counters", metavar="DIR",
                    help="turn DIR/{fetch,write,copy_fetch,copy_write}.csv (rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE "
                         "of a --counters-pass and a --copy-calibration run) and DIR/pass.json (the counters "
                         "pass's output) into the per-kernel traffic record profiles/traffic_qwen3_share.json "
                         "and print its table")
    return ap.parse_args()


def copy_calibration() -> int:
    """Three device copies of 1 GiB: a kernel whose HBM bytes are known, so
    that FETCH_SIZE / WRITE_SIZE counter readings can be scaled to bytes."""
    import torch
    x = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    x.fill_(1)
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print("copied 3 x 1 GiB", flush=True)
    return 0


def main() -> int:
    args = parse()
    if args.copy_calibration:
        return copy_calibration()
    if args.summarize_counters:
        return summarize_counters(args.summarize_counters)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU's share of the expert layer; --gpus {args.gpus} "
              f"(WORLD_SIZE={world}) is not supported: the multi-GPU path (EP All-to-All over xGMI) "
              "is not implemented here", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2606_11867_amd import _lib, api
    from paper_2606_11867_amd.hip_events import Event
    from paper_2606_11867_amd.policy_update import PHASES, MicroStep, PolicyUpdate
    from workload import make_workload
    from workload import accounting as acc

    lib = _lib.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t0 = time.time()
    w = make_workload("qwen3-30b-a3b-ep8-policy-update")
    spec = w.spec
    n_micro = min(args.micro_steps, len(w.micro))
    T, K, d, F, E = spec.T, spec.K, spec.d, spec.F, spec.E
    bf = torch.bfloat16

    def dv(a, dt=bf):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev).to(dt)

    # ---- resident inputs: routing, plans, activations, upstream grads, weights
    local = w.micro[0].plan.local_experts
    gu_h, dn_h = w.weights(w.micro[0].plan)
    gu, dn = dv(gu_h), dv(dn_h)
    G = int(len(local))
    mss = []
    for i in range(n_micro):
        m = w.micro[i]
        assert np.array_equal(m.plan.local_experts, local)
        mss.append(MicroStep(ids=torch.from_numpy(m.ids).to(dev), gates=torch.from_numpy(m.gates).to(dev),
                             x=dv(w.x(i)), dy=dv(w.dy(i)), plan=api.DevicePlan.from_host(m.plan, dev)))
    S_max = max(ms.S for ms in mss)
    # buffers, workspaces and the two streams of the benchmark's schedule
    M = args.wgrad_group  # a last incomplete group is launched by pu.finish(), inside the timed region
    pu = PolicyUpdate(T, K, d, F, E, G, S_max, gu, dn, dev, split=not args.no_split, wgrad_group=M)
    stream = pu.main
    setup_s = time.time() - t0

    def run_step(i, ev=None, overlap=False, pipelined=False, last=None):
        # last: the index of the last micro-step of this run (early_hist
        # launches the next micro-step's histogram only if there is one)
        nxt = mss[(i + 1) % n_micro] if last is not None and i < last else None
        pu.run(i, mss[i % n_micro], ev, overlap, pipelined, args.side_gathers, args.fwd_after_side,
               next_ms=nxt, early_hist=not args.no_early_hist)

    # ---- realised per-micro-step sizes (read back once, outside the timed region)
    Ns, Gs = [], []
    for i in range(n_micro):
        run_step(i)
        torch.cuda.synchronize()
        S = mss[i].S
        buf = pu.set_of(i, pipelined=False)
        sc = buf["slot_count"][:S].cpu().numpy()
        Ns.append(int(buf["slot_offset"][S].item()))
        gidx = mss[i].plan.slot_gidx.cpu().numpy()
        Gs.append(int(len(set(gidx[sc > 0].tolist()))))
    pu.finish()

    if args.counters_pass:
        # after the one-stream pass above, each micro-step twice in the timed
        # region's schedule: every micro-step is dispatched three times, so
        # per-dispatch counters average over the 16 micro-steps evenly
        pu.start()
        for r in range(2):
            for i in range(n_micro):
                run_step(r * n_micro + i, overlap=not args.no_overlap, pipelined=not args.no_pipeline,
                         last=2 * n_micro - 1)
        pu.finish()
        torch.cuda.synchronize()
        print(json.dumps({"counters_pass": {"micro_steps": n_micro, "dispatches_per_micro_step": 3, "N": Ns,
                                            "G": Gs, "T": T, "K": K, "d": d, "F": F, "wgrad_group": M}}),
              flush=True)
        return 0

    overlap = not args.no_overlap
    for i in range(args.warmup):
        run_step(i, overlap=overlap)
    pu.finish()
    torch.cuda.synchronize()

    def new_events(phases=PHASES):
        # timing events without the system-scope fence: a launch-attached
        # pair costs about 3 us of stream time instead of 7 us
        return {p: (Event(timing=True), Event(timing=True)) for p in phases}

    def phase_sums(evs, phases=PHASES):
        # step s carries weight-gradient events only if it launched them
        # (grouped: the last step of each group, counted from 0 after a finish())
        def ran(p, s):
            return p not in ("gate_up_wgrad", "down_wgrad") or M == 1 or pu.wgrad_launches_at(s)
        return {p: sum(ev[p][0].elapsed_time(ev[p][1]) for s, ev in enumerate(evs) if ran(p, s)) for p in phases}

    # ---- per-kernel pass: every phase timed by HIP events, one kernel after
    # another, so that every phase's duration is its own (row GEMMs: events
    # attached to the kernel launch, i.e. the kernel's start and end; other
    # phases: event records around the call)
    evs_seq = [new_events() for _ in range(args.steps)]
    torch.cuda.synchronize()
    seq0, seq1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    seq0.record(stream)
    flush_ev = new_events(["gate_up_wgrad", "down_wgrad"])
    for s in range(args.steps):
        run_step(s, evs_seq[s])
    flushed = pu.finish(ev=flush_ev)  # grouped weight gradients: an incomplete last group's
    seq1.record(stream)
    torch.cuda.synchronize()
    phase_ms = phase_sums(evs_seq)
    if flushed:
        for p in ("gate_up_wgrad", "down_wgrad"):
            phase_ms[p] += flush_ev[p][0].elapsed_time(flush_ev[p][1])
    seq_ms_per_step = seq0.elapsed_time(seq1) / args.steps
    # the dominant single-launch kernel; in the timed region only its calls
    # carry events (on the stream it runs on)
    dom = max((p for p in PHASES if p in SINGLE_LAUNCH), key=lambda p: phase_ms[p])

    # ---- timed region: the step as it runs (backward GEMMs overlapped);
    # only the dominant kernel's calls carry HIP events, attached to its
    # launches so that no event command sits between kernels (event records
    # around every call cost about 80 us per step; a record pair around one
    # kernel left two gaps of about 6 us). Replaying the step from
    # HIP graphs was measured slower than launching the calls (0.87 vs
    # 0.83 ms per step), so the calls are launched one by one.
    evs = [new_events([dom]) for _ in range(args.steps)]

    pipelined = overlap and not args.no_pipeline

    def timed_step(i, ev, last):
        run_step(i, ev, overlap=overlap, pipelined=pipelined, last=last)

    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    pu.start()
    for i in range(2):
        timed_step(i, None, 1)
    pu.finish()
    torch.cuda.synchronize()
    start.record(stream)
    for s in range(args.steps):
        timed_step(s, evs[s], args.steps - 1)
    pu.finish()
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps
    live_ms = phase_sums(evs, [dom])

    # ---- algorithmic work of the timed steps
    work = {p: {"flop": 0.0, "bytes": 0.0} for p in PHASES}
    for s in range(args.steps):
        N, g = Ns[s % n_micro], Gs[s % n_micro]
        for p, by in acc.phase_bytes(N, g, T, K, d, F, wgrad_group=M).items():
            work[p]["bytes"] += by
        for p in ("gate_up_fwd", "gate_up_dgrad", "gate_up_wgrad"):
            work[p]["flop"] += acc.gate_up_flops(N, d, F)
        for p in ("down_fwd", "down_dgrad", "down_wgrad"):
            work[p]["flop"] += acc.down_flops(N, d, F)

    def rates(p, ms):
        t_s = ms / 1e3
        fl, by = work[p]["flop"], work[p]["bytes"]
        t_mfma = fl / acc.PEAK_BF16_DENSE_FLOPS
        t_hbm = by / acc.PEAK_HBM_BYTES_PER_S
        if fl > 0 and t_mfma >= t_hbm:
            return "mfma", fl / t_s / 1e12, acc.PEAK_BF16_DENSE_FLOPS / 1e12, "TFLOP/s"
        return "hbm", by / t_s / 1e9, acc.PEAK_HBM_BYTES_PER_S / 1e9, "GB/s"

    kernels = {}
    for p in PHASES:
        t_s = phase_ms[p] / 1e3
        fl, by = work[p]["flop"], work[p]["bytes"]
        bound, ach, peak, unit = rates(p, phase_ms[p])
        tr = measured_traffic(p)
        kernels[p] = {"us_per_step": round(phase_ms[p] * 1e3 / args.steps, 2), "bound": bound,
                      "achieved": round(ach, 2), "unit": unit, "frac": round(ach / peak, 4),
                      "tflops": round(fl / t_s / 1e12, 2) if fl else None,
                      "gbs": round(by / t_s / 1e9, 1),
                      "algorithmic_bytes_per_micro_step": round(by / args.steps, 0),
                      "traffic_bytes_per_micro_step": tr,
                      "traffic_over_algorithmic": round(tr / (by / args.steps), 3) if tr else None}
    # the dominant single-launch kernel, timed live in the timed region on
    # the stream it runs on
    bound, ach, peak, unit = rates(dom, live_ms[dom])
    roofline = {"bound": bound, "achieved": round(ach, 2), "peak": round(peak, 1), "unit": unit,
                "frac": round(ach / peak, 4), "traffic": measured_traffic(dom), "kernel": dom,
                "avg_launch_us": round(live_ms[dom] * 1e3 / args.steps, 2)}

    ffn = ["gate_up_fwd", "down_fwd", "down_dgrad", "gate_up_dgrad", "gate_up_wgrad", "down_wgrad"]
    ffn_flop = sum(work[p]["flop"] for p in ffn)
    ffn_s = sum(phase_ms[p] for p in ffn) / 1e3
    fwd_ph = ["histogram_assign", "permute", "gate_up_fwd", "down_fwd", "combine"]
    fwd_s = sum(phase_ms[p] for p in fwd_ph) / 1e3
    ffn_fwd_s = (phase_ms["gate_up_fwd"] + phase_ms["down_fwd"]) / 1e3
    ffn_fwd_flop = work["gate_up_fwd"]["flop"] + work["down_fwd"]["flop"]
    value = T * args.steps / (total_ms / 1e3)

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Zipf s=1.1 + Dirichlet a=0.3 routing; N(0,1) tokens and upstream grads; "
                "N(0,1/fan_in) weights)",
        "config": {"workload": "qwen3-30b-a3b EP=8 rank share, policy-update micro-step (fwd+bwd)",
                   "T": T, "d": d, "F": F, "E": E, "K": K, "local_experts": G, "slots": S_max,
                   "micro_steps": n_micro, "n_pairs_mean": round(float(np.mean(Ns)), 1),
                   "n_pairs_min": int(min(Ns)), "n_pairs_max": int(max(Ns)),
                   "backward_overlap": overlap, "tail_split": not args.no_split,
                   "pipelined_micro_steps": pipelined,
                   "side_gathers": args.side_gathers if overlap else 0, "wgrad_group": M,
                   "early_hist": bool(pipelined and not args.no_early_hist)},
        "ms_per_step_sequential": round(seq_ms_per_step, 4),
        "roofline": roofline,
        "grouped_ffn_tflops": round(ffn_flop / ffn_s / 1e12, 2),
        "grouped_ffn_frac_bf16_peak": round(ffn_flop / ffn_s / acc.PEAK_BF16_DENSE_FLOPS, 4),
        "grouped_ffn_fwd_tflops": round(ffn_fwd_flop / ffn_fwd_s / 1e12, 2),
        "permute_gbs": kernels["permute"]["gbs"],
        "combine_gbs": kernels["combine"]["gbs"],
        "forward_tokens_per_s": round(T * args.steps / fwd_s, 1),
        "kernels": kernels,
        "setup_s": round(setup_s, 1),
    }
    if not args.no_reference_peaks:
        ref = reference_peaks(dev)
        ref["dominant_kernel_frac"] = round(roofline["achieved"] / ref["bf16_gemm_tflops"], 4) \
            if roofline["unit"] == "TFLOP/s" else None
        ref["grouped_ffn_frac"] = round(out["grouped_ffn_tflops"] / ref["bf16_gemm_tflops"], 4)
        ref["permute_frac"] = round(out["permute_gbs"] / ref["copy_gbs"], 4)
        ref["combine_frac"] = round(out["combine_gbs"] / ref["copy_gbs"], 4)
        out["measured_peaks"] = ref
    if not args.no_cache_report:
        out["cache"] = cache_report(pu, mss, n_micro, dom, dev)
    if not args.no_planner:
        out["planner"] = planner_report(w, api, dev, n_micro)
    if not args.no_transfer:
        out["transfer"] = transfer_report(w, api, dev, pu, mss, n_micro)
    if not args.no_other_configs:
        del pu, mss, buf
        torch.cuda.empty_cache()
        out["other_configs"] = {name: config_report(name, api, dev)
                                for name in ("mixtral-8x7b-share", "deepseek-v3-ep32-share")}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)
    return 0


def cache_report(pu, mss, n_micro: int, dom: str, dev, flush_mib: int = 512) -> dict:
    """Each micro-step alone, one stream, with its own weight gradients,
    every phase between HIP events: once right after a warm-up run of the
    same micro-step (warm: its inputs, weights and buffers partly in the L2s
    and the 256 MB Infinity Cache) and once after a flush_mib scratch write
    (cold: caches hold the scratch buffer). Medians over the micro-steps."""
    import numpy as np
    import torch

    from paper_2606_11867_amd.hip_events import Event
    from paper_2606_11867_amd.policy_update import PHASES

    scratch = torch.empty(flush_mib << 20, dtype=torch.uint8, device=dev)
    main = pu.main

    def one(i):
        ev = {p: (Event(timing=True), Event(timing=True)) for p in PHASES}
        wev = {p: (Event(timing=True), Event(timing=True)) for p in ("gate_up_wgrad", "down_wgrad")}
        a, b = Event(timing=True), Event(timing=True)
        a.record(main)
        pu.run(i, mss[i % n_micro], ev)
        flushed = pu.finish(ev=wev)
        b.record(main)
        torch.cuda.synchronize()
        ph = {p: ev[p][0].elapsed_time(ev[p][1]) * 1e3 for p in PHASES if p not in wev or not flushed}
        if flushed:
            ph.update({p: wev[p][0].elapsed_time(wev[p][1]) * 1e3 for p in wev})
        return a.elapsed_time(b), ph

    warm, cold = [], []
    for i in range(n_micro):
        one(i)
        warm.append(one(i))
        scratch.fill_(i & 0xFF)
        cold.append(one(i))
    med = lambda xs: float(np.median(xs))  # noqa: E731
    phases = {p: {"warm_us": round(med([x[1][p] for x in warm]), 2), "cold_us": round(med([x[1][p] for x in cold]), 2)}
              for p in PHASES}
    return {"micro_step_ms": {"warm": round(med([x[0] for x in warm]), 4), "cold": round(med([x[0] for x in cold]), 4)},
            "dominant_kernel": dom, "phases": phases,
            "method": f"each of the {n_micro} micro-steps alone on one stream with its own weight gradients, "
                      f"after a warm-up run of itself (warm) or after a {flush_mib} MiB scratch write (cold); "
                      "medians over the micro-steps"}


def reference_peaks(dev) -> dict:
    """Context for the rooflines, measured outside the timed region: a large
    square bf16 GEMM through torch (hipBLASLt) and a 1 GiB device copy (far
    larger than the caches). Neither is part of the path."""
    import torch
    n = 8192
    a = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    b = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    c = torch.empty(n, n, device=dev, dtype=torch.bfloat16)
    for _ in range(3):
        torch.matmul(a, b, out=c)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        torch.matmul(a, b, out=c)
    e1.record()
    torch.cuda.synchronize()
    gemm = 2.0 * n ** 3 * 10 / (e0.elapsed_time(e1) / 1e3) / 1e12
    del a, b, c
    x = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    x.fill_(1)
    y = torch.empty_like(x)
    for _ in range(2):
        y.copy_(x)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(5):
        y.copy_(x)
    e1.record()
    torch.cuda.synchronize()
    copy = 2.0 * (1 << 30) * 5 / (e0.elapsed_time(e1) / 1e3) / 1e9
    return {"bf16_gemm_tflops": round(gemm, 1), "bf16_gemm": "torch.matmul 8192^3 (hipBLASLt)",
            "copy_gbs": round(copy, 1), "copy": "1 GiB device copy, bytes read + written"}


def config_report(name: str, api, dev, reps: int = 5) -> dict:
    """One micro-step of another rank share (its measured micro-step: the one
    whose local pair count is closest to the share's nominal T * K / P),
    forward and backward, every phase on one stream between HIP events,
    averaged over `reps` runs after a warm-up. Routing and the slot table come
    from the seeded generator; activations, upstream gradients and weights are
    drawn on the device (N(0,1), N(0, 1/fan_in)): values do not change the
    work. Rates are against the same algorithmic work as the main line."""
    import numpy as np
    import torch

    from paper_2606_11867_amd.hip_events import Event
    from paper_2606_11867_amd.policy_update import PHASES, MicroStep, PolicyUpdate
    from workload import accounting as acc
    from workload import make_workload

    w = make_workload(name)
    spec = w.spec
    T, K, d, F, E = spec.T, spec.K, spec.d, spec.F, spec.E
    m = w.micro[w.measured]
    bf = torch.bfloat16
    g = torch.Generator(device=dev).manual_seed(23)
    G = int(m.plan.G)
    gu = (torch.randn((m.plan.W, 2 * F, d), generator=g, device=dev) / d ** 0.5).to(bf)
    dn = (torch.randn((m.plan.W, d, F), generator=g, device=dev) / F ** 0.5).to(bf)
    ms = MicroStep(ids=torch.from_numpy(m.ids).to(dev), gates=torch.from_numpy(m.gates).to(dev),
                   x=torch.randn((T, d), generator=g, device=dev).to(bf),
                   dy=torch.randn((T, d), generator=g, device=dev).to(bf),
                   plan=api.DevicePlan.from_host(m.plan, dev))
    n_cap = int(w.stats.get("local_pairs_max", T * K))
    pu = PolicyUpdate(T, K, d, F, E, G, m.plan.S, gu, dn, dev, n_cap=n_cap)
    pu.run(0, ms)
    torch.cuda.synchronize()
    st = pu.set_of(0, False)
    N = int(st["slot_offset"][m.plan.S].item())
    sc = st["slot_count"][:m.plan.S].cpu().numpy()
    gidx = m.plan.slot_gidx
    gn = int(len(set(np.asarray(gidx)[sc > 0].tolist())))
    evs = [{p: (Event(timing=True), Event(timing=True)) for p in PHASES} for _ in range(reps)]
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(pu.main)
    for ev in evs:
        pu.run(0, ms, ev)
    t1.record(pu.main)
    torch.cuda.synchronize()
    step_us = t0.elapsed_time(t1) * 1e3 / reps
    by = acc.phase_bytes(N, gn, T, K, d, F)
    fl = {p: 0.0 for p in PHASES}
    for p in ("gate_up_fwd", "gate_up_dgrad", "gate_up_wgrad"):
        fl[p] = acc.gate_up_flops(N, d, F)
    for p in ("down_fwd", "down_dgrad", "down_wgrad"):
        fl[p] = acc.down_flops(N, d, F)
    phases = {}
    for p in PHASES:
        us = sum(ev[p][0].elapsed_time(ev[p][1]) for ev in evs) * 1e3 / reps
        e = {"us": round(us, 2), "gbs": round(by[p] / (us * 1e-6) / 1e9, 1),
             "hbm_frac": round(by[p] / (us * 1e-6) / acc.PEAK_HBM_BYTES_PER_S, 4)}
        if fl[p]:
            e["tflops"] = round(fl[p] / (us * 1e-6) / 1e12, 1)
            e["mfma_frac"] = round(fl[p] / (us * 1e-6) / acc.PEAK_BF16_DENSE_FLOPS, 4)
        phases[p] = e
    ffn = ["gate_up_fwd", "down_fwd", "down_dgrad", "gate_up_dgrad", "gate_up_wgrad", "down_wgrad"]
    ffn_us = sum(phases[p]["us"] for p in ffn)
    ffn_fl = sum(fl[p] for p in ffn)
    out = {"micro_step": int(w.measured), "T": T, "d": d, "F": F, "E": E, "K": K, "slots": int(m.plan.S),
           "n_pairs": N, "slot_counts": sorted((int(c) for c in sc), reverse=True),
           "us_per_micro_step_one_stream": round(step_us, 1),
           "tokens_per_s_one_stream": round(T / (step_us * 1e-6), 1),
           "grouped_ffn_tflops": round(ffn_fl / (ffn_us * 1e-6) / 1e12, 1),
           "grouped_ffn_frac_bf16_peak": round(ffn_fl / (ffn_us * 1e-6) / acc.PEAK_BF16_DENSE_FLOPS, 4),
           "phases": phases,
           "data": "routing from the seeded generator; activations, gradients and weights drawn on the device"}
    del pu, ms, gu, dn
    torch.cuda.empty_cache()
    return out


def transfer_report(w, api, dev, pu, mss, n_micro: int) -> dict:
    """The one-GPU half of the Expert Transfer Engine (Sec. 6), measured
    outside the timed region with HIP events:

    * Copy-out / Copy-in (Sec. 6.2) of every expert of the share (16 local
      + 4 replica slots) with bf16 parameters and fp32 gradients, 27 MiB per
      record (App. A.3/A.4), and Copy-in adding 4 replica partial gradients
      into their main experts; HBM bytes read + written per second.
    * CPU-assisted prefetch (Sec. 6.1): App. A.4's worst case of N_s = 10
      experts (90 MiB of bf16 parameters) from a pinned host master copy,
      alone, and on an auxiliary stream beside the forward of a micro-step
      (dispatch, expert FFN forward, combine: the recompute stage), to show
      how much of it the forward hides.
    """
    import numpy as np
    import torch

    spec = w.spec
    d, F, E = spec.d, spec.F, spec.E
    bf = torch.bfloat16
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731

    def timed(fn, reps=5, stream=None):
        st = stream or torch.cuda.current_stream(dev)
        fn()
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record(st)
        for _ in range(reps):
            fn()
        b.record(st)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps  # us

    n = 20
    g = torch.Generator(device=dev).manual_seed(17)
    wgu = torch.randn((n, 2 * F, d), generator=g, device=dev).to(bf)
    wdn = torch.randn((n, d, F), generator=g, device=dev).to(bf)
    ggu = torch.randn((n, 2 * F, d), generator=g, device=dev)
    gdn = torch.randn((n, d, F), generator=g, device=dev)
    both = api._lib.XFER_PARAMS | api._lib.XFER_GRADS
    rb = api.xfer_record_bytes(d, F, bf, both)
    idx = list(range(n))
    send = api.copy_out(wgu, wdn, ggu, gdn, idx, idx, both)
    recv = send.clone()
    wgu2, wdn2, ggu2, gdn2 = (torch.empty_like(t) for t in (wgu, wdn, ggu, gdn))
    t_out = timed(lambda: api.copy_out(wgu, wdn, ggu, gdn, idx, idx, both, buf=send))
    t_in = timed(lambda: api.copy_in(recv, idx, idx, [0] * n, both, wgu2, wdn2, ggu2, gdn2))
    grads = api._lib.XFER_GRADS
    rbg = api.xfer_record_bytes(d, F, bf, grads)
    part = api.copy_out(wgu, wdn, ggu, gdn, [0, 1, 2, 3], [16, 17, 18, 19], grads)
    t_add = timed(lambda: api.copy_in(part, [-1] * 4, [0, 1, 2, 3], [1] * 4, grads, wgu2, wdn2, ggu2, gdn2))
    by_out = 2.0 * n * rb
    by_add = 4 * rbg * 3.0

    # CPU-assisted prefetch from a pinned master copy of all E experts
    n_pf = 10
    master_gu = torch.empty((E, 2 * F, d), dtype=bf, pin_memory=True)
    master_dn = torch.empty((E, d, F), dtype=bf, pin_memory=True)
    master_gu.copy_(torch.randn((E, 2 * F, d), generator=torch.Generator().manual_seed(1)).to(bf))
    master_dn.copy_(torch.randn((E, d, F), generator=torch.Generator().manual_seed(2)).to(bf))
    slots_gu = torch.empty((n_pf, 2 * F, d), dtype=bf, device=dev)
    slots_dn = torch.empty((n_pf, d, F), dtype=bf, device=dev)
    experts = list(range(0, 2 * n_pf, 2))
    aux = torch.cuda.Stream(dev)
    pf = lambda: api.prefetch_experts(master_gu, master_dn, experts, list(range(n_pf)), slots_gu, slots_dn,  # noqa
                                      stream=aux)
    t_pf = timed(pf, stream=aux)
    pf_bytes = n_pf * api.xfer_record_bytes(d, F, bf, api._lib.XFER_PARAMS)
    # the forward of micro-step i (recompute stage) alone, then with the prefetch beside it
    fwd_phases = {"histogram_assign", "permute", "gate_up_fwd", "down_fwd", "combine"}

    def forward(i):
        for ph, op in pu.ops(i, mss[i % n_micro]):
            if ph in fwd_phases:
                op()

    main = torch.cuda.current_stream(dev)
    reps = 2 * n_micro
    forward(0)
    torch.cuda.synchronize()
    a, b = ev(), ev()
    a.record(main)
    for i in range(reps):
        forward(i)
    b.record(main)
    torch.cuda.synchronize()
    t_fwd = a.elapsed_time(b) * 1e3 / reps
    # the prefetch for micro-step i + 1 goes out with micro-step i's forward.
    # Its slots were last read by micro-step i - 1, so the host waits for that
    # forward's event before queueing it: on this runtime, host-to-device
    # copies queued on a stream that waits on a not yet completed event of
    # another stream are carried out synchronously by the host (measured:
    # the copy calls then block for the whole transfer), so the aux stream
    # never waits on the main stream here; the main stream waits for the
    # aux stream before the next forward.
    fwd_done = [torch.cuda.Event(), torch.cuda.Event()]
    a.record(main)
    for i in range(reps):
        if i >= 1:
            fwd_done[(i - 1) % 2].synchronize()
        pf()
        forward(i)
        fwd_done[i % 2].record(main)
        main.wait_stream(aux)
    b.record(main)
    torch.cuda.synchronize()
    t_both = a.elapsed_time(b) * 1e3 / reps
    hidden = max(0.0, min(1.0, (t_fwd + t_pf - t_both) / t_pf)) if t_pf > 0 else None
    # App. A.2's overlap condition on this GPU: the smallest per-rank token
    # count n whose layer time covers this prefetch (N_s = 10 experts), with
    # the measured PCIe rate and the measured large-GEMM rate as F
    from workload import accounting as acc
    n_min = acc.n_min_cpu(d, F, spec.K, E, n_pf, 2, 1.0e15, pf_bytes / (t_pf * 1e-6))
    return {
        "copy_out": {"records": n, "record_mib": round(rb / 2 ** 20, 2), "us": round(t_out, 1),
                     "gbs": round(by_out / (t_out * 1e-6) / 1e9, 1),
                     "frac_hbm": round(by_out / (t_out * 1e-6) / 8e12, 4)},
        "copy_in_assign": {"records": n, "us": round(t_in, 1), "gbs": round(by_out / (t_in * 1e-6) / 1e9, 1),
                           "frac_hbm": round(by_out / (t_in * 1e-6) / 8e12, 4)},
        "copy_in_add_replica_grads": {"records": 4, "us": round(t_add, 1),
                                      "gbs": round(by_add / (t_add * 1e-6) / 1e9, 1),
                                      "frac_hbm": round(by_add / (t_add * 1e-6) / 8e12, 4)},
        "prefetch": {"experts": n_pf, "mib": round(pf_bytes / 2 ** 20, 1), "us": round(t_pf, 1),
                     "gbs": round(pf_bytes / (t_pf * 1e-6) / 1e9, 1),
                     "paper_h20": "90 MiB in 1.47 ms over PCIe Gen5 x16 (App. A.4)"},
        "prefetch_beside_forward": {"forward_us": round(t_fwd, 1), "prefetch_us": round(t_pf, 1),
                                    "together_us": round(t_both, 1), "hidden_frac": None if hidden is None
                                    else round(hidden, 3),
                                    "note": "forward of one micro-step (dispatch, FFN forward, combine) on the "
                                            "main stream, the 10-expert prefetch on an auxiliary stream"},
        "app_a_n_min_cpu": {"tokens": round(n_min), "note": "App. A.2 Eq. cpu_n_min with N_s = 10, p_w = 2, "
                                                            "F = 1 PFLOP/s (about the measured large bf16 GEMM "
                                                            "rate), B_PCIe = the prefetch rate above; the paper "
                                                            "gives 1862 tokens on H20"},
    }


def planner_report(w, api, dev, n_micro: int, N_r: int = 4, C_max: int = 8) -> dict:
    """The placement planner on the same micro-steps (Sec. 8 Alg. 1; App. D
    Alg. 3; host C++), and the per-source dispatch of the measured rank's
    planned share on the GPU (Sec. 7.2 r_{s,e,j} as water-filled counts).

    Reported: the planner's host time per micro-step, the compute imbalance
    L_max / L_mean over the 8 ranks (natural placement e -> e / (E/P), Stage 1
    base placement, after Stages 2-4; medians over the micro-steps, the
    metric of Sec. 10.4), the planned share's local pairs, and the GPU time of
    histogram_src + assign_replicas + permute for it. Then the whole layer
    (dispatch, expert FFN forward and backward, combine and the backward
    gathers, one stream) on the share of each micro-step's slowest rank,
    under the natural placement and under the plan: all ranks wait for the
    slowest one (Sec. 7.1, Eq. 1), so these are the layer times per
    micro-step that the two placements give on this GPU.
    """
    import numpy as np
    import torch
    from workload import Plan

    spec = w.spec
    P, E, T, K = spec.P, spec.E, spec.T, spec.K
    tb = (np.arange(P + 1) * (T // P)).astype(np.int32)

    def src_loads(ids):
        out = np.zeros((P, E), dtype=np.int64)
        for s in range(P):
            v = ids[tb[s]:tb[s + 1]].reshape(-1)
            out[s] = np.bincount(v[v >= 0], minlength=E)
        return out

    loads = [src_loads(m.ids) for m in w.micro[:n_micro]]
    base = api.plan_base(np.sum(loads, axis=0), 1, P, E // P)
    natural = np.arange(E) // (E // P)
    imb = {"natural": [], "base": [], "planned": []}
    plans, host_s = [], 0.0

    def share_plan(copy_rank, counts, rank):
        sl = api.plan_rank_slots(copy_rank, rank)
        return Plan(E=E, R_max=C_max, slot_expert=sl["slot_expert"], slot_replica=sl["slot_replica"],
                    expert_nrep=sl["expert_nrep"], expert_rep_weight=None, slot_widx=sl["slot_widx"],
                    slot_gidx=sl["slot_widx"].copy(), local_experts=sl["local_experts"],
                    src_token_begin=tb, src_rep_weight=counts)

    # the natural placement as a plan: one copy per expert, on rank e / (E/P)
    nat_rank = np.full((E, C_max), -1, dtype=np.int32)
    nat_rank[:, 0] = natural
    slowest = {"natural": [], "planned": []}  # (plan, expected local pairs) per micro-step
    for i, W in enumerate(loads):
        t0 = time.perf_counter()
        copy_rank, counts, rank_load = api.plan_micro_step(W, base, 1, P, E // P, N_r, C_max)
        plans.append(share_plan(copy_rank, counts, w.rank))
        host_s += time.perf_counter() - t0
        we = W.sum(axis=0)
        for name, pl in (("natural", natural), ("base", base)):
            L = np.bincount(pl, weights=we, minlength=P)
            imb[name].append(float(L.max() / L.mean()))
        imb["planned"].append(float(rank_load.max() / rank_load.mean()))
        L_nat = np.bincount(natural, weights=we, minlength=P).astype(np.int64)
        nat_counts = np.zeros((P, E, C_max), dtype=np.int32)
        nat_counts[:, :, 0] = W
        p_nat, p_pl = int(np.argmax(L_nat)), int(np.argmax(rank_load))
        slowest["natural"].append((share_plan(nat_rank, nat_counts, p_nat), int(L_nat[p_nat])))
        slowest["planned"].append((share_plan(copy_rank, counts, p_pl), int(rank_load[p_pl])))
    # GPU: per-source dispatch of the measured rank's planned share
    bf = torch.bfloat16
    d = spec.d
    n_cap = T * K
    ws = api.workspace(T, K, E * P, dev)
    x_perm = torch.empty((n_cap, d), dtype=bf, device=dev)
    r2p = torch.empty(n_cap, dtype=torch.int32, device=dev)
    p2r = torch.empty(T * K, dtype=torch.int32, device=dev)
    ms = []
    for i, pl in enumerate(plans):
        dp = api.DevicePlan.from_host(pl, dev)
        ms.append(dict(ids=torch.from_numpy(w.micro[i].ids).to(dev),
                       x=torch.from_numpy(np.ascontiguousarray(w.x(i), dtype=np.float32)).to(dev).to(bf),
                       plan=dp, cplan=dp.c_struct()))
    lib = api._lib.load()
    sp = torch.cuda.current_stream(dev).cuda_stream
    Ns = []

    def dispatch(m):
        counts = api.histogram_src(m["ids"], E, m["plan"].src_token_begin, ws)
        rb, sc, so = api.assign_replicas(counts.reshape(-1), m["plan"], ws)
        api.check(lib.foremoe_permute(m["x"].data_ptr(), api._lib.BF16, T, d, m["ids"].data_ptr(), K,
                                      ctypes.byref(m["cplan"]), rb.data_ptr(), so.data_ptr(), n_cap,
                                      x_perm.data_ptr(), r2p.data_ptr(), p2r.data_ptr(), ws.data_ptr(),
                                      ws.numel(), sp), "foremoe_permute")
        return so

    for m in ms:
        Ns.append(int(dispatch(m)[-1].item()))
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    rounds = 3
    e0.record()
    for _ in range(rounds):
        for m in ms:
            dispatch(m)
    e1.record()
    torch.cuda.synchronize()
    dispatch_us = e0.elapsed_time(e1) * 1e3 / (rounds * len(ms))

    # the whole layer on the slowest rank's share, natural vs planned
    F = spec.F
    gen = torch.Generator(device=dev).manual_seed(11)
    W_max = max(pl.W for v in slowest.values() for pl, _ in v)
    gu = (torch.randn((W_max, 2 * F, d), generator=gen, device=dev) / d ** 0.5).to(bf)
    dn = (torch.randn((W_max, d, F), generator=gen, device=dev) / F ** 0.5).to(bf)
    dwgu = torch.zeros((W_max, 2 * F, d), dtype=torch.float32, device=dev)
    dwdn = torch.zeros((W_max, d, F), dtype=torch.float32, device=dev)
    dy = torch.randn((T, d), generator=gen, device=dev).to(bf)
    rws, wws = api.ffn_workspace(dev), api.wgrad_workspace(d, F, dev)
    gates = [torch.from_numpy(w.micro[i].gates).to(dev) for i in range(len(ms))]

    def layer(m, g):
        so = dispatch(m)
        h, y_perm, au = api.grouped_ffn_fwd(x_perm, so, m["plan"].slot_widx, gu, dn, ws=rws)
        api.combine(y_perm, p2r, g, out_dtype=bf)
        dy_perm, _ = api.combine_bwd(dy, y_perm, p2r, g)
        d_au, dx_perm = api.grouped_ffn_dgrad(dy_perm, au, so, m["plan"].slot_widx, gu, dn, ws=rws)
        api.grouped_ffn_wgrad(x_perm, h, dy_perm, d_au, so, m["plan"].slot_gidx, dwgu, dwdn, ws=wws)
        api.permute_bwd(dx_perm, p2r, T, K, out_dtype=bf)
        return so

    layer_us, pairs = {}, {}
    for name, v in slowest.items():
        mm = []
        for i, (pl, n_exp) in enumerate(v):
            dp = api.DevicePlan.from_host(pl, dev)
            m = dict(ms[i], plan=dp, cplan=dp.c_struct())
            got = int(layer(m, gates[i])[-1].item())  # warm-up pass, checked against the planner
            if got != n_exp:
                raise RuntimeError(f"{name} share of micro-step {i}: {got} local pairs, planner says {n_exp}")
            mm.append(m)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(2):
            for i, m in enumerate(mm):
                layer(m, gates[i])
        e1.record()
        torch.cuda.synchronize()
        layer_us[name] = round(e0.elapsed_time(e1) * 1e3 / (2 * len(mm)), 1)
        pairs[name] = round(float(np.mean([n for _, n in v])), 1)
    med = {k: round(float(np.median(v)), 3) for k, v in imb.items()}
    return {"plan_us_per_micro_step": round(host_s / len(loads) * 1e6, 1),
            "imbalance_median": med,
            "imbalance_max": {k: round(float(np.max(v)), 3) for k, v in imb.items()},
            "planned_share": {"rank": int(w.rank), "n_pairs_mean": round(float(np.mean(Ns)), 1),
                              "n_pairs_max": int(max(Ns)), "n_pairs_min": int(min(Ns)),
                              "dispatch_us_per_micro_step": round(dispatch_us, 2),
                              "note": "histogram_src + assign_replicas + permute, (source, expert) keys"},
            "slowest_rank_layer": {"us_per_micro_step": layer_us, "n_pairs_mean": pairs,
                                   "speedup": round(layer_us["natural"] / layer_us["planned"], 3),
                                   "note": "dispatch + expert FFN fwd/dgrad/wgrad + combine + backward "
                                           "gathers, one stream, on the slowest rank's share"}}


TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "traffic_qwen3_share.json")
# the kernels of every phase; a name that serves two phases is dispatched
# once for each per micro-step, in this order (one-stream and overlapped
# schedules alike)
PHASE_KERNELS = [
    ("hist_count_kernel", ["histogram_assign"], "paper_2606_11867_amd/csrc/dispatch.hip"),
    ("hist_scan_assign_kernel", ["histogram_assign"], "paper_2606_11867_amd/csrc/dispatch.hip"),
    ("permute_gather_kernel", ["permute"], "paper_2606_11867_amd/csrc/dispatch.hip"),
    ("gemm_rows_kernel<true, 1>", ["gate_up_fwd"], "paper_2606_11867_amd/csrc/grouped_gemm.hip"),
    ("gemm_rows_kernel<true, 0>", ["down_fwd"], "paper_2606_11867_amd/csrc/grouped_gemm.hip"),
    ("combine_kernel", ["combine", "permute_bwd"], "paper_2606_11867_amd/csrc/dispatch.hip"),
    ("combine_bwd_kernel", ["combine_bwd"], "paper_2606_11867_amd/csrc/dispatch.hip"),
    ("gemm_rows_kernel<false, 2>", ["down_dgrad"], "paper_2606_11867_amd/csrc/grouped_gemm.hip"),
    ("gemm_rows_kernel<false, 0>", ["gate_up_dgrad"], "paper_2606_11867_amd/csrc/grouped_gemm.hip"),
    ("gemm_wgrad_kernel", ["down_wgrad", "gate_up_wgrad"], "paper_2606_11867_amd/csrc/grouped_gemm.hip"),
    ("wgrad_reduce_kernel", ["down_wgrad", "gate_up_wgrad"], "paper_2606_11867_amd/csrc/grouped_gemm.hip"),
]


def _kernel_key(name: str):
    """The PHASE_KERNELS key of a demangled kernel name, or None."""
    import re
    m = re.search(r"gemm_rows_kernel<([^>]*)>", name)
    if m:
        args = [a.strip() for a in m.group(1).split(",")]
        return f"gemm_rows_kernel<{args[-2]}, {args[-1]}>"
    for key, _, _ in PHASE_KERNELS:
        if "<" not in key and re.search(r"\b" + key + r"\b", name):
            return key
    return None


def _file_sha(rel: str) -> str:
    import hashlib
    with open(os.path.join(ROOT, rel), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def summarize_counters(folder: str) -> int:
    """Per-kernel HBM traffic from rocprofv3 counter CSVs (FETCH_SIZE and
    WRITE_SIZE in KiB, summed over a dispatch's rows), each scaled by what
    the same counter reads for the calibration copies (bytes of a 1 GiB
    copy), against the algorithmic bytes of the same dispatches (the
    counters pass dispatches every micro-step three times, so per-dispatch
    averages are averages over the micro-steps). Writes TRAFFIC_RECORD."""
    import collections
    import csv

    from workload import accounting as acc

    def per_dispatch(path, counter):
        tot = collections.defaultdict(float)
        names = {}
        with open(path) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] != counter:
                    continue
                k = int(r["Dispatch_Id"])
                tot[k] += float(r["Counter_Value"])
                names[k] = r["Kernel_Name"]
        return [(k, names[k], tot[k]) for k in sorted(tot)]

    with open(os.path.join(folder, "pass.json")) as f:
        cp = json.loads([ln for ln in f if ln.startswith("{")][-1])["counters_pass"]
    cal = {}
    for counter, fn in (("FETCH_SIZE", "copy_fetch.csv"), ("WRITE_SIZE", "copy_write.csv")):
        vals = [v for _, n, v in per_dispatch(os.path.join(folder, fn), counter) if "copy" in n.lower()]
        cal[counter] = sum(vals) / len(vals) * 1024.0 / (1 << 30)  # counter bytes per copied byte
    per_phase = collections.defaultdict(lambda: {"fetch": [], "write": [], "kernels": set(), "sources": set()})
    for counter, fn in (("FETCH_SIZE", "fetch.csv"), ("WRITE_SIZE", "write.csv")):
        seen = collections.Counter()
        for _, name, v in per_dispatch(os.path.join(folder, fn), counter):
            key = _kernel_key(name)
            if key is None:
                continue
            phases, src = next((ph, sr) for k, ph, sr in PHASE_KERNELS if k == key)
            phase = phases[seen[key] % len(phases)]
            seen[key] += 1
            rec = per_phase[phase]
            rec["fetch" if counter == "FETCH_SIZE" else "write"].append(v * 1024.0 / cal[counter])
            rec["kernels"].add(key)
            rec["sources"].add(src)
    T, K, d, F = cp["T"], cp["K"], cp["d"], cp["F"]
    M = cp.get("wgrad_group", 1)
    alg = collections.defaultdict(float)
    for N, g in zip(cp["N"], cp["G"]):
        for p, by in acc.phase_bytes(N, g, T, K, d, F, wgrad_group=M).items():
            alg[p] += by / len(cp["N"])
    kernels = {}
    for phase, rec in per_phase.items():
        n_k = len(rec["kernels"])
        # launches of the phase: dispatches of its kernels / kernels per phase;
        # a weight-gradient launch serves M micro-steps
        launches = len(rec["fetch"]) // n_k
        per = M if phase in ("gate_up_wgrad", "down_wgrad") else 1
        fetch = sum(rec["fetch"]) / launches / per
        write = sum(rec["write"]) / launches / per
        kernels[phase] = {"kernels": sorted(rec["kernels"]), "launches": launches, "micro_steps_per_launch": per,
                          "read_bytes_per_micro_step": round(fetch), "write_bytes_per_micro_step": round(write),
                          "hbm_bytes_per_micro_step": round(fetch + write),
                          "algorithmic_bytes_per_micro_step": round(alg[phase]),
                          "ratio": round((fetch + write) / alg[phase], 3),
                          "sources": {s: _file_sha(s) for s in sorted(rec["sources"])}}
    out = {"workload": "qwen3-30b-a3b EP=8 rank share, policy-update micro-steps (bench.py --counters-pass: "
                       "every micro-step three times, one stream once then twice pipelined)",
           "calibration": {"fetch_size_per_copied_byte": round(cal["FETCH_SIZE"], 4),
                           "write_size_per_copied_byte": round(cal["WRITE_SIZE"], 4),
                           "copy": "torch device copy of 1 GiB (bench.py --copy-calibration)"},
           "kernels": {p: kernels[p] for p in PHASES_ORDER if p in kernels}}
    with open(TRAFFIC_RECORD, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print("| phase | kernels | launches | micro-steps per launch | read MB | written MB | HBM MB | "
          "algorithmic MB | ratio |")
    print("|---|---|---|---|---|---|---|---|---|")
    for p, k in out["kernels"].items():
        print(f"| {p} | {', '.join('`' + x + '`' for x in k['kernels'])} | {k['launches']} | "
              f"{k['micro_steps_per_launch']} | {k['read_bytes_per_micro_step'] / 1e6:.1f} | "
              f"{k['write_bytes_per_micro_step'] / 1e6:.1f} | {k['hbm_bytes_per_micro_step'] / 1e6:.1f} | "
              f"{k['algorithmic_bytes_per_micro_step'] / 1e6:.1f} | {k['ratio']:.2f} |")
    return 0


PHASES_ORDER = ["histogram_assign", "permute", "gate_up_fwd", "down_fwd", "combine", "combine_bwd",
                "down_dgrad", "gate_up_dgrad", "gate_up_wgrad", "down_wgrad", "permute_bwd"]


def measured_traffic(phase: str):
    """HBM bytes per micro-step of a phase (FETCH_SIZE + WRITE_SIZE, each
    scaled by a calibration copy; one launch per micro-step except the
    grouped weight gradients) from the committed counter record, or None
    when there is none or a source of the phase's kernels changed since."""
    if not os.path.exists(TRAFFIC_RECORD):
        return None
    with open(TRAFFIC_RECORD) as f:
        rec = json.load(f)
    k = rec.get("kernels", {}).get(phase)
    if not k or "sources" not in k:
        return None
    if any(_file_sha(src) != sha for src, sha in k["sources"].items()):
        return None
    return float(k["hbm_bytes_per_micro_step"])


def cpu_baseline(w, budget_s: float = 10.0) -> dict:
    """The fp64 oracle on whole micro-steps (forward + backward, gradients
    accumulated over micro-steps), run until about `budget_s` of CPU time."""
    import numpy as np

    import oracle.foremoe_oracle as O
    # the BLAS threads numpy runs with (pinned by OPENBLAS_NUM_THREADS before
    # numpy was imported, see the top of this file), the CPUs this process may
    # use, the CPU model and the BLAS build
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        threads = max([int(i.get("num_threads", 1)) for i in info] or [1])
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')} ({info[0].get('architecture')})"
    except Exception:  # pragma: no cover - threadpoolctl is optional
        threads = int(os.environ.get("OPENBLAS_NUM_THREADS", "1"))
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), cpu_model)
    except OSError:
        pass
    T, K = w.micro[0].ids.shape
    gu, dn = w.weights(w.micro[0].plan)
    G = w.micro[0].plan.G
    dwgu = np.zeros((G, gu.shape[1], gu.shape[2]))
    dwdn = np.zeros((G, dn.shape[1], dn.shape[2]))
    done, pairs, dt = 0, 0, 0.0
    while done < len(w.micro) and (done == 0 or dt < budget_s):
        m = w.micro[done]
        x, dy = w.x(done), w.dy(done)
        t0 = time.perf_counter()
        fwd = O.layer_forward(x, m.ids, m.gates, m.plan, gu, dn, n_cap=T * K)
        O.layer_backward(fwd, dy, m.gates, m.plan, gu, dn, T, K, dwgu, dwdn)
        dt += time.perf_counter() - t0
        pairs += int(fwd["slot_offset"][-1])
        done += 1
    return {"value": round(T * done / dt, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "affinity_cpus": AFFINITY_CPUS, "cpu_model": cpu_model, "blas": blas,
            "sample": f"micro-steps 0..{done - 1} of the same workload ({done} x {T} tokens, {pairs} local "
                      f"pairs), forward + backward in fp64 numpy, gradients accumulated; "
                      f"{dt:.1f} s"}


if __name__ == "__main__":
    sys.exit(main())
