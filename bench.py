"""Benchmark: candidate plans scored per second on one MI355X.

A step is one pass of the whole hot path over one batch already resident in
HBM: score every plan of the batch (plan decode, unit formation, resource
order, lifecycle and memory simulation, timeline, reductions) and select the
best feasible plan.  The default workload is the throughput configuration:
one 256-activation window (16 workflows x 16 activations, 8 devices, 16
models) and 1,048,576 candidate plans (about 0.9 GB of packed plans).

Prints one JSON line (see the fields at the end of main()).
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X published HBM3E bandwidth
# 32-bit vector lane operations per second: 256 CUs x 64 lanes x 2.4 GHz (the
# published 157.3 TFLOP/s fp32 vector peak counts an FMA as two operations and
# packed fp32 as two more)
VALU_PEAK_TLANE = 256 * 64 * 2.4e9 / 1e12
CSRC = os.path.join(ROOT, "paper_2609_03335_amd", "csrc")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "score_lean_traffic.json")


def algorithmic_bytes_per_plan(n_act: int) -> int:
    """Packed plan row read once (int8 device + uint16 priority + 2 flag
    bits per activation) plus the 32-byte score record written once."""
    return 3 * n_act + (n_act + 3) // 4 + 32


def kernel_source_digest() -> str:
    """sha256 over the scoring kernel's sources, its launch planner and the
    compiler flags: a stored counter measurement is only valid for the code
    it was taken on."""
    import hashlib
    from paper_2609_03335_amd import build
    h = hashlib.sha256()
    for name in ("score_kernel.h", "mutation.h", "score.hip", "lean.hip", "kernels.h", "host.hip"):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    h.update(" ".join(build.HIP_FLAGS).encode())
    return h.hexdigest()


def measured_counters(config: int, n_plans: int):
    """The committed counter record of this workload, or None when there is
    none or the kernel changed since it was taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    e = rec.get("configs", {}).get(str(config))
    if not e or e.get("n_plans") != n_plans or rec.get("kernel_source_sha256") != kernel_source_digest():
        return None
    return e


def measured_traffic(config: int, n_plans: int):
    """HBM bytes per scoring launch (FETCH_SIZE + WRITE_SIZE, each scaled by
    the copy-kernel factor), or None."""
    e = measured_counters(config, n_plans)
    return int(e["fetch_bytes"] + e["write_bytes"]) if e else None


def valu_roofline(config: int, n_plans: int, kernel_ms: float):
    """Vector-instruction issue of the scoring launch against the chip's
    32-bit lane-operation peak, from the committed SQ counters (wave
    instructions per dispatch) and this run's kernel time; None without a
    counter record for the current kernel."""
    e = measured_counters(config, n_plans)
    sq = (e or {}).get("sq_per_dispatch")
    if not sq or "SQ_INSTS_VALU" not in sq:
        return None
    achieved = sq["SQ_INSTS_VALU"] * 64 / (kernel_ms * 1e-3) / 1e12
    out = {"bound": "valu-issue", "achieved": round(achieved, 2), "peak": round(VALU_PEAK_TLANE, 2),
           "unit": "Tlane-op/s", "frac": round(achieved / VALU_PEAK_TLANE, 4),
           "valu_insts_per_plan": round(sq["SQ_INSTS_VALU"] / n_plans, 1)}
    for k, name in (("SQ_INSTS_SALU", "salu_insts_per_plan"), ("SQ_INSTS_LDS", "lds_insts_per_plan")):
        if k in sq:
            out[name] = round(sq[k] / n_plans, 1)
    return out


def copy_probe(nbytes: int) -> None:
    """A plain streaming kernel of known size (read nbytes, write nbytes):
    the calibration run for the HBM byte counters."""
    import torch
    src = torch.randint(0, 255, (nbytes,), dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.bitwise_not(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": nbytes, "copy_probe_bytes_written": nbytes,
                      "launches": 3, "kernel": "bitwise_not"}))


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=4, help="benchmark configuration 0-4")
    ap.add_argument("--plans", type=int, default=None, help="override the number of plans")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="plans in the CPU-baseline sample (default: about 10 s of CPU work)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--check", type=int, default=4096,
                    help="plans per leg checked against the oracle in the CPU-baseline leg (0 = none)")
    ap.add_argument("--search-mut", type=int, default=2,
                    help="mutations per generated candidate in the search leg (-1 = skip it)")
    ap.add_argument("--prefetch-slack-us", type=int, default=None,
                    help="dispatch slack of the rule-guided search leg (default: median load time)")
    ap.add_argument("--no-paper-order", action="store_true",
                    help="skip the leg that scores with the paper's reclamation order")
    ap.add_argument("--no-keys", action="store_true",
                    help="skip the ranking-key leg (Eq. 12 keys and their argmin)")
    ap.add_argument("--no-prefix", action="store_true",
                    help="skip the prefix-commit leg (Algorithm 1's last step, one plan)")
    ap.add_argument("--batch-limit", type=int, default=4,
                    help="units per device at once in the batch-limit leg (1 = skip it)")
    ap.add_argument("--replica-cap", type=int, default=6,
                    help="copies per model in the replica-cap leg (0 = skip it)")
    ap.add_argument("--copy-probe", type=int, default=None, metavar="BYTES",
                    help="only run a plain copy kernel of BYTES bytes (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py scores plans on one GPU only; runs on several GPUs are not supported "
              "(plans are independent: a batch would split into one range per GPU, with one "
              "exchange of the per-GPU argmin keys)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_03335_amd as pkg
    from paper_2609_03335_amd import workload

    assert torch.cuda.is_available(), "bench.py needs a HIP device"
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    t0 = time.time()
    win, plans = workload.make_config(args.config, n_plans=args.plans)
    # dispatch slack of the rule-guided prefetch alternative: the median load
    # time of the window (used only by the rule-guided search leg)
    win.prefetch_slack_us = int(np.median(win.load_us)) if args.prefetch_slack_us is None \
        else args.prefetch_slack_us
    P, N, D = plans.n_plans, win.n_act, win.n_dev
    print(f"[bench] config {args.config}: N={N} W={win.n_wf} D={D} M={win.n_models} P={P} "
          f"generated in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    ctx = pkg.Context(0)
    ctx.wf_plan_upload_window(win)
    # times as uint32 offsets or fp64, memory as int32 MiB
    dtype = {32: "u32", 64: "f64"}[ctx.wf_plan_time_bits()]
    dev, prio, flags = pkg.device_plans(plans, "cuda:0")
    scores = torch.empty((P, 32), dtype=torch.uint8, device="cuda:0")
    best = torch.empty(1, dtype=torch.int64, device="cuda:0")
    stream = torch.cuda.current_stream()

    def step():
        ctx.wf_plan_score_batch(dev, prio, flags, P, scores, None, stream)
        ctx.wf_plan_argmin(scores, P, best, stream)

    # samples of every leg's GPU records, checked against the oracle in the
    # CPU-baseline leg (the one part of this script that runs the oracle):
    # (what, GPU bytes, function of the oracle module giving its bytes)
    checks = []
    T = min(16, os.cpu_count() or 1)
    if args.check:
        step()
        torch.cuda.synchronize()
        idx = np.unique(np.linspace(0, P - 1, min(P, args.check)).astype(np.int64))
        got = pkg.scores_to_numpy(scores, P)[idx]
        checks.append(("scores", got.tobytes(),
                       lambda o, idx=idx: o.score(win, plans.take(idx), threads=T).tobytes()))

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # per-launch durations of the scoring kernel, on the stream it runs on
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    if torch.distributed.is_available() and torch.distributed.is_initialized():
        torch.distributed.barrier()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        ctx.wf_plan_score_batch(dev, prio, flags, P, scores, None, stream)
        ev[i][1].record(stream)
        ctx.wf_plan_argmin(scores, P, best, stream)
    torch.cuda.synchronize()
    t_total = time.perf_counter() - t_start
    if torch.distributed.is_available() and torch.distributed.is_initialized():
        torch.distributed.barrier()
    kernel_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    # the argmin on its own
    aev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, b in aev:
        a.record(stream)
        ctx.wf_plan_argmin(scores, P, best, stream)
        b.record(stream)
    torch.cuda.synchronize()
    argmin_ms = float(np.mean([a.elapsed_time(b) for a, b in aev]))
    # a plain streaming kernel over the same number of bytes: the bandwidth
    # this GPU actually delivers
    bpp0 = algorithmic_bytes_per_plan(N)
    nbytes = bpp0 * P // 2
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    torch.bitwise_not(src, out=dst)
    cev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(5)]
    for a, b in cev:
        a.record(stream)
        torch.bitwise_not(src, out=dst)
        b.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 2 * nbytes / (float(np.median([a.elapsed_time(b) for a, b in cev])) * 1e-3) / 1e9
    del src, dst
    ms_per_step = t_total * 1e3 / args.steps
    value = P * args.steps / t_total

    bpp = algorithmic_bytes_per_plan(N)
    achieved = bpp * P / (kernel_ms * 1e-3) / 1e9
    traffic = measured_traffic(args.config, P)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": ctx.wf_plan_score_kernel(), "kernel_ms": round(kernel_ms, 4),
                "bytes_per_plan": bpp, "copy_gbs_measured": round(copy_gbs, 1),
                "frac_of_copy": round(achieved / copy_gbs, 4), "argmin_ms": round(argmin_ms, 4)}

    # the prefix commit of the selected plan (Algorithm 1's last step): the
    # plan scored again with its schedule, then the actions to commit before
    # the next predicted event
    prefix_leg = None
    b_idx = int(best.item())
    if b_idx >= 0 and not args.no_prefix:
        rows = (dev[b_idx:b_idx + 1], prio[b_idx:b_idx + 1], flags[b_idx:b_idx + 1])
        _, sch = pkg.score_batch(ctx, *rows, 1, schedule=True, n_act=N, n_dev=D, reclaims=True,
                                 stream=stream)
        commit = torch.empty(max(N, 1), dtype=torch.uint8, device="cuda:0")
        crec = torch.empty(max(N, 1), dtype=torch.int64, device="cuda:0")
        t_next = torch.empty(1, dtype=torch.int64, device="cuda:0")
        pargs = (rows[0][0], sch[0][0], sch[1][0], sch[2][0], sch[4][0], commit, crec, t_next)
        ctx.wf_plan_prefix(*pargs, stream)
        torch.cuda.synchronize()
        if args.check:
            got = (np.array([t_next.item()], np.int64).tobytes() + commit.cpu().numpy()[:N].tobytes()
                   + crec.cpu().numpy()[:N].tobytes())

            def prefix_ref(o, b_idx=b_idx):
                one = plans.take(np.array([b_idx]))
                _, rs = o.score(win, one, schedule=True, reclaims=True)
                c, cr, t = o.prefix(win, one.dev[0], rs[0][0], rs[1][0], rs[2][0], rs[4][0])
                return np.array([t], np.int64).tobytes() + c.tobytes() + cr.tobytes()
            checks.append(("prefix commit", got, prefix_ref))
        pev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        for a, b in pev:
            a.record(stream)
            ctx.wf_plan_prefix(*pargs, stream)
            b.record(stream)
        torch.cuda.synchronize()
        cm = commit.cpu().numpy()[:N]
        prefix_leg = {"us": round(float(np.mean([a.elapsed_time(b) for a, b in pev])) * 1e3, 2),
                      "plan": b_idx, "t_next_us": int(t_next.item()),
                      "grants": int((cm & 1).astype(bool).sum()),
                      "loads": int((cm & 2).astype(bool).sum()),
                      "note": "prefix commit of the selected plan (Algorithm 1): the grants, loads "
                              "and reclamations that begin before its next predicted event"}

    # candidates generated around plan 0 on the GPU and scored (no plan rows
    # in HBM): the same number of plans, same window; uniform alternatives
    # and the rule-guided ones of Algorithm 1
    search, search_rules = None, None
    if args.search_mut >= 0:
        sd, sp_, sf = dev[0].contiguous(), prio[0].contiguous(), flags[0].contiguous()
        seed = 0x5EED
        legs = {}
        for mname, mode in (("uniform", pkg.WF_SEARCH_UNIFORM), ("rules", pkg.WF_SEARCH_RULES)):
            if args.check:
                n_chk = min(P, args.check)
                ctx.wf_plan_search_batch(sd, sp_, sf, seed, args.search_mut, 0, n_chk, scores, stream,
                                         mode=mode)
                torch.cuda.synchronize()

                def search_ref(o, n_chk=n_chk, seed=seed, mode=mode):
                    inc = (plans.dev[0], plans.prio[0], plans.flags[0])
                    cand = workload.PlanBatch(*o.search_candidates(win, *inc, seed, args.search_mut, 0,
                                                                   n_chk, mode=mode))
                    return o.score(win, cand, threads=T).tobytes()
                checks.append((f"generated candidates ({mname})",
                               pkg.scores_to_numpy(scores, n_chk).tobytes(), search_ref))
            for _ in range(args.warmup):
                ctx.wf_plan_search_batch(sd, sp_, sf, seed, args.search_mut, 0, P, scores, stream,
                                         mode=mode)
            torch.cuda.synchronize()
            sev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                   for _ in range(args.steps)]
            for i in range(args.steps):
                sev[i][0].record(stream)
                ctx.wf_plan_search_batch(sd, sp_, sf, seed, args.search_mut, i * P, P, scores, stream,
                                         mode=mode)
                sev[i][1].record(stream)
            torch.cuda.synchronize()
            s_ms = float(np.mean([a.elapsed_time(b) for a, b in sev]))
            legs[mname] = {"value": round(P / (s_ms * 1e-3), 1), "unit": "candidates/s",
                           "kernel_ms": round(s_ms, 4), "n_mut": args.search_mut}
        search = dict(legs["uniform"], note="candidates generated around one incumbent plan inside "
                      "the scoring kernel (no plan rows in HBM), same window and count")
        search_rules = dict(legs["rules"], prefetch_slack_us=int(win.prefetch_slack_us),
                            note="the same with Algorithm 1's rules for re-placed devices "
                                 "(BestFeasibleBinding) and prefetch bits (PlanPrefetch)")

    # the ranking keys of Eq. 12 for the same plans, and their lexicographic
    # argmin
    keys_leg = None
    if not args.no_keys:
        keys = scores  # 32 bytes per plan as well
        if args.check:
            n_chk = min(P, args.check)
            idx = np.unique(np.linspace(0, P - 1, n_chk).astype(np.int64))
            ctx.wf_plan_score_keys(dev, prio, flags, P, keys, stream)
            torch.cuda.synchronize()
            checks.append(("ranking keys", pkg.keys_to_numpy(keys, P)[idx].tobytes(),
                           lambda o, idx=idx: o.phi_keys(win, plans.take(idx), threads=T).tobytes()))
        out_k = torch.empty(1, dtype=torch.int64, device="cuda:0")
        for _ in range(args.warmup):
            ctx.wf_plan_score_keys(dev, prio, flags, P, keys, stream)
            ctx.wf_plan_argmin_keys(keys, P, out_k, stream)
        torch.cuda.synchronize()
        kev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
                torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        for a, b, c in kev:
            a.record(stream)
            ctx.wf_plan_score_keys(dev, prio, flags, P, keys, stream)
            b.record(stream)
            ctx.wf_plan_argmin_keys(keys, P, out_k, stream)
            c.record(stream)
        torch.cuda.synchronize()
        k_ms = float(np.mean([a.elapsed_time(b) for a, b, c in kev]))
        ka_ms = float(np.mean([b.elapsed_time(c) for a, b, c in kev]))
        keys_leg = {"value": round(P / ((k_ms + ka_ms) * 1e-3), 1), "unit": "plans/s",
                    "kernel_ms": round(k_ms, 4), "argmin_ms": round(ka_ms, 4),
                    "note": "ranking keys of Eq. 12 (admitted ready work, its latest completion, "
                            "timely prefetches, lifecycle overhead) for the same plans, then "
                            "their lexicographic argmin"}

    def window_leg(win_v, what):
        """The same plans scored under a variant of the window: a sample kept
        for the oracle check, then timed like the main leg."""
        ctx.wf_plan_upload_window(win_v)
        if args.check:
            n_chk = min(P, args.check)
            idx = np.unique(np.linspace(0, P - 1, n_chk).astype(np.int64))
            ctx.wf_plan_score_batch(dev, prio, flags, P, scores, None, stream)
            torch.cuda.synchronize()
            checks.append((what, pkg.scores_to_numpy(scores, P)[idx].tobytes(),
                           lambda o, idx=idx: o.score(win_v, plans.take(idx), threads=T).tobytes()))
        for _ in range(args.warmup):
            ctx.wf_plan_score_batch(dev, prio, flags, P, scores, None, stream)
        torch.cuda.synchronize()
        pev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        for a, b in pev:
            a.record(stream)
            ctx.wf_plan_score_batch(dev, prio, flags, P, scores, None, stream)
            b.record(stream)
        torch.cuda.synchronize()
        ctx.wf_plan_upload_window(win)
        return float(np.mean([a.elapsed_time(b) for a, b in pev]))

    import dataclasses
    # the same plans under the paper's reclamation order (copies held on
    # another device, then next-use distance per reload time, then recency)
    paper_leg = None
    if not args.no_paper_order:
        p_ms = window_leg(dataclasses.replace(win, victim_order=1), "paper reclamation order")
        paper_leg = {"value": round(P / (p_ms * 1e-3), 1), "unit": "plans/s",
                     "kernel_ms": round(p_ms, 4),
                     "note": "the same plans scored with the paper's reclamation order "
                             "(victim_order = 1: a scan over the resident set per reclamation)"}
    # the same plans with a batch limit on every device (several units run
    # at once; memory is checked against the running units)
    batch_leg = None
    if args.batch_limit > 1:
        bl = np.full(D, args.batch_limit, np.int32)
        b_ms = window_leg(dataclasses.replace(win, dev_batch=bl), "batch limits")
        batch_leg = {"value": round(P / (b_ms * 1e-3), 1), "unit": "plans/s",
                     "kernel_ms": round(b_ms, 4), "batch_limit": args.batch_limit,
                     "note": "the same plans with up to batch_limit units per device at once "
                             "(slots, memory of running units, leases on their models)"}

    # the same plans with a replica cap on every model (Sec. 3.5 scale-out):
    # the window moves to the scanned-residency kernel with a per-level check
    replica_leg = None
    if args.replica_cap > 0:
        rc = np.full(win.n_models, args.replica_cap, np.int32)
        r_ms = window_leg(dataclasses.replace(win, model_replica_cap=rc), "replica caps")
        replica_leg = {"value": round(P / (r_ms * 1e-3), 1), "unit": "plans/s",
                       "kernel_ms": round(r_ms, 4), "replica_cap": args.replica_cap,
                       "note": "the same plans with every model capped at replica_cap copies "
                               "held per topological level (status bit 4 beyond it)"}

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        threads = max(1, min(16, os.cpu_count() or 1))
        # the whole batch is about 20 core-seconds of oracle work at the
        # throughput workload; larger batches are sampled evenly
        n_cpu = min(P, args.cpu_sample or 2_000_000)
        idx = np.arange(n_cpu) * max(1, P // n_cpu)
        sample = plans.take(idx)
        t, c = time.perf_counter(), time.process_time()
        oracle.score(win, sample, threads=threads)
        dt, dc = time.perf_counter() - t, time.process_time() - c
        what = "the whole batch" if n_cpu == P else f"{n_cpu} evenly spaced plans of the batch"
        # one thread on a smaller evenly spaced sample
        n1 = min(P, 50_000)
        s1 = plans.take(np.arange(n1) * max(1, P // n1))
        t = time.perf_counter()
        oracle.score(win, s1, threads=1)
        d1 = time.perf_counter() - t
        cpu = {"value": round(n_cpu / dt, 1), "unit": "plans/s", "cores": threads, "kind": "oracle",
               "sample": f"{what}, {threads} threads, {dt:.2f} s wall, {dc:.1f} s CPU "
                         f"({cpu_model()}, {os.cpu_count()} logical CPUs visible)",
               "value_1_thread": round(n1 / d1, 1)}
        # every leg's sampled records against the oracle
        for name, got, ref_fn in checks:
            if got != ref_fn(oracle):
                print(f"[bench] {name}: GPU records differ from the oracle", file=sys.stderr)
                sys.exit(1)
        if checks:
            print(f"[bench] {len(checks)} legs' sampled records bit-exact vs the oracle",
                  file=sys.stderr, flush=True)
    elif checks:
        print("[bench] no CPU-baseline leg: the sampled records were not checked against the oracle",
              file=sys.stderr, flush=True)

    line = {
        "metric": "candidate plans scored/sec at 1 GPU; achieved HBM GB/s vs peak",
        "value": round(value, 1), "unit": "plans/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": "synthetic",
        "config": {"workload": workload.CONFIGS[args.config]["name"], "n_act": N,
                   "n_wf": win.n_wf, "n_dev": D, "n_models": win.n_models, "n_plans": P,
                   "batch_bytes": bpp * P,
                   # batches below the 256 MB last-level cache can be read from it
                   "cache_resident": bool(bpp * P < 256 * 2 ** 20)},
        "roofline": roofline,
        # the bound that holds: vector-instruction issue of the per-device walk
        "valu_roofline": valu_roofline(args.config, P, kernel_ms),
        "cpu_baseline": cpu,
        "search": search,
        "search_rules": search_rules,
        "keys": keys_leg,
        "paper_order": paper_leg,
        "batch_limit": batch_leg,
        "replica_cap": replica_leg,
        "prefix": prefix_leg,
    }
    print(json.dumps(line))
    ctx.close()


if __name__ == "__main__":
    main()
