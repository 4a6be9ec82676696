#!/usr/bin/env python3
"""Benchmark of the eviction-by-design hot path on one MI355X.

The default run measures three workloads (legs) and prints one JSON line:

  llama8b_16k (the headline: the largest workload by bytes): 32 layers x batch 32 x 8 KV heads =
      8192 unit caches of 16384 tokens, 4 query heads per KV head, 25% budget.  One step is one
      eviction (ebd_evict: lambda solve, Poisson mask, compaction) followed by 64 decode steps,
      each appending the new token with pi = 1 (ebd_append_certain; the draw is reused) and
      running certified attention over the retained rows (ebd_attend_certify: Hajek output,
      Theorem 2 variance, eq. (4) radius).
  long_128k (the largest by context): 1024 caches of 131072 tokens, G = 4, 10% budget, floor
      0.005, heavy-tailed scores; one eviction, then 128 decode steps.
  qwen7b_6k: 1792 caches of 6144 tokens, G = 7; an eviction and one certified step at each of
      the 10/25/50% budgets.

`value` is the headline leg's retained-KV bandwidth of certified decode: K + V bytes of every
retained row read by the 64 decode steps, divided by the decode loops' elapsed time (HIP events
around the appends and attention launches).  Inputs are resident in HBM before timing starts.
Each leg reports its own value, fraction of the 8 TB/s HBM peak, evictions/s and the roofline
of its dominant kernel; the oracle runs on a sample of the headline leg's units on the host.
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published peak (8 TB/s)
METRIC = "certified decode attention: retained-KV GB/s (% HBM peak); evictions/sec"


def kernel_sources_hash() -> str:
    """Hash of the library sources with comments and blank space removed (a comment edit does not
    make the committed counter summary stale; any code change does)."""
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2607_21475_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".hpp", ".cpp")):
            src = open(os.path.join(d, f)).read()
            src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)  # block comments
            src = re.sub(r"//[^\n]*", "", src)  # line comments
            h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


def load_traffic(workload: str, kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it is current."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic_%s.json" % workload)
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_sources_hash") != kernel_sources_hash():
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else k.get("bytes_per_launch")


def summarize_pmc(fetch_dir: str, write_dir: str, workload: str, command: str,
                  out_dir: str = "", req_dir: str = "") -> int:
    """Per-launch HBM bytes of the library's kernels from two rocprofv3 --pmc csv runs.

    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are each scaled by what the same counter reads
    for the 1 GiB device copy that --copy-calibration runs (1 GiB read, 1 GiB written).  The
    1 GiB read-only sum it also runs gives a second FETCH_SIZE scale, reported beside the first:
    the two agree when the counter's scale does not depend on the access mix.
    With req_dir (a third run counting the L2's memory read requests by size,
    TCC_EA0_RDREQ_{32B,64B,128B}_sum and TCC_EA0_RDREQ_sum), the fetched bytes are also summed
    directly, 32, 64 or 128 bytes per request, with no calibration; both are reported.
    Writes profiles/hbm_traffic_<workload>.json (read by the benchmark while the kernel sources
    are unchanged), or the same file under out_dir.
    """
    import csv
    import glob
    import statistics

    def load(d, counter):
        """Per library kernel: its readings.  Calibration: the 1 GiB copies and sums that
        copy_calibration runs after every library kernel (the last dispatches of the run; the
        inputs' own copies, earlier in the run, are of other sizes)."""
        per, calib, rcal = {}, [], []
        rows = []
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            rows += [r for r in csv.DictReader(open(f)) if r["Counter_Name"] == counter]
        last_lib = max((int(r["Dispatch_Id"]) for r in rows if "ebd::" in r["Kernel_Name"]), default=-1)
        for r in rows:
            name, v = r["Kernel_Name"], float(r["Counter_Value"])
            if "ebd::" in name:
                k = name.split("(")[0].replace("void ", "").replace("ebd::", "")
                k = k.replace("_kernel", "").split("<")[0]
                per.setdefault(k, []).append(v)
            elif int(r["Dispatch_Id"]) > last_lib and v > 0.25 * (1 << 20):
                if "copyBuffer" in name:
                    calib.append(v)  # the 1 GiB calibration copies
                elif "reduce" in name:
                    rcal.append(v)  # the 1 GiB read-only calibration sums
        return per, calib, rcal

    fetch, fcal, frcal = load(fetch_dir, "FETCH_SIZE")
    write, wcal, _ = load(write_dir, "WRITE_SIZE")
    if not fcal or not wcal:
        print("no calibration copy found in the counter runs", file=sys.stderr)
        return 1
    gib_kib = float(1 << 20)
    fscale = gib_kib / statistics.median(fcal)  # true KiB per counted KiB
    wscale = gib_kib / statistics.median(wcal)
    sized = {}  # per kernel: mean fetched bytes from the request counts, and the sized share
    sized_calib = None
    if req_dir:
        per = {n: load(req_dir, "TCC_EA0_RDREQ_%s_sum" % n) for n in ("32B", "64B", "128B")}
        tot = load(req_dir, "TCC_EA0_RDREQ_sum")
        for k in tot[0]:
            b = sum(w * statistics.mean(per[n][0].get(k, [0.0]))
                    for n, w in (("32B", 32), ("64B", 64), ("128B", 128)))
            cnt = sum(statistics.mean(per[n][0].get(k, [0.0])) for n in ("32B", "64B", "128B"))
            sized[k] = (b, cnt / max(statistics.mean(tot[0][k]), 1.0))
        if per["128B"][1]:
            sized_calib = sum(w * statistics.median(per[n][1]) for n, w in
                              (("32B", 32), ("64B", 64), ("128B", 128)) if per[n][1]) / (1 << 30)
    kernels = {}
    for k in sorted(set(fetch) | set(write)):
        fb = statistics.mean(fetch.get(k, [0.0])) * fscale * 1024
        wb = statistics.mean(write.get(k, [0.0])) * wscale * 1024
        kernels[k] = {"fetch_bytes_per_launch": int(fb), "write_bytes_per_launch": int(wb),
                      "bytes_per_launch": int(fb + wb),
                      "launches_profiled": len(fetch.get(k, []))}
        if k in sized:
            kernels[k]["fetch_bytes_by_request_size"] = int(sized[k][0])
            kernels[k]["sized_request_share"] = round(sized[k][1], 4)
    rec = {"workload": workload, "kernel_sources_hash": kernel_sources_hash(),
           "fetch_scale": fscale, "write_scale": wscale,
           "fetch_scale_read_only_sum": (gib_kib / statistics.median(frcal)) if frcal else None,
           "calibration_copy_gib_by_request_size": sized_calib,
           "kernels": kernels, "command": command}
    out_dir = out_dir or os.path.join(ROOT, "profiles")
    os.makedirs(out_dir, exist_ok=True)
    path = os.path.join(out_dir, "hbm_traffic_%s.json" % workload)
    json.dump(rec, open(path, "w"), indent=1)
    print(json.dumps(rec, indent=1))
    return 0


def summarize_trace(trace_dir: str) -> int:
    """Markdown table of the library's kernel durations from a rocprofv3 --kernel-trace csv run,
    grouped by kernel and launch shape (work-groups x threads), so that the same kernel template
    on different workloads is listed apart."""
    import csv
    import glob
    import statistics

    groups = {}
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            name = r["Kernel_Name"]
            if "ebd::" not in name:
                continue
            name = name.split("(")[0].replace("void ", "")
            wg = int(r["Workgroup_Size_X"])
            key = (name, int(r["Grid_Size_X"]) // max(wg, 1), wg)
            dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3  # ns -> us
            groups.setdefault(key, []).append(dur)
    print("| Kernel | Work-groups x threads | Calls | Average (us) | Min (us) | Max (us) |")
    print("|---|---|---|---|---|---|")
    for (name, nwg, wg), d in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        print("| `%s` | %d x %d | %d | %.1f | %.1f | %.1f |"
              % (name, nwg, wg, len(d), statistics.mean(d), min(d), max(d)))
    return 0


DEFAULT_LEGS = "llama8b_16k,long_128k,qwen7b_6k"
LEG_KERNELS = ("evict_select", "evict_copy", "append_certain", "attend_split", "attend_finalize")


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3,
                    help="timed steps per leg (decode legs: one eviction + all decode steps each)")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--legs", default=DEFAULT_LEGS,
                    help="comma list of workloads; the first is the headline")
    ap.add_argument("--workload", default="", help="a single workload as the only leg")
    ap.add_argument("--decode-steps", type=int, default=0,
                    help="decode steps per eviction for decode legs (0: the workload's)")
    ap.add_argument("--budgets", default="", help="comma list overriding the workload's budgets")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, run a plain 1 GiB device copy and a 1 GiB read-only sum "
                         "(profiler counter scale)")
    ap.add_argument("--scores-steps", type=int, default=3,
                    help="also time the importance-score kernels on the headline leg (0: skip)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate host time for the oracle baseline (0 disables it)")
    ap.add_argument("--cpu-min-gb", type=float, default=1.0,
                    help="least retained KV (GB) the oracle baseline covers")
    ap.add_argument("--cpu-wall-seconds", type=float, default=40.0,
                    help="wall-clock cap of the oracle baseline, host copies included, once its "
                         "least retained KV is covered")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write profiles/hbm_traffic_<workload>.json from rocprofv3 --pmc csv runs")
    ap.add_argument("--pmc-command", default="", help="command recorded in the summary")
    ap.add_argument("--summarize-trace", default="", metavar="TRACE_DIR",
                    help="print the library's kernel durations from a rocprofv3 --kernel-trace run")
    ap.add_argument("--pmc-requests", default="", metavar="REQ_DIR",
                    help="with --summarize-pmc: a third counter run of the read requests by size")
    ap.add_argument("--compare-arms", action="store_true",
                    help="instead of timing: errors of the sampling designs against full attention")
    ap.add_argument("--compare-units", type=int, default=256)
    ap.add_argument("--next-steps", type=int, default=3,
                    help="timed repetitions of the rows built after the hot path (0: skip)")
    ap.add_argument("--replay-grid", action="store_true",
                    help="instead of the legs: the whole replay grid (12096 cells x 8 KV heads, "
                         "G = 1), evicted chunk by chunk, certified in one launch, with coverage "
                         "of the full-cache error per (budget, context)")
    ap.add_argument("--replay-chunks", type=int, default=8,
                    help="chunks the replay grid's full caches are generated and evicted in")
    ap.add_argument("--replay-chunk", type=int, default=-1, metavar="CHUNK",
                    help="instead of a workload: time one chunk (0..7) of 1512 cells of the replay "
                         "grid (8 KV heads per cell, G = 1, per-unit budgets and contexts)")
    args = ap.parse_args()

    if args.summarize_trace:
        return summarize_trace(args.summarize_trace)
    if args.summarize_pmc:
        return summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1],
                             args.workload or args.legs.split(",")[0], args.pmc_command,
                             req_dir=args.pmc_requests)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(units are independent; see the design notes on sharding). Run with --gpus 1.",
              file=sys.stderr)
        return 2

    import torch

    import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.compare_arms:
        wl = synth.WORKLOADS[args.workload or "qwen7b_6k"]
        budgets = [float(b) for b in args.budgets.split(",")] if args.budgets else list(wl.budgets)
        return compare_arms(args, wl, budgets)
    if args.replay_chunk >= 0:
        return replay_chunk(args)
    if args.replay_grid:
        return replay_grid(args)

    names = [args.workload] if args.workload else [w for w in args.legs.split(",") if w]
    legs = {}
    headline = None
    for i, name in enumerate(names):
        wl = synth.WORKLOADS[name]
        t0 = time.time()
        if wl.decode_steps > 1:
            leg = decode_leg(wl, args, headline=(i == 0))
        else:
            leg = budgets_leg(wl, args, headline=(i == 0))
        leg["wall_s"] = round(time.time() - t0, 1)
        print("leg %s: %.1f GB/s (%.3f of peak), %.0f evictions/s, %.1f s" %
              (name, leg["value"], leg["value_frac_hbm"], leg["evictions_per_s"], leg["wall_s"]),
              file=sys.stderr, flush=True)
        legs[name] = leg
        if i == 0:
            headline = leg
        torch.cuda.empty_cache()

    calib = copy_calibration(torch, args.copy_calibration)
    h = headline
    h["roofline"]["measured_copy_gbs"] = calib["copy_gbs"]
    line = {
        "metric": METRIC,
        "value": h["value"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": h["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 K/V/q, fp32 accumulate",
        "data": "synthetic (seeded N(0,1) bf16 K/V/q, 2% heavy-hitter keys x4, 32-query window "
                "importance scores; Pareto(1.5) scores for the long-context leg); the paper's "
                "models and datasets are not used",
        "config": h["config"],
        "value_frac_hbm": h["value_frac_hbm"],
        "evictions_per_s": h["evictions_per_s"],
        "roofline": h["roofline"],
        "cpu_baseline": h.pop("cpu_baseline", None),
        "legs": legs,
        "kernel_sources_hash": kernel_sources_hash(),
    }
    print(json.dumps(line), flush=True)
    return 0


def copy_calibration(torch, under_profiler: bool):
    """A plain 1 GiB device copy (1 GiB read + 1 GiB written) and a 1 GiB read-only sum, outside
    the timed regions: their rates are what this GPU sustains for a copy and for a streaming read
    (the ceilings of the copy-bound and read-bound kernels), and under rocprofv3 --pmc their
    FETCH_SIZE / WRITE_SIZE readings calibrate the counters (each reads a known byte count)."""
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    flt = src.view(torch.float32)
    flt.zero_()
    acc = flt.sum()
    best_c = best_r = float("inf")
    for _ in range(3 if under_profiler else 5):
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record()
        dst.copy_(src)
        e1.record()
        acc = flt.sum()
        e2.record()
        torch.cuda.synchronize()
        best_c = min(best_c, e0.elapsed_time(e1))
        best_r = min(best_r, e1.elapsed_time(e2))
    del src, dst, flt, acc
    return {"copy_gbs": round(2 * (1 << 30) / (best_c * 1e-3) / 1e9, 1),
            "read_gbs": round((1 << 30) / (best_r * 1e-3) / 1e9, 1)}


def _alloc_retained(torch, cache, cap_host, U):
    rows = cap_host[-1]
    return cache.RetainedCache(
        Kc=torch.empty((rows, 128), dtype=torch.bfloat16, device="cuda"),
        Vc=torch.empty((rows, 128), dtype=torch.bfloat16, device="cuda"),
        pic=torch.empty((rows,), dtype=torch.float32, device="cuda"),
        idxc=torch.empty((rows,), dtype=torch.int32, device="cuda"),
        count=torch.empty((U,), dtype=torch.int32, device="cuda"),
        status=torch.empty((U,), dtype=torch.int32, device="cuda"),
        cap_off=torch.tensor(cap_host, dtype=torch.int64, device="cuda"),
        max_cap=max(cap_host[i + 1] - cap_host[i] for i in range(U)))


def _outputs(torch, U, G):
    return {k: torch.empty(s, dtype=torch.float32, device="cuda")
            for k, s in (("y", (U, G, 128)), ("vhat", (U, G)), ("lse", (U, G)), ("b", (U, G)),
                         ("r", (U, G)))}


def _kernel_table(kt, alg, steps):
    """Per kernel: total and average launch time (HIP events on the launch stream) and the
    achieved rate of its algorithmic bytes."""
    kern = {}
    for k, (ms, launches) in kt.items():
        if launches == 0:
            continue
        avg_ms = ms / launches
        gbs = alg[k] * steps / (ms * 1e-3) / 1e9
        kern[k] = dict(total_ms=round(ms, 4), launches=int(launches), avg_us=round(avg_ms * 1e3, 2),
                       alg_bytes_per_step=int(alg[k]), achieved_gbs=round(gbs, 1),
                       frac_hbm=round(gbs / HBM_PEAK_GBS, 4))
    return kern


def _roofline(kern, alg, steps, workload):
    dom = max(kern, key=lambda k: kern[k]["total_ms"])
    dk = kern[dom]
    launch_bytes = alg[dom] / (dk["launches"] / steps)
    return {"bound": "hbm", "achieved": dk["achieved_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(dk["achieved_gbs"] / HBM_PEAK_GBS, 4),
            "traffic": load_traffic(workload, dom), "kernel": dom,
            "alg_bytes_per_launch": int(launch_bytes), "avg_launch_us": dk["avg_us"]}


def decode_leg(wl, args, headline: bool):
    """Evict once, then the workload's decode steps (append a pi = 1 token, certified attention)
    per timed step; HIP events bracket the eviction and the decode loop of every step."""
    import torch

    import synth
    import paper_2607_21475_amd as ebd
    from paper_2607_21475_amd import cache

    U, n, G = wl.units, wl.context, wl.group
    T = args.decode_steps or wl.decode_steps
    budget = float(args.budgets.split(",")[0]) if args.budgets else wl.budgets[0]
    t0 = time.time()
    inp = synth.make_workload_inputs(wl, seed=args.seed, device="cuda")
    cap_host = cache.plan_capacity([n] * U, budget, wl.n_sink, wl.n_recent, extra=T, pi_min=wl.pi_min)
    rc = _alloc_retained(torch, cache, cap_host, U)
    ep = ebd.evict_params(U, n, rc.max_cap, inp["seq_off"], rc.cap_off, wl.n_sink, wl.n_recent,
                          budget, None, wl.pi_min, 0, args.seed, None, 0)
    ews = ebd.workspace(ebd.ebd_workspace_size(ebd.EBD_WS_EVICT, ep))
    apar = ebd.attend_params(U, G, rc.max_cap, rc.cap_off)
    aws_bytes = ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, apar)
    aws = ebd.workspace(aws_bytes)
    o = _outputs(torch, U, G)
    ast = torch.empty((U,), dtype=torch.int32, device="cuda")
    # decode-step inputs: a query block, a new key/value row and its position per step
    qs = torch.stack([synth.make_queries(U, G, seed=args.seed + 30000 + t, device="cuda")
                      for t in range(T)])
    kn = torch.stack([synth.make_queries(U, 1, seed=args.seed + 10000 + t, device="cuda")[:, 0]
                      for t in range(T)])
    vn = torch.stack([synth.make_queries(U, 1, seed=args.seed + 20000 + t, device="cuda")[:, 0]
                      for t in range(T)])
    pos = (n + torch.arange(T, dtype=torch.int32, device="cuda"))[:, None].expand(T, U).contiguous()
    torch.cuda.synchronize()
    print("%s: inputs ready, %d units x %d tokens, G=%d, %d decode steps (%.1f s)"
          % (wl.name, U, n, G, T, time.time() - t0), file=sys.stderr, flush=True)

    def evict():
        ebd.ebd_evict(ep, inp["scores"], inp["K"], inp["V"], rc.Kc, rc.Vc, rc.pic, rc.idxc,
                      rc.count, rc.status, ews)

    def decode():
        for t in range(T):
            ebd.ebd_append_certain(U, rc.cap_off, rc.count, kn[t], vn[t], rc.Kc, rc.Vc, rc.pic,
                                   rc.idxc, pos[t], rc.status)
            ebd.ebd_attend_certify(apar, qs[t], rc.Kc, rc.Vc, rc.pic, rc.count, o["y"], o["vhat"],
                                   o["lse"], aws, brange=o["b"], radius=o["r"], status=ast)

    for _ in range(args.warmup):
        evict()
        decode()
    evict()
    torch.cuda.synchronize()
    base = rc.count.cpu().numpy().astype(np.int64)
    decode()
    torch.cuda.synchronize()
    if (rc.status.cpu().numpy() & ebd.EBD_ST_CAP_OVERFLOW).any() or ast.cpu().numpy().any():
        raise RuntimeError("%s: capacity overflow or unseen rows" % wl.name)

    ebd.ebd_timing_enable(True)
    for k in LEG_KERNELS:
        ebd.ebd_timing_read(k)  # clear
    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    torch.cuda.synchronize()
    for k in range(K):
        ev[k][0].record()
        evict()
        ev[k][1].record()
        decode()
        ev[k][2].record()
    torch.cuda.synchronize()
    kt = {k: ebd.ebd_timing_read(k) for k in LEG_KERNELS}
    ebd.ebd_timing_enable(False)
    evict_ms = sum(e[0].elapsed_time(e[1]) for e in ev)
    decode_ms = sum(e[1].elapsed_time(e[2]) for e in ev)
    total_ms = ev[0][0].elapsed_time(ev[-1][2])

    rows0 = int(base.sum())
    kv_step = 512 * (T * rows0 + U * T * (T + 1) // 2)  # K + V of every row each decode step reads
    value = kv_step * K / (decode_ms * 1e-3) / 1e9
    att_rows = T * rows0 + U * T * (T + 1) // 2  # summed over the decode steps of one step
    gathers = kt["evict_copy"][1] == 0
    fused = kt["attend_finalize"][1] == 0  # the split kernel finalized every unit itself
    alg = {
        "evict_select": 4 * U * n + 8 * rows0 + (1024 * rows0 if gathers else 0),
        "evict_copy": 0 if gathers else 1024 * rows0,
        "append_certain": T * U * 512,
        "attend_split": 516 * att_rows + T * U * G * 256 + (T * U * G * 528 if fused else 0),
        "attend_finalize": 0 if fused else T * U * G * 528,
    }
    kern = _kernel_table(kt, alg, K)
    t_evict_k = (kt["evict_select"][0] + kt["evict_copy"][0]) * 1e-3
    leg = {
        "value": round(value, 1),
        "unit": "GB/s",
        "value_frac_hbm": round(value / HBM_PEAK_GBS, 4),
        "ms_per_step": round(total_ms / K, 3),
        "decode_ms_per_step": round(decode_ms / K, 3),
        "decode_step_us": round(decode_ms / K / T * 1e3, 2),
        "evict_ms_per_step": round(evict_ms / K, 4),
        "evictions_per_s": round(U * K / (evict_ms * 1e-3), 1),
        "evictions_per_s_kernels": round(U * K / t_evict_k, 1),
        "evicted_tokens_per_s": round(U * n * K / (evict_ms * 1e-3), 1),
        "evict_gbs": round((4 * U * n + 1032 * rows0) * K / (evict_ms * 1e-3) / 1e9, 1),
        "config": {"workload": wl.name, "description": wl.description, "units": U, "context": n,
                   "group": G, "head_dim": 128, "budgets": [budget], "pi_min": wl.pi_min,
                   "protected": [wl.n_sink, wl.n_recent], "scores": wl.scores,
                   "decode_steps": T, "step": "one eviction, then %d decode steps (append a "
                   "pi = 1 token, certified attention)" % T, "parallelism": "single GPU"},
        "retained_rows_after_eviction": rows0,
        "mean_retained_per_unit": round(rows0 / U, 1),
        "fused_finalize": bool(fused),
        "evict_select_gathers": bool(gathers),
        "range_term_rescans_last_step": cache.rescans(aws, U, G),
        "direct_variance_heads_last_step": cache.direct_variances(aws, U, G),
        "kernels": kern,
        "roofline": _roofline(kern, alg, K, wl.name),
    }
    if headline and args.scores_steps > 0:
        leg["importance_scores"] = time_scores(args, wl, inp, ebd, torch)
    if headline and args.cpu_seconds > 0:
        # a clean state: the eviction again (deterministic, now also writing every position's pi)
        # and the first decode query, no appends
        pf = torch.empty((U * n,), dtype=torch.float32, device="cuda")
        ebd.ebd_evict(ep, inp["scores"], inp["K"], inp["V"], rc.Kc, rc.Vc, rc.pic, rc.idxc,
                      rc.count, rc.status, ews, pi_full=pf)
        o0 = _outputs(torch, U, G)
        ebd.ebd_attend_certify(apar, qs[0], rc.Kc, rc.Vc, rc.pic, rc.count, o0["y"], o0["vhat"],
                               o0["lse"], aws, brange=o0["b"], radius=o0["r"])
        torch.cuda.synchronize()
        leg["cpu_baseline"] = cpu_baseline(wl, args, inp, rc, pf, qs[0], o0, budget, torch)
    del inp, rc, qs, kn, vn, o
    return leg


def budgets_leg(wl, args, headline: bool):
    """One eviction and one certified decode step at each of the workload's budgets per timed
    step (evictions first, so that no retained cache is still in the last-level cache when
    attention reads it)."""
    import torch

    import synth
    import paper_2607_21475_amd as ebd
    from paper_2607_21475_amd import cache

    U, n, G = wl.units, wl.context, wl.group
    budgets = [float(b) for b in args.budgets.split(",")] if args.budgets else list(wl.budgets)
    lengths = [n] * U
    t0 = time.time()
    inp = synth.make_workload_inputs(wl, seed=args.seed, device="cuda")
    torch.cuda.synchronize()
    print("%s: inputs ready, %d units x %d tokens, G=%d (%.1f s)" % (wl.name, U, n, G, time.time() - t0),
          file=sys.stderr, flush=True)
    plans = []
    for b in budgets:
        cap_host = cache.plan_capacity(lengths, b, wl.n_sink, wl.n_recent, pi_min=wl.pi_min)
        rc = _alloc_retained(torch, cache, cap_host, U)
        ep = ebd.evict_params(U, n, rc.max_cap, inp["seq_off"], rc.cap_off, wl.n_sink, wl.n_recent,
                              b, None, wl.pi_min, 0, args.seed, None, 0)
        ews = ebd.workspace(ebd.ebd_workspace_size(ebd.EBD_WS_EVICT, ep))
        ap_ = ebd.attend_params(U, G, rc.max_cap, rc.cap_off)
        aws_bytes = ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, ap_)
        plans.append(dict(budget=b, rc=rc, ep=ep, ews=ews, ap=ap_, aws=ebd.workspace(aws_bytes),
                          out=_outputs(torch, U, G)))

    def evict_all():
        for p in plans:
            rc = p["rc"]
            ebd.ebd_evict(p["ep"], inp["scores"], inp["K"], inp["V"], rc.Kc, rc.Vc, rc.pic, rc.idxc,
                          rc.count, rc.status, p["ews"])

    def attend_all():
        for p in plans:
            rc, o = p["rc"], p["out"]
            ebd.ebd_attend_certify(p["ap"], inp["q"], rc.Kc, rc.Vc, rc.pic, rc.count, o["y"],
                                   o["vhat"], o["lse"], p["aws"], brange=o["b"], radius=o["r"])

    for _ in range(args.warmup):
        evict_all()
        attend_all()
    torch.cuda.synchronize()
    ebd.ebd_timing_enable(True)
    for p in plans:  # which budgets' evictions gather their rows inside evict_select
        ebd.ebd_timing_read("evict_copy")
        rc = p["rc"]
        ebd.ebd_evict(p["ep"], inp["scores"], inp["K"], inp["V"], rc.Kc, rc.Vc, rc.pic, rc.idxc,
                      rc.count, rc.status, p["ews"])
        torch.cuda.synchronize()
        p["gathers"] = ebd.ebd_timing_read("evict_copy")[1] == 0
        # ... and whose attention finalizes inside the split kernel (no attend_finalize launch)
        ebd.ebd_timing_read("attend_finalize")
        o = p["out"]
        ebd.ebd_attend_certify(p["ap"], inp["q"], rc.Kc, rc.Vc, rc.pic, rc.count, o["y"],
                               o["vhat"], o["lse"], p["aws"], brange=o["b"], radius=o["r"])
        torch.cuda.synchronize()
        p["fused"] = ebd.ebd_timing_read("attend_finalize")[1] == 0
    for p in plans:
        if (p["rc"].status.cpu().numpy() & ebd.EBD_ST_CAP_OVERFLOW).any():
            raise RuntimeError("capacity overflow at budget %s" % p["budget"])
    for k in LEG_KERNELS:
        ebd.ebd_timing_read(k)  # clear
    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    torch.cuda.synchronize()
    for k in range(K):
        ev[k][0].record()
        evict_all()
        ev[k][1].record()
        attend_all()
        ev[k][2].record()
    torch.cuda.synchronize()
    kt = {k: ebd.ebd_timing_read(k) for k in LEG_KERNELS}
    ebd.ebd_timing_enable(False)
    evict_ms = sum(e[0].elapsed_time(e[1]) for e in ev)
    attend_ms = sum(e[1].elapsed_time(e[2]) for e in ev)
    total_ms = ev[0][0].elapsed_time(ev[-1][2])

    per_budget, retained_total, gathered = [], 0, 0
    for p in plans:
        cnt = p["rc"].count.cpu().numpy().astype(np.int64)
        per_budget.append(dict(budget=p["budget"], retained_rows=int(cnt.sum()),
                               mean_retained_per_unit=round(float(cnt.mean()), 1),
                               range_term_rescans=cache.rescans(p["aws"], U, G),
                               direct_variance_heads=cache.direct_variances(p["aws"], U, G),
                               fused_finalize=bool(p["fused"]), select_gathers=bool(p["gathers"])))
        retained_total += int(cnt.sum())
        gathered += int(cnt.sum()) if p["gathers"] else 0
    nb = len(plans)
    nfused = sum(1 for p in plans if p["fused"])
    alg = {
        "evict_select": 4 * U * n * nb + 8 * retained_total + 1024 * gathered,
        "evict_copy": 1024 * (retained_total - gathered),
        "append_certain": 0,
        "attend_split": 516 * retained_total + nb * U * G * 256 + nfused * U * G * 528,
        "attend_finalize": (nb - nfused) * U * G * 528,
    }
    kern = _kernel_table(kt, alg, K)
    value = 512 * retained_total * K / (attend_ms * 1e-3) / 1e9
    leg = {
        "value": round(value, 1),
        "unit": "GB/s",
        "value_frac_hbm": round(value / HBM_PEAK_GBS, 4),
        "ms_per_step": round(total_ms / K, 4),
        "attend_ms_per_step": round(attend_ms / K, 4),
        "evict_ms_per_step": round(evict_ms / K, 4),
        "evictions_per_s": round(U * nb * K / (evict_ms * 1e-3), 1),
        "evicted_tokens_per_s": round(U * n * nb * K / (evict_ms * 1e-3), 1),
        "config": {"workload": wl.name, "description": wl.description, "units": U, "context": n,
                   "group": G, "head_dim": 128, "budgets": budgets, "pi_min": wl.pi_min,
                   "protected": [wl.n_sink, wl.n_recent], "scores": wl.scores,
                   "step": "an eviction and one certified decode step at every budget",
                   "parallelism": "single GPU"},
        "per_budget": per_budget,
        "kernels": kern,
        "roofline": _roofline(kern, alg, K, wl.name),
    }
    if headline and args.scores_steps > 0:
        leg["importance_scores"] = time_scores(args, wl, inp, ebd, torch)
    if args.next_steps > 0:
        leg["next_rows"] = next_rows(args, wl, inp, plans, ebd, torch)
    del inp, plans
    return leg


def time_scores(args, wl, inp, ebd, torch):
    """The step before the path (not part of `value`): importance scores from 32 observation-
    window queries per unit, timed alone."""
    import synth

    U, n = wl.units, wl.context
    qw = synth.make_queries(U, 32, seed=args.seed + 7, device="cuda")
    sp_ = ebd.scores_params(U, 32, n, inp["seq_off"])
    sws = ebd.workspace(ebd.ebd_workspace_size(ebd.EBD_WS_SCORES, sp_))
    sco = torch.empty_like(inp["scores"])
    ebd.ebd_scores(sp_, qw, inp["K"], sco, sws)
    torch.cuda.synchronize()
    ebd.ebd_timing_enable(True)
    for k in ("scores_stats", "scores_accum"):
        ebd.ebd_timing_read(k)
    for _ in range(args.scores_steps):
        ebd.ebd_scores(sp_, qw, inp["K"], sco, sws)
    torch.cuda.synchronize()
    st = {k: ebd.ebd_timing_read(k) for k in ("scores_stats", "scores_accum")}
    ebd.ebd_timing_enable(False)
    toks = U * n
    # each pass reads every cached key once (256 B); the second also writes the score (4 B)
    sb = {"scores_stats": 256 * toks, "scores_accum": 260 * toks}
    imp = {"queries_per_unit": 32, "steps": args.scores_steps}
    tot_ms = 0.0
    for k, (ms, nl) in st.items():
        avg = ms / max(nl, 1)
        tot_ms += ms
        imp[k] = {"avg_us": round(avg * 1e3, 2), "achieved_gbs": round(sb[k] / (avg * 1e-3) / 1e9, 1),
                  "frac_hbm": round(sb[k] / (avg * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    imp["tokens_per_s"] = round(toks * args.scores_steps / (tot_ms * 1e-3), 1)
    del qw, sws, sco
    return imp


def next_rows(args, wl, inp, plans, ebd, torch):
    """Timing of the rows built after the hot path, on the benchmark's own inputs: the
    per-block variance contributions and the deployed certificate step over the middle budget's
    retained caches and attention outputs, then the other sampling designs (fixed-size
    systematic, top-k, uniform) evicting the same units at every budget."""
    U, n, G = wl.units, wl.context, wl.group
    res = {}
    p = plans[len(plans) // 2]
    rc, o = p["rc"], p["out"]
    retained = int(rc.count.sum().item())
    nblocks = (n + 63) // 64
    blocks = torch.empty((U, nblocks), dtype=torch.float32, device="cuda")
    # units are (layer, sequence, KV head) with the KV head fastest; each holds G query heads
    useq = torch.tensor([(u // wl.kv_heads) % wl.batch for u in range(U)], dtype=torch.int32,
                        device="cuda")
    uh0 = torch.tensor([(u % wl.kv_heads) * G for u in range(U)], dtype=torch.int32, device="cuda")
    cert = torch.zeros(wl.batch, dtype=torch.float32, device="cuda")
    ebd.ebd_block_contributions(U, G, nblocks, rc.max_cap, rc.cap_off, inp["q"], rc.Kc, rc.Vc,
                                rc.pic, rc.idxc, rc.count, o["y"], o["lse"], blocks)
    torch.cuda.synchronize()
    ebd.ebd_timing_enable(True)
    for k in ("block_contrib", "cert_step"):
        ebd.ebd_timing_read(k)
    for _ in range(args.next_steps):
        ebd.ebd_block_contributions(U, G, nblocks, rc.max_cap, rc.cap_off, inp["q"], rc.Kc, rc.Vc,
                                    rc.pic, rc.idxc, rc.count, o["y"], o["lse"], blocks)
        ebd.ebd_certificate_step(U, G, wl.batch, useq, o["r"], cert, unit_head0=uh0)
    torch.cuda.synchronize()
    bc, cs = ebd.ebd_timing_read("block_contrib"), ebd.ebd_timing_read("cert_step")
    bc_us = bc[0] / max(bc[1], 1) * 1e3
    bbytes = 520 * retained * ((G + 7) // 8)  # K, V, pi, index per retained row and head block
    res["block_contrib"] = {"budget": p["budget"], "avg_us": round(bc_us, 2),
                            "alg_bytes_per_launch": bbytes,
                            "achieved_gbs": round(bbytes / (bc_us * 1e-6) / 1e9, 1),
                            "frac_hbm": round(bbytes / (bc_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    res["cert_step"] = {"avg_us": round(cs[0] / max(cs[1], 1) * 1e3, 2), "sequences": wl.batch}
    designs = {}
    for name, design in (("systematic", ebd.EBD_DESIGN_SYSTEMATIC), ("topk", ebd.EBD_DESIGN_TOPK),
                         ("uniform", ebd.EBD_DESIGN_UNIFORM)):
        eps = [ebd.evict_params(U, n, q["rc"].max_cap, inp["seq_off"], q["rc"].cap_off, wl.n_sink,
                                wl.n_recent, q["budget"], None, wl.pi_min, 0, args.seed, None, 0,
                                design) for q in plans]

        def evict_all():
            for q, ep in zip(plans, eps):
                r = q["rc"]
                ebd.ebd_evict(ep, inp["scores"], inp["K"], inp["V"], r.Kc, r.Vc, r.pic, r.idxc,
                              r.count, r.status, q["ews"])

        evict_all()
        torch.cuda.synchronize()
        for k in ("evict_select", "evict_copy"):
            ebd.ebd_timing_read(k)
        for _ in range(args.next_steps):
            evict_all()
        torch.cuda.synchronize()
        ms = sum(ebd.ebd_timing_read(k)[0] for k in ("evict_select", "evict_copy"))
        calls = args.next_steps * len(plans)
        overflow = any(bool((q["rc"].status.cpu().numpy() & ebd.EBD_ST_CAP_OVERFLOW).any())
                       for q in plans)
        designs[name] = {"evict_us_per_call": round(ms / calls * 1e3, 2),
                         "evictions_per_s": round(U * calls / (ms * 1e-3), 1),
                         "retained_rows": [int(q["rc"].count.sum().item()) for q in plans],
                         "capacity_overflow": overflow}
    ebd.ebd_timing_enable(False)
    res["designs"] = designs
    return res


def replay_grid(args) -> int:
    """The whole replay grid: 12096 cells x 8 KV heads = 96768 units (G = 1), cell c with budget
    5/10/15/25/50% (c mod 5) and context 2048/6144/16384 ((c div 5) mod 3).  Their full caches
    (406 GB) exceed the GPU's memory, so they are generated and evicted chunk by chunk into one
    compacted cache of all units; while a chunk's full cache is resident, its full-cache output
    y (eq. (1)) is computed by the certified kernel itself over the uncompacted rows with pi = 1
    (the Hajek output then is eq. (1), and the certificate is 0).  Then one certified step over
    all 96768 units (one launch per kernel) gives yhat and the radius r, and coverage
    |yhat - y| / |y| <= r, the median error and radius and the Spearman correlation of radius and
    error are reported per (budget, context).  Timed: the chunk evictions (HIP events) and the
    all-unit certified step (args.steps repetitions)."""
    import torch

    import synth
    import paper_2607_21475_amd as ebd
    from paper_2607_21475_amd import cache

    H = synth.REPLAY_KV_HEADS
    ncell = synth.REPLAY_CELLS
    cells = [synth.replay_cell(c) for c in range(ncell)]
    lengths = [ctx for (_, ctx, _, _) in cells for _ in range(H)]
    budgets = [b for (b, _, _, _) in cells for _ in range(H)]
    U = len(lengths)
    t0 = time.time()
    cap_host = cache.plan_capacity(lengths, budgets, 4, 64, pi_min=0.01)
    rc = _alloc_retained(torch, cache, cap_host, U)
    q = synth.make_queries(U, 1, seed=args.seed + 7, device="cuda")
    bpu = torch.tensor(budgets, dtype=torch.float32, device="cuda")
    yfull = torch.empty((U, 1, 128), dtype=torch.float32, device="cuda")
    per = -(-ncell // args.replay_chunks)
    ev_ms, ev_calls, full_rows = 0.0, 0, 0
    for k in range(args.replay_chunks):
        c0, c1 = k * per, min(ncell, (k + 1) * per)
        if c0 >= c1:
            break
        u0, u1 = c0 * H, c1 * H
        lens = lengths[u0:u1]
        Uc = u1 - u0
        K, V, seq_off = synth.make_cache(lens, seed=args.seed + 100 + k, device="cuda")
        sc = synth.window_scores(K, seq_off, seed=args.seed + 200 + k)
        r0, r1 = cap_host[u0], cap_host[u1]
        coff = torch.tensor([x - r0 for x in cap_host[u0:u1 + 1]], dtype=torch.int64, device="cuda")
        maxcap = max(cap_host[i + 1] - cap_host[i] for i in range(u0, u1))
        ep = ebd.evict_params(Uc, max(lens), maxcap, seq_off, coff, 4, 64, 0.0, bpu[u0:u1], 0.01, 0,
                              args.seed + k, None, 0)
        ews = ebd.workspace(ebd.ebd_workspace_size(ebd.EBD_WS_EVICT, ep))

        def evict():
            ebd.ebd_evict(ep, sc, K, V, rc.Kc[r0:r1], rc.Vc[r0:r1], rc.pic[r0:r1], rc.idxc[r0:r1],
                          rc.count[u0:u1], rc.status[u0:u1], ews)

        evict()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            evict()
        e1.record()
        # full-cache reference output: every row kept with pi = 1
        ones = torch.ones((K.shape[0],), dtype=torch.float32, device="cuda")
        nfull = torch.tensor(lens, dtype=torch.int32, device="cuda")
        fp = ebd.attend_params(Uc, 1, max(lens), seq_off)
        fws = ebd.workspace(ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, fp))
        scratch = _outputs(torch, Uc, 1)
        ebd.ebd_attend_certify(fp, q[u0:u1], K, V, ones, nfull, yfull[u0:u1], scratch["vhat"],
                               scratch["lse"], fws)
        torch.cuda.synchronize()
        ev_ms += e0.elapsed_time(e1)
        ev_calls += args.steps
        full_rows += int(K.shape[0])
        print("replay grid: chunk %d cells %d..%d, %d units, %.1f GB of full cache (%.0f s)"
              % (k, c0, c1, Uc, 512 * K.shape[0] / 1e9, time.time() - t0), file=sys.stderr, flush=True)
        del K, V, seq_off, sc, ones, nfull, fws, scratch, ews
        torch.cuda.empty_cache()
    if (rc.status.cpu().numpy() & ebd.EBD_ST_CAP_OVERFLOW).any():
        raise RuntimeError("capacity overflow in the replay grid")
    retained = int(rc.count.sum().item())

    # one certified step over every unit
    ap_ = ebd.attend_params(U, 1, rc.max_cap, rc.cap_off)
    aws = ebd.workspace(ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, ap_))
    o = _outputs(torch, U, 1)
    ast = torch.empty((U,), dtype=torch.int32, device="cuda")

    def attend():
        ebd.ebd_attend_certify(ap_, q, rc.Kc, rc.Vc, rc.pic, rc.count, o["y"], o["vhat"], o["lse"],
                               aws, brange=o["b"], radius=o["r"], status=ast)

    attend()
    torch.cuda.synchronize()
    ebd.ebd_timing_enable(True)
    for k in ("attend_split", "attend_finalize"):
        ebd.ebd_timing_read(k)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        attend()
    e1.record()
    torch.cuda.synchronize()
    kt = {k: ebd.ebd_timing_read(k) for k in ("attend_split", "attend_finalize")}
    ebd.ebd_timing_enable(False)
    att_ms = e0.elapsed_time(e1) / args.steps
    if ast.cpu().numpy().any():
        raise RuntimeError("rows the certified step could not see")

    # coverage of the full-cache error, per (budget, context)
    err = (torch.linalg.norm(o["y"] - yfull, dim=2) / torch.linalg.norm(yfull, dim=2)).flatten()
    r = o["r"].flatten()
    cell_of = torch.arange(U, device="cuda") // H
    bi, ci = cell_of % 5, (cell_of // 5) % 3
    table = []
    for b in range(5):
        for c in range(3):
            m = (bi == b) & (ci == c)
            e_, r_ = err[m], r[m]
            table.append({"budget": synth.REPLAY_BUDGETS[b], "context": synth.REPLAY_CONTEXTS[c],
                          "units": int(m.sum()),
                          "coverage": round(float((e_ <= r_).float().mean()), 4),
                          "median_rel_err": float("%.4g" % float(e_.median())),
                          "median_radius": float("%.4g" % float(r_.median())),
                          "spearman_radius_error": round(_spearman(r_, e_), 4)})
    kv = 512 * retained
    line = {"mode": "replay_grid", "cells": ncell, "units": U, "group": 1,
            "full_cache_rows": full_rows, "full_cache_gb": round(512 * full_rows / 1e9, 1),
            "retained_rows": retained, "retained_kv_gb": round(kv / 1e9, 2),
            "chunks": args.replay_chunks, "steps": args.steps,
            "evict_ms_per_pass": round(ev_ms / ev_calls * args.replay_chunks, 3),
            "evictions_per_s": round(U * ev_calls / args.replay_chunks / (ev_ms * 1e-3), 1),
            "evict_gbs": round((4 * full_rows + 1032 * retained) * ev_calls / args.replay_chunks
                               / (ev_ms * 1e-3) / 1e9, 1),
            "attend_ms": round(att_ms, 3),
            "attend_launches_per_step": {k: kt[k][1] // args.steps for k in kt},
            "attend_kernel_ms": {k: round(kt[k][0] / max(kt[k][1], 1), 3) for k in kt},
            "retained_kv_gbs": round(kv / (att_ms * 1e-3) / 1e9, 1),
            "retained_kv_frac_hbm": round(kv / (att_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "coverage_all": round(float((err <= r).float().mean()), 4),
            "per_budget_context": table,
            "data": "synthetic caches in the replay grid's shapes (the paper's models and prompts "
                    "are not used); coverage is reported, not gated"}
    print(json.dumps(line), flush=True)
    return 0


def replay_chunk(args) -> int:
    """One chunk of the replay grid as one eviction and one certified decode step: cells
    c0 .. c0 + 1511 (c0 = 1512 x chunk), 8 KV heads each (G = 1), every cell with its own budget
    (5 .. 50%) and context (2048 / 6144 / 16384); its full caches (about 50 GB) fit one GPU, the
    whole grid's (406 GB) are evicted chunk by chunk."""
    import torch

    import synth
    import paper_2607_21475_amd as ebd
    from paper_2607_21475_amd import cache

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    ncell = 1512
    c0 = ncell * args.replay_chunk
    cells = [synth.replay_cell(c) for c in range(c0, c0 + ncell)]
    H = synth.REPLAY_KV_HEADS
    lengths = [ctx for (_, ctx, _, _) in cells for _ in range(H)]
    budgets = [b for (b, _, _, _) in cells for _ in range(H)]
    U = len(lengths)
    K, V, seq_off = synth.make_cache(lengths, seed=args.seed + 5, device="cuda")
    sc = synth.window_scores(K, seq_off, seed=args.seed + 6)
    q = synth.make_queries(U, 1, seed=args.seed + 7, device="cuda")
    bpu = torch.tensor(budgets, dtype=torch.float32, device="cuda")
    out = cache.evict(K, V, sc, seq_off, lengths, budget_per_unit=bpu, seed=args.seed)
    res = cache.attend_certify(out, q)
    torch.cuda.synchronize()
    if (out.status.cpu().numpy() & ebd.EBD_ST_CAP_OVERFLOW).any():
        raise RuntimeError("capacity overflow in the replay chunk")
    retained = int(out.count.sum().item())
    names = ("evict_select", "evict_copy", "attend_split", "attend_finalize")
    ebd.ebd_timing_enable(True)
    for k in names:
        ebd.ebd_timing_read(k)
    for _ in range(args.steps):
        out2 = cache.evict(K, V, sc, seq_off, lengths, budget_per_unit=bpu, seed=args.seed)
        del out2
        cache.attend_certify(out, q, ws=res["ws"])
    torch.cuda.synchronize()
    t = {k: ebd.ebd_timing_read(k) for k in names}
    ebd.ebd_timing_enable(False)
    att_ms = (t["attend_split"][0] + t["attend_finalize"][0]) / args.steps
    ev_ms = (t["evict_select"][0] + t["evict_copy"][0]) / args.steps
    kv = 512 * retained
    line = {"mode": "replay_chunk", "chunk": args.replay_chunk, "cells": ncell, "units": U,
            "group": 1, "rows": int(sum(lengths)), "retained_rows": retained, "steps": args.steps,
            "attend_us": round(att_ms * 1e3, 1),
            "attend_launches_per_call": {k: t[k][1] // args.steps for k in names[2:]},
            "retained_kv_gbs": round(kv / (att_ms * 1e-3) / 1e9, 1),
            "retained_kv_frac_hbm": round(kv / (att_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "evict_us": round(ev_ms * 1e3, 1),
            "evict_launches_per_call": {k: t[k][1] // args.steps for k in names[:2]},
            "evictions_per_s": round(U / (ev_ms * 1e-3), 1),
            "evict_gbs": round((4 * sum(lengths) + 1032 * retained) / (ev_ms * 1e-3) / 1e9, 1)}
    print(json.dumps(line), flush=True)
    return 0


def compare_arms(args, wl, budgets) -> int:
    """Relative error of each sampling design against full attention on a sample of units, and
    the certificate's coverage; then the value-permutation demonstration for top-k: permuting
    the evicted values leaves every retained-set statistic of top-k unchanged while its true
    error moves (comparative only; synthetic caches stand in for the paper's models)."""
    import torch

    import paper_2607_21475_amd as ebd
    import synth
    from paper_2607_21475_amd import cache

    U = min(args.compare_units, wl.units)
    n, G = wl.context, wl.group
    inp = synth.make_workload_inputs(wl, units=U, seed=args.seed, device="cuda")
    lengths = [n] * U
    kw = dict(n_sink=wl.n_sink, n_recent=wl.n_recent, pi_min=wl.pi_min, seed=args.seed)

    def full_output(V):
        full = cache.evict(inp["K"], V, inp["scores"], inp["seq_off"], lengths, budget_frac=1.0, **kw)
        return cache.attend_certify(full, inp["q"])["y"]

    def rel_err(y, yref):
        return (torch.linalg.norm(y - yref, dim=2) / torch.linalg.norm(yref, dim=2)).flatten()

    yref = full_output(inp["V"])
    arms = (("poisson_hajek", ebd.EBD_DESIGN_POISSON, True),
            ("poisson_no_offset", ebd.EBD_DESIGN_POISSON, False),
            ("systematic_hajek", ebd.EBD_DESIGN_SYSTEMATIC, True),
            ("topk", ebd.EBD_DESIGN_TOPK, True),
            ("uniform_hajek", ebd.EBD_DESIGN_UNIFORM, True))
    table = []
    for b in budgets:
        row = {"budget": b}
        for name, design, offset in arms:
            rc = cache.evict(inp["K"], inp["V"], inp["scores"], inp["seq_off"], lengths,
                             budget_frac=b, design=design, **kw)
            res = cache.attend_certify(rc, inp["q"], offset=offset)
            err = rel_err(res["y"], yref)
            ent = {"median_rel_err": round(float(err.median()), 5),
                   "mean_retained": round(float(rc.count.float().mean()), 1)}
            if design != ebd.EBD_DESIGN_TOPK:
                r = res["r"].flatten()
                ent["coverage"] = round(float((err <= r).float().mean()), 4)
                ent["median_radius"] = round(float(r.median()), 5)
                ent["spearman_radius_error"] = round(_spearman(r, err), 4)
            row[name] = ent
        table.append(row)

    # Theorem 1 by construction: permute each unit's evicted value rows (top-k at the first budget)
    b = budgets[0]
    rc = cache.evict(inp["K"], inp["V"], inp["scores"], inp["seq_off"], lengths, budget_frac=b,
                     design=ebd.EBD_DESIGN_TOPK, **kw)
    y_top = cache.attend_certify(rc, inp["q"])["y"]
    cnt = rc.count.cpu().tolist()
    coff = rc.cap_off.cpu().tolist()
    idx = rc.idxc.cpu()
    g = torch.Generator(device="cpu")
    g.manual_seed(args.seed + 99)
    errs, same = [], True
    for world in range(6):
        perm = torch.arange(U * n)
        for u in range(U):
            kept = torch.zeros(n, dtype=torch.bool)
            kept[idx[coff[u]:coff[u] + cnt[u]].long()] = True
            ev = torch.nonzero(~kept).flatten() + u * n
            perm[ev] = ev[torch.randperm(ev.numel(), generator=g)]
        Vp = inp["V"][perm.to("cuda")]
        rc2 = cache.evict(inp["K"], Vp, inp["scores"], inp["seq_off"], lengths, budget_frac=b,
                          design=ebd.EBD_DESIGN_TOPK, **kw)
        y2 = cache.attend_certify(rc2, inp["q"])["y"]
        rows = torch.cat([torch.arange(coff[u], coff[u] + cnt[u]) for u in range(U)]).to("cuda")
        same = (same and bool(torch.equal(y2, y_top)) and bool(torch.equal(rc2.count, rc.count))
                and bool(torch.equal(rc2.idxc[rows], rc.idxc[rows]))
                and bool(torch.equal(rc2.Vc[rows], rc.Vc[rows])))
        errs.append(float(rel_err(y_top, full_output(Vp)).median()))
    line = {"mode": "compare_arms", "workload": wl.name, "units": U, "group": G, "context": n,
            "data": "synthetic (seeded); the paper's models and prompts are not used",
            "arms": table,
            "topk_value_permutation": {"budget": b, "worlds": 6,
                                       "median_rel_err_per_world": [round(e, 5) for e in errs],
                                       "max_over_min": round(max(errs) / max(min(errs), 1e-30), 3),
                                       "retained_set_and_output_identical": same}}
    print(json.dumps(line), flush=True)
    return 0


def _spearman(a, b) -> float:
    ra = a.argsort().argsort().double()
    rb = b.argsort().argsort().double()
    ra -= ra.mean()
    rb -= rb.mean()
    return float((ra * rb).sum() / (ra.norm() * rb.norm() + 1e-300))


def cpu_baseline(wl, args, inp, rc, pi_gpu, q, o, budget, torch):
    """The fp64 oracle on the host cores, on a sample of the leg's units with their global ids
    (so it draws the same Philox streams): eviction (its own lambda solve), then one certified
    step with the first decode query, timed with the host clock.  Units are taken in blocks of 64
    (a fixed random order) until at least args.cpu_min_gb of retained KV are covered and either
    about args.cpu_seconds of oracle time or args.cpu_wall_seconds of wall time (host copies
    included) have passed.  Parity on exactly that sample (untimed): pi against the GPU's within
    1e-5; the oracle's mask and compaction given the GPU's fp32 pi against the GPU's retained
    rows, bit for bit; and the oracle's certified step on those rows against the GPU's yhat
    (2e-3) and Vhat, b, r (1e-2, floors 1e-12 |yhat|^2, 1e-12 |yhat|, 1e-12)."""
    import oracle
    import synth

    U, n, G = wl.units, wl.context, wl.group
    nthreads = oracle.max_threads()
    order = np.random.default_rng(1).permutation(U)
    coff_all = rc.cap_off.cpu().numpy()
    cnt_all = rc.count.cpu().numpy()
    t_evict = t_attend = 0.0
    kv_bytes = 0
    done = 0
    pi_err = 0.0
    sets_equal = 0
    worst = {"y": 0.0, "vhat": 0.0, "b": 0.0, "r": 0.0}
    bad_cert = 0
    wall0 = time.perf_counter()
    while done < U and (kv_bytes < args.cpu_min_gb * 1e9 or
                        ((t_evict + t_attend) < args.cpu_seconds and
                         time.perf_counter() - wall0 < args.cpu_wall_seconds)):
        us = np.sort(order[done:done + 64])
        done += len(us)
        rows = torch.cat([torch.arange(int(u) * n, (int(u) + 1) * n) for u in us]).to("cuda")
        Kb, Vb = synth.bf16_bits(inp["K"][rows]), synth.bf16_bits(inp["V"][rows])
        sc = inp["scores"][rows].cpu().numpy()
        uidx = torch.as_tensor(us, device="cuda")
        qb = synth.bf16_bits(q[uidx])
        off = np.arange(len(us) + 1, dtype=np.int64) * n
        caps = coff_all[us + 1] - coff_all[us]
        coff = np.concatenate([[0], np.cumsum(caps)]).astype(np.int64)
        uid = us.astype(np.uint32)
        t0 = time.perf_counter()
        ev = oracle.evict_batch(off, coff, sc, Kb, Vb, wl.n_sink, wl.n_recent, budget_frac=budget,
                                pi_min=wl.pi_min, seed=args.seed, nthreads=nthreads, unit_ids=uid)
        t1 = time.perf_counter()
        oracle.attend_batch(coff, ev["count"], qb, ev["Kc"], ev["Vc"], ev["pic"], nthreads=nthreads)
        t2 = time.perf_counter()
        t_evict += t1 - t0
        t_attend += t2 - t1
        kv_bytes += 512 * int(ev["count"].sum())
        # parity on the sample
        pg = pi_gpu[rows].cpu().numpy()
        pi_err = max(pi_err, float(np.max(np.abs(pg.astype(np.float64) - ev["pi_full"]))))
        same = oracle.evict_batch(off, coff, sc, Kb, Vb, wl.n_sink, wl.n_recent, pi_given=pg,
                                  seed=args.seed, nthreads=nthreads, unit_ids=uid)
        gi = torch.cat([torch.arange(int(coff_all[u]), int(coff_all[u] + cnt_all[u])) for u in us]).to("cuda")
        g_idx, g_pic = rc.idxc[gi].cpu().numpy(), rc.pic[gi].cpu().numpy()
        g_K, g_V = synth.bf16_bits(rc.Kc[gi]), synth.bf16_bits(rc.Vc[gi])
        pos = 0
        for i, u in enumerate(us):
            c = int(cnt_all[u])
            a = coff[i]
            sl = slice(pos, pos + c)
            pos += c
            sets_equal += int(int(same["count"][i]) == c
                              and np.array_equal(same["idx"][a:a + c], g_idx[sl])
                              and np.array_equal(same["pic"][a:a + c].view(np.uint32), g_pic[sl].view(np.uint32))
                              and np.array_equal(same["Kc"][a:a + c], g_K[sl])
                              and np.array_equal(same["Vc"][a:a + c], g_V[sl]))
        at = oracle.attend_batch(coff, same["count"], qb, same["Kc"], same["Vc"], same["pic"],
                                 nthreads=nthreads)
        gy = o["y"][uidx].cpu().numpy().astype(np.float64)
        nrm = np.linalg.norm(at["y"], axis=2)
        worst["y"] = max(worst["y"], float(np.max(np.linalg.norm(gy - at["y"], axis=2) / nrm)))
        floors = {"vhat": 1e-12 * nrm ** 2, "b": 1e-12 * nrm, "r": np.full_like(nrm, 1e-12)}
        for k in ("vhat", "b", "r"):
            g = o[k][uidx].cpu().numpy().astype(np.float64)
            rel = np.abs(g - at[k]) / np.maximum(np.abs(at[k]), floors[k])
            worst[k] = max(worst[k], float(rel.max()))
            bad_cert += int((rel > 1e-2).sum())
    parity = {"units": done, "pi_max_abs_err": float("%.3g" % pi_err),
              "retained_sets_bit_exact_given_gpu_pi": sets_equal,
              "max_rel_err": {k: float("%.3g" % v) for k, v in worst.items()},
              "certificates_beyond_1e-2": bad_cert,
              "ok": bool(pi_err <= 1e-5 and sets_equal == done and worst["y"] <= 2e-3
                         and bad_cert == 0)}
    return {"value": round(kv_bytes / t_attend / 1e9, 4), "unit": "GB/s", "cores": int(nthreads),
            "kind": "oracle",
            "sample": "%d of %d units of %s (global unit ids), %.2f GB of retained KV; oracle "
                      "eviction %.2f s, one certified step %.2f s" %
                      (done, U, wl.name, kv_bytes / 1e9, t_evict, t_attend),
            "evictions_per_s": round(done / t_evict, 2),
            "parity_on_sample": parity}


if __name__ == "__main__":
    sys.exit(main())
