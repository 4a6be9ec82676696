#!/usr/bin/env python3
"""Benchmark of the eviction-by-design hot path on one MI355X.

A step is one pass of the whole path over one batch of synthetic input: for every budget of the
workload, ebd_evict (lambda solve, Poisson mask, compaction of K/V/pi), then for every budget one
certified decode step ebd_attend_certify (Hajek attention, Theorem 2 variance, eq. (4) radius).
Evictions for all budgets run before the attention steps so that no retained cache is still in
the 256 MB last-level cache when it is read.

The default workload is the Qwen2.5-7B-shaped configuration: 28 layers x batch 16 x 4 KV heads
(1792 unit caches), 7 query heads per KV head, context 6144, budgets 10/25/50%, bf16.

Prints one JSON line.  `value` is the retained-KV bandwidth of certified attention
(K + V bytes of every retained row, summed over the timed steps and budgets, divided by the
summed duration of the attention kernels).  Inputs are resident in HBM before timing starts.
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
KERNELS = ("evict_select", "evict_copy", "attend_split", "attend_finalize")


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
                  out_dir: str = "") -> int:
    """Per-launch HBM bytes of the library's kernels from two rocprofv3 --pmc csv runs.

    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are each scaled by what the same counter reads
    for the 1 GiB device copy that --copy-calibration runs (1 GiB read, 1 GiB written).
    Writes profiles/hbm_traffic_<workload>.json (read by the benchmark while the kernel sources
    are unchanged), or the same file under out_dir.
    """
    import csv
    import glob
    import statistics

    def load(d, counter):
        per, calib = {}, []
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for row in csv.DictReader(open(f)):
                if row["Counter_Name"] != counter:
                    continue
                name, v = row["Kernel_Name"], float(row["Counter_Value"])
                if "ebd::" in name:
                    k = name.split("(")[0].replace("void ", "").replace("ebd::", "")
                    k = k.replace("_kernel", "").split("<")[0]
                    per.setdefault(k, []).append(v)
                elif "copyBuffer" in name and v > 0.25 * (1 << 20):
                    calib.append(v)  # the 1 GiB calibration copies
        return per, calib

    fetch, fcal = load(fetch_dir, "FETCH_SIZE")
    write, wcal = load(write_dir, "WRITE_SIZE")
    if not fcal or not wcal:
        print("no calibration copy found in the counter runs", file=sys.stderr)
        return 1
    gib_kib = float(1 << 20)
    fscale = gib_kib / statistics.median(fcal)  # true KiB per counted KiB
    wscale = gib_kib / statistics.median(wcal)
    kernels = {}
    for k in sorted(set(fetch) | set(write)):
        fb = statistics.mean(fetch.get(k, [0.0])) * fscale * 1024
        wb = statistics.mean(write.get(k, [0.0])) * wscale * 1024
        kernels[k] = {"fetch_bytes_per_launch": int(fb), "write_bytes_per_launch": int(wb),
                      "bytes_per_launch": int(fb + wb),
                      "launches_profiled": len(fetch.get(k, []))}
    rec = {"workload": workload, "kernel_sources_hash": kernel_sources_hash(),
           "fetch_scale": fscale, "write_scale": wscale, "kernels": kernels, "command": command}
    out_dir = out_dir or os.path.join(ROOT, "profiles")
    os.makedirs(out_dir, exist_ok=True)
    path = os.path.join(out_dir, "hbm_traffic_%s.json" % workload)
    json.dump(rec, open(path, "w"), indent=1)
    print(json.dumps(rec, indent=1))
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen7b_6k")
    ap.add_argument("--budgets", default="", help="comma list overriding the workload's budgets")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, run a plain 1 GiB device copy (profiler counter scale)")
    ap.add_argument("--scores-steps", type=int, default=10,
                    help="also time the importance-score kernels alone (0: skip)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate host time for the oracle baseline (0 disables it)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write profiles/hbm_traffic_<workload>.json from rocprofv3 --pmc csv runs")
    ap.add_argument("--pmc-command", default="", help="command recorded in the summary")
    ap.add_argument("--compare-arms", action="store_true",
                    help="instead of timing: errors of the sampling designs against full attention")
    ap.add_argument("--compare-units", type=int, default=256)
    ap.add_argument("--next-steps", type=int, default=3,
                    help="timed repetitions of the rows built after the hot path (0: skip)")
    ap.add_argument("--replay-chunk", type=int, default=-1, metavar="CHUNK",
                    help="instead of a workload: time one chunk (0..7) of 1512 cells of the replay "
                         "grid (8 KV heads per cell, G = 1, per-unit budgets and contexts)")
    args = ap.parse_args()

    if args.summarize_pmc:
        return summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.workload,
                             args.pmc_command)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(units are independent; see the design notes on sharding). Run with --gpus 1.",
              file=sys.stderr)
        return 2

    import torch

    import synth
    import paper_2607_21475_amd as ebd
    from paper_2607_21475_amd import cache

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    wl = synth.WORKLOADS[args.workload]
    budgets = [float(b) for b in args.budgets.split(",")] if args.budgets else list(wl.budgets)
    if args.compare_arms:
        return compare_arms(args, wl, budgets)
    if args.replay_chunk >= 0:
        return replay_chunk(args)
    U, n, G = wl.units, wl.context, wl.group
    lengths = [n] * U

    t0 = time.time()
    inp = synth.make_workload_inputs(wl, seed=args.seed, device="cuda")
    torch.cuda.synchronize()
    print("inputs ready: %d units x %d tokens, G=%d (%.1f s)" % (U, n, G, time.time() - t0),
          file=sys.stderr, flush=True)

    # Pre-plan every launch: outputs, workspaces and parameter blocks are allocated once.
    plans = []
    for b in budgets:
        cap_host = cache.plan_capacity(lengths, b, wl.n_sink, wl.n_recent, pi_min=wl.pi_min)
        cap_off = torch.tensor(cap_host, dtype=torch.int64, device="cuda")
        rows = cap_host[-1]
        rc = cache.RetainedCache(
            Kc=torch.empty((rows, 128), dtype=torch.bfloat16, device="cuda"),
            Vc=torch.empty((rows, 128), dtype=torch.bfloat16, device="cuda"),
            pic=torch.empty((rows,), dtype=torch.float32, device="cuda"),
            idxc=torch.empty((rows,), dtype=torch.int32, device="cuda"),
            count=torch.empty((U,), dtype=torch.int32, device="cuda"),
            status=torch.empty((U,), dtype=torch.int32, device="cuda"),
            cap_off=cap_off, max_cap=max(cap_host[i + 1] - cap_host[i] for i in range(U)))
        ep = ebd.evict_params(U, n, rc.max_cap, inp["seq_off"], cap_off, wl.n_sink, wl.n_recent,
                              b, None, wl.pi_min, 0, args.seed, None, 0)
        ews = ebd.workspace(ebd.ebd_workspace_size(ebd.EBD_WS_EVICT, ep))
        ap_ = ebd.attend_params(U, G, rc.max_cap, cap_off)
        aws_bytes = ebd.ebd_workspace_size(ebd.EBD_WS_ATTEND, ap_)
        aws = ebd.workspace(aws_bytes)
        out = {k: torch.empty(s, dtype=torch.float32, device="cuda")
               for k, s in (("y", (U, G, 128)), ("vhat", (U, G)), ("lse", (U, G)),
                            ("b", (U, G)), ("r", (U, G)))}
        plans.append(dict(budget=b, rc=rc, ep=ep, ews=ews, ap=ap_, aws=aws, out=out,
                          fused=cache.fused_finalize(aws_bytes, U, G)))

    def step():
        for p in plans:
            rc = p["rc"]
            ebd.ebd_evict(p["ep"], inp["scores"], inp["K"], inp["V"], rc.Kc, rc.Vc, rc.pic, rc.idxc,
                          rc.count, rc.status, p["ews"])
        for p in plans:
            rc, o = p["rc"], p["out"]
            ebd.ebd_attend_certify(p["ap"], inp["q"], rc.Kc, rc.Vc, rc.pic, rc.count, o["y"],
                                   o["vhat"], o["lse"], p["aws"], brange=o["b"], radius=o["r"])

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # which budgets' evictions gather their rows inside evict_select (no evict_copy launch)
    ebd.ebd_timing_enable(True)
    for p in plans:
        ebd.ebd_timing_read("evict_copy")
        rc = p["rc"]
        ebd.ebd_evict(p["ep"], inp["scores"], inp["K"], inp["V"], rc.Kc, rc.Vc, rc.pic, rc.idxc,
                      rc.count, rc.status, p["ews"])
        torch.cuda.synchronize()
        p["gathers"] = ebd.ebd_timing_read("evict_copy")[1] == 0
    ebd.ebd_timing_enable(False)
    for p in plans:
        st = p["rc"].status.cpu().numpy()
        if (st & ebd.EBD_ST_CAP_OVERFLOW).any():
            raise RuntimeError("capacity overflow at budget %s" % p["budget"])
    ebd.ebd_timing_enable(True)
    for k in KERNELS:
        ebd.ebd_timing_read(k)  # clear
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    total_ms = ev0.elapsed_time(ev1)
    kt = {k: ebd.ebd_timing_read(k) for k in KERNELS}
    ebd.ebd_timing_enable(False)

    # Work per step, from the (deterministic) retained counts.
    per_budget = []
    retained_total = 0
    gathered = 0  # retained rows of budgets whose evict_select also gathers
    for p in plans:
        cnt = p["rc"].count.cpu().numpy().astype(np.int64)
        rescans = cache.rescans(p["aws"], U, G)
        per_budget.append(dict(budget=p["budget"], retained_rows=int(cnt.sum()),
                               mean_retained_per_unit=float(cnt.mean()),
                               range_term_rescans=int(rescans), fused_finalize=bool(p["fused"]),
                               select_gathers=bool(p["gathers"])))
        retained_total += int(cnt.sum())
        if p["gathers"]:
            gathered += int(cnt.sum())
    K = args.steps
    nb = len(plans)
    kv_bytes = 512 * retained_total  # K + V bf16 rows retained, per step (all budgets)
    nfused = sum(1 for p in plans if p["fused"])
    alg = {
        # scores read once per cached token; pi and index written per retained row; rows read and
        # written (1024 B) where the selection also gathers them
        "evict_select": 4 * U * n * nb + 8 * retained_total + 1024 * gathered,
        # read K+V rows (512 B) and write Kc+Vc rows (512 B) per retained row
        "evict_copy": 1024 * (retained_total - gathered),
        # K, V, pi per retained row (516 B) and the query heads; a split kernel that finalizes
        # its units itself also writes y (512 B), vhat, lse, b, r per query head
        "attend_split": 516 * retained_total + nb * U * G * 256 + nfused * U * G * (512 + 16),
        # y, vhat, lse, b, r per query head of budgets whose units span several splits
        "attend_finalize": (nb - nfused) * U * G * (512 + 16),
    }
    kern = {}
    for k in KERNELS:
        ms, launches = kt[k]
        if launches == 0:
            continue
        avg_ms = ms / launches
        gbs = alg[k] * K / (ms * 1e-3) / 1e9
        kern[k] = dict(total_ms=round(ms, 4), launches=int(launches), avg_us=round(avg_ms * 1e3, 2),
                       alg_bytes_per_step=int(alg[k]), achieved_gbs=round(gbs, 1),
                       frac_hbm=round(gbs / HBM_PEAK_GBS, 4))
    t_attend = (kt["attend_split"][0] + kt["attend_finalize"][0]) * 1e-3
    t_evict = (kt["evict_select"][0] + kt["evict_copy"][0]) * 1e-3
    value = kv_bytes * K / t_attend / 1e9
    evictions_per_s = U * nb * K / t_evict
    dom = max(kern, key=lambda k: kern[k]["total_ms"])
    dk = kern[dom]
    dom_launch_bytes = alg[dom] / (dk["launches"] / K)
    traffic = load_traffic(args.workload, dom)
    roofline = {"bound": "hbm", "achieved": dk["achieved_gbs"], "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(dk["achieved_gbs"] / HBM_PEAK_GBS, 4),
                "traffic": traffic, "kernel": dom,
                "alg_bytes_per_launch": int(dom_launch_bytes), "avg_launch_us": dk["avg_us"]}

    # A plain 1 GiB device copy (read 1 GiB, write 1 GiB) outside the timed region: its rate is
    # what this GPU sustains for a copy (the evict_copy kernel's own ceiling), and its byte
    # counters calibrate a profiler's HBM counters (--copy-calibration runs it under them).
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    best = float("inf")
    for _ in range(5 if not args.copy_calibration else 3):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del src, dst
    roofline["measured_copy_gbs"] = round(2 * (1 << 30) / (best * 1e-3) / 1e9, 1)

    # The step before the path (not part of `value`): importance scores from 32 observation-
    # window queries per unit, the same recipe as the synthetic inputs' scores, timed alone.
    imp = None
    if args.scores_steps > 0:
        qw = synth.make_queries(U, 32, seed=args.seed + 7, device="cuda")
        sp_ = ebd.scores_params(U, 32, n, inp["seq_off"])
        sws = ebd.workspace(ebd.ebd_workspace_size(ebd.EBD_WS_SCORES, sp_))
        sco = torch.empty_like(inp["scores"])
        for _ in range(2):
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
        imp["gbs"] = round(sum(sb.values()) * args.scores_steps / (tot_ms * 1e-3) / 1e9, 1)
        del qw, sws, sco

    nxt = next_rows(args, wl, inp, plans, ebd, torch) if args.next_steps > 0 else None

    # CPU baseline: the fp64 oracle on a bounded sample of the same units, same budgets.
    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(inp, plans, wl, args, torch)

    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / K, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 K/V/q, fp32 accumulate",
        "data": "synthetic (seeded N(0,1) bf16 K/V/q, 2% heavy-hitter keys x4, 32-query window "
                "importance scores); the paper's models and datasets are not used",
        "config": {"workload": wl.name, "description": wl.description, "units": U, "context": n,
                   "group": G, "head_dim": 128, "budgets": budgets, "pi_min": wl.pi_min,
                   "protected": [wl.n_sink, wl.n_recent], "parallelism": "single GPU"},
        "value_frac_hbm": round(value / HBM_PEAK_GBS, 4),
        "evictions_per_s": round(evictions_per_s, 1),
        "evicted_tokens_per_s": round(U * n * nb * K / t_evict, 1),
        "attend_ms_per_step": round(t_attend * 1e3 / K, 4),
        "evict_ms_per_step": round(t_evict * 1e3 / K, 4),
        "per_budget": per_budget,
        "kernels": kern,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "importance_scores": imp,
        "next_rows": nxt,
        "kernel_sources_hash": kernel_sources_hash(),
    }
    print(json.dumps(line), flush=True)
    return 0


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


def cpu_baseline(inp, plans, wl, args, torch):
    import oracle
    import synth

    U, n, G = wl.units, wl.context, wl.group
    nthreads = oracle.max_threads()
    # Sample units in blocks of 16 (spread over the workload) until the time budget is spent.
    order = np.random.default_rng(1).permutation(U)
    done = 0
    t_evict = t_attend = 0.0
    kv_bytes = 0
    units_done = 0
    block = 16
    while done < U and (t_evict + t_attend) < args.cpu_seconds:
        us = np.sort(order[done:done + block])
        done += len(us)
        rows = np.concatenate([np.arange(u * n, (u + 1) * n) for u in us])
        Kb = synth.bf16_bits(inp["K"][rows])
        Vb = synth.bf16_bits(inp["V"][rows])
        sc = inp["scores"][rows].cpu().numpy()
        qb = synth.bf16_bits(inp["q"][torch.as_tensor(us, device="cuda")])
        off = np.arange(len(us) + 1, dtype=np.int64) * n
        for p in plans:
            b = p["budget"]
            caps = [p["rc"].cap_off[u + 1].item() - p["rc"].cap_off[u].item() for u in us]
            coff = np.concatenate([[0], np.cumsum(caps)]).astype(np.int64)
            t0 = time.perf_counter()
            ev = oracle.evict_batch(off, coff, sc, Kb, Vb, wl.n_sink, wl.n_recent, budget_frac=b,
                                    pi_min=wl.pi_min, seed=args.seed, nthreads=nthreads)
            t1 = time.perf_counter()
            oracle.attend_batch(coff, ev["count"], qb, ev["Kc"], ev["Vc"], ev["pic"],
                                nthreads=nthreads)
            t2 = time.perf_counter()
            t_evict += t1 - t0
            t_attend += t2 - t1
            kv_bytes += 512 * int(ev["count"].sum())
        units_done += len(us)
    return {"value": round(kv_bytes / t_attend / 1e9, 4), "unit": "GB/s", "cores": int(nthreads),
            "kind": "oracle",
            "sample": "%d of %d units (x %d budgets), same inputs; oracle evict %.2f s, attend %.2f s"
                      % (units_done, U, len(plans), t_evict, t_attend),
            "evictions_per_s": round(units_done * len(plans) / t_evict, 2)}


if __name__ == "__main__":
    sys.exit(main())
