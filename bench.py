#!/usr/bin/env python3
"""Benchmark of PaDoc tree attention on one MI355X.

    python bench.py [--steps K] [--warmup W] [--gpus 1]

A step is one decode step of masked parallel decoding over the paged cache of
the concurrent-decode workload (64 pages x [prefix 3072, layout stream 256,
24 branches with lengths U[1,1024]]; 1600 live streams, Hq=16, Hkv=2, d=128,
bf16, 16-token blocks shuffled across a pool that fills most of HBM): the
decode plan is uploaded, one kernel runs the shared-key tile items and the
private-key streaming items side by side, and the split partials are combined.  Inputs (Q, the paged K/V cache, the block table) are resident in
HBM before timing starts.  The headline value is branch tokens (queries) per
second of one attention-layer call.  The same run also times the packed
forward of the 8-page training/branch-creation workload (TFLOP/s) and its
backward.

The oracle leg runs the CPU oracle on the decode step (its time is the
reported CPU baseline) and compares the outputs of the timed calls with it in
the same job: every query of the decode step on the timed pool, the other
decode configurations, sampled rows of the timed forward and of the baselines
beside it, and one whole page of the timed backward.  The errors go into the
JSON line under "parity"; a miss makes the run exit with status 1.

One JSON line is printed (rank 0, one GPU).  Kernel durations for the
roofline come from HIP events the library records around all kernels of a
call on the launch stream; the decode roofline is taken on the median of
cold-cache calls (a 1 GiB write between calls), the warm mean is secondary.
`roofline.traffic` comes from the committed rocprofv3 counter summary in
profiles/ while it matches the library sources (`--summarize-profile`
writes it).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "branch-decode tokens/s + HBM GB/s; packed tree-attn TFLOP/s (% roofline)"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2516.6
PROFILE_TAG = "concurrent_decode_64pages_packed_forward_8pages"
TRACE_SUMMARY = os.path.join(ROOT, "profiles", f"kernel_trace_{PROFILE_TAG}.md")
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", f"hbm_traffic_{PROFILE_TAG}.txt")
DECODE_KERNELS = ("decode_step_kernel<128>", "lse_combine_kernel<128, true, 8>")
FORWARD_KERNEL = "tile_mfma_bf16_kernel<128>"
COUNTER_SUMMARY = os.path.join(ROOT, "profiles", f"sq_counters_{PROFILE_TAG}.md")
# SQ counter passes (at most 8 SQ counters each, plus GRBM_GUI_ACTIVE)
SQ_PASSES = {
    "sqA": "SQ_BUSY_CYCLES SQ_VALU_MFMA_BUSY_CYCLES SQ_WAVE_CYCLES SQ_WAIT_INST_LDS SQ_WAIT_ANY "
           "SQ_ACTIVE_INST_LDS SQ_ACTIVE_INST_VALU SQ_ACTIVE_INST_ANY GRBM_GUI_ACTIVE",
    "sqB": "SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_INSTS_LDS SQ_LDS_ADDR_CONFLICT SQ_WAIT_INST_ANY "
           "SQ_VALU_MFMA_COEXEC_CYCLES SQ_BUSY_CU_CYCLES SQ_WAVES GRBM_GUI_ACTIVE",
    "sqC": "SQ_INSTS_MFMA SQ_INSTS_VALU SQ_INSTS_SALU SQ_INSTS_VMEM_RD SQ_INSTS_SMEM SQ_ACTIVE_INST_VMEM "
           "SQ_ACTIVE_INST_SCA SQ_INSTS_BRANCH GRBM_GUI_ACTIVE",
}
SQ_KERNELS = (FORWARD_KERNEL, DECODE_KERNELS[0], "bwd_dkdv_kernel<128>", "bwd_dq_kernel<128>")
BACKWARD_KERNELS = ("bwd_prep_kernel<128>", "bwd_dq_kernel<128>", "bwd_dkdv_kernel<128>", "bwd_finalize_kernel")
COPY_KERNEL = "__amd_rocclr_copyBuffer"
COPY_BYTES = 1 << 30


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--workload", default="concurrent_decode_64pages")
    ap.add_argument("--forward-workload", default="packed_forward_8pages",
                    help="packed-forward workload timed alongside ('none' to skip)")
    ap.add_argument("--pool-gib", type=float, default=0.0,
                    help="bytes of each of the K and V pools in GiB (0: 45%% of HBM each, backing off on failure)")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle leg (CPU baseline and the parity check of the timed outputs)")
    ap.add_argument("--cold-steps", type=int, default=100,
                    help="cold-cache decode calls timed (a 1 GiB write between calls); at least 10")
    ap.add_argument("--no-backward", action="store_true", help="skip the backward of the forward workload")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache decode timing")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the single-page and dense-page decode configurations")
    ap.add_argument("--no-baselines", action="store_true",
                    help="skip the baselines (dense-mask SDPA, gather-varlen, per-stream decode)")
    ap.add_argument("--driver-steps", type=int, default=60,
                    help="decode-session steps timed on the decode workload's streams (0 to skip)")
    ap.add_argument("--budget-pages", type=int, default=16,
                    help="pages of complete traces decoded under a row budget (0 skips that leg)")
    ap.add_argument("--budget-rows", type=int, default=256, help="rows per step in the budgeted leg")
    ap.add_argument("--budget-layers", type=int, default=28,
                    help="attention calls per step in the budgeted leg (a model's layers over one tree)")
    ap.add_argument("--decode-chunk", type=int, default=0,
                    help="decode plan: max keys per work item (0 = planner's choice)")
    ap.add_argument("--decode-target-wg", type=int, default=0,
                    help="decode plan: workgroups the planner aims for when it chooses chunks (0 = default)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy three times (reference for HBM counters)")
    ap.add_argument("--summarize-profile", metavar="DIR",
                    help="only summarize rocprofv3 outputs under DIR into profiles/ (no GPU needed)")
    return ap.parse_args(argv)


# ---------------------------------------------------------------- helpers

def visible_pairs_of(segs):
    """Visible (query, key) pairs of a segment tree: ancestors' fork prefixes
    plus the causal own part, for each of the last q_len tokens."""
    import numpy as np
    n = len(segs)
    anc = np.zeros(n, dtype=np.int64)
    for i in range(n):
        p = int(segs["parent"][i])
        if p >= 0:
            anc[i] = anc[p] + int(segs["fork"][i])
    L = segs["len"].astype(np.int64)
    Q = segs["q_len"].astype(np.int64)
    # sum over p in [L-Q, L) of (anc + p + 1)
    own = Q * L - Q * (Q - 1) // 2
    return int((Q * anc + own).sum())


def timed_steps(fn, steps, warmup, torch, pa):
    """Run `fn` warmup + steps times; returns (ms_per_step, [kernel ms])."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    evs = []
    for _ in range(steps):
        b = torch.cuda.Event(enable_timing=True)
        a = torch.cuda.Event(enable_timing=True)
        b.record()  # creates the underlying events
        a.record()
        evs.append((b, a))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for b, a in evs:
        pa.set_kernel_events(b, a)
        fn()
    te = time.perf_counter()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    pa.set_kernel_events()
    kms = [b.elapsed_time(a) for b, a in evs]
    timed_steps.enqueue_ms = (te - t0) * 1e3 / steps  # host time to submit one step
    return (t1 - t0) * 1e3 / steps, kms


def alloc_pools(torch, n_blocks_needed, Hkv, d, pool_gib, dev):
    """K and V pools sized to most of HBM (each pool gets half), backing off
    8 GiB at a time until both allocations succeed."""
    block_bytes = Hkv * 16 * d * 2
    total = torch.cuda.get_device_properties(dev).total_memory
    want = int(pool_gib * (1 << 30)) if pool_gib > 0 else int(0.45 * total)
    while want > 0:
        n = max(n_blocks_needed, want // block_bytes)
        try:
            kc = torch.empty((n, Hkv, d // 8, 16, 8), dtype=torch.bfloat16, device=dev)  # chunk-major K blocks
            vc = torch.empty((n, Hkv, d, 16), dtype=torch.bfloat16, device=dev)  # d-major V blocks
            return kc, vc, n
        except RuntimeError:
            torch.cuda.empty_cache()
            if want <= 8 << 30:
                break
            want -= 8 << 30
    n = n_blocks_needed
    return (torch.empty((n, Hkv, d // 8, 16, 8), dtype=torch.bfloat16, device=dev),
            torch.empty((n, Hkv, d, 16), dtype=torch.bfloat16, device=dev), n)


# ---------------------------------------------------------------- profile summaries

def source_digest() -> str:
    """SHA-256 over the library sources (kernels, planner, C ABI header):
    a counter summary applies only to the sources it was taken on."""
    import glob
    import hashlib
    files = sorted(f for f in glob.glob(os.path.join(ROOT, "paper_2608_06146_amd", "csrc", "**", "*"), recursive=True)
                   if f.endswith((".hip", ".hpp", ".cpp", ".h")))
    files.append(os.path.join(ROOT, "include", "padoc_attn.h"))
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.relpath(f, ROOT).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def short_kernel_name(name: str) -> str:
    n = name.replace("void ", "").replace("padoc::(anonymous namespace)::", "").replace("padoc::", "")
    return n.split("(")[0].strip()


def measured_traffic():
    """HBM bytes per decode call and per forward launch from the committed
    counter summary, or (None, None) when it was taken on other sources."""
    try:
        with open(TRAFFIC_SUMMARY) as fh:
            kv = dict(line.split(":", 1) for line in fh if ":" in line and not line.startswith("#"))
    except OSError:
        return None, None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("sources_sha256") != source_digest():
        return None, None
    return float(kv["decode_call_bytes"]), float(kv["forward_launch_bytes"])


def measured_counters():
    """Per-kernel derived SQ counter figures from the committed summary, or
    {} when it was taken on other sources."""
    try:
        with open(COUNTER_SUMMARY) as fh:
            lines = [ln.strip() for ln in fh if ln.startswith("value ")]
            fh.seek(0)
            tag = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("sources_sha256:")), None)
    except OSError:
        return {}
    if tag != source_digest():
        return {}
    out = {}
    for ln in lines:  # value <kernel> | <name>: <number>
        kern, rest = ln[len("value "):].split(" | ", 1)
        name, val = rest.split(":", 1)
        out.setdefault(kern.strip(), {})[name.strip()] = float(val)
    return out


def summarize_counters(d: str) -> None:
    """Derived SQ figures per kernel from the three counter passes.  Busy
    fractions divide by the kernel's cycles: GRBM_GUI_ACTIVE sums the 8 XCDs'
    graphics-busy cycles, so a dispatch lasts GRBM_GUI_ACTIVE / 8 cycles, on
    256 CUs x 4 SIMDs; SQ_*_CYCLES-type counters of the SQ block count per
    SIMD (MFMA busy) or per CU (LDS active) over the whole chip."""
    import csv
    import glob
    import statistics
    vals = {}
    dur = {}
    for p in SQ_PASSES:
        for f in glob.glob(os.path.join(d, p, "**", "*counter_collection.csv"), recursive=True):
            with open(f) as fh:
                for r in csv.DictReader(fh):
                    k = short_kernel_name(r["Kernel_Name"])
                    vals.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
                    dur.setdefault(k, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
    lines = ["# SQ counters: bench.py default workloads (packed forward, 8 pages, and its backward; concurrent "
             "decode, 64 pages)", "",
             "Commands (GPU host, repository root as $R): as in kernel_trace_" + PROFILE_TAG + ".md; counters of",
             "each pass (one rocprofv3 run per pass, at most 8 SQ counters):", ""]
    for p, c in SQ_PASSES.items():
        lines.append(f"- {p}: `{c}`")
    lines += ["", f"sources_sha256: {source_digest()}", ""]
    for k in SQ_KERNELS:
        if k not in vals:
            continue
        v = {c: statistics.mean(x) for c, x in vals[k].items()}
        cyc = v["GRBM_GUI_ACTIVE"] / 8.0  # cycles of one dispatch
        us = statistics.mean(dur[k])
        mf = max(v.get("SQ_INSTS_MFMA", 0.0), 1.0)
        derived = {
            "clock_ghz": cyc / (us * 1e3),
            "mfma_busy": v["SQ_VALU_MFMA_BUSY_CYCLES"] / (1024 * cyc),
            "valu_insts_per_mfma": v["SQ_INSTS_VALU"] / mf,
            "salu_insts_per_mfma": v["SQ_INSTS_SALU"] / mf,
            "lds_insts_per_mfma": v["SQ_INSTS_LDS"] / mf,
            "lds_active": v["SQ_LDS_IDX_ACTIVE"] / (256 * cyc),
            "lds_bank_conflict_per_active": v["SQ_LDS_BANK_CONFLICT"] / max(v["SQ_LDS_IDX_ACTIVE"], 1.0),
            "wait_any_per_wave_cycle": v["SQ_WAIT_ANY"] / max(v["SQ_WAVE_CYCLES"], 1.0),
            "valu_active_per_wave_cycle": v["SQ_ACTIVE_INST_VALU"] / max(v["SQ_WAVE_CYCLES"], 1.0),
        }
        lines += [f"## `{k}`", "", f"dispatches: {len(vals[k]['GRBM_GUI_ACTIVE'])}, mean duration under counters "
                  f"{us:.1f} us", "", "| counter | mean per dispatch |", "|---|---|"]
        lines += [f"| {c} | {x:.4g} |" for c, x in sorted(v.items())]
        lines += ["", "| derived | value |", "|---|---|"] + [f"| {n} | {x:.3f} |" for n, x in derived.items()]
        lines += [""] + [f"value {k} | {n}: {x:.5g}" for n, x in derived.items()] + [""]
    with open(COUNTER_SUMMARY, "w") as fh:
        fh.write("\n".join(lines))
    print(f"wrote {COUNTER_SUMMARY}")


PROFILE_COMMANDS = """\
    R=<repository root>; OUT=<output directory>; cd /tmp && export TMPDIR=/tmp
    rocprofv3 --kernel-trace --stats -d $OUT/trace -o bench -- \\
        python3 $R/bench.py --steps 30 --warmup 5 --no-cpu-baseline --no-baselines --driver-steps 0 --no-secondary --no-cold > $OUT/trace/bench.json
    rocprofv3 --pmc FETCH_SIZE --kernel-include-regex padoc -f csv -d $OUT/fetch -o p -- \\
        python3 $R/bench.py --steps 30 --warmup 5 --no-cpu-baseline --no-baselines --driver-steps 0 --no-secondary --no-cold
    rocprofv3 --pmc WRITE_SIZE --kernel-include-regex padoc -f csv -d $OUT/write -o p -- \\
        python3 $R/bench.py --steps 30 --warmup 5 --no-cpu-baseline --no-baselines --driver-steps 0 --no-secondary --no-cold
    rocprofv3 --pmc FETCH_SIZE -f csv -d $OUT/copy_fetch -o c -- python3 $R/bench.py --calibrate-copy
    rocprofv3 --pmc WRITE_SIZE -f csv -d $OUT/copy_write -o c -- python3 $R/bench.py --calibrate-copy
    for P in sqA sqB sqC; do   # counters of each pass: SQ_PASSES in bench.py
      rocprofv3 --pmc <SQ_PASSES[$P]> --kernel-include-regex "tile_mfma|decode_step|bwd_dkdv|bwd_dq" -f csv -d $OUT/$P -o p -- \\
          python3 $R/bench.py --steps 3 --warmup 1 --no-cpu-baseline --no-baselines --driver-steps 0 --budget-pages 0 --no-secondary --no-cold
    done
    python3 $R/bench.py --summarize-profile $OUT
"""


def summarize_profile(d: str) -> None:
    """Write the kernel-trace table and the HBM-traffic summary under
    profiles/ from the outputs of the profiling commands above."""
    import csv
    import glob
    import sqlite3
    import statistics

    if not os.path.isdir(os.path.join(d, "trace")):  # counter passes only
        summarize_counters(d)
        return
    db = sorted(glob.glob(os.path.join(d, "trace", "**", "*.db"), recursive=True))[0]
    con = sqlite3.connect(db)
    rows = con.execute("select name, count(*), avg(duration), min(duration), max(duration), max(lds_size), "
                       "max(grid_x), max(workgroup_x) from kernels "
                       "where name like '%padoc%' group by name order by avg(duration) desc").fetchall()
    ev = {}
    try:
        with open(os.path.join(d, "trace", "bench.json")) as fh:
            ev = json.loads(fh.read().strip().splitlines()[-1])
    except (OSError, ValueError, IndexError):
        pass

    def counter(sub, name):
        out = {}
        for f in glob.glob(os.path.join(d, sub, "**", "*counter_collection.csv"), recursive=True):
            with open(f) as fh:
                for r in csv.DictReader(fh):
                    if r["Counter_Name"] == name:
                        out.setdefault(short_kernel_name(r["Kernel_Name"]), []).append(float(r["Counter_Value"]))
        return {k: statistics.mean(v) for k, v in out.items()}

    fetch, write = counter("fetch", "FETCH_SIZE"), counter("write", "WRITE_SIZE")
    fetch_factor = COPY_BYTES / 1024 / counter("copy_fetch", "FETCH_SIZE")[COPY_KERNEL]
    write_factor = COPY_BYTES / 1024 / counter("copy_write", "WRITE_SIZE")[COPY_KERNEL]

    def traffic(k):
        return (fetch[k] * fetch_factor + write[k] * write_factor) * 1024

    dec_bytes = sum(traffic(k) for k in DECODE_KERNELS)
    fwd_bytes = traffic(FORWARD_KERNEL)
    lines = [f"# Kernel trace: bench.py default run (concurrent decode, 64 pages x 24 branches; packed forward, 8 pages)",
             "", "Commands (GPU host, repository root as $R):", "", PROFILE_COMMANDS,
             "| kernel | calls | avg us | min us | max us | LDS B | workgroups | threads |",
             "|---|---|---|---|---|---|---|---|"]
    for name, n, avg, mn, mx, lds, gx, wx in rows:
        lines.append(f"| `{short_kernel_name(name)}` | {n} | {avg / 1e3:.1f} | {mn / 1e3:.1f} | {mx / 1e3:.1f} | "
                     f"{lds} | {gx // max(wx, 1)} | {wx} |")
    dec_avg = sum(r[2] for r in rows if short_kernel_name(r[0]) in DECODE_KERNELS) / 1e3
    lines += ["", f"Decode call (sum of the decode kernels' averages: step + combine): {dec_avg:.1f} us."]
    if ev:
        lines.append(f"Same run, HIP events around each call (bench.py): decode call "
                     f"{ev['decode']['kernel_ms'] * 1e3:.1f} us, forward {ev['forward']['kernel_ms'] * 1e3:.1f} us.")
    lines += ["", f"HBM traffic per launch (FETCH_SIZE x {fetch_factor:.3f} + WRITE_SIZE x {write_factor:.3f}, factors "
              f"from a 1 GiB device copy): see {os.path.basename(TRAFFIC_SUMMARY)}.", ""]
    with open(TRACE_SUMMARY, "w") as fh:
        fh.write("\n".join(lines))
    tl = ["# HBM traffic from rocprofv3 FETCH_SIZE / WRITE_SIZE (KiB per dispatch), scaled by a 1 GiB copy.",
          "# Commands: as in " + os.path.basename(TRACE_SUMMARY) + ". bench.py reports these bytes as",
          "# roofline.traffic only while sources_sha256 matches the library sources.",
          f"sources_sha256: {source_digest()}",
          f"fetch_factor: {fetch_factor:.4f}", f"write_factor: {write_factor:.4f}"]
    for k in DECODE_KERNELS + (FORWARD_KERNEL,) + BACKWARD_KERNELS:
        if k in fetch and k in write:
            tl.append(f"kernel {k} fetch_kib: {fetch[k]:.1f}")
            tl.append(f"kernel {k} write_kib: {write[k]:.1f}")
    tl += [f"decode_call_bytes: {dec_bytes:.0f}", f"forward_launch_bytes: {fwd_bytes:.0f}", ""]
    with open(TRAFFIC_SUMMARY, "w") as fh:
        fh.write("\n".join(tl))
    print(f"wrote {TRACE_SUMMARY} and {TRAFFIC_SUMMARY}")
    if any(os.path.isdir(os.path.join(d, p)) for p in SQ_PASSES):
        summarize_counters(d)


# ---------------------------------------------------------------- decode leg

def run_decode(args, torch, np, syn, pa, dev, name=None, pool_gib=None, steps=None, check=None):
    """One decode step of workload `name` (default: the headline workload),
    timed warm (consecutive calls) and cold (a 1 GiB write between calls,
    outside the timed span, so no K/V stays in L2 / the memory-side cache).
    `check(wl, q, kc, vc, ids, o, lse)`, when given, runs while the timed
    pool and the outputs of the last timed call are still resident (the
    oracle leg); its result is returned under "oracle"."""
    wl = syn.make_workload(name or args.workload, args.seed)
    steps = args.steps if steps is None else steps
    pool_gib = args.pool_gib if pool_gib is None else pool_gib
    assert wl.kind == "decode"
    Hq, Hkv, d = wl.num_heads_q, wl.num_heads_kv, wl.head_dim
    T = syn.count_tokens(wl.pages)
    nq = syn.count_queries(wl.pages)
    nb = syn.count_blocks(wl.pages)
    segs_paged = pa.segments_from_pages(wl.pages, 16)
    segs_packed = pa.segments_from_pages(wl.pages, 0)

    kc, vc, n_pool = alloc_pools(torch, nb, Hkv, d, pool_gib, dev)
    pool_gib = 2 * n_pool * Hkv * 16 * d * 2 / (1 << 30)
    log(f"decode workload {wl.name}: {len(wl.pages)} pages, {T} cached tokens, {nq} queries, "
        f"{nb} blocks in a {pool_gib:.1f} GiB K+V pool")
    ids = syn.draw_block_ids(nb, n_pool, args.seed)

    # plan creation (host) is timed on its own
    pts = []
    for _ in range(5):
        t0 = time.perf_counter()
        plan = pa.TreePlan(segs_paged, Hq, Hkv, d, "bf16", 16, num_kv_rows=n_pool, num_q_rows=nq,
                           block_table_len=nb, max_chunk_keys=args.decode_chunk,
                           target_workgroups=args.decode_target_wg)
        pts.append((time.perf_counter() - t0) * 1e3)
    plan_ms = statistics.median(pts)

    # fill the used blocks: token t of segment s -> block ids[bt_off + t//16], slot t%16
    k = syn.draw_normal((T, Hkv, d), args.seed, 2, "bf16", device=dev)
    v = syn.draw_normal((T, Hkv, d), args.seed, 3, "bf16", device=dev)
    q = syn.draw_normal((nq, Hq, d), args.seed, 1, "bf16", device=dev)
    blk = np.empty(T, dtype=np.int64)
    slot = np.empty(T, dtype=np.int64)
    for s in range(len(segs_paged)):
        L = int(segs_paged["len"][s])
        r0 = int(segs_packed["kv_off"][s])
        t = np.arange(L)
        blk[r0:r0 + L] = ids[int(segs_paged["kv_off"][s]) + t // 16]
        slot[r0:r0 + L] = t % 16
    bi = torch.as_tensor(blk, device=dev)
    si = torch.as_tensor(slot, device=dev)
    # K blocks are chunk-major: token t's 8-dim piece c at [c][slot], slot =
    # t with bits 2 and 3 exchanged (the library's documented cache layout)
    ci = (si & 3) | ((si >> 3) & 1) << 2 | ((si >> 2) & 1) << 3
    kc[bi, :, :, ci, :] = k.reshape(T, Hkv, d // 8, 8)
    vc[bi, :, :, si] = v
    del k, v, bi, si
    bt = torch.as_tensor(ids, device=dev)
    o = torch.empty(nq, Hq, d, dtype=torch.bfloat16, device=dev)
    lse = torch.empty(nq, Hq, dtype=torch.float32, device=dev)
    ws = plan.workspace(dev)
    torch.cuda.synchronize()

    # The schedule is an input like the caches: resident in HBM before the
    # timed region (one upload serves every layer of a model's decode step).
    pa.plan_upload(plan, ws)

    def step():
        pa.branch_decode_resident(q, kc, vc, bt, plan, o, lse, ws)

    ms, kms = timed_steps(step, steps, args.warmup, torch, pa)
    enqueue_ms = timed_steps.enqueue_ms
    k_ms = statistics.mean(kms)

    def step_with_upload():  # the schedule copied from host memory in every call (one layer per step)
        pa.branch_decode(q, kc, vc, bt, plan, out=o, lse=lse, workspace=ws)

    ms_up, _ = timed_steps(step_with_upload, steps, args.warmup, torch, pa)
    # cold: flush between calls (not timed)
    flush = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    cold = []
    n_cold = 0 if args.no_cold else max(10, args.cold_steps)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_cold)]
    for b, a in evs:
        b.record()  # creates the underlying events
        a.record()
    torch.cuda.synchronize()
    for i, (b, a) in enumerate(evs):
        flush.fill_(i & 255)
        pa.set_kernel_events(b, a)
        step()
        pa.set_kernel_events()
        cold.append((b, a))
    torch.cuda.synchronize()
    cold_ms = [b.elapsed_time(a) for b, a in cold] or [float("nan")]
    del flush

    # algorithmic bytes: every cached K/V token read once, Q read, O/LSE written,
    # block-table ids of the referenced blocks read
    kv_bytes = T * Hkv * d * 2 * 2
    q_bytes = nq * Hq * d * 2
    o_bytes = nq * Hq * d * 2 + nq * Hq * 4
    bt_bytes = nb * 4
    step_bytes = kv_bytes + q_bytes + bt_bytes + o_bytes
    kernel_bytes = step_bytes  # the timed span covers every kernel of the call
    naive = 0
    anc = {}
    for s in range(len(segs_paged)):
        p = int(segs_paged["parent"][s])
        anc[s] = (anc[p] + int(segs_paged["fork"][s])) if p >= 0 else 0
        if int(segs_paged["q_len"][s]) > 0:
            naive += anc[s] + int(segs_paged["len"][s])
    flops = 4 * d * Hq * visible_pairs_of(segs_paged)
    ex = plan.export()
    res = {
        "workload": wl.name, "ms_per_step": ms, "enqueue_ms": enqueue_ms, "kernel_ms": k_ms,
        "ms_per_step_with_upload": ms_up, "tokens_per_s_with_upload": nq / (ms_up * 1e-3),
        "kernel_ms_p10": float(np.percentile(kms, 10)), "kernel_ms_p90": float(np.percentile(kms, 90)),
        "kernel_ms_cold_p10": float(np.percentile(cold_ms, 10)), "kernel_ms_cold_p50": float(np.median(cold_ms)),
        "kernel_ms_cold_p90": float(np.percentile(cold_ms, 90)),
        "kernel_gbps_cold": kernel_bytes / (float(np.median(cold_ms)) * 1e-3) / 1e9,
        "tokens_per_s": nq / (ms * 1e-3), "step_gbps": step_bytes / (ms * 1e-3) / 1e9,
        "kernel_gbps": kernel_bytes / (k_ms * 1e-3) / 1e9, "kernel_bytes": kernel_bytes,
        "kv_bytes": kv_bytes, "naive_per_stream_kv_bytes": naive * Hkv * d * 2 * 2,
        "sharing_factor": naive / T, "flops": flops, "kernel_tflops": flops / (k_ms * 1e-3) / 1e12,
        "plan_ms": plan_ms, "tokens_per_s_with_plan": nq / ((ms_up + plan_ms) * 1e-3),
        "work_items": int(len(ex["work"])), "partial_slots": int(ex["n_slots"]), "pool_gib": pool_gib,
        "pages": len(wl.pages), "queries": nq, "cached_tokens": T, "Hq": Hq, "Hkv": Hkv, "d": d,
    }
    if check is not None:
        torch.cuda.synchronize()
        res["oracle"] = check(wl, q, kc, vc, ids, o, lse)
    del kc, vc
    torch.cuda.empty_cache()
    return res, wl


# ---------------------------------------------------------------- session (step driver) leg

class _DriverSet:
    """A DecodeSession holding some pages of the decode workload, built as
    the decoding loop builds them: prefix prefill, layout stream, then the
    content streams at their forks (App. E loop), plus its step buffers."""

    def __init__(self, args, torch, np, syn, pa, dev, wl, pages, steps, seed, stream=None):
        Hq, Hkv, d = wl.num_heads_q, wl.num_heads_kv, wl.head_dim
        nb = syn.count_blocks(pages)
        rows0 = syn.count_queries(pages)
        n_pool = int(nb * 1.25) + (steps + args.warmup + 2) * (rows0 // 16 + 64) + 4096
        self.torch, self.np = torch, np
        self.kc = torch.empty((n_pool, Hkv, d // 8, 16, 8), dtype=torch.bfloat16, device=dev)
        self.vc = torch.empty((n_pool, Hkv, d, 16), dtype=torch.bfloat16, device=dev)
        self.bt = torch.full((4 * n_pool,), -1, dtype=torch.int32, device=dev)
        sess = pa.DecodeSession(Hq, Hkv, d, n_pool, "bf16", k_cache=self.kc, v_cache=self.vc, block_table=self.bt,
                                max_chunk_keys=args.decode_chunk, target_workgroups=args.decode_target_wg)
        self.sess, self.n_pool = sess, n_pool
        gen = torch.Generator(device=dev)
        gen.manual_seed(seed * 1000003 + 17)

        def rows(n, h):
            return torch.randn((n, h, d), generator=gen, device=dev, dtype=torch.float32).to(torch.bfloat16)

        def build_step(n_new, n_q):
            nk, nq, _ = sess.prepare(np.asarray(n_new, np.int32), np.asarray(n_q, np.int32))
            sess.launch(rows(nq, Hq) if nq else None, rows(nk, Hkv), rows(nk, Hkv))
            torch.cuda.synchronize()

        roots = [sess.open(-1, 0) for _ in pages]
        build_step([p.prefix_len for p in pages], [0] * len(pages))
        lay = [sess.open(r, p.prefix_len) for r, p in zip(roots, pages)]
        for r in roots:
            sess.close(r)
        build_step([p.stream_len - 1 for p in pages], [0] * len(pages))
        self.kind = {x: ("layout", i) for i, x in enumerate(lay)}
        for i, p in enumerate(pages):
            for b in p.branches:
                self.kind[sess.open(lay[i], b.fork)] = ("content", i)
        ids = [int(x) for x in sess.view(block_table=False)["row_id"]]
        branch_len = {i: iter([b.length - 1 for b in p.branches]) for i, p in enumerate(pages)}
        build_step([0 if self.kind[x][0] == "layout" else next(branch_len[self.kind[x][1]]) for x in ids],
                   [0] * len(ids))
        self.lay_len = {x: p.stream_len - 1 for x, p in zip(lay, pages)}
        self.live = ids  # open streams, ascending id (the session's row order)
        self.q_buf = rows(rows0 + 4096, Hq)
        self.k_buf = rows(rows0 + 4096, Hkv)
        self.v_buf = rows(rows0 + 4096, Hkv)
        self.o_buf = torch.empty_like(self.q_buf)
        self.l_buf = torch.empty(self.q_buf.shape[:2], dtype=torch.float32, device=dev)
        self.rng = np.random.default_rng(seed + 5)
        self.done = torch.cuda.Event()
        self.stream = stream  # None: the current stream

    def prepare_launch(self):
        """Host plan of the step, then its launch; returns (rows, prepare s, launch s)."""
        t0 = time.perf_counter()
        nk, nq, _ = self.sess.prepare()
        t1 = time.perf_counter()
        if nq > self.q_buf.shape[0]:
            raise RuntimeError("driver: more live streams than the step buffers hold")
        if self.stream is None:
            self.sess.launch(self.q_buf[:nq], self.k_buf[:nk], self.v_buf[:nk], out=self.o_buf[:nq],
                             lse=self.l_buf[:nq])
            self.done.record()
        else:
            with self.torch.cuda.stream(self.stream):
                self.sess.launch(self.q_buf[:nq], self.k_buf[:nk], self.v_buf[:nk], out=self.o_buf[:nq],
                                 lse=self.l_buf[:nq])
                self.done.record()
        return nq, t1 - t0, time.perf_counter() - t1

    def events(self):
        """The step's events: a content stream ends with probability 1/512, a
        layout stream opens a content stream with probability 24/512."""
        sess, np = self.sess, self.np
        for x in self.lay_len:
            self.lay_len[x] += 1
        u = self.rng.random(len(self.live))
        ended, born = set(), []
        for j in np.nonzero(u < 24.0 / 512)[0]:     # only these streams can have an event
            x = self.live[j]
            k_, pg = self.kind[x]
            if k_ == "content" and u[j] < 1.0 / 512:
                sess.close(x)
                ended.add(x)
            elif k_ == "layout":
                c = sess.open(x, self.lay_len[x])
                self.kind[c] = ("content", pg)
                born.append(c)
        for x in ended:
            self.live.remove(x)
        self.live += born

    def free_blocks(self):
        return int(self.sess.view(block_table=False)["free_blocks"])

    def destroy(self):
        self.sess.destroy()
        del self.kc, self.vc, self.bt, self.q_buf, self.k_buf, self.v_buf, self.o_buf


def run_driver(args, torch, np, syn, pa, dev, wl):
    """Masked parallel decoding steps through DecodeSessions (App. E loop).
    Each step prepares (host plan), launches (append of one new token per
    live stream + attention) and waits for the outputs, as a decoding loop
    must before it samples; then the step's events are applied (content
    streams end with probability 1/512, i.e. mean length 512 as U[1,1024];
    layout streams open content streams with probability 24/512, keeping
    about 24 per page).
    serial: one session holds every page; per step prepare -> launch -> wait
      -> events, so the host work and the GPU work add up.
    pipelined: two sessions hold half the pages each and alternate, a
      serving loop's two micro-batches, each on a stream of its own (default
      priority): while the GPU runs one session's step the host waits for,
      samples and prepares the other's, so the host work hides behind the
      GPU, and the two sessions' kernels may overlap on the GPU (each
      session still waits for its own outputs before its next step).
    Reported: per-step wall time split into prepare / launch / wait /
    events, and tokens/s with and without the host work."""
    steps = args.driver_steps
    res = {}
    # ---- serial: one session, all pages
    D = _DriverSet(args, torch, np, syn, pa, dev, wl, wl.pages, steps, args.seed)
    log(f"driver: session holds {len(D.live)} streams, {D.free_blocks()} of {D.n_pool} blocks free")
    rec = []
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for b, a in ev:
        b.record()
        a.record()
    torch.cuda.synchronize()
    for s in range(args.warmup + steps):
        timed = s >= args.warmup
        if timed:
            pa.set_kernel_events(*ev[s - args.warmup])
        nq, t_prep, t_launch = D.prepare_launch()
        t2 = time.perf_counter()
        D.done.synchronize()
        t3 = time.perf_counter()
        D.events()
        t4 = time.perf_counter()
        if timed:
            pa.set_kernel_events()
            rec.append((nq, t_prep, t_launch, t3 - t2, t4 - t3))
    gpu = [b.elapsed_time(a) for b, a in ev]
    n_rows = sum(r[0] for r in rec)
    wall = sum(r[1] + r[2] + r[3] + r[4] for r in rec)
    res.update({
        "steps": steps, "rows_per_step": n_rows / steps,
        "step_ms": wall * 1e3 / steps,
        "prepare_ms": 1e3 * statistics.mean(r[1] for r in rec),
        "launch_ms": 1e3 * statistics.mean(r[2] for r in rec),
        "wait_ms": 1e3 * statistics.mean(r[3] for r in rec),
        "events_ms": 1e3 * statistics.mean(r[4] for r in rec),
        "gpu_ms": statistics.mean(gpu),
        "tokens_per_s": n_rows / wall,
        "tokens_per_s_gpu": n_rows / (sum(gpu) * 1e-3),
        "pool_blocks": D.n_pool, "free_blocks_end": D.free_blocks(),
    })
    D.destroy()
    torch.cuda.empty_cache()

    # ---- pipelined: two sessions of half the pages each, alternating
    half = len(wl.pages) // 2
    sets = [_DriverSet(args, torch, np, syn, pa, dev, wl, wl.pages[:half], steps, args.seed, torch.cuda.Stream()),
            _DriverSet(args, torch, np, syn, pa, dev, wl, wl.pages[half:], steps, args.seed + 1, torch.cuda.Stream())]
    torch.cuda.synchronize()
    rows_done = 0
    host = {"prepare": 0.0, "launch": 0.0, "events": 0.0, "wait": 0.0}
    t_start = None
    for X in sets:  # first step of each session in flight
        X.prepare_launch()
    for s in range(args.warmup + steps):
        if s == args.warmup:
            t_start = time.perf_counter()
            rows_done = 0
            host = dict.fromkeys(host, 0.0)
        for X in sets:
            t0 = time.perf_counter()
            X.done.synchronize()   # this session's step is done: sample, apply its events
            t1 = time.perf_counter()
            X.events()
            t2 = time.perf_counter()
            nq, t_prep, t_launch = X.prepare_launch()
            rows_done += nq
            host["wait"] += t1 - t0
            host["events"] += t2 - t1
            host["prepare"] += t_prep
            host["launch"] += t_launch
    for X in sets:
        X.done.synchronize()
    wall = time.perf_counter() - t_start
    # rows launched in the timed loop; the last launches finish inside `wall`
    res["pipelined"] = {
        "sessions": 2, "pages_per_session": [half, len(wl.pages) - half], "steps": steps,
        "rows_per_step": rows_done / steps, "step_ms": wall * 1e3 / steps,
        "prepare_ms": 1e3 * host["prepare"] / steps, "launch_ms": 1e3 * host["launch"] / steps,
        "events_ms": 1e3 * host["events"] / steps, "wait_ms": 1e3 * host["wait"] / steps,
        "tokens_per_s": rows_done / wall, "streams": "one per session (default priority)",
    }
    for X in sets:
        X.destroy()
    torch.cuda.empty_cache()

    return res


# ---------------------------------------------------------------- budgeted steps (critical-path order)

class BudgetedReplay:
    """A known decoding tree (the segments of complete traces: page roots
    prefilled, every other segment decoded one token per step) run through a
    DecodeSession with at most ``max_rows`` rows per step.  Each step the
    session's open streams are ranked by ``padoc_session_select``: oldest
    first, or (``by_priority``) by their remaining critical path from
    ``padoc_tree_remaining`` at the step's progress (Sec. 3.1).  A segment is
    opened once it has started (a child of a root with its page, a deeper one
    once its parent has produced ``fork`` tokens; newly started segments in
    index order) and closed once it has produced all its tokens.  ``launch``
    runs a prepared step on the GPU (``launch(replay, n_kv_rows, n_q_rows)``);
    without it the session is host-only and steps are committed."""

    def __init__(self, pa, np, sess, nodes, max_rows, by_priority, launch=None):
        self.pa, self.np, self.sess = pa, np, sess
        self.nodes = [tuple(int(x) for x in nd) for nd in nodes]
        n = len(self.nodes)
        seg = np.zeros(n, dtype=pa.SEGMENT_DTYPE)
        seg["parent"] = [nd[0] for nd in self.nodes]
        seg["fork"] = [nd[1] for nd in self.nodes]
        seg["len"] = [nd[2] for nd in self.nodes]
        self.seg = seg
        self.max_rows, self.by_priority, self.launch = int(max_rows), bool(by_priority), launch
        self.produced = np.zeros(n, np.int32)
        self.id_of = {}
        self.seg_of = {}
        self.seg_by_id = np.full(n, -1, np.int64)   # session ids are 0, 1, ... in opening order
        self.open_ids = []
        self.children = [[] for _ in range(n)]
        for s, nd in enumerate(self.nodes):
            if nd[0] >= 0:
                self.children[nd[0]].append(s)
        roots = [s for s in range(n) if self.nodes[s][0] < 0]
        for s in roots:
            self._open(s, -1, 0)
        self._run([self.nodes[s][2] for s in roots], [0] * len(roots))
        self._open_started()
        for s in roots:
            self._close(s)
        self.steps = []   # advanced segments per step

    def _open(self, s, parent_id, fork):
        i = self.sess.open(parent_id, fork)
        self.id_of[s], self.seg_of[i] = i, s
        self.seg_by_id[i] = s
        self.open_ids.append(i)

    def _close(self, s):
        i = self.id_of[s]
        self.sess.close(i)
        self.open_ids.remove(i)

    def _run(self, n_new, n_query):
        nk, nq, _ = self.sess.prepare(self.np.asarray(n_new, self.np.int32), self.np.asarray(n_query, self.np.int32))
        if self.launch is None:
            self.sess.commit()
        else:
            self.launch(self, nk, nq)
        return nq

    def _open_started(self, advanced=None):
        """Open the segments that have started and are not open yet, in index
        order (every parent before its children).  Only children of
        `advanced` (the segments that just produced a token) and, through
        fork offsets of 0, their descendants can start after the first call."""
        if advanced is None:
            cand = [s for s in range(len(self.nodes)) if self.nodes[s][0] >= 0]
        else:
            cand = [c for s in advanced for c in self.children[s]]
        new = []
        seen = set()
        while cand:
            nxt = []
            for s in cand:
                if s in self.id_of or s in seen:
                    continue
                parent, fork = self.nodes[s][0], self.nodes[s][1]
                root_child = self.nodes[parent][0] < 0
                if root_child or ((parent in self.id_of or parent in seen) and self.produced[parent] >= fork):
                    seen.add(s)
                    new.append(s)
                    nxt.extend(self.children[s])  # a fork of 0 starts with its parent
            cand = nxt
        for s in sorted(new):
            parent, fork = self.nodes[s][0], self.nodes[s][1]
            self._open(s, self.id_of[parent], fork if self.nodes[parent][0] >= 0 else self.nodes[parent][2])

    def done(self):
        return not self.open_ids

    def step(self):
        """One step; returns its query rows."""
        np = self.np
        pr = None
        open_seg = self.seg_by_id[np.asarray(self.open_ids, np.int64)]
        if self.by_priority:
            pr = self.pa.tree_remaining(self.seg, self.produced)[open_seg]
        n_new, n_query = self.sess.select(self.max_rows, pr)
        nq = self._run(n_new, n_query)
        adv = open_seg[n_new > 0].tolist()
        self.produced[adv] += 1
        self.steps.append(sorted(adv))
        self._open_started(adv)
        for s in adv:
            if self.produced[s] == self.nodes[s][2]:
                self._close(s)
        return nq


def schedule_trace_pages(np, n_pages, seed):
    """Complete decoding traces shaped as the decode workload's pages: per
    page a 3,072-token prefix (prefilled), a 256-token layout stream and 24
    content streams with forks f ~ U{1..255} (sorted) and lengths
    L ~ U{1..1024}; the layout stream starts at its first token."""
    rng = np.random.default_rng(seed)
    nodes = []
    for _ in range(n_pages):
        L = rng.integers(1, 1025, size=24)
        f = np.sort(rng.integers(1, 256, size=24))
        r = len(nodes)
        nodes.append((-1, 0, 3072, 0))
        nodes.append((r, 3072, 256, 256))
        nodes += [(r + 1, int(a), int(b), int(b)) for a, b in zip(f, L)]
    return nodes


def run_budgeted(args, torch, np, pa, dev):
    """Steps to decode complete traces with a row budget per step, oldest
    streams first against critical-path first (the remaining paths of
    padoc_tree_remaining as the session's priorities), on the GPU: each step
    appends the new rows and runs the attention of `--budget-layers` layers
    over the step's tree (the same caches stand in for every layer's), and
    the loop waits for each step's outputs."""
    nodes = schedule_trace_pages(np, args.budget_pages, args.seed + 11)
    segs = np.zeros(len(nodes), dtype=pa.SEGMENT_DTYPE)
    segs["parent"] = [x[0] for x in nodes]
    segs["fork"] = [x[1] for x in nodes]
    segs["len"] = [x[2] for x in nodes]
    _, d_seq, d_crit = pa.tree_depths(segs)
    decoded = int(d_seq.sum())
    budget = args.budget_rows
    Hq, Hkv, d = 16, 2, 128
    tokens = sum(x[2] for x in nodes)
    n_pool = tokens // 16 + len(nodes) + 1024
    kc = torch.empty((n_pool, Hkv, d // 8, 16, 8), dtype=torch.bfloat16, device=dev)
    vc = torch.empty((n_pool, Hkv, d, 16), dtype=torch.bfloat16, device=dev)
    bt = torch.full((4 * n_pool,), -1, dtype=torch.int32, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed + 29)
    big = max(x[2] for x in nodes if x[0] < 0) * args.budget_pages
    kv_buf = torch.randn((big, Hkv, d), generator=gen, device=dev).to(torch.bfloat16)
    q_buf = torch.randn((max(budget, 1) + 64 * args.budget_pages, Hq, d), generator=gen, device=dev).to(torch.bfloat16)
    o_buf = torch.empty_like(q_buf)
    l_buf = torch.empty(q_buf.shape[:2], dtype=torch.float32, device=dev)

    import ctypes as C
    from paper_2608_06146_amd import _lib
    layers = max(1, args.budget_layers)
    lws = torch.empty(64 << 20, dtype=torch.uint8, device=dev)

    def launch(R, nk, nq):
        # the step's append and its first layer's attention, then the
        # attention of the other layers on the same tree (a model's decode
        # step attends over one tree in every layer)
        v = R.sess.view(block_table=False) if layers > 1 and nq else None  # the prepared step's plan
        R.sess.launch(q_buf[:nq] if nq else None, kv_buf[:nk], kv_buf[:nk], out=o_buf[:nq], lse=l_buf[:nq])
        if v is not None:
            if v["workspace_bytes"] > lws.numel():
                raise RuntimeError("budgeted leg: layer workspace too small")
            st = torch.cuda.current_stream(dev).cuda_stream
            for _ in range(layers - 1):
                _lib.check(_lib.lib().padoc_branch_decode(
                    C.c_void_p(v["plan"]), C.c_void_p(q_buf.data_ptr()), C.c_void_p(kc.data_ptr()),
                    C.c_void_p(vc.data_ptr()), C.c_void_p(bt.data_ptr()), C.c_void_p(o_buf.data_ptr()),
                    C.c_void_p(l_buf.data_ptr()), C.c_void_p(lws.data_ptr()), lws.numel(), C.c_void_p(st)))

    out = {"pages": args.budget_pages, "max_rows": budget, "layers_per_step": layers, "decoded_tokens": decoded,
           "d_crit_max": int(d_crit.max()), "lower_bound_steps": int(max(d_crit.max(), -(-decoded // budget)))}
    for name, by_pr in (("oldest_first", False), ("critical_path_first", True)):
        bt.fill_(-1)
        sess = pa.DecodeSession(Hq, Hkv, d, n_pool, "bf16", k_cache=kc, v_cache=vc, block_table=bt)
        R = BudgetedReplay(pa, np, sess, nodes, budget, by_pr, launch)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        host = 0.0
        rows = 0
        while not R.done():
            h0 = time.perf_counter()
            rows += R.step()
            host += time.perf_counter() - h0
            torch.cuda.synchronize()   # a decoding loop waits for its outputs before it samples
        wall = time.perf_counter() - t0
        out[name] = {"steps": len(R.steps), "wall_s": wall, "host_s": host, "rows": rows,
                     "tokens_per_s": rows / wall, "mean_rows_per_step": rows / max(1, len(R.steps))}
        sess.destroy()
        log(f"budgeted steps ({name}): {len(R.steps)} steps, {wall:.2f} s")
    del kc, vc, bt, kv_buf, q_buf, o_buf, l_buf, lws
    torch.cuda.empty_cache()
    out["steps_saved"] = out["oldest_first"]["steps"] - out["critical_path_first"]["steps"]
    return out


# ---------------------------------------------------------------- attainable rates on this machine

def attainable(torch, dev):
    """Measured references next to the published peaks: a 2 GiB device copy
    (PyTorch's copy kernel; 2 GiB read + 2 GiB written) and a large bf16
    matrix product (library GEMM, 8192^3)."""
    x = torch.ones(1 << 30, dtype=torch.bfloat16, device=dev)
    y = torch.empty_like(x)
    ms_copy = _event_ms(torch, lambda: y.copy_(x), 5)
    del x, y
    a = torch.randn(8192, 8192, device=dev).to(torch.bfloat16)
    b = torch.randn(8192, 8192, device=dev).to(torch.bfloat16)
    ms_mm = _event_ms(torch, lambda: a @ b, 10)
    del a, b
    torch.cuda.empty_cache()
    return {"copy_gbps": (4 << 30) / (ms_copy * 1e-3) / 1e9, "copy_bytes_read_plus_written": 4 << 30,
            "gemm_bf16_tflops": 2 * 8192 ** 3 / (ms_mm * 1e-3) / 1e12, "gemm_shape": [8192, 8192, 8192]}


def secondary_decode(args, torch, np, syn, pa, dev, name):
    """A smaller decode configuration (its own pool size), summarised; the
    oracle leg checks every query row (at most 17) or 64 sampled rows."""
    wl = syn.make_workload(name, args.seed)
    check = None
    if not args.no_cpu_baseline:
        check = decode_check(args, np, torch, rows_of=lambda nq, w: sampled_rows(np, nq, 64, args.seed + 7,
                                                                                  (0, nq - 1)))
    r, _ = run_decode(args, torch, np, syn, pa, dev, name=name, pool_gib=(wl.pool_bytes or (16 << 30)) / (1 << 30),
                      steps=max(20, args.steps), check=check)
    return {"workload": name, "queries": r["queries"], "cached_tokens": r["cached_tokens"],
            "kernel_us": r["kernel_ms"] * 1e3, "kernel_us_cold_p50": r["kernel_ms_cold_p50"] * 1e3,
            "kernel_us_cold_p10": r["kernel_ms_cold_p10"] * 1e3, "kernel_us_cold_p90": r["kernel_ms_cold_p90"] * 1e3,
            "tokens_per_s": r["tokens_per_s"], "kernel_gbps": r["kernel_gbps"],
            "hbm_frac": r["kernel_gbps"] / HBM_PEAK_GBS, "kernel_tflops": r["kernel_tflops"],
            "mfma_frac": r["kernel_tflops"] / BF16_PEAK_TFLOPS, "sharing_factor": r["sharing_factor"],
            "plan_ms": r["plan_ms"], "oracle": r.get("oracle")}


# ---------------------------------------------------------------- decoding-depth accounting

def depth_accounting(pa, syn, np, name, seed):
    """Per-page sequential depth D_seq, concurrent critical path D_crit and
    forward-step reduction R_step = 1 - D_crit / D_seq (Sec. 3.1, App. D) of
    a workload's pages, taken as complete decoding traces (the layout stream
    and every branch at its full length)."""
    wl = syn.make_workload(name, seed)
    _, d_seq, d_crit = pa.tree_depths(pa.segments_from_pages(wl.pages, 0))
    r = 1.0 - d_crit / np.maximum(d_seq, 1)
    return {"workload": name, "pages": int(len(d_seq)), "d_seq_mean": float(d_seq.mean()),
            "d_crit_mean": float(d_crit.mean()), "r_step_mean": float(r.mean()),
            "r_step_median": float(np.median(r)), "r_step_min": float(r.min()), "r_step_max": float(r.max()),
            "steps_ratio_total": float(d_seq.sum() / max(int(d_crit.sum()), 1))}


# ---------------------------------------------------------------- forward leg

def run_forward(args, torch, np, syn, pa, dev):
    """Packed forward (and its backward) of the forward workload, timed;
    returns (the tensors the oracle leg checks, the summary)."""
    wl = syn.make_workload(args.forward_workload, args.seed)
    assert wl.kind == "forward"
    Hq, Hkv, d = wl.num_heads_q, wl.num_heads_kv, wl.head_dim
    T = syn.count_tokens(wl.pages)
    nq = syn.count_queries(wl.pages)
    segs = pa.segments_from_pages(wl.pages, 0)
    t0 = time.perf_counter()
    plan = pa.TreePlan(segs, Hq, Hkv, d, wl.dtype, 0, num_kv_rows=T, num_q_rows=nq)
    plan_ms = (time.perf_counter() - t0) * 1e3
    q = syn.draw_normal((nq, Hq, d), args.seed, 1, wl.dtype, device=dev)
    k = syn.draw_normal((T, Hkv, d), args.seed, 2, wl.dtype, device=dev)
    v = syn.draw_normal((T, Hkv, d), args.seed, 3, wl.dtype, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty(nq, Hq, dtype=torch.float32, device=dev)
    ws = plan.workspace(dev)
    log(f"forward workload {wl.name}: {len(wl.pages)} pages, {T} tokens")

    def step():
        pa.tree_attn_fwd(q, k, v, plan, out=o, lse=lse, workspace=ws)

    ms, kms = timed_steps(step, max(10, args.steps), args.warmup, torch, pa)
    k_ms = statistics.mean(kms)
    pairs = visible_pairs_of(segs)
    flops = 4 * d * Hq * pairs
    bwd = None
    if not args.no_backward and wl.dtype == "bf16":
        # Backward of the same forward: dO drawn like the inputs; algorithmic
        # flops = 5 products per visible pair (S recomputed, dP, dV, dQ, dK).
        dout = syn.draw_normal((nq, Hq, d), args.seed, 4, wl.dtype, device=dev)
        dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
        bws = plan.backward_workspace(dev)

        def bstep():
            pa.tree_attn_bwd(q, k, v, o, lse, dout, plan, dq=dq, dk=dk, dv=dv, workspace=bws)

        log("backward of the forward workload")
        bms, bkms = timed_steps(bstep, max(10, args.steps // 2), args.warmup, torch, pa)
        bk = statistics.mean(bkms)
        bflops = 10 * d * Hq * pairs
        ex = plan.export()
        bwd = {"ms_per_step": bms, "kernel_ms": bk, "flops": bflops, "kernel_tflops": bflops / (bk * 1e-3) / 1e12,
               "dkdv_items": int(len(ex["bwd"])), "dq_items": int(len(ex["work"])),
               "roofline": {"bound": "mfma", "achieved": bflops / (bk * 1e-3) / 1e12, "peak": BF16_PEAK_TFLOPS,
                            "unit": "TFLOP/s", "frac": bflops / (bk * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
                            "kernel": "backward call: " + " + ".join(BACKWARD_KERNELS)}}
    base, base_out = None, None
    if not args.no_baselines:
        log("forward baselines: dense-mask SDPA, tree-varlen")
        base, base_out = forward_baselines(torch, np, segs, q, k, v, o, Hq, Hkv, d, max(3, args.steps // 5))
        for b in base.values():
            b["useful_tflops"] = flops / (b.get("total_ms", b["ms"]) * 1e-3) / 1e12
            b["tree_speedup"] = b.get("total_ms", b["ms"]) / k_ms
    tensors = {"wl": wl, "q": q, "k": k, "v": v, "o": o, "lse": lse, "baseline_outputs": base_out,
               "grads": (dout, dq, dk, dv) if bwd is not None else None}
    return tensors, {
        "workload": wl.name, "tokens": T, "visible_pairs": pairs, "flops": flops,
        "ms_per_step": ms, "kernel_ms": k_ms, "tflops": flops / (ms * 1e-3) / 1e12,
        "kernel_tflops": flops / (k_ms * 1e-3) / 1e12, "plan_ms": plan_ms,
        "roofline": {"bound": "mfma", "achieved": flops / (k_ms * 1e-3) / 1e12, "peak": BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": flops / (k_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
                     "traffic": measured_traffic()[1], "kernel": FORWARD_KERNEL,
                     "mfma_busy": measured_counters().get(FORWARD_KERNEL, {}).get("mfma_busy")},
        "backward": bwd,
        "baselines": base,
    }


def small_forward(args, torch, np, syn, pa, dev, name="tiny_fp32_forward"):
    """A latency-bound forward configuration (the fp32 path): per-call time
    (HIP events, median of the calls and after a cache flush) and, with the
    CPU leg, every output row against the oracle."""
    wl = syn.make_workload(name, args.seed)
    Hq, Hkv, d = wl.num_heads_q, wl.num_heads_kv, wl.head_dim
    T = syn.count_tokens(wl.pages)
    nq = syn.count_queries(wl.pages)
    segs = pa.segments_from_pages(wl.pages, 0)
    plan = pa.TreePlan(segs, Hq, Hkv, d, wl.dtype, 0, num_kv_rows=T, num_q_rows=nq)
    q = syn.draw_normal((nq, Hq, d), args.seed, 1, wl.dtype, device=dev)
    k = syn.draw_normal((T, Hkv, d), args.seed, 2, wl.dtype, device=dev)
    v = syn.draw_normal((T, Hkv, d), args.seed, 3, wl.dtype, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty(nq, Hq, dtype=torch.float32, device=dev)
    ws = plan.workspace(dev)
    ms, kms = timed_steps(lambda: pa.tree_attn_fwd(q, k, v, plan, out=o, lse=lse, workspace=ws),
                          max(20, args.steps), args.warmup, torch, pa)
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    cold = []
    for _ in range(max(10, args.cold_steps // 5)):
        flush.fill_(1.0)
        b, a = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        b.record()  # creates the underlying events
        a.record()
        pa.set_kernel_events(b, a)
        pa.tree_attn_fwd(q, k, v, plan, out=o, lse=lse, workspace=ws)
        pa.set_kernel_events()
        torch.cuda.synchronize()
        cold.append(b.elapsed_time(a))
    del flush
    pairs = visible_pairs_of(segs)
    res = {"workload": name, "dtype": wl.dtype, "tokens": T, "flops": 4 * d * Hq * pairs,
           "kernel_us": statistics.median(kms) * 1e3, "kernel_us_cold_p50": statistics.median(cold) * 1e3,
           "ms_per_step": ms, "bound": "latency"}
    if not args.no_cpu_baseline:
        import oracle
        from oracle import dense as od
        t0 = time.perf_counter()
        O, L = oracle.tree_attention(od.page_nodes(wl.pages), q, k, v, 1.0 / math.sqrt(d), Hq, Hkv)
        rows = np.arange(nq)
        res["oracle"] = _compare(np, torch, o, lse, O, L, rows, wl.dtype)
        res["oracle"]["oracle_s"] = time.perf_counter() - t0
        log(f"oracle: {name} {nq} rows, O max-abs {res['oracle']['o_max_abs']:.3g}, "
            f"{'ok' if res['oracle']['ok'] else 'FAILED'}")
    return res


# ---------------------------------------------------------------- baselines (measurement only)

def _page_row_ranges(segs):
    """[begin, end) packed rows and segment index range of each page."""
    out = []
    n = len(segs)
    s = 0
    while s < n:
        e = s + 1
        while e < n and int(segs["parent"][e]) >= 0:
            e += 1
        a = int(segs["kv_off"][s])
        b = int(segs["kv_off"][e - 1] + segs["len"][e - 1])
        out.append((a, b, s, e))
        s = e
    return out


def _event_ms(torch, fn, reps):
    fn()
    torch.cuda.synchronize()
    b = torch.cuda.Event(enable_timing=True)
    a = torch.cuda.Event(enable_timing=True)
    b.record()
    for _ in range(reps):
        fn()
    a.record()
    torch.cuda.synchronize()
    return b.elapsed_time(a) / reps


def forward_baselines(torch, np, segs, q, k, v, o_tree, Hq, Hkv, d, reps):
    """The paper's attention backends for the packed tree (App. C), built from
    PyTorch-ROCm operations on the same inputs: (1) dense SDPA with the
    materialised Boolean ancestor mask of each page, (2) tree-varlen: one
    causal problem for prefix + stream and one per branch over the gathered
    [prefix, stream[:fork], branch] keys with bottom-right causal alignment,
    run as one variable-length flash-attention call (or, when that entry is
    missing, one SDPA call per problem).  Returns (timings, outputs); the
    oracle leg checks the outputs against the oracle on sampled rows."""
    import torch.nn.functional as F
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(d)
    pages = _page_row_ranges(segs)
    res = {}
    # (1) dense mask per page
    dev = q.device
    masks, qs, ks, vs = [], [], [], []
    t0 = time.perf_counter()
    for a, b, s0, s1 in pages:
        ns = s1 - s0
        lim = np.zeros((ns, ns), np.int64)
        for s in range(s0, s1):
            t, child = int(segs["parent"][s]), s
            while t >= 0:
                lim[s - s0, t - s0] = int(segs["fork"][child])
                child, t = t, int(segs["parent"][t])
        seg_row = np.repeat(np.arange(ns), segs["len"][s0:s1].astype(np.int64))
        pos_row = np.concatenate([np.arange(int(L)) for L in segs["len"][s0:s1]])
        sr = torch.as_tensor(seg_row, device=dev)
        pr = torch.as_tensor(pos_row, device=dev)
        limt = torch.as_tensor(lim, device=dev)
        m = pr[None, :] < limt[sr[:, None], sr[None, :]]
        same = sr[:, None] == sr[None, :]
        m = torch.where(same, pr[None, :] <= pr[:, None], m)
        masks.append(m[None, None])
        qs.append(q[a:b].transpose(0, 1).unsqueeze(0).contiguous())
        ks.append(k[a:b].repeat_interleave(G, dim=1).transpose(0, 1).unsqueeze(0).contiguous())
        vs.append(v[a:b].repeat_interleave(G, dim=1).transpose(0, 1).unsqueeze(0).contiguous())
    torch.cuda.synchronize()
    mask_ms = (time.perf_counter() - t0) * 1e3

    def dense():
        return [F.scaled_dot_product_attention(qq, kk, vv, attn_mask=mm, scale=scale)
                for qq, kk, vv, mm in zip(qs, ks, vs, masks)]

    outs = dense()
    o_dense = torch.cat([x[0].transpose(0, 1) for x in outs])
    res["dense_sdpa"] = {"ms": _event_ms(torch, dense, reps), "mask_build_ms": mask_ms,
                         "mask_bytes": int(sum(m.numel() for m in masks)),
                         "max_abs_diff_vs_tree": float((o_dense.float() - o_tree.float()).abs().max())}
    del masks, qs, ks, vs, outs
    torch.cuda.empty_cache()

    # (2) tree-varlen: gather the keys of each causal problem
    idx_k, cq, ck = [], [0], [0]
    for a, b, s0, s1 in pages:
        P, S = int(segs["len"][s0]), int(segs["len"][s0 + 1])
        m_rows = np.arange(a, a + P + S)
        idx_k.append(m_rows)
        cq.append(cq[-1] + P + S)
        ck.append(ck[-1] + P + S)
        for s in range(s0 + 2, s1):
            f, L, r0 = int(segs["fork"][s]), int(segs["len"][s]), int(segs["kv_off"][s])
            rows = np.concatenate([np.arange(a, a + P + f), np.arange(r0, r0 + L)])
            idx_k.append(rows)
            cq.append(cq[-1] + L)
            ck.append(ck[-1] + len(rows))
    idx = torch.as_tensor(np.concatenate(idx_k), device=dev)
    cum_q = torch.as_tensor(np.array(cq, np.int32), device=dev)
    cum_k = torch.as_tensor(np.array(ck, np.int32), device=dev)
    max_q = int(np.diff(cq).max())
    max_k = int(np.diff(ck).max())

    def gather():
        return (k.index_select(0, idx).repeat_interleave(G, dim=1),
                v.index_select(0, idx).repeat_interleave(G, dim=1))

    kg, vg = gather()
    method = "aten._flash_attention_forward (varlen, causal)"

    def varlen():
        return torch.ops.aten._flash_attention_forward(q, kg, vg, cum_q, cum_k, max_q, max_k, 0.0, True, False,
                                                        scale=scale)[0]

    from torch.nn.attention.bias import causal_lower_right
    probs = [(cq[i], cq[i + 1], ck[i], ck[i + 1]) for i in range(len(cq) - 1)]

    def per_problem():
        out = torch.empty_like(q)
        for q0, q1, k0, k1 in probs:
            qq = q[q0:q1].transpose(0, 1).unsqueeze(0)
            kk = kg[k0:k1].transpose(0, 1).unsqueeze(0)
            vv = vg[k0:k1].transpose(0, 1).unsqueeze(0)
            out[q0:q1] = F.scaled_dot_product_attention(
                qq, kk, vv, attn_mask=causal_lower_right(q1 - q0, k1 - k0), scale=scale)[0].transpose(0, 1)
        return out

    try:
        o_var = varlen()
        torch.cuda.synchronize()
        # A gross disagreement (e.g. top-left causal alignment, which is not
        # the tree-varlen relation) means the entry does not compute this
        # problem: use the per-problem form.  Whether either form is right
        # is decided against the oracle, not here.
        bad = float((o_var.float() - o_tree.float()).abs().max())
        if not bad < 0.1:
            raise ValueError(f"varlen output differs from the tree's by {bad:.3g}")
    except Exception as e:  # the entry is not built into every PyTorch
        log(f"varlen flash entry not usable ({type(e).__name__}: {e}); one SDPA call per problem instead")
        method = "SDPA per problem, causal_lower_right"
        varlen = per_problem
        o_var = varlen()
    res["tree_varlen"] = {"ms": _event_ms(torch, varlen, reps), "gather_ms": _event_ms(torch, gather, reps),
                          "method": method, "problems": len(cq) - 1, "gathered_key_rows": int(idx.numel()),
                          "max_abs_diff_vs_tree": float((o_var.float() - o_tree.float()).abs().max())}
    res["tree_varlen"]["total_ms"] = res["tree_varlen"]["ms"] + res["tree_varlen"]["gather_ms"]
    return res, {"dense_sdpa": o_dense, "tree_varlen": o_var}


def decode_baselines(args, torch, np, syn, pa, dev, wl, tree_ms):
    """The decode step without tree sharing, on the same kernels: every
    stream as its own sequence (root) holding its whole visible path --
    (a) with private copies of every block, (b) with prefix blocks reused
    across the streams of a page (block-granular prefix caching: full blocks
    of the prefix and of the stream up to the fork are shared, the rest of
    the path is the stream's own).  The kernels then read each stream's path
    once per stream."""
    Hq, Hkv, d = wl.num_heads_q, wl.num_heads_kv, wl.head_dim
    paths = []   # per stream: (page, prefix tokens, stream tokens seen, own tokens)
    for pg, p in enumerate(wl.pages):
        paths.append((pg, p.prefix_len, p.stream_len, 0))   # the layout stream: prefix + its own tokens
        for b in p.branches:
            paths.append((pg, p.prefix_len, b.fork, b.length))
    n = len(paths)
    lens = np.array([P + f + L for _, P, f, L in paths], np.int64)
    nodes = [(-1, 0, int(x), 1) for x in lens]
    segs = pa.segments_layout(nodes, 16)
    q = torch.randn((n, Hq, d), device=dev).to(torch.bfloat16)
    out = {}
    for variant in ("private_copies", "prefix_block_reuse"):
        if variant == "private_copies":
            nb = int(sum(-(-int(x) // 16) for x in lens))
            table = np.arange(nb, dtype=np.int32)
            n_pool = nb
        else:
            # the page's [prefix | stream] tokens fill its own blocks; a
            # stream's sequence shares the ones entirely inside its first
            # prefix + fork tokens, the rest of its blocks are its own
            ids, nxt, page_blocks = [], 0, {}
            for pg, p in enumerate(wl.pages):
                nb_pg = -(-(p.prefix_len + p.stream_len) // 16)
                page_blocks[pg] = np.arange(nxt, nxt + nb_pg)
                nxt += nb_pg
            for pg, P, f, L in paths:
                sh = (P + f) // 16
                total = -(-(P + f + L) // 16)
                ids.append(np.concatenate([page_blocks[pg][:sh], np.arange(nxt, nxt + total - sh)]))
                nxt += total - sh
            table = np.concatenate(ids).astype(np.int32)
            n_pool = nxt
        assert len(table) == int(sum(-(-int(x) // 16) for x in lens))
        kc = torch.randn((n_pool, Hkv, d // 8, 16, 8), device=dev).to(torch.bfloat16)
        vc = torch.randn((n_pool, Hkv, d, 16), device=dev).to(torch.bfloat16)
        bt = torch.as_tensor(table, device=dev)
        plan = pa.TreePlan(segs, Hq, Hkv, d, "bf16", 16, num_kv_rows=n_pool, num_q_rows=n,
                           block_table_len=len(table))
        o = torch.empty_like(q)
        lse = torch.empty(n, Hq, dtype=torch.float32, device=dev)
        ws = plan.workspace(dev)

        def step():
            pa.branch_decode(q, kc, vc, bt, plan, out=o, lse=lse, workspace=ws)

        _, kms = timed_steps(step, max(10, args.steps // 2), args.warmup, torch, pa)
        km = statistics.mean(kms)
        path_bytes = int(lens.sum()) * Hkv * d * 2 * 2
        out[variant] = {"kernel_ms": km, "tokens_per_s": n / (km * 1e-3), "path_kv_bytes": path_bytes,
                        "pool_bytes": 2 * n_pool * Hkv * 16 * d * 2, "path_gbps": path_bytes / (km * 1e-3) / 1e9,
                        "tree_speedup": km / tree_ms}
        del kc, vc, bt, plan, ws
        torch.cuda.empty_cache()
    return out


# ---------------------------------------------------------------- oracle leg (CPU baseline, parity)
#
# The oracle runs here only.  Its dense-mask attention over the decode
# workload is the reported CPU baseline, and its outputs are compared with
# the GPU outputs of the same run: the headline decode call on the timed
# pool, the other decode configurations, the timed packed forward, the
# baselines next to it, and the timed backward.

TOL = {"bf16": (1.5e-2, 2e-3), "f32": (1e-5, 1e-5)}
# Backward: the bf16 bounds in units of each gradient's scale (the larger of
# the tensor's RMS and the element's row RMS for the max, the tensor's RMS for
# the mean), plus one bf16 ulp of the element for the max (the output is
# rounded to nearest even after fp32 accumulation).
BWD_ULP = 2.0 ** -8


def cpu_info():
    """(CPU model as lscpu names it, BLAS threads the oracle uses)."""
    import subprocess
    model = ""
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        kv = {l.split(":", 1)[0].strip(): l.split(":", 1)[1].strip() for l in out.splitlines() if ":" in l}
        model = kv.get("Model name", "")
        # a virtual machine may name only the vendor line; family / model /
        # stepping and the core count still identify the part
        extra = [f"{k.lower()} {kv[k]}" for k in ("CPU family", "Model", "Stepping") if kv.get(k)]
        if model and extra:
            model += " (" + ", ".join(extra) + f"; {kv.get('CPU(s)', '?')} CPUs)"
    except (OSError, subprocess.SubprocessError):
        pass
    if not model:
        try:
            with open("/proc/cpuinfo") as fh:
                model = next((l.split(":", 1)[1].strip() for l in fh if l.startswith("model name")), "")
        except OSError:
            pass
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        cores = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    return model, int(cores)


def _compare(np, torch, o_gpu, lse_gpu, O, L, rows, dtype):
    """Element-wise errors of GPU rows against the oracle's (fp64) rows."""
    rows = np.asarray(sorted(set(int(r) for r in rows)), dtype=np.int64)
    ri = torch.as_tensor(rows, device=o_gpu.device)
    o = o_gpu.index_select(0, ri).to("cpu", torch.float64).numpy()
    finite = bool(np.isfinite(o).all())
    eo = np.abs(o - O[rows])
    mx, mn = TOL[dtype]
    r = {"rows": int(rows.size), "o_max_abs": float(eo.max()), "o_mean_abs": float(eo.mean())}
    ok = finite and r["o_max_abs"] <= mx and (dtype != "bf16" or r["o_mean_abs"] <= mn)
    if lse_gpu is not None:
        l = lse_gpu.index_select(0, ri).to("cpu", torch.float64).numpy()
        el = np.abs(l - L[rows])
        r.update(lse_max_abs=float(el.max()), lse_mean_abs=float(el.mean()))
        finite = finite and bool(np.isfinite(l).all())
        ok = ok and finite and r["lse_max_abs"] <= mx and (dtype != "bf16" or r["lse_mean_abs"] <= mn)
    r["finite"] = finite
    r["ok"] = bool(ok)
    return r


def decode_check(args, np, torch, rows_of=None, baseline=False):
    """Oracle check of a decode call, run while its pool is resident: the
    oracle gathers the used blocks from the timed pool with its own code
    (untimed), then computes the dense-mask attention of the selected query
    rows (all rows when `rows_of` is None).  With `baseline`, the oracle's
    wall time is the CPU baseline."""
    import oracle
    from oracle import dense as od

    def check(wl, q, kc, vc, ids, o, lse):
        nodes = od.page_nodes(wl.pages)
        nq = q.shape[0]
        rows = list(range(nq)) if rows_of is None else rows_of(nq, wl)
        k = od.gather_paged(nodes, kc, ids, 16, layout="chunked")
        v = od.gather_paged(nodes, vc, ids, 16, d_major=True)
        q64 = q.to("cpu", torch.float64).numpy()
        t0 = time.perf_counter()
        O, L = oracle.tree_attention(nodes, q64, k, v, 1.0 / math.sqrt(wl.head_dim), wl.num_heads_q,
                                     wl.num_heads_kv, rows=None if rows_of is None else rows)
        dt = time.perf_counter() - t0
        r = _compare(np, torch, o, lse, O, L, rows, wl.dtype)
        r["oracle_s"] = dt
        if baseline:
            model, cores = cpu_info()
            T = syn_count_tokens(wl)
            r["cpu_baseline"] = {
                "value": len(rows) / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle", "cpu_model": model,
                "sample": f"all {len(wl.pages)} pages of the decode step ({len(rows)} queries, {T} cached tokens): "
                          f"fp64 dense ancestor mask per page, {dt:.1f} s wall (after the oracle's own gather "
                          "of the used blocks from the timed pool, not timed)"}
        log(f"oracle: {wl.name} {r['rows']} rows, O max-abs {r['o_max_abs']:.3g} mean-abs {r['o_mean_abs']:.3g}, "
            f"LSE max-abs {r['lse_max_abs']:.3g}, {'ok' if r['ok'] else 'FAILED'} ({dt:.1f} s)")
        return r

    return check


def syn_count_tokens(wl):
    return sum(p.prefix_len + p.stream_len + sum(b.length for b in p.branches) for p in wl.pages)


def sampled_rows(np, nq, n_random, seed, must=()):
    rng = np.random.default_rng(seed)
    return sorted(set(rng.choice(nq, min(n_random, nq), replace=False).tolist()) | set(int(x) for x in must))


def forward_check(np, torch, fwd_t, seed):
    """Oracle check of the timed packed forward (sampled rows: 400 random plus
    the first and last query of every fourth segment), of the baselines'
    outputs on the same rows, and of the timed backward on one whole page
    (every dQ row of its queries, every dK / dV row of its keys)."""
    import oracle
    from oracle import dense as od
    wl, q, k, v, o, lse = fwd_t["wl"], fwd_t["q"], fwd_t["k"], fwd_t["v"], fwd_t["o"], fwd_t["lse"]
    Hq, Hkv, d = wl.num_heads_q, wl.num_heads_kv, wl.head_dim
    scale = 1.0 / math.sqrt(d)
    nodes = od.page_nodes(wl.pages)
    kv_off, q_off = od.canonical_layout(nodes, 0)
    must = []
    for s, n in enumerate(nodes):
        if s % 4 == 0 and n[3] > 0:
            must += [int(q_off[s]), int(q_off[s] + n[3] - 1)]
    rows = sampled_rows(np, q.shape[0], 400, seed + 11, must)
    q64, k64, v64 = (x.to("cpu", torch.float64).numpy() for x in (q, k, v))
    t0 = time.perf_counter()
    O, L = oracle.tree_attention(nodes, q64, k64, v64, scale, Hq, Hkv, rows=rows)
    out = {"forward": _compare(np, torch, o, lse, O, L, rows, wl.dtype)}
    out["forward"]["oracle_s"] = time.perf_counter() - t0
    log(f"oracle: forward {len(rows)} rows, O max-abs {out['forward']['o_max_abs']:.3g}, "
        f"{'ok' if out['forward']['ok'] else 'FAILED'}")
    for name, ob in (fwd_t.get("baseline_outputs") or {}).items():
        out[f"baseline_{name}"] = _compare(np, torch, ob, None, O, L, rows, wl.dtype)
        log(f"oracle: baseline {name} O max-abs {out[f'baseline_{name}']['o_max_abs']:.3g}, "
            f"{'ok' if out[f'baseline_{name}']['ok'] else 'FAILED'}")
    if fwd_t.get("grads") is not None:
        dout, dq, dk, dv = fwd_t["grads"]
        roots = [s for s, n in enumerate(nodes) if n[0] < 0]
        sizes = []
        for i, r0 in enumerate(roots):
            r1 = roots[i + 1] if i + 1 < len(roots) else len(nodes)
            sizes.append((sum(n[2] for n in nodes[r0:r1]), r0, r1))
        _, r0, r1 = min(sizes)   # the smallest page (prefix, stream and branches)
        sub = nodes[r0:r1]
        sub = [(-1 if p < 0 else p - r0, f, n, ql) for p, f, n, ql in sub]
        t0 = time.perf_counter()
        dQ, dK, dV = oracle.tree_attention_backward(sub, q64, k64, v64, dout.to("cpu", torch.float64).numpy(),
                                                    scale, Hq, Hkv, kv_off=kv_off[r0:r1], q_off=q_off[r0:r1],
                                                    o=o.to("cpu", torch.float64).numpy())
        qrows = np.concatenate([q_off[s] + np.arange(nodes[s][3]) for s in range(r0, r1)]).astype(np.int64)
        krows = np.concatenate([kv_off[s] + np.arange(nodes[s][2]) for s in range(r0, r1)]).astype(np.int64)
        b = {"page": int(roots.index(r0)), "q_rows": int(qrows.size), "kv_rows": int(krows.size),
             "oracle_s": time.perf_counter() - t0}
        ok = True
        for name, g, ref, rr in (("dq", dq, dQ, qrows), ("dk", dk, dK, krows), ("dv", dv, dV, krows)):
            x = g.index_select(0, torch.as_tensor(rr, device=g.device)).to("cpu", torch.float64).numpy()
            r = ref[rr]
            s = float(np.sqrt(np.mean(r * r))) or 1.0
            err = np.abs(x - r)
            s_el = np.maximum(s, np.sqrt(np.mean(r * r, axis=2, keepdims=True)))
            e_max = float(np.max(np.maximum(err - BWD_ULP * np.abs(r), 0.0) / s_el))
            e_mean = float(err.mean() / s)
            good = bool(np.isfinite(x).all()) and e_max <= TOL["bf16"][0] and e_mean <= TOL["bf16"][1]
            b[name] = {"rms": s, "max_err_minus_ulp_over_scale": e_max, "mean_err_over_rms": e_mean, "ok": good}
            ok = ok and good
        b["ok"] = ok
        out["backward"] = b
        log(f"oracle: backward page {b['page']} ({b['q_rows']} query rows, {b['kv_rows']} key rows), "
            f"{'ok' if ok else 'FAILED'} ({b['oracle_s']:.1f} s)")
    return out


def main(argv=None) -> int:
    args = parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on exactly one GPU (asked for --gpus {args.gpus}, WORLD_SIZE={world}); pages are "
              "independent trees, so several GPUs would shard by page with no exchange -- not built here.",
              file=sys.stderr)
        return 2
    if args.summarize_profile:
        summarize_profile(args.summarize_profile)
        return 0
    import numpy as np
    import torch

    import padoc_synth as syn
    import paper_2608_06146_amd as pa

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calibrate_copy:
        src = torch.ones(1 << 29, dtype=torch.bfloat16, device=dev)   # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": src.numel() * 2, "copy_bytes_written": dst.numel() * 2}))
        return 0
    pa.version()  # loads the library (fails loudly if it was not built)

    dec, wl = run_decode(args, torch, np, syn, pa, dev,
                         check=None if args.no_cpu_baseline else decode_check(args, np, torch, baseline=True))
    others = None
    if not args.no_secondary:
        others = [secondary_decode(args, torch, np, syn, pa, dev, n)
                  for n in ("single_page_decode", "dense_page_mixed_step")]
    refs = None if args.no_baselines else attainable(torch, dev)
    drv = run_driver(args, torch, np, syn, pa, dev, wl) if args.driver_steps > 0 else None
    if drv is not None and args.budget_pages > 0:
        drv["budgeted"] = run_budgeted(args, torch, np, pa, dev)
    if not args.no_baselines:
        log("decode baselines: per-stream sequences without tree sharing")
        dec["baselines"] = decode_baselines(args, torch, np, syn, pa, dev, wl, dec["kernel_ms"])
    fwd, fwd_check = None, None
    small = None
    if args.forward_workload != "none" and not args.no_secondary:
        small = [small_forward(args, torch, np, syn, pa, dev)]
    if args.forward_workload != "none":
        fwd_t, fwd = run_forward(args, torch, np, syn, pa, dev)
        if not args.no_cpu_baseline:
            fwd_check = forward_check(np, torch, fwd_t, args.seed)
        del fwd_t
    cpu, parity = None, None
    if not args.no_cpu_baseline:
        dec_or = dec.pop("oracle")
        cpu = dec_or.pop("cpu_baseline")
        parity = {"tolerance": {"bf16_max_abs": TOL["bf16"][0], "bf16_mean_abs": TOL["bf16"][1],
                                "f32_max_abs": TOL["f32"][0]},
                  "decode": dec_or}
        for x in (others or []) + (small or []):
            parity[x["workload"]] = x.pop("oracle")
        if fwd_check:
            parity.update(fwd_check)
        parity["ok"] = all(v.get("ok", True) for k, v in parity.items() if k not in ("tolerance",))

    line = {
        "metric": METRIC,
        "value": dec["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dec["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": dec["workload"], "pages": dec["pages"], "branches_per_page": 24,
                   "queries": dec["queries"], "cached_tokens": dec["cached_tokens"], "Hq": dec["Hq"],
                   "Hkv": dec["Hkv"], "d": dec["d"], "block": 16, "pool_gib": round(dec["pool_gib"], 1)},
        "hbm_gbps": dec["step_gbps"],
        # headline roofline: the cold-cache median call (a 1 GiB write
        # between calls); the warm mean of back-to-back calls is secondary
        "roofline": {"bound": "hbm", "achieved": dec["kernel_gbps_cold"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": dec["kernel_gbps_cold"] / HBM_PEAK_GBS, "traffic": measured_traffic()[0],
                     "kernel": "decode call: " + " + ".join(DECODE_KERNELS),
                     "kernel_ms": dec["kernel_ms_cold_p50"], "kernel_ms_p10": dec["kernel_ms_cold_p10"],
                     "kernel_ms_p90": dec["kernel_ms_cold_p90"], "timing": "cold-cache median",
                     "warm_kernel_ms": dec["kernel_ms"], "warm_frac": dec["kernel_gbps"] / HBM_PEAK_GBS,
                     "bytes_per_launch": dec["kernel_bytes"]},
        "cpu_baseline": cpu,
        "parity": parity,
        "decode": dec,
        "other_decode_configs": others,
        "other_forward_configs": small,
        "attainable": refs,
        "driver": drv,
        "accounting": [depth_accounting(pa, syn, np, n, args.seed)
                       for n in ("concurrent_decode_64pages", "packed_forward_8pages")],
        "forward": fwd,
    }
    print(json.dumps(line), flush=True)
    if parity is not None and not parity["ok"]:
        log("PARITY FAILED: a timed output is outside the oracle tolerance (see \"parity\")")
        return 1
    return 0


if __name__ == "__main__":
    sys.exit(main())
