#!/usr/bin/env python3
"""Throughput of the paged KV-cache transfer path on one MI355X.

One step is one pass of the whole path over one batch of requests on
synthetic pools already resident in HBM.  With no flags the headline is the
largest workload, the MLA latent cache:
- 61 layers x one 576-wide latent (512 + 64 rope), bf16, 64-token pages;
- about 18.7k-page pools on both sides, layout [layer][page][kv][token][head][dim];
- 64 requests with lengths uniform in [4096, 32768], copying positions
  [p, len) with p uniform in [0, len/2), so pages start unaligned.
A step is one planned transfer (kvx_transfer_planned) of all 64 requests.
The library picks between its two launches by timing both on the first
warmup steps (``--launch-choice``), and ``roofline.launch`` names the one the
timed steps took.  The same run then measures
the other three transfer workloads of the benchmark set, one at a time
(each allocates its pools, is timed, sample-checked against the CPU oracle
and freed before the next), and reports them under ``context.configs``:
- handoff: 36 layers x 8 KV heads x 128, 4096 x 64-token pools, 32
  requests of 1024-8192 tokens, one fused transfer;
- relayout: 28 x 4 x 128, 16-token token-major pages into 64-token
  head-major pages, 16 requests of 2048-16384 tokens;
- host_tier: the handoff pool, 1820 pages (16 GiB) gathered into pinned host
  memory and scattered back into fresh pages (PCIe-bound).

``--workload`` measures one workload alone instead: those four, tp_reshard
(a head range into a narrower pool), cow_fork (copy-on-write inside one
pool), handoff_layered (the handoff in 4-layer groups with an event each),
small_requests (16384 requests of 1-4 tokens), host_tier_v (the host tier
for the V half only) or page_hash (chained page hashes of token ids).

GB/s counts algorithmic bytes, GB = 1e9: every copied token position is read
once and written once, 2 * tokens * L*C*H*D*e per step.

Printed as one JSON line:
- ``value``: algorithmic bytes per step / wall time per step.
- ``roofline``: the transfer kernel's own rate.  Its bytes per launch are
  divided by the average launch duration, measured with HIP events on the
  launch stream, and compared with the 8 TB/s HBM peak (63 GB/s per
  direction of PCIe 5.0 x16 for the host tier).
- ``cpu_baseline``: the CPU oracle timed on this host over a sample of
  layers, which are also compared bit for bit with the GPU result.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "KV transfer GB/s (read+write) and % of HBM/host-link peak, 1 MI355X"
HBM_PEAK_GBPS = 8000.0        # MI355X HBM3E, published
PCIE_PEAK_GBPS = 63.0         # PCIe 5.0 x16 per direction: 32 GT/s x 16 x 128/130 / 8
HEADLINE = "mla"
CONTEXT = ("handoff", "relayout", "host_tier")
# Sources of each kernel and its launch shape; a change here invalidates the
# committed HBM counter records of the workloads that run it.
COPY_SOURCES = ["paper_2606_31093_amd/csrc/kvx_kernels.hip",
                "paper_2606_31093_amd/csrc/kvx_internal.h"]
HASH_SOURCES = ["paper_2606_31093_amd/csrc/kvx_hash.hip",
                "paper_2606_31093_amd/csrc/kvx_hash.h"]


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_sha(workload: str = "handoff") -> str:
    h = hashlib.sha256()
    for p in HASH_SOURCES if workload == "page_hash" else COPY_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_record(key: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary,
    if it was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{key}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_sha") != kernel_sha(key):
        return None
    return rec


# --launch-choice values and their KVX_CHOOSE_* modes
LAUNCH_CHOICES = {"measured": 0, "sweep": 1, "grid": 2}
# Calls the library's measured launch choice takes on a pool pair before it
# keeps one launch (six untimed, four timed).
CHOICE_CALLS = 10

WORKLOADS = ["mla", "handoff", "relayout", "host_tier", "tp_reshard", "cow_fork",
             "handoff_layered", "small_requests", "host_tier_v", "page_hash"]


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=None, choices=WORKLOADS,
                    help="measure one workload alone (default: the MLA headline plus the "
                         "handoff, relayout and host tier under context.configs)")
    ap.add_argument("--cpu-layers", type=int, default=12,
                    help="layers of the headline workload the CPU oracle runs (0: skip)")
    ap.add_argument("--check-layers", type=int, default=4,
                    help="layers of each context workload compared with the oracle (0: skip)")
    ap.add_argument("--cpu-threads", type=int, default=16,
                    help="most host threads for the multi-threaded oracle timing")
    ap.add_argument("--no-memcpy", action="store_true", help="skip the hipMemcpy reference")
    ap.add_argument("--unplanned", action="store_true",
                    help="launch transfers with kvx_transfer(_slice, _layered) instead of their planned forms")
    ap.add_argument("--launch-choice", default="measured", choices=("measured", "sweep", "grid"),
                    help="how planned transfers that can sweep pick their launch (kvx_set_launch_choice); "
                         "measured, the library's default, times both on the warmup steps")
    ap.add_argument("--calibrate-copy", type=float, default=0.0, metavar="GIB",
                    help="only run a plain device copy of this many GiB (counter calibration)")
    return ap.parse_args()


def calibrate_copy(gib: float) -> None:
    """A plain copy kernel of known size, for scaling rocprofv3 byte counters."""
    import torch
    n = int(gib * 2**30)
    a = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": n, "launches": 3}), flush=True)


def main() -> int:
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "kvx is measured on one GPU; the library has no multi-GPU path, "
                                   "so --gpus must be 1", "n_gpus": args.gpus}), flush=True)
        return 2
    if int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only (WORLD_SIZE must be 1)", file=sys.stderr)
        return 2

    import torch

    if args.calibrate_copy > 0:
        calibrate_copy(args.calibrate_copy)
        return 0

    from paper_2606_31093_amd import build_lib, kvx

    if not os.path.exists(build_lib.LIBRARY):
        log("libkvx.so missing: building")
        build_lib.build()
    kvx.lib()
    kvx.kvx_set_launch_choice(LAUNCH_CHOICES[args.launch_choice])
    if args.workload == "page_hash":
        return hash_bench(args)

    name = args.workload or HEADLINE
    res = measure(name, args, cpu_layers=args.cpu_layers, time_cpu=True)
    if res is None:
        return 1
    context = res.pop("context")
    if args.workload is None:
        context["configs"] = {}
        for k in CONTEXT:
            torch.cuda.empty_cache()
            r = measure(k, args, cpu_layers=args.check_layers, time_cpu=False)
            if r is None:
                return 1
            context["configs"][k] = summary(r)
    out = {
        "metric": METRIC, "value": res["value"], "unit": "GB/s", "n_gpus": 1,
        "steps": res["steps"], "warmup": res["warmup"], "ms_per_step": res["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u16",
        "data": "synthetic (seeded N(0,1) bf16 source, offset-coded destination prefill)",
        "config": res["config"],
        "roofline": res["roofline"],
        "cpu_baseline": res["cpu_baseline"],
        "context": context,
    }
    print(json.dumps(out), flush=True)
    return 0


def summary(r: dict) -> dict:
    """The per-workload entry of context.configs."""
    c = r["context"]
    s = {"workload": r["config"]["workload"], "steps": r["steps"], "ms_per_step": r["ms_per_step"],
         "value_GBps": r["value"], "roofline": r["roofline"],
         "sample_bit_exact": r["sample_bit_exact"], "sample_layers": r["sample_layers"]}
    for k in ("per_step_kernel_ms", "per_step_kernel_ms_median", "per_step_kernel_ms_min",
              "hip_memcpy_d2d_GBps_read_plus_write", "hip_memcpy_d2h_GBps",
              "hip_memcpy_h2d_GBps", "per_op", "both_launches_GBps"):
        if k in c:
            s[k] = c[k]
    return s


def launch_step(kvx, wl, mem, d, errw):
    st = d["st"]
    S, D = wl.sides[st.src], wl.sides[st.dst]
    if st.op == "transfer" and d.get("plan") is not None and st.layer_group:
        kvx.kvx_transfer_layered_planned(mem[st.src], S, mem[st.dst], D, d["spt"], d["dpt"], d["reqs"],
                                         st.layer_group, d["events"], d["plan"], d["plan_pages"],
                                         d["plan_tokens"], st.slice, errw)
    elif st.op == "transfer" and d.get("plan") is not None:
        kvx.kvx_transfer_planned(mem[st.src], S, mem[st.dst], D, d["spt"], d["dpt"], d["reqs"],
                                 d["plan"], d["plan_pages"], d["plan_tokens"], st.slice, errw)
    elif st.op == "transfer" and st.layer_group:
        kvx.kvx_transfer_layered(mem[st.src], S, mem[st.dst], D, d["spt"], d["dpt"], d["reqs"],
                                 st.layer_group, d["events"], st.slice, errw)
    elif st.op == "transfer" and st.slice is not None:
        kvx.kvx_transfer_slice(mem[st.src], S, mem[st.dst], D, st.slice, d["spt"], d["dpt"],
                               d["reqs"], errw)
    elif st.op == "transfer":
        kvx.kvx_transfer(mem[st.src], S, mem[st.dst], D, d["spt"], d["dpt"], d["reqs"], errw)
    elif st.op == "gather" and st.slice is not None:
        kvx.kvx_gather_slice(mem[st.src], S, mem[st.dst], D, st.slice, d["spt"], d["reqs"], errw)
    elif st.op == "gather":
        kvx.kvx_gather(mem[st.src], S, mem[st.dst], D, d["spt"], d["reqs"], errw)
    elif st.slice is not None:
        kvx.kvx_scatter_slice(mem[st.src], S, mem[st.dst], D, st.slice, d["dpt"], d["reqs"], errw)
    else:
        kvx.kvx_scatter(mem[st.src], S, mem[st.dst], D, d["dpt"], d["reqs"], errw)


def measure(name: str, args, cpu_layers: int, time_cpu: bool):
    """Allocate, fill, time, check and free one workload.  Returns a dict of
    the line's fields for it, or None if the device reported an error or a
    checked layer differs from the oracle."""
    import torch

    from paper_2606_31093_amd import kvx, workloads

    dev = torch.device("cuda", 0)
    wl = workloads.get(name)
    log(f"workload: {wl.title}")
    mem = {}
    for side, spec in wl.sides.items():
        pinned = side in wl.host_sides
        log(f"allocating side {side}: {spec.nbytes / 2**30:.2f} GiB "
            f"{'pinned host' if pinned else 'HBM'}")
        mem[side] = workloads.alloc_side(spec, dev, pinned=pinned)
    log("filling source values and destination prefill")
    workloads.init_sides_(wl, mem)
    dsteps = []
    for st in wl.steps:
        dsteps.append(dict(
            st=st,
            spt=kvx.device_table(st.src_pt, dev) if st.src_pt is not None else None,
            dpt=kvx.device_table(st.dst_pt, dev) if st.dst_pt is not None else None,
            reqs=kvx.device_reqs(st.reqs, dev),
            events=[torch.cuda.Event(enable_timing=True)
                    for _ in range(-(-wl.sides[st.src].L // st.layer_group))]
            if st.layer_group else None,
            # the plan of destination pages, built on the host from the records
            # and uploaded with them (kvx_transfer_planned)
            **(dict(zip(("plan", "plan_pages", "plan_tokens"),
                        kvx.device_plan(st.reqs, wl.sides[st.src].T, wl.sides[st.dst].T, dev)))
               if st.op == "transfer" and not args.unplanned else {})))
    errw = torch.zeros(1, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()

    # A copy inside one pool, and the host tier's offload + onload (whose
    # onload pages may overlap the offloaded ones), change what the next step
    # reads: they are checked on one extra step from a snapshot of the pool.
    replay = len({st.dst for st in wl.steps} & {st.src for st in wl.steps}) > 0
    host_leg = bool(wl.host_sides)
    steps = args.steps if not host_leg else min(args.steps, 5)
    warmup = args.warmup if not host_leg else min(args.warmup, 1)

    # A planned transfer in the measured launch choice settles on one launch
    # within CHOICE_CALLS calls; fewer warmup steps get the missing calls
    # first, untimed, so that the timed steps all take the kept launch.
    choosing = (kvx.kvx_launch_choice() == kvx.CHOOSE_MEASURED and
                any(d.get("plan") is not None and not d["st"].layer_group for d in dsteps))
    choice_calls = max(0, CHOICE_CALLS - warmup) if choosing else 0
    log(f"warmup: {warmup} steps" + (f" after {choice_calls} launch-choice calls" if choice_calls else ""))
    for _ in range(choice_calls + warmup):
        for d in dsteps:
            launch_step(kvx, wl, mem, d, errw)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    events = [[] for _ in dsteps]
    launches = [set() for _ in dsteps]     # the launch kinds each step took while timed
    log(f"timing: {steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        for i, d in enumerate(dsteps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            launch_step(kvx, wl, mem, d, errw)
            e1.record(stream)
            events[i].append((e0, e1))
            launches[i].add(kvx.LAUNCH_NAMES[kvx.kvx_last_launch()])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    dev_err = int(errw.item())
    if dev_err:
        log(f"device error bits {dev_err}")
        return None

    ms_per_step = (t1 - t0) * 1e3 / steps
    step_bytes = sum(wl.algorithmic_bytes(st) for st in wl.steps)
    value = step_bytes / (ms_per_step / 1e3) / 1e9
    kern_ms = [sum(a.elapsed_time(b) for a, b in ev) / len(ev) for ev in events]
    log(f"{ms_per_step:.3f} ms/step, {value:.1f} GB/s; kernel ms {kern_ms}")

    i_dom = max(range(len(dsteps)), key=lambda i: kern_ms[i])
    dom = wl.steps[i_dom]
    dom_bytes = wl.algorithmic_bytes(dom)
    launch = "+".join(sorted(launches[i_dom]))
    log(f"launch of the timed steps: {launch}")
    tr = traffic_record(name)
    traffic = tr.get("by_launch", {}).get(launch) if tr else None
    if host_leg:
        one_way = dom_bytes / 2
        rate = one_way / (kern_ms[i_dom] / 1e3) / 1e9
        roofline = {"bound": "pcie", "achieved": round(rate, 2), "peak": PCIE_PEAK_GBPS,
                    "unit": "GB/s", "frac": round(rate / PCIE_PEAK_GBPS, 4),
                    "traffic": traffic, "kernel": f"kvx {dom.op}", "launch": launch,
                    "bytes_per_launch": int(one_way), "kernel_ms": round(kern_ms[i_dom], 4)}
    else:
        rate = dom_bytes / (kern_ms[i_dom] / 1e3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(rate, 1), "peak": HBM_PEAK_GBPS,
                    "unit": "GB/s", "frac": round(rate / HBM_PEAK_GBPS, 4),
                    "traffic": traffic, "kernel": f"kvx {dom.op}", "launch": launch,
                    "bytes_per_launch": int(dom_bytes), "kernel_ms": round(kern_ms[i_dom], 4)}

    reps = [sorted(a.elapsed_time(b) for a, b in ev) for ev in events]
    context = {"kernel_sha": kernel_sha(name),
               "launch_choice": {v: k for k, v in LAUNCH_CHOICES.items()}[kvx.kvx_launch_choice()],
               "launches": ["+".join(sorted(x)) for x in launches],
               "launch_choice_calls": choice_calls,
               "per_step_kernel_ms": [round(x, 4) for x in kern_ms],
               "per_step_kernel_ms_median": [round(r[len(r) // 2], 4) for r in reps],
               "per_step_kernel_ms_min": [round(r[0], 4) for r in reps]}
    if host_leg:
        context["per_op"] = {st.op: {"kernel_ms": round(kern_ms[i], 4),
                                     "one_way_GBps": round(wl.algorithmic_bytes(st) / 2 /
                                                           (kern_ms[i] / 1e3) / 1e9, 2),
                                     "frac_of_pcie": round(wl.algorithmic_bytes(st) / 2 /
                                                           (kern_ms[i] / 1e3) / 1e9 /
                                                           PCIE_PEAK_GBPS, 4)}
                             for i, st in enumerate(wl.steps)}
    for i, d in enumerate(dsteps):
        if d["events"]:
            # completion time of each layer group, from the start of the last timed step
            e_start = events[i][-1][0]
            context["layer_group_done_ms"] = [round(e_start.elapsed_time(ev), 4)
                                              for ev in d["events"]]

    # Oracle comparison of sampled layers (and the CPU baseline timing), before
    # the hipMemcpy reference below overwrites the buffers.
    snap = None
    if replay and cpu_layers > 0:
        snap = {side: mem[side].clone() for side in wl.sides if side not in wl.host_sides}
        for d in dsteps:
            launch_step(kvx, wl, mem, d, errw)
        torch.cuda.synchronize()
        if int(errw.item()):
            log(f"device error bits {int(errw.item())}")
            return None
    picks, exact, cpu = [], None, None
    if cpu_layers > 0:
        st = wl.steps[0]
        S = wl.sides[st.src]
        L = st.slice[2] if st.slice is not None else S.L
        picks = _layer_picks(L, cpu_layers)
        if len(wl.steps) == 2:
            ok = _check_gather_scatter(wl, mem, snap, picks)
            exact, results = all(ok), []
            log(f"oracle on layers {picks}: bit-exact={exact}")
        else:
            results = []
            for l in picks:
                r = _check_transfer(wl, mem, snap, st, l)
                if time_cpu:
                    log(f"cpu oracle layer {l}: {r.oracle_seconds:.2f} s, bit-exact={r.equal}")
                results.append(r)
            exact = all(r.equal for r in results)
            log(f"oracle on layers {picks}: bit-exact={exact}")
        if not exact:
            log("GPU result differs from the oracle on a sampled layer")
            return None
        if time_cpu and results:
            secs = sum(r.oracle_seconds for r in results)
            moved = sum(r.moved_bytes for r in results)
            threads = _cpu_threads(args, len(results))
            wall = _threaded_seconds([r.rerun for r in results], threads)
            log(f"cpu oracle, {len(results)} layers on {threads} threads: {wall:.2f} s")
            cpu = {"value": round(moved / wall / 1e9, 4), "unit": "GB/s", "cores": threads,
                   "kind": "oracle",
                   "sample": f"layers {picks} of {L}: all {len(st.reqs)} requests, "
                             f"{moved / 1e9:.2f} GB moved; one layer per thread, {threads} "
                             f"threads, {wall:.2f} s wall",
                   "single_thread": {"value": round(moved / secs / 1e9, 4),
                                     "seconds": round(secs, 2)},
                   "sample_bit_exact": exact,
                   "cpu_model": _cpu_model(), "host_cpu_count": os.cpu_count()}
        results = None
    del snap

    if not args.no_memcpy and not host_leg and not replay:
        # hipMemcpyAsync D2D of the same byte count, as the achievable copy rate
        st = wl.steps[0]
        nb = min(dom_bytes // 2, mem[st.src].numel(), mem[st.dst].numel())
        ev = []
        cpy_a, cpy_b = mem[st.src][:nb], mem[st.dst][:nb]
        nrep = 5
        for r in range(nrep + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            cpy_b.copy_(cpy_a)
            e1.record(stream)
            if r:
                ev.append((e0, e1))
        torch.cuda.synchronize()
        ms = sum(a.elapsed_time(b) for a, b in ev) / nrep
        context["hip_memcpy_d2d_GBps_read_plus_write"] = round(2 * nb / (ms / 1e3) / 1e9, 1)

    if not args.no_memcpy and host_leg:
        # hipMemcpyAsync between the same pinned buffer and HBM, per direction
        hs = wl.host_sides[0]
        host = mem[hs]
        other = [n for n in wl.sides if n != hs][0]
        nb = min(host.numel(), mem[other].numel())
        for key, fn in (("hip_memcpy_d2h_GBps",
                         lambda: host[:nb].copy_(mem[other][:nb], non_blocking=True)),
                        ("hip_memcpy_h2d_GBps",
                         lambda: mem[other][:nb].copy_(host[:nb], non_blocking=True))):
            fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            context[key] = round(nb / (e0.elapsed_time(e1) / 1e3) / 1e9, 2)

    if any(d.get("plan") is not None and not d["st"].layer_group for d in dsteps) and len(dsteps) == 1:
        # after everything else: both launches fixed in turn on the same pools,
        # to show what the launch kept for the timed steps was chosen from
        d = dsteps[0]
        mode = kvx.kvx_launch_choice()
        rates = {}
        try:
            for key, fixed in (("sweep", kvx.CHOOSE_SWEEP), ("grid", kvx.CHOOSE_GRID)):
                kvx.kvx_set_launch_choice(fixed)
                launch_step(kvx, wl, mem, d, errw)
                if kvx.kvx_last_launch() != {"sweep": kvx.LAUNCH_SWEEP, "grid": kvx.LAUNCH_GRID}[key]:
                    continue                     # this step cannot take that launch
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for _ in range(4):
                    launch_step(kvx, wl, mem, d, errw)
                e1.record(stream)
                torch.cuda.synchronize()
                rates[key] = round(dom_bytes / (e0.elapsed_time(e1) / 4 / 1e3) / 1e9, 1)
        finally:
            kvx.kvx_set_launch_choice(mode)
        if int(errw.item()):
            log(f"device error bits {int(errw.item())}")
            return None
        context["both_launches_GBps"] = rates
        log(f"both launches, fixed, after the run: {rates}")

    n_tok = sum(st.n_tokens for st in wl.steps)
    config = {"workload": wl.title, "name": name,
              "ops": [("transfer_planned" if d.get("plan") is not None else st.op)
                      for st, d in zip(wl.steps, dsteps)],
              "requests": len(wl.steps[0].reqs),
              "tokens_per_step": n_tok, "bytes_per_step": step_bytes,
              "pools": {k: {"bytes": v.nbytes, **({"layout": v.layout, "page_tokens": v.T}
                                                  if hasattr(v, "layout") else {})}
                        for k, v in wl.sides.items()},
              "host_sides": list(wl.host_sides)}
    del mem, dsteps, events
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return {"value": round(value, 1), "ms_per_step": round(ms_per_step, 4), "config": config,
            "steps": steps, "warmup": warmup,
            "roofline": roofline, "cpu_baseline": cpu, "context": context,
            "sample_bit_exact": exact, "sample_layers": picks}


def _check_transfer(wl, mem, snap, st, l):
    """Layer l of a pool -> pool step against the oracle; ``snap`` holds the
    pools as they were before the checked step (a copy inside one pool)."""
    from oracle import layer_check
    S, D = wl.sides[st.src], wl.sides[st.dst]
    if st.slice is not None:
        return layer_check.check_transfer_slice_layer(mem[st.src], S, mem[st.dst], D, st, l,
                                                      wl.prefill_tag)
    before = layer_check.pool_layer(snap[st.dst], D, l) if snap is not None else None
    return layer_check.check_transfer_layer(mem[st.src], S, mem[st.dst], D, st, l,
                                            wl.prefill_tag, before)


def _check_gather_scatter(wl, mem, snap, picks) -> list:
    """Sampled layers of an offload (gather) and onload (scatter) into the
    pool it came from, from the snapshot taken before the checked step."""
    from oracle import layer_check
    g, s = wl.steps
    S, B = wl.sides[g.src], wl.sides[g.dst]
    out = []
    for l in picks:
        before = layer_check.pool_layer(snap[g.src], S, l)
        after = layer_check.pool_layer(mem[g.src], S, l)
        if g.slice is not None:
            ok = layer_check.gather_scatter_slice_layer(before, S, mem[g.dst], B, after, g, s, l)
        else:
            ok = layer_check.gather_scatter_layer(before, S, mem[g.dst], B, after, g, s, l)
        out.append(all(ok))
    return out


# Valu instruction cost of one payload byte in the page-digest loop of the
# hash kernel (gfx950 assembly): one quarter-rate 64-bit multiply-add, one
# quarter-rate 32-bit multiply and three full-rate operations, i.e. 11 SIMD
# cycles per byte per lane.  Peak: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
# / 11 cycles per byte.
HASH_CYCLES_PER_BYTE = 11
HASH_PEAK_GBPS = 256 * 4 * 16 * 2.4e9 / HASH_CYCLES_PER_BYTE / 1e9


def hash_bench(args) -> int:
    """Chained page hashes over token ids: GB/s of payload hashed."""
    import numpy as np
    import torch

    from paper_2606_31093_amd import kvx, workloads
    wl = workloads.page_hash()
    log(f"workload: {wl.title}")
    pay_np = workloads.hash_payload(wl)
    dev = torch.device("cuda", 0)
    pay = torch.from_numpy(pay_np.view(np.uint8).copy()).to(dev)
    reqs = kvx.device_hash_reqs(wl.rows, dev)
    out = torch.zeros(wl.out_len, dtype=torch.int64, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)

    def go():
        kvx.kvx_page_hashes(pay, wl.rec_bytes, wl.T, reqs, out, err)

    for _ in range(args.warmup):
        go()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        go()
        e1.record(stream)
        ev.append((e0, e1))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if int(err.item()):
        log(f"device error bits {int(err.item())}")
        return 1
    nbytes = wl.payload_bytes()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    kern_ms = sum(a.elapsed_time(b) for a, b in ev) / len(ev)
    achieved = nbytes / (kern_ms / 1e3) / 1e9
    cpu = None
    if args.cpu_layers > 0:
        from oracle import kvx_oracle
        want = np.zeros(wl.out_len, np.uint64)
        O = kvx_oracle.default()
        t2 = time.perf_counter()
        e = O.page_hashes(pay_np, wl.rec_bytes, wl.T, wl.rows, want)
        secs = time.perf_counter() - t2
        exact = e == 0 and np.array_equal(out.cpu().numpy().view(np.uint64), want)
        log(f"cpu oracle: {secs:.2f} s, bit-exact={exact}")
        if not exact:
            return 1
        # the same call over disjoint groups of requests, one group per thread
        threads = _cpu_threads(args, len(wl.rows))
        cuts = np.linspace(0, len(wl.rows), threads + 1).astype(int)
        want2 = np.zeros_like(want)
        jobs = [lambda a=a, b=b: O.page_hashes(pay_np, wl.rec_bytes, wl.T, wl.rows[a:b], want2)
                for a, b in zip(cuts[:-1], cuts[1:])]
        wall = _threaded_seconds(jobs, threads)
        exact = exact and np.array_equal(want2, want)
        log(f"cpu oracle on {threads} threads: {wall:.2f} s, same={exact}")
        if not exact:
            return 1
        cpu = {"value": round(nbytes / wall / 1e9, 4), "unit": "GB/s", "cores": threads,
               "kind": "oracle",
               "sample": f"the whole workload ({nbytes / 1e6:.1f} MB of token ids); requests split "
                         f"into {threads} groups, one per thread, {wall:.2f} s wall",
               "single_thread": {"value": round(nbytes / secs / 1e9, 4), "seconds": round(secs, 2)},
               "sample_bit_exact": exact, "cpu_model": _cpu_model(), "host_cpu_count": os.cpu_count()}
    tr = traffic_record("page_hash")
    out_line = {
        "metric": "chained page hash GB/s of payload, 1 MI355X", "value": round(nbytes / (ms_per_step / 1e3) / 1e9, 2),
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u64", "data": "synthetic (seeded int32 token ids)",
        "config": {"workload": wl.title, "name": wl.name, "requests": len(wl.rows),
                   "positions": wl.positions, "pages": wl.out_len, "payload_bytes": nbytes},
        "roofline": {"bound": "alu", "achieved": round(achieved, 2), "peak": round(HASH_PEAK_GBPS, 1),
                     "unit": "GB/s", "frac": round(achieved / HASH_PEAK_GBPS, 4),
                     "traffic": tr["traffic_bytes_per_launch"] if tr else None,
                     "kernel": "kvx page hashes (digest and chain roles in one launch)", "bytes_per_launch": nbytes,
                     "kernel_ms": round(kern_ms, 4)},
        "cpu_baseline": cpu,
        "context": {"kernel_sha": kernel_sha("page_hash"),
                    "kernel_ms_median": round(sorted(a.elapsed_time(b) for a, b in ev)[len(ev) // 2], 4),
                    "kernel_ms_min": round(min(a.elapsed_time(b) for a, b in ev), 4)},
    }
    print(json.dumps(out_line), flush=True)
    return 0


def _cpu_threads(args, jobs: int) -> int:
    """Threads for the multi-threaded oracle timing: the host CPUs this
    process may use (at most --cpu-threads), at most one per job."""
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    return max(1, min(avail, args.cpu_threads, jobs))


def _threaded_seconds(jobs, threads: int) -> float:
    """Wall time of running every job (oracle calls through ctypes, which
    release the GIL) on a pool of ``threads`` threads."""
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(threads) as ex:
        t0 = time.perf_counter()
        errs = list(ex.map(lambda f: f(), jobs))
        wall = time.perf_counter() - t0
    if any(errs):
        raise RuntimeError(f"oracle reported error bits {errs}")
    return wall


def _layer_picks(L: int, k: int) -> list:
    """k layers spread evenly over [0, L)."""
    return sorted({round(i * (L - 1) / max(1, k - 1)) for i in range(min(k, L))})


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    sys.exit(main())
