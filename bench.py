#!/usr/bin/env python3
"""Benchmark of the synthesis matcher on one MI355X.

One step = one full pccl_synthesize call on the 512-NPU All-to-All over the
2-level rail-switch topology (64 nodes x 8 NPUs, 400 GB/s intra-node, 8
switches at 50 GB/s, 128 KiB chunks): conditions, shortest paths, relays,
priority order, the matching event loop and the canonical schedule, with the
pre/postcondition bitmaps already resident in HBM.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config k] [--no-cpu-baseline]
    python bench.py --sweep   # chunk-count sweep: 64-NPU All-to-All, 1..64 chunks per pair
    python bench.py --switch-model   # the same 512-NPU All-to-All with finite switch buffers / no multicast
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
# Algorithmic bytes of the matching kernel, per launch: 16 B per scanned
# word position (one 8-byte word of the source's holds row and one of the
# destination's needs row) plus 96 B per committed transfer (the two words
# holding its bit, the needs-word read-modify-write, the holds-word set at
# arrival, link state, the send record and one atomic).
BYTES_PER_SCANNED_WORD = 16
BYTES_PER_MATCH = 96


COUNTERS = os.path.join(ROOT, "profiles", "k_match_switch2level_512_a2a_hbm_counters.md")
MATCH_SRC = os.path.join(ROOT, "paper_2606_07019_amd", "csrc", "pccl_match.hip")


def code_sha256(path: str) -> str:
    """sha256 of a source file's code: // comments, surrounding blanks and
    empty lines dropped, so that a comment edit keeps the hash."""
    import hashlib
    lines = []
    with open(path) as f:
        for line in f:
            code = line.split("//", 1)[0].strip()
            if code:
                lines.append(code)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()


def measured_traffic(config: int):
    """HBM bytes per k_match launch from the committed counter summary, or
    None when the kernel's code changed since the counters were taken."""
    if config != 4 or not os.path.exists(COUNTERS):
        return None
    want, traffic = None, None
    with open(COUNTERS) as f:
        for line in f:
            if "k_match code sha256:" in line:
                want = line.split(":", 1)[1].strip()
            elif "k_match traffic bytes per launch:" in line:
                traffic = int(line.split(":", 1)[1].strip())
    return traffic if want == code_sha256(MATCH_SRC) else None


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(wl, budget_s: float = 30.0):
    """The CPU oracle as it stands, single-threaded, on the same workload."""
    from oracle import oracle as O
    t0 = time.perf_counter()
    r = O.run_workload(wl)
    dt = time.perf_counter() - t0
    if r.status != 0:
        raise RuntimeError(r.message)
    cpu = platform.processor() or platform.machine()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": len(r.sends) / dt, "unit": "matches/s", "cores": 1, "kind": "oracle",
            "sample": f"the whole {wl.name} synthesis, one run ({dt:.1f} s, 1 thread, "
                      f"host {os.cpu_count()} threads of {cpu})",
            "seconds": dt, "n_sends": len(r.sends), "collective_time_ns": r.collective_time}


def end_to_end(wl, Synthesizer, torch, n_expected, runs: int = 5):
    """Synthesis from host bitmaps to a host schedule: pccl_set_collective
    (the library copies the host pre/postconditions), pccl_set_workspace,
    pccl_synthesize (upload, setup, matching, output) and pccl_get_schedule
    into host memory.  One warm-up, then the median of `runs`; HIP
    initialisation and module loading are outside (the context exists)."""
    import numpy as np
    from paper_2606_07019_amd import pccl as P
    syn = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed, device=0)
    c = wl.coll
    host = np.zeros((n_expected, 4), np.uint32)
    times = []
    try:
        for i in range(runs + 1):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            P.pccl_set_collective(syn.h, c.n_chunks, c.chunk_bytes, c.pre, c.post, c.group_masks,
                                  c.chunk_group, c.op)
            P.pccl_set_workspace(syn.h, syn.ws.data_ptr(), syn.ws.numel(), syn.max_sends, syn.stream.cuda_stream)
            got, _ = P.pccl_synthesize(syn.h)
            P.pccl_get_schedule(syn.h, host.ctypes.data, got)
            dt = time.perf_counter() - t0
            if got != n_expected:
                raise RuntimeError("end-to-end synthesis gave another schedule size")
            if i:
                times.append(dt)
    finally:
        syn.close()
    med = sorted(times)[len(times) // 2]
    return {"seconds_median": med, "matches_per_s": n_expected / med, "runs": runs,
            "schedule_bytes_to_host": int(host.nbytes), "bitmap_bytes_from_host": int(c.pre.nbytes + c.post.nbytes),
            "what": "host pre/post bitmaps -> set_collective + set_workspace + synthesize -> schedule in host memory"}


def sweep(args, W, Synthesizer, torch):
    """Synthesis wall time against the number of 128 KiB chunks per pair
    (the collective-size experiment of Sec. 6.1, Scalability) on both 64-NPU topologies."""
    steps = max(1, min(args.steps, 5))
    points = []
    for name, make in W.SWEEP_TOPOLOGIES.items():
        for k in W.SWEEP_K:
            wl = make(k)
            syn = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed, device=0)
            syn.synthesize()
            torch.cuda.synchronize()
            match_ms = []
            t0 = time.perf_counter()
            for _ in range(steps):
                syn.synthesize()
                match_ms.append(syn.profile()["match_ms"])
            torch.cuda.synchronize()
            step_s = (time.perf_counter() - t0) / steps
            st = syn.stats()
            pt = {"topology": name, "chunks_per_pair": k, "chunks": wl.coll.n_chunks,
                  "buffer_MiB_per_npu": 64 * k * wl.coll.chunk_bytes / 2 ** 20, "sends": syn.n_sends,
                  "collective_time_ns": syn.collective_time, "windows": st["windows"],
                  "synthesis_ms": step_s * 1e3, "match_ms": sum(match_ms) / len(match_ms),
                  "matches_per_s": syn.n_sends / step_s}
            syn.close()
            log(f"[sweep] {wl.name}: {pt['synthesis_ms']:.2f} ms, {pt['sends']} sends, {pt['windows']} windows")
            points.append(pt)
    last = points[-1]
    print(json.dumps({
        "metric": "synthesis wall time vs chunks per pair, 64-NPU All-to-All (Sec. 6.1 collective size)",
        "value": last["matches_per_s"], "unit": "matches/s", "n_gpus": 1, "steps": steps, "warmup": 1,
        "ms_per_step": last["synthesis_ms"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": "grid4x4x4_a2a_k64 (last point)", "points": len(points)},
        "points": points,
        "context": {"paper_hypercube_512MiB_a2a_synthesis_s": 109.8, "paper_hardware": "not stated"},
    }), flush=True)


SWITCH_POINTS = ((64, 8, 0, True), (64, 8, 64, True), (64, 8, 16, False), (16, 8, 4, True))


def switch_model(args, W, Synthesizer, torch):
    """Rail-cluster All-to-All with explicit switch nodes (Sec. 4.7): the
    switch-group matching kernel on the 512-NPU topology (unicast rail
    switches, with and without a buffer limit) and on 16 nodes x 8 NPUs,
    where the oracle is also timed."""
    steps = max(1, min(args.steps, 3))
    points = []
    for nn, pn, buf, uni in SWITCH_POINTS:
        wl = W.switch2level_model(nn, pn, buf, uni)
        syn = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed, device=0)
        syn.synthesize()
        torch.cuda.synchronize()
        match_ms = []
        t0 = time.perf_counter()
        for _ in range(steps):
            syn.synthesize()
            match_ms.append(syn.profile()["match_ms"])
        torch.cuda.synchronize()
        step_s = (time.perf_counter() - t0) / steps
        st, pr = syn.stats(), syn.profile()
        # the switch-group kernel, or the plain one when the device found
        # that the no-multicast rule cannot act (and no buffer limit binds)
        kern = "k_match_sw" if syn.matcher() == "switch" else "k_match"
        kms = sum(match_ms) / len(match_ms)
        alg = BYTES_PER_SCANNED_WORD * pr["scan_words"] + BYTES_PER_MATCH * syn.n_sends
        pt = {"workload": wl.name, "npus": nn * pn, "buffer_chunks": buf, "unicast": bool(uni),
              "sends": syn.n_sends, "collective_time_ns": syn.collective_time, "windows": st["windows"],
              "synthesis_ms": step_s * 1e3, "match_ms": kms, "matches_per_s": syn.n_sends / step_s,
              "matcher": kern,
              "roofline": {"bound": "hbm", "kernel": kern, "achieved": round(alg / (kms * 1e-3) / 1e9, 3),
                           "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                           "frac": round(alg / (kms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 6),
                           "alg_bytes_per_launch": alg, "scan_words": pr["scan_words"]}}
        syn.close()
        if nn * pn <= 128 and not args.no_cpu_baseline:
            log(f"[switch] timing the CPU oracle on {wl.name} ...")
            pt["cpu_baseline"] = cpu_baseline(wl)
        log(f"[switch] {wl.name}: {pt['synthesis_ms']:.1f} ms, {pt['sends']} sends, collective {syn.collective_time} ns")
        points.append(pt)
    head = points[1]
    print(json.dumps({
        "metric": "synthesis wall time + link-chunk matches/s, 512-NPU All-to-All with a switch model (Sec. 4.7)",
        "value": head["matches_per_s"], "unit": "matches/s", "n_gpus": 1, "steps": steps, "warmup": 1,
        "ms_per_step": head["synthesis_ms"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": head["workload"], "points": len(points)},
        "points": points,
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--switch-model", action="store_true",
                    help="512-NPU All-to-All with finite switch buffers / no multicast (Sec. 4.7)")
    ap.add_argument("--sweep", action="store_true",
                    help="time the chunk-count sweep (8x8 mesh and 4x4x4 grid All-to-All, k = 1..64)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (to scale HBM counters)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration << 18  # int32 elements
        src = torch.ones(n, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4}), flush=True)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: the synthesis matcher runs on one GPU; there is no multi-GPU path "
              "(--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_07019_amd import workloads as W
    from paper_2606_07019_amd.pccl import Synthesizer

    if not torch.cuda.is_available():
        raise RuntimeError("no GPU visible")
    if args.sweep:
        sweep(args, W, Synthesizer, torch)
        return
    if args.switch_model:
        switch_model(args, W, Synthesizer, torch)
        return
    wl = W.CONFIGS[args.config]()
    log(f"[bench] workload {wl.name}: {wl.topo.n_devices} devices, {wl.topo.n_links} links, "
        f"{wl.coll.n_chunks} chunks")
    syn = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed, device=0)
    for i in range(args.warmup):
        syn.synthesize()
        log(f"[bench] warmup {i}: {syn.n_sends} sends, collective time {syn.collective_time} ns")
    torch.cuda.synchronize()
    match_ms, setup_ms, output_ms, each_s = [], [], [], []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        ts = time.perf_counter()
        syn.synthesize()  # returns once the schedule is complete on the device
        each_s.append(time.perf_counter() - ts)
        p = syn.profile()
        match_ms.append(p["match_ms"])
        setup_ms.append(p["setup_ms"])
        output_ms.append(p["output_ms"])
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    step_s = dt / max(args.steps, 1)
    prof = syn.profile()
    st = syn.stats()
    n = syn.n_sends
    busy, bins, bin_ns = syn.link_usage(20)
    ct = max(syn.collective_time, 1)
    frac = busy / ct
    schedule_metrics = {
        "link_busy_fraction": {"mean": round(float(frac.mean()), 4), "max": round(float(frac.max()), 4),
                               "min": round(float(frac.min()), 4), "links_unused": int((busy == 0).sum())},
        "utilization_over_time": {"bins": 20, "bin_ns": bin_ns,
                                  "fraction_of_links_busy": [round(float(b) / (len(busy) * bin_ns), 4) for b in bins]},
    }
    log(f"[bench] {args.steps} steps in {dt:.3f} s; stages (ms, last step) {prof}")

    avg_match_s = sum(match_ms) / len(match_ms) / 1e3
    alg_bytes = BYTES_PER_SCANNED_WORD * prof["scan_words"] + BYTES_PER_MATCH * n
    achieved = alg_bytes / avg_match_s / 1e9
    traffic = measured_traffic(args.config)
    roofline = {"bound": "hbm", "achieved": round(achieved, 3), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBPS, 6), "traffic": traffic,
                "kernel": "k_match", "kernel_ms": round(avg_match_s * 1e3, 4),
                "alg_bytes_per_launch": alg_bytes, "scan_words": prof["scan_words"], "matches": n,
                # the counter bytes (FETCH_SIZE + WRITE_SIZE, calibrated) over the same
                # kernel time: HBM GB/s as the hardware counts it, MALL hits included
                "traffic_GBps": None if traffic is None else round(traffic / avg_match_s / 1e9, 3)}

    out = {
        "metric": "synthesis wall time (s) + link-chunk matches/s, 512-NPU All-to-All; HBM GB/s",
        "value": n / step_s,
        "unit": "matches/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": wl.name, "npus": wl.topo.n_npus, "switches": wl.topo.n_switches,
                   "links": wl.topo.n_links, "chunks": wl.coll.n_chunks, "chunk_bytes": wl.coll.chunk_bytes,
                   "sends": n, "collective_time_ns": syn.collective_time, "windows": st["windows"],
                   "events": st["events"], "rounds": st["rounds"], "clashes": st["clashes"]},
        "synthesis_wall_s": step_s,
        "synthesis_wall_s_median": sorted(each_s)[len(each_s) // 2],
        "stage_ms": {"setup": sum(setup_ms) / len(setup_ms), "match": sum(match_ms) / len(match_ms),
                     "output": sum(output_ms) / len(output_ms)},
        "roofline": roofline,
        "schedule_metrics": schedule_metrics,
        "context": {"paper_512npu_a2a_synthesis_s": 700.8, "paper_hardware": "not stated",
                    "paper_topology": "2D Mesh / 3D Hypercube family (not this topology)"},
    }
    syn.close()
    out["end_to_end"] = end_to_end(wl, Synthesizer, torch, n)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on the same workload ...")
        cb = cpu_baseline(wl)
        if cb["n_sends"] != n or cb["collective_time_ns"] != out["config"]["collective_time_ns"]:
            raise RuntimeError("GPU and oracle schedules differ in size or collective time")
        out["cpu_baseline"] = {k: cb[k] for k in ("value", "unit", "cores", "kind", "sample")}
        out["cpu_baseline"]["seconds"] = cb["seconds"]
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
