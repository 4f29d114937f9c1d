"""Benchmark: one step = append the turn's new K/V + extend attention over
the reused prefix, on one GPU, through the C-ABI library.

Default workload: the long ReAct turn -- one sequence, 131072 reused prefix
tokens, 2048 new tokens (an appended tool output), Hq=96, Hkv=8, D=128, bf16,
pages scattered at random over a 2^20-page pool.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

Without --steps the timed region holds 20 steps, or as many as fill about
0.2 s when 20 steps would take under 0.1 s (short workloads, where one
launch's latency would otherwise weigh on the wall-clock step time); short
workloads also warm up for at least 0.1 s, so the clock has settled.

``--gpus N`` with N > 1 exits: the benchmark measures one GPU only.
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

METRIC = "extend-attention TFLOP/s and new tokens/s at 128K reused prefix; % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X published dense bf16 MFMA peak
PEAK_HBM_GBPS = 8000.0      # MI355X published HBM3E bandwidth
PEAK_HOST_LINK_GBPS = 64.0  # PCIe 5.0 x16, one direction


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def load_traffic(workload: str, kind: str = "extend"):
    """HBM bytes per launch of the extend, decode or append kernel from
    committed rocprofv3 counters, if they were taken on the current kernel
    sources; else None."""
    from paper_2609_39819_amd.profiling import APPEND_SOURCES, DECODE_SOURCES, EXTEND_SOURCES, read_traffic, \
        source_sha
    name = workload if workload.startswith(kind) else f"{kind}_{workload}"
    t = read_traffic(os.path.join(ROOT, "profiles", f"{name}_traffic.md"))
    srcs = {"extend": EXTEND_SOURCES, "decode": DECODE_SOURCES, "append": APPEND_SOURCES}[kind]
    if t is None or t[0] != source_sha(srcs):
        return None
    return t[1]


def cpu_baseline(w, target_s: float):
    """Time the fp64 oracle on a bounded sample of the same workload."""
    from oracle import oracle_append, oracle_extend
    from paper_2609_39819_amd.workloads import algorithmic_flops
    try:
        import threadpoolctl
        threads = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    kp, vp = oracle_append(w.k_pool_c, w.v_pool_c, w.compact_table, w.prefix_len, w.suffix_len, w.k_new, w.v_new)

    def run(n):
        rows, flops = [], 0
        for b in range(w.num_seqs):
            S = int(w.suffix_len[b])
            r = np.unique(np.linspace(0, S - 1, max(1, min(S, n))).astype(np.int64))
            rows.append(r)
            P = int(w.prefix_len[b])
            flops += 4 * w.head_dim * w.num_q_heads * int((P + r + 1).sum())
        t0 = time.perf_counter()
        oracle_extend(w.q, kp, vp, w.compact_table, w.prefix_len, w.suffix_len, w.num_kv_heads, w.scale, rows=rows)
        return time.perf_counter() - t0, flops, sum(len(r) for r in rows)

    n = 2
    dt, fl, nt = run(n)
    while dt < target_s / 3 and n < int(w.suffix_len.max()):
        n = min(int(w.suffix_len.max()), int(n * max(2.0, min(16.0, target_s / max(dt, 1e-3)))))
        dt, fl, nt = run(n)
    tflops = fl / dt / 1e12
    toks = nt / dt
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:
        pass
    return {
        "value": tflops, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
        "cpu_model": model, "nproc": os.cpu_count(),
        "sample": f"{nt} of {w.total_tokens} new tokens (evenly spaced), all {w.num_q_heads} query heads, "
                  f"full reused prefix; fp64 numpy oracle; {dt:.1f} s",
        "seconds": dt, "new_tokens_per_s": toks,
    }


def sample_power(step, ms_per_step: float):
    """Socket power and GFX clocks while steps run back to back: about 4 s of
    steps are queued, amd-smi is read 1.5 s in, then the queue drains."""
    import re
    import subprocess
    import torch
    n = max(10, int(4000.0 / max(ms_per_step, 1e-3)))
    for _ in range(n):
        step()
    time.sleep(1.5)
    try:
        r = subprocess.run(["amd-smi", "metric", "-p", "-c"], capture_output=True, text=True, timeout=60)
        text = r.stdout
    except (OSError, subprocess.TimeoutExpired) as e:
        text = ""
        log(f"amd-smi unavailable: {e}")
    torch.cuda.synchronize()
    power = re.search(r"SOCKET_POWER:\s*([0-9.]+)\s*W", text)
    clocks = [int(x) for x in re.findall(r"GFX_\d+:\s*\n\s*CLK:\s*([0-9]+)\s*MHz", text)]
    return {"socket_power_w": float(power.group(1)) if power else None,
            "gfx_clock_mhz": clocks or None, "source": "amd-smi metric -p -c"}


def bench_copy(args, w, d, dev):
    """Offload every used page of the workload to pinned host memory and
    reload it into the same pages; HIP events around each launch."""
    import torch
    from paper_2609_39819_amd import kvt
    ids = torch.from_numpy(np.ascontiguousarray(w.phys_ids, dtype=np.int32)).to(dev)
    n = int(ids.numel())
    host = torch.empty((n, 2) + tuple(d["k_pool"].shape[1:]), dtype=d["k_pool"].dtype, pin_memory=True)
    nbytes = host.numel() * host.element_size()
    stream = torch.cuda.current_stream(dev)
    for _ in range(args.warmup):
        kvt.copy_blocks(d["k_pool"], d["v_pool"], ids, host, to_host=True)
        kvt.copy_blocks(d["k_pool"], d["v_pool"], ids, host, to_host=False)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    for e in evs:
        e[0].record(stream)
        kvt.copy_blocks(d["k_pool"], d["v_pool"], ids, host, to_host=True)
        e[1].record(stream)
        kvt.copy_blocks(d["k_pool"], d["v_pool"], ids, host, to_host=False)
        e[2].record(stream)
    torch.cuda.synchronize()
    off = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    rel = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    log(f"{n} pages, {nbytes / 1e6:.1f} MB: offload {off:.3f} ms ({nbytes / off / 1e6:.1f} GB/s), "
        f"reload {rel:.3f} ms ({nbytes / rel / 1e6:.1f} GB/s)")
    step_ms = off + rel
    return {
        "metric": "HBM <-> pinned-host page moves (offload + reload of every page of the workload)",
        "value": 2 * nbytes / (step_ms * 1e-3) / 1e9, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": step_ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u8", "data": "synthetic",
        "config": {"workload": f"{w.name} pages", "pages": n, "bytes_each_way": nbytes},
        "offload_ms": off, "reload_ms": rel,
        "offload_gbps": nbytes / (off * 1e-3) / 1e9, "reload_gbps": nbytes / (rel * 1e-3) / 1e9,
        "roofline": {"bound": "host link", "achieved": 2 * nbytes / (step_ms * 1e-3) / 1e9,
                     "peak": PEAK_HOST_LINK_GBPS, "unit": "GB/s",
                     "frac": 2 * nbytes / (step_ms * 1e-3) / 1e9 / PEAK_HOST_LINK_GBPS, "traffic": None},
        "gpu": torch.cuda.get_device_name(dev),
    }


def bench_manager(args):
    """Replay the seeded agent trace through the library's block manager
    (host code, no GPU): natively through kvt_mgr_replay (the value), and
    call by call through the binding; the oracle model replays a bounded
    prefix of the same trace, and both must report the same there."""
    from paper_2609_39819_amd import kvt
    from paper_2609_39819_amd.workloads import agent_events
    events = list(agent_events())
    encoded = kvt.Manager.encode(events)
    pages = args.manager_pages

    def one_by_one(m, evs, deadline=None):
        reps, totals = [], {}
        t0 = time.perf_counter()
        for n, (op, a) in enumerate(evs):
            r = getattr(m, op)(*a)
            if r is not None:
                reps.append(r)
                for k, v in r.items():
                    totals[k] = totals.get(k, 0) + v
            if deadline is not None and (n & 63) == 0 and time.perf_counter() - t0 > deadline:
                return time.perf_counter() - t0, n + 1, reps, totals
        return time.perf_counter() - t0, len(evs), reps, totals

    for _ in range(args.warmup):
        kvt.Manager(pages).replay(encoded)
    times = []
    for _ in range(max(1, args.steps)):
        m = kvt.Manager(pages)
        t0 = time.perf_counter()
        ok, tot = m.replay(encoded)
        times.append(time.perf_counter() - t0)
    if ok != len(events):
        raise SystemExit(f"trace replay: {len(events) - ok} calls failed")
    dt = float(np.median(times))
    py_dt, _, _, py_tot = one_by_one(kvt.Manager(pages), events)
    if py_tot != tot:
        raise SystemExit("trace replay and call-by-call reports differ")
    hit = tot["hit_tokens"] / max(1, tot["hit_tokens"] + tot["miss_tokens"])
    log(f"{len(events)} calls: native {dt * 1e3:.1f} ms ({len(events) / dt:.0f} calls/s), through the binding "
        f"{py_dt * 1e3:.1f} ms ({len(events) / py_dt:.0f} calls/s); hit ratio {hit:.3f}, {tot}")
    res = {
        "metric": "host block-manager calls per second over a seeded ReAct agent trace",
        "value": len(events) / dt, "unit": "calls/s", "n_gpus": 1, "steps": len(times), "warmup": args.warmup,
        "ms_per_step": dt * 1e3, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int64", "data": "synthetic",
        "config": {"workload": "agent_events(seed=9): 256 agents, 32 at once, 8-40 calls each", "calls": len(events),
                   "pool_pages": pages, "page_size": 16},
        "binding_calls_per_s": len(events) / py_dt,
        "hit_ratio_tokens": hit, **tot,
        "roofline": None,
        "note": "host code; value = kvt_mgr_replay over the encoded trace, binding_calls_per_s = one ctypes call "
                "per event",
    }
    if not args.no_cpu_baseline:
        from oracle import OracleManager
        log("replaying a prefix of the trace through the oracle model")
        odt, on, oreps, _ = one_by_one(OracleManager(pages), events, deadline=args.cpu_seconds)
        _, _, lreps, _ = one_by_one(kvt.Manager(pages), events[:on])
        res["cpu_baseline"] = {"value": on / odt, "unit": "calls/s", "cores": 1, "kind": "oracle",
                               "sample": f"first {on} of {len(events)} calls of the same trace, {odt:.1f} s",
                               "reports_match": oreps == lreps}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default: 20, more for steps under 5 ms; see above)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="react_128k")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--cascade", action="store_true",
                    help="for a workload whose sequences share a prefix (forked_agents), run the cascade extend "
                         "(shared keys once for the whole batch, then the private keys, then an LSE merge)")
    ap.add_argument("--cascade-mode", choices=("auto", "shared", "plain"), default="auto",
                    help="with --cascade: let the library's estimate choose between the shared pass and the plain "
                         "extend plan (auto, the default), or force one")
    ap.add_argument("--copy", action="store_true",
                    help="instead of attention, time moving every page of the workload to pinned host memory "
                         "and back (kvt_copy_blocks)")
    ap.add_argument("--cold-mib", type=int, default=0,
                    help="write a scratch buffer of this size before every step, outside the timed "
                         "region, so the step starts with cold caches; times then come from HIP events")
    ap.add_argument("--sample-power", action="store_true",
                    help="after the timed steps, keep the extend kernel running for a few seconds and "
                         "record socket power and GFX clocks from amd-smi (reported, not timed)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="run one plain fp32 copy kernel (torch.neg) of this size first, as the "
                         "reference a rocprofv3 FETCH_SIZE/WRITE_SIZE pass is scaled by")
    ap.add_argument("--manager", action="store_true",
                    help="instead of attention, time the host block manager (lifecycle states, Algorithm 1 "
                         "admission, MRU inside Suspended) over a seeded agent event trace; no GPU work")
    ap.add_argument("--manager-pages", type=int, default=32768,
                    help="page pool of the --manager run (the trace needs about 50K pages to fit)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)
    if args.manager or args.copy:
        args.steps = 20 if args.steps is None else args.steps
    if args.manager:
        bench_manager(args)
        return

    import torch
    from paper_2609_39819_amd import kvt
    from paper_2609_39819_amd.workloads import algorithmic_flops, kv_bytes, make_config, stage_on_device

    kvt.lib()   # fail loudly if the library is missing
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    log(f"generating {args.workload}")
    t0 = time.time()
    w = make_config(args.workload)
    log(f"generated in {time.time() - t0:.1f}s; staging on {torch.cuda.get_device_name(dev)}")
    calib_src = None
    if args.calibrate_copy_mib:
        # written before the pool staging below, so no cache holds it when it is copied
        calib_src = torch.ones(args.calibrate_copy_mib * 262144, dtype=torch.float32, device=dev)
    d = stage_on_device(w, dev)
    torch.cuda.synchronize()

    if args.copy:
        print(json.dumps(bench_copy(args, w, d, dev)), flush=True)
        return
    Hq, D = w.num_q_heads, w.head_dim
    flops = algorithmic_flops(w.prefix_len, w.suffix_len, Hq, D)
    elem = 2 if w.dtype == "bf16" else 4
    append_bytes = 2 * 2 * w.total_tokens * w.num_kv_heads * D * elem   # K+V, read + write
    # a decoding step (one new token per sequence) runs the decode kernel,
    # which is bound by streaming K/V from HBM
    decode = w.name.startswith("decode")
    attn_bytes = kv_bytes(w.prefix_len, w.suffix_len, w.num_kv_heads, D, elem) + 2 * w.total_tokens * Hq * D * elem
    out = torch.empty_like(d["q"])
    shared = 0
    if args.cascade:
        from paper_2609_39819_amd.workloads import config_shapes
        shared = int(config_shapes(w.name).get("shared_prefix", 0))
        if not shared:
            print(f"--cascade needs a workload with a shared prefix; {w.name} has none", file=sys.stderr)
            sys.exit(2)
    if decode:
        need = kvt.decode_workspace_bytes(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, Hq)
    elif shared:
        cmode = {"auto": kvt.CASCADE_AUTO, "shared": kvt.CASCADE_SHARED_PASS, "plain": kvt.CASCADE_PLAIN}[
            args.cascade_mode]
        need = kvt.cascade_workspace_bytes(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len,
                                           shared, Hq, mode=cmode)
        cascade_plan = ("shared pass" if args.cascade_mode == "shared" else "plain" if args.cascade_mode == "plain"
                        else "shared pass" if kvt.cascade_uses_shared_pass(d["k_pool"], d["v_pool"], d["block_table"],
                                                                           w.prefix_len, w.suffix_len, shared, Hq)
                        else "plain")
        log(f"cascade mode {args.cascade_mode}: {cascade_plan}")
    else:
        need = kvt.extend_workspace_bytes(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len, Hq)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev) if need else None
    stream = torch.cuda.current_stream(dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        kvt.append_kv(d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len, d["k_new"], d["v_new"])
        if ev is not None:
            ev[1].record(stream)
        if decode:
            kvt.decode_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.scale,
                                 out=out, workspace=ws, use_workspace=need > 0)
        elif shared:
            kvt.cascade_extend_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len,
                                         w.suffix_len, shared, w.scale, out=out, workspace=ws,
                                         use_workspace=need > 0, mode=cmode)
        else:
            kvt.extend_attention(d["q"], d["k_pool"], d["v_pool"], d["block_table"], w.prefix_len, w.suffix_len,
                                 w.scale, out=out, workspace=ws, use_workspace=need > 0)
        if ev is not None:
            ev[2].record(stream)

    if calib_src is not None:
        dst = torch.empty_like(calib_src)
        torch.cuda.synchronize()
        torch.neg(calib_src, out=dst)
        torch.cuda.synchronize()
        del calib_src, dst
    scratch = torch.empty(args.cold_mib * 262144, dtype=torch.float32, device=dev) if args.cold_mib else None
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.steps is None:
        # size the timed region from a short untimed probe of back-to-back steps
        t0 = time.perf_counter()
        for _ in range(5):
            step()
        torch.cuda.synchronize()
        est = (time.perf_counter() - t0) / 5
        args.steps = 20 if 20 * est >= 0.1 else int(min(20000, np.ceil(0.2 / est)))
        if 20 * est < 0.1:
            extra = int(np.ceil(0.1 / est))
            for _ in range(extra):
                step()
            args.warmup += 5 + extra
            torch.cuda.synchronize()
        else:
            args.warmup += 5
        log(f"about {est * 1e3:.3f} ms per step: {args.steps} timed steps after {args.warmup} warm-up steps")
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        if scratch is not None:
            scratch.fill_(float(i))
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    app_ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    ext_ms = np.array([e[1].elapsed_time(e[2]) for e in evs])
    # with cold caches the scratch writes sit between the steps, so the step
    # time is the sum of the kernels' event times instead of the wall clock
    ms_per_step = float((app_ms + ext_ms).mean()) if scratch is not None else wall * 1e3 / args.steps
    value = flops / (ms_per_step * 1e-3) / 1e12
    ext_avg = float(ext_ms.mean())
    achieved = flops / (ext_avg * 1e-3) / 1e12
    log(f"extend avg {ext_avg:.3f} ms (min {ext_ms.min():.3f}), append avg {app_ms.mean():.4f} ms, "
        f"step {ms_per_step:.3f} ms, extend {achieved:.1f} TFLOP/s = {100 * achieved / PEAK_BF16_TFLOPS:.1f}% of peak")

    res = {
        "metric": METRIC,
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "num_seqs": w.num_seqs,
            "prefix_len": int(w.prefix_len.max()) if w.num_seqs == 1 else [int(x) for x in w.prefix_len],
            "suffix_len": int(w.suffix_len.max()) if w.num_seqs == 1 else [int(x) for x in w.suffix_len],
            "num_q_heads": Hq, "num_kv_heads": w.num_kv_heads, "head_dim": D,
            "page_size": 16, "pool_pages": w.num_blocks, "key_splits": "auto",
        },
        "new_tokens_per_s": w.total_tokens / (ms_per_step * 1e-3),
        "pct_bf16_peak": 100.0 * value / PEAK_BF16_TFLOPS,
        "attention_kernel": "decode" if decode else (f"cascade extend ({args.cascade_mode}: {cascade_plan})"
                                                     if shared else "extend"),
        "extend_ms": ext_avg,
        "extend_ms_median": float(np.median(ext_ms)),
        "extend_ms_min": float(ext_ms.min()),
        "caches": f"cold ({args.cold_mib} MiB scratch write before each step)" if args.cold_mib else "warm",
        "extend_tflops": achieved,
        "append_ms": float(app_ms.mean()),
        "append_gbps": append_bytes / (float(app_ms.mean()) * 1e-3) / 1e9,
        "roofline": {
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            "traffic": load_traffic(w.name),
        } if not decode else {
            "bound": "hbm",
            "achieved": attn_bytes / (ext_avg * 1e-3) / 1e9,
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": attn_bytes / (ext_avg * 1e-3) / 1e9 / PEAK_HBM_GBPS,
            "traffic": load_traffic(w.name, "decode"),
        },
        # the scatter of the new tokens' K/V (HBM-bound; launch-bound below ~100 MB)
        "append_roofline": {
            "bound": "hbm",
            "achieved": append_bytes / (float(app_ms.mean()) * 1e-3) / 1e9,
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": append_bytes / (float(app_ms.mean()) * 1e-3) / 1e9 / PEAK_HBM_GBPS,
            "traffic": load_traffic(w.name, "append"),
        },
        "gpu": torch.cuda.get_device_name(dev),
        "gcn_arch": torch.cuda.get_device_properties(dev).gcnArchName,
        "hip": torch.version.hip,
    }
    if args.sample_power:
        res["power_sample"] = sample_power(lambda: step(), ms_per_step)
    del d, out, ws, scratch
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on a sample")
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
