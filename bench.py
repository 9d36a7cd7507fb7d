"""Throughput of the CoSpec verify-and-arbitrate step on one MI355X.

One step = one cospec_verify_block call (all of: vocabulary reductions of the
target and draft rows, merge/Delta/compaction, MFMA head on the mismatch rows,
first-stop scan and emission, features written) over one batch that is already
resident in HBM.  Default workload: the large chain batch B=256, K=7,
V=151936 bf16 logits, head 5120->512->1, lambda 0.5.

Prints one JSON line: rows/s (B*(K+1) verified rows per second), the roofline
of the dominant kernel (the vocabulary reduction, timed with HIP events on the
stream it runs on), and the CPU oracle timed on a bounded sample of the same
workload on this host, with a parity re-check of the timed outputs.
`--sample` times the temperature-1 variant (candidates sampled by inversion of
seeded uniforms) instead of the greedy one; `--sps` times the standard
speculative-sampling baseline on the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "verified rows/sec (B×(k+1)) and achieved HBM GB/s vs peak, V=151936 bf16"
HBM_PEAK_GBPS = 8000.0


def measured_traffic(kernel_source: str):
    """HBM bytes per launch of the reduction kernel from the committed rocprofv3 counter
    summary, or None when that kernel's source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "k_vocab_reduce_large_chain_traffic.json")
    try:
        rec = json.load(open(path))
        sha = hashlib.sha256(open(os.path.join(ROOT, kernel_source), "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("source") != kernel_source or rec.get("source_sha256") != sha:
        return None
    return rec.get("traffic_bytes_per_launch")


def gpu_state(tag, torch=None):
    """Current shader and memory clocks (MHz) and average power (W) of the benchmarked GPU,
    read from its sysfs files (no other program is started: this process may already
    have initialised the GPU); {} when the device cannot be identified or read."""
    import glob
    out = {}
    try:
        dev = None
        if torch is not None:
            prop = torch.cuda.get_device_properties(0)
            dev = "/sys/bus/pci/devices/%04x:%02x:%02x.0" % (prop.pci_domain_id, prop.pci_bus_id,
                                                            prop.pci_device_id)
        else:
            cards = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
            if len(cards) == 1:                  # only when the device is unambiguous
                dev = os.path.dirname(cards[0])
        if dev is None or not os.path.isdir(dev):
            return out
        for clk in ("sclk", "mclk"):
            for ln in open(os.path.join(dev, "pp_dpm_" + clk)):
                if ln.rstrip().endswith("*"):    # e.g. "1: 2100Mhz *"
                    out[f"{clk}_mhz_{tag}"] = float(ln.split(":")[1].split("Mhz")[0])
        for pw in glob.glob(os.path.join(dev, "hwmon", "hwmon*", "power1_average")):
            out[f"power_w_{tag}"] = int(open(pw).read()) / 1e6
    except Exception:
        pass
    return out


def host_info():
    """ROCm release, the GPU state before this process touches the GPU (idle clocks, not
    the clocks under load) and the host's CPU model; fields that cannot be read are left
    out."""
    info = {}
    try:
        info["rocm"] = open("/opt/rocm/.info/version").read().strip()
    except OSError:
        pass
    info.update(gpu_state("idle_at_start"))
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                info["cpu_model"] = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return info


def device_info(torch):
    prop = torch.cuda.get_device_properties(0)
    return {"name": prop.name, "arch": getattr(prop, "gcnArchName", None),
            "compute_units": prop.multi_processor_count, "hip": torch.version.hip}


def step_percentiles(torch, np, step, steps, flush=None):
    """Per-step HIP-event times (ms) of `steps` calls: p10, median, p90.  With `flush`,
    that callable runs before every step, outside the step's events."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        if flush is not None:
            flush()
        a.record()
        step()
        b.record()
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    return {"p10": float(np.percentile(ms, 10)), "p50": float(np.median(ms)), "p90": float(np.percentile(ms, 90))}


def oracle_threads():
    """Threads for the parallel oracle run: the CPUs this process may use, at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=4, help="named workload 1..5 (default 4)")
    ap.add_argument("--splits", type=int, default=0, help="workgroups per row (0 = automatic)")
    ap.add_argument("--overlap", action="store_true",
                    help="run the head on a second stream, overlapping the draft-row reduction "
                         "(slower on the large chain batch: the reduction fills every CU)")
    ap.add_argument("--sample", action="store_true",
                    help="temperature-1 target candidates (inversion of seeded uniforms) instead "
                         "of the greedy argmax")
    ap.add_argument("--sps", action="store_true",
                    help="time the standard speculative-sampling baseline (chain workloads) instead "
                         "of the CoSpec step")
    ap.add_argument("--attention", action="store_true",
                    help="time the arbitrator's hybrid attention over the region queries "
                         "(B=64 sequences, 2048 context tokens, K=7, 32 query / 8 key-value heads, "
                         "D=128) instead of the verify step")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of one step captured in a HIP graph (no per-launch host "
                         "work: what a serving loop that captures its step sees)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU budget of the oracle baseline sample (0 disables it)")
    return ap.parse_args()


def bench_attention(args):
    """The arbitrator's hybrid attention for one round's region queries: each sequence's
    2K+3 new positions attend to its cached context and the region (bf16, fp32
    accumulation).  Roofline: the key/value bytes every launch must read."""
    hinfo = host_info()
    import numpy as np
    import torch

    import paper_2605_24793_amd as cs
    from paper_2605_24793_amd.workloads import bf16_bits
    dev = torch.device("cuda:0")
    B, ctx_len, K, Hq, Hkv, D = 64, 2048, 7, 32, 8, 128
    nq = 2 * K + 3
    l = ctx_len + nq
    L = (l + 15) // 16 * 16
    g = torch.Generator().manual_seed(11)
    q = (torch.randn(B, nq, Hq, D, generator=g)).to(torch.bfloat16)
    k = (torch.randn(B, L, Hkv, D, generator=g)).to(torch.bfloat16)
    v = (torch.randn(B, L, Hkv, D, generator=g)).to(torch.bfloat16)
    ctx = torch.full((B,), ctx_len, dtype=torch.int32)
    qd, kd, vd, cd = q.to(dev), k.to(dev), v.to(dev), ctx.to(dev)
    scale = 1.0 / np.sqrt(D)
    for _ in range(args.warmup):
        out = cs.hybrid_attention(qd, kd, vd, cd, cd, K, scale)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(args.steps):
        out = cs.hybrid_attention(qd, kd, vd, cd, cd, K, scale)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    kv_bytes = B * Hkv * l * D * 2 * 2                   # keys and values each sequence's group reads
    flops = B * Hq * nq * l * D * 2 * 2                  # q k^T and p v
    achieved = kv_bytes / (ms * 1e-3) / 1e9
    cpu = None
    if args.cpu_seconds > 0:
        import oracle
        got = out.float().cpu().numpy()
        c0 = time.perf_counter()
        n = 0
        while n < B and time.perf_counter() - c0 < args.cpu_seconds:
            ref = oracle.hybrid_attention(bf16_bits(q[n:n + 1]), bf16_bits(k[n:n + 1]), bf16_bits(v[n:n + 1]),
                                          [ctx_len], [ctx_len], K, scale)
            tol = 6e-3 * float(v[n].float().abs().max())
            assert np.abs(got[n:n + 1] - ref).max() <= tol, "attention parity re-check failed"
            n += 1
        spent = time.perf_counter() - c0
        cpu = {"value": n * nq / spent, "unit": "query positions/s", "cores": 1, "kind": "oracle",
               "sample": f"first {n} of {B} sequences, fp64 oracle, single thread, {spent:.1f} s"}
    line = {"metric": "hybrid-attention region queries/sec", "value": B * nq / (ms * 1e-3),
            "unit": "query positions/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"arbitrator region attention B={B} context={ctx_len} K={K} Hq={Hq} "
                                   f"Hkv={Hkv} D={D}"},
            "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                         "kernel": "k_hybrid_attention", "kernel_ms": ms,
                         "algorithmic_bytes_per_launch": kv_bytes},
            "tflops": flops / (ms * 1e-3) / 1e12, "device": dict(device_info(torch), **hinfo),
            "cpu_baseline": cpu}
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py measures one GPU (sequences shard across GPUs with no exchange); --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.attention:
        bench_attention(args)
        return
    hinfo = host_info()
    import numpy as np
    import torch

    import paper_2605_24793_amd as cs
    from paper_2605_24793_amd import workloads
    from paper_2605_24793_amd.workloads import bf16_bits

    dev = torch.device("cuda:0")
    print(f"[bench] generating workload {args.config}", file=sys.stderr, flush=True)
    wl = workloads.make_config(args.config)
    tree = isinstance(wl, workloads.TreeBatch)
    lam = wl.lambdas[len(wl.lambdas) // 2]
    head = workloads.Head(wl.head.w1.to(dev), None if wl.head.b1 is None else wl.head.b1.to(dev),
                          wl.head.w2.to(dev), wl.head.b2)
    tgt, drf, hid = wl.target.to(dev), wl.draft.to(dev), wl.hidden.to(dev)
    u_host = None
    if args.sample:
        R = wl.N if tree else wl.K + 1
        u_host = torch.rand((wl.B, R), generator=torch.Generator().manual_seed(2024))
    u_dev = None if u_host is None else u_host.to(dev)
    sps_u = None
    if args.sps:
        if tree:
            print(json.dumps({"error": "--sps runs on chain workloads"}))
            sys.exit(2)
        sps_u = torch.rand((wl.B, wl.K + 1), generator=torch.Generator().manual_seed(2025))
    if tree:
        par, tok = wl.parent.to(dev), wl.node_tokens.to(dev)
        p = cs.prepare_tree(tgt, drf, par, tok, hid, head, lam, features=True, splits=args.splits,
                            overlap=args.overlap, sample_u=u_dev)
        rows = wl.B * wl.N
        internal = np.zeros((wl.B, wl.N), bool)
        pn = wl.parent.numpy()
        for b in range(wl.B):
            for n in range(1, wl.N):
                internal[b, pn[b, n]] = True
        reduced_rows = rows + int(internal.sum())
    else:
        tok = wl.draft_tokens.to(dev)
        if args.sps:
            p = cs.prepare_sps(tgt, drf, tok, sps_u.to(dev), features=True, splits=args.splits)
        else:
            p = cs.prepare_block(tgt, drf, tok, hid, head, lam, features=True, splits=args.splits,
                                 overlap=args.overlap, sample_u=u_dev)
        rows = wl.B * (wl.K + 1)
        reduced_rows = wl.B * (2 * wl.K + 1)
    elem = tgt.element_size()
    logit_bytes = reduced_rows * wl.V * elem       # algorithmic bytes of the two reduction launches

    torch.cuda.synchronize()

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        p.launch()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    step = p.launch
    if args.graph:
        if args.overlap:
            print(json.dumps({"error": "--graph does not capture the aux stream"}))
            sys.exit(2)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            p.launch()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            p.launch()
        step = graph.replay
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()

    # timed region 1: the whole step, back to back, nothing else on the stream
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record()
    for _ in range(args.steps):
        step()
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t0.elapsed_time(t1)

    # timed region 2: the same steps with HIP events recorded by the library around
    # the two vocabulary-reduction launches (target rows, draft rows), on the stream
    # they run on
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for e in (x for row in ev for x in row):
        e.record()                                 # materialise the HIP events
    torch.cuda.synchronize()
    print(f"[bench] timing the reduction kernel over {args.steps} steps", file=sys.stderr, flush=True)
    for i in range(args.steps):
        p.launch(timing=ev[i])
    torch.cuda.synchronize()
    # per-step distribution: back to back, and with the 256 MB last-level cache (MALL)
    # flushed before every step by writing a 512 MB buffer outside the step's events
    print(f"[bench] per-step times, warm and with the cache flushed, {args.steps} steps each",
          file=sys.stderr, flush=True)
    warm_pct = step_percentiles(torch, np, step, args.steps)
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cold_pct = step_percentiles(torch, np, step, args.steps, flush=lambda: scratch.fill_(0x5A))
    hinfo.update(gpu_state("right_after_timing", torch))
    del scratch
    launches = 2 if args.overlap else 1             # the draft rows get their own launch
    k_ms = [e[0].elapsed_time(e[1]) + e[2].elapsed_time(e[3]) for e in ev]
    k_raw = float(np.mean(k_ms)) / launches         # event interval per launch
    # Without the overlap stream the library records the second pair back to back with
    # no launch between them, so that pair measures what an event interval adds on its
    # own (barrier packets, timestamps); it is taken off the kernel's interval.
    ev_overhead = 0.0 if args.overlap else float(np.mean([e[2].elapsed_time(e[3]) for e in ev]))
    k_avg = k_raw - ev_overhead                     # average duration of one launch
    ms_per_step = total_ms / args.steps
    value = rows / (ms_per_step * 1e-3)
    launch_bytes = logit_bytes / launches
    achieved = launch_bytes / (k_avg * 1e-3) / 1e9
    res = p.result()
    out = {k: v.cpu() for k, v in res.items()}

    # CPU oracle on a bounded sample (first sequences of the same workload), also a
    # parity re-check of the timed outputs on those sequences
    cpu = cpu_par = None
    if args.cpu_seconds > 0:
        import oracle
        from oracle import parity

        def conv(t):
            return bf16_bits(t) if t.dtype == torch.bfloat16 else t.contiguous().numpy()
        head_np = (conv(wl.head.w1), None if wl.head.b1 is None else conv(wl.head.b1),
                   conv(wl.head.w2), wl.head.b2)
        done, spent, chunk = 0, 0.0, 8
        checked = 0
        while done < wl.B and spent < args.cpu_seconds:
            seqs = list(range(done, min(wl.B, done + chunk)))
            sub = wl.take(seqs)
            us = None if u_host is None else u_host[seqs].double().numpy()
            c0 = time.perf_counter()
            if args.sps:
                ref = oracle.sps_block(conv(sub.target), conv(sub.draft), sub.draft_tokens.numpy(),
                                       sps_u[seqs].double().numpy())
            elif tree:
                ref = oracle.verify_tree(conv(sub.target), conv(sub.draft), sub.parent.numpy(),
                                         sub.node_tokens.numpy(), conv(sub.hidden), head_np, lam,
                                         sample_u=us)
            else:
                ref = oracle.verify_block(conv(sub.target), conv(sub.draft), sub.draft_tokens.numpy(),
                                          conv(sub.hidden), head_np, lam, sample_u=us)
            spent += time.perf_counter() - c0
            gsub = {k: v[seqs] for k, v in out.items()}
            if args.sps:
                parity.check_sps(gsub, ref, conv(sub.target), conv(sub.draft), sps_u[seqs].double().numpy())
                checked += len(seqs)
                done += len(seqs)
                continue
            if us is not None:
                # candidates at a cumulative boundary may differ; the check validates
                # them and the rest of the step is compared on the GPU's candidates
                cand = parity.check_candidates(gsub["tgt_candidate"], conv(sub.target), us)
                if not np.array_equal(cand, ref["tgt_cand"]):
                    fn = oracle.verify_tree if tree else oracle.verify_block
                    ref = (fn(conv(sub.target), conv(sub.draft), sub.parent.numpy(), sub.node_tokens.numpy(),
                              conv(sub.hidden), head_np, lam, sample_u=us, cand_override=cand) if tree else
                           fn(conv(sub.target), conv(sub.draft), sub.draft_tokens.numpy(), conv(sub.hidden),
                              head_np, lam, sample_u=us, cand_override=cand))
            (parity.check_tree if tree else parity.check_block)(gsub, ref)
            checked += len(seqs)
            done += len(seqs)
        cpu_rows = done * (wl.N if tree else wl.K + 1)
        cpu = {"value": cpu_rows / spent, "unit": "rows/s", "cores": 1, "kind": "oracle",
               "sample": f"first {done} of {wl.B} sequences ({cpu_rows} verified rows) of the same "
                         f"workload, fp64 oracle, single thread, {spent:.1f} s",
               "parity_checked_sequences": checked}

        # the same sequences again, one chunk per task on a thread pool: the oracle's C
        # loops release the interpreter lock, so its row reductions run in parallel
        from concurrent.futures import ThreadPoolExecutor
        nth = oracle_threads()

        def run_chunk(seqs):
            sub = wl.take(seqs)
            us = None if u_host is None else u_host[seqs].double().numpy()
            if args.sps:
                oracle.sps_block(conv(sub.target), conv(sub.draft), sub.draft_tokens.numpy(),
                                 sps_u[seqs].double().numpy())
            elif tree:
                oracle.verify_tree(conv(sub.target), conv(sub.draft), sub.parent.numpy(), sub.node_tokens.numpy(),
                                   conv(sub.hidden), head_np, lam, sample_u=us)
            else:
                oracle.verify_block(conv(sub.target), conv(sub.draft), sub.draft_tokens.numpy(),
                                    conv(sub.hidden), head_np, lam, sample_u=us)
        chunks = [list(range(s, min(done, s + chunk))) for s in range(0, done, chunk)]
        c0 = time.perf_counter()
        with ThreadPoolExecutor(max_workers=nth) as pool:
            list(pool.map(run_chunk, chunks))
        par_spent = time.perf_counter() - c0
        cpu_par = {"value": cpu_rows / par_spent, "unit": "rows/s", "cores": nth, "kind": "oracle",
                   "sample": f"the same {done} sequences, {len(chunks)} chunks of up to {chunk} on "
                             f"{nth} threads, {par_spent:.1f} s"}

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if elem == 2 else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, ("N" if tree else "K"): (wl.N if tree else wl.K),
                   "V": wl.V, "d": wl.head.d, "h": wl.head.h, "lambda": lam,
                   "splits": args.splits or "auto", "head_overlap": args.overlap,
                   "hip_graph": args.graph,
                   "temperature": 1 if args.sample or args.sps else 0,
                   "rule": "speculative sampling" if args.sps else "cospec",
                   "rows_per_step": rows,
                   "reduced_rows_per_step": reduced_rows},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": (measured_traffic("paper_2605_24793_amd/csrc/reduce.hip")
                                 if args.config == 4 and not args.splits and not args.sample
                                 and not args.sps else None),
                     "kernel": "k_vocab_reduce", "kernel_ms": k_avg,
                     "event_interval_ms": k_raw, "empty_event_interval_ms": ev_overhead,
                     "launches_per_step": launches, "algorithmic_bytes_per_launch": launch_bytes},
        "step_hbm_gbps": logit_bytes / (ms_per_step * 1e-3) / 1e9,
        "wall_s": wall,
        "mean_accept_len": float(out["accept_len"].float().mean()),
        "step_ms_warm": warm_pct,
        "step_ms_cache_flushed": cold_pct,
        "device": dict(device_info(torch), **hinfo),
        "cpu_baseline": cpu,
        "cpu_baseline_threads": cpu_par,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
