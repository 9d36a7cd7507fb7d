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
# Chain batches of at most this many decision slots run the head's first layer in the
# reduction's launch (kEverySlotMax in paper_2605_24793_amd/csrc/cospec_api.hip).
EVERY_SLOT_MAX = 256
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
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the records of the peaked serving chain, the tree batch and the small "
                         "and tiny chains that the default run appends")
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


def _conv(torch, bf16_bits, t):
    return bf16_bits(t) if t.dtype == torch.bfloat16 else t.contiguous().numpy()


class Step:
    """One workload resident on the GPU with its pre-marshalled verify call."""

    def __init__(self, cs, workloads, torch, np, wl, dev, lam, args, u_host=None, sps_u=None):
        self.wl, self.lam, self.torch = wl, lam, torch
        self.tree = isinstance(wl, workloads.TreeBatch)
        head = workloads.Head(wl.head.w1.to(dev), None if wl.head.b1 is None else wl.head.b1.to(dev),
                              wl.head.w2.to(dev), wl.head.b2)
        tgt, drf, hid = wl.target.to(dev), wl.draft.to(dev), wl.hidden.to(dev)
        u_dev = None if u_host is None else u_host.to(dev)
        if self.tree:
            par, tok = wl.parent.to(dev), wl.node_tokens.to(dev)
            self.p = cs.prepare_tree(tgt, drf, par, tok, hid, head, lam, features=True, splits=args.splits,
                                     sample_u=u_dev)
            self.rows = wl.B * wl.N
            internal = np.zeros((wl.B, wl.N), bool)
            pn = wl.parent.numpy()
            for b in range(wl.B):
                for n in range(1, wl.N):
                    internal[b, pn[b, n]] = True
            self.reduced_rows = self.rows + int(internal.sum())
        else:
            tok = wl.draft_tokens.to(dev)
            if sps_u is not None:
                self.p = cs.prepare_sps(tgt, drf, tok, sps_u.to(dev), features=True, splits=args.splits)
            else:
                self.p = cs.prepare_block(tgt, drf, tok, hid, head, lam, features=True, splits=args.splits,
                                          sample_u=u_dev)
            self.rows = wl.B * (wl.K + 1)
            self.reduced_rows = wl.B * (2 * wl.K + 1)
        self.elem = tgt.element_size()
        self.kernel = "k_vocab_reduce"
        if not self.tree and sps_u is None and 0 < wl.B * wl.K <= EVERY_SLOT_MAX:
            # the library runs the head's first layer over every decision slot in the
            # reduction's launch: the timed launch holds both
            self.kernel = "k_vocab_reduce_head (reduction + the head's first layer on every slot)"
        self.logit_bytes = self.reduced_rows * wl.V * self.elem   # algorithmic bytes of the reductions
        self.step = self.p.launch

    def warmup(self, n):
        for _ in range(n):
            self.step()
        self.torch.cuda.synchronize()

    def timed(self, n):
        """n back-to-back steps between two events on the stream: ms per step, wall s."""
        torch = self.torch
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        t0.record()
        for _ in range(n):
            self.step()
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / n, time.perf_counter() - wall0

    def reduction_events(self, np, n, flush=None):
        """HIP events recorded by the library around the vocabulary-reduction launches (on
        the stream they run on) over n steps; with `flush`, that callable runs before every
        step.  Returns (average launch ms, raw event interval ms, empty-pair ms)."""
        torch = self.torch
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(n)]
        for e in (x for row in ev for x in row):
            e.record()                                 # materialise the HIP events
        torch.cuda.synchronize()
        for i in range(n):
            if flush is not None:
                flush()
            self.p.launch(timing=ev[i])
        torch.cuda.synchronize()
        k_raw = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
        # The library records the second pair back to back with no launch between them, so
        # that pair measures what an event interval adds on its own (barrier packets,
        # timestamps); it is taken off the kernel's interval.
        overhead = float(np.mean([e[2].elapsed_time(e[3]) for e in ev]))
        return k_raw - overhead, k_raw, overhead


def oracle_parity(torch, np, bf16_bits, wl, out, lam, tree, u_host=None, sps_u=None, nthreads=1,
                  budget_s=None):
    """Oracle over the workload's sequences, chunks of eight on `nthreads` threads (the
    oracle's C loops release the interpreter lock), each chunk's timed GPU outputs
    checked against it.  With budget_s the chunks run in order on one thread until the
    budget is spent.  Returns (sequences checked, CPU seconds of oracle work)."""
    import oracle
    from oracle import parity

    def conv(t):
        return _conv(torch, bf16_bits, t)
    head_np = (conv(wl.head.w1), None if wl.head.b1 is None else conv(wl.head.b1), conv(wl.head.w2),
               wl.head.b2)

    def run(seqs):
        sub = wl.take(seqs)
        us = None if u_host is None else u_host[seqs].double().numpy()
        c0 = time.perf_counter()
        if sps_u is not None:
            ref = oracle.sps_block(conv(sub.target), conv(sub.draft), sub.draft_tokens.numpy(),
                                   sps_u[seqs].double().numpy())
        elif tree:
            ref = oracle.verify_tree(conv(sub.target), conv(sub.draft), sub.parent.numpy(),
                                     sub.node_tokens.numpy(), conv(sub.hidden), head_np, lam, sample_u=us)
        else:
            ref = oracle.verify_block(conv(sub.target), conv(sub.draft), sub.draft_tokens.numpy(),
                                      conv(sub.hidden), head_np, lam, sample_u=us)
        spent = time.perf_counter() - c0
        gsub = {k: v[seqs] for k, v in out.items()}
        if sps_u is not None:
            parity.check_sps(gsub, ref, conv(sub.target), conv(sub.draft), sps_u[seqs].double().numpy())
            return len(seqs), spent
        if us is not None:
            # candidates at a cumulative boundary may differ; the check validates them and
            # the rest of the step is compared on the GPU's candidates
            cand = parity.check_candidates(gsub["tgt_candidate"], conv(sub.target), us)
            if not np.array_equal(cand, ref["tgt_cand"]):
                ref = (oracle.verify_tree(conv(sub.target), conv(sub.draft), sub.parent.numpy(),
                                          sub.node_tokens.numpy(), conv(sub.hidden), head_np, lam,
                                          sample_u=us, cand_override=cand) if tree else
                       oracle.verify_block(conv(sub.target), conv(sub.draft), sub.draft_tokens.numpy(),
                                           conv(sub.hidden), head_np, lam, sample_u=us, cand_override=cand))
        (parity.check_tree if tree else parity.check_block)(gsub, ref)
        return len(seqs), spent

    chunk = 8
    chunks = [list(range(s, min(wl.B, s + chunk))) for s in range(0, wl.B, chunk)]
    if budget_s is not None:
        done, spent = 0, 0.0
        for c in chunks:
            if spent >= budget_s:
                break
            n, t = run(c)
            done, spent = done + n, spent + t
        return done, spent
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=nthreads) as pool:
        parts = list(pool.map(run, chunks))
    return sum(n for n, _ in parts), sum(t for _, t in parts)


def extra_workload(cs, workloads, torch, np, bf16_bits, cfg, dev, args, nthreads):
    """Compact record of another named workload, same binary and launch sequence: step
    time back to back, the reduction kernel's HBM fraction by HIP events with the
    last-level cache flushed before every step, and a parity re-check of every sequence
    (every threshold the workload names) against the oracle."""
    wl = workloads.make_config(cfg)
    tree = isinstance(wl, workloads.TreeBatch)
    lam = wl.lambdas[len(wl.lambdas) // 2]
    st = Step(cs, workloads, torch, np, wl, dev, lam, args)
    st.warmup(args.warmup)
    ms, _ = st.timed(args.steps)
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    k_avg, k_raw, _ = st.reduction_events(np, args.steps, flush=lambda: scratch.fill_(0x5A))
    cold = step_percentiles(torch, np, st.step, args.steps, flush=lambda: scratch.fill_(0x5A))
    del scratch
    checked = 0
    for lam_i in wl.lambdas:
        p = st if lam_i == lam else Step(cs, workloads, torch, np, wl, dev, lam_i, args)
        if p is not st:
            p.warmup(1)
        out = {k: v.cpu() for k, v in p.p.result().items()}
        n, _ = oracle_parity(torch, np, bf16_bits, wl, out, lam_i, tree, nthreads=nthreads)
        checked += n
    launch_bytes = st.logit_bytes
    gbps = launch_bytes / (k_avg * 1e-3) / 1e9
    return {"workload": wl.name, "lambda": lam, "ms_per_step": ms, "rows_per_s": st.rows / (ms * 1e-3),
            "step_ms_cache_flushed": cold,
            "reduction_cache_flushed": {"kernel": st.kernel, "kernel_ms": k_avg,
                                        "event_interval_ms": k_raw, "achieved_gbps": gbps,
                                        "frac": gbps / HBM_PEAK_GBPS,
                                        "algorithmic_bytes_per_launch": launch_bytes},
            "parity_checked_sequences": checked, "lambdas_checked": list(wl.lambdas)}


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
    u_host = None
    if args.sample:
        R = wl.N if tree else wl.K + 1
        u_host = torch.rand((wl.B, R), generator=torch.Generator().manual_seed(2024))
    sps_u = None
    if args.sps:
        if tree:
            print(json.dumps({"error": "--sps runs on chain workloads"}))
            sys.exit(2)
        sps_u = torch.rand((wl.B, wl.K + 1), generator=torch.Generator().manual_seed(2025))
    st = Step(cs, workloads, torch, np, wl, dev, lam, args, u_host=u_host, sps_u=sps_u)
    torch.cuda.synchronize()

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    st.warmup(args.warmup)
    if args.graph:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            st.p.launch()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            st.p.launch()
        st.step = graph.replay
        st.warmup(args.warmup)

    # Measurement loops that report on the same step run first, each exactly `steps`
    # steps: the reduction kernel's own launches by HIP events, then the per-step time
    # distribution back to back and with the 256 MB last-level cache (MALL) flushed before
    # every step by writing a 512 MB buffer outside the step's events.  The headline loop
    # then times `steps` steps of a GPU that has been running this step.
    print(f"[bench] timing the reduction kernel over {args.steps} steps", file=sys.stderr, flush=True)
    k_avg, k_raw, ev_overhead = st.reduction_events(np, args.steps)
    print(f"[bench] per-step times, warm and with the cache flushed, {args.steps} steps each",
          file=sys.stderr, flush=True)
    warm_pct = step_percentiles(torch, np, st.step, args.steps)
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cold_pct = step_percentiles(torch, np, st.step, args.steps, flush=lambda: scratch.fill_(0x5A))
    del scratch
    st.warmup(args.warmup)
    hinfo.update(gpu_state("before_headline", torch))

    # the headline: `steps` whole steps back to back, nothing else on the stream
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    ms_per_step, wall = st.timed(args.steps)
    hinfo.update(gpu_state("right_after_timing", torch))
    value = st.rows / (ms_per_step * 1e-3)
    launch_bytes = st.logit_bytes
    achieved = launch_bytes / (k_avg * 1e-3) / 1e9
    out = {k: v.cpu() for k, v in st.p.result().items()}

    nth = oracle_threads()
    extras = {}
    default_mode = (args.config == 4 and not (args.sample or args.sps or args.graph or args.splits)
                    and not args.no_extras)
    if default_mode:
        for key, cfg in (("peaked_chain", 3), ("tree", 5), ("small_chain", 2), ("tiny_chain", 1)):
            print(f"[bench] workload {cfg}: timing, flushed reduction events, parity of every sequence",
                  file=sys.stderr, flush=True)
            extras[key] = extra_workload(cs, workloads, torch, np, bf16_bits, cfg, dev, args, nth)

    # CPU oracle on a bounded sample (first sequences of the same workload), also a parity
    # re-check of the timed outputs on those sequences; then the same sequences on a pool
    cpu = cpu_par = None
    if args.cpu_seconds > 0:
        print("[bench] oracle baseline", file=sys.stderr, flush=True)
        done, spent = oracle_parity(torch, np, bf16_bits, wl, out, lam, tree, u_host, sps_u,
                                    budget_s=args.cpu_seconds)
        cpu_rows = done * (wl.N if tree else wl.K + 1)
        host_cpus = os.cpu_count()
        cpu = {"value": cpu_rows / spent, "unit": "rows/s", "cores": 1, "kind": "oracle",
               "sample": f"first {done} of {wl.B} sequences ({cpu_rows} verified rows) of the same "
                         f"workload, fp64 oracle, single thread, {spent:.1f} s",
               "parity_checked_sequences": done, "host_cpus": host_cpus}
        sub = wl.take(list(range(done)))
        sout = {k: v[:done] for k, v in out.items()}
        c0 = time.perf_counter()
        oracle_parity(torch, np, bf16_bits, sub, sout, lam, tree, None if u_host is None else u_host[:done],
                      None if sps_u is None else sps_u[:done], nthreads=nth)
        par_spent = time.perf_counter() - c0
        cpu_par = {"value": cpu_rows / par_spent, "unit": "rows/s", "cores": nth, "kind": "oracle",
                   "sample": f"the same {done} sequences, chunks of up to 8 on {nth} threads "
                             f"(of {host_cpus} host CPUs), {par_spent:.1f} s",
                   "host_cpus": host_cpus}

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
        "dtype": "bf16" if st.elem == 2 else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, ("N" if tree else "K"): (wl.N if tree else wl.K),
                   "V": wl.V, "d": wl.head.d, "h": wl.head.h, "lambda": lam,
                   "splits": args.splits or "auto",
                   "hip_graph": args.graph,
                   "temperature": 1 if args.sample or args.sps else 0,
                   "rule": "speculative sampling" if args.sps else "cospec",
                   "rows_per_step": st.rows,
                   "reduced_rows_per_step": st.reduced_rows,
                   "loops_before_headline": "warmup, reduction-kernel events, warm and flushed "
                                            f"per-step times ({args.steps} steps each), warmup"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": (measured_traffic("paper_2605_24793_amd/csrc/reduce.hip")
                                 if args.config == 4 and not args.splits and not args.sample
                                 and not args.sps else None),
                     "kernel": st.kernel, "kernel_ms": k_avg,
                     "event_interval_ms": k_raw, "empty_event_interval_ms": ev_overhead,
                     "launches_per_step": 1, "algorithmic_bytes_per_launch": launch_bytes},
        "step_hbm_gbps": st.logit_bytes / (ms_per_step * 1e-3) / 1e9,
        "wall_s": wall,
        "mean_accept_len": float(out["accept_len"].float().mean()),
        "step_ms_warm": warm_pct,
        "step_ms_cache_flushed": cold_pct,
        "device": dict(device_info(torch), **hinfo),
        "cpu_baseline": cpu,
        "cpu_baseline_threads": cpu_par,
    }
    line.update({f"workload_{k}": v for k, v in extras.items()})
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
