"""Benchmark: paged prefix-reuse prefill attention + KV prefetch on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

One step is one serving pass over the workload's agents in dispatch order:
for each agent, its invocations run cs_prefill_paged_attn on the main stream
while cs_kv_prefetch brings the next agent's CPU-tier anchor blocks into the
pool on a side stream; the main stream waits on the prefetch's event before
the next agent's attention.  Inputs are resident in HBM (and the prefetch
sources in pinned host memory) before timing starts.

Prints one JSON line.  ``value`` is the attention throughput of the whole step
(algorithmic FLOP of all attention launches / wall time of the step);
``roofline`` rates the attention kernel from its own average launch duration
(HIP events on the main stream, inside the timed region); ``prefetch`` rates
the copy from its launch durations on the side stream; ``cpu_baseline`` times
the float64 oracle on a bounded sample of the same workload on the host.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "prefill-attn TFLOP/s (% bf16 MFMA peak) + KV prefetch GB/s, 1 MI355X"
PEAK_BF16_TFLOPS = 2500.0        # MI355X dense bf16 MFMA
PEAK_SCLK_MHZ = 2400.0           # the clock that peak is quoted at
PEAK_HBM_GBS = 8000.0
PEAK_PCIE5_X16_GBS = 63.0        # PCIe 5.0 x16, one direction, 128b/130b
KERNEL_SOURCES = ("paper_2608_14624_amd/csrc/prefill_paged_attn.hip",
                  "paper_2608_14624_amd/csrc/kv_prefetch.hip")

DESCRIPTIONS = {
    "llama70b_prefetch": "16 invocations over 4 agents, 64 query / 8 KV heads, head_dim 128, "
                         "cached prefix 4096 + suffix 512 tokens, 16-token blocks in a "
                         "16384-block pool; 64 of each agent's 256 anchor blocks are "
                         "prefetched from pinned host memory on a side stream while the "
                         "previous agent's attention runs",
    "tiny": "1 request, 8 query / 2 KV heads, head_dim 64, cached prefix 256 + suffix 64 "
            "tokens, prefix blocks at a seeded permutation of a 64-block pool (a correctness "
            "shape: one launch of 4 work-groups)",
    "llama8b": "1 request, 32 query / 8 KV heads, head_dim 128, cached prefix 2048 + suffix "
               "1024 tokens, 16384-block pool",
    "agent_batch": "32 invocations over 4 agents, anchors U[1536,3072], suffixes U[256,2048], "
                   "32 query / 8 KV heads, head_dim 128, 16384-block pool",
    "long_mixed": "128 invocations over 8 agents, anchors U[4096,8192], lognormal suffixes "
                  "(median 512) in [128,4096], 77 hits / 51 full-prompt misses, 32 query / 8 "
                  "KV heads, head_dim 128, pool at 90% occupancy",
    "decode_batch": "128 sequences over 8 agents, anchors U[4096,8192] + lognormal history "
                    "(median 512) in [128,4096], one token decoded per sequence, 32 query / 8 "
                    "KV heads, head_dim 128",
    "decode_private": "128 sequences with the decode_batch length mix and nothing shared (each "
                      "its own anchor U[4096,8192] + history), one token decoded per sequence, "
                      "32 query / 8 KV heads, head_dim 128",
    "llama70b_prefetch_tp8": "one GPU's shard of llama70b_prefetch split 8 ways by KV head: "
                             "the same 16 invocations and prefetches with 8 query / 1 KV head",
    "agent_batch_tp8": "one GPU's shard of agent_batch split 8 ways by KV head: the same 32 "
                       "invocations with 4 query / 1 KV head",
}


def source_hash(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel, workload, kernel_hash):
    """HBM bytes per launch of `kernel` on `workload` from a committed
    rocprofv3 --pmc summary (FETCH_SIZE + WRITE_SIZE, each scaled by a plain
    copy's reading); None unless the kernel source is the one measured."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    entry = data.get(f"{kernel}|{workload}")
    if not entry or entry.get("kernel_sha") != kernel_hash:
        return None
    return entry.get("bytes_per_launch")


def attention_kernel_name(batch, max_q_len, num_q_heads, num_kv_heads, head_dim, parts=1):
    """Which attention kernel a launch runs (the library's own launch rule,
    asked through cs_prefill_paged_attn_launch_shape; ``parts`` > 1: the
    workspace call's key parts and their merge)."""
    from paper_2608_14624_amd import ops
    if parts > 1:
        return (f"prefill_paged_attn_ppd_split_kernel<{head_dim}, true> + "
                f"prefill_split_merge_kernel<{head_dim}>")
    kernel, _, tail = ops.prefill_launch_shape(batch, max_q_len, num_q_heads, num_kv_heads)
    if kernel == ops.ATTN_PING_PONG:
        return f"prefill_paged_attn_ppd_kernel<{head_dim}, {'true' if tail else 'false'}>"
    return f"prefill_paged_attn_ppd_split_kernel<{head_dim}, false>"


def key_parts(sb, wl, workspace):
    """Key parts the attention call of sub-batch ``sb`` takes (1: none)."""
    from paper_2608_14624_amd import ops
    if workspace is None or sb.hi <= sb.lo:
        return 1
    need = ops.prefill_workspace_bytes(sb.hi - sb.lo, sb.q1 - sb.q0, sb.max_q_len, sb.max_kv_len,
                                       wl.num_q_heads, wl.num_kv_heads, wl.head_dim)
    return max(1, need // ((sb.q1 - sb.q0) * wl.num_q_heads * (wl.head_dim + 2) * 4))


def _oracle_invocations(wl, kp, vp, rs):
    """Run the float64 oracle on invocations ``rs`` one by one; returns
    (seconds, algorithmic FLOP)."""
    import numpy as np
    import oracle
    cu = wl.cu_q_lens.astype(np.int64)
    flops, t0 = 0, time.perf_counter()
    for r in rs:
        s = int(cu[r + 1] - cu[r])
        p = int(wl.prefix_lens[r])
        oracle.prefill_paged_attn(wl.q[cu[r]:cu[r + 1]], kp, vp, wl.block_tables[r:r + 1],
                                  wl.prefix_lens[r:r + 1], np.array([0, s]), wl.num_q_heads,
                                  wl.num_kv_heads, wl.scale)
        flops += 4 * wl.head_dim * wl.num_q_heads * (s * p + s * (s + 1) // 2)
    return time.perf_counter() - t0, flops


def cpu_baseline(wl, sample_s=2.0, repeats=3):
    """The float64 oracle timed on the host, in TFLOP/s of algorithmic work.

    Main figure: whole invocations of the same workload, taken in order until
    the first pass holds about ``sample_s`` seconds of work (at least one),
    run ``repeats`` times with all BLAS threads; the median is reported.
    Beside it, single-thread figures for the tiny and Llama-3-8B-shape
    configurations (median of 3 and one run)."""
    import statistics
    import oracle
    from paper_2608_14624_amd.workload import make_config
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threadpool_limits = None
        threads = os.cpu_count()
    kp, vp = wl.k_pool, wl.v_pool
    if wl.prefetch_dst is not None:
        kp, vp = oracle.kv_prefetch(wl.host_k, wl.host_v, wl.prefetch_dst, kp, vp)
    rs, first = [], 0.0
    for r in range(wl.batch):
        dt, _ = _oracle_invocations(wl, kp, vp, [r])
        rs.append(r)
        first += dt
        if first >= sample_s:
            break
    runs = [_oracle_invocations(wl, kp, vp, rs) for _ in range(repeats)]
    flops = runs[0][1]
    secs = [t for t, _ in runs]
    med = statistics.median(secs)
    single = {}
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            for name, reps in (("tiny", 3), ("llama8b", 1)):
                w = make_config(name)
                allr = list(range(w.batch))
                ts = [_oracle_invocations(w, w.k_pool, w.v_pool, allr) for _ in range(reps)]
                t1 = statistics.median([t for t, _ in ts])
                single[name] = {"value": round(ts[0][1] / t1 / 1e12, 6), "unit": "TFLOP/s",
                                "seconds": round(t1, 3), "runs": reps}
    return {"value": round(flops / med / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle", "host": host_description(),
            "runs_s": [round(t, 3) for t in secs],
            "sample": f"invocations {rs[0]}..{rs[-1]} ({len(rs)} of {wl.batch}) of {wl.name}, "
                      f"full float64 oracle, median of {repeats} runs "
                      f"({med:.2f} s each, {int(threads)} BLAS threads)",
            "single_thread": single}


def _time_launches(fn, steps, warmup, stream):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    t0 = time.perf_counter()
    for e0, e1 in evs:
        e0.record(stream)
        fn()
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = [e0.elapsed_time(e1) for e0, e1 in evs]
    return wall, sum(ms) / steps, ms


def hbm_reference(dev, stream, nbytes=2 << 30):
    """What plain library kernels reach on this GPU's HBM, measured beside an
    HBM-bound component: torch's device-to-device copy (reads and writes
    nbytes each) and its float32 sum (reads nbytes).  A practical ceiling for
    comparison; the roofline fraction stays against the published peak."""
    import torch
    src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).uniform_()
    dst = torch.empty_like(src)
    acc = torch.empty((), dtype=torch.float32, device=dev)
    _, ms_copy, _ = _time_launches(lambda: dst.copy_(src), 10, 2, stream)
    _, ms_sum, _ = _time_launches(lambda: torch.sum(src, 0, out=acc), 10, 2, stream)
    del src, dst
    torch.cuda.empty_cache()
    return {"bytes": nbytes,
            "copy_gbs": round(2 * nbytes / (ms_copy * 1e-3) / 1e9, 1),
            "read_sum_gbs": round(nbytes / (ms_sum * 1e-3) / 1e9, 1),
            "note": "torch copy_ (read + write) and sum (read) of a 2 GiB float32 tensor"}


def percentiles_us(ms_list):
    """Median, p10 and p90 of launch durations given in milliseconds, in us."""
    import numpy as np
    a = np.asarray(ms_list, dtype=np.float64) * 1e3
    return {"p10_us": round(float(np.percentile(a, 10)), 2),
            "median_us": round(float(np.percentile(a, 50)), 2),
            "p90_us": round(float(np.percentile(a, 90)), 2)}


def host_description():
    """CPU model and BLAS library of the host the oracle runs on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')}"
    except Exception:  # pragma: no cover
        pass
    lscpu = {}
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            k, _, v = line.partition(":")
            if k.strip() in ("Model name", "Vendor ID", "CPU family", "Model", "Socket(s)",
                             "Core(s) per socket", "Thread(s) per core", "CPU(s)",
                             "CPU max MHz", "Hypervisor vendor"):
                lscpu[k.strip()] = v.strip()
    except Exception:  # pragma: no cover
        pass
    return {"cpu_model": model, "lscpu": lscpu, "blas": blas, "logical_cpus": os.cpu_count(),
            "affinity_cpus": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity")
            else None}


def _find_values(obj, want, inner=None):
    """Numeric ``value`` fields under every key accepted by ``want`` anywhere
    in a parsed amd-smi JSON document (``key: {inner: {"value": x}}`` when
    ``inner`` is given, else ``key: {"value": x}``)."""
    found = []
    if isinstance(obj, dict):
        for k, v in obj.items():
            if want(k) and isinstance(v, dict):
                leaf = v.get(inner) if inner else v
                val = leaf.get("value") if isinstance(leaf, dict) else None
                if isinstance(val, (int, float)):
                    found.append(float(val))
            found += _find_values(v, want, inner)
    elif isinstance(obj, list):
        for v in obj:
            found += _find_values(v, want, inner)
    return found


def sample_clock_power(fn, seconds=3.0):
    """Run ``fn`` back to back for about ``seconds`` while a thread samples the
    shader clock (mean over the XCDs' gfx clocks) and the socket power with
    ``amd-smi metric``; returns medians and sample counts, or the reason it
    could not sample."""
    import shutil
    import statistics
    import subprocess
    import threading
    import torch
    smi = shutil.which("amd-smi") or ("/opt/rocm/bin/amd-smi"
                                      if os.path.exists("/opt/rocm/bin/amd-smi") else None)
    if smi is None:
        return {"error": "amd-smi not found"}
    clocks, powers, errors = [], [], []
    stop = threading.Event()

    def poll():
        while not stop.is_set():
            try:
                r = subprocess.run([smi, "metric", "--clock", "--power", "--json"],
                                   capture_output=True, text=True, timeout=20)
                doc = json.loads(r.stdout)
            except Exception as e:  # pragma: no cover
                errors.append(repr(e)[:200])
                time.sleep(0.2)
                continue
            gfx = _find_values(doc, lambda k: str(k).startswith("gfx_"), inner="clk")
            pw = _find_values(doc, lambda k: str(k) in ("socket_power", "current_socket_power",
                                                        "average_socket_power"))
            if gfx:
                clocks.append(sum(gfx) / len(gfx))
            if pw:
                powers.append(pw[0])
            if not gfx and not pw:
                errors.append(r.stdout[:300])

    th = threading.Thread(target=poll, daemon=True)
    th.start()
    t0, n = time.perf_counter(), 0
    while time.perf_counter() - t0 < seconds or (not clocks and n < 100000 and
                                                  time.perf_counter() - t0 < 4 * seconds):
        for _ in range(20):
            fn()
            n += 1
        torch.cuda.synchronize()
    stop.set()
    th.join(timeout=30)
    res = {"window_s": round(time.perf_counter() - t0, 2), "steps": n, "samples": len(clocks)}
    if clocks:
        res["sclk_mhz_median"] = round(statistics.median(clocks), 1)
        res["sclk_mhz_min"] = round(min(clocks), 1)
        res["sclk_mhz_max"] = round(max(clocks), 1)
    if powers:
        res["socket_power_w_median"] = round(statistics.median(powers), 1)
    if errors and not clocks:
        res["error"] = errors[0]
    return res


def bench_copy(args, dev):
    """The write-back scatter (HBM bound) or the offload (host-link bound) alone."""
    import numpy as np
    import torch
    from paper_2608_14624_amd import ops
    from paper_2608_14624_amd.workload import make_config
    wl = make_config(args.workload)
    stream = torch.cuda.current_stream(dev)
    k_pool = torch.from_numpy(wl.k_pool.view(np.int16)).view(torch.bfloat16).to(dev)
    v_pool = torch.from_numpy(wl.v_pool.view(np.int16)).view(torch.bfloat16).to(dev)
    hkv, d = wl.num_kv_heads, wl.head_dim
    if args.component in ("decode", "cascade_decode"):
        from paper_2608_14624_amd.workload import cascade_view, decode_view
        # the batch ordered by agent group (the order cascade decode needs;
        # plain decode runs on the same order)
        cv = cascade_view(wl)
        q_np, seq_lens_np = decode_view(wl)
        order = cv["order"]
        q_np, seq_lens_np = np.ascontiguousarray(q_np[order]), np.ascontiguousarray(seq_lens_np[order])
        bt_np = np.ascontiguousarray(wl.block_tables[order])
        q = torch.from_numpy(q_np.view(np.int16)).view(torch.bfloat16).to(dev)
        out = torch.empty_like(q)
        bt = torch.from_numpy(bt_np).to(dev)
        seq_lens = torch.from_numpy(seq_lens_np).to(dev)
        max_len = int(seq_lens_np.max())
        # K and V of every key every sequence attends to (what a per-sequence
        # kernel reads), and the distinct pool blocks among them (the least a
        # kernel must read from HBM); both plus q and out
        qo = 2 * q.numel() * 2
        logical = int(seq_lens_np.astype(np.int64).sum()) * hkv * d * 2 * 2 + qo
        unique_blocks = len(np.unique(np.concatenate(
            [bt_np[r, :-(-int(L) // 16)] for r, L in enumerate(seq_lens_np)])))
        unique_bytes = unique_blocks * hkv * 16 * d * 2 * 2 + qo
        moved = unique_bytes
        if args.component == "decode":
            def fn():
                ops.cs_paged_decode_attn(q, k_pool, v_pool, bt, seq_lens, out,
                                         max_seq_len=max_len, scale=wl.scale, stream=stream)
        else:
            cu = torch.from_numpy(cv["cu_groups"]).to(dev)
            shared = torch.from_numpy(cv["shared_lens"]).to(dev)
            need = ops.cs_cascade_decode_workspace_bytes(wl.batch, wl.num_q_heads, d,
                                                         cv["max_shared_len"],
                                                         cv["max_rest_len"])
            ws = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)

            def fn():
                ops.cs_cascade_decode_attn(q, k_pool, v_pool, bt, seq_lens, cu, shared, out,
                                           max_seq_len=max_len,
                                           max_group_seqs=cv["max_group_seqs"],
                                           max_shared_len=cv["max_shared_len"],
                                           max_rest_len=cv["max_rest_len"], scale=wl.scale,
                                           workspace=ws, stream=stream)
        peak, bound = PEAK_HBM_GBS, "hbm"
        unit_desc = (f"{wl.batch} sequences in {len(cv['shared_lens'])} agent groups, "
                     f"{int(seq_lens_np.sum())} keys, {unique_blocks} distinct pool blocks "
                     f"({unique_blocks * hkv * 16 * d * 4 / 1e6:.0f} MB of unique K/V)")
    elif args.component == "kv_write":
        # the suffix tokens of every invocation, written to their own slots
        slots = []
        for r in range(wl.batch):
            p, s = int(wl.prefix_lens[r]), int(wl.q_lens[r])
            j = np.arange(p, p + s)
            slots.append(wl.block_tables[r, j // 16].astype(np.int64) * 16 + j % 16)
        slots = torch.from_numpy(np.concatenate(slots).astype(np.int32)).to(dev)
        t = slots.numel()
        k_new = torch.randn((t, hkv, d), device=dev).to(torch.bfloat16)
        v_new = torch.randn((t, hkv, d), device=dev).to(torch.bfloat16)
        moved = 2 * 2 * t * hkv * d * 2        # K and V, read once and written once

        def fn():
            ops.cs_kv_write(k_new, v_new, slots, k_pool, v_pool, stream=stream)
        peak, bound, unit_desc = PEAK_HBM_GBS, "hbm", f"{t} tokens"
    elif args.component == "kv_prefetch":
        # the prefetch alone: 256 blocks (16 MiB) is the line's value; the
        # sweep and a plain pinned host-to-device copy of the same bytes (the
        # link as the runtime's own copy reaches it) go beside it
        sweep, n_main = {}, 256
        g = torch.Generator().manual_seed(7)
        for n in (64, 256, 1024, 4096):
            ids_n = torch.from_numpy(np.random.default_rng(n).choice(wl.num_blocks, n, replace=False)
                                     .astype(np.int32)).to(dev)
            hk = torch.empty((n, hkv, 16, d), dtype=torch.bfloat16, pin_memory=True)
            hv = torch.empty_like(hk, pin_memory=True)
            hk.copy_(torch.randn(hk.shape, generator=g).to(torch.bfloat16))
            hv.copy_(torch.randn(hv.shape, generator=g).to(torch.bfloat16))
            nbytes = 2 * n * hkv * 16 * d * 2

            def pf(hk=hk, hv=hv, ids_n=ids_n):
                ops.cs_kv_prefetch(hk, hv, ids_n, k_pool, v_pool, stream=stream)
            _, ms, _ = _time_launches(pf, max(5, args.steps // 5), 2, stream)
            sweep[str(n)] = {"bytes": nbytes, "avg_launch_us": round(ms * 1e3, 2),
                             "gbs": round(nbytes / (ms * 1e-3) / 1e9, 2)}
            if n == n_main:
                host_k, host_v, ids, moved = hk, hv, ids_n, nbytes
        flat = host_k.view(-1)
        dev_buf = torch.empty(flat.shape, dtype=flat.dtype, device=dev)

        def h2d():
            dev_buf.copy_(flat, non_blocking=True)
        _, ms, _ = _time_launches(h2d, 20, 3, stream)
        memcpy = {"bytes": flat.numel() * 2, "gbs": round(flat.numel() * 2 / (ms * 1e-3) / 1e9, 2),
                  "note": "torch copy_ from the pinned K buffer: the runtime's own host-to-"
                          "device copy, a measured reference for the link"}

        def fn():
            ops.cs_kv_prefetch(host_k, host_v, ids, k_pool, v_pool, stream=stream)
        peak, bound, unit_desc = PEAK_PCIE5_X16_GBS, "host_link", f"{n_main} blocks"
    else:
        n = 256
        ids = torch.from_numpy(np.random.default_rng(5).choice(wl.num_blocks, n, replace=False)
                               .astype(np.int32)).to(dev)
        host_k = torch.empty((n, hkv, 16, d), dtype=torch.bfloat16, pin_memory=True)
        host_v = torch.empty_like(host_k, pin_memory=True)
        moved = 2 * n * hkv * 16 * d * 2        # K and V blocks over the host link

        def fn():
            ops.cs_kv_offload(ids, k_pool, v_pool, host_k, host_v, stream=stream)
        peak, bound, unit_desc = PEAK_PCIE5_X16_GBS, "host_link", f"{n} blocks"
    kernel, sources = {
        "decode": ("paged_decode_attn_kernel<128, false>",
                   ("paper_2608_14624_amd/csrc/paged_decode_attn.hip",)),
        "cascade_decode": ("shared_prefix_partials_kernel<128> + paged_decode_attn_kernel<128, true>"
                           " + cascade_merge_kernel<128>",
                           ("paper_2608_14624_amd/csrc/prefill_paged_attn.hip",
                            "paper_2608_14624_amd/csrc/paged_decode_attn.hip",
                            "paper_2608_14624_amd/csrc/internal.h")),
        "kv_write": ("kv_write_kernel", ("paper_2608_14624_amd/csrc/kv_copy.hip",)),
        "kv_offload": ("kv_offload_kernel", ("paper_2608_14624_amd/csrc/kv_copy.hip",
                                             "paper_2608_14624_amd/csrc/block_copy.h")),
        "kv_prefetch": ("kv_prefetch_kernel", ("paper_2608_14624_amd/csrc/kv_prefetch.hip",
                                               "paper_2608_14624_amd/csrc/block_copy.h")),
    }[args.component]
    traffic = load_traffic(kernel, args.workload, source_hash(sources))
    wall, avg_ms, all_ms = _time_launches(fn, args.steps, args.warmup, stream)
    gbs = moved / (avg_ms * 1e-3) / 1e9
    extra = {}
    if args.component == "kv_prefetch":
        extra = {"sweep_blocks": sweep, "memcpy_h2d": memcpy}
    if args.component in ("decode", "cascade_decode"):
        extra = {"logical_bytes": logical,
                 "logical_rate_gbs": round(logical / (avg_ms * 1e-3) / 1e9, 2),
                 "note": "achieved counts each distinct K/V block once (plus q and out); "
                         "logical counts the K/V of every key of every sequence"}
    if args.component in ("decode", "cascade_decode", "kv_write"):
        extra["hbm_reference"] = hbm_reference(dev, stream)
    return {"metric": f"{args.component} GB/s, 1 MI355X", "value": round(gbs, 2), "unit": "GB/s",
            "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": round(wall / args.steps * 1e3, 4), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"{args.component} of {unit_desc} of {args.workload}",
                       "bytes_per_launch": moved},
            "roofline": {"bound": bound, "achieved": round(gbs, 2), "peak": peak, "unit": "GB/s",
                         "frac": round(gbs / peak, 4), "traffic": traffic, "kernel": kernel,
                         "avg_launch_us": round(avg_ms * 1e3, 2),
                         "launch_us": percentiles_us(all_ms), **extra},
            "cpu_baseline": None}


def bench_control_plane(args):
    """The host-side control plane (cs_scout_*) on a synthetic agent trace:
    24 agents whose successor is a fixed one 80% of the time, each turn
    touching 64 blocks of a 16384-block pool.  Native costs come from batched
    calls (no per-touch FFI); per-call costs include one ctypes round trip,
    reported alongside as `ffi_floor_us`.  Host only: no GPU is used."""
    import numpy as np
    from paper_2608_14624_amd import ops
    import oracle.control_plane as oracle_cp

    agents, blocks, per_turn, turns = 24, 16384, 64, 4096
    rng = np.random.default_rng(11)
    succ = rng.permutation(agents)
    seq = np.empty(turns, dtype=np.int32)
    a = 0
    for t in range(turns):
        seq[t] = a
        a = succ[a] if rng.random() < 0.8 else rng.integers(agents)
    tr_agents = np.repeat(seq, per_turn)
    tr_blocks = rng.integers(0, blocks, tr_agents.size, dtype=np.int32)
    tr_tokens = np.full(tr_agents.size, 16, dtype=np.int32)
    tr_now = np.repeat(np.arange(turns, dtype=np.int64), per_turn)
    dispatches = int(np.count_nonzero(np.diff(seq)) + 1)

    def best_of(fn, reps=5):
        best = float("inf")
        for _ in range(reps):
            t0 = time.perf_counter()
            fn()
            best = min(best, time.perf_counter() - t0)
        return best

    def replay():
        sc = ops.Scout(agents, blocks)
        sc.observe_touches(tr_blocks, tr_agents, tr_tokens, tr_now)
        return sc
    t_trace = best_of(replay)
    # every touch a dispatch: the transition update plus the hop-table rebuild
    alt = np.tile(np.arange(agents, dtype=np.int32), 2000)
    alt_b = rng.integers(0, blocks, alt.size, dtype=np.int32)
    alt_tok = np.full(alt.size, 16, dtype=np.int32)
    alt_now = np.arange(alt.size, dtype=np.int64)
    sc = replay()
    t_disp = best_of(lambda: sc.observe_touches(alt_b, alt, alt_tok, alt_now))

    n_calls = 20000
    floor = best_of(lambda: [sc.current for _ in range(n_calls)]) / n_calls
    t_surv = best_of(lambda: [sc.survival_all() for _ in range(n_calls // 10)]) / (n_calls // 10)
    cands = [int(b) for b in rng.integers(0, blocks, 32)]
    t_victim = best_of(lambda: [sc.select_victim(cands, turns) for _ in range(n_calls)]) / n_calls
    t_between = best_of(lambda: [sc.between_step() for _ in range(n_calls)]) / n_calls

    # the oracle on a bounded prefix of the same trace
    n_or = 20000
    t0 = time.perf_counter()
    plane = oracle_cp.ControlPlane(agents, blocks)
    for i in range(n_or):
        plane.observe_touch(int(tr_blocks[i]), int(tr_agents[i]), 16, int(tr_now[i]))
    t_oracle = time.perf_counter() - t0

    touch_us = t_trace / tr_agents.size * 1e6
    return {"metric": "control-plane ObserveTouch us per block touch (host)",
            "value": round(touch_us, 4), "unit": "us", "n_gpus": 0, "steps": 1, "warmup": 0,
            "ms_per_step": round(t_trace * 1e3, 3), "higher_is_better": False,
            "scaling": "weak", "vs_baseline": round(touch_us / 1.0, 4), "dtype": "f64",
            "data": "synthetic",
            "config": {"workload": f"{agents} agents, {turns} turns x {per_turn} block touches, "
                                   f"{blocks}-block pool, dominant successor p=0.8",
                       "touches": int(tr_agents.size), "dispatches": dispatches},
            "control_plane": {
                "observe_touch_us": round(touch_us, 4),
                "dispatch_us": round(t_disp / alt.size * 1e6, 4),
                "survival_all_us": round(t_surv * 1e6, 3),
                "select_victim_32_us": round(t_victim * 1e6, 3),
                "between_step_us": round(t_between * 1e6, 3),
                "ffi_floor_us": round(floor * 1e6, 3),
                "state_bytes_24_agents": ops.Scout(agents, 0).state_bytes(),
                "state_bytes_with_pool": sc.state_bytes(),
                "paper": {"observe_touch_us": 1.0, "predict_survival_us": 6.0,
                          "state_bytes": 25 * 1024}},
            "roofline": None,
            "cpu_baseline": {"value": round(t_oracle / n_or * 1e6, 3), "unit": "us", "cores": 1,
                             "kind": "oracle",
                             "sample": f"first {n_or} touches of the same trace"}}


# (prefix, suffix, invocations, query heads, KV heads, head_dim): one agent's
# invocations, all hits on the same prefix
SWEEP = [(0, 512, 16, 32, 8, 128), (2048, 512, 16, 32, 8, 128), (4096, 512, 16, 32, 8, 128),
         (2048, 2048, 4, 32, 8, 128), (8192, 1024, 4, 32, 8, 128), (1024, 128, 64, 32, 8, 128),
         (4096, 512, 16, 64, 8, 128), (2048, 1024, 8, 16, 8, 128), (2048, 1024, 8, 8, 8, 128),
         (2048, 512, 16, 32, 8, 64)]


def bench_attn_sweep(args, dev):
    """Prefill attention alone, one launch per shape, back to back with HIP
    events on the launch stream; value = geometric mean of the shapes' rates."""
    import math
    import torch
    from paper_2608_14624_amd import ops, pipeline
    from paper_2608_14624_amd.workload import Invocation, build_workload
    stream = torch.cuda.current_stream(dev)
    rows = []
    for i, (P, S, B, hq, hkv, d) in enumerate(SWEEP):
        nb = P // 16 + B * (-(-(P % 16 + S) // 16) + 1) + 64
        wl = build_workload(f"sweep{i}", 40 + i, [P], [Invocation(0, S) for _ in range(B)],
                            num_q_heads=hq, num_kv_heads=hkv, head_dim=d, num_blocks=nb)
        dw = pipeline.DeviceWorkload(wl)
        sb = pipeline.SubBatch(dw, 0, wl.batch)
        kernel, grid, tail = ops.prefill_launch_shape(wl.batch, wl.max_q_len, hq, hkv)
        fn = lambda: sb.attention(stream=stream)
        _, avg_ms, _ = _time_launches(fn, max(args.steps, 20), max(args.warmup, 3), stream)
        avg_us = avg_ms * 1e3
        rows.append({"prefix": P, "suffix": S, "invocations": B, "q_heads": hq, "kv_heads": hkv,
                     "head_dim": d, "kernel": attention_kernel_name(wl.batch, wl.max_q_len, hq, hkv, d),
                     "work_groups": grid, "tail_work_groups": tail, "avg_launch_us": round(avg_us, 2),
                     "tflops": round(sb.flops / (avg_us * 1e-6) / 1e12, 1)})
        del dw, sb
        torch.cuda.empty_cache()
    gm = math.exp(sum(math.log(r["tflops"]) for r in rows) / len(rows))
    return {"metric": "prefill-attn TFLOP/s across shapes (geometric mean), 1 MI355X",
            "value": round(gm, 1), "unit": "TFLOP/s", "n_gpus": 1, "steps": max(args.steps, 20),
            "warmup": max(args.warmup, 3), "ms_per_step": None, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"{len(rows)} single-agent shapes (prefix, suffix, "
                                   "invocations, heads, head_dim); see sweep"},
            "roofline": {"bound": "mfma", "achieved": round(gm, 1), "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(gm / PEAK_BF16_TFLOPS, 4), "traffic": None},
            "cpu_baseline": None, "sweep": rows}


def bench_kv_locality(args, dev):
    """What the K/V fetches cost the prefill attention: the workload's batch in
    one launch with its real block tables, then the same launch (same
    lengths, the same FLOP) with every table entry pointing at one of 16 pool
    slots of the first invocation, so that every K/V read after the first
    few hits in L2.  The difference bounds what any scheme that reads each
    shared anchor block only once (a shared-prefix cascade) can save; the
    cascade's own partial results would add HBM traffic on top."""
    import numpy as np
    import torch
    from paper_2608_14624_amd import ops, pipeline
    from paper_2608_14624_amd.workload import make_config
    stream = torch.cuda.current_stream(dev)
    wl = make_config(args.workload)
    dw = pipeline.DeviceWorkload(wl)
    dw.prefetch_all()
    sb = pipeline.SubBatch(dw, 0, wl.batch)
    steps, warm = max(args.steps, 20), max(args.warmup, 3)
    _, real_ms, real_list = _time_launches(lambda: sb.attention(stream=stream), steps, warm, stream)
    n0 = -(-int(wl.kv_lens[0]) // wl.block_size)
    hot = wl.block_tables[0, :min(16, n0)].astype(np.int32)
    bt_hot = hot[np.arange(wl.block_tables.shape[1]) % len(hot)][None, :].repeat(wl.batch, axis=0)
    bt_hot_d = torch.from_numpy(np.ascontiguousarray(bt_hot)).to(dev)
    out_hot = torch.empty_like(dw.out)

    def hot_call():
        ops.cs_prefill_paged_attn(dw.q, dw.k_pool, dw.v_pool, bt_hot_d, dw.prefix_lens,
                                  dw.cu_q_lens, out_hot, max_q_len=wl.max_q_len,
                                  max_kv_len=wl.max_kv_len, scale=wl.scale, stream=stream)
    _, hot_ms, hot_list = _time_launches(hot_call, steps, warm, stream)
    torch.cuda.synchronize()
    assert torch.isfinite(out_hot.float()).all().item()
    flops = wl.flops()
    rows = wl.total_q * wl.num_q_heads
    # a cascade writes and reads back two fp32 partials (O, m, l) per row:
    # the shared-anchor part and the own-key part
    partial_bytes = 2 * 2 * rows * (wl.head_dim + 2) * 4
    real_us, hot_us = real_ms * 1e3, hot_ms * 1e3
    return {"metric": "prefill-attn us per launch, real block tables vs K/V served from L2",
            "value": round(real_us, 2), "unit": "us", "n_gpus": 1, "steps": steps,
            "warmup": warm, "ms_per_step": round(real_ms, 4), "higher_is_better": False,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": f"{args.workload}: {DESCRIPTIONS.get(args.workload, '')}",
                       "launch": "all invocations in one cs_prefill_paged_attn call",
                       "hot_slots": int(len(hot))},
            "real_tables": {"avg_launch_us": round(real_us, 2), "launch_us": percentiles_us(real_list),
                            "tflops": round(flops / (real_ms * 1e-3) / 1e12, 1)},
            "kv_from_l2": {"avg_launch_us": round(hot_us, 2), "launch_us": percentiles_us(hot_list),
                           "tflops": round(flops / (hot_ms * 1e-3) / 1e12, 1)},
            "kv_fetch_share_of_time": round(1.0 - hot_us / real_us, 4),
            "cascade_partial_bytes": partial_bytes,
            "cascade_partial_us_at_5tbs": round(partial_bytes / 5e12 * 1e6, 1),
            "roofline": None, "cpu_baseline": None}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama70b_prefetch",
                    choices=sorted(DESCRIPTIONS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-clock", action="store_true",
                    help="skip the amd-smi clock / power sampling after the timed region")
    ap.add_argument("--no-workspace", action="store_true",
                    help="run the plain cs_prefill_paged_attn; by default the attention runs "
                         "cs_prefill_paged_attn_ws, which splits launches too small to fill the "
                         "GPU into key parts (launches of a round or more are unchanged)")
    ap.add_argument("--overlap", action="store_true",
                    help="serving step: consecutive agents' attention launches alternate between "
                         "two streams, so one launch's last round runs beside the next one's "
                         "first (known order only; the per-launch events still time launches "
                         "one after another)")
    ap.add_argument("--policy", default="order", choices=("order", "scout"),
                    help="prefetch target: the next agent in dispatch order (default) or the "
                         "control plane's between-step decision (cs_scout_*); the warmup "
                         "steps let it learn the dispatch cycle")
    ap.add_argument("--component", default="pipeline",
                    choices=("pipeline", "kv_write", "kv_offload", "kv_prefetch", "decode",
                             "cascade_decode", "control_plane", "attn_sweep", "kv_locality"),
                    help="pipeline (default): the serving step; kv_write / kv_offload / "
                         "kv_prefetch: the write-back scatter, the offload copy and the "
                         "prefetch (with a sweep over 64-4096 blocks) on their own; "
                         "decode / cascade_decode: paged decode attention, per sequence or "
                         "with each agent's anchor read once (use --workload decode_batch); "
                         "control_plane: the host-side scout on a synthetic agent trace; "
                         "attn_sweep: prefill attention alone over a grid of prefix / "
                         "suffix lengths, GQA groups and head dims; kv_locality: one "
                         "launch of the workload with its real block tables and with every "
                         "K/V read served from L2 (what a shared-prefix cascade could save)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run only a plain 1 GiB device-to-device copy (the reference kernel "
                         "for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE readings)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the path "
              "shards by KV head or by invocation with no exchange inside it, see the "
              "design notes)", file=sys.stderr)
        sys.exit(2)

    if args.component == "control_plane":
        print(json.dumps(bench_control_plane(args)), flush=True)
        return

    import numpy as np
    import torch
    from paper_2608_14624_amd import build, ops, pipeline
    from paper_2608_14624_amd.workload import make_config

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_probe:
        nbytes = 1 << 30
        src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device=dev).normal_()
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": nbytes, "copy_probe_bytes_written": nbytes,
                          "launches": 5}), flush=True)
        return
    if args.component == "attn_sweep":
        print(json.dumps(bench_attn_sweep(args, dev)), flush=True)
        return
    if args.component == "kv_locality":
        print(json.dumps(bench_kv_locality(args, dev)), flush=True)
        return
    if args.component != "pipeline":
        print(json.dumps(bench_copy(args, dev)), flush=True)
        return
    wl = make_config(args.workload)
    dw = pipeline.DeviceWorkload(wl, dev, workspace=None if args.no_workspace else "auto")
    main_stream = torch.cuda.current_stream(dev)
    if wl.prefetch_dst is not None:
        # serving order with the next agent's prefetch overlapped on a side stream
        policy = None
        if args.policy == "scout":
            policy = pipeline.ScoutPolicy(wl, sorted({inv.agent for inv in wl.invocations}))
        pipe = pipeline.AgentPipeline(dw, policy=policy, overlap=args.overlap)
        pipe.stage_first()
        n_launch = len(pipe.agents)
        step_flops, step_bytes, warm = pipe.flops, pipe.prefetch_bytes, pipe.step
        # the per-launch events time launches one after another, so with
        # --overlap they come from a pipeline of the same work without it
        pipe_ev = pipe if not pipe.overlap else pipeline.AgentPipeline(dw)
    else:
        # no CPU-tier blocks: the whole batch is one attention launch
        pipe = pipe_ev = None
        n_launch = 1
        step_flops, step_bytes, warm = wl.flops(), 0, dw.attention
    for _ in range(args.warmup):
        warm()
    torch.cuda.synchronize()

    # per-launch events: attention on the main stream, prefetch on the side stream
    def events():
        return [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                 for _ in range(n_launch)] for _ in range(args.steps)]
    a_ev, p_ev = events(), events()

    def timed_step(si):
        if pipe is None:
            a_ev[si][0][0].record(main_stream)
            dw.attention(stream=main_stream)
            a_ev[si][0][1].record(main_stream)
            return
        # AgentPipeline.step with events around each launch
        pipe_ev.step(timing=list(zip(p_ev[si], a_ev[si])))

    torch.cuda.synchronize()
    pipes = [] if pipe is None else ([pipe] if pipe_ev is pipe else [pipe, pipe_ev])
    hits0, misses0 = sum(q.hits for q in pipes), sum(q.misses for q in pipes)
    # the timed region: exactly `steps` serving steps, nothing recorded inside
    t0 = time.perf_counter()
    for _ in range(args.steps):
        warm()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # then the same steps again with events around every launch, for the
    # per-launch durations of the roofline (the events themselves cost a few
    # percent of the step, so they stay out of the timed region)
    for si in range(args.steps):
        timed_step(si)
    torch.cuda.synchronize()

    ms_per_step = wall / args.steps * 1e3
    value = step_flops * args.steps / wall / 1e12
    attn_ms = sum(e0.elapsed_time(e1) for row in a_ev for e0, e1 in row)
    n_attn = args.steps * n_launch
    attn_avg_ms = attn_ms / n_attn
    achieved = step_flops * args.steps / (attn_ms * 1e-3) / 1e12
    pf_bytes_per_step = step_bytes
    prefetch = None
    if pf_bytes_per_step:
        pf_ms = [e0.elapsed_time(e1) for row in p_ev for e0, e1 in row]
        # the same copies with nothing else on the GPU (after the timed region)
        iso_ms = []
        for _ in range(3):
            for a in pipe.agents:
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(main_stream)
                pipe.prefetch_agent(a, main_stream)
                e1.record(main_stream)
                iso_ms.append((e0, e1))
        torch.cuda.synchronize()
        iso = sum(e0.elapsed_time(e1) for e0, e1 in iso_ms) / len(iso_ms)
        iso_gbs = pf_bytes_per_step / n_launch / (iso * 1e-3) / 1e9
        pf_gbs = pf_bytes_per_step * args.steps / (sum(pf_ms) * 1e-3) / 1e9
        # the attention launches of a step alone, back to back on one stream
        # (all of their work, no copy beside them): how much the prefetch
        # running beside them costs, and the serial sum the overlap beats
        def attention_only():
            for b in pipe.batches:
                b.attention(stream=main_stream)
        for _ in range(args.warmup):
            attention_only()
        torch.cuda.synchronize()
        al_ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(n_launch)] for _ in range(args.steps)]
        for row in al_ev:
            for b, (e0, e1) in zip(pipe.batches, row):
                e0.record(main_stream)
                b.attention(stream=main_stream)
                e1.record(main_stream)
        torch.cuda.synchronize()
        alone_ms = [e0.elapsed_time(e1) for row in al_ev for e0, e1 in row]
        alone_step_ms = sum(alone_ms) / args.steps
        prefetch = {"value": round(pf_gbs, 2), "unit": "GB/s",
                    "frac_link": round(pf_gbs / PEAK_PCIE5_X16_GBS, 4),
                    "link_peak": PEAK_PCIE5_X16_GBS, "frac_hbm": round(pf_gbs / PEAK_HBM_GBS, 5),
                    "bytes_per_step": pf_bytes_per_step, "launches_per_step": n_launch,
                    "avg_launch_us": round(sum(pf_ms) / len(pf_ms) * 1e3, 2),
                    "launch_us": percentiles_us(pf_ms),
                    "overlapped_with_attention": True,
                    "isolated": {"value": round(iso_gbs, 2), "unit": "GB/s",
                                 "frac_link": round(iso_gbs / PEAK_PCIE5_X16_GBS, 4),
                                 "avg_launch_us": round(iso * 1e3, 2)},
                    "attention_alone": {
                        "avg_launch_us": round(sum(alone_ms) / len(alone_ms) * 1e3, 2),
                        "launch_us": percentiles_us(alone_ms),
                        "slowdown_beside_prefetch": round(
                            (attn_ms / n_attn) / (sum(alone_ms) / len(alone_ms)), 4),
                        "serial_sum_ms_per_step": round(alone_step_ms + iso * n_launch, 4),
                        "overlapped_ms_per_step": round(ms_per_step, 4)}}
    khash = source_hash(KERNEL_SOURCES[:1])
    batches = pipe.batches if pipe is not None else [pipeline.SubBatch(dw, 0, wl.batch)]
    kernel_names = sorted({attention_kernel_name(b.hi - b.lo, b.max_q_len, wl.num_q_heads,
                                                 wl.num_kv_heads, wl.head_dim,
                                                 key_parts(b, wl, dw.workspace))
                           for b in batches})
    kernel_name = " + ".join(kernel_names)
    traffic = load_traffic(kernel_name, args.workload, khash)
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {DESCRIPTIONS[args.workload]}",
                   "attention_flop_per_step": step_flops,
                   "attention_launches_per_step": n_launch,
                   "total_q": wl.total_q, "num_blocks": wl.num_blocks},
        "frac_of_bf16_peak": round(value / PEAK_BF16_TFLOPS, 4),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic,
                     "kernel": kernel_name,
                     "avg_launch_us": round(attn_avg_ms * 1e3, 2),
                     "launch_us": percentiles_us(
                         [e0.elapsed_time(e1) for row in a_ev for e0, e1 in row]),
                     "flop_per_launch": step_flops // n_launch,
                     "timing": "HIP events around every launch, in a second pass of the "
                               "same steps after the timed region"},
        "prefetch": prefetch,
        "prefetch_policy": None if pipe is None else {
            "name": args.policy, "hits": sum(q.hits for q in pipes) - hits0,
            "misses": sum(q.misses for q in pipes) - misses0,
            "launches_overlapped": pipe.overlap},
        "kernel_sha": khash,
        "library_digest": ops.source_digest(),
        "source_digest": build.source_digest(),
        "cpu_baseline": None,
    }
    # the clock the chip holds under this load, sampled over a few seconds of
    # the same steps after everything above (the timed region is too short
    # for amd-smi), and the fraction of the peak at that clock
    clk = {"skipped": True} if args.no_clock else sample_clock_power(warm)
    result["clock"] = clk
    if clk.get("sclk_mhz_median"):
        peak_at = PEAK_BF16_TFLOPS * clk["sclk_mhz_median"] / PEAK_SCLK_MHZ
        result["roofline"]["frac_at_measured_sclk"] = round(achieved / peak_at, 4)
        result["roofline"]["peak_at_measured_sclk"] = round(peak_at, 1)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
