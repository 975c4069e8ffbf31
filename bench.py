"""Benchmark: prefix-shared beam decode attention on one MI355X.

One step = one decode-attention call of one transformer layer for every beam
of the batch (``tts_prefix_decode_attn``), i.e. one pass of the hot path
over one batch. Steps rotate over ``--layers`` independent layer KV pools
(same beam tree and block tables, different K/V values and queries), so the
working set exceeds the 256 MB Infinity Cache and the timed KV reads come
from HBM. The prefix metadata is built once per tree (once per reasoning
step of the search); its host time is reported separately.

Metric: beam-tokens/s = beams advanced by one token / time per layer call,
plus the fraction of HBM peak achieved on the unique KV bytes of one call.

Prints one JSON line. ``--gpus`` above 1 is refused: the library runs on one
GPU.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "beam-tokens/s per decode step + % HBM peak (unique KV bytes), 1 MI355X"
HBM_PEAK_GBS = 8000.0
KERNEL_SRC = os.path.join(ROOT, "paper_2509_00195_amd", "csrc", "tts_kernels.hip")
PLANNER_SRC = os.path.join(ROOT, "paper_2509_00195_amd", "csrc", "tts_plan.cpp")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def kernel_sha() -> str:
    """Hash of the attention kernel's source, the work planner's source and the device compile flags (a traffic
    record is valid only for the code and the plans it was measured on)."""
    from paper_2509_00195_amd.build import DEVICE

    h = hashlib.sha256()
    for src in (KERNEL_SRC, PLANNER_SRC):
        with open(src, "rb") as f:
            h.update(f.read())
    h.update(" ".join(DEVICE).encode())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=560)
    ap.add_argument("--warmup", type=int, default=56)
    ap.add_argument("--config", default="7b64")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--layers", type=int, default=28,
                    help="independent layer pools to rotate over (raised until they hold twice the 256 MB cache)")
    ap.add_argument("--variant", choices=["prefix", "paged"], default="prefix")
    ap.add_argument("--graph", action="store_true", help="replay the steps from a captured HIP graph")
    ap.add_argument("--q-len", type=int, default=1,
                    help="verification: every beam's last Q tokens are causal queries (prefix variant only; "
                         "value is then query tokens/s)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=16.0,
                    help="host time for the oracle leg, split between one thread and all threads")
    ap.add_argument("--no-check", action="store_true",
                    help="skip comparing the call on layer 0 with the oracle (on by default; the oracle output "
                         "of the cpu_baseline leg is reused)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after the timed region, stream this many MiB device-to-device three times with a plain "
                         "elementwise copy (dst = ~src; counter calibration runs)")
    ap.add_argument("--ingest-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="read two rocprofv3 counter_collection.csv files (FETCH_SIZE run, WRITE_SIZE run, both "
                         "made with --copy-mib) and record the attention kernel's HBM bytes per launch in "
                         "profiles/traffic.json; runs no GPU work")
    return ap.parse_args()


def make_layers(wl, x, layers, seed):
    """Per-layer K/V pools and queries: layer 0 is the generator's; others drawn on the GPU."""
    import torch

    sh = wl.shape
    pools = [(x.q, x.k_cache, x.v_cache, x.k_scale, x.v_scale)]
    g = torch.Generator(device=x.q.device)
    g.manual_seed(1000 + seed)
    for _ in range(1, layers):
        def draw(shape, kind):
            v = torch.randn(shape, generator=g, device=x.q.device, dtype=torch.float32)
            if kind == "bf16":
                return v.to(torch.bfloat16)
            if kind == "fp8":
                return v.clamp(-448, 448).to(torch.float8_e4m3fn).view(torch.uint8)
            return v
        q = draw(tuple(x.q.shape), sh.q_dtype)
        k = draw(tuple(x.k_cache.shape), sh.kv_dtype)
        v = draw(tuple(x.v_cache.shape), sh.kv_dtype)
        ks = vs = None
        if sh.kv_dtype == "fp8":
            ks = torch.rand(wl.num_blocks, generator=g, device=x.q.device) * 0.01 + 0.001
            vs = torch.rand(wl.num_blocks, generator=g, device=x.q.device) * 0.01 + 0.001
        pools.append((q, k, v, ks, vs))
    return pools


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:  # pragma: no cover
        pass
    return "unknown"


def cpu_baseline(wl, budget_s):
    """The oracle, as is, on the same batch: whole layer calls, first on one BLAS thread, then on all of them,
    about half the budget each; the faster leg is the reported value. Returns the record and the oracle's output
    of the first call."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle.attention import oracle_attn_workload

    info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = max([i.get("num_threads", 1) for i in info] + [1])
    blas = ", ".join(f"{i.get('internal_api')} {i.get('version')} ({i.get('threading_layer')})" for i in info) or "none"

    def run(limit, budget):
        n, first = 0, None
        with threadpool_limits(limits=limit, user_api="blas"):
            t0 = time.perf_counter()
            while True:
                out = oracle_attn_workload(wl)
                if first is None:
                    first = out
                n += 1
                el = time.perf_counter() - t0
                if el >= budget or n >= 64:
                    break
        return n, el, first

    n1, el1, ref = run(1, 0.5 * budget_s)
    na, ela, _ = run(threads, 0.5 * budget_s)
    v1, va = wl.num_seqs / (el1 / n1), wl.num_seqs / (ela / na)
    # the faster of the two legs is the baseline; `cores` is the thread count of that leg
    rec = {"value": max(v1, va), "unit": "beam-tokens/s", "cores": 1 if v1 >= va else int(threads), "kind": "oracle",
           "value_1_thread": v1, "value_all_threads": va, "all_threads": int(threads),
           "host": {"os_cpu_count": os.cpu_count(), "cpu_model": _cpu_model(), "blas": blas},
           "sample": f"{wl.name} batch ({wl.num_seqs} beams, all heads), whole layer calls, numpy fp32 oracle: "
                     f"{n1} calls in {el1:.1f} s on 1 BLAS thread, {na} calls in {ela:.1f} s on {threads}"}
    return rec, ref


def meta_timings(wl, desc, prev, reps=5):
    """Host cost of the metadata (median of warm runs, ms): the trie, segments and beam order alone; the same
    plus the work plan (host only, no allocation); the full build with the device upload; and the update after a
    fork, re-planned warm from the previous metadata (tts_fork_prefix_meta; timed on the same tables, whose
    sizes set its cost)."""
    from paper_2509_00195_amd import tts as T

    def med(fn):
        fn()
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter()
            fn()
            ts.append((time.perf_counter() - t0) * 1e3)
        return float(np.median(ts))

    ncu = 256
    try:
        import torch

        ncu = torch.cuda.get_device_properties(0).multi_processor_count
    except Exception:  # pragma: no cover
        pass
    args = (wl.req_seq_offsets, wl.block_tables, wl.seq_lens, wl.shape.block_size, wl.num_blocks)
    return {
        "host_trie_ms": med(lambda: T.tts_build_prefix_meta(*args)),
        "host_trie_and_plan_ms": med(lambda: T.tts_plan_units_host(*args, desc, ncu)),
        "build_with_upload_ms": med(lambda: T.tts_build_prefix_meta(*args, desc=desc)),
        "fork_update_ms": med(lambda: T.tts_fork_prefix_meta(prev, *args)),
    }


COPY_KERNEL = "bitwise_not"  # the calibration copy: dst = ~src, one read and one write per byte
ATTN_KERNEL = "attn_kernel"


def _counter_rows(path, counter):
    import csv

    with open(path, newline="") as f:
        return [r for r in csv.DictReader(f) if r["Counter_Name"] == counter]


def ingest_traffic(args):
    """HBM bytes per attention launch from FETCH_SIZE / WRITE_SIZE counter runs.

    Each counter (KiB per dispatch) is scaled by bytes / counter of the plain
    copy kernel of ``--copy-mib`` MiB (read once, written once) recorded in
    the same run, then averaged over every attention dispatch."""
    if args.copy_mib <= 0:
        raise SystemExit("--ingest-traffic needs the --copy-mib the counter runs used")
    copy_kib = args.copy_mib * 1024.0
    rec = {"kernel_sha": kernel_sha(), "entries": {}}
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            old = json.load(f)
        if old.get("kernel_sha") == rec["kernel_sha"]:
            rec = old
    ent = {"copy_mib": args.copy_mib}
    total = 0.0
    for path, counter in zip(args.ingest_traffic, ("FETCH_SIZE", "WRITE_SIZE")):
        rows = _counter_rows(path, counter)
        attn = [float(r["Counter_Value"]) for r in rows if ATTN_KERNEL in r["Kernel_Name"]]
        copy = [float(r["Counter_Value"]) for r in rows if COPY_KERNEL in r["Kernel_Name"]
                and int(r["Grid_Size"]) > 0]
        if not attn or not copy:
            raise SystemExit(f"{path}: no {ATTN_KERNEL} or {COPY_KERNEL} dispatches with {counter}")
        copy_kib_meas = copy[-1]  # the last copy dispatches are the calibration copies
        factor = copy_kib / copy_kib_meas
        kib = float(np.mean(attn))
        ent[counter.lower()] = {"attn_kib_mean": kib, "attn_dispatches": len(attn), "copy_kib": copy_kib_meas,
                                "factor": factor}
        total += kib * factor * 1024.0
    ent["bytes_per_launch"] = total
    rec["entries"][f"{args.config}:{args.variant}"] = ent
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(ent))


def main():
    args = parse()
    if args.ingest_traffic:
        ingest_traffic(args)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no multi-GPU path",
              file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2509_00195_amd import tts as T
    from paper_2509_00195_amd.runner import PagedAttention, PrefixAttention
    from tts_synth import CONFIGS, make_workload
    from tts_synth.device import to_device

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = CONFIGS[args.config]
    wl = make_workload(cfg, args.seed, poison=False)
    sh = wl.shape
    x = to_device(wl, dev)
    # All work runs on one non-default stream (graph capture needs one);
    # the timing events are recorded on it too.
    stream = torch.cuda.Stream(device=dev)
    torch.cuda.set_stream(stream)

    t0 = time.perf_counter()
    pref = PrefixAttention(x, wl.req_seq_offsets, wl.block_tables, wl.seq_lens, wl.num_blocks, stream=stream)
    meta_ms = (time.perf_counter() - t0) * 1e3
    meta_warm = meta_timings(wl, pref.desc, pref.meta) if args.q_len <= 1 else None
    view = pref.meta.export()
    units, slots = pref.meta.stats()
    eb = {"f32": 4, "bf16": 2, "fp8": 1}[sh.kv_dtype]
    unique_kv = view["unique_tokens"] * sh.num_kv_heads * sh.head_dim * 2 * eb
    if sh.kv_dtype == "fp8":
        unique_kv += view["unique_blocks"] * 8
    logical_tokens = int(wl.seq_lens.sum())
    logical_kv = logical_tokens * sh.num_kv_heads * sh.head_dim * 2 * eb
    paged = PagedAttention(x, wl.max_seq_len, wl.num_blocks)

    pool_bytes = sum(t.numel() * t.element_size() for t in (x.k_cache, x.v_cache))
    layers = max(args.layers, min(512, -(-2 * 256 * 2 ** 20 // max(pool_bytes, 1))))
    pools = make_layers(wl, x, layers, args.seed)
    out = pref.out
    qlen = max(1, args.q_len)
    if qlen > 1:
        if args.variant != "prefix":
            raise SystemExit("--q-len needs the prefix variant")
        vmeta = T.tts_build_verify_meta(wl.req_seq_offsets, wl.block_tables, wl.seq_lens, qlen, 16, wl.num_blocks,
                                        desc=pref.desc, stream=stream)
        vws_bytes = T.tts_prefix_decode_workspace_size(pref.desc, vmeta)
        vws = torch.zeros(max(vws_bytes, 1), dtype=torch.uint8, device=dev)
        out = torch.zeros((wl.num_seqs, qlen, sh.num_q_heads, sh.head_dim), dtype=torch.float32, device=dev)
        gq = torch.Generator(device=dev)
        gq.manual_seed(2000 + args.seed)
        qv = torch.randn((wl.num_seqs, qlen, sh.num_q_heads, sh.head_dim), generator=gq, device=dev)
        qv = qv if sh.q_dtype == "f32" else qv.to(torch.bfloat16)
        units, slots = vmeta.stats()
    tabs, lens = x.block_tables, x.seq_lens
    maxb = int(tabs.shape[1])

    # One rotation for every phase below: step i uses pool i mod L, and every
    # phase continues from the last index, so a pool comes back only after
    # the other L - 1 (at least twice the 256 MB cache of traffic).
    rot = [0]

    def step(i, partials_only=False):
        q, k, v, ks, vs = pools[i % len(pools)]
        if qlen > 1:
            fn = T.tts_prefix_decode_partials if partials_only else T.tts_prefix_verify_attn
            fn(pref.desc, vmeta, qv, k, v, ks, vs, tabs, maxb, lens, wl.num_blocks, out, vws, vws_bytes, stream)
        elif args.variant == "prefix":
            fn = T.tts_prefix_decode_partials if partials_only else T.tts_prefix_decode_attn
            fn(pref.desc, pref.meta, q, k, v, ks, vs, tabs, maxb, lens, wl.num_blocks, out, pref.ws, pref.ws_bytes,
               stream)
        else:
            T.tts_paged_decode_attn(paged.desc, wl.num_seqs, q, k, v, ks, vs, tabs, maxb, lens, wl.max_seq_len,
                                    wl.num_blocks, out, paged.ws, paged.ws_bytes, stream)

    # Layer 0's output, for the comparison with the oracle (layer 0 holds the
    # generator's inputs, the ones the oracle sees).
    out0 = None
    if not args.no_check and qlen == 1:
        step(0)
        torch.cuda.synchronize()
        out0 = out.cpu().numpy().copy()
    rot[0] = 1

    def steps(n, partials_only=False):
        for _ in range(n):
            step(rot[0], partials_only)
            rot[0] += 1

    steps(args.warmup)
    torch.cuda.synchronize()

    graph = None
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=stream):
            steps(len(pools))
        graph.replay()
        torch.cuda.synchronize()

    def timed(fn, n):
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        fn(n)
        end.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(end)

    # The step: one full call (all launches) per layer, rotating layers.
    if graph is not None:
        reps = max(1, args.steps // len(pools))
        ms = timed(lambda n: [graph.replay() for _ in range(n)], reps)
        nsteps = reps * len(pools)
    else:
        ms = timed(steps, args.steps)
        nsteps = args.steps
    ms_per_step = ms / nsteps
    value = wl.num_seqs * qlen / (ms_per_step * 1e-3)

    # For reference: the same calls replayed from one captured HIP graph per
    # rotation of the layer pools (what a serving loop that captures its
    # decode step would see); `value` stays the eager rate.
    graph_call_us = ms_per_step * 1e3 if graph is not None else None
    if graph is None:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            steps(len(pools))
        g.replay()
        reps = max(1, args.steps // len(pools))
        graph_call_us = timed(lambda n: [g.replay() for _ in range(n)], reps) * 1e3 / (reps * len(pools))
        del g

    # The dominant kernel alone (the attention work units of each call), same
    # rotation, events on the stream it runs on.
    if args.variant == "prefix":
        kms = timed(lambda n: steps(n, partials_only=True), args.steps) / args.steps
    else:
        kms = ms_per_step
    kv_bytes = unique_kv if args.variant == "prefix" else logical_kv
    achieved = kv_bytes / (kms * 1e-3) / 1e9

    # The KV steps around the call, on layer 0's pool: appending every beam's
    # token (tts_append_kv) and the copy-on-write copies of a duplication
    # step (tts_copy_blocks, one partial block per beam).
    q0, k0, v0, ks0, vs0 = pools[0]
    kv_src = torch.zeros((wl.num_seqs, sh.num_kv_heads, sh.head_dim),
                         dtype=torch.float32 if sh.kv_dtype == "f32" else torch.bfloat16, device=dev)
    kv_src.normal_()
    # (Timed as replays of a captured HIP graph of 50 calls: eager, each call
    # is bound by the host's launch path, not by the GPU.)
    def graph_ms(call, reps=50):
        call()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for _ in range(reps):
                call()
        g.replay()
        return timed(lambda n: [g.replay() for _ in range(n)], 4) / (4 * reps)

    append_ms = graph_ms(lambda: T.tts_append_kv(pref.desc, wl.num_seqs, kv_src, kv_src, tabs, maxb, lens,
                                                 wl.num_blocks, k0, v0, ks0, vs0, stream))
    used = set()
    src_ids = []
    for b in range(wl.num_seqs):
        nblk = -(-int(wl.seq_lens[b]) // 16)
        used.update(wl.block_tables[b, :nblk].tolist())
        src_ids.append(int(wl.block_tables[b, max(nblk - 1, 0)]))
    spare = [i for i in range(wl.num_blocks) if i not in used][: wl.num_seqs]
    pairs = torch.tensor(list(zip(src_ids, spare)), dtype=torch.int32, device=dev).reshape(-1, 2).contiguous()
    copy_ms = graph_ms(lambda: T.tts_copy_blocks(pref.desc, int(pairs.shape[0]), pairs, wl.num_blocks, k0, v0, ks0,
                                                 vs0, stream))

    # Streaming calibration on the same GPU: an elementwise copy of 1 GiB
    # (dst = ~src), one read and one write per byte, timed the same way.
    csrc = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
    cdst = torch.empty_like(csrc)
    torch.bitwise_not(csrc, out=cdst)
    cms = timed(lambda n: [torch.bitwise_not(csrc, out=cdst) for _ in range(n)], 20) / 20
    stream_gbs = 2.0 * csrc.numel() / (cms * 1e-3) / 1e9
    del csrc, cdst
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        key = f"{args.config}:{args.variant}"
        if tr.get("kernel_sha") == kernel_sha() and key in tr.get("entries", {}):
            traffic = tr["entries"][key]["bytes_per_launch"]

    rec = {
        "metric": METRIC,
        "value": value,
        "unit": "beam-tokens/s" if qlen == 1 else "query-tokens/s",
        "n_gpus": 1,
        "steps": nsteps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if sh.kv_dtype in ("bf16", "fp8") else "f32",
        "data": "synthetic (seeded beam-search tree; random K/V/Q)",
        "config": {
            "workload": f"{args.config}: {cfg.description}",
            "seed": args.seed,
            "variant": args.variant,
            "kv_dtype": sh.kv_dtype,
            "beams": wl.num_seqs,
            "layers_rotated": len(pools),
            "layer_pool_bytes": int(pool_bytes),
            "graph_replay": bool(args.graph),
            "graph_call_us": graph_call_us,
            "q_len": qlen,
            "unique_kv_bytes": int(unique_kv),
            # per call, beside the KV bytes: queries read, outputs written, the block-table rows the
            # kernels read (the metadata's own buffer aside)
            "q_bytes": int(wl.num_seqs * qlen * sh.num_q_heads * sh.head_dim * (4 if sh.q_dtype == "f32" else 2)),
            "out_bytes": int(wl.num_seqs * qlen * sh.num_q_heads * sh.head_dim * 4),
            "table_bytes": int(wl.block_tables.size * 4 + wl.num_seqs * 4),
            "logical_kv_bytes": int(logical_kv),
            "sharing": logical_kv / max(unique_kv, 1),
            "unique_kv_hbm_frac_per_call": unique_kv / (ms_per_step * 1e-3) / (HBM_PEAK_GBS * 1e9),
            "stream_copy_gbs": stream_gbs,
            "append_kv_us": append_ms * 1e3,
            "copy_blocks_us": copy_ms * 1e3,
            "attention_frac_of_stream_copy": achieved / stream_gbs,
            "attention_kernel_us": kms * 1e3,
            "merge_and_gaps_us": (ms_per_step - kms) * 1e3,
            "per_28_layer_step_beam_tokens_per_s": value / 28.0,
            "work_units": units,
            "partial_slots": slots,
            "meta_first_build_ms": meta_ms,
            "meta_warm_ms": meta_warm,
            "max_abs_err_vs_oracle": None,
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "attn_kernel (work units of tts_prefix_decode_partials)" if args.variant == "prefix"
                      else "attn_kernel + merge_kernel (tts_paged_decode_attn)",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "frac_per_call": kv_bytes / (ms_per_step * 1e-3) / (HBM_PEAK_GBS * 1e9),
        },
    }
    if args.copy_mib > 0:
        src = torch.ones(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.bitwise_not(src, out=dst)
        torch.cuda.synchronize()
    ref = None
    if not args.no_cpu_baseline:
        rec["cpu_baseline"], ref = cpu_baseline(wl, args.cpu_seconds)
    if out0 is not None:
        if ref is None:
            from oracle.attention import oracle_attn_workload

            ref = oracle_attn_workload(wl)
        rec["config"]["max_abs_err_vs_oracle"] = float(np.max(np.abs(out0.astype(np.float64) - ref)))
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
