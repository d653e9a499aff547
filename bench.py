"""Benchmark of the evidence-retrieval hot path on one MI355X.

One step = one ss_retrieve call over the whole workload (query prep, sampled
cut-off, the streaming MFMA scoring pass over every stored key, exact top-k,
votes, pool and max-min), with the index already resident in HBM.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config C4]

Prints one JSON line.  ``value`` is key vectors scored per second (a key vector
is one stored d-dim bf16 row at one (layer, KV head); each is scored against
its G query heads).  ``roofline`` covers the streaming scoring kernel, timed
with HIP events recorded around it on the call's stream.  ``cpu_baseline`` is
the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

HBM_PEAK_GBS = 8000.0
METRIC = "index keys scored/sec + % HBM roofline; p50 ss_retrieve latency, 1-hour index"
KERNEL_SRC = os.path.join(ROOT, "paper_2609_02780_amd", "csrc", "ss_kernels.hip")
# committed PMC summaries of the streaming kernel per (workload, score mode)
TRAFFIC_FILES = {("C4", 0): "k_stream_c4_traffic.md", ("C5", 0): "k_stream_c5_traffic.md",
                 ("P4", 0): "k_stream_hm_p4_traffic.md", ("P4", 1): "k_stream_hp_p4_traffic.md"}
HOT_KERNEL = "k_stream<128>"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_hash() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def stored_traffic(cfg_name: str, score_mode: int):
    """HBM bytes per launch of the hot kernel from the committed PMC summary of
    this workload, if there is one and it was taken on the current kernel
    source; else None."""
    name = TRAFFIC_FILES.get((cfg_name, score_mode))
    path = os.path.join(ROOT, "profiles", name) if name else None
    if path is None or not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"kernel source sha256\[:16\]:\s*([0-9a-f]{16})", text)
    m_bytes = re.search(r"HBM bytes per launch:\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != kernel_hash():
        return None
    return float(m_bytes.group(1))


def dev_bf16(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def build_streams(torch, P, cfg, block=600):
    """Generate and append every stream of the workload; returns the indices, the
    per-stream device queries and stream 0's queries and host key blocks (for the
    CPU baseline)."""
    specs = W.stream_specs(cfg)
    idxs, queries, host0 = [], [], None
    t0 = time.time()
    for spec in specs:
        q = W.make_queries(cfg, 0, spec.stream)
        T = cfg.tokens_per_frame
        rpf = T if spec.compress is None else min(spec.compress[0], T)
        idx = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, spec.n_frames,
                             spec.n_frames * rpf)
        blocks = []
        for f0 in range(0, spec.n_frames, block):
            f1 = min(spec.n_frames, f0 + block)
            kb = W.frame_block_keys(cfg, spec, q, f0, f1)
            idx.append([dev_bf16(torch, k) for k in kb], f1 - f0, T, spec.compress)
            if spec.stream == 0:
                blocks.append((kb, f1 - f0))
            torch.cuda.synchronize()
        if spec.stream == 0:
            host0 = (q, blocks, spec.compress)
        idxs.append(idx)
        queries.append([dev_bf16(torch, x) for x in q])
        log(f"stream {spec.stream}: {spec.n_frames} frames appended ({time.time() - t0:.1f} s)")
    return specs, idxs, queries, host0


def time_append(torch, P, cfg, frames=64):
    """Compressed append latency: one frame at a time and one batch of frames."""
    spec = W.stream_specs(cfg)[0]
    q = W.make_queries(cfg, 0, 0)
    T = cfg.tokens_per_frame
    kb = W.frame_block_keys(cfg, spec, q, 0, frames)
    dev = [dev_bf16(torch, k) for k in kb]
    n_c = spec.compress[0] if spec.compress else T
    idx = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, 4 * frames, 4 * frames * n_c)
    one = [d[:, :T, :].contiguous() for d in dev]
    for _ in range(3):
        idx.append(one, 1, T, spec.compress)
    torch.cuda.synchronize()
    lat = []
    for _ in range(frames):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        idx.append(one, 1, T, spec.compress)
        b.record()
        b.synchronize()
        lat.append(a.elapsed_time(b))
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    idx.append(dev, frames, T, spec.compress)
    b.record()
    b.synchronize()
    batch_ms = a.elapsed_time(b)
    return {"per_frame_p50_ms": float(np.median(lat)), "batch_frames": frames,
            "batch_frames_per_s": frames / (batch_ms / 1e3)}


def timed_calls(torch, r, queries, calls, kernel=None):
    """Per-call times in ms from HIP events: around each whole call, or (with
    `kernel`, the package) around its streaming kernel, recorded by the library
    on the call's stream.  The calls are queued back to back."""
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(calls)]
    for e2 in ev:   # torch reads elapsed times only of events it has recorded once
        for e in e2:
            e.record()
    torch.cuda.synchronize()
    for a, b in ev:
        if kernel is not None:
            kernel.set_profile_events(a, b)
            r(queries)
        else:
            a.record()
            r(queries)
            b.record()
    if kernel is not None:
        kernel.set_profile_events(None, None)
    torch.cuda.synchronize()
    return np.array([a.elapsed_time(b) for a, b in ev])


def time_serving(torch, P, idxs, queries, cfg, score_mode, key_vectors, key_bytes, want_ids, calls=100):
    """Two queries in flight, as a serving loop may keep them: two retrievers
    (each its own workspace and outputs) take the calls in turn on two HIP
    streams of default priority, so one call's small kernels can run beside the
    other's streaming pass.  Whole-loop wall time per call; every call's frame
    ids must equal the single-stream call's."""
    rs = [P.Retriever(idxs, cfg.top_k, cfg.n_select, cfg.pool_mult, cfg.head_mode, score_mode) for _ in range(2)]
    sts = [torch.cuda.Stream(), torch.cuda.Stream()]
    for i in range(4):
        rs[i % 2](queries, stream=sts[i % 2])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(calls):
        rs[i % 2](queries, stream=sts[i % 2])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for r2 in rs:
        if not torch.equal(r2.frame_ids, want_ids):
            raise RuntimeError("a two-stream call's frame ids differ from the single-stream call's")
    ms = (t1 - t0) * 1e3 / calls
    return {"streams": 2, "calls": calls, "ms_per_call": ms, "keys_per_s": key_vectors / (ms / 1e3),
            "hbm_frac": key_bytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS}


def time_cold(torch, P, r, queries, key_bytes, calls=20, scratch_bytes=512 << 20):
    """Cold-cache retrieval: before each call a 512 MB scratch buffer is written,
    which evicts the index from L2 and the 256 MB Infinity Cache; the call and its
    streaming kernel are timed with HIP events (the scratch writes are outside)."""
    scratch = torch.empty(scratch_bytes // 4, dtype=torch.int32, device="cuda")
    lat, hot = [], []
    for i in range(calls + 2):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        for x in e:   # torch reads elapsed times only of events it has recorded once
            x.record()
        scratch.fill_(i)
        P.set_profile_events(e[2], e[3])
        e[0].record()
        r(queries)
        e[1].record()
        P.set_profile_events(None, None)
        torch.cuda.synchronize()
        if i >= 2:
            lat.append(e[0].elapsed_time(e[1]))
            hot.append(e[2].elapsed_time(e[3]))
    del scratch
    hot_ms = float(np.mean(hot))
    return {"p50_latency_ms": float(np.percentile(lat, 50)), "p10_latency_ms": float(np.percentile(lat, 10)),
            "p90_latency_ms": float(np.percentile(lat, 90)), "avg_kernel_ms": hot_ms,
            "kernel_gbs": key_bytes / (hot_ms / 1e3) / 1e9, "calls": calls,
            "scratch_bytes": scratch_bytes}


def time_evidence(torch, P, idxs, frame_ids, calls=20):
    """Evidence assembly after the retrieval, with the paper's settings: 6
    recent units and one preceding unit per selected unit."""
    for _ in range(3):
        P.assemble_evidence(idxs, frame_ids, 6, 1, 0, True)
    torch.cuda.synchronize()
    lat = []
    for _ in range(calls):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        units, _, n_units = P.assemble_evidence(idxs, frame_ids, 6, 1, 0, True)
        b.record()
        b.synchronize()
        lat.append(a.elapsed_time(b))
    return {"p50_ms": float(np.median(lat)), "n_recent": 6, "n_before": 1, "n_after": 0,
            "units_stream0": int(n_units[0].item())}


def sweep(torch, P, cfg, points=(64, 128, 256, 512, 1024, 2048, 3600), calls=20):
    """History-length sweep on one growing stream of the workload's shape: at
    each length the token-vote retrieval (with its streaming kernel), the
    pooled Q-K ranker and the evidence assembly are timed with HIP events."""
    spec = W.stream_specs(cfg)[0]
    q = W.make_queries(cfg, 0, 0)
    T = cfg.tokens_per_frame
    F_max = max(points)
    spec = W.StreamSpec(0, F_max, cfg.n_planted, None, W.planted_frames(F_max, cfg.n_planted))
    idx = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, F_max, F_max * T)
    qd = [[dev_bf16(torch, x) for x in q]]
    r = P.Retriever([idx], cfg.top_k, cfg.n_select, cfg.pool_mult)
    pr = P.PooledRanker([idx], cfg.n_select)

    def timed(fn, with_kernel=False):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(calls)]
        for e4 in ev:            # torch times only events it has recorded once itself
            for e in e4:
                e.record()
        torch.cuda.synchronize()
        for e4 in ev:
            if with_kernel:
                P.set_profile_events(e4[2], e4[3])
            e4[0].record()
            fn()
            e4[1].record()
        torch.cuda.synchronize()
        P.set_profile_events(None, None)
        lat = float(np.median([e[0].elapsed_time(e[1]) for e in ev]))
        ker = float(np.median([e[2].elapsed_time(e[3]) for e in ev])) if with_kernel else None
        return lat, ker

    def graph_ms(fn, outs):
        """GPU time of one call replayed from a HIP graph (no host launch
        overhead); the replays' outputs must equal the eager call's."""
        fn()
        torch.cuda.synchronize()
        want = [o.clone() for o in outs]
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            fn()
        for _ in range(3):
            g.replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(calls):
            g.replay()
        b.record()
        b.synchronize()
        for o, w in zip(outs, want):
            if not torch.equal(o, w):
                raise RuntimeError("graph replay differs from the eager call")
        return a.elapsed_time(b) / calls

    # long-history compression on: a second index keeps the newest 6 frames as
    # recent context and the 512 before them in detail; older frames leave into
    # long-term clusters as the stream grows
    n_recent, n_detail, tau = 6, 512, 0.1
    lidx = P.ShallowIndex(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, F_max, F_max * T, n_recent)
    lcl = P.LongClusters(lidx, T, 4096, tau)
    lr = P.Retriever([lidx], cfg.top_k, cfg.n_select, cfg.pool_mult)
    absorbed, absorb_ms = 0, []

    rows = []
    have = 0
    for F in points:
        while have < F:
            f1 = min(F, have + 600)
            kb = W.frame_block_keys(cfg, spec, q, have, f1)
            idx.append([dev_bf16(torch, k) for k in kb], f1 - have, T)
            lidx.append([dev_bf16(torch, k) for k in kb], f1 - have, T)
            have = f1
        torch.cuda.synchronize()
        hi = max(0, F - n_recent - n_detail)
        if hi > absorbed:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            lcl.absorb(hi, hi - absorbed)
            b.record()
            b.synchronize()
            absorb_ms.append((a.elapsed_time(b), hi - absorbed))
            absorbed = hi
        lat, ker = timed(lambda: r(qd), with_kernel=True)
        plat, _ = timed(lambda: pr(qd))
        elat, _ = timed(lambda: P.assemble_evidence([idx], r.frame_ids, 6, 1, 0, True))
        llat, lker = timed(lambda: lr(qd), with_kernel=True)
        clat, _ = timed(lambda: lcl.retrieve(qd[0], 4))
        n_clusters = lcl.export()["n_clusters"] if absorbed else 0
        glat = graph_ms(lambda: r(qd), [r.frame_ids, r.votes, r.n_out])
        gplat = graph_ms(lambda: pr(qd), [pr.frame_ids, pr.n_out])
        key_bytes = idx.n_rows * cfg.n_layers * cfg.n_kv_heads * cfg.head_dim * 2
        rows.append({"frames": F, "key_bytes": key_bytes, "retrieve_p50_ms": lat, "retrieve_graph_ms": glat,
                     "stream_kernel_ms": ker, "stream_kernel_gbs": key_bytes / (ker / 1e3) / 1e9,
                     "pooled_p50_ms": plat, "pooled_graph_ms": gplat, "evidence_p50_ms": elat,
                     "lc_detailed_frames": F - absorbed - min(F, n_recent), "lc_retrieve_p50_ms": llat,
                     "lc_stream_kernel_ms": lker, "lc_clusters": n_clusters, "lc_cluster_retrieve_p50_ms": clat})
        log(f"{F} frames: retrieve {lat:.3f} ms (graph {glat:.3f}, kernel {ker:.3f}), "
            f"pooled {plat:.3f} ms (graph {gplat:.3f}), evidence {elat:.3f} ms; "
            f"compression on: retrieve {llat:.3f} ms over {F - absorbed - min(F, n_recent)} detailed frames, "
            f"{n_clusters} clusters ranked in {clat:.3f} ms")
    per_frame = [ms / n for ms, n in absorb_ms]
    log("absorb ms per frame", [round(x, 4) for x in per_frame])
    return rows, {"n_recent": n_recent, "n_detail": n_detail, "tau": tau,
                  "absorb_ms_per_frame": per_frame}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def hot_kernel(cfg, score_mode: int) -> str:
    """The streaming scoring kernel of the workload's mode."""
    if cfg.head_mode == 0:
        return HOT_KERNEL
    if score_mode == 1:
        return f"k_stream_hp<{cfg.head_dim}, {cfg.n_kv_heads}>"
    return f"k_stream_hm<{cfg.head_dim}>"


def cpu_baseline(cfg, host0, score_mode: int = 0):
    """The oracle's retrieval over stream 0 of the workload, with its queries and
    retrieval parameters, every frame of the stream.  A compressed stream keeps,
    per frame, its first n_centroids token rows as the stored rows: the same
    number of rows the centroids would fill, so the same retrieval work, without
    the oracle's float64 k-means (append work, outside the timed retrieval).
    Runs of under 3 s are repeated and the median of three is reported."""
    from oracle import oracle as O
    q, blocks, comp = host0
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = 1
    oi = O.Index(cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim)
    T = cfg.tokens_per_frame
    if comp is None:
        for kb, nf in blocks:
            oi.append(kb, nf, T)
        what = f"all {oi.n_frames} frames"
    else:
        rpf = min(comp[0], T)
        for kb, nf in blocks:
            rows = [np.concatenate([k[:, f * T:f * T + rpf, :] for f in range(nf)], axis=1) for k in kb]
            descs = [O.descriptor(O.decode_bf16(kb[-1][:, f * T:(f + 1) * T, :])) for f in range(nf)]
            oi.append_stored(rows, [rpf] * nf, descs)
        what = (f"all {oi.n_frames} frames, {rpf} stored rows each (the frame's first {rpf} token rows "
                f"in place of its k-means centroids)")
    times = []
    while True:
        t0 = time.perf_counter()
        O.retrieve(oi, q, cfg.top_k, cfg.n_select, cfg.pool_mult, cfg.head_mode, score_mode=score_mode)
        times.append(time.perf_counter() - t0)
        if times[0] >= 3.0 or len(times) == 3:
            break
    dt = float(np.median(times))
    keys = oi.n_rows * cfg.n_layers * cfg.n_kv_heads
    return {"value": keys / dt, "unit": "keys/s", "cores": int(cores), "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"float64 oracle retrieval (scores, top-k, votes, pool, max-min) over {what} "
                      f"({oi.n_rows} rows per (layer, KV head)) of stream 0 of {cfg.name} with its queries "
                      f"and parameters: {keys} key vectors in {dt:.2f} s "
                      f"({'median of ' + str(len(times)) + ' runs' if len(times) > 1 else 'one run'})"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--samples", type=int, default=20,
                    help="calls timed one by one with HIP events (latency percentiles, streaming kernel)")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="C4", choices=sorted(W.CONFIGS))
    ap.add_argument("--score-mode", type=int, default=0, choices=(0, 1),
                    help="list values: 0 scaled logits (the workloads' default), 1 attention probabilities")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--serving", action="store_true",
                    help="also time two queries in flight on two streams (serving_two_streams)")
    ap.add_argument("--cold", action="store_true",
                    help="also time cold-cache calls (on by default for indices of at most 1 GiB)")
    ap.add_argument("--sweep", action="store_true",
                    help="history-length sweep (64..3600 frames of the workload's shape) instead of the benchmark")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (calibrates the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the retrieval has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.calibrate_copy:
        # a plain copy of known size: 2^30 bytes read and 2^30 bytes written
        torch.cuda.set_device(0)
        a = torch.ones(1 << 28, dtype=torch.int32, device="cuda")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes": 1 << 30}), flush=True)
        return

    import paper_2609_02780_amd as P
    if not os.path.exists(P._lib.LIB_PATH):
        from paper_2609_02780_amd.build import build_library
        build_library()
    torch.cuda.set_device(0)
    cfg = W.CONFIGS[args.config]
    if args.sweep:
        rows, lc = sweep(torch, P, cfg)
        print(json.dumps({"sweep": "history length", "workload": cfg.name, "top_k": cfg.top_k,
                          "n_select": cfg.n_select, "data": "synthetic", "points": rows,
                          "long_history_compression": lc}), flush=True)
        return
    specs, idxs, queries, host0 = build_streams(torch, P, cfg)
    r = P.Retriever(idxs, cfg.top_k, cfg.n_select, cfg.pool_mult, cfg.head_mode, args.score_mode)
    for _ in range(args.warmup):
        r(queries)
    torch.cuda.synchronize()

    # the timed steps run back to back with no event between them, as a serving
    # loop would (a HIP event costs about 5 us of stream time); the latency
    # percentiles and the streaming kernel's time come from separate passes of
    # `samples` calls, each bracketed by its own events
    K = args.steps
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        r(queries)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    lat = timed_calls(torch, r, queries, args.samples)
    hot = timed_calls(torch, r, queries, args.samples, kernel=P)

    rows = [x.n_rows for x in idxs]
    key_vectors = sum(x.n_rows for x in idxs) * cfg.n_layers * cfg.n_kv_heads
    key_bytes = key_vectors * cfg.head_dim * 2
    ms_per_step = (t1 - t0) * 1e3 / K
    value = key_vectors / (ms_per_step / 1e3)
    achieved = key_bytes / (hot.mean() / 1e3) / 1e9
    traffic = stored_traffic(cfg.name, args.score_mode)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "keys/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.description}; {cfg.n_layers} shallow layers, "
                               f"{cfg.n_q_heads} query / {cfg.n_kv_heads} KV heads, d={cfg.head_dim}, "
                               f"{cfg.n_q} query tokens, top-k {cfg.top_k}, {cfg.n_select} frames selected"
                               + (", head-averaged lists" if cfg.head_mode else "")
                               + (", attention probabilities" if args.score_mode else ""),
                   "streams": len(idxs), "rows_per_layer_kv_head": rows, "key_vectors": key_vectors,
                   "key_bytes": key_bytes},
        "p10_latency_ms": float(np.percentile(lat, 10)),
        "p50_latency_ms": float(np.percentile(lat, 50)),
        "p90_latency_ms": float(np.percentile(lat, 90)),
        "scores_per_s": value * cfg.group,
        "hbm_frac_end_to_end": key_bytes / (np.percentile(lat, 50) / 1e3) / 1e9 / HBM_PEAK_GBS,
        "roofline": {"kernel": hot_kernel(cfg, args.score_mode), "bound": "hbm", "achieved": achieved,
                     "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "avg_kernel_ms": float(hot.mean()), "bytes_per_launch": key_bytes,
                     "event_samples": len(hot)},
    }
    if args.serving:
        out["serving_two_streams"] = time_serving(torch, P, idxs, queries, cfg, args.score_mode, key_vectors,
                                                  key_bytes, r.frame_ids.clone())
    out["evidence"] = time_evidence(torch, P, idxs, r.frame_ids)
    if args.cold or key_bytes <= (1 << 30):   # indices that a warm Infinity Cache could hold
        out["cold"] = time_cold(torch, P, r, queries, key_bytes)
    if cfg.compress is not None:
        out["append"] = time_append(torch, P, cfg)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, host0, args.score_mode)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
