#!/usr/bin/env python3
"""Benchmark of the LSA hot path on one MI355X.

One step = the whole hot path over one synthetic single-sequence prefill of L = 131072 tokens:
block cache (lsa_block_means, or lsa_block_minmax with --pooling minmax), hierarchical indexer with streaming merge and runs
(lsa_index_prefill), then sparse attention for the 4 layers of one cross-layer group, all reading
the same index list (lsa_sparse_attn x 4). Inputs are resident in HBM before timing starts.

Prints one JSON line: tokens/s of the whole step, a roofline entry for the dominant kernel
(sparse attention: algorithmic bytes per launch over its HIP-event duration against 8 TB/s), the
indexer's MFMA fraction, and the float64 oracle timed on the host's cores over a bounded sample.
Diagnostics go to stderr.
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
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2608_01662_amd import lsa, synth  # noqa: E402
from paper_2608_01662_amd import workloads as W  # noqa: E402

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "mla_attn_kernel_L131072_hbm_traffic.txt")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_01662_amd", "csrc", f) for f in ("attention.hip", "device.hpp")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """SHA-256 of the attention kernel's sources with comments and blank lines removed (so that
    an edit of the comments alone keeps the committed traffic figure valid), and of the extra
    compiler flags of attention.hip."""
    from paper_2608_01662_amd.build import EXTRA_FLAGS
    h = hashlib.sha256()
    h.update((" ".join(EXTRA_FLAGS.get("attention.hip", [])) + "\n").encode())
    for f in KERNEL_SOURCES:
        with open(f) as fh:
            text = re.sub(r"/\*.*?\*/", "", fh.read(), flags=re.S)
        for line in text.splitlines():
            code = line.split("//", 1)[0].rstrip()
            if code:
                h.update((code + "\n").encode())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per attention launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary,
    or None when that summary is missing, was taken on another workload or on different kernel
    sources."""
    try:
        kv = {}
        with open(TRAFFIC_FILE) as fh:
            for line in fh:
                if ":" in line and not line.startswith("#"):
                    k, v = line.split(":", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("workload") != workload or kv.get("kernel_sources_sha256") != kernel_source_hash():
            return None
        return int(kv["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def copy_probe(nbytes: int):
    """A plain device copy of known size, run under rocprofv3 --pmc to calibrate FETCH_SIZE and
    WRITE_SIZE (each copy reads and writes exactly nbytes)."""
    dev = torch.device("cuda:0")
    src = torch.ones(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes, "copies": 3}), flush=True)


def gather_probe(n_rows: int, table_rows: int):
    """Random-row gather of known size, shaped like the attention's KV reads, run under rocprofv3
    --pmc to check the FETCH_SIZE calibration on scattered 1152-byte rows: n_rows rows of 576 bf16
    (1152 bytes) drawn at random from a table of table_rows rows (torch.index_select: every
    gathered row is read once and written once)."""
    dev = torch.device("cuda:0")
    table = torch.ones((table_rows, 576), dtype=torch.bfloat16, device=dev)
    g = torch.Generator(device=dev)
    g.manual_seed(1234)
    idx = torch.randint(0, table_rows, (n_rows,), generator=g, device=dev)
    out = torch.empty((n_rows, 576), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.index_select(table, 0, idx, out=out)
    torch.cuda.synchronize()
    print(json.dumps({"gather_probe_rows": n_rows, "row_bytes": 1152, "table_rows": table_rows,
                      "gathered_bytes": n_rows * 1152, "index_bytes": n_rows * 8,
                      "table_bytes": table_rows * 1152, "gathers": 3}), flush=True)


def index_sweep(lengths, pooling):
    """Indexer time of one whole prefill (every row) at each cache length, hierarchical (the
    benchmark workload's M and P) against flat (dense causal scoring of every eligible token): the
    measurement behind the adaptive dispatch length hi_min_kv. One JSON line per length."""
    from dataclasses import replace
    dev = torch.device("cuda:0")
    base = replace(W.L128K_CLI4, pooling=pooling)
    for L in lengths:
        w = replace(base, seq_len=L)
        qI = synth.device_normal_bf16((L, w.n_heads, w.head_dim), w.seed, synth.T_QI, dev,
                                      scale=1.0 / math.sqrt(w.head_dim))
        wI = synth.device_uniform_f32((L, w.n_heads), w.seed, synth.T_W, dev)
        kI, ks = synth.device_fp8_keys(L, w.head_dim, w.seed, dev)
        res = {"seq_len": L, "rows": L}
        for mode, keep in (("hierarchical", w.keep_pages), ("flat", 0)):
            prm = replace(w, keep_pages=keep).index_params()
            bk = lsa.block_keys(prm, kI, ks)
            out = lsa.index_prefill(prm, qI, wI, kI, ks, bk, 0, n_kv=L, runs=True)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(3):
                lsa.index_prefill(prm, qI, wI, kI, ks, bk, 0, n_kv=L, runs=True, out=out)
            e1.record()
            torch.cuda.synchronize()
            res[f"{mode}_ms"] = e0.elapsed_time(e1) / 3
            del out, bk
            torch.cuda.empty_cache()
        res["faster"] = "flat" if res["flat_ms"] < res["hierarchical_ms"] else "hierarchical"
        print(json.dumps(res), flush=True)
        del qI, wI, kI, ks
        torch.cuda.empty_cache()


def bench_decode(w, args):
    """Batched decode step: the indexer for one new token per sequence over the paged key cache
    (lsa_index_decode), then the paged sparse attention of each layer (lsa_sparse_attn). With
    --graph the step is captured once into a HIP graph (torch.cuda.CUDAGraph) and replayed, which
    removes the per-kernel launch cost of this small, launch-bound step. One JSON line."""
    dev = torch.device("cuda:0")
    prm, aprm = w.index_params(), w.attn_params()
    H, dqk, dv = w.attn_dims
    ctx, table, n_phys = synth.decode_layout(w.seed, w.batch, w.ctx_lo, w.ctx_hi, w.kv_page)
    n_tok = n_phys * w.kv_page
    B = w.batch
    log(f"[bench] {w.name}: {B} sequences, {n_tok} cached tokens in {n_phys} pages")
    qI = synth.device_normal_bf16((B, w.n_heads, w.head_dim), w.seed, synth.T_QI, dev, scale=1.0 / math.sqrt(w.head_dim))
    wI = synth.device_uniform_f32((B, w.n_heads), w.seed, synth.T_W, dev)
    kI, ks = synth.device_fp8_keys(n_tok, w.head_dim, w.seed, dev)
    bk = lsa.block_keys(prm, kI, ks)
    Q = [synth.device_normal_bf16((B, H, dqk), w.seed, synth.T_Q + l, dev) for l in range(w.layers)]
    KV = [synth.device_normal_bf16((n_tok, dqk), w.seed, synth.T_KV + l, dev).view(n_phys, w.kv_page, dqk)
          for l in range(w.layers)]
    ctx_d = torch.from_numpy(ctx).to(dev)
    table_d = torch.from_numpy(table).to(dev)
    out = dict(idx=torch.empty((B, w.k_cap), dtype=torch.int32, device=dev),
               count=torch.empty((B,), dtype=torch.int32, device=dev),
               runs=torch.empty((B, w.k_cap, 2), dtype=torch.int32, device=dev),
               run_count=torch.empty((B,), dtype=torch.int32, device=dev))
    ws_idx = torch.empty(max(1, lsa.index_workspace_size(prm, B, table.shape[1] * w.kv_page)), dtype=torch.uint8, device=dev)
    ws_attn = torch.empty(max(1, lsa.attn_workspace_size(aprm, B, w.k_cap, True)), dtype=torch.uint8, device=dev)
    O = [torch.empty((B, H, dv), dtype=torch.bfloat16, device=dev) for _ in range(w.layers)]
    LSE = [torch.empty((B, H), dtype=torch.float32, device=dev) for _ in range(w.layers)]

    def step():
        lsa.index_decode(prm, ctx_d, table_d, w.kv_page, n_phys, qI, wI, kI, ks, bk, runs=True, workspace=ws_idx,
                         out=out)
        for l in range(w.layers):
            lsa.sparse_attn(aprm, Q[l], KV[l], None, out["idx"], out["count"], page_table=table_d,
                            kv_page_size=w.kv_page, out=O[l], lse=LSE[l], workspace=ws_attn)

    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    # the two calls timed apart: each repeated back to back (steady state), on the library's stream
    def timed(fn, reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps
    idx_ms = timed(lambda: lsa.index_decode(prm, ctx_d, table_d, w.kv_page, n_phys, qI, wI, kI, ks, bk, runs=True,
                                            workspace=ws_idx, out=out), args.steps)
    attn_ms = timed(lambda: [lsa.sparse_attn(aprm, Q[l], KV[l], None, out["idx"], out["count"], page_table=table_d,
                                             kv_page_size=w.kv_page, out=O[l], lse=LSE[l], workspace=ws_attn)
                             for l in range(w.layers)], args.steps) / w.layers
    graph = None
    if args.graph:
        s_cap = torch.cuda.Stream()
        s_cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s_cap):
            step()                               # one more warm call on the capture stream
        torch.cuda.current_stream().wait_stream(s_cap)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
    run = graph.replay if graph is not None else step
    for _ in range(max(1, args.warmup)):
        run()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        run()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    cnt = out["count"].cpu().numpy().astype(np.int64)
    sum_s = int(cnt.sum())
    attn_bytes = sum_s * (dqk * 2 + 4) + B * H * (dqk + dv) * 2 + B * H * 4 + B * 4
    # indexer bytes per step: each sequence's block keys of its eligible pages (Eq. 9), the keys and
    # scales of its candidates on the recalled pages (Eq. 11), its query and weights, and idx/count/runs out
    t_pos = ctx.astype(np.int64) - 1
    hi_pos = t_pos - w.k_swa
    n_elig = np.where(hi_pos >= w.k_sink, hi_pos // w.page - w.k_sink // w.page + 1, 0)
    n_cand = np.where(hi_pos >= w.k_sink, np.minimum(n_elig, w.keep_pages) * w.page, 0)
    key_bytes = w.head_dim * (1 if w.fp8 else 2) + (4 if w.fp8 else 0)
    idx_bytes = int((n_elig * (w.page // w.sub_block) * prm.block_width * 2).sum() + (n_cand * key_bytes).sum()
                    + B * w.n_heads * (w.head_dim * 2 + 4) + B * w.k_cap * 12 + B * 8)
    attn_gbs = attn_bytes / (attn_ms * 1e-3) / 1e9
    res = {
        "metric": f"LSA decode tokens/s, {B} sequences of {w.ctx_lo // 1024}K-{w.ctx_hi // 1024}K context (indexer+attn)",
        "value": B / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "context": [int(ctx.min()), int(ctx.max())],
                   "kv_page": w.kv_page, "layers": w.layers, "hip_graph": bool(graph is not None),
                   "indexer": {"heads": w.n_heads, "head_dim": w.head_dim, "page": w.page, "keep_pages": w.keep_pages,
                               "k_sparse": w.k_sparse, "k_sink": w.k_sink, "k_swa": w.k_swa}},
        "roofline": {"kernel": "mla_attn_kernel (split over the list) + attn_combine_kernel", "bound": "hbm",
                     "achieved": attn_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": attn_gbs / HBM_PEAK_GBS,
                     "traffic": None, "algorithmic_bytes_per_launch": attn_bytes, "launch_ms": attn_ms},
        "breakdown": {"index_ms": idx_ms, "attn_ms_per_layer": attn_ms,
                      "index_algorithmic_bytes": idx_bytes, "index_hbm_gbs": idx_bytes / (idx_ms * 1e-3) / 1e9,
                      "index_hbm_frac": idx_bytes / (idx_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                      "mean_index_list_len": sum_s / B},
    }
    print(json.dumps(res), flush=True)


def make_inputs(w, dev, n_q):
    """Indexer and attention inputs: the key caches of all L tokens, the queries of the n_q rows
    of one step."""
    n = w.seq_len
    H, dqk, dv = w.attn_dims
    t = {}
    t["qI"] = synth.device_normal_bf16((n_q, w.n_heads, w.head_dim), w.seed, synth.T_QI, dev,
                                       scale=1.0 / math.sqrt(w.head_dim))
    t["wI"] = synth.device_uniform_f32((n_q, w.n_heads), w.seed, synth.T_W, dev)
    if w.fp8:
        t["kI"], t["ks"] = synth.device_fp8_keys(n, w.head_dim, w.seed, dev)
    else:
        t["kI"] = synth.device_normal_bf16((n, w.head_dim), w.seed, synth.T_KI, dev, scale=1.0 / math.sqrt(w.head_dim))
        t["ks"] = None
    t["Q"] = [synth.device_normal_bf16((n_q, H, dqk), w.seed, synth.T_Q + l, dev, rows_per_chunk=2048)
              for l in range(w.layers)]
    t["KV"] = [synth.device_normal_bf16((n, dqk), w.seed, synth.T_KV + l, dev) for l in range(w.layers)]
    t["V"] = [None if w.attn == "mla" else synth.device_normal_bf16((n, dv), w.seed, synth.T_V + l, dev)
              for l in range(w.layers)]
    return t


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


_CPU = {}   # worker state: the oracle's inputs, memory-mapped from files the parent wrote


def _cpu_worker_init(shm_dir, layers, prm_kw, dv, sm_scale):
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)                     # one BLAS thread per worker process
    import oracle.lsa_oracle as orc
    ld = lambda name: np.load(os.path.join(shm_dir, name + ".npy"), mmap_mode="r")
    _CPU.update(orc=orc, k_hat=ld("k_hat"), k_mean=ld("k_mean"), q=ld("q"), w=ld("w"),
                Q=[ld(f"Q{l}") for l in range(layers)], KV=[ld(f"KV{l}") for l in range(layers)],
                V=[ld(f"V{l}") if os.path.exists(os.path.join(shm_dir, f"V{l}.npy")) else None for l in range(layers)],
                prm=orc.IndexParams(**prm_kw), dv=dv, sm_scale=sm_scale)
    if prm_kw["pooling"] == "minmax":
        _CPU["k_mean"] = (ld("k_mean"), ld("k_min"))


def _cpu_worker_rows(job):
    """Oracle index row and every layer's attention for the sample rows job = [(i, t), ...]."""
    c = _CPU
    for i, t in job:
        r = c["orc"].index_row(int(t), c["q"][i], c["w"][i], c["k_hat"], c["k_mean"], c["prm"])
        for l in range(len(c["Q"])):
            c["orc"].attention_for_set(c["Q"][l][i], c["KV"][l], c["V"][l], r["S"], c["dv"], c["sm_scale"])
    return len(job)


def cpu_baseline(w, t, seconds, q_start=0):
    """The float64 oracle on a bounded sample of query rows of the same workload (rows of the
    step: positions q_start .. L-1), in a pool of one process per core this process may run on
    (os.sched_getaffinity), each with one BLAS thread. The pool's processes are started fresh
    (spawn: they never touch the GPU) and read the inputs memory-mapped from /dev/shm."""
    import multiprocessing as mp
    import shutil
    import tempfile
    import oracle.lsa_oracle as orc
    cores = len(os.sched_getaffinity(0))
    n = w.seq_len
    H, dqk, dv = w.attn_dims
    g = np.random.default_rng(1234)
    lo = max(w.k_cap, q_start)
    rows = np.sort(g.choice(np.arange(lo, n), size=min(8192, n - lo), replace=False))
    kb = t["kI"].cpu().numpy() if w.fp8 else t["kI"].view(torch.int16).cpu().numpy().view(np.uint16)
    ks = t["ks"].cpu().numpy() if w.fp8 else None
    ridx = torch.from_numpy(rows - q_start).cuda()
    shm_dir = tempfile.mkdtemp(prefix="lsa_oracle_", dir="/dev/shm" if os.path.isdir("/dev/shm") else None)
    try:
        save = lambda name, arr: np.save(os.path.join(shm_dir, name + ".npy"), np.ascontiguousarray(arr))
        save("q", t["qI"].index_select(0, ridx).float().cpu().numpy().astype(np.float64))
        save("w", t["wI"].index_select(0, ridx).cpu().numpy())
        for l in range(w.layers):
            save(f"Q{l}", t["Q"][l].index_select(0, ridx).view(torch.int16).cpu().numpy().view(np.uint16))
            save(f"KV{l}", t["KV"][l].view(torch.int16).cpu().numpy().view(np.uint16))
            if t["V"][l] is not None:
                save(f"V{l}", t["V"][l].view(torch.int16).cpu().numpy().view(np.uint16))
        # one-off work of the step, timed in this process: key decode and the block cache
        t0 = time.perf_counter()
        k_hat = orc.dequantized_keys(kb, ks)
        if w.pooling == "minmax":
            k_max, k_min = orc.sub_block_minmax_keys(k_hat, w.sub_block)
        else:
            k_max, k_min = orc.sub_block_mean_keys(k_hat, w.sub_block), None
        t_once = time.perf_counter() - t0
        save("k_hat", k_hat)
        save("k_mean", k_max)
        if k_min is not None:
            save("k_min", k_min)
        del k_hat, k_max, k_min
        prm_kw = dict(page=w.page, sub_block=w.sub_block, keep_pages=w.keep_pages, k_sparse=w.k_sparse,
                      k_sink=w.k_sink, k_swa=w.k_swa, run_align=w.run_align, pooling=w.pooling)
        jobs = [[(i, int(rows[i])) for i in range(j, min(j + 4, len(rows)))] for j in range(0, len(rows), 4)]
        ctx = mp.get_context("spawn")
        with ctx.Pool(cores, initializer=_cpu_worker_init,
                      initargs=(shm_dir, w.layers, prm_kw, dv, w.sm_scale)) as pool:
            pool.map(_cpu_worker_rows, [jobs[0]] * cores, chunksize=1)   # warm every worker (imports, page-in)
            done = 0
            t1 = time.perf_counter()
            pending = [pool.apply_async(_cpu_worker_rows, (j,)) for j in jobs[:2 * cores]]
            nxt = len(pending)
            while pending:
                done += pending.pop(0).get()
                if time.perf_counter() - t1 < seconds and nxt < len(jobs):
                    pending.append(pool.apply_async(_cpu_worker_rows, (jobs[nxt],)))
                    nxt += 1
            wall = time.perf_counter() - t1
    finally:
        shutil.rmtree(shm_dir, ignore_errors=True)
    per_row = wall / done                    # pool wall time per row (all workers busy)
    n_q = n - q_start
    full = t_once + n_q * per_row
    return {"value": n_q / full, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu": _cpu_model(),
            "sample": (f"{done} query rows at random positions in [{lo}, L) through the indexer and "
                       f"{w.layers} attention layers in {cores} worker processes with one BLAS thread each "
                       f"({wall:.1f} s wall), plus the one-off key decode and block cache ({t_once:.2f} s); "
                       f"tokens/s extrapolated to all {n_q} rows of the step ({per_row * 1e3:.2f} ms of pool "
                       f"wall time per row)")}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default=W.L128K_CLI4.name, choices=[w.name for w in W.FULL],
                    help="single-call prefill workloads time the whole prefill; chunked ones time the last "
                         "chunk (its block-cache update, indexer and attention) against the full cache; "
                         "the decode workload times one batched decode step")
    ap.add_argument("--graph", action="store_true", help="decode: replay the step as a captured HIP graph")
    ap.add_argument("--pooling", default="mean", choices=["mean", "minmax"],
                    help="coarse-stage block summary: mean keys (Eq. 9) or min-max extrema (Eq. 13)")
    ap.add_argument("--attn", default="fused", choices=["fused", "runs", "split"],
                    help="sparse attention as one fused pass over S_t (lsa_sparse_attn), the same pass "
                         "reading S_t from its run encoding (lsa_sparse_attn_runs), or split into "
                         "the listed part and the contiguous window on two streams, merged by log-sum-exp "
                         "(lsa_hfa_attn)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--index-sweep", default="", metavar="L1,L2,...",
                    help="only time the indexer, hierarchical against flat, at these cache lengths, and exit")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES (counter calibration) and exit")
    ap.add_argument("--gather-probe", default="", metavar="ROWS,TABLE_ROWS",
                    help="only gather ROWS random 1152-byte rows from a table of TABLE_ROWS rows "
                         "(counter calibration for scattered reads) and exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures the hot path on one GPU; running across several GPUs is not "
              "implemented (how it would shard is a design note); use --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.steps < 1 or args.warmup < 0:
        sys.exit("--steps must be >= 1 and --warmup >= 0")
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gather_probe:
        n_rows, table_rows = (int(x) for x in args.gather_probe.split(","))
        gather_probe(n_rows, table_rows)
        return
    if args.index_sweep:
        index_sweep([int(x) for x in args.index_sweep.split(",")], args.pooling)
        return

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = W.BY_NAME[args.workload]
    if w.decode:
        bench_decode(w, args)
        return
    if args.pooling != w.pooling:
        from dataclasses import replace
        w = replace(w, name=f"{w.name}_{args.pooling}", pooling=args.pooling)
    n = w.seq_len
    q_start = n - w.chunk if w.chunk else 0   # chunked workloads: the step is the last chunk
    n_q = n - q_start
    H, dqk, dv = w.attn_dims
    prm, aprm = w.index_params(), w.attn_params()
    log(f"[bench] {w.name}: generating inputs on {torch.cuda.get_device_name(dev)}")
    t = make_inputs(w, dev, n_q)
    bk = torch.empty((n // w.sub_block, prm.block_width), dtype=torch.bfloat16, device=dev)
    chunk_rows = torch.arange(q_start, n, dtype=torch.int64, device=dev)
    if w.chunk:
        lsa.block_keys(prm, t["kI"], t["ks"], out=bk)   # the earlier chunks' block cache exists already
    out = dict(idx=torch.empty((n_q, w.k_cap), dtype=torch.int32, device=dev),
               count=torch.empty((n_q,), dtype=torch.int32, device=dev),
               runs=torch.empty((n_q, w.k_cap, 2), dtype=torch.int32, device=dev),
               run_count=torch.empty((n_q,), dtype=torch.int32, device=dev))
    ws_idx = torch.empty(max(1, lsa.index_workspace_size(prm, n_q, n)), dtype=torch.uint8, device=dev)
    split_attn = args.attn == "split"
    runs_attn = args.attn == "runs"
    ws_attn_n = (lsa.hfa_workspace_size(aprm, n_q) if split_attn else
                 lsa.attn_runs_workspace_size(aprm, n_q, w.k_cap, False) if runs_attn else
                 lsa.attn_workspace_size(aprm, n_q, w.k_cap, False))
    ws_attn = torch.empty(max(1, ws_attn_n), dtype=torch.uint8, device=dev)
    O = [torch.empty((n_q, H, dv), dtype=torch.bfloat16, device=dev) for _ in range(w.layers)]
    LSE = [torch.empty((n_q, H), dtype=torch.float32, device=dev) for _ in range(w.layers)]
    torch.cuda.synchronize()
    log(f"[bench] inputs ready; {torch.cuda.memory_allocated() / 2**30:.1f} GiB allocated")

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        if w.chunk:   # the chunk's own keys just entered the cache: refresh their sub-blocks
            lsa.block_keys_update(prm, chunk_rows, t["kI"], t["ks"], bk)
        else:
            lsa.block_keys(prm, t["kI"], t["ks"], out=bk)
        if ev is not None:
            ev[1].record()
        lsa.index_prefill(prm, t["qI"], t["wI"], t["kI"], t["ks"], bk, q_start, n_kv=n, runs=True,
                          workspace=ws_idx, out=out)
        if ev is not None:
            ev[2].record()
        for l in range(w.layers):
            if split_attn:
                lsa.hfa_attn(aprm, t["Q"][l], t["KV"][l], out["idx"], out["count"], q_start, w.k_swa, out=O[l],
                             lse=LSE[l], workspace=ws_attn)
            elif runs_attn:
                lsa.sparse_attn_runs(aprm, t["Q"][l], t["KV"][l], out["runs"], out["run_count"], out=O[l],
                                     lse=LSE[l], workspace=ws_attn if ws_attn_n else None, v=t["V"][l])
            else:
                lsa.sparse_attn(aprm, t["Q"][l], t["KV"][l], t["V"][l], out["idx"], out["count"], out=O[l],
                                lse=LSE[l], workspace=ws_attn if ws_attn_n else None)
            if ev is not None:
                ev[3 + l].record()

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"[bench] warmup step {i + 1}/{args.warmup} done")
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3 + w.layers)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for s in range(args.steps):
        step(events[s])
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / args.steps
    bm_ms = np.mean([e[0].elapsed_time(e[1]) for e in events])
    idx_ms = np.mean([e[1].elapsed_time(e[2]) for e in events])
    attn_ms = [np.mean([e[2 + l].elapsed_time(e[3 + l]) for e in events]) for l in range(w.layers)]
    attn_avg = float(np.mean(attn_ms))
    log(f"[bench] {args.steps} steps: {ms_per_step:.2f} ms/step (block cache {bm_ms:.3f}, index {idx_ms:.2f}, "
        f"attention per layer {attn_avg:.2f} ms)")

    # ---- algorithmic work (per launch / per step)
    cnt = out["count"].cpu().numpy().astype(np.int64)
    sum_s = int(cnt.sum())
    row_kv_bytes = dqk * 2 if w.attn == "mla" else (dqk + dv) * 2
    attn_bytes = (sum_s * row_kv_bytes + sum_s * 4                       # gathered rows + their indices
                  + n_q * H * dqk * 2 + n_q * H * dv * 2 + n_q * H * 4 + n_q * 4)  # Q in, O and lse out, count
    attn_flops = 2.0 * H * sum_s * (dqk + dv)
    tpos = np.arange(q_start, n)
    hi = tpos - w.k_swa
    n_elig_pages = np.where(hi >= w.k_sink, hi // w.page - w.k_sink // w.page + 1, 0)
    cand = np.where(hi >= w.k_sink, np.minimum(n_elig_pages, w.keep_pages) * w.page, 0)
    sub_per_page = w.page // w.sub_block
    coarse_dim = prm.block_width      # min-max pooling scores [q+ | q-] . [k_max | k_min]
    idx_flops = 2.0 * w.n_heads * (coarse_dim * float(n_elig_pages.sum()) * sub_per_page + w.head_dim * float(cand.sum()))
    attn_gbs = attn_bytes / (attn_avg * 1e-3) / 1e9
    res = {
        "metric": ("LSA prefill tokens/s at L=128K (indexer+attn)" if not w.chunk else
                   f"LSA chunked-prefill tokens/s, last {w.chunk}-row chunk at L={n} (indexer+attn)"),
        "value": n_q / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "seq_len": n, "rows_per_step": n_q, "q_start": q_start,
                   "layers_sharing_index": w.layers,
                   "indexer": {"heads": w.n_heads, "head_dim": w.head_dim, "keys": "fp8_e4m3fn" if w.fp8 else "bf16",
                               "page": w.page, "sub_block": w.sub_block, "keep_pages": w.keep_pages,
                               "k_sparse": w.k_sparse, "k_sink": w.k_sink, "k_swa": w.k_swa,
                               "run_align": w.run_align, "pooling": w.pooling},
                   "attention": {"kind": w.attn, "heads": H, "d_qk": dqk, "d_v": dv,
                                 "operator": ("split (listed part + window, two streams)" if split_attn else
                                              "fused, list read as runs" if runs_attn else "fused")}},
        "roofline": {"kernel": ("lsa_hfa_attn (two mla_attn_kernel parts + attn_combine_kernel)" if split_attn
                                else "mla_attn_kernel"),
                     "bound": "hbm", "achieved": attn_gbs, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": attn_gbs / HBM_PEAK_GBS,
                     "traffic": None if (split_attn or runs_attn) else measured_traffic(w.name),
                     "algorithmic_bytes_per_launch": attn_bytes, "launch_ms": attn_avg},
        "breakdown": {
            "block_cache_ms": float(bm_ms), "index_ms": float(idx_ms), "attn_ms_per_layer": attn_ms,
            "indexer_scoring_tflops": idx_flops / (idx_ms * 1e-3) / 1e12,
            "indexer_mfma_frac": idx_flops / (idx_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
            "attn_tflops": attn_flops / (attn_avg * 1e-3) / 1e12,
            "attn_mfma_frac": attn_flops / (attn_avg * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
            "attn_gather_gbs": sum_s * row_kv_bytes / (attn_avg * 1e-3) / 1e9,
            "attn_tokens_per_s_per_layer": n_q / (attn_avg * 1e-3),
            "tokens_per_s_layer_equivalent": n_q * w.layers / (ms_per_step * 1e-3),
            "mean_index_list_len": sum_s / n_q,
        },
    }
    tr = res["roofline"]["traffic"]
    if tr is not None:   # HBM (data-fabric) bytes from the committed counter passes over this launch time
        res["breakdown"]["attn_fabric_gbs"] = tr / (attn_avg * 1e-3) / 1e9
        res["breakdown"]["attn_fabric_frac"] = res["breakdown"]["attn_fabric_gbs"] / HBM_PEAK_GBS
    # beside the algorithmic fraction: the counter-measured HBM fraction (the L2 serves the window
    # rows that neighbouring queries share) and the MFMA fraction of the same launch
    res["roofline"]["traffic_frac"] = res["breakdown"].get("attn_fabric_frac")
    res["roofline"]["mfma_frac"] = res["breakdown"]["attn_mfma_frac"]
    if not args.no_cpu_baseline:
        log(f"[bench] timing the oracle for ~{args.cpu_seconds:.0f} s on the host")
        res["cpu_baseline"] = cpu_baseline(w, t, args.cpu_seconds, q_start)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
