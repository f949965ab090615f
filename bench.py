#!/usr/bin/env python3
"""Response-replay attention benchmark on one MI355X.

One step = the whole replay hot path over one batch of synthetic input: the
split-KV forward over a 2,097,152-position paged bf16 prefix (8 contiguous
shards x 4 splits + the causal response split), the two-level LSE merge, and
the backward (dq accumulated over the shards, response dK/dV).  Inputs are
resident in HBM before the timed region.  Prints one JSON line.

FLOP convention: fwd = 4*Hq*D*sum_i |V_i|; bwd = Hq*D*(6*sum_i |V_i & prefix| +
10*sum_i |V_i & response|) (recompute counted, prefix dK/dV not counted); the
"useful" rate drops the backward's Q K^T recompute (4 and 8 instead of 6 and 10).
Besides the step it reports HBM-bound page streaming (the split forward over
the whole prefix with 16 query rows), ceilings measured on the same GPU (bf16
GEMM, 4 GiB copy), the clocks, and the cost of the production composition
(the cross-shard merge with its numerator reduced in bf16: time and distance
from the fp32 composition on the same shard results).  ``--ownership cyclic``
deals prefix pages to the shards block-cyclically (page p to shard p mod 8)
and ``--bf16-numerator`` makes the step's cross-shard merge the bf16 one.
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

METRIC = "replay attention TFLOP/s (fwd+bwd) & % of bf16 MFMA peak at 2M-position prefix"
METRIC_FWD = "replay attention forward TFLOP/s & % of bf16 MFMA peak (one 262,144-position shard)"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0


def visible_counts(cfg):
    """sum_i |V_i & prefix| and sum_i |V_i & response| over the response rows."""
    R, P = cfg.resp_len, cfg.prefix_len
    return R * P, R * (R + 1) // 2


def flops(cfg):
    pre, resp = visible_counts(cfg)
    Hq, D = cfg.n_q_heads, cfg.head_dim
    fwd = 4 * Hq * D * (pre + resp)
    bwd = Hq * D * (6 * pre + 10 * resp)
    return fwd, bwd


def sparse_flops(cfg):
    """Sparse latent replay: each row visits its top-k prefix entries plus the
    causal response window.  Forward: Q.K^T over Dk and P.V over Dv; backward
    (dq only): the QK^T recompute (Dk), dO.V^T (Dv) and dS.K (Dk)."""
    R, H, Dk, Dv = cfg.resp_len, cfg.n_q_heads, cfg.head_dim, cfg.head_dim_v
    vis = R * cfg.topk + R * (R + 1) // 2
    return 2 * H * (Dk + Dv) * vis, 2 * H * (2 * Dk + Dv) * vis


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def useful_flops(cfg):
    """The FLOP convention without the backward's recompute of Q K^T."""
    pre, resp = visible_counts(cfg)
    Hq, D = cfg.n_q_heads, cfg.head_dim
    return 4 * Hq * D * (pre + resp) + Hq * D * (4 * pre + 8 * resp)


def time_ms(fn, reps, stream=None, lead=0):
    """GPU time per call (ms): `reps` calls enqueued back to back between two
    HIP events, after one untimed call.  Only the first call's host-side
    argument marshalling can fall inside the interval (the GPU is idle when the
    start event is recorded); later calls are enqueued while earlier ones run,
    so for calls whose GPU time exceeds their host time the rest is hidden.
    With `lead` > 0, that many untimed calls run back to back right before the
    start event, with no synchronisation in between: the timed calls then run
    at the clock the chip settles at under that load (after idle it first runs
    fast, then lowers its clock for a few milliseconds and recovers part of
    it), and their marshalling overlaps the lead calls."""
    import torch
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(lead):
        fn()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def measured_ceilings():
    """Ceilings measured on this GPU: a large bf16 GEMM through torch (hipBLASLt)
    and a 4 GiB device-to-device copy (read + write bytes per second)."""
    import torch
    n = 8192
    a = torch.randn((n, n), dtype=torch.bfloat16, device="cuda")
    b = torch.randn((n, n), dtype=torch.bfloat16, device="cuda")
    c = torch.empty((n, n), dtype=torch.bfloat16, device="cuda")
    ms = time_ms(lambda: torch.matmul(a, b, out=c), 10)
    gemm = 2 * n ** 3 / (ms * 1e-3) / 1e12
    del a, b, c
    src = torch.empty(1 << 30, dtype=torch.float32, device="cuda")
    src.fill_(1.0)
    dst = torch.empty_like(src)
    ms = time_ms(lambda: dst.copy_(src), 10, lead=10)
    copy = 2 * src.numel() * 4 / (ms * 1e-3) / 1e9
    del dst
    torch.cuda.empty_cache()
    return {"bf16_gemm_tflops": round(gemm, 1), "gemm_shape": [n, n, n],
            "d2d_copy_gbs": round(copy, 1), "copy_bytes": 1 << 32,
            **hbm_read_ceiling(src)}


def hbm_read_ceiling(buf=None):
    """Read-only ceiling: ls_hbm_read_probe over a 4 GiB buffer (each byte read
    once, 8 loads of 16 bytes in flight per lane, XOR of the words)."""
    import torch
    from paper_2607_14952_amd import binding as B
    if buf is None:
        buf = torch.empty(1 << 30, dtype=torch.float32, device="cuda")
        buf.fill_(1.0)
    out = torch.zeros(1, dtype=torch.int32, device=buf.device)
    ms = time_ms(lambda: B.hbm_read_probe(buf, out), 20, lead=20)
    nbytes = buf.numel() * buf.element_size()
    return {"hbm_read_gbs": round(nbytes / (ms * 1e-3) / 1e9, 1), "read_bytes": nbytes}


def gpu_clocks():
    """The DPM levels of the shader and memory clocks, read in-process from the
    amdgpu sysfs files (the level marked '*' is the current one; no tool is
    started).  None when the files are not readable.  This is a snapshot after
    the timed steps: the clock the chip holds under MFMA load comes from
    counters (GRBM_GUI_ACTIVE over the kernel time, in the utilization
    summaries)."""
    import glob
    out = {}
    for path in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
        dev = os.path.dirname(path)
        for name in ("pp_dpm_sclk", "pp_dpm_mclk"):
            try:
                with open(os.path.join(dev, name)) as f:
                    lines = [ln.strip() for ln in f if ln.strip()]
            except OSError:
                continue
            cur = [ln for ln in lines if ln.endswith("*")]
            out[name] = {"levels": lines, "current": cur[0] if cur else None}
        if out:
            out["device"] = dev
            break
    return out or None


def host_cpu():
    """Logical CPUs this process may run on, and the CPU model."""
    model = platform.processor() or platform.machine()
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.lower().startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return len(os.sched_getaffinity(0)), model


def bf16_numerator_cost(step, stream, reps=20):
    """The cross-shard merge of the step's shard results with the numerator
    reduced in bf16 and in fp32 (both to fp32 outputs): times and differences."""
    import torch
    from paper_2607_14952_amd import binding as B
    R, Hq, Dv = step.out.shape
    o32 = torch.empty((R, Hq, Dv), dtype=torch.float32, device=step.out.device)
    o16 = torch.empty_like(o32)
    l32, l16 = torch.empty_like(step.lse), torch.empty_like(step.lse)
    f32 = lambda: B.lse_merge(step.shard_out, step.shard_lse, out=o32, lse=l32,  # noqa: E731
                              stream=stream)
    b16 = lambda: B.lse_merge(step.shard_out, step.shard_lse, out=o16, lse=l16,  # noqa: E731
                              flags=B.FLAG_BF16_NUMERATOR, stream=stream)
    t32, t16 = time_ms(f32, reps, stream), time_ms(b16, reps, stream)
    torch.cuda.synchronize()
    d = (o16 - o32).abs()
    return {"parts": int(step.shard_out.shape[0]), "merge_ms_fp32": round(t32, 4),
            "merge_ms_bf16": round(t16, 4), "max_abs_diff": float(d.max()),
            "max_abs_out": float(o32.abs().max()),
            "rel_l2_diff": float(torch.linalg.norm(o16 - o32) / torch.linalg.norm(o32)),
            "lse_identical": bool(torch.equal(l16, l32))}


def page_streaming(cfg, dev, rows=16, n_splits=256):
    """The split forward over the whole prefix with only `rows` query rows: an
    HBM-bound pass that reads every K and V row of the prefix once."""
    from paper_2607_14952_amd import binding as B
    q = dev["q"][:rows].contiguous()
    kv = B.PagedKV(dev["k_pool"], dev["v_pool"], dev["page_table"])
    P = cfg.prefix_len
    bounds = [P * i // n_splits for i in range(n_splits + 1)]
    splits = list(zip(bounds[:-1], bounds[1:]))
    op, lp = B.prefix_attn_fwd(q, kv, splits, prefix_len=P, q_pos0=P, scale=cfg.scale)
    ms = time_ms(lambda: B.prefix_attn_fwd(q, kv, splits, prefix_len=P, q_pos0=P,
                                           scale=cfg.scale, out_part=op, lse_part=lp), 40,
                 lead=20)
    nbytes = 2 * P * cfg.n_kv_heads * cfg.head_dim * 2
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"rows": rows, "splits": n_splits, "bytes": nbytes, "ms": round(ms, 3),
            "gbs": round(gbs, 1), "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4)}


def cpu_baseline(cfg, host, n_rows=16, n_shards=2):
    """The fp64 oracle as it stands, on this host's cores, over a bounded sample:
    forward and dq of the first n_rows query rows (all heads) against the first
    n_shards prefix shards, the same paged store and page table as the GPU run."""
    import numpy as np
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        blas_threads = os.cpu_count() or 1
    rows = np.arange(n_rows)
    b, e = cfg.shard_ranges()[0][0], cfg.shard_ranges()[n_shards - 1][1]
    kw = dict(page_size=cfg.page_size, q_pos0=cfg.q_pos0, scale=cfg.scale)
    t0 = time.perf_counter()
    o, l = O.attn_fwd(host["q"], host["k_pool"], host["v_pool"], host["page_table"], rows=rows,
                      kv_begin=b, kv_end=e, **kw)
    R, Hq, Dv = cfg.resp_len, cfg.n_q_heads, cfg.head_dim_v
    o_full = np.zeros((R, Hq, Dv))
    l_full = np.zeros((Hq, R))
    o_full[rows], l_full[:, rows] = o, l
    O.attn_bwd(host["q"], host["k_pool"], host["v_pool"], host["page_table"], host["d_out"],
               rows=rows, resp_keys=np.zeros(0, np.int64), out=o_full, lse=l_full,
               prefix_len=cfg.prefix_len, kv_begin=b, kv_end=e, **kw)
    dt = time.perf_counter() - t0
    fl = (4 + 6) * Hq * cfg.head_dim * n_rows * (e - b)
    affinity, model = host_cpu()
    return {"value": fl / dt / 1e12, "unit": "TFLOP/s", "cores": int(blas_threads),
            "cores_note": "BLAS threads the oracle ran on (its matmuls are the only "
                          "multithreaded part)",
            "affinity_cpus": affinity, "cpu_model": model, "blas_threads": int(blas_threads),
            "kind": "oracle",
            "sample": f"fp64 numpy oracle: split forward + dq of query rows 0..{n_rows - 1} "
                      f"(all {Hq} heads) over prefix keys [{b}, {e}) of the paged store; "
                      f"{fl / 1e9:.1f} GFLOP in {dt:.1f} s",
            "seconds": dt}


def run_blockwise(cfg, args):
    """G members replayed blockwise (reverse 2,048-row blocks) against one resident
    prefix; every member appends its response pages and pops them afterwards."""
    import torch
    from paper_2607_14952_amd import inputs
    from paper_2607_14952_amd.blockwise import BlockwiseReplay, ResidentPrefix, block_flops
    from paper_2607_14952_amd.replay import to_device
    log(f"generating the resident prefix for {cfg.name}")
    store = inputs.prefix_store(cfg)
    prefix = ResidentPrefix(cfg, store)
    del store
    members = []
    for m in range(cfg.members):
        r = inputs.response_inputs(cfg, m)
        members.append({k: to_device(v) for k, v in r.items()})
    rep = BlockwiseReplay(cfg, prefix)
    fl = sum(sum(block_flops(cfg, b)) for b in range(cfg.blocks)) * cfg.members
    for w in range(args.warmup):
        rep.run_member(members[0])
        torch.cuda.synchronize()
        log(f"warmup {w + 1}/{args.warmup} done")
    torch.cuda.synchronize()
    E = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    evs = [{b: (E(), E()) for b in range(cfg.blocks)} for _ in range(cfg.members)]
    t0 = time.perf_counter()
    for m in range(cfg.members):
        rep.run_member(members[m], block_events=evs[m])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    value = fl / wall / 1e12
    blocks = {}
    for b in range(cfg.blocks):
        ms = sorted(evs[m][b][0].elapsed_time(evs[m][b][1]) for m in range(cfg.members))
        bf = sum(block_flops(cfg, b))
        blocks[str(b)] = {"median_ms": round(ms[len(ms) // 2], 2), "min_ms": round(ms[0], 2),
                          "tflops_at_median": round(bf / (ms[len(ms) // 2] * 1e-3) / 1e12, 1)}
    print(json.dumps({
        "metric": "replay attention TFLOP/s (fwd+bwd), G blockwise members on a resident prefix",
        "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": 1,
        "warmup": args.warmup, "ms_per_step": round(wall * 1e3, 1), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.members} members x {cfg.resp_len} tokens in "
                               f"{cfg.rows_per_call}-row reverse blocks, prefix {cfg.prefix_len} "
                               f"in a {cfg.n_phys_pages}-page pool (sampled, with free pages)",
                   "parallelism": "single-gpu"},
        "frac_of_peak": round(value / PEAK_BF16_TFLOPS, 4), "flop_per_step": fl,
        "blocks": blocks, "gpu": torch.cuda.get_device_name(0)}), flush=True)


def run_sparse(cfg, args):
    """Sparse latent replay (MLA keys, DSA-style top-k selection + response window):
    forward and dq backward over all response rows."""
    import torch
    from paper_2607_14952_amd import binding as B
    from paper_2607_14952_amd import inputs
    from paper_2607_14952_amd.replay import to_device
    log(f"generating inputs for {cfg.name}")
    h = inputs.sparse_inputs(cfg)
    q = to_device(h["q"])
    lat = to_device(h["latent_pool"])
    table = to_device(h["page_table"])
    kv = B.PagedKV(lat, lat, table)
    idx = to_device(h["idx"])
    d_out = to_device(h["d_out"])
    sel = None
    if cfg.index_heads:
        from paper_2607_14952_amd.dsa import DsaSelect
        sel = DsaSelect(cfg, {"q_index": to_device(h["q_index"]), "w_index": to_device(h["w_index"]),
                              "k_index_pool": to_device(h["k_index_pool"]), "page_table": table},
                        mode=args.dsa_mode)
    del h
    kw = dict(prefix_len=cfg.prefix_len, q_pos0=cfg.q_pos0, scale=cfg.scale)
    ws = B.sparse_workspace(q, kv, cfg.topk, backward=True, prefix_len=cfg.prefix_len,
                            q_pos0=cfg.q_pos0)
    out = torch.empty((cfg.resp_len, cfg.n_q_heads, cfg.head_dim_v), dtype=torch.float32, device="cuda")
    lse = torch.empty((cfg.n_q_heads, cfg.resp_len), dtype=torch.float32, device="cuda")
    dq = torch.empty((cfg.resp_len, cfg.n_q_heads, cfg.head_dim), dtype=torch.float32, device="cuda")

    def step(ev=None):
        nonlocal idx
        if sel is not None:   # the step selects its indices (Eq. dsa-index, top-k)
            if ev:
                ev[3].record()
            sel.score()
            if ev:
                ev[4].record()
            idx = sel.select()
        if ev:
            ev[0].record()
        B.sparse_attn_fwd(q, kv, idx, out=out, lse=lse, workspace=ws, **kw)
        if ev:
            ev[1].record()
        # the backward takes the forward's fp32 output as written (Delta = rowsum(dO * O))
        B.sparse_attn_bwd(q, kv, idx, d_out, out, lse, dq=dq, workspace=ws, **kw)
        if ev:
            ev[2].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    R, H = cfg.resp_len, cfg.n_q_heads
    vis = R * cfg.topk + R * (R + 1) // 2
    fwd_fl, bwd_fl = sparse_flops(cfg)
    gathered = vis * 1152
    fwd_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
    bwd_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps
    ms = wall * 1e3 / args.steps
    extra = {}
    if sel is not None:
        score_ms = sum(e[3].elapsed_time(e[4]) for e in evs) / args.steps
        topk_ms = sum(e[4].elapsed_time(e[0]) for e in evs) / args.steps
        score_fl = 2 * R * cfg.prefix_len * cfg.index_heads * 128
        extra["selection"] = {
            "mode": args.dsa_mode, "index_heads": cfg.index_heads, "topk": cfg.topk,
            "score_ms": round(score_ms, 3),
            "score_tflops": round(score_fl / (score_ms * 1e-3) / 1e12, 2),
            "topk_ms": round(topk_ms, 3),
            "topk_score_gbs_per_pass": round(R * cfg.prefix_len * 4 / (topk_ms * 1e-3) / 1e9, 1),
            "score_flop": score_fl}
    print(json.dumps({
        "metric": "sparse latent replay TFLOP/s (fwd+bwd dq), MLA 576/512 with top-k selection",
        "value": round((fwd_fl + bwd_fl + extra.get("selection", {}).get("score_flop", 0))
                       / (ms * 1e-3) / 1e12, 2), "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {H} heads sharing one 576-wide latent row, prefix "
                               f"{cfg.prefix_len} in {cfg.page_size}-entry pages, {R} tokens x "
                               f"top-{cfg.topk} + causal window"
                               + (f"; indices selected in the step by DSA index scores "
                                  f"({cfg.index_heads} heads x 128, counted in the FLOP) and "
                                  f"top-{cfg.topk} ({args.dsa_mode})" if sel is not None else
                                  "; seeded indices"), "parallelism": "single-gpu"},
        "fwd_ms": round(fwd_ms, 3), "fwd_tflops": round(fwd_fl / (fwd_ms * 1e-3) / 1e12, 2),
        "fwd_gather_gbs": round(gathered / (fwd_ms * 1e-3) / 1e9, 1),
        "bwd_ms": round(bwd_ms, 3), "bwd_tflops": round(bwd_fl / (bwd_ms * 1e-3) / 1e12, 2),
        "flop_per_step": {"fwd": fwd_fl, "bwd": bwd_fl}, "gpu": torch.cuda.get_device_name(0),
        **extra}),
        flush=True)


def run_capture(cfg, args):
    """Chunked no-grad capture of one attention layer's prompt into the paged
    store: every chunk's K/V scatter, split forward and merge, timed over the
    whole prompt with its rows resident in HBM."""
    import torch
    from paper_2607_14952_amd import inputs
    from paper_2607_14952_amd.capture import PrefixCapture
    from paper_2607_14952_amd.replay import to_device
    log(f"generating inputs for {cfg.name}")
    t = time.perf_counter()
    h = inputs.capture_inputs(cfg)
    log(f"inputs ready in {time.perf_counter() - t:.1f} s; copying to HBM")
    dev = {k: to_device(v) for k, v in h.items()}
    del h
    stream = torch.cuda.current_stream()
    cap = PrefixCapture(cfg, dev, stream=stream)
    for c in range(min(args.warmup, cfg.n_chunks)):   # warm the kernels on the first chunks
        cap.chunk(c)
    torch.cuda.synchronize()
    E = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    probes = sorted({0, cfg.n_chunks // 4, cfg.n_chunks // 2, cfg.n_chunks - 1})
    pev = {c: (E(), E()) for c in probes}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for c in range(cfg.n_chunks):
        if c in pev:
            pev[c][0].record(stream)
        cap.chunk(c)
        if c in pev:
            pev[c][1].record(stream)
        if c % 64 == 63:
            log(f"captured {c + 1}/{cfg.n_chunks} chunks")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fl = 4 * cfg.n_q_heads * cfg.head_dim * cfg.visible()
    chunk_ms = {str(c): round(pev[c][0].elapsed_time(pev[c][1]), 3) for c in probes}
    result = {
        "metric": "prefix capture, one attention layer (s)",
        "value": round(wall, 3), "unit": "s", "n_gpus": 1, "steps": 1, "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3, 1), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.length} prompt positions in "
                               f"{cfg.n_chunks} chunks of {cfg.chunk}, bf16 GQA "
                               f"{cfg.n_q_heads}q/{cfg.n_kv_heads}kv, head_dim {cfg.head_dim}, "
                               f"{cfg.page_size}-position pages; per chunk: K/V scatter into "
                               f"its pages, split forward over earlier + own keys, merge",
                   "length": cfg.length, "chunk": cfg.chunk, "page_size": cfg.page_size},
        "tflops": round(fl / wall / 1e12, 2),
        "flop": fl,
        "chunk_ms": chunk_ms,
        "gpu": torch.cuda.get_device_name(0),
    }
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c3")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=96)
    ap.add_argument("--calib-copy", action="store_true",
                    help="run a 1 GiB device copy first (reference for rocprofv3 byte counters)")
    ap.add_argument("--ownership", choices=("contiguous", "cyclic"), default="contiguous",
                    help="prefix pages to shards: contiguous ranges or page p to shard p mod 8")
    ap.add_argument("--bf16-numerator", action="store_true",
                    help="the step's cross-shard merge reduces the numerator in bf16")
    ap.add_argument("--dsa-select", action="store_true",
                    help="c5: select each row's top-k with the DSA index scores inside the step")
    ap.add_argument("--dsa-mode", choices=("global", "candidates"), default="global",
                    help="selection: one top-k per row, or per-shard candidates and a merge")
    ap.add_argument("--streaming-only", action="store_true",
                    help="c3 inputs: time only the page streaming pass (R = 16) and the read "
                         "ceiling (for counter runs on that pass alone)")
    ap.add_argument("--skip-extras", action="store_true",
                    help="skip page streaming, measured ceilings and clocks (profiling runs: the "
                         "streaming pass reuses the forward kernel)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_14952_amd import binding, configs, inputs
    from paper_2607_14952_amd.replay import ReplayStep, device_inputs

    binding.load_library()
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    cfg = configs.get(args.config)
    if args.calib_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if isinstance(cfg, configs.CaptureConfig):
        run_capture(cfg, args)
        return
    if args.dsa_select:
        cfg = cfg.scaled(index_heads=32)
    if args.ownership != "contiguous" or args.bf16_numerator:
        cfg = cfg.scaled(ownership=args.ownership, bf16_numerator=args.bf16_numerator)
    if cfg.members > 1:
        run_blockwise(cfg, args)
        return
    if cfg.sparse:
        run_sparse(cfg, args)
        return
    log(f"generating inputs for {cfg.name}")
    t = time.perf_counter()
    host = inputs.dense_inputs(cfg)
    log(f"inputs ready in {time.perf_counter() - t:.1f} s; copying to HBM")
    dev = device_inputs(host)
    stream = torch.cuda.current_stream()
    if args.streaming_only:
        ps = page_streaming(cfg, dev)
        del dev
        torch.cuda.empty_cache()
        ceil = hbm_read_ceiling()
        ps["frac_of_read_ceiling"] = round(ps["gbs"] / ceil["hbm_read_gbs"], 4)
        print(json.dumps({"page_streaming": ps, "read_ceiling": ceil,
                          "gpu": torch.cuda.get_device_name(0)}), flush=True)
        return
    # a forward-only configuration (c2: one shard of c3, out and lse) times the
    # forward and the merge alone
    with_bwd = cfg.backward
    step = ReplayStep(cfg, dev, backward=with_bwd, stream=stream)
    fwd_fl, bwd_fl = flops(cfg)
    if not with_bwd:
        bwd_fl = 0

    for w in range(args.warmup):
        step.step()
        torch.cuda.synchronize()
        log(f"warmup {w + 1}/{args.warmup} done")

    E = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    n_r = len(step.shards) if with_bwd else 0
    ev = [[E() for _ in range(3 + n_r + 1)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        e = ev[s]
        e[0].record(stream)
        step.forward_splits()
        e[1].record(stream)
        step.merge()
        e[2].record(stream)
        for r in range(n_r):
            step.backward_range(r)
            e[3 + r].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    log(f"timed {args.steps} steps in {wall:.3f} s")

    fwd_ms = [e[0].elapsed_time(e[1]) for e in ev]
    merge_ms = [e[1].elapsed_time(e[2]) for e in ev]
    bwd_ms = [[e[2 + r].elapsed_time(e[3 + r]) for r in range(n_r)] for e in ev]
    step_ms = [e[0].elapsed_time(e[3 + n_r - 1]) for e in ev]
    ms_per_step = wall * 1e3 / args.steps
    value = (fwd_fl + bwd_fl) / (ms_per_step * 1e-3) / 1e12

    avg = lambda xs: sum(xs) / len(xs)  # noqa: E731
    fwd_avg = avg(fwd_ms)
    fwd_tf = fwd_fl / (fwd_avg * 1e-3) / 1e12
    if with_bwd:
        pre_ranges = [r for r, (b, e) in enumerate(step.shards) if e <= cfg.prefix_len]
        dq_launch_ms = avg([bwd_ms[s][r] for s in range(args.steps) for r in pre_ranges])
        shard_len = step.shards[pre_ranges[0]][1] - step.shards[pre_ranges[0]][0]
        dq_launch_fl = 6 * cfg.n_q_heads * cfg.head_dim * cfg.resp_len * shard_len
        dq_tf = dq_launch_fl / (dq_launch_ms * 1e-3) / 1e12
        fwd_total, dq_total = fwd_avg, dq_launch_ms * len(pre_ranges)
    else:
        dq_tf = None
        fwd_total, dq_total = fwd_avg, 0.0
    if fwd_total >= dq_total:
        roof = {"kernel": "fwd_bf16_d256_kernel (all splits: one launch, one per shard "
                          "when cyclic)",
                "achieved": fwd_tf, "flop_per_launch": fwd_fl, "avg_launch_ms": fwd_avg}
    else:
        roof = {"kernel": "bwd_dq_bf16_d256_kernel (one 262,144-key shard per launch)",
                "achieved": dq_tf, "flop_per_launch": dq_launch_fl, "avg_launch_ms": dq_launch_ms}
    from paper_2607_14952_amd import profiling
    kname = "fwd_bf16_d256_kernel" if fwd_total >= dq_total else "bwd_dq_bf16_d256_kernel"
    traffic = profiling.traffic_for(kname, os.path.join(ROOT, "profiles", f"traffic_{cfg.name}.json"))
    roofline = {"bound": "mfma", "achieved": round(roof["achieved"], 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(roof["achieved"] / PEAK_BF16_TFLOPS, 4),
                "traffic": None if traffic is None else round(traffic),
                "kernel": roof["kernel"], "flop_per_launch": roof["flop_per_launch"],
                "avg_launch_ms": round(roof["avg_launch_ms"], 3)}
    # merge bytes: split partials read + shard results written and re-read + output
    R, Hq, Dv = cfg.resp_len, cfg.n_q_heads, cfg.head_dim_v
    ns, nsh = len(step.splits), len(step.shards)
    merge_bytes = (ns * R * Hq * (Dv + 1) * 4 + nsh * R * Hq * (Dv + 1) * 4 * 2
                   + R * Hq * (Dv * 2 + 4))
    result = {
        "metric": METRIC if with_bwd else METRIC_FWD,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: bf16 GQA {cfg.n_q_heads}q/{cfg.n_kv_heads}kv, "
                               f"head_dim {cfg.head_dim}, prefix {cfg.prefix_len} in "
                               f"{cfg.page_size}-position pages (seeded permutation), "
                               f"{cfg.n_shards} {cfg.ownership} shards x "
                               f"{cfg.splits_per_shard} splits + response split, response "
                               f"{cfg.resp_len} causal, " + ("fwd+bwd" if with_bwd else "fwd only")
                               + (", bf16-numerator merge" if cfg.bf16_numerator else ""),
                   "ownership": cfg.ownership, "bf16_numerator": cfg.bf16_numerator,
                   "prefix_len": cfg.prefix_len, "resp_len": cfg.resp_len,
                   "n_q_heads": cfg.n_q_heads, "n_kv_heads": cfg.n_kv_heads,
                   "head_dim": cfg.head_dim, "page_size": cfg.page_size,
                   "splits": ns, "shards": nsh, "parallelism": "single-gpu"},
        "frac_of_peak": round(value / PEAK_BF16_TFLOPS, 4),
        "roofline": roofline,
        "phases_ms": {"fwd_splits": round(fwd_avg, 3), "merge": round(avg(merge_ms), 3),
                      "bwd_ranges": [round(avg([b[r] for b in bwd_ms]), 3) for r in range(n_r)],
                      "step_events": round(avg(step_ms), 3),
                      "step_events_median": round(sorted(step_ms)[len(step_ms) // 2], 3),
                      "step_events_min": round(min(step_ms), 3)},
        "fwd_tflops": round(fwd_tf, 2),
        "dq_tflops": None if dq_tf is None else round(dq_tf, 2),
        "merge_gbs": round(merge_bytes / (avg(merge_ms) * 1e-3) / 1e9, 1),
        "flop_per_step": {"fwd": fwd_fl, "bwd": bwd_fl},
        "gpu": torch.cuda.get_device_name(0),
    }
    useful = useful_flops(cfg) if with_bwd else fwd_fl
    result["useful_tflops"] = round(useful / (ms_per_step * 1e-3) / 1e12, 2)
    if not args.skip_extras:
        log("bf16-numerator merge cost")
        result["bf16_numerator"] = bf16_numerator_cost(step, stream)
        log("page streaming, clocks")
        result["page_streaming"] = page_streaming(cfg, dev)
        result["gpu_clocks"] = gpu_clocks()
    if not args.no_cpu_baseline:
        del dev, step
        torch.cuda.empty_cache()
        log("timing the CPU oracle sample")
        cb = cpu_baseline(cfg, host, args.cpu_rows)
        result["cpu_baseline"] = {k: (round(v, 6) if isinstance(v, float) else v)
                                  for k, v in cb.items()}
    else:
        del dev, step
        torch.cuda.empty_cache()
    if not args.skip_extras:
        log("measured ceilings")
        ceil = measured_ceilings()
        ceil["frac_of_gemm"] = round(value / ceil["bf16_gemm_tflops"], 4)
        ceil["roofline_frac_of_gemm"] = round(roofline["achieved"] / ceil["bf16_gemm_tflops"], 4)
        result["measured_ceilings"] = ceil
        ps = result["page_streaming"]
        ps["frac_of_read_ceiling"] = round(ps["gbs"] / ceil["hbm_read_gbs"], 4)
        ps["frac_of_copy_ceiling"] = round(ps["gbs"] / ceil["d2d_copy_gbs"], 4)
        result["merge_frac_of_hbm_peak"] = round(result["merge_gbs"] / PEAK_HBM_GBS, 4)
        result["merge_frac_of_read_ceiling"] = round(result["merge_gbs"] / ceil["hbm_read_gbs"], 4)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
