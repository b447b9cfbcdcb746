#!/usr/bin/env python3
"""Benchmark of owner-local paged MLA decode attention on one MI355X.

A step is one whole pass of the path over one batch (one layer): the split
planner, the attend kernel and the combine kernel, through the library's
C-ABI, with inputs already resident in HBM.  Prints ONE JSON line.

Default workload: many short requests (B=256, H=128, q=1, s ~ U[1024,4096],
bf16 cache).  --config selects another of the five workloads.
"""
import argparse
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0        # MI355X HBM3E
KERNEL_SOURCES = ["paper_2609_37626_amd/csrc/kernels.hip", "paper_2609_37626_amd/csrc/splash_common.hpp",
                  "paper_2609_37626_amd/csrc/kernels.hpp"]
BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
METRIC = "us/step and achieved KV GB/s + MFMA TFLOP/s (% of roofline), paged MLA decode"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_digest():
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per attend launch from the committed counter summary, if it
    was taken on the kernel sources as they stand (else None)."""
    path = os.path.join(ROOT, "profiles", "attend_kernel_hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                fields.setdefault(k.strip(), []).append(v.strip())
    digests = fields.get("kernel_source_sha256", [])
    if not digests or digests[0] != kernel_source_digest():
        return None
    for w, fb, wb in zip(fields.get("workload", []), fields.get("fetch_bytes_per_launch", []),
                         fields.get("write_bytes_per_launch", [])):
        if w == workload:
            return {"fetch_bytes": int(fb), "write_bytes": int(wb), "total_bytes": int(fb) + int(wb)}
    return None


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(batch, budget_s):
    """Time the fp64 oracle (as it stands) on the first requests of the batch,
    then scale by visible (row, key) pairs to the whole batch: once with the
    BLAS threads numpy has on this host, once limited to one thread."""
    import numpy as np
    import oracle
    q = batch.q_chunk
    vis = [int(s) * q - q * (q - 1) // 2 for s in batch.seq_lens]
    total_vis = sum(vis)

    def timed(budget):
        done_vis, n, t_used = 0, 0, 0.0
        while n < batch.B and t_used < budget:
            t0 = time.perf_counter()
            oracle.mla_attention(batch.q, batch.kv, batch.block_table, batch.seq_lens, q, batch.softmax_scale,
                                 kv_dtype=batch.kv_dtype, kv_scales=batch.kv_scales, requests=[n])
            t_used += time.perf_counter() - t0
            done_vis += vis[n]
            n += 1
        return t_used * 1e6 * total_vis / done_vis, n, done_vis, t_used

    threads = os.cpu_count() or 1
    one = None
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([d.get("num_threads", 1) for d in threadpool_info() if d.get("user_api") == "blas"] or [1])
        with threadpool_limits(limits=1, user_api="blas"):
            u1, n1, v1, t1 = timed(budget_s / 3)
        one = {"value": round(u1, 1), "unit": "us/step", "cores": 1,
               "sample": f"first {n1} of {batch.B} requests ({v1} of {total_vis} visible row-key pairs, "
                         f"{t1:.1f} s), scaled by visible row-key pairs"}
    except ImportError:
        pass
    us_per_step, n, done_vis, t_used = timed(budget_s)
    res = {"value": round(us_per_step, 1), "unit": "us/step", "cores": int(threads), "kind": "oracle",
           "sample": f"first {n} of {batch.B} requests ({done_vis} of {total_vis} visible row-key pairs, "
                     f"{t_used:.1f} s), scaled by visible row-key pairs",
           "cpu_model": cpu_model(), "cpu_threads_available": len(os.sched_getaffinity(0)),
           "blas_threads": int(threads)}
    if one is not None:
        res["one_thread"] = one
    return res


def run_topk(args, spec, batch):
    """--topk K: every row n attends min(K, visible) distinct positions of its
    request's history, drawn uniformly (seeded) and listed in position order;
    a step is one splash_mla_attend_topk call (plan, attend, combine)."""
    import numpy as np
    import torch

    from paper_2609_37626_amd import binding as B
    from paper_2609_37626_amd import workloads as W
    from paper_2609_37626_amd.device import to_device

    K = args.topk
    rng = np.random.Generator(np.random.PCG64(spec.seed + 1000))
    N = batch.B * batch.q_chunk
    idx = np.full((N, K), -1, dtype=np.int32)
    cnt = np.zeros(N, dtype=np.int32)
    for n in range(N):
        b, i = divmod(n, batch.q_chunk)
        vis = int(batch.seq_lens[b]) - batch.q_chunk + i + 1
        c = min(K, vis)
        idx[n, :c] = np.sort(rng.choice(vis, size=c, replace=False))
        cnt[n] = c
    db = to_device(batch)
    out, lse = db.alloc_outputs()
    ws = db.workspace()
    desc = db.desc()
    idx_d, cnt_d = torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda()
    stream = torch.cuda.current_stream()

    def step():
        B.splash_mla_attend_topk(db.q, db.kv, db.block_table, db.seq_lens, batch.q_chunk, idx_d, cnt_d, out, lse,
                                 desc, ws, stream)

    t_w = time.perf_counter()
    warm = 0
    while warm < args.warmup or ((time.perf_counter() - t_w) * 1e3 < args.min_warmup_ms and warm < 5000):
        step()
        warm += 1
        if warm % 10 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    for k in range(args.steps):
        ev[k][0].record(stream)
        step()
        ev[k][1].record(stream)
    torch.cuda.synchronize()
    call_us = float(np.mean([e[0].elapsed_time(e[1]) for e in ev])) * 1e3

    sel = int(cnt.sum())
    row_bytes = {W.KV_BF16: 1152, W.KV_FP8_E4M3: 580, W.KV_FP8_LATENT: W.LATENT_ROW_BYTES}[batch.kv_dtype]
    H = batch.H
    alg_bytes = sel * row_bytes + N * H * (576 * 2 + 512 * 2 + 4) + sel * 4
    flops = 2.0 * H * (576 + 512) * sel
    hbm_t, mfma_t = alg_bytes / (HBM_PEAK_GBPS * 1e9), flops / (BF16_PEAK_TFLOPS * 1e12)
    if hbm_t >= mfma_t:
        ach = alg_bytes / (call_us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBPS, 4)}
    else:
        ach = flops / (call_us * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / BF16_PEAK_TFLOPS, 4)}
    roof.update({"traffic": None, "kernel": "splash_mla_attend_topk (plan, attend, combine) timed together",
                 "kernel_avg_us": round(call_us, 2), "alg_bytes_per_launch": int(alg_bytes),
                 "alg_flops_per_launch": int(flops), "roofline_us": round(max(hbm_t, mfma_t) * 1e6, 1)})
    result = {
        "metric": METRIC + ", top-k",
        "value": round(ms * 1e3, 2), "unit": "us/step", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "warmup_run": warm, "ms_per_step": round(ms, 4), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded PCG64 draws of the workload's length mix; N(0,1) cache rows and queries; "
                "uniform position choice)",
        "config": {"workload": spec.name, "B": batch.B, "H": H, "q_chunk": batch.q_chunk,
                   "kv_cache": W.KV_LABELS[batch.kv_dtype], "seed": spec.seed, "topk": K,
                   "selected_rows": sel},
        "kv_gbps": round(sel * row_bytes / (ms * 1e-3) / 1e9, 1),
        "roofline": roof,
    }
    print(json.dumps(result), flush=True)


def run_dop(args, spec, batch):
    """--dop-ranks T: one GPU's share of a layer's DOP regroup.  As a rank it
    packs its H/T heads of all N rows by owner and later puts its output rows
    back in order; as an owner it assembles its N/T rows (requests dealt out
    round-robin) with all heads and splits its output by rank.  The
    all-to-all between them is not timed (it is not part of the library)."""
    import numpy as np
    import torch

    from paper_2609_37626_amd import binding as B

    T = args.dop_ranks
    N = args.dop_rows if args.dop_rows > 0 else batch.B * batch.q_chunk
    H = batch.H
    if H % T:
        raise SystemExit(f"--dop-ranks {T} must divide the {H} heads")
    hl = H // T
    owner = (np.arange(N) // batch.q_chunk) % T                  # request b's rows go to owner b % T
    order = np.concatenate([np.flatnonzero(owner == o) for o in range(T)]).astype(np.int32)
    n_own = int(np.count_nonzero(owner == 0))
    order_d = torch.from_numpy(order).cuda()
    g = torch.Generator(device="cuda").manual_seed(spec.seed)
    rnd = lambda *shape: torch.randint(-32768, 32767, shape, dtype=torch.int16, device="cuda", generator=g)
    q_nope, q_rope = rnd(N, hl, 512), rnd(N, hl, 64)
    send_q, recv_q, q_owner = rnd(N, hl, 576), rnd(T * n_own, hl, 576), rnd(n_own, H, 576)
    out_owner, send_o, recv_o, out = rnd(n_own, H, 512), rnd(T * n_own, hl, 512), rnd(N, hl, 512), rnd(N, hl, 512)
    stream = torch.cuda.current_stream()
    kernels = [
        ("pack_q", lambda: B.splash_dop_pack_q(q_nope, q_rope, order_d, send_q, stream), 2 * N * hl * 576 * 2),
        ("unpack_q", lambda: B.splash_dop_unpack_q(recv_q, T, q_owner, stream), 2 * n_own * H * 576 * 2),
        ("pack_out", lambda: B.splash_dop_pack_out(out_owner, T, send_o, stream), 2 * n_own * H * 512 * 2),
        ("unpack_out", lambda: B.splash_dop_unpack_out(recv_o, order_d, out, stream), 2 * N * hl * 512 * 2),
    ]

    def layer():
        for _, fn, _ in kernels:
            fn()

    t_w = time.perf_counter()
    warm = 0
    while warm < args.warmup or ((time.perf_counter() - t_w) * 1e3 < args.min_warmup_ms and warm < 20000):
        layer()
        warm += 1
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        layer()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(kernels) + 1)] for _ in range(args.steps)]
    for k in range(args.steps):
        for i, (_, fn, _) in enumerate(kernels):
            ev[k][i].record(stream)
            fn()
        ev[k][len(kernels)].record(stream)
    torch.cuda.synchronize()
    per = {name: float(np.mean([e[i].elapsed_time(e[i + 1]) for e in ev])) * 1e3
           for i, (name, _, _) in enumerate(kernels)}
    gbps = {name: round(nbytes / (per[name] * 1e-6) / 1e9, 1) for name, _, nbytes in kernels}
    total_bytes = sum(nb for _, _, nb in kernels)
    dom = max(per, key=per.get)
    dom_bytes = dict((n, nb) for n, _, nb in kernels)[dom]
    achieved = dom_bytes / (per[dom] * 1e-6) / 1e9
    result = {
        "metric": "us per layer and GB/s of one GPU's DOP query + output regroup (pack, unpack; all-to-all not "
                  "included)",
        "value": round(ms * 1e3, 2), "unit": "us/layer", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (random bf16 bit patterns)",
        "config": {"workload": spec.name, "ranks": T, "rows": N, "H": H, "heads_per_rank": hl,
                   "rows_owned": n_own, "owner_of_request": "b mod ranks"},
        "kernel_us": {k: round(v, 2) for k, v in per.items()}, "kernel_gbps": gbps,
        "bytes_per_layer": total_bytes, "gbps_per_layer": round(total_bytes / (ms * 1e-3) / 1e9, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": None, "kernel": f"dop {dom}",
                     "kernel_avg_us": round(per[dom], 2), "alg_bytes_per_launch": dom_bytes},
    }
    print(json.dumps(result), flush=True)


def run_sharded(args, spec, batch, db):
    """--shards N: every history cut into N page-aligned position shards of
    (nearly) equal length; a step is the N shard calls (each: plan, attend,
    the shard's own combine) and one splash_mla_combine over the N partials,
    i.e. what N position-sharded ranks compute, on one GPU."""
    import numpy as np
    import torch

    from paper_2609_37626_amd import binding as B
    from paper_2609_37626_amd import workloads as W

    N = args.shards
    s = batch.seq_lens.astype(np.int64)
    cuts = np.stack([np.minimum(s, (s * k // N) // 64 * 64) for k in range(N)] + [s], axis=1).astype(np.int32)
    kb = [torch.from_numpy(np.ascontiguousarray(cuts[:, k])).cuda() for k in range(N)]
    ke = [torch.from_numpy(np.ascontiguousarray(cuts[:, k + 1])).cuda() for k in range(N)]
    part_out = torch.empty((batch.B * N * batch.q_chunk, batch.H, 512), dtype=torch.float32, device="cuda")
    part_lse = torch.empty((batch.B * N * batch.q_chunk, batch.H), dtype=torch.float32, device="cuda")
    indptr = torch.arange(0, (batch.B + 1) * N, N, dtype=torch.int32, device="cuda")
    out, lse = db.alloc_outputs()
    ws = db.workspace()
    desc = db.desc()
    stream = torch.cuda.current_stream()

    def sharded_step(ev=None):
        for k in range(N):
            if ev is not None:
                ev[k].record(stream)
            B.splash_mla_attend_shard(db.q, db.kv, db.block_table, db.seq_lens, db.q_chunk, kb[k], ke[k], N, k,
                                      part_out, part_lse, desc, ws, stream)
        if ev is not None:
            ev[N].record(stream)
        B.splash_mla_combine(part_out, part_lse, indptr, batch.B, batch.q_chunk, batch.H, out, lse, stream)
        if ev is not None:
            ev[N + 1].record(stream)

    t_w = time.perf_counter()
    warmup_run = 0
    while warmup_run < args.warmup or ((time.perf_counter() - t_w) * 1e3 < args.min_warmup_ms and warmup_run < 5000):
        sharded_step()
        warmup_run += 1
        if warmup_run % 10 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        sharded_step()
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t_start) * 1e3 / args.steps
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(N + 2)] for _ in range(args.steps)]
    for k in range(args.steps):
        sharded_step(events[k])
    torch.cuda.synchronize()
    per_shard = np.array([[e[k].elapsed_time(e[k + 1]) for k in range(N)] for e in events]).mean(axis=0)
    merge_ms = float(np.mean([e[N].elapsed_time(e[N + 1]) for e in events]))
    shard_s = float(per_shard.sum()) * 1e-3

    kv_bytes, alg_bytes, flops = W.workload_bytes_flops(batch)
    hbm_time = alg_bytes / (HBM_PEAK_GBPS * 1e9)
    mfma_time = flops / (BF16_PEAK_TFLOPS * 1e12)
    if hbm_time >= mfma_time:
        achieved = alg_bytes / shard_s / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4)}
    else:
        achieved = flops / shard_s / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / BF16_PEAK_TFLOPS, 4)}
    roof.update({"traffic": None, "kernel": f"splash_mla_attend_shard x {N} (plan, attend and the shard's combine "
                                            f"each), timed together",
                 "kernel_avg_us": round(shard_s * 1e6, 2), "roofline_us": round(max(hbm_time, mfma_time) * 1e6, 1)})
    result = {
        "metric": METRIC + ", position-sharded",
        "value": round(ms_per_step * 1e3, 2),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_run": warmup_run,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded PCG64 draws of the workload's length mix; N(0,1) cache rows and queries)",
        "config": {"workload": spec.name, "B": batch.B, "H": batch.H, "q_chunk": batch.q_chunk,
                   "kv_cache": W.KV_LABELS[batch.kv_dtype], "seed": spec.seed,
                   "shards": N, "shard_cuts": "history b cut at floor(s_b k / N) rounded down to a page, k < N"},
        "phases_us": {"shards": [round(float(x) * 1e3, 2) for x in per_shard], "merge": round(merge_ms * 1e3, 2)},
        "roofline": roof,
    }
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--min-warmup-ms", type=float, default=200.0,
                    help="keep warming up (beyond --warmup steps) until this much wall time has passed: "
                         "the first ~30 steps of a process run ~10%% slow")
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (reference for HBM byte counters)")
    ap.add_argument("--topk", type=int, default=0,
                    help="top-k variant: every row attends this many of its visible positions (a seeded uniform "
                         "choice, in position order) through splash_mla_attend_topk")
    ap.add_argument("--dop-ranks", type=int, default=0,
                    help="DOP regroup: time one GPU's share of a layer's query and output regroup for this many "
                         "ranks (pack its head slice, assemble its own rows, and back)")
    ap.add_argument("--dop-rows", type=int, default=0,
                    help="with --dop-ranks: current query rows N (default: the workload's B * q_chunk)")
    ap.add_argument("--exact-qk", action="store_true",
                    help="fp8 caches: QK with K converted to bf16 (SPLASH_FLAG_EXACT_QK) instead of the fp8 pipe")
    ap.add_argument("--kv-format", choices=["workload", "latent"], default="workload",
                    help="latent: the workload's lengths over the fp8 latent-row cache (656-byte rows)")
    ap.add_argument("--shards", type=int, default=0,
                    help="position-sharded variant: cut every history into this many page-aligned shards, "
                         "run splash_mla_attend_shard per shard and splash_mla_combine over them")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (each owner GPU runs the same "
              "kernel on its own requests); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_37626_amd import binding as B
    from paper_2609_37626_amd import calib as CAL
    from paper_2609_37626_amd import workloads as W
    from paper_2609_37626_amd.device import to_device
    globals()["B"], globals()["CAL"] = B, CAL

    assert torch.cuda.is_available(), "bench needs a GPU"
    spec = W.CONFIGS[args.config]
    t0 = time.perf_counter()
    if args.kv_format == "latent" and args.dop_ranks > 0:
        print("--kv-format latent applies to the attention modes, not the DOP regroup", file=sys.stderr)
        sys.exit(2)
    if args.kv_format == "latent":
        batch = W.make_config(args.config, kv_dtype=W.KV_FP8_LATENT)
        spec = dataclasses.replace(spec, name=spec.name.replace(" e4m3", "") + " fp8-latent-rows",
                                   kv_dtype=W.KV_FP8_LATENT)
    else:
        batch = W.make_config(args.config)
    log(f"workload {spec.name}: generated in {time.perf_counter() - t0:.1f} s")
    if args.dop_ranks > 0:
        return run_dop(args, spec, batch)
    if args.topk > 0:
        return run_topk(args, spec, batch)
    db = to_device(batch)
    if args.shards > 0:
        return run_sharded(args, spec, batch, db)
    out, lse = db.alloc_outputs()
    ws = db.workspace()
    desc = db.desc(B.FLAG_EXACT_QK if args.exact_qk else 0)
    stream = torch.cuda.current_stream()

    def step_plain():
        # the product entry point: plan, attend and combine in one call
        B.splash_mla_attend(db.q, db.kv, db.block_table, db.seq_lens, db.q_chunk, out, lse, desc, ws, stream)

    def step(ev=None):
        # the same work as three calls, with events around each phase
        if ev is not None:
            ev[0].record(stream)
        B.splash_mla_plan(db.seq_lens, db.q_chunk, desc, ws, stream)
        if ev is not None:
            ev[1].record(stream)
        B.splash_mla_attend_units(db.q, db.kv, db.block_table, db.seq_lens, db.q_chunk, out, lse, desc, ws, stream)
        if ev is not None:
            ev[2].record(stream)
        B.splash_mla_combine_splits(db.q_chunk, out, lse, desc, ws, stream)
        if ev is not None:
            ev[3].record(stream)

    t_w = time.perf_counter()
    warmup_run = 0
    for _ in range(args.warmup):
        step_plain()
        warmup_run += 1
    torch.cuda.synchronize()
    while (time.perf_counter() - t_w) * 1e3 < args.min_warmup_ms and warmup_run < 5000:
        for _ in range(10):
            step_plain()
        warmup_run += 10
        torch.cuda.synchronize()

    # Warm region: K steps back to back with nothing else on the stream (the
    # KV of one step can still sit partly in the 256 MB MALL for the next).
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        step_plain()
    torch.cuda.synchronize()
    warm_ms = (time.perf_counter() - t_start) * 1e3 / args.steps

    # Same K steps with HIP events on the launch stream around each phase.
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    warm_ph = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(3)] + [e[0].elapsed_time(e[3])]
                        for e in events]) * 1e3

    # Cold region (the headline): before each step the whole cache hierarchy
    # (L2 and the 256 MB MALL) is flushed by READING a 1 GiB buffer, outside
    # the events, so no dirty line is written back during the timed step.
    # The headline times the product entry point, one call, between two
    # events; a second cold pass runs the three phase calls with events
    # between them for the breakdown (an event between two kernels costs
    # them a few microseconds, so its step is a little longer).
    flush_buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    flush_buf.zero_()
    sink = torch.empty(512 * 1024, dtype=torch.uint8, device="cuda")
    # (the two kinds of step alternate, so both see the same chip state)
    sev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    cev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        CAL.stream_read(flush_buf, sink, 512, stream)
        sev[k][0].record(stream)
        step_plain()
        sev[k][1].record(stream)
        CAL.stream_read(flush_buf, sink, 512, stream)
        step(cev[k])
    torch.cuda.synchronize()
    cold_wall_ms = (time.perf_counter() - t_start) * 1e3 / (2 * args.steps)
    cold_steps = np.array([e[0].elapsed_time(e[1]) for e in sev]) * 1e3
    cold_ph = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(3)] + [e[0].elapsed_time(e[3])]
                        for e in cev]) * 1e3
    del flush_buf

    # Achievable peaks of this chip, measured in the same run: a streaming
    # read of 1 GiB and a loop of bf16 MFMAs on random N(0,1) operands.
    peaks = measured_peaks(torch, stream)

    offs, _ = B.workspace_offsets(batch.B, batch.q_chunk, batch.H, 0)
    hdr = ws[offs[0]:offs[0] + 64].cpu().numpy().view(np.int32)

    kv_bytes, alg_bytes, flops = W.workload_bytes_flops(batch)
    hbm_time = alg_bytes / (HBM_PEAK_GBPS * 1e9)
    mfma_time = flops / (BF16_PEAK_TFLOPS * 1e12)
    roof_us = max(hbm_time, mfma_time) * 1e6
    hbm_bound = hbm_time >= mfma_time

    def pct(a, q):
        return round(float(np.percentile(a, q)), 2)

    cold_step, cold_att = np.median(cold_steps), np.median(cold_ph[:, 1])
    warm_att = float(warm_ph[:, 1].mean())
    us = float(cold_step)
    if hbm_bound:
        achieved = alg_bytes / (cold_att * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": None}
        measured_peak = peaks["stream_read_gbps"]
    else:
        achieved = flops / (cold_att * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": None}
        measured_peak = peaks["mfma_random_tflops"]
    traffic = measured_traffic(spec.name)
    if traffic is not None:
        roof["traffic"] = traffic["total_bytes"]
        roof["traffic_detail"] = traffic
    roof.update({
        "kernel": "attend_kernel",
        "kernel_avg_us": round(float(cold_att), 2),
        "kernel_timing": "median over the cold steps (events on the launch stream)",
        "frac_warm": round(roof_us / warm_att, 4),
        "kernel_avg_us_warm": round(warm_att, 2),
        "frac_whole_step": round(roof_us / us, 4),
        "frac_whole_step_warm": round(roof_us / float(np.mean(warm_ph[:, 3])), 4),
        "frac_of_measured_peak": round(roof["achieved"] / measured_peak, 4),
        "alg_bytes_per_launch": int(alg_bytes), "alg_flops_per_launch": int(flops),
        "roofline_us": round(roof_us, 1)})

    result = {
        "metric": METRIC,
        "value": round(us, 2),
        "unit": "us/step",
        "value_kind": "median step over the cold steps: one splash_mla_attend call (plan + attend + combine) "
                      "between two events, L2 and MALL flushed by a 1 GiB read before each, outside the events",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_run": warmup_run,
        "ms_per_step": round(us * 1e-3, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded PCG64 draws of the workload's length mix; N(0,1) cache rows and queries)",
        "config": {"workload": spec.name, "B": batch.B, "H": batch.H, "q_chunk": batch.q_chunk,
                   "lengths": list(spec.lengths), "kv_cache": W.KV_LABELS[batch.kv_dtype],
                   "qk": "bf16 MFMA" if batch.kv_dtype == W.KV_BF16 else (
                       "bf16 MFMA, K converted (exact)" if args.exact_qk else "fp8 MFMA, split query"),
                   "seed": spec.seed, "sum_seq_len": int(batch.seq_lens.sum()), "page_size": 64},
        "kv_gbps": round(kv_bytes / (us * 1e-6) / 1e9, 1),
        "alg_gbps": round(alg_bytes / (us * 1e-6) / 1e9, 1),
        "tflops": round(flops / (us * 1e-6) / 1e12, 1),
        "cold": {"step_us": {"p10": pct(cold_steps, 10), "p50": pct(cold_steps, 50),
                             "p90": pct(cold_steps, 90)},
                 "instrumented_step_us_median": round(float(np.median(cold_ph[:, 3])), 2),
                 "phases_us_median": {"plan": round(float(np.median(cold_ph[:, 0])), 2),
                                      "attend": round(float(cold_att), 2),
                                      "combine": round(float(np.median(cold_ph[:, 2])), 2)},
                 "wall_us_per_step_incl_flush": round(cold_wall_ms * 1e3, 2)},
        "warm": {"wall_us_per_step": round(warm_ms * 1e3, 2),
                 "step_event_us": {"mean": round(float(warm_ph[:, 3].mean()), 2), "p10": pct(warm_ph[:, 3], 10),
                                   "p50": pct(warm_ph[:, 3], 50), "p90": pct(warm_ph[:, 3], 90)},
                 "phases_us_mean": {"plan": round(float(warm_ph[:, 0].mean()), 2),
                                    "attend": round(warm_att, 2),
                                    "combine": round(float(warm_ph[:, 2].mean()), 2)}},
        "plan": {"kind": "fold" if int(hdr[9]) > 0 else "unit size",
                 "units": int(hdr[1]), "partials": int(hdr[2]), "pages_per_unit": int(hdr[3]),
                 "fold_cap_pages": int(hdr[10]), "split_tiles": int(hdr[6]), "workers": B.device_workers()},
        "measured_peaks": peaks,
        "roofline": roof,
    }
    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = 1 << 30
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(batch, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def measured_peaks(torch, stream):
    """Streaming-read bandwidth (1 GiB, non-temporal 16-byte loads, best of
    five) and bf16 MFMA rate on random N(0,1) operands (every CU, four
    chains per wave, best of three), from the calibration library."""
    import numpy as np
    G = B.device_workers()
    buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    buf.zero_()
    sink = torch.empty(4 * G * 1024, dtype=torch.uint8, device="cuda")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    best_read = 0.0
    for _ in range(5):
        ev[0].record(stream)
        CAL.stream_read(buf, sink, 2 * G, stream)
        ev[1].record(stream)
        torch.cuda.synchronize()
        best_read = max(best_read, (1 << 30) / (ev[0].elapsed_time(ev[1]) * 1e-3) / 1e9)
    del buf
    ops_bytes = CAL.mfma_ops_bytes(G)
    g = torch.Generator(device="cuda").manual_seed(0)
    ops = torch.randn(ops_bytes // 2, generator=g, device="cuda").to(torch.bfloat16)
    iters = 1000
    best_mfma = 0.0
    for _ in range(3):
        ev[0].record(stream)
        CAL.mfma_loop(ops, iters, sink, G, stream)
        ev[1].record(stream)
        torch.cuda.synchronize()
        best_mfma = max(best_mfma, CAL.mfma_flops(G, iters) / (ev[0].elapsed_time(ev[1]) * 1e-3) / 1e12)
    return {"stream_read_gbps": round(best_read, 1), "mfma_random_tflops": round(best_mfma, 1),
            "how": "streaming read of 1 GiB (2 x CUs workgroups, best of 5); bf16 32x32x16 MFMA loop on "
                   "random N(0,1) operands on every CU (best of 3)"}


if __name__ == "__main__":
    main()
