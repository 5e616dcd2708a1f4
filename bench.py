"""Benchmark: dynamic block-sparse attention request (plan + forward) on one MI355X.

A step is one complete request on resident inputs: bsa_plan (mask state,
statistics copy, regime lookup, launch preparation) followed by bsa_forward
(attention kernel and, for Split-K plans, the merge), ending when the stream
is idle.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload c2_window15]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA, 256 CU x 4096 flop/clk x 2.4 GHz
PEAK_HBM_GBS = 8000.0


FLUSH_BYTES = 512 << 20
KERNEL_SRC = os.path.join(HERE, "paper_2609_25869_amd", "csrc", "attn_fwd.hip")
ORDER_SRC = os.path.join(HERE, "paper_2609_25869_amd", "csrc", "task_order.hip")  # dispatch order: sets L2 reuse
SLOTMAP_SRC = os.path.join(HERE, "paper_2609_25869_amd", "csrc", "slot_map.h")  # which XCD runs which task
TRAFFIC_FILE = os.path.join(HERE, "profiles", "attn_fwd_c2_window15_traffic.md")


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def effective_flops(mask, d):
    """4*d per token pair of E(M) (Section 2.3 accounting), summed over the mask."""
    total = 0
    for b in range(mask.B):
        for h in range(mask.H):
            m = mask.head(b, h) != 0
            bq, bkv = int(mask.bq[h]), int(mask.bkv[h])
            rows = np.full(m.shape[0], bq, dtype=np.int64)
            rows[-1] = mask.nq - (m.shape[0] - 1) * bq
            cols = np.full(m.shape[1], bkv, dtype=np.int64)
            cols[-1] = mask.nkv - (m.shape[1] - 1) * bkv
            total += int(rows @ m.astype(np.int64) @ cols)
    return 4 * d * total


def gemm_probe(torch, n=16384, reps=5, batches=3):
    """A practical bf16 MFMA ceiling on this machine: a large, contiguous
    n x n x n bf16 matrix product through the vendor GEMM library (fp32
    accumulate), timed with HIP events after warm-up; the best of `batches`
    batches of `reps` products.  Returns TFLOP/s."""
    a = torch.randn((n, n), device="cuda", dtype=torch.float32).to(torch.bfloat16)
    b = torch.randn((n, n), device="cuda", dtype=torch.float32).to(torch.bfloat16)
    c = torch.empty((n, n), device="cuda", dtype=torch.bfloat16)
    for _ in range(2):
        torch.matmul(a, b, out=c)
    best = float("inf")
    for _ in range(batches):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            torch.matmul(a, b, out=c)
        e1.record()
        e1.synchronize()
        best = min(best, e0.elapsed_time(e1) / reps)
    del a, b, c
    return 2.0 * n ** 3 / (best * 1e-3) / 1e12


def copy_probe(torch, mib):
    """A plain device-to-device copy of known size, for scaling FETCH_SIZE / WRITE_SIZE."""
    n = (mib << 20) // 4
    src = torch.ones(n, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n * 4, "launches": 5}), flush=True)


def measured_traffic(workload, plan_ids):
    """HBM bytes per launch of the attention kernel from the committed counter summary.

    Reported only when that summary was taken on this workload and plan with
    the current kernel, slot-map and dispatch-order sources; otherwise None.
    """
    import hashlib
    if not os.path.exists(TRAFFIC_FILE):
        return None
    text = open(TRAFFIC_FILE).read()
    a = text.find("```json")
    if a < 0:
        return None
    rec = json.loads(text[a + 7:text.index("```", a + 7)])
    src_hash = hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()
    order_hash = hashlib.sha256(open(ORDER_SRC, "rb").read()).hexdigest()
    slot_hash = hashlib.sha256(open(SLOTMAP_SRC, "rb").read()).hexdigest()
    if rec.get("workload") != workload or rec.get("plan_ids") != plan_ids or rec.get("attn_fwd_sha256") != src_hash \
            or rec.get("task_order_sha256") != order_hash or rec.get("slot_map_sha256") != slot_hash:
        return None
    return rec["hbm_bytes_per_launch"]


def cpu_baseline(q, k, v, mask, eff_flops_total, budget_s, seed=1234):
    """Time the fp64 oracle on a seeded sample of query rows of the same workload."""
    from oracle import attn as oattn
    rng = np.random.default_rng(seed)
    B, Nq, H, d = q.shape
    # active keys per query row, to count the sample's effective flops
    def row_flops(rows):
        f = 0
        for b, h, i in rows:
            m = mask.head(b, h)
            bq, bkv = int(mask.bq[h]), int(mask.bkv[h])
            act = np.nonzero(m[i // bq])[0]
            widths = np.minimum((act + 1) * bkv, mask.nkv) - act * bkv
            f += 4 * d * int(widths.sum())
        return f

    def draw(n):
        return np.stack([rng.integers(0, B, n), rng.integers(0, H, n), rng.integers(0, Nq, n)], axis=1)

    # batches of rows until the budget is spent (the first batch also warms the thread pool)
    n, done, dt, f = 128, 0, 0.0, 0
    while dt < budget_s:
        rows = draw(n)
        t0 = time.perf_counter()
        oattn.masked_attention(q, k, v, mask, rows=rows)
        t = time.perf_counter() - t0
        dt += t
        f += row_flops(rows)
        done += n
        if t < 2.0:
            n *= 2
    return {
        "value": f / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": oattn.num_threads(),
        "kind": "oracle",
        "sample": "%d seeded random query rows of the same workload (%.3g of %d rows, %.3g effective GFLOP), "
                  "fp64 C oracle, %.1f s" % (done, done / (B * H * Nq), B * H * Nq, f / 1e9, dt),
        "seconds": dt,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c2_window15")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gemm-probe", action="store_true", help="skip the vendor-GEMM ceiling probe")
    ap.add_argument("--force-plan", type=int, default=-1)
    ap.add_argument("--no-flush", action="store_true", help="skip the cache-evicting write before each step")
    ap.add_argument("--sparsify", action="store_true",
                    help="top-k workloads: build the mask on the device inside every request "
                         "(bsa_sparsify_topk -> bsa_plan -> bsa_forward) instead of reading a resident one")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (HBM counter calibration) and exit")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the block-sparse request path runs within a single device; "
              "multi-GPU runs are not part of this build (got --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe:
        copy_probe(torch, args.copy_probe)
        return
    import paper_2609_25869_amd as bsa
    from workloads import CONFIGS, make_mask, make_qkv

    cfg = CONFIGS[args.workload]
    t0 = time.perf_counter()
    q, k, v = make_qkv(cfg)
    mask = make_mask(cfg, q, k)
    log("generated %s in %.1f s" % (cfg.name, time.perf_counter() - t0))
    d = cfg.d
    eff = effective_flops(mask, d)

    dev = torch.device("cuda:0")
    to_dev = lambda x: torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev)
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    od = torch.empty_like(qd)
    lse = torch.empty((cfg.B, cfg.H, cfg.N), dtype=torch.float32, device=dev)
    md = torch.from_numpy(mask.data).to(dev)
    shapes = bsa.shapes_of(qd, kd, vd, od)
    topk = None
    if args.sparsify:
        if cfg.kind != "topk":
            print("--sparsify applies to the top-k workloads only", file=sys.stderr)
            sys.exit(2)
        bq0, bkv0 = cfg.geometry[0]
        topk = int(np.floor(cfg.params["frac"] * (-(-cfg.N // bkv0)) + 0.5))
        dev_mask = bsa.sparsify_topk(qd, kd, bq0, bkv0, topk)
        torch.cuda.synchronize()
        # the device sparsifier reproduces the workload's mask recipe; report any difference
        n_diff = int((dev_mask.cpu().numpy().reshape(-1) != mask.data.reshape(-1)).sum())
        log("device sparsifier: %d of %d mask entries differ from the workload mask" % (n_diff, mask.data.size))
    per_head = not mask.uniform_geometry
    bq = [int(x) for x in mask.bq] if per_head else int(mask.bq[0])
    bkv = [int(x) for x in mask.bkv] if per_head else int(mask.bkv[0])
    stream = torch.cuda.current_stream()
    # written before every step so that each request starts with the inputs
    # out of the L2 and last-level caches (512 MiB is twice the MALL)
    flush = None if args.no_flush else torch.empty(FLUSH_BYTES // 4, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()

    sp_ms = []

    def evict_caches():
        # outside the request: the write and its completion precede the timer
        if flush is not None:
            flush.fill_(1)
        torch.cuda.synchronize()

    def request():
        if topk is not None:
            s0 = torch.cuda.Event(enable_timing=True)
            s1 = torch.cuda.Event(enable_timing=True)
            s0.record(stream)
            bsa.sparsify_topk(qd, kd, cfg.geometry[0][0], cfg.geometry[0][1], topk, mask=md.view(dev_mask.shape),
                              stream=stream)
            s1.record(stream)
            sp_ms.append((s0, s1))
        p = bsa.plan(md, bq, bkv, shapes, head_offset=list(mask.head_offset), stride_b=mask.stride_b,
                     force_plan=args.force_plan, stream=stream)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        bsa.forward(p, qd, kd, vd, od, lse, stream=stream)
        e1.record(stream)
        return p, e0, e1

    for _ in range(args.warmup):
        evict_caches()
        p, _, _ = request()
        torch.cuda.synchronize()
        p.destroy()

    # K timed steps, each a complete request between two synchronisations;
    # the timed region is their sum
    req_ms, kern = [], []
    for _ in range(args.steps):
        evict_caches()
        t1 = time.perf_counter()
        p, e0, e1 = request()
        stream.synchronize()
        req_ms.append((time.perf_counter() - t1) * 1e3)
        kern.append((e0, e1))
        if _ < args.steps - 1:
            p.destroy()
    torch.cuda.synchronize()
    total_s = sum(req_ms) * 1e-3
    kernel_ms = [a.elapsed_time(b) for a, b in kern]
    info = [p.info(s) for s in range(p.num_segments())]

    # warm exact repeats: forward on the kept plan
    warm = []
    for _ in range(max(3, args.steps // 2)):
        t1 = time.perf_counter()
        bsa.forward(p, qd, kd, vd, od, lse, stream=stream)
        stream.synchronize()
        warm.append((time.perf_counter() - t1) * 1e3)
    p.destroy()

    ms_per_step = total_s * 1e3 / args.steps
    k_avg = float(np.mean(kernel_ms))
    kernel_tflops = eff / (k_avg * 1e-3) / 1e12
    executed = sum(4 * d * i["n_tiles"] * i["tq"] * i["tkv"] for i in info)   # MFMA work incl. masked entries
    tiles_bytes = sum(4 * d * i["n_tiles"] * i["tkv"] for i in info)   # K/V bytes streamed, bf16
    traffic = measured_traffic(cfg.name, [i["plan_id"] for i in info])
    out = {
        "metric": "effective active-block TFLOP/s + request latency incl. planning, 1x MI355X",
        "value": eff / (ms_per_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Philox normals; 3D-window block mask standing in for the paper's vDiT masks)",
        "config": {
            "workload": cfg.name,
            "description": cfg.description,
            "batch": cfg.B, "heads": cfg.H, "seq_len": cfg.N, "head_dim": d,
            "block": [int(mask.bq[0]), int(mask.bkv[0])],
            "density": float(mask.data.mean()),
            "effective_gflop": eff / 1e9,
            "parallelism": "single GPU",
        },
        "request_ms": {"median": float(np.median(req_ms)), "p95": float(np.percentile(req_ms, 95)),
                       "cache_flush_before_each_step": flush is not None,
                       "warm_median": float(np.median(warm))},
        "kernel_ms": {"mean": k_avg, "median": float(np.median(kernel_ms)),
                      "p95": float(np.percentile(kernel_ms, 95))},
        "kernel_tflops": kernel_tflops,
        "executed_kernel_tflops": executed / (k_avg * 1e-3) / 1e12,
        "plans": [{k2: i[k2] for k2 in ("plan_id", "tq", "tkv", "split", "mapping_name", "regime_hit", "n_tasks",
                                          "n_tiles")} for i in info],
        "roofline": {
            "bound": "mfma",
            "kernel": "attn_fwd_kernel (bsa_forward)",
            "achieved": kernel_tflops,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": kernel_tflops / PEAK_BF16_TFLOPS,
            "traffic": traffic,
            "kv_stream_gbs": tiles_bytes / (k_avg * 1e-3) / 1e9,
        },
    }
    if topk is not None:
        sp = [a.elapsed_time(b) for a, b in sp_ms[-args.steps:]]
        out["sparsify_ms"] = {"mean": float(np.mean(sp)), "median": float(np.median(sp)), "topk": topk,
                              "in_request": True}
    # outside the timed region: the practical MFMA ceiling of this machine
    if not args.no_gemm_probe:
        probe = gemm_probe(torch)
        out["roofline"]["gemm_probe"] = {"tflops": probe, "frac": kernel_tflops / probe,
                                         "what": "16384^3 bf16 torch.matmul (vendor GEMM), best of 3 batches of 5, "
                                                 "HIP events"}
    if not args.no_cpu_baseline:
        log("timing the CPU oracle (about %.0f s)" % args.cpu_budget)
        out["cpu_baseline"] = cpu_baseline(q, k, v, mask, eff, args.cpu_budget)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
