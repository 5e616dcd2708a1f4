"""Host-side pieces of bench.py: the effective-flop count and the gate on the
committed traffic record (no GPU)."""
import hashlib
import importlib.util
import json
import os

import numpy as np

from workloads import random_case

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_host", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_effective_flops_counts_token_pairs_of_active_blocks():
    bench = _bench()
    # ragged tails on both sides, two geometries, N_q != N_kv
    _, _, _, mask = random_case(7, 2, 2, 333, 517, 8, [(64, 32), (32, 128)], 0.3, diag=False, empty_rows=1)
    pairs = 0
    for b in range(mask.B):
        for h in range(mask.H):
            m = mask.head(b, h) != 0
            bq, bkv = int(mask.bq[h]), int(mask.bkv[h])
            for i in range(mask.nq):            # token-level expansion, brute force
                row = m[i // bq]
                pairs += sum(1 for j in range(mask.nkv) if row[j // bkv])
    assert bench.effective_flops(mask, 128) == 4 * 128 * pairs


def test_traffic_record_is_used_only_for_its_kernel_workload_and_plan():
    bench = _bench()
    text = open(bench.TRAFFIC_FILE).read()
    rec = json.loads(text[text.index("```json") + 7:text.index("```", text.index("```json") + 7)])
    src = hashlib.sha256(open(bench.KERNEL_SRC, "rb").read()).hexdigest()
    order = hashlib.sha256(open(bench.ORDER_SRC, "rb").read()).hexdigest()
    got = bench.measured_traffic(rec["workload"], rec["plan_ids"])
    if rec["attn_fwd_sha256"] == src and rec.get("task_order_sha256") == order:
        assert got == rec["hbm_bytes_per_launch"] and got > 0
    else:
        assert got is None   # the kernel or the dispatch order changed since the counters were taken
    assert bench.measured_traffic(rec["workload"], [p + 1 for p in rec["plan_ids"]]) is None
    assert bench.measured_traffic("another_workload", rec["plan_ids"]) is None
