"""Offline profiling of the plan catalog on MI355X (Section 5.1, Algorithm 1).

Runs every eligible catalog plan on a corpus of seeded synthetic masks and
records, per case, the request key, the regime features the online path will
see (the library's own mask statistics) and the kernel latency of each plan
whose output passed validation (``kernel_time``: the median of three timed
batches; launches shorter than a millisecond are timed as batches of
back-to-back launches, so event and launch jitter average out).  The output is one JSON line per case;
``compile.py`` turns those lines into the plan table.

Validation (Algorithm 1 keeps only plans whose output passes): every plan's
output must be finite everywhere and, on 64 seeded query rows per case, agree
within 2e-2 absolute with masked attention evaluated from its definition
(Eq. 1) in fp32 on the device: the row's active keys gathered from the
logical mask, softmax of their scaled scores, the weighted sum of their
values, and zero for a row with no active key.

Corpus (the paper's profiling masks are not available; these stand in):
  geometries: the nine logical geometries of the paper's workloads plus the
  alternating (128,32) / (32,128) pair; sequence lengths 16K, 64K and 115K
  tokens; 4 or 24 (batch x heads); masks from three families at several
  densities -- frame-window masks (long runs, like spatiotemporal windows),
  Bernoulli masks with the diagonal (few runs) and per-row top-k of pooled
  q.k block scores with the diagonal.  Inputs are N(0,1) in bf16.  The
  wide, mixture and large splits widen this grid (see their constants).

    python -m paper_2609_25869_amd.lut.profile --out PATH [--split profile|eval] [--budget SECONDS]

Plans added to the catalog later (or whose launch changed) are timed into
existing records and then put on each split's original clock:

    python -m paper_2609_25869_amd.lut.profile --split S --add-plans 30,31 --base gfx950_S.jsonl --out NEW
    python -m paper_2609_25869_amd.lut.profile --out NEW --finalize
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

GEOMETRIES = [(128, 128), (128, 64), (64, 64), (64, 32), (32, 32), (32, 16), (16, 16), (128, 32), (32, 128)]
SEQ_LENS = [16384, 65536, 115200]
BATCH_HEADS = [4, 24]
FAMILIES = [("window", 0.05), ("window", 0.15), ("bernoulli", 0.03), ("bernoulli", 0.10), ("bernoulli", 0.30),
            ("topk", 0.12)]
SPLIT_SEED = {"profile": 0, "eval": 1, "wide": 2, "wide_eval": 3, "mixture": 4, "mixture_eval": 5, "large": 6,
              "large_eval": 7, "grid2": 8}
FRAMES = 16

# The wide splits draw, per request key, random combinations of a larger
# grid: short and long sequences, few and many heads, twelve mask sources.
WIDE_SEQ = [2048, 4096, 8192, 16384, 32768, 65536, 115200]
WIDE_BH = [1, 2, 4, 8, 24]
WIDE_SOURCES = [("window", 0.03), ("window", 0.08), ("window", 0.15), ("window", 0.30),
                ("bernoulli", 0.02), ("bernoulli", 0.05), ("bernoulli", 0.10), ("bernoulli", 0.20),
                ("bernoulli", 0.40), ("topk", 0.06), ("topk", 0.12), ("topk", 0.25)]
WIDE_PER_KEY = {"wide": 96, "wide_eval": 48}

# The mixture splits: requests whose heads draw their masks from different
# families (window 40%, top-k 40%, Bernoulli 20%) at densities from
# {2, 5, 10, 25, 50}%, per head, as in a model whose heads attend
# differently; long sequences and many heads.
MIX_SEQ = [16384, 32768, 65536, 115200, 131072]
MIX_BH = [8, 24, 48]
MIX_PER_KEY = {"mixture": 12, "mixture_eval": 6}
MIX_FAMILIES = [("window", 0.4), ("topk", 0.4), ("bernoulli", 0.2)]
MIX_RHO = [0.02, 0.05, 0.10, 0.25, 0.50]

# The large splits: the request sizes of video generation (64K to 131K
# tokens, 8 to 48 batch x heads), each case drawing one of the twelve wide
# sources or a per-head mixture (a quarter of the cases).
LARGE_SEQ = [65536, 98304, 115200, 131072]
LARGE_BH = [8, 16, 24, 48]
LARGE_SOURCES = WIDE_SOURCES + [("mixture", 0.0)] * 4
LARGE_PER_KEY = {"large": 12, "large_eval": 6}

# The second grid split (held out): the grid split's geometries and
# sources at the batch x heads between its two (8 and 16), from 32K to 115K
# tokens.
GRID2_SEQ = [32768, 65536, 115200]
GRID2_BH = [8, 16]


def log(msg):
    print("[profile] " + msg, flush=True)


def corpus(split):
    """The deterministic case list of one split."""
    cases = []
    if split in MIX_PER_KEY:
        import random
        rng = random.Random(1000 + SPLIT_SEED[split])
        for geom in GEOMETRIES:
            for _ in range(MIX_PER_KEY[split]):
                cases.append(dict(id="%s-%d" % (split, len(cases)), geometry=list(geom), N=rng.choice(MIX_SEQ),
                                  bh=rng.choice(MIX_BH), family="mixture", rho=0.0, seed=rng.randrange(1 << 30)))
        return cases
    if split in LARGE_PER_KEY:
        import random
        rng = random.Random(1000 + SPLIT_SEED[split])
        for geom in GEOMETRIES:
            for _ in range(LARGE_PER_KEY[split]):
                fam, rho = rng.choice(LARGE_SOURCES)
                cases.append(dict(id="%s-%d" % (split, len(cases)), geometry=list(geom), N=rng.choice(LARGE_SEQ),
                                  bh=rng.choice(LARGE_BH), family=fam, rho=rho, seed=rng.randrange(1 << 30)))
        return cases
    if split in WIDE_PER_KEY:
        import random
        rng = random.Random(1000 + SPLIT_SEED[split])
        for gi, geom in enumerate(GEOMETRIES):
            for _ in range(WIDE_PER_KEY[split]):
                fam, rho = rng.choice(WIDE_SOURCES)
                cases.append(dict(id="%s-%d" % (split, len(cases)), geometry=list(geom), N=rng.choice(WIDE_SEQ),
                                  bh=rng.choice(WIDE_BH), family=fam, rho=rho, seed=rng.randrange(1 << 30)))
        return cases
    seqs, bhs = (GRID2_SEQ, GRID2_BH) if split == "grid2" else (SEQ_LENS, BATCH_HEADS)
    for gi, geom in enumerate(GEOMETRIES):
        for N in seqs:
            for bh in bhs:
                for fi, (fam, rho) in enumerate(FAMILIES):
                    seed = ((SPLIT_SEED[split] * 16 + gi) * 8 + seqs.index(N)) * 64 + bhs.index(bh) * 8 + fi
                    cases.append(dict(id="%s-%d" % (split, len(cases)), geometry=list(geom), N=N, bh=bh, family=fam,
                                      rho=rho, seed=seed))
    return cases


def make_mask(torch, case, q, k):
    """[bh, nqb, nkb] uint8 mask for the case, built on the device."""
    bq, bkv = case["geometry"]
    N, bh, rho = case["N"], case["bh"], case["rho"]
    nqb, nkb = -(-N // bq), -(-N // bkv)
    dev = q.device
    g = torch.Generator(device=dev)
    g.manual_seed(case["seed"])
    cq = (torch.arange(nqb, device=dev, dtype=torch.float64) + 0.5) * bq
    ck = (torch.arange(nkb, device=dev, dtype=torch.float64) + 0.5) * bkv
    diag = (torch.arange(nqb, device=dev)[:, None] * bq < (torch.arange(nkb, device=dev)[None, :] + 1) * bkv) & \
           (torch.arange(nkb, device=dev)[None, :] * bkv < (torch.arange(nqb, device=dev)[:, None] + 1) * bq)
    out = torch.empty((bh, nqb, nkb), dtype=torch.uint8, device=dev)
    if case["family"] == "mixture":
        import random
        pick = random.Random(case["seed"])
        for h in range(bh):
            u, acc, fam = pick.random(), 0.0, MIX_FAMILIES[-1][0]
            for name, w in MIX_FAMILIES:
                acc += w
                if u < acc:
                    fam = name
                    break
            rho = pick.choice(MIX_RHO)
            one = dict(case, family=fam, rho=rho, bh=1, seed=pick.randrange(1 << 30))
            out[h] = make_mask(torch, one, q[:, :, h:h + 1, :], k[:, :, h:h + 1, :])[0]
        return out
    if case["family"] == "window":
        # tokens as FRAMES frames of N/FRAMES positions; active when the block
        # centres are within one frame and within a spatial half-width w
        F = N / FRAMES
        fq, fk = torch.floor(cq / F), torch.floor(ck / F)
        sq, sk = cq - fq * F, ck - fk * F
        w = rho * FRAMES / 3.0 * F / 2.0
        for h in range(bh):
            jitter = float(torch.rand(1, generator=g, device=dev).item()) * 0.2 + 0.9
            m = ((fq[:, None] - fk[None, :]).abs() <= 1) & ((sq[:, None] - sk[None, :]).abs() <= w * jitter)
            out[h] = (m | diag).to(torch.uint8)
    elif case["family"] == "bernoulli":
        for h in range(bh):
            m = torch.rand((nqb, nkb), generator=g, device=dev) < rho
            out[h] = (m | diag).to(torch.uint8)
    else:
        kk = max(1, int(math.floor(rho * nkb + 0.5)))
        for h in range(bh):
            pq = q[0, :nqb * bq, h, :].float().reshape(nqb, bq, -1).mean(1) if N % bq == 0 else \
                torch.stack([q[0, i * bq:min(N, (i + 1) * bq), h, :].float().mean(0) for i in range(nqb)])
            pk = k[0, :nkb * bkv, h, :].float().reshape(nkb, bkv, -1).mean(1) if N % bkv == 0 else \
                torch.stack([k[0, i * bkv:min(N, (i + 1) * bkv), h, :].float().mean(0) for i in range(nkb)])
            idx = torch.topk(pq @ pk.T, kk, dim=1).indices
            m = torch.zeros((nqb, nkb), dtype=torch.bool, device=dev)
            m.scatter_(1, idx, True)
            out[h] = (m | diag).to(torch.uint8)
    return out


BATCH_MS = 1.0   # a timed batch of short launches lasts about this long
MAX_BATCH = 64


def kernel_time(torch, stream, launch, reps=3):
    """Kernel time of one launch (ms): one warm-up launch sizes a batch of
    back-to-back launches lasting about BATCH_MS; the median over `reps`
    batches of the mean per launch (HIP events around each batch).  Kernels
    longer than BATCH_MS are timed one launch per batch."""
    def batch(n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n):
            launch()
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) / n
    first = batch(1)
    n = max(1, min(MAX_BATCH, int(math.ceil(BATCH_MS / max(first, 1e-3)))))
    ts = sorted(batch(n) for _ in range(reps))
    return ts[len(ts) // 2]


def reference_rows(torch, q, k, v, mask, bq, bkv, rows):
    """Masked attention (Eq. 1) for query rows [(h, i), ...] of batch 0, in
    fp32, from the logical mask: a plain per-row evaluation, independent of
    every plan."""
    N = q.shape[1]
    out = torch.zeros((len(rows), q.shape[3]), dtype=torch.float32, device=q.device)
    scale = 1.0 / math.sqrt(q.shape[3])
    for r, (h, i) in enumerate(rows):
        blocks = torch.nonzero(mask[h, i // bq]).flatten()
        if blocks.numel() == 0:
            continue
        keys = (blocks[:, None] * bkv + torch.arange(bkv, device=q.device)[None, :]).flatten()
        keys = keys[keys < N]
        s = (k[0, keys, h, :].float() @ q[0, i, h, :].float()) * scale
        out[r] = torch.softmax(s, 0) @ v[0, keys, h, :].float()
    return out


def profile_case(torch, bsa, case, reps=3, only=None):
    bq, bkv = case["geometry"]
    N, bh = case["N"], case["bh"]
    dev = torch.device("cuda")
    g = torch.Generator(device=dev)
    g.manual_seed(case["seed"] + 7)
    q = torch.randn((1, N, bh, 128), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    k = torch.randn((1, N, bh, 128), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    v = torch.randn((1, N, bh, 128), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    mask = make_mask(torch, case, q, k)
    nqb, nkb = mask.shape[1], mask.shape[2]
    head_offset = [h * nqb * nkb for h in range(bh)]
    shapes = bsa.shapes_of(q, k, v, q)
    o = torch.empty_like(q)
    stream = torch.cuda.current_stream()
    base = bsa.base_plan(bq, bkv)
    plans = [e["id"] for e in bsa.catalog() if bsa.plan_eligible(e["id"], bq, bkv, shapes)]
    plans = [base] + [p for p in plans if p != base]
    if only is not None:
        plans = [p for p in plans if p in only]
    rng = torch.Generator()
    rng.manual_seed(case["seed"] + 11)
    rows = [(int(h), int(i)) for h, i in zip(torch.randint(0, bh, (64,), generator=rng).tolist(),
                                             torch.randint(0, N, (64,), generator=rng).tolist())]
    ref = reference_rows(torch, q, k, v, mask, bq, bkv, rows)
    ri = torch.tensor([i for _, i in rows], device=dev)
    rh = torch.tensor([h for h, _ in rows], device=dev)
    lat, invalid, feats = {}, [], None
    for pid in plans:
        try:
            p = bsa.plan(mask, bq, bkv, shapes, head_offset=head_offset, stride_b=0, force_plan=pid, stream=stream)
        except bsa.BsaError as e:   # e.g. a Split-K workspace that does not fit
            log("  plan %d not run: %s" % (pid, e))
            invalid.append(pid)
            continue
        if feats is None:
            info = p.info(0)
            feats = {"seq_q": N, "seq_kv": N, "batch_heads": bh, "nnz": info["nnz"], "blocks": info["blocks"],
                     "run_blocks": info["run_blocks"], "max_row_nnz": info["max_row_nnz"]}
        t = kernel_time(torch, stream, lambda: bsa.forward(p, q, k, v, o, None, stream=stream), reps)
        p.destroy()
        ok = bool(torch.isfinite(o).all().item())
        if ok:
            ok = float((o[0, ri, rh, :].float() - ref).abs().max().item()) <= 2e-2
        if ok:
            lat[pid] = t
        else:
            invalid.append(pid)
    del q, k, v, o, mask, ref
    return {"id": case["id"], "key": [bq, bkv, 0, 128], "family": case["family"], "rho": case["rho"],
            "features": feats, "latency_ms": {str(p): t for p, t in lat.items()}, "invalid": invalid}


def case_features(torch, bsa, case):
    """The regime features of a case alone (mask statistics from bsa_plan
    with the base plan), without timing any plan."""
    bq, bkv = case["geometry"]
    N, bh = case["N"], case["bh"]
    dev = torch.device("cuda")
    g = torch.Generator(device=dev)
    g.manual_seed(case["seed"] + 7)
    q = torch.randn((1, N, bh, 128), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    k = torch.randn((1, N, bh, 128), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    mask = make_mask(torch, case, q, k)
    nqb, nkb = mask.shape[1], mask.shape[2]
    p = bsa.plan(mask, bq, bkv, bsa.shapes_of(q, k, k, q), head_offset=[h * nqb * nkb for h in range(bh)],
                 stride_b=0, force_plan=bsa.base_plan(bq, bkv))
    info = p.info(0)
    p.destroy()
    return {"seq_q": N, "seq_kv": N, "batch_heads": bh, "nnz": info["nnz"], "blocks": info["blocks"],
            "run_blocks": info["run_blocks"], "max_row_nnz": info["max_row_nnz"]}


def refeature(args):
    """Add max_row_nnz to the records of a split profiled before it was
    recorded: the masks are regenerated from the case seeds, and the other
    statistics must come out as recorded."""
    import torch
    import paper_2609_25869_amd as bsa
    by_id = {c["id"]: c for c in corpus(args.split)}
    recs = [json.loads(l) for l in open(args.out) if l.strip()]
    t0 = time.time()
    for r in recs:
        if "max_row_nnz" in (r["features"] or {}):
            continue
        f = case_features(torch, bsa, by_id[r["id"]])
        old = r["features"]
        assert all(f[k] == old[k] for k in old), (r["id"], old, f)
        r["features"] = f
    with open(args.out + ".tmp", "w") as fo:
        for r in recs:
            fo.write(json.dumps(r) + "\n")
    os.replace(args.out + ".tmp", args.out)
    log("refeatured %d records of %s in %.1f s" % (len(recs), args.split, time.time() - t0))


def add_plans(args):
    """Time plans added to the catalog after a split was profiled (or plans
    whose kernels or launch changed since), and merge them into its records
    (--base, written to --out).  Every case re-times the two fastest
    recorded plans outside the timed set beside them and keeps the geometric
    mean of recorded / re-timed over those reference plans (`scale`) with the
    raw latencies; `finalize_added` then puts the new latencies on the clock
    the split was first profiled at.  The regenerated mask must give the
    recorded statistics.  (Passes for plans 30-34 took the fastest recorded
    plan and the base plan as references.)"""
    import torch
    import paper_2609_25869_amd as bsa
    new = [int(x) for x in args.add_plans.split(",")]
    by_id = {c["id"]: c for c in corpus(args.split)}
    recs = [json.loads(l) for l in open(args.base) if l.strip()]
    done = set()
    if os.path.exists(args.out):
        done = {json.loads(l)["id"] for l in open(args.out) if l.strip()}
    todo = [r for r in recs if r["id"] not in done]
    log("%d cases to extend with plans %s (%d already in %s)" % (len(todo), new, len(done), args.out))
    t0 = time.time()
    with open(args.out, "a") as f:
        for i, rec in enumerate(todo):
            if time.time() - t0 > args.budget:
                log("budget reached after %d cases" % i)
                break
            tc = time.time()
            case = by_id[rec["id"]]
            old = rec["latency_ms"]
            # the reference plans: the two fastest recorded plans outside the
            # timed set (a plan timed again because its kernel changed cannot
            # measure the box)
            outside = sorted((p for p in old if int(p) not in new), key=lambda p: old[p])
            refs = sorted(outside[:2], key=int)
            r = profile_case(torch, bsa, case, only=set(new) | {int(p) for p in refs})
            assert all(r["features"][k] == v for k, v in rec["features"].items()), (rec["id"], rec["features"])
            got = [old[p] / r["latency_ms"][p] for p in refs if p in r["latency_ms"]]
            scale = math.exp(sum(math.log(x) for x in got) / len(got)) if got else 1.0
            raw = {}
            for p in new:
                if str(p) in r["latency_ms"]:
                    raw[str(p)] = r["latency_ms"][str(p)]
                    old[str(p)] = raw[str(p)] * scale
                elif p in r["invalid"] and p not in rec["invalid"]:
                    rec["invalid"].append(p)
            entry = {"plans": new, "refs": [int(p) for p in refs], "scale": scale, "raw": raw,
                     "ref_ms": min(old[p] for p in refs) if refs else 0.0}
            prev = rec.get("added")
            rec["added"] = (prev if isinstance(prev, list) else [prev] if prev else []) + [entry]
            f.write(json.dumps(rec) + "\n")
            f.flush()
            log("%s: scale %.4f, %s (%.1f s)" % (rec["id"], scale, ", ".join(
                "%d %.3f" % (p, old[str(p)]) for p in new if str(p) in old), time.time() - tc))
            torch.cuda.empty_cache()
    log("done in %.1f s" % (time.time() - t0))


FINALIZE_MIN_MS = 0.5


def finalize_added(path):
    """One clock factor per pass of --add-plans over a split (one pass runs on
    one box): the geometric mean of the per-case reference ratios over the
    cases whose reference kernels take at least FINALIZE_MIN_MS, where timing
    noise is small.  Each added latency becomes its raw time times that
    factor; per-case ratios of short kernels are too noisy to scale by alone.
    Entries written before raw times were kept carry them implicitly as the
    stored latency divided by the per-case scale."""
    recs = [json.loads(l) for l in open(path) if l.strip()]
    npass = max((len(r["added"]) if isinstance(r.get("added"), list) else 1) for r in recs)
    for k in range(npass):
        logs = []
        for r in recs:
            e = r["added"][k] if isinstance(r["added"], list) else r["added"]
            ref_ms = e.get("ref_ms")
            if ref_ms is None:
                ref_ms = min(r["latency_ms"][str(p)] for p in e["refs"]) if e["refs"] else 0.0
                e["ref_ms"] = ref_ms
            if ref_ms >= FINALIZE_MIN_MS and e["scale"] > 0:
                logs.append(math.log(e["scale"]))
        factor = math.exp(sum(logs) / len(logs)) if logs else 1.0
        for r in recs:
            e = r["added"][k] if isinstance(r["added"], list) else r["added"]
            if "raw" not in e:
                e["raw"] = {str(p): r["latency_ms"][str(p)] / e["scale"] for p in e["plans"] if str(p) in r["latency_ms"]}
            for p, t in e["raw"].items():
                r["latency_ms"][p] = t * factor
            e["factor"] = factor
        log("%s pass %d: factor %.4f from %d of %d cases" % (path, k, factor, len(logs), len(recs)))
    with open(path + ".tmp", "w") as f:
        for r in recs:
            f.write(json.dumps(r) + "\n")
    os.replace(path + ".tmp", path)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", required=True)
    ap.add_argument("--split", default="profile", choices=sorted(SPLIT_SEED))
    ap.add_argument("--budget", type=float, default=600.0, help="stop starting new cases after this many seconds")
    ap.add_argument("--only", default="", help="comma-separated geometries 'bq:bkv' to profile")
    ap.add_argument("--refeature", action="store_true",
                    help="only add the max_row_nnz statistic to the existing records in --out (no timing)")
    ap.add_argument("--add-plans", default="",
                    help="comma-separated catalog ids to time and merge into the records of --base")
    ap.add_argument("--base", default="", help="records of --split to extend (with --add-plans)")
    ap.add_argument("--finalize", action="store_true",
                    help="put the plans added to the records in --out on one clock factor per pass (no timing)")
    args = ap.parse_args()
    if args.finalize:
        finalize_added(args.out)
        return
    if args.refeature:
        refeature(args)
        return
    if args.add_plans:
        add_plans(args)
        return
    import torch
    import paper_2609_25869_amd as bsa

    done = set()
    if os.path.exists(args.out):
        for line in open(args.out):
            if line.strip():
                done.add(json.loads(line)["id"])
    cases = [c for c in corpus(args.split) if c["id"] not in done]
    if args.only:
        keep = {tuple(int(x) for x in s.split(":")) for s in args.only.split(",")}
        cases = [c for c in cases if tuple(c["geometry"]) in keep]
    log("%d cases to profile (%d already in %s)" % (len(cases), len(done), args.out))
    t0 = time.time()
    with open(args.out, "a") as f:
        for i, c in enumerate(cases):
            if time.time() - t0 > args.budget:
                log("budget reached after %d cases" % i)
                break
            tc = time.time()
            rec = profile_case(torch, bsa, c)
            f.write(json.dumps(rec) + "\n")
            f.flush()
            best = min(rec["latency_ms"].items(), key=lambda kv: kv[1])
            log("%s geom %s N %d bh %d %s %.2f: density %.4f best plan %s %.3f ms, %d invalid (%.1f s)" % (
                c["id"], c["geometry"], c["N"], c["bh"], c["family"], c["rho"],
                rec["features"]["nnz"] / rec["features"]["blocks"], best[0], best[1], len(rec["invalid"]),
                time.time() - tc))
            torch.cuda.empty_cache()
    log("done in %.1f s" % (time.time() - t0))


if __name__ == "__main__":
    main()
