"""Helpers shared by the GPU tests: uploads, plans, and comparisons with the oracle."""
from __future__ import annotations

import sys
from typing import Dict, Optional, Tuple

import numpy as np

# tolerance on O against the fp64 oracle, absolute over the compared elements
# (unit-variance inputs; bf16 operands and P rounded to bf16)
MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev_bf16(bits: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def bf16_to_f64(t) -> np.ndarray:
    import torch
    return t.detach().float().cpu().numpy().astype(np.float64)


def mask_to_dev(mask):
    import torch
    return torch.from_numpy(np.ascontiguousarray(mask.data)).cuda()


def run_plan(bsa, mask, q, k, v, force_plan: int = -1, lse: bool = True, select_mode: int = 0,
             geometry_per_head: Optional[bool] = None, keep_row_order: bool = False):
    """Plan and run on device; returns (plan, O tensor, LSE tensor or None, device inputs).

    O and LSE start as NaN, so a row that no task writes cannot pass for a
    correct one left in reused memory by an earlier run."""
    import torch
    qd, kd, vd = to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v)
    od = torch.full_like(qd, float("nan"))
    B, Nq, H, d = q.shape
    lsed = torch.full((B, H, Nq), float("nan"), dtype=torch.float32, device="cuda") if lse else None
    md = mask_to_dev(mask)
    shapes = bsa.shapes_of(qd, kd, vd, od)
    per_head = (not mask.uniform_geometry) if geometry_per_head is None else geometry_per_head
    bq = list(mask.bq) if per_head else int(mask.bq[0])
    bkv = list(mask.bkv) if per_head else int(mask.bkv[0])
    p = bsa.plan(md, bq, bkv, shapes, head_offset=list(mask.head_offset), stride_b=mask.stride_b,
                 force_plan=force_plan, select_mode=select_mode, keep_row_order=keep_row_order)
    bsa.forward(p, qd, kd, vd, od, lsed)
    torch.cuda.synchronize()
    return p, od, lsed, (qd, kd, vd, md)


def compare(O_gpu: np.ndarray, O_ref: np.ndarray, what: str = "") -> Dict[str, float]:
    err = np.abs(O_gpu - O_ref)
    out = {"max_abs": float(err.max()) if err.size else 0.0, "mean_abs": float(err.mean()) if err.size else 0.0}
    assert np.all(np.isfinite(O_gpu)), "%s: non-finite output" % what
    assert out["max_abs"] <= MAX_ABS, "%s: max-abs %.3g > %.3g" % (what, out["max_abs"], MAX_ABS)
    assert out["mean_abs"] <= MEAN_ABS, "%s: mean-abs %.3g > %.3g" % (what, out["mean_abs"], MEAN_ABS)
    return out


def compare_lse(L_gpu: np.ndarray, L_ref: np.ndarray, what: str = "", tol: float = 2e-3):
    fin = np.isfinite(L_ref)
    assert np.array_equal(np.isfinite(L_gpu), fin), "%s: LSE finiteness differs" % what
    assert np.all(L_gpu[~fin] == -np.inf), "%s: empty rows must have LSE -inf" % what
    if fin.any():
        rel = np.abs(L_gpu[fin] - L_ref[fin]) / np.maximum(1.0, np.abs(L_ref[fin]))
        assert rel.max() <= tol, "%s: LSE error %.3g" % (what, rel.max())


def expected_dispatch(tasks: np.ndarray, tile_kv: np.ndarray, member: Optional[np.ndarray]) -> np.ndarray:
    """The dispatch order the planner documents, from exported plan metadata:
    row order, with every task moved up to the first task (in row order) of
    the same (batch, head) that has the same KV tile list and member bits."""
    first = {}
    rep = []
    for i, (bh, _pq, lo, hi, _s, _ns) in enumerate(np.asarray(tasks).tolist()):
        mem = tuple(member[lo:hi].tolist()) if member is not None and len(member) else ()
        rep.append(first.setdefault((bh, tuple(tile_kv[lo:hi].tolist()), mem), i))
    return np.array(sorted(range(len(rep)), key=lambda i: (rep[i], i)), dtype=np.int64)
