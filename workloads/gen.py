"""Seeded synthetic workloads for dynamic block-sparse attention.

Inputs follow the shapes of the paper's vDiT workloads (about 115K tokens for
a five-second 720p clip, Section 1; logical blocks of 16 to 128 tokens and
mean densities near 10%, Section 7.1 and Table 3).  The paper's real mask
corpus is not available, so these generators stand in for it:

* Q, K, V: i.i.d. N(0, 1) in float32 rounded to bfloat16, drawn per
  (batch, head) slice by a counter-based generator (``philox_normal.c``), in
  the layout [B, N, H, d] with d contiguous.
* Logical masks (one byte per logical block, nonzero = active):
  Bernoulli with forced diagonal, a spatiotemporal 3D window over
  token cubes, per-row top-k by mean-pooled q.k block scores, and a seeded
  mixture of the three.

Nothing here computes attention.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libwlgen.so")
_LIB = None
_LIB_LOCK = threading.Lock()

# RNG stream ids of one (config, batch, head) slice.
STREAM_Q, STREAM_K, STREAM_V, STREAM_MASK, STREAM_CHOICE = 0, 1, 2, 3, 4


def build_generator(force: bool = False) -> str:
    """Compile the counter-based normal generator with gcc (OpenMP)."""
    src = os.path.join(_HERE, "philox_normal.c")
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(src):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", src, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _lib():
    global _LIB
    with _LIB_LOCK:
        if _LIB is None:
            if not os.path.exists(_LIB_PATH):
                build_generator()
            lib = ctypes.CDLL(_LIB_PATH)
            lib.wl_fill_normal_bf16.restype = ctypes.c_int
            lib.wl_fill_normal_bf16.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                                ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint32]
            _LIB = lib
    return _LIB


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    t = u >> 16
    t &= 1
    t += u
    t += 0x7FFF
    t >>= 16
    return t.astype(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _key(cfg_id: int, stream: int, b: int, h: int) -> Tuple[int, int]:
    return ((cfg_id & 0xFFFF) << 16 | (stream & 0xFFFF), (b & 0xFFFF) << 16 | (h & 0xFFFF))


def qkv_slice(cfg_id: int, stream: int, b: int, h: int, n: int, d: int) -> np.ndarray:
    """The [n, d] bfloat16 slice of tensor `stream` (0=Q, 1=K, 2=V) at (b, h)."""
    out = np.empty((n, d), dtype=np.uint16)
    k0, k1 = _key(cfg_id, stream, b, h)
    rc = _lib().wl_fill_normal_bf16(out.ctypes.data, n, d, d, k0, k1)
    if rc != 0:
        raise ValueError("head_dim must be a multiple of 4")
    return out


def make_tensor(cfg_id: int, stream: int, B: int, n: int, H: int, d: int) -> np.ndarray:
    """A [B, n, H, d] bfloat16 tensor (as uint16 bits), each (b, h) slice seeded on its own."""
    out = np.empty((B, n, H, d), dtype=np.uint16)
    lib = _lib()
    for b in range(B):
        for h in range(H):
            k0, k1 = _key(cfg_id, stream, b, h)
            ptr = out.ctypes.data + ((b * n * H + h) * d) * 2
            rc = lib.wl_fill_normal_bf16(ptr, n, d, H * d, k0, k1)
            if rc != 0:
                raise ValueError("head_dim must be a multiple of 4")
    return out


@dataclass
class BlockMask:
    """A logical block mask with per-head geometry.

    ``data`` holds one byte per logical block (nonzero = active).  Head h of
    batch b is the row-major [nqb(h), nkb(h)] matrix that starts at
    ``b * stride_b + head_offset[h]``; ``stride_b == 0`` broadcasts over batch.
    """

    data: np.ndarray
    head_offset: np.ndarray
    stride_b: int
    bq: np.ndarray
    bkv: np.ndarray
    B: int
    H: int
    nq: int
    nkv: int

    def nqb(self, h: int) -> int:
        return -(-self.nq // int(self.bq[h]))

    def nkb(self, h: int) -> int:
        return -(-self.nkv // int(self.bkv[h]))

    def head(self, b: int, h: int) -> np.ndarray:
        start = b * self.stride_b + int(self.head_offset[h])
        n = self.nqb(h) * self.nkb(h)
        return self.data[start:start + n].reshape(self.nqb(h), self.nkb(h))

    @property
    def uniform_geometry(self) -> bool:
        return bool(np.all(self.bq == self.bq[0]) and np.all(self.bkv == self.bkv[0]))

    @staticmethod
    def from_heads(heads: Sequence[Sequence[np.ndarray]], bq: Sequence[int], bkv: Sequence[int],
                   nq: int, nkv: int) -> "BlockMask":
        """Pack masks given as heads[b][h] 2-D arrays (one per batch and head)."""
        B = len(heads)
        H = len(heads[0])
        sizes = [heads[0][h].size for h in range(H)]
        offs = np.zeros(H, dtype=np.int64)
        if H > 1:
            offs[1:] = np.cumsum(sizes)[:-1]
        per_b = int(sum(sizes))
        data = np.empty(B * per_b, dtype=np.uint8)
        for b in range(B):
            for h in range(H):
                m = np.asarray(heads[b][h])
                assert m.shape == (-(-nq // bq[h]), -(-nkv // bkv[h])), (m.shape, bq[h], bkv[h])
                data[b * per_b + offs[h]: b * per_b + offs[h] + m.size] = (m != 0).astype(np.uint8).ravel()
        return BlockMask(data=data, head_offset=offs, stride_b=per_b if B > 1 else per_b,
                         bq=np.asarray(bq, dtype=np.int32), bkv=np.asarray(bkv, dtype=np.int32),
                         B=B, H=H, nq=nq, nkv=nkv)


# ----------------------------------------------------------------------------
# Mask generators
# ----------------------------------------------------------------------------

def diagonal_blocks(nq: int, nkv: int, bq: int, bkv: int) -> np.ndarray:
    """Blocks whose token rectangle meets the token diagonal i == j."""
    nqb, nkb = -(-nq // bq), -(-nkv // bkv)
    out = np.zeros((nqb, nkb), dtype=bool)
    n = min(nq, nkv)
    for qb in range(nqb):
        lo, hi = qb * bq, min((qb + 1) * bq, n)
        if lo >= hi:
            continue
        out[qb, lo // bkv:(hi - 1) // bkv + 1] = True
    return out


def bernoulli_mask(rng: np.random.Generator, nqb: int, nkb: int, rho: float) -> np.ndarray:
    return rng.random((nqb, nkb)) < rho


def window_mask(grid: Tuple[int, int, int], half: Tuple[int, int, int]) -> np.ndarray:
    """Cube-grid window: block (q, k) active iff |dt|, |dh|, |dw| <= half-widths.

    Tokens are ordered cube by cube; cubes are numbered row-major over `grid`.
    """
    gt, gh, gw = grid
    t, hh, w = np.meshgrid(np.arange(gt), np.arange(gh), np.arange(gw), indexing="ij")
    t, hh, w = t.ravel(), hh.ravel(), w.ravel()
    return ((np.abs(t[:, None] - t[None, :]) <= half[0])
            & (np.abs(hh[:, None] - hh[None, :]) <= half[1])
            & (np.abs(w[:, None] - w[None, :]) <= half[2]))


def pooled_means(x_bits: np.ndarray, block: int) -> np.ndarray:
    """Mean of each `block`-token group of an [n, d] bfloat16 slice, in fp64."""
    x = f32_from_bf16_bits(x_bits).astype(np.float64)
    n, d = x.shape
    nb = -(-n // block)
    pad = nb * block - n
    if pad:
        x = np.concatenate([x, np.zeros((pad, d))])
    sums = x.reshape(nb, block, d).sum(axis=1)
    counts = np.full(nb, float(block))
    counts[-1] = n - (nb - 1) * block
    return sums / counts[:, None]


def topk_mask(q_bits: np.ndarray, k_bits: np.ndarray, bq: int, bkv: int, k: int) -> np.ndarray:
    """Per query-block row, the k KV blocks with the largest pooled q.k score.

    Ties keep the lower KV block (stable sort on the negated score).
    """
    pq = pooled_means(q_bits, bq)
    pk = pooled_means(k_bits, bkv)
    scores = pq @ pk.T
    order = np.argsort(-scores, axis=1, kind="stable")[:, :k]
    out = np.zeros(scores.shape, dtype=bool)
    np.put_along_axis(out, order, True, axis=1)
    return out


# ----------------------------------------------------------------------------
# Workload configurations
# ----------------------------------------------------------------------------

@dataclass
class WorkloadConfig:
    name: str
    cfg_id: int
    B: int
    H: int
    N: int
    geometry: List[Tuple[int, int]]  # per head (B_Q, B_KV)
    kind: str
    params: Dict = field(default_factory=dict)
    d: int = 128
    description: str = ""


# Window half-widths (in cubes) that realise each target density of the
# mixed-density sweep on the (8, 16, 16) grid of 64-token cubes.
MIXED_WINDOW_HALF = {0.02: (3, 1, 1), 0.05: (1, 3, 3), 0.10: (3, 3, 3), 0.25: (1, 9, 9), 0.50: (6, 7, 7)}
MIXED_DENSITIES = (0.02, 0.05, 0.10, 0.25, 0.50)

CONFIGS: Dict[str, WorkloadConfig] = {
    "c1_tiny": WorkloadConfig(
        "c1_tiny", 1, 1, 2, 2048, [(64, 64)] * 2, "bernoulli_diag", {"rho": 0.3},
        description="B1 H2 N2048, (64,64) blocks, Bernoulli(0.3) + diagonal"),
    "c2_window": WorkloadConfig(
        "c2_window", 2, 1, 24, 115200, [(128, 128)] * 24, "window",
        {"grid": (15, 6, 10), "half": (1, 3, 5)},
        description="B1 H24 N115200, (128,128) blocks over (2,8,8) token cubes, window half-widths (1,3,5): 12.74%"),
    "c2_window15": WorkloadConfig(
        "c2_window15", 2, 1, 24, 115200, [(128, 128)] * 24, "window",
        {"grid": (15, 6, 10), "half": (1, 5, 5)},
        description="B1 H24 N115200, (128,128) blocks, window half-widths (1,5,5): 15.29%"),
    "c3_topk": WorkloadConfig(
        "c3_topk", 3, 1, 24, 115200, [(64, 64)] * 24, "topk", {"frac": 0.12},
        description="B1 H24 N115200, (64,64) blocks, top 12% by pooled q.k + diagonal"),
    "c4_asym": WorkloadConfig(
        "c4_asym", 4, 1, 16, 65536, [(128, 32) if h % 2 == 0 else (32, 128) for h in range(16)],
        "bernoulli_diag", {"rho_range": (0.05, 0.5)},
        description="B1 H16 N65536, (128,32)/(32,128) alternating, Bernoulli(U[0.05,0.5]) + diagonal"),
    "c5_mixed": WorkloadConfig(
        "c5_mixed", 5, 2, 24, 131072, [(64, 64)] * 24, "mixture", {"grid": (8, 16, 16)},
        description="B2 H24 N131072, (64,64) blocks, window/top-k/uniform mixture over {2,5,10,25,50}%"),
}


def scaled_config(cfg: WorkloadConfig, N: int, H: Optional[int] = None, B: Optional[int] = None,
                  name: Optional[str] = None) -> WorkloadConfig:
    """The same generator recipe at a smaller size (for fast parity tests)."""
    H = cfg.H if H is None else H
    geom = [cfg.geometry[h % len(cfg.geometry)] for h in range(H)]
    return WorkloadConfig(name or "%s_n%d" % (cfg.name, N), cfg.cfg_id, cfg.B if B is None else B, H, N, geom,
                          cfg.kind, dict(cfg.params), cfg.d, cfg.description + " (scaled to N=%d)" % N)


def make_qkv(cfg: WorkloadConfig) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Q, K, V as [B, N, H, d] bfloat16 bit arrays."""
    return tuple(make_tensor(cfg.cfg_id, s, cfg.B, cfg.N, cfg.H, cfg.d) for s in (STREAM_Q, STREAM_K, STREAM_V))


def _head_mask(cfg: WorkloadConfig, b: int, h: int, q: Optional[np.ndarray], k: Optional[np.ndarray]) -> np.ndarray:
    bq, bkv = cfg.geometry[h]
    N = cfg.N
    nqb, nkb = -(-N // bq), -(-N // bkv)
    rng_mask = np.random.default_rng([cfg.cfg_id, STREAM_MASK, b, h])
    rng_choice = np.random.default_rng([cfg.cfg_id, STREAM_CHOICE, b, h])

    def qk_slices():
        qs = q[b, :, h, :] if q is not None else qkv_slice(cfg.cfg_id, STREAM_Q, b, h, N, cfg.d)
        ks = k[b, :, h, :] if k is not None else qkv_slice(cfg.cfg_id, STREAM_K, b, h, N, cfg.d)
        return np.ascontiguousarray(qs), np.ascontiguousarray(ks)

    if cfg.kind == "bernoulli_diag":
        if "rho_range" in cfg.params:
            lo, hi = cfg.params["rho_range"]
            rho = float(rng_choice.uniform(lo, hi))
        else:
            rho = cfg.params["rho"]
        m = bernoulli_mask(rng_mask, nqb, nkb, rho)
        return m | diagonal_blocks(N, N, bq, bkv)
    if cfg.kind == "window":
        grid, half = cfg.params["grid"], cfg.params["half"]
        m = window_mask(grid, half)
        if m.shape != (nqb, nkb):
            raise ValueError("cube grid %s does not match %d x %d blocks" % (grid, nqb, nkb))
        return m
    if cfg.kind == "topk":
        kk = int(np.floor(cfg.params["frac"] * nkb + 0.5))
        qs, ks = qk_slices()
        return topk_mask(qs, ks, bq, bkv, kk) | diagonal_blocks(N, N, bq, bkv)
    if cfg.kind == "mixture":
        u = float(rng_choice.random())
        rho = MIXED_DENSITIES[int(rng_choice.integers(len(MIXED_DENSITIES)))]
        if u < 0.4:
            grid = cfg.params["grid"]
            if grid[0] * grid[1] * grid[2] != nqb:
                # Smaller test sizes: fall back to a 1-D window of matching density.
                w = max(0, int(round(rho * nkb / 2)))
                idx = np.arange(nqb)
                return np.abs(idx[:, None] - idx[None, :]) <= w
            return window_mask(grid, MIXED_WINDOW_HALF[rho])
        if u < 0.8:
            kk = max(1, int(np.floor(rho * nkb + 0.5)))
            qs, ks = qk_slices()
            return topk_mask(qs, ks, bq, bkv, kk) | diagonal_blocks(N, N, bq, bkv)
        return bernoulli_mask(rng_mask, nqb, nkb, rho)
    raise ValueError("unknown mask kind %r" % cfg.kind)


def make_mask(cfg: WorkloadConfig, q: Optional[np.ndarray] = None, k: Optional[np.ndarray] = None) -> BlockMask:
    """The config's logical block mask (top-k kinds pool from Q/K, regenerated if not given)."""
    heads = [[_head_mask(cfg, b, h, q, k) for h in range(cfg.H)] for b in range(cfg.B)]
    return BlockMask.from_heads(heads, [g[0] for g in cfg.geometry], [g[1] for g in cfg.geometry], cfg.N, cfg.N)


def random_case(seed: int, B: int, H: int, nq: int, nkv: int, d: int,
                geometry: Sequence[Tuple[int, int]], density: float, diag: bool = False,
                empty_rows: int = 0) -> Tuple[np.ndarray, np.ndarray, np.ndarray, BlockMask]:
    """A small random case (Q, K, V bfloat16 bits and a Bernoulli block mask).

    `empty_rows` query-block rows of each head are cleared so that fully
    masked query rows appear.
    """
    rng = np.random.default_rng([seed, 7])
    q = bf16_bits_from_f32(rng.standard_normal((B, nq, H, d), dtype=np.float32))
    k = bf16_bits_from_f32(rng.standard_normal((B, nkv, H, d), dtype=np.float32))
    v = bf16_bits_from_f32(rng.standard_normal((B, nkv, H, d), dtype=np.float32))
    heads = []
    for b in range(B):
        row = []
        for h in range(H):
            bq, bkv = geometry[h]
            nqb, nkb = -(-nq // bq), -(-nkv // bkv)
            m = rng.random((nqb, nkb)) < density
            if diag:
                m |= diagonal_blocks(nq, nkv, bq, bkv)
            if empty_rows:
                rows = rng.choice(nqb, size=min(empty_rows, nqb), replace=False)
                m[rows, :] = False
            row.append(m)
        heads.append(row)
    mask = BlockMask.from_heads(heads, [g[0] for g in geometry], [g[1] for g in geometry], nq, nkv)
    return q, k, v, mask
