"""Seeded synthetic workloads for the detached-block training step.

This module only *draws* inputs: model descriptions, initial parameters,
batches and labels.  It holds none of the training step's arithmetic, so the
CPU oracle and the HIP path can both consume what it produces without sharing
any computation.

Workloads (the paper's models and data are not available; these stand in for
them with the shapes and value distributions of the paper's settings):

* ``tiny``      -- 2 detached blocks on a shared 16-wide input, fp32, M=64.
* ``ctr_mlp``   -- CTR-shaped input (13 log1p dense features + 26 sum-pooled
                   embedding bags of width 64 = 1677 features), 6 detached
                   dense subarchitectures 1677->512->256->128 each with a local
                   Linear(128->1) sigmoid-BCE head, bf16, M=4096.  Stands in
                   for the paper's CTR model with six detached dense
                   subarchitectures (Section 3.2).
* ``ctr_dcn``   -- the same input at M=16384, 6 blocks of 2 DCNv2 cross layers
                   followed by 1677->1024->1024->512, bf16.
* ``deep_chain``-- 12 blocks chained through the stop-gradient of Eq. (1),
                   each 256->256->256, bf16, M=1024.

Random draw order for one seed: parameters (block -> layer -> W, b -> head
w, head c), then embedding tables, then batches (x then labels per batch).

Model description (plain dict, consumed by both sides):

    {"name", "dtype": "f32"|"bf16", "batch", "in_dim",
     "blocks": [{"input": "x"|"prev", "layers": [(kind, in, out), ...],
                 "lam": float}, ...],
     "adam": {"lr", "beta1", "beta2", "eps"}}

with ``kind`` one of ``"linear_relu"`` and ``"cross"``.
"""
from __future__ import annotations

import copy

import numpy as np

ADAM_DEFAULT = {"lr": 1e-3, "beta1": 0.9, "beta2": 0.999, "eps": 1e-8}

# CTR input recipe (13 dense + 26 bags x 64 = 1677 features).
CTR_DENSE = 13
CTR_TABLES = 26
CTR_DIM = 64
CTR_ROWS = 100_000
CTR_BAG_MIN, CTR_BAG_MAX = 1, 20
CTR_ZIPF_S = 1.1
CTR_TABLE_STD = 0.01


def _mlp_block(widths, inp="x", lam=1.0):
    layers = [("linear_relu", widths[i], widths[i + 1]) for i in range(len(widths) - 1)]
    return {"input": inp, "layers": layers, "lam": float(lam)}


def config(name: str, **over) -> dict:
    """Return the model/workload description for a named workload.

    Keyword overrides replace top-level keys (``batch`` is the usual one), so
    tests can shrink a workload while keeping its structure.
    """
    if name == "tiny":
        cfg = {"name": name, "dtype": "f32", "batch": 64, "in_dim": 16,
               "blocks": [_mlp_block([16, 32, 32]) for _ in range(2)],
               "label_p": 0.5, "input_kind": "normal"}
    elif name == "tiny_chain":
        cfg = {"name": name, "dtype": "f32", "batch": 64, "in_dim": 16,
               "blocks": [_mlp_block([16, 32, 32]), _mlp_block([32, 32, 32], inp="prev")],
               "label_p": 0.5, "input_kind": "normal"}
    elif name == "ctr_mlp":
        cfg = {"name": name, "dtype": "bf16", "batch": 4096, "in_dim": 1677,
               "blocks": [_mlp_block([1677, 512, 256, 128]) for _ in range(6)],
               "label_p": 0.03, "input_kind": "ctr"}
    elif name == "ctr_dcn":
        blocks = []
        for _ in range(6):
            layers = [("cross", 1677, 1677), ("cross", 1677, 1677),
                      ("linear_relu", 1677, 1024), ("linear_relu", 1024, 1024),
                      ("linear_relu", 1024, 512)]
            blocks.append({"input": "x", "layers": layers, "lam": 1.0})
        cfg = {"name": name, "dtype": "bf16", "batch": 16384, "in_dim": 1677,
               "blocks": blocks, "label_p": 0.03, "input_kind": "ctr"}
    elif name == "deep_chain":
        blocks = [_mlp_block([256, 256, 256], inp="x" if b == 0 else "prev") for b in range(12)]
        cfg = {"name": name, "dtype": "bf16", "batch": 1024, "in_dim": 256,
               "blocks": blocks, "label_p": 0.03, "input_kind": "normal"}
    else:
        raise KeyError(f"unknown workload {name!r}")
    cfg["adam"] = dict(ADAM_DEFAULT)
    cfg["ctr_rows"] = CTR_ROWS
    for k, v in over.items():
        cfg[k] = v
    return cfg


def custom(dtype, batch, in_dim, blocks, label_p=0.5, input_kind="normal", adam=None, name="custom"):
    """Build a description from explicit blocks (used by tests for odd shapes)."""
    return {"name": name, "dtype": dtype, "batch": int(batch), "in_dim": int(in_dim),
            "blocks": copy.deepcopy(blocks), "label_p": float(label_p),
            "input_kind": input_kind, "adam": dict(adam or ADAM_DEFAULT), "ctr_rows": CTR_ROWS}


# ----------------------------------------------------------------------------
# bf16 value rounding for *inputs*: x and initial parameters are drawn in
# float64, then rounded once to bf16 (round-to-nearest-even) and handed to
# both sides as float32 arrays holding bf16-representable values.
# ----------------------------------------------------------------------------
def round_to_bf16_values(a: np.ndarray) -> np.ndarray:
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)).astype(np.uint32)
    return r.view(np.float32).reshape(f.shape)


def _as_input(cfg, a):
    a = np.asarray(a, dtype=np.float32)
    return round_to_bf16_values(a) if cfg["dtype"] == "bf16" else a


def make_params(cfg: dict, rng: np.random.Generator) -> list:
    """Initial parameters, ``nn.Linear`` default init: U(+-1/sqrt(fan_in)).

    Returns one dict per block: ``{"layers": [(W[out,in], b[out]), ...],
    "head": (w[last], c[1])}`` as float32 arrays.
    """
    out = []
    for blk in cfg["blocks"]:
        layers = []
        for (_kind, fin, fout) in blk["layers"]:
            bound = 1.0 / np.sqrt(fin)
            W = rng.uniform(-bound, bound, size=(fout, fin))
            b = rng.uniform(-bound, bound, size=(fout,))
            layers.append((_as_input(cfg, W), _as_input(cfg, b)))
        last = blk["layers"][-1][2]
        bound = 1.0 / np.sqrt(last)
        w = rng.uniform(-bound, bound, size=(last,))
        c = rng.uniform(-bound, bound, size=(1,))
        out.append({"layers": layers, "head": (_as_input(cfg, w), _as_input(cfg, c))})
    return out


def zero_state(params: list) -> list:
    """Adam moments, all zeros, same structure as ``params``."""
    return [{"layers": [(np.zeros_like(W), np.zeros_like(b)) for (W, b) in p["layers"]],
             "head": (np.zeros_like(p["head"][0]), np.zeros_like(p["head"][1]))} for p in params]


def _bounded_zipf_cdf(n: int, s: float) -> np.ndarray:
    ranks = np.arange(1, n + 1, dtype=np.float64)
    w = ranks ** (-s)
    cdf = np.cumsum(w)
    return cdf / cdf[-1]


class CtrTables:
    """Frozen embedding tables N(0, 0.01^2), one per sparse feature."""

    def __init__(self, rng: np.random.Generator, rows: int = CTR_ROWS):
        self.rows = rows
        self.tables = [rng.normal(0.0, CTR_TABLE_STD, size=(rows, CTR_DIM)).astype(np.float32)
                       for _ in range(CTR_TABLES)]
        self.cdf = _bounded_zipf_cdf(rows, CTR_ZIPF_S)


def make_ctr_raw(tables: CtrTables, M: int, rng: np.random.Generator) -> dict:
    """Raw CTR features of M rows: LogNormal(0,1) dense values and, per
    table, bags of 1..20 bounded-Zipf(1.1) row ids.  ``offsets[t][m]`` ..
    ``offsets[t][m+1]`` delimit bag (t, m) in the flat ``indices`` list."""
    dense = rng.lognormal(0.0, 1.0, size=(M, CTR_DENSE))
    offsets = np.zeros((CTR_TABLES, M + 1), dtype=np.int64)
    ids_all = []
    base = 0
    for t in range(CTR_TABLES):
        lens = rng.integers(CTR_BAG_MIN, CTR_BAG_MAX + 1, size=M)
        total = int(lens.sum())
        u = rng.random(total)
        ids = np.minimum(np.searchsorted(tables.cdf, u, side="left"), tables.rows - 1)
        offsets[t, 0] = base
        offsets[t, 1:] = base + np.cumsum(lens)
        ids_all.append(ids.astype(np.int32))
        base += total
    return {"dense": dense, "offsets": offsets, "indices": np.concatenate(ids_all)}


def make_ctr_x(tables: CtrTables, M: int, rng: np.random.Generator) -> np.ndarray:
    """CTR input rows: log1p(LogNormal(0,1)) dense features followed by 26
    sum-pooled bags of 1..20 bounded-Zipf(1.1) row ids each (bags summed in
    float32 in index order)."""
    raw = make_ctr_raw(tables, M, rng)
    x = np.empty((M, CTR_DENSE + CTR_TABLES * CTR_DIM), dtype=np.float32)
    x[:, :CTR_DENSE] = np.log1p(raw["dense"])
    for t in range(CTR_TABLES):
        o = raw["offsets"][t]
        ids = raw["indices"][o[0]:o[-1]]
        seg = np.repeat(np.arange(M), np.diff(o))
        pooled = np.zeros((M, CTR_DIM), dtype=np.float32)
        np.add.at(pooled, seg, tables.tables[t][ids])
        x[:, CTR_DENSE + t * CTR_DIM: CTR_DENSE + (t + 1) * CTR_DIM] = pooled
    return x


def make_batches(cfg: dict, rng: np.random.Generator, n_batches: int, tables: CtrTables | None = None):
    """``n_batches`` (x[M,in_dim] float32, y[M] float32 in {0,1}) pairs."""
    M, K = cfg["batch"], cfg["in_dim"]
    if cfg["input_kind"] == "ctr" and tables is None:
        tables = CtrTables(rng, rows=cfg.get("ctr_rows", CTR_ROWS))
    out = []
    for _ in range(n_batches):
        if cfg["input_kind"] == "ctr":
            x = make_ctr_x(tables, M, rng)
        else:
            x = rng.normal(0.0, 1.0, size=(M, K))
        y = (rng.random(M) < cfg["label_p"]).astype(np.float32)
        out.append((_as_input(cfg, x), y))
    return out


def make_workload(cfg: dict, seed: int = 0, n_batches: int = 1):
    """Parameters and batches for ``cfg`` from one seeded PCG64 stream."""
    rng = np.random.Generator(np.random.PCG64(seed))
    params = make_params(cfg, rng)
    tables = None
    if cfg["input_kind"] == "ctr":
        tables = CtrTables(rng, rows=cfg.get("ctr_rows", CTR_ROWS))
    batches = make_batches(cfg, rng, n_batches, tables)
    return params, batches


def param_count(cfg: dict) -> int:
    n = 0
    for blk in cfg["blocks"]:
        for (_k, fin, fout) in blk["layers"]:
            n += fout * fin + fout
        n += blk["layers"][-1][2] + 1
    return n


def gemm_flops_per_step(cfg: dict) -> int:
    """Algorithmic GEMM FLOPs of one step: forward, weight gradient and, for
    every layer but a block's first, input gradient (2*M*N*K each)."""
    M = cfg["batch"]
    f = 0
    for blk in cfg["blocks"]:
        for i, (_k, fin, fout) in enumerate(blk["layers"]):
            f += 2 * 2 * M * fin * fout
            if i > 0:
                f += 2 * M * fin * fout
    return f
