"""Seeded synthetic workloads for the detached small-transformer step.

Like ``synth``, this module only draws inputs (model description, initial
parameters, token batches) and holds none of the step's arithmetic, so the
CPU oracle and the HIP path can both consume what it produces.

Workloads (NanoChat, the paper's transformer of Section 3.1, is not
available; ``tf_c5`` has the shape of the small-transformer setting: vocabulary
32768, width 512, 8 heads of 64, 8 layers, sequences of 1024, batch 16,
token ids uniform over the vocabulary):

* ``tf_tiny``  -- vocabulary 64, width 64, 1 head, 2 layers, T=16, B=2.
* ``tf_small`` -- vocabulary 512, width 128, 2 heads, 2 layers, T=128, B=2.
* ``tf_c5``    -- the full shape above.

Description (plain dict):

    {"name", "vocab", "d", "heads", "layers", "seq", "batch", "lam",
     "adam": {"lr", "beta1", "beta2", "eps"}}

Parameters: one dict per block with ``wqkv`` [3d, d], ``wo`` [d, d],
``w1`` [4d, d], ``w2`` [d, 4d], ``wh`` [V, d], and ``emb`` [V, d] in block 1.
Random draw order for one seed: block 1's embedding, then per block wqkv,
wo, w1, w2, wh, then the token batches.  Every parameter is drawn in
float64 and rounded once to bf16 values (the workload is bf16), and the same
values go to both sides.
"""
from __future__ import annotations

import numpy as np

from .synth import ADAM_DEFAULT, round_to_bf16_values

PARAM_ORDER = ("emb", "wqkv", "wo", "w1", "w2", "wh")


def tf_config(name: str, **over) -> dict:
    shapes = {
        "tf_tiny": dict(vocab=64, d=64, heads=1, layers=2, seq=16, batch=2),
        "tf_small": dict(vocab=512, d=128, heads=2, layers=2, seq=128, batch=2),
        "tf_c5": dict(vocab=32768, d=512, heads=8, layers=8, seq=1024, batch=16),
    }
    if name not in shapes:
        raise KeyError(f"unknown transformer workload {name!r}")
    cfg = {"name": name, **shapes[name], "lam": 1.0, "adam": dict(ADAM_DEFAULT), "dtype": "bf16"}
    cfg.update(over)
    return cfg


def param_shapes(cfg: dict, block: int) -> list:
    """[(name, shape)] of one block in flat order."""
    V, d = cfg["vocab"], cfg["d"]
    out = [("emb", (V, d))] if block == 0 else []
    return out + [("wqkv", (3 * d, d)), ("wo", (d, d)), ("w1", (4 * d, d)), ("w2", (d, 4 * d)), ("wh", (V, d))]


def param_count(cfg: dict, block: int) -> int:
    return sum(int(np.prod(s)) for _, s in param_shapes(cfg, block))


def make_params(cfg: dict, rng: np.random.Generator, round_bf16: bool = True) -> list:
    """Embedding ~ N(0, 1) (``nn.Embedding``'s default), linear weights
    ~ U(+-1/sqrt(fan_in)) (``nn.Linear``'s default), no biases."""
    rnd = round_to_bf16_values if round_bf16 else (lambda a: np.asarray(a, dtype=np.float32))
    out = []
    for b in range(cfg["layers"]):
        p = {}
        for name, shape in param_shapes(cfg, b):
            if name == "emb":
                a = rng.normal(0.0, 1.0, size=shape)
            else:
                bound = 1.0 / np.sqrt(shape[1])
                a = rng.uniform(-bound, bound, size=shape)
            p[name] = rnd(a)
        out.append(p)
    return out


def zero_state(params: list) -> list:
    return [{k: np.zeros_like(a) for k, a in p.items()} for p in params]


def make_tokens(cfg: dict, rng: np.random.Generator, n_batches: int = 1) -> list:
    """Token batches [batch, seq + 1] int32, uniform over the vocabulary."""
    return [rng.integers(0, cfg["vocab"], size=(cfg["batch"], cfg["seq"] + 1)).astype(np.int32)
            for _ in range(n_batches)]


def make_workload(cfg: dict, seed: int = 0, n_batches: int = 1):
    rng = np.random.Generator(np.random.PCG64(seed))
    params = make_params(cfg, rng)
    return params, make_tokens(cfg, rng, n_batches)


def pack_block(cfg: dict, block: int, p: dict) -> np.ndarray:
    """Flat float32 vector of a block's parameters in the library's order."""
    return np.concatenate([np.asarray(p[n], dtype=np.float32).reshape(-1) for n, _ in param_shapes(cfg, block)])


def unpack_block(cfg: dict, block: int, flat: np.ndarray) -> dict:
    out, o = {}, 0
    for n, s in param_shapes(cfg, block):
        k = int(np.prod(s))
        out[n] = np.asarray(flat[o:o + k]).reshape(s)
        o += k
    return out


def flops_per_step(cfg: dict) -> dict:
    """Algorithmic FLOPs of one step (multiply-add = 2): the GEMMs of every
    block forward and backward and the attention products (causal: half of
    the T x T scores), with no input-gradient GEMM into a detached input."""
    V, d, L, T, B = cfg["vocab"], cfg["d"], cfg["layers"], cfg["seq"], cfg["batch"]
    N = B * T
    body = 2 * N * d * (3 * d + d + 4 * d + 4 * d)          # qkv, o, up, down
    head = 2 * N * d * V
    att_f = 2 * 2 * B * d * T * (T + 1) / 2                  # q k^T and p v over the causal triangle
    fwd = L * (body + head + att_f)
    # backward: weight gradients of every matrix, input gradients of every
    # matrix but qkv (except block 1), the head's input gradient, and the
    # attention backward (recompute of q k^T, then dv, dp, dq, dk)
    wgrad = L * (body + head)
    dgrad = L * (body - 2 * N * d * 3 * d + head) + 2 * N * d * 3 * d
    att_b = L * 2 * B * d * T * (T + 1) / 2 * 5
    return {"forward": fwd, "backward": wgrad + dgrad + att_b, "total": fwd + wgrad + dgrad + att_b}
