"""CPU oracle of one ERASE training step on a network of detached blocks.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, links or runs
this module: only the test-suite, the smoke check and the CPU-baseline leg of
the benchmark do.  It shares no code with the HIP library.

What it computes (paper, Section 2):

* Eq. (1): block b reads sg[z_{b-1}] (or the shared input x for independent
  subarchitectures), so no gradient crosses a block boundary.
* A local loss on the block's own (undetached) output updates that block's
  parameters alone; the aggregate objective of Eq. (2) is L = sum_b lam_b l_b,
  so grad_{theta_b} L = lam_b grad_{theta_b} l_b.
* ERASE changes *when* each block's backward runs, never *what* it computes
  (Sections 2.2 and 5: gradients inside a piece stay exact), so the oracle is
  the plain definition: forward every block with the current parameters,
  form each block's local gradient, then apply Adam per block.

Readings where the paper is silent (it never names the optimizer, the
precision, the loss of the CTR heads or the init): sigmoid binary
cross-entropy with logits averaged over the batch; ReLU after every linear
layer and none after a DCNv2 cross layer; Adam with PyTorch semantics (bias
correction, eps outside the square root, no weight decay) with gradients
overwritten every step; the next block reads z_b computed with the
pre-update parameters.

Arithmetic is float64 unless ``dtype`` says otherwise.  ``emulate_bf16=True``
additionally rounds to bf16 exactly the tensors the GPU stores in bf16 (the
GEMM copy of each weight matrix, layer outputs, and stored activation
gradients); it is a diagnostic for tighter comparisons, not the reference.

Pins (tests/test_oracle_*.py): central finite differences, torch CPU autograd
with .detach() at every cut, torch.optim.Adam, closed forms (zero head gives
log 2, cross with W=0,b=0 is the identity, Adam's first step), the
detachment invariants (exact equality), and lam-scaling.
"""
from __future__ import annotations

import numpy as np

__all__ = ["bce_with_logits", "sigmoid", "block_forward", "block_backward",
           "adam_update", "step", "forward_all"]


def _bf16(a: np.ndarray) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even) via torch's own cast."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy().astype(a.dtype)


def _ident(a):
    return a


def sigmoid(s: np.ndarray) -> np.ndarray:
    """Logistic function, evaluated without overflow for either sign."""
    out = np.empty_like(s)
    pos = s >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-s[pos]))
    e = np.exp(s[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def bce_with_logits(s: np.ndarray, y: np.ndarray) -> np.ndarray:
    """Per-sample binary cross-entropy of logit s against label y:
    -[y log sigma(s) + (1-y) log(1-sigma(s))] = max(s,0) - s*y + log(1+e^{-|s|})."""
    return np.maximum(s, 0) - s * y + np.log1p(np.exp(-np.abs(s)))


def block_forward(blk: dict, p: dict, a0: np.ndarray, emulate_bf16: bool = False) -> dict:
    """Forward of one detached block f_b(sg[z_{b-1}]; theta_b) and its head.

    Layer kinds:
      linear_relu:   a_l = max(a_{l-1} W_l^T + b_l, 0)
      cross (DCNv2): a_l = a_0 * (a_{l-1} W_l^T + b_l) + a_{l-1}
    Head: s = z w + c with z = a_L.
    Returns the cache needed by ``block_backward``.
    """
    rnd = _bf16 if emulate_bf16 else _ident
    acts = [a0]
    pre = []
    a = a0
    for (kind, _fin, _fout), (W, b) in zip(blk["layers"], p["layers"]):
        h = a @ rnd(W).T + b
        pre.append(h)
        if kind == "linear_relu":
            a = np.maximum(h, 0)
        elif kind == "cross":
            a = a0 * h + a
        else:
            raise ValueError(kind)
        a = rnd(a)
        acts.append(a)
    w, c = p["head"]
    s = acts[-1] @ w + c[0]
    return {"acts": acts, "pre": pre, "s": s}


def block_backward(blk: dict, p: dict, cache: dict, y: np.ndarray,
                   emulate_bf16: bool = False, g_out=None, want_input_grad: bool = False,
                   trace: dict | None = None):
    """Local loss and exact gradient of lam_b * l_b w.r.t. theta_b only.

    l_b = mean_i BCE(s_i, y_i).  With g_s = lam (sigma(s) - y) / M:
      dw = z^T g_s, dc = sum g_s, g = g_s w^T   (g is the gradient at z = a_L)
    then for l = L..1, with g the gradient at a_l:
      linear_relu: u = g * [a_l > 0]; dW_l = u^T a_{l-1}; db_l = sum_rows u;
                   gradient at a_{l-1} = u W_l             (only if l > 1)
      cross:       u = g * a_0;       dW_l = u^T a_{l-1}; db_l = sum_rows u;
                   gradient at a_{l-1} = u W_l + g         (only if l > 1)
    No gradient is formed for the block input a_0: it is detached (Eq. 1).
    Returns (loss, grads) with grads shaped like p.

    ``trace`` (a dict, optional) receives the activation gradients the step
    stores per layer -- "u" (the GEMM operand u above), "g" (a cross layer's
    gradient at its output) and "wcopy" (the weight matrix as the GEMMs
    read it) -- for checks of where emulation rounds; nothing else changes.

    For the undetached baseline (conventional backpropagation through the
    cuts, the comparison of Section 3): ``g_out`` is added to g at z (the
    gradient later blocks send back), and ``want_input_grad`` also forms the
    gradient at a_0, u W_1 (+ g for a first cross layer) plus g_l * h_l for
    every cross layer l (a_0 enters each cross layer as a factor).  Then the
    return value is (loss, grads, gradient at a_0).
    """
    rnd = _bf16 if emulate_bf16 else _ident
    acts, s = cache["acts"], cache["s"]
    M = s.shape[0]
    lam = blk["lam"]
    loss = np.mean(bce_with_logits(s, y))
    gs = lam * (sigmoid(s) - y) / M
    w, _c = p["head"]
    dw = acts[-1].T @ gs
    dc = np.array([gs.sum()], dtype=s.dtype)
    g = np.outer(gs, w)
    if g_out is not None:
        if emulate_bf16 and blk["layers"][-1][0] == "linear_relu":
            # the head's term is stored (bf16, under the last layer's ReLU
            # mask) before the gradient from the next block is added to it
            g = rnd(g * (acts[-1] > 0))
        g = g + g_out
    a0 = acts[0]
    kinds = [k for (k, _i, _o) in blk["layers"]]
    grads = [None] * len(kinds)
    g_in = np.zeros_like(a0) if want_input_grad else None
    for l in range(len(kinds), 0, -1):
        W, _b = p["layers"][l - 1]
        if kinds[l - 1] == "linear_relu":
            u = rnd(g * (acts[l] > 0))
        else:
            g = rnd(g)
            u = rnd(g * a0)
            if want_input_grad:
                g_in = g_in + g * cache["pre"][l - 1]
        if trace is not None:
            trace.setdefault("u", {})[l] = u
            trace.setdefault("wcopy", {})[l] = rnd(W)
            if kinds[l - 1] == "cross":
                trace.setdefault("g", {})[l] = g
        grads[l - 1] = (u.T @ acts[l - 1], u.sum(axis=0))
        if l > 1 or want_input_grad:
            g_below = u @ rnd(W)
            if kinds[l - 1] == "cross":
                g_below = g_below + g
            if l > 1:
                g = g_below
            else:
                g_in = g_in + g_below
    if want_input_grad:
        return loss, {"layers": grads, "head": (dw, dc)}, g_in
    return loss, {"layers": grads, "head": (dw, dc)}


def adam_update(theta, m, v, g, t, lr, beta1, beta2, eps):
    """One Adam step at step count t >= 1 (bias-corrected, eps outside sqrt):
    m <- b1 m + (1-b1) g ; v <- b2 v + (1-b2) g^2 ;
    theta <- theta - lr * (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps)."""
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** t)
    vhat = v / (1.0 - beta2 ** t)
    theta = theta - lr * mhat / (np.sqrt(vhat) + eps)
    return theta, m, v


def _cast(tree, dtype):
    return {"layers": [(np.asarray(W, dtype=dtype), np.asarray(b, dtype=dtype)) for (W, b) in tree["layers"]],
            "head": (np.asarray(tree["head"][0], dtype=dtype), np.asarray(tree["head"][1], dtype=dtype))}


def forward_all(cfg: dict, params: list, x: np.ndarray, emulate_bf16: bool = False,
                dtype=np.float64) -> list:
    """Forward caches of every block with the given parameters."""
    caches = []
    prev = None
    for blk, p in zip(cfg["blocks"], params):
        p = _cast(p, dtype)
        a0 = np.asarray(x, dtype=dtype) if blk["input"] == "x" else prev
        cache = block_forward(blk, p, a0, emulate_bf16)
        caches.append(cache)
        prev = cache["acts"][-1]  # sg[z_b]: a constant for the next block
    return caches


def step(cfg: dict, params: list, m: list, v: list, t: int, x: np.ndarray, y: np.ndarray,
         emulate_bf16: bool = False, dtype=np.float64, detach: bool = True) -> dict:
    """One training step of the detached network.

    ``params``, ``m``, ``v``: one dict per block ({"layers": [(W, b)...],
    "head": (w, c)}).  ``t`` is the step count before this step; the Adam
    update uses t+1.  Returns losses (unweighted l_b), grads (of
    L = sum lam_b l_b), and the updated params/m/v and step count.

    ``detach=False`` is the conventional (undetached) baseline: the same
    forward and objective, but the gradient of L flows back across every cut
    of a chain (a block reading the previous block's output sends the
    gradient at its input back to that block).  For blocks reading the
    shared input x nothing crosses a cut, so both give the same result.
    """
    y = np.asarray(y, dtype=dtype)
    caches = forward_all(cfg, params, x, emulate_bf16, dtype)
    ad = cfg["adam"]
    t1 = t + 1
    nb = len(cfg["blocks"])
    back = [None] * nb   # (loss, grads) per block
    g_next = [None] * nb  # gradient sent back to block b's output
    for b in range(nb - 1, -1, -1):
        blk = cfg["blocks"][b]
        p = _cast(params[b], dtype)
        send = (not detach) and blk["input"] == "prev" and b > 0
        if send:
            loss, gr, g_in = block_backward(blk, p, caches[b], y, emulate_bf16, g_next[b], True)
            g_next[b - 1] = g_in
        else:
            loss, gr = block_backward(blk, p, caches[b], y, emulate_bf16, g_next[b])
        back[b] = (loss, gr)
    losses, grads, new_p, new_m, new_v = [], [], [], [], []
    for blk, p, mb, vb, (loss, gr) in zip(cfg["blocks"], params, m, v, back):
        p, mb, vb = _cast(p, dtype), _cast(mb, dtype), _cast(vb, dtype)
        losses.append(float(loss))
        grads.append(gr)
        pl, ml, vl = [], [], []
        for (W, b), (mW, mbias), (vW, vbias), (gW, gb) in zip(p["layers"], mb["layers"], vb["layers"], gr["layers"]):
            W2, mW2, vW2 = adam_update(W, mW, vW, gW, t1, **ad)
            b2, mb2, vb2 = adam_update(b, mbias, vbias, gb, t1, **ad)
            pl.append((W2, b2)); ml.append((mW2, mb2)); vl.append((vW2, vb2))
        hp = [adam_update(p["head"][i], mb["head"][i], vb["head"][i], gr["head"][i], t1, **ad) for i in range(2)]
        new_p.append({"layers": pl, "head": (hp[0][0], hp[1][0])})
        new_m.append({"layers": ml, "head": (hp[0][1], hp[1][1])})
        new_v.append({"layers": vl, "head": (hp[0][2], hp[1][2])})
    return {"losses": losses, "grads": grads, "params": new_p, "m": new_m, "v": new_v, "t": t1}


def total_loss(cfg: dict, params: list, x: np.ndarray, y: np.ndarray, dtype=np.float64) -> float:
    """Aggregate objective of Eq. (2) with every block loss local: sum_b lam_b l_b."""
    caches = forward_all(cfg, params, x, False, dtype)
    yy = np.asarray(y, dtype=dtype)
    return float(sum(blk["lam"] * np.mean(bce_with_logits(c["s"], yy))
                     for blk, c in zip(cfg["blocks"], caches)))
