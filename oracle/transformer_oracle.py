"""CPU oracle of one ERASE training step of the small causal transformer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, links or runs
this module: only the test-suite, the smoke check and the CPU-baseline leg of
the benchmark do.  It shares no code with the HIP library.

What it computes.  Section 3.1 partitions NanoChat's attention stack into
detached subgraphs, each sending no gradient to the one before it (Eq. 1),
and trains each piece on its own objective (Section 2.1); the aggregate
objective is Eq. 2.  The workload reads this as: every layer is one detached
block with its own local next-token head, and the chain of blocks is

    a0_1 = E[tokens[:, :-1]]                 (block 1 owns the embedding E)
    a0_b = sg[z_{b-1}]                       (b > 1)
    n1 = rms(a0);   [q | k | v] = n1 Wqkv^T
    o  = per head h: softmax(q_h k_h^T / sqrt(dh) + causal mask) v_h
    a1 = a0 + o Wo^T
    n2 = rms(a1);   u = n2 W1^T;   z = a1 + gelu(u) W2^T
    loss_b = mean over the B*T positions of  -log softmax(rms(z) Wh_b^T)[next token]

with rms(x) = x / sqrt(mean(x^2) + eps) over the model width (no gain) and
gelu the tanh form.  The gradient of L = sum_b lam_b loss_b reaches block b's
parameters from loss_b alone; block 1 also sends it into the embedding rows
its tokens selected.  Adam (PyTorch semantics) then updates every parameter.

Readings where the paper is silent (it names NanoChat, not its layers):
no positional encoding; no biases; RMSNorm eps 1e-6 without a learnable gain;
the tanh form of GELU; attention scale 1/sqrt(dh); embedding ~ N(0, 1) and
every linear weight ~ U(+-1/sqrt(fan_in)); loss averaged over all B*T
positions; lam_b = 1.

Arithmetic is float64 unless ``dtype`` says otherwise.  ``emulate_bf16=True``
rounds to bf16 the tensors the GPU stores in bf16 (weight copies, block
activations, stored activation gradients, and the head's exponentials and
row-scaled input, which stand in for a stored logit gradient); it is a
diagnostic for tighter comparisons, not the reference.

Pins (tests/test_oracle_transformer.py): torch CPU autograd of the same
network with .detach() at every cut (and torch.nn.functional's
scaled_dot_product_attention, rms_norm, gelu and cross_entropy), central
finite differences, closed forms (zero head gives log V; one position
attends only to itself), causality and detachment invariants (exact
equality), and torch.optim.Adam.
"""
from __future__ import annotations

import numpy as np

from .erase_oracle import adam_update

__all__ = ["PARAM_ORDER", "rms_norm", "rms_norm_backward", "gelu_tanh", "gelu_tanh_grad",
           "causal_attention", "causal_attention_backward", "softmax_xent",
           "tf_block_forward", "tf_block_backward", "tf_step", "tf_forward_losses"]

# flat order of a block's parameters (block 1 starts with the embedding)
PARAM_ORDER = ("emb", "wqkv", "wo", "w1", "w2", "wh")
RMS_EPS = 1e-6
_GELU_C = np.sqrt(2.0 / np.pi)
_GELU_A = 0.044715


def _bf16(a: np.ndarray) -> np.ndarray:
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy().astype(a.dtype)


def _ident(a):
    return a


def rms_norm(x: np.ndarray, eps: float = RMS_EPS):
    """y = x * r with r = 1 / sqrt(mean(x^2) + eps) per row (last axis)."""
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * r, r


def rms_norm_backward(dy: np.ndarray, x: np.ndarray, r: np.ndarray) -> np.ndarray:
    """Gradient at x of y = x r(x): with y = x r and d the width,
    dx = r (dy - y * mean(dy * y)), since dr/dx_j = -r^3 x_j / d."""
    y = x * r
    return r * (dy - y * np.mean(dy * y, axis=-1, keepdims=True))


def gelu_tanh(u: np.ndarray) -> np.ndarray:
    """0.5 u (1 + tanh(c (u + a u^3))), c = sqrt(2/pi), a = 0.044715."""
    return 0.5 * u * (1.0 + np.tanh(_GELU_C * (u + _GELU_A * u ** 3)))


def gelu_tanh_grad(u: np.ndarray) -> np.ndarray:
    """d gelu / du = 0.5 (1 + t) + 0.5 u (1 - t^2) c (1 + 3 a u^2), t = tanh(c (u + a u^3))."""
    t = np.tanh(_GELU_C * (u + _GELU_A * u ** 3))
    return 0.5 * (1.0 + t) + 0.5 * u * (1.0 - t * t) * _GELU_C * (1.0 + 3.0 * _GELU_A * u * u)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray):
    """q, k, v [B, H, T, dh].  Position i attends to positions j <= i:
    P = softmax_j(q_i . k_j / sqrt(dh)) over j <= i, o_i = sum_j P_ij v_j.
    Returns o and P."""
    T, dh = q.shape[2], q.shape[3]
    s = np.matmul(q, np.swapaxes(k, -1, -2)) / np.sqrt(dh)
    future = np.triu(np.ones((T, T), dtype=bool), 1)
    s = np.where(future, -np.inf, s)
    s = s - np.max(s, axis=-1, keepdims=True)
    e = np.exp(s)
    p = e / np.sum(e, axis=-1, keepdims=True)
    return np.matmul(p, v), p


def causal_attention_backward(do: np.ndarray, q: np.ndarray, k: np.ndarray, v: np.ndarray, p: np.ndarray):
    """Gradients at q, k, v of o = P v with P = softmax(q k^T / sqrt(dh) + mask):
    dv = P^T do;  dP = do v^T;  dS = P * (dP - rowsum(dP * P));
    dq = dS k / sqrt(dh);  dk = dS^T q / sqrt(dh).  Masked entries have P = 0."""
    sc = 1.0 / np.sqrt(q.shape[-1])
    dv = np.matmul(np.swapaxes(p, -1, -2), do)
    dp = np.matmul(do, np.swapaxes(v, -1, -2))
    ds = p * (dp - np.sum(dp * p, axis=-1, keepdims=True))
    dq = np.matmul(ds, k) * sc
    dk = np.matmul(np.swapaxes(ds, -1, -2), q) * sc
    return dq, dk, dv


def softmax_xent(logits: np.ndarray, target: np.ndarray):
    """Per-row -log softmax(logits)[target] = lse(logits) - logits[target] and
    the gradient of the per-row loss, softmax(logits) - onehot(target)."""
    mx = np.max(logits, axis=-1, keepdims=True)
    e = np.exp(logits - mx)
    se = np.sum(e, axis=-1, keepdims=True)
    lse = (mx + np.log(se))[:, 0]
    rows = np.arange(logits.shape[0])
    loss = lse - logits[rows, target]
    g = e / se
    g[rows, target] -= 1.0
    return loss, g


def _heads(x, B, T, H):
    """[B*T, H*dh] -> [B, H, T, dh]"""
    return x.reshape(B, T, H, -1).transpose(0, 2, 1, 3)


def _unheads(x):
    """[B, H, T, dh] -> [B*T, H*dh]"""
    B, H, T, dh = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B * T, H * dh)


def tf_block_forward(cfg: dict, p: dict, a0: np.ndarray, emulate_bf16: bool = False) -> dict:
    """Forward of one block and its local head (loss not yet reduced).
    a0: [B*T, d] block input.  Returns the cache for ``tf_block_backward``."""
    rb = _bf16 if emulate_bf16 else _ident
    B, T, H = cfg["batch"], cfg["seq"], cfg["heads"]
    d = a0.shape[1]
    W = {k: rb(p[k]) for k in ("wqkv", "wo", "w1", "w2", "wh")}
    n1, r1 = rms_norm(a0)
    n1 = rb(n1)
    qkv = rb(n1 @ W["wqkv"].T)
    q, k, v = (_heads(qkv[:, i * d:(i + 1) * d], B, T, H) for i in range(3))
    o4, P = causal_attention(q, k, v)
    o = rb(_unheads(o4))
    a1 = rb(a0 + o @ W["wo"].T)
    n2, r2 = rms_norm(a1)
    n2 = rb(n2)
    uf = n2 @ W["w1"].T
    u = rb(uf)
    g = rb(gelu_tanh(uf))
    z = rb(a1 + g @ W["w2"].T)
    hn, r3 = rms_norm(z)
    hn = rb(hn)
    logits = hn @ W["wh"].T
    return {"a0": a0, "n1": n1, "r1": r1, "q": q, "k": k, "v": v, "P": P, "o": o, "a1": a1,
            "n2": n2, "r2": r2, "u": u, "g": g, "z": z, "hn": hn, "r3": r3, "logits": logits, "W": W}


def tf_block_backward(cfg: dict, c: dict, target: np.ndarray, lam: float, emulate_bf16: bool = False,
                      g_out: np.ndarray | None = None, need_input_grad: bool = False,
                      trace: dict | None = None):
    """Local loss and the gradient of lam * loss (+ <g_out, z> when the
    undetached baseline sends a gradient into z) at the block's weights, and
    at its input a0 when ``need_input_grad``.  Returns (loss, grads, g_a0).
    ``trace`` (a dict, optional) receives the activation gradients the step
    stores (dhn, dz, du, dn2, da1, do, dqkv, and dn1 when formed; the head's
    pexp and hns under emulation, the logit gradient dlog otherwise), for
    checks of where emulation rounds; nothing else changes."""
    rb = _bf16 if emulate_bf16 else _ident
    B, T = cfg["batch"], cfg["seq"]
    N = B * T
    W = c["W"]
    rows, dlog = softmax_xent(c["logits"], target)
    loss = float(np.mean(rows))
    head = {}
    if emulate_bf16:
        # The head as the GPU stores it in bf16: exponentials relative to the
        # target logit, e = exp(x - x_target), with row sums S; the target
        # entry replaced by e - S; the head input scaled per row by
        # s = lam / (N S).  Then lam (softmax - onehot) / N = s (e - S onehot),
        # so dWh = e^T (s hn) and dhn = s (e Wh), the row scale applied after
        # the stored product.
        x = c["logits"]
        idx = np.arange(N)
        e = rb(np.exp(x - x[idx, target][:, None]))
        S = e.sum(axis=1)
        e[idx, target] = rb(e[idx, target] - S)
        s = (lam / N) / S
        hns = rb(s[:, None] * c["hn"])
        gr = {"wh": e.T @ hns}
        dhn = rb(e @ W["wh"])
        dz = rms_norm_backward(s[:, None] * dhn, c["z"], c["r3"])
        head = {"pexp": e, "hns": hns}
    else:
        dlog = dlog * (lam / N)
        gr = {"wh": dlog.T @ c["hn"]}
        dhn = dlog @ W["wh"]
        dz = rms_norm_backward(dhn, c["z"], c["r3"])
        head = {"dlog": dlog}
    if g_out is not None:
        dz = dz + g_out
    dz = rb(dz)
    gr["w2"] = dz.T @ c["g"]
    du = rb((dz @ W["w2"]) * gelu_tanh_grad(c["u"]))
    gr["w1"] = du.T @ c["n2"]
    dn2 = rb(du @ W["w1"])
    da1 = rb(dz + rms_norm_backward(dn2, c["a1"], c["r2"]))
    gr["wo"] = da1.T @ c["o"]
    do = rb(da1 @ W["wo"])
    H = c["q"].shape[1]
    dq, dk, dv = causal_attention_backward(_heads(do, B, T, H), c["q"], c["k"], c["v"], c["P"])
    dqkv = rb(np.concatenate([_unheads(dq), _unheads(dk), _unheads(dv)], axis=1))
    gr["wqkv"] = dqkv.T @ c["n1"]
    g_a0 = None
    dn1 = None
    if need_input_grad:
        dn1 = rb(dqkv @ W["wqkv"])
        g_a0 = da1 + rms_norm_backward(dn1, c["a0"], c["r1"])
    if trace is not None:
        trace.update(head, dhn=dhn, dz=dz, du=du, dn2=dn2, da1=da1, do=do, dqkv=dqkv)
        if dn1 is not None:
            trace["dn1"] = dn1
    return loss, gr, g_a0


def _cast(p: dict, dtype) -> dict:
    return {k: np.asarray(a, dtype=dtype) for k, a in p.items()}


def _inputs(tokens):
    tokens = np.asarray(tokens)
    return tokens[:, :-1].reshape(-1), tokens[:, 1:].reshape(-1)


def _forward(cfg, params, tokens, emulate_bf16, dtype):
    rb = _bf16 if emulate_bf16 else _ident
    inp, tgt = _inputs(tokens)
    caches = []
    a0 = rb(np.asarray(params[0]["emb"], dtype=dtype))[inp]
    for b, p in enumerate(params):
        c = tf_block_forward(cfg, _cast(p, dtype), a0, emulate_bf16)
        caches.append(c)
        a0 = c["z"]
    return caches, inp, tgt


def tf_forward_losses(cfg: dict, params: list, tokens: np.ndarray, dtype=np.float64) -> list:
    """Unweighted local losses loss_b of every block."""
    caches, _, tgt = _forward(cfg, params, tokens, False, dtype)
    return [float(np.mean(softmax_xent(c["logits"], tgt)[0])) for c in caches]


def tf_step(cfg: dict, params: list, m: list, v: list, t: int, tokens: np.ndarray,
            emulate_bf16: bool = False, dtype=np.float64, detach: bool = True) -> dict:
    """One training step.  ``params``, ``m``, ``v``: one dict per block with the
    keys of PARAM_ORDER (``emb`` in block 1 only).  ``tokens`` [B, T+1]:
    positions [:, :-1] are the inputs, [:, 1:] the next-token targets.
    ``t`` is the step count before this step.  Returns losses, grads (of
    L = sum_b lam_b loss_b), the updated params / m / v and the step count.

    ``detach=False`` is the conventional baseline: the same forward and
    objective, with the gradient at every block's input sent back into the
    block before it (and from block 1 into the embedding as before)."""
    caches, inp, tgt = _forward(cfg, params, tokens, emulate_bf16, dtype)
    nb = len(params)
    lam = cfg.get("lam", 1.0)
    losses, grads = [None] * nb, [None] * nb
    g_next = None
    for b in range(nb - 1, -1, -1):
        need = b == 0 or not detach
        loss, gr, g_a0 = tf_block_backward(cfg, caches[b], tgt, lam, emulate_bf16,
                                           None if detach else g_next, need)
        if b == 0:
            # the embedding rows each input position selected, summed per row
            ge = np.zeros_like(np.asarray(params[0]["emb"], dtype=dtype))
            np.add.at(ge, inp, g_a0)
            gr = {"emb": ge, **gr}
        losses[b], grads[b] = loss, gr
        g_next = g_a0
    ad = cfg["adam"]
    t1 = t + 1
    new_p, new_m, new_v = [], [], []
    for b in range(nb):
        p, mb, vb = _cast(params[b], dtype), _cast(m[b], dtype), _cast(v[b], dtype)
        pp, mm, vv = {}, {}, {}
        for key in grads[b]:
            pp[key], mm[key], vv[key] = adam_update(p[key], mb[key], vb[key], grads[b][key], t1, **ad)
        new_p.append(pp)
        new_m.append(mm)
        new_v.append(vv)
    return {"losses": losses, "grads": grads, "params": new_p, "m": new_m, "v": new_v, "t": t1}
