"""Pins of the small-transformer oracle against definitions that do not use it:
torch CPU autograd of the same network (float64, .detach() at every cut),
torch.nn.functional's rms_norm / gelu / scaled_dot_product_attention /
cross_entropy as library routines, central finite differences, closed forms
(zero head gives log V; one position attends only to itself), exact
causality and detachment invariants, and torch.optim.Adam."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import transformer_oracle as to
from paper_2608_18469_amd import synth_tf


def _cfg(**over):
    base = dict(vocab=37, d=12, heads=3, layers=3, seq=7, batch=2)
    base.update(over)
    return synth_tf.tf_config("tf_tiny", **base)


def _work(cfg, seed=0):
    rng = np.random.Generator(np.random.PCG64(seed))
    params = synth_tf.make_params(cfg, rng, round_bf16=False)
    tokens = synth_tf.make_tokens(cfg, rng)[0]
    return params, tokens


def _torch_losses(cfg, params, tokens, detach=True):
    """The network written with torch.nn.functional, float64 autograd."""
    B, T, H, d = cfg["batch"], cfg["seq"], cfg["heads"], cfg["d"]
    P = [{k: torch.tensor(np.asarray(a, dtype=np.float64), requires_grad=True) for k, a in p.items()} for p in params]
    inp = torch.from_numpy(tokens[:, :-1].astype(np.int64))
    tgt = torch.from_numpy(tokens[:, 1:].astype(np.int64)).reshape(-1)
    x = F.embedding(inp, P[0]["emb"])  # [B, T, d]
    losses = []
    for b, p in enumerate(P):
        a0 = x.detach() if (detach and b > 0) else x
        n1 = F.rms_norm(a0, (d,), eps=to.RMS_EPS)
        q, k, v = (n1 @ p["wqkv"].T).split(d, dim=-1)
        sh = lambda t: t.reshape(B, T, H, d // H).transpose(1, 2)
        o = F.scaled_dot_product_attention(sh(q), sh(k), sh(v), is_causal=True)
        a1 = a0 + o.transpose(1, 2).reshape(B, T, d) @ p["wo"].T
        n2 = F.rms_norm(a1, (d,), eps=to.RMS_EPS)
        z = a1 + F.gelu(n2 @ p["w1"].T, approximate="tanh") @ p["w2"].T
        logits = F.rms_norm(z, (d,), eps=to.RMS_EPS) @ p["wh"].T
        losses.append(F.cross_entropy(logits.reshape(B * T, -1), tgt))
        x = z
    return P, losses


def _rel(a, b):
    a, b = np.asarray(a, dtype=np.float64), np.asarray(b, dtype=np.float64)
    n = np.linalg.norm(b)
    return np.linalg.norm(a - b) / n if n > 0 else np.linalg.norm(a - b)


def test_components_match_torch_functional():
    rng = np.random.Generator(np.random.PCG64(1))
    x = rng.normal(size=(5, 16)) * 3
    y, r = to.rms_norm(x)
    np.testing.assert_allclose(y, F.rms_norm(torch.from_numpy(x), (16,), eps=to.RMS_EPS).numpy(), rtol=1e-13)
    u = rng.normal(size=200) * 4
    np.testing.assert_allclose(to.gelu_tanh(u), F.gelu(torch.from_numpy(u), approximate="tanh").numpy(),
                               rtol=1e-13, atol=1e-15)
    ut = torch.from_numpy(u).requires_grad_(True)
    F.gelu(ut, approximate="tanh").sum().backward()
    np.testing.assert_allclose(to.gelu_tanh_grad(u), ut.grad.numpy(), rtol=1e-12, atol=1e-14)
    q, k, v = (rng.normal(size=(2, 3, 9, 4)) for _ in range(3))
    o, P = to.causal_attention(q, k, v)
    ref = F.scaled_dot_product_attention(*(torch.from_numpy(a) for a in (q, k, v)), is_causal=True).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-13)
    logits = rng.normal(size=(11, 29)) * 5
    tgt = rng.integers(0, 29, size=11)
    rows, g = to.softmax_xent(logits, tgt)
    lt = torch.from_numpy(logits).requires_grad_(True)
    ce = F.cross_entropy(lt, torch.from_numpy(tgt), reduction="none")
    np.testing.assert_allclose(rows, ce.detach().numpy(), rtol=1e-13)
    ce.sum().backward()
    np.testing.assert_allclose(g, lt.grad.numpy(), rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("detach", [True, False])
def test_losses_and_gradients_match_torch_autograd(detach):
    cfg = _cfg(lam=0.7)
    params, tokens = _work(cfg)
    m = synth_tf.zero_state(params)
    r = to.tf_step(cfg, params, m, m, 0, tokens, detach=detach)
    P, losses = _torch_losses(cfg, params, tokens, detach=detach)
    sum(cfg["lam"] * l for l in losses).backward()
    for b in range(cfg["layers"]):
        lb = losses[b].item()
        assert abs(r["losses"][b] - lb) <= 1e-13 * abs(lb)
        for k, t in P[b].items():
            assert _rel(r["grads"][b][k], t.grad.numpy()) < 1e-11, (b, k)


def test_detached_vs_undetached_differ_only_across_cuts():
    cfg = _cfg()
    params, tokens = _work(cfg, seed=3)
    m = synth_tf.zero_state(params)
    a = to.tf_step(cfg, params, m, m, 0, tokens, detach=True)
    b = to.tf_step(cfg, params, m, m, 0, tokens, detach=False)
    last = cfg["layers"] - 1
    for k in a["grads"][last]:   # nothing is sent into the last block
        assert np.array_equal(a["grads"][last][k], b["grads"][last][k])
    assert _rel(a["grads"][0]["wqkv"], b["grads"][0]["wqkv"]) > 1e-3   # the first block receives the rest


def test_central_differences():
    cfg = _cfg(vocab=11, d=6, heads=2, layers=2, seq=4, batch=2)
    params, tokens = _work(cfg, seed=5)
    m = synth_tf.zero_state(params)
    r = to.tf_step(cfg, params, m, m, 0, tokens)
    rng = np.random.Generator(np.random.PCG64(6))

    def total(ps):
        return to.tf_forward_losses(cfg, ps, tokens)

    for b in range(cfg["layers"]):
        for k in params[b]:
            for _ in range(3):
                idx = tuple(int(rng.integers(0, s)) for s in params[b][k].shape)
                if k == "emb" and idx[0] not in set(tokens[:, :-1].reshape(-1)):
                    assert r["grads"][b][k][idx] == 0.0
                    continue
                h = 1e-6 * max(1.0, abs(float(params[b][k][idx])))
                vals = []
                for sgn in (1, -1):
                    ps = [{kk: np.array(a, dtype=np.float64) for kk, a in p.items()} for p in params]
                    ps[b][k][idx] += sgn * h
                    vals.append(total(ps)[b])  # detached: only the block's own loss carries its gradient
                fd = (vals[0] - vals[1]) / (2 * h)
                g = r["grads"][b][k][idx]
                assert abs(fd - g) <= 1e-6 * max(1e-3, abs(g)), (b, k, idx, fd, g)


def test_zero_head_closed_form():
    cfg = _cfg()
    params, tokens = _work(cfg, seed=7)
    for p in params:
        p["wh"] = np.zeros_like(p["wh"])
    m = synth_tf.zero_state(params)
    r = to.tf_step(cfg, params, m, m, 0, tokens)
    V, N = cfg["vocab"], cfg["batch"] * cfg["seq"]
    for b in range(cfg["layers"]):
        assert abs(r["losses"][b] - math.log(V)) <= 1e-14 * math.log(V)
        # dlogits = (1/V - onehot)/N and the head input has unit RMS rows, so
        # every body gradient is zero (wh = 0 blocks the path) ...
        for k in ("wqkv", "wo", "w1", "w2"):
            assert np.all(r["grads"][b][k] == 0.0)
        # ... and grad wh = dlogits^T hn
        c = to._forward(cfg, params, tokens, False, np.float64)[0][b]
        tgt = tokens[:, 1:].reshape(-1)
        dl = np.full((N, V), 1.0 / V)
        dl[np.arange(N), tgt] -= 1.0
        np.testing.assert_allclose(r["grads"][b]["wh"], (dl / N).T @ c["hn"], rtol=1e-12, atol=1e-15)


def test_single_position_attends_to_itself():
    rng = np.random.Generator(np.random.PCG64(8))
    q, k, v = (rng.normal(size=(3, 2, 1, 5)) for _ in range(3))
    o, P = to.causal_attention(q, k, v)
    assert np.array_equal(P, np.ones_like(P))
    assert np.array_equal(o, v)


def test_attention_is_causal_exactly():
    rng = np.random.Generator(np.random.PCG64(9))
    q, k, v = (rng.normal(size=(2, 2, 10, 4)) for _ in range(3))
    o, _ = to.causal_attention(q, k, v)
    k2, v2 = k.copy(), v.copy()
    k2[:, :, 6:] += rng.normal(size=k2[:, :, 6:].shape)
    v2[:, :, 6:] += 5.0
    o2, _ = to.causal_attention(q, k2, v2)
    assert np.array_equal(o[:, :, :6], o2[:, :, :6])


def test_later_blocks_do_not_change_earlier_gradients():
    cfg = _cfg()
    params, tokens = _work(cfg, seed=10)
    m = synth_tf.zero_state(params)
    a = to.tf_step(cfg, params, m, m, 0, tokens)
    ps = [dict(p) for p in params]
    ps[2] = {k: x * 1.5 + 0.01 for k, x in ps[2].items()}
    b = to.tf_step(cfg, ps, m, m, 0, tokens)
    for blk in (0, 1):
        assert a["losses"][blk] == b["losses"][blk]
        for k in a["grads"][blk]:
            assert np.array_equal(a["grads"][blk][k], b["grads"][blk][k])


def test_embedding_gradient_rows():
    cfg = _cfg(vocab=50)
    params, tokens = _work(cfg, seed=11)
    m = synth_tf.zero_state(params)
    r = to.tf_step(cfg, params, m, m, 0, tokens)
    used = set(int(t) for t in tokens[:, :-1].reshape(-1))
    ge = r["grads"][0]["emb"]
    for row in range(cfg["vocab"]):
        if row not in used:
            assert np.all(ge[row] == 0.0)
    assert all(np.any(ge[row] != 0.0) for row in used)


def test_adam_matches_torch_optim():
    cfg = _cfg(layers=2)
    params, tokens = _work(cfg, seed=12)
    m = synth_tf.zero_state(params)
    r1 = to.tf_step(cfg, params, m, m, 0, tokens)
    r2 = to.tf_step(cfg, r1["params"], r1["m"], r1["v"], r1["t"], tokens)
    ad = cfg["adam"]
    for b in range(cfg["layers"]):
        for k in params[b]:
            t = torch.tensor(np.asarray(params[b][k], dtype=np.float64), requires_grad=True)
            opt = torch.optim.Adam([t], lr=ad["lr"], betas=(ad["beta1"], ad["beta2"]), eps=ad["eps"])
            for g in (r1["grads"][b][k], r2["grads"][b][k]):
                t.grad = torch.from_numpy(np.asarray(g, dtype=np.float64))
                opt.step()
            np.testing.assert_allclose(r2["params"][b][k], t.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_emulated_bf16_is_close():
    cfg = _cfg()
    params, tokens = _work(cfg, seed=13)
    m = synth_tf.zero_state(params)
    a = to.tf_step(cfg, params, m, m, 0, tokens)
    b = to.tf_step(cfg, params, m, m, 0, tokens, emulate_bf16=True)
    for blk in range(cfg["layers"]):
        assert abs(a["losses"][blk] - b["losses"][blk]) < 2e-2 * a["losses"][blk]
        for k in a["grads"][blk]:
            assert _rel(b["grads"][blk][k], a["grads"][blk][k]) < 0.1


def test_emulated_head_reproduces_the_logit_gradient():
    """The emulated head (exponentials relative to the target logit, the
    target entry minus the row sum, the row scale on the head input and after
    the input-gradient product) gives the head weight gradient and dz of the
    float64 logit gradient lam (softmax - onehot) / N up to bf16 rounding; a
    dropped one-hot entry or a wrong scale would be off by O(1)."""
    cfg = _cfg(vocab=96, d=32, heads=2, layers=1, seq=24, batch=3)
    params, tokens = _work(cfg, seed=5)
    inp, tgt = tokens[:, :-1].reshape(-1), tokens[:, 1:].reshape(-1)
    p = {k: np.asarray(a, np.float64) for k, a in params[0].items()}
    a0 = np.asarray(params[0]["emb"], np.float64)[inp]
    c = to.tf_block_forward(cfg, p, a0, False)
    out = {}
    for emulate in (False, True):
        tr = {}
        _loss, gr, _ga0 = to.tf_block_backward(cfg, c, tgt, 0.7, emulate, trace=tr)
        out[emulate] = (gr["wh"], tr["dz"])
    assert _rel(out[True][0], out[False][0]) < 1e-2
    assert _rel(out[True][1], out[False][1]) < 2e-2
    # the stored head tensors: the target entries are the only negatives
    tr = {}
    to.tf_block_backward(cfg, c, tgt, 0.7, True, trace=tr)
    neg = tr["pexp"] < 0
    assert np.array_equal(np.argwhere(neg)[:, 1], tgt) and neg.sum() == tgt.size


def _is_bf16(a):
    """Elementwise: a bf16 number (a float32 whose low 16 bits are zero)."""
    a = np.asarray(a, dtype=np.float64)
    f = a.astype(np.float32)
    return (f.astype(np.float64) == a) & ((f.view(np.uint32) & np.uint32(0xFFFF)) == 0)


def _share(arrays):
    a = np.concatenate([np.ravel(np.asarray(x, dtype=np.float64)) for x in arrays])
    a = a[a != 0]
    return float(np.mean(_is_bf16(a))) if a.size else 0.0


def test_bf16_emulation_rounds_exactly_the_stored_tensors():
    """emulate_bf16 rounds what the GPU stores in bf16 -- the weight copies,
    the block's activations (n1, q/k/v, o, a1, n2, u, g, z, hn), the head's
    exponentials and row-scaled input, and the stored activation gradients
    (dhn, dz, du, dn2, da1, do, dqkv, dn1) -- and leaves the fp32 ones alone:
    the RMSNorm statistics, the attention probabilities, the logits and the
    weight gradients.  Without emulation the stored tensors are not bf16
    (the check is not vacuous)."""
    cfg = _cfg(vocab=64, d=32, heads=2, layers=2, seq=16, batch=3)
    params, tokens = _work(cfg, seed=21)
    inp, tgt = tokens[:, :-1].reshape(-1), tokens[:, 1:].reshape(-1)
    acts = ("n1", "q", "k", "v", "o", "a1", "n2", "u", "g", "z", "hn")
    body = ("dhn", "dz", "du", "dn2", "da1", "do", "dqkv", "dn1")
    for emulate in (True, False):
        grads = (("pexp", "hns") if emulate else ("dlog",)) + body
        rb = to._bf16 if emulate else (lambda a: a)
        a0 = rb(np.asarray(params[0]["emb"], np.float64))[inp]
        c = to.tf_block_forward(cfg, {k: np.asarray(a, np.float64) for k, a in params[0].items()}, a0, emulate)
        tr = {}
        _loss, gr, _ga0 = to.tf_block_backward(cfg, c, tgt, 1.0, emulate, None, True, trace=tr)
        stored = [c[k] for k in acts] + [tr[k] for k in grads]
        if emulate:
            for k in acts:
                assert np.all(_is_bf16(c[k])), k
            for k in grads:
                assert np.all(_is_bf16(tr[k])), k
            for k, Wc in c["W"].items():
                assert np.all(_is_bf16(Wc)), k
        else:
            assert _share(stored) < 0.05
        assert _share([c["r1"], c["r2"], c["r3"], c["P"], c["logits"]] + list(gr.values())) < 0.05
