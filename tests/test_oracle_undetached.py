"""Pins of the oracle's undetached baseline (conventional backpropagation of
the aggregate objective of Eq. 2 through every cut of a chain, the comparison
point of the paper's Section 3) against mathematics that does not use the
oracle's own backward:

* torch CPU autograd of the same network with no .detach() anywhere;
* central finite differences of L = sum_b lam_b l_b (the total derivative,
  which is what the undetached gradient is);
* on shared-input topologies nothing crosses a cut, so detached and
  undetached steps agree exactly.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_18469_amd import synth

F64 = np.float64


def _chain_cfg():
    # a chain whose middle block starts with two cross layers, so the gradient
    # at a block input also collects the g * h terms of the cross layers
    blocks = [
        {"input": "x", "layers": [("linear_relu", 6, 5), ("linear_relu", 5, 4)], "lam": 1.0},
        {"input": "prev", "layers": [("cross", 4, 4), ("cross", 4, 4), ("linear_relu", 4, 6)], "lam": 0.6},
        {"input": "prev", "layers": [("linear_relu", 6, 5)], "lam": 1.4},
    ]
    return synth.custom("f32", batch=10, in_dim=6, blocks=blocks, label_p=0.4)


def _workload(cfg, seed):
    params, batches = synth.make_workload(cfg, seed, 1)
    x, y = batches[0]
    params = [{"layers": [(W.astype(F64).copy(), b.astype(F64).copy()) for (W, b) in p["layers"]],
               "head": (p["head"][0].astype(F64).copy(), p["head"][1].astype(F64).copy())} for p in params]
    return params, x.astype(F64), y.astype(F64)


def _leaves(tree):
    out = []
    for (W, b) in tree["layers"]:
        out += [W, b]
    return out + [tree["head"][0], tree["head"][1]]


def _zeros(params):
    return [{"layers": [(np.zeros_like(W), np.zeros_like(b)) for (W, b) in p["layers"]],
             "head": (np.zeros_like(p["head"][0]), np.zeros_like(p["head"][1]))} for p in params]


def _step(cfg, params, x, y, detach):
    return oracle.step(cfg, params, _zeros(params), _zeros(params), 0, x, y, detach=detach)


def _torch_undetached(cfg, params, x, y):
    """The same network in torch autograd, one backward of sum lam_b l_b, no cut."""
    tp = []
    for p in params:
        layers = [(torch.tensor(W, requires_grad=True), torch.tensor(b, requires_grad=True)) for (W, b) in p["layers"]]
        head = (torch.tensor(p["head"][0], requires_grad=True), torch.tensor(p["head"][1], requires_grad=True))
        tp.append((layers, head))
    xt, yt = torch.tensor(x), torch.tensor(y)
    total, prev = 0.0, None
    for blk, (layers, head) in zip(cfg["blocks"], tp):
        a0 = xt if blk["input"] == "x" else prev
        a = a0
        for (kind, _i, _o), (W, b) in zip(blk["layers"], layers):
            h = torch.nn.functional.linear(a, W, b)
            a = torch.relu(h) if kind == "linear_relu" else a0 * h + a
        s = a @ head[0] + head[1]
        total = total + blk["lam"] * torch.nn.functional.binary_cross_entropy_with_logits(s, yt)
        prev = a
    total.backward()
    return [{"layers": [(W.grad.numpy(), b.grad.numpy()) for (W, b) in layers],
             "head": (head[0].grad.numpy(), head[1].grad.numpy())} for layers, head in tp]


def test_undetached_chain_matches_torch_autograd_without_detach():
    cfg = _chain_cfg()
    params, x, y = _workload(cfg, 3)
    r = _step(cfg, params, x, y, detach=False)
    tg = _torch_undetached(cfg, params, x, y)
    for b in range(len(cfg["blocks"])):
        for G, T in zip(_leaves(r["grads"][b]), _leaves(tg[b])):
            np.testing.assert_allclose(np.asarray(G).reshape(-1), T.reshape(-1), rtol=1e-10, atol=1e-14)


def test_undetached_gradient_is_the_total_derivative():
    """Central differences of L with respect to every parameter of the first
    two blocks of the chain (whose gradients collect later blocks' losses)."""
    cfg = _chain_cfg()
    params, x, y = _workload(cfg, 5)
    g = _step(cfg, params, x, y, detach=False)["grads"]
    for b in (0, 1):
        for P, G in zip(_leaves(params[b]), _leaves(g[b])):
            flat, gflat = P.reshape(-1), np.asarray(G).reshape(-1)
            for i in range(flat.size):
                h = 1e-6 * max(1.0, abs(flat[i]))
                old = flat[i]
                flat[i] = old + h
                lp = oracle.total_loss(cfg, params, x, y)
                flat[i] = old - h
                lm = oracle.total_loss(cfg, params, x, y)
                flat[i] = old
                fd = (lp - lm) / (2 * h)
                assert abs(fd - gflat[i]) <= 1e-6 * max(1e-3, abs(fd)) + 1e-9, (b, i, fd, gflat[i])


def test_undetached_differs_from_detached_exactly_where_gradient_crosses_a_cut():
    cfg = _chain_cfg()
    params, x, y = _workload(cfg, 7)
    det = _step(cfg, params, x, y, detach=True)
    und = _step(cfg, params, x, y, detach=False)
    # the last block sends nothing further back: identical
    for G, H in zip(_leaves(det["grads"][2]), _leaves(und["grads"][2])):
        assert np.array_equal(G, H)
    # earlier blocks' body gradients change; their heads (local only) do not
    for b in (0, 1):
        assert max(float(np.abs(G - H).max()) for G, H in
                   zip(_leaves(det["grads"][b])[:-2], _leaves(und["grads"][b])[:-2])) > 1e-6
        for G, H in zip(_leaves(det["grads"][b])[-2:], _leaves(und["grads"][b])[-2:]):
            assert np.array_equal(G, H)
    assert det["losses"] == und["losses"]


@pytest.mark.parametrize("name", ["tiny", "ctr_mlp"])
def test_shared_input_topology_is_unchanged_by_detachment(name):
    cfg = synth.config(name, batch=32) if name == "ctr_mlp" else synth.config(name)
    if name == "ctr_mlp":
        cfg["blocks"] = cfg["blocks"][:2]
        cfg["ctr_rows"] = 1000
    params, x, y = _workload(cfg, 2)
    det = _step(cfg, params, x, y, detach=True)
    und = _step(cfg, params, x, y, detach=False)
    for a, b in zip(det["grads"], und["grads"]):
        for G, H in zip(_leaves(a), _leaves(b)):
            assert np.array_equal(G, H)
