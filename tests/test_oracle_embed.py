"""Pins of the oracle's embedding-bag input stage against definitions that do
not use it: torch's embedding_bag (sum mode) and math.log1p as library
routines, a count-matrix product as a second construction, closed forms
(single id, empty bag, repeated id, linearity), permutation invariance, and
the input generator's own pooling."""
import math

import numpy as np
import torch

import oracle
from paper_2608_18469_amd import synth


def _raw(seed, M=23, T=4, rows=50, dim=8, n_dense=5, max_len=6, allow_empty=True):
    rng = np.random.Generator(np.random.PCG64(seed))
    tables = [rng.normal(0, 1, size=(rows, dim)) for _ in range(T)]
    dense = rng.lognormal(0, 1, size=(M, n_dense))
    offsets = np.zeros((T, M + 1), dtype=np.int64)
    ids, base = [], 0
    for t in range(T):
        lens = rng.integers(0 if allow_empty else 1, max_len + 1, size=M)
        offsets[t, 0] = base
        offsets[t, 1:] = base + np.cumsum(lens)
        ids.append(rng.integers(0, rows, size=int(lens.sum())))
        base += int(lens.sum())
    return dense, offsets, np.concatenate(ids), tables


def test_matches_torch_embedding_bag_and_log1p():
    dense, offsets, indices, tables = _raw(1)
    x = oracle.embed_bags(dense, offsets, indices, tables)
    n_dense, dim = dense.shape[1], tables[0].shape[1]
    for m in range(dense.shape[0]):
        for j in range(n_dense):
            # two libm implementations: equal to a few ulp
            assert abs(x[m, j] - math.log1p(dense[m, j])) <= 4e-16 * max(1.0, abs(x[m, j]))
    for t, tab in enumerate(tables):
        o = offsets[t]
        ref = torch.nn.functional.embedding_bag(torch.from_numpy(indices[o[0]:o[-1]]),
                                                torch.from_numpy(tab), torch.from_numpy(o[:-1] - o[0]),
                                                mode="sum").numpy()
        np.testing.assert_allclose(x[:, n_dense + t * dim: n_dense + (t + 1) * dim], ref, rtol=1e-13, atol=1e-13)


def test_equals_count_matrix_product():
    dense, offsets, indices, tables = _raw(2, rows=17)
    x = oracle.embed_bags(dense, offsets, indices, tables)
    M, n_dense, dim = dense.shape[0], dense.shape[1], tables[0].shape[1]
    for t, tab in enumerate(tables):
        C = np.zeros((M, tab.shape[0]))
        for m in range(M):
            for r in indices[offsets[t, m]:offsets[t, m + 1]]:
                C[m, r] += 1
        np.testing.assert_allclose(x[:, n_dense + t * dim: n_dense + (t + 1) * dim], C @ tab, rtol=1e-12, atol=1e-12)


def test_closed_forms():
    rng = np.random.Generator(np.random.PCG64(3))
    tab = rng.normal(0, 1, size=(9, 4))
    # bags: [5], [], [2, 2, 2], [7, 1]
    offsets = np.array([[0, 1, 1, 4, 6]])
    indices = np.array([5, 2, 2, 2, 7, 1])
    dense = np.zeros((4, 0))
    x = oracle.embed_bags(dense, offsets, indices, [tab])
    assert np.array_equal(x[0], tab[5])
    assert np.array_equal(x[1], np.zeros(4))
    np.testing.assert_allclose(x[2], 3 * tab[2], rtol=1e-15)
    np.testing.assert_allclose(x[3], tab[7] + tab[1], rtol=1e-15)
    # linear in the table
    x2 = oracle.embed_bags(dense, offsets, indices, [2.5 * tab - 1.0])
    cnt = np.array([1, 0, 3, 2])[:, None]
    np.testing.assert_allclose(x2, 2.5 * x - cnt, rtol=1e-13, atol=1e-13)


def test_permutation_within_bags():
    dense, offsets, indices, tables = _raw(4)
    x = oracle.embed_bags(dense, offsets, indices, tables)
    rng = np.random.Generator(np.random.PCG64(5))
    perm = indices.copy()
    for t in range(offsets.shape[0]):
        for m in range(offsets.shape[1] - 1):
            a, b = offsets[t, m], offsets[t, m + 1]
            perm[a:b] = rng.permutation(perm[a:b])
    np.testing.assert_allclose(oracle.embed_bags(dense, offsets, perm, tables), x, rtol=1e-13, atol=1e-13)


def test_generator_pooling_agrees():
    """The CTR input generator pools in float32; the float64 oracle on the
    same raw features agrees to float32 rounding."""
    rng = np.random.Generator(np.random.PCG64(6))
    tabs = synth.CtrTables(rng, rows=2000)
    state = rng.bit_generator.state
    raw = synth.make_ctr_raw(tabs, 40, rng)
    rng.bit_generator.state = state
    x32 = synth.make_ctr_x(tabs, 40, rng)
    x = oracle.embed_bags(raw["dense"], raw["offsets"], raw["indices"], tabs.tables)
    # 20 terms of |v| <~ 0.05 each: float32 rounding well under 1e-7 absolute
    np.testing.assert_allclose(x32, x, rtol=1e-6, atol=2e-8)


def test_backward_matches_torch_embedding_bag_autograd():
    dense, offsets, indices, tables = _raw(7, rows=30)
    M, n_dense, dim, T = dense.shape[0], dense.shape[1], tables[0].shape[1], len(tables)
    rng = np.random.Generator(np.random.PCG64(8))
    dx = rng.normal(size=(M, n_dense + T * dim + 3))
    g = oracle.embed_bags_backward(offsets, indices, dx, n_dense, 30, dim)
    for t, tab in enumerate(tables):
        w = torch.tensor(tab, dtype=torch.float64, requires_grad=True)
        o = offsets[t]
        out = torch.nn.functional.embedding_bag(torch.from_numpy(indices[o[0]:o[-1]]), w,
                                                torch.from_numpy(o[:-1] - o[0]), mode="sum")
        out.backward(torch.from_numpy(dx[:, n_dense + t * dim: n_dense + (t + 1) * dim]))
        np.testing.assert_allclose(g[t], w.grad.numpy(), rtol=1e-13, atol=1e-13)


def test_backward_is_the_adjoint_of_the_forward():
    """<embed_bags(tables), dx> over the pooled columns = <tables, backward(dx)>:
    the forward is linear in the tables."""
    dense, offsets, indices, tables = _raw(9, rows=21)
    M, n_dense, dim, T = dense.shape[0], dense.shape[1], tables[0].shape[1], len(tables)
    rng = np.random.Generator(np.random.PCG64(10))
    dx = rng.normal(size=(M, n_dense + T * dim))
    x = oracle.embed_bags(np.zeros_like(dense), offsets, indices, tables)
    lhs = float(np.sum(x[:, n_dense:] * dx[:, n_dense:]))
    g = oracle.embed_bags_backward(offsets, indices, dx, n_dense, 21, dim)
    rhs = float(sum(np.sum(g[t] * tables[t]) for t in range(T)))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))
    # rows no bag selects get zero
    used = {(t, int(r)) for t in range(T) for r in indices[offsets[t, 0]:offsets[t, -1]]}
    for t in range(T):
        for r in range(21):
            if (t, r) not in used:
                assert np.all(g[t, r] == 0.0)
