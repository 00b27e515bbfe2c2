"""CPU oracle of the embedding-bag input stage of the CTR workload.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, links or runs
this module: only the test-suite and the smoke check do.  It shares no code
with the HIP library.

What it computes.  The paper trains its CTR model (Section 3.2) from an input
embedding x (Section 2.1) and does not describe the features behind it; the
benchmark workload's reading is the usual CTR input: the dense features
through log1p, then, for every sparse feature (table), the sum of the table
rows its bag of ids selects, all concatenated into one row:

    x[m] = [ log1p(dense[m]) | sum_{i in bag(0, m)} T_0[idx_i] | ... |
             sum_{i in bag(T-1, m)} T_{T-1}[idx_i] ]

Bag (t, m) is indices[offsets[t][m] : offsets[t][m+1]].  Arithmetic is
float64: the result is the exact sum up to float64 rounding, which any
summation order reaches within the error bound the tests use.
"""
from __future__ import annotations

import numpy as np


def embed_bags(dense, offsets, indices, tables):
    """x [M][n_dense + T*dim] in float64.

    dense:   [M][n_dense] raw dense features (log1p is applied here);
    offsets: [T][M+1] bag boundaries into ``indices``;
    indices: flat row ids;
    tables:  sequence of T arrays [rows][dim].
    """
    dense = np.asarray(dense, dtype=np.float64)
    offsets = np.asarray(offsets, dtype=np.int64)
    indices = np.asarray(indices, dtype=np.int64)
    M = offsets.shape[1] - 1
    T = offsets.shape[0]
    dim = np.asarray(tables[0]).shape[1]
    n_dense = dense.shape[1] if dense.size else 0
    x = np.zeros((M, n_dense + T * dim), dtype=np.float64)
    if n_dense:
        x[:, :n_dense] = np.log1p(dense)
    for t in range(T):
        tab = np.asarray(tables[t], dtype=np.float64)
        for m in range(M):
            ids = indices[offsets[t, m]:offsets[t, m + 1]]
            # the bag's rows, summed (a sum of a selection: a library matmul
            # of the bag's multiplicity vector with the table is the same)
            x[m, n_dense + t * dim: n_dense + (t + 1) * dim] = tab[ids].sum(axis=0)
    return x


def embed_bags_backward(offsets, indices, dx, n_dense, rows, dim):
    """Gradient of the tables given the gradient dx [M][>= n_dense + T*dim]
    at x, in float64:

        grad[t][r] = sum over the entries i of table t with indices[i] == r
                     of dx[bag(i)][n_dense + t*dim : n_dense + (t+1)*dim]

    where bag(i) is the bag (row of x) entry i belongs to.  The dense
    features take no table gradient.  Returns [T][rows][dim]."""
    offsets = np.asarray(offsets, dtype=np.int64)
    indices = np.asarray(indices, dtype=np.int64)
    dx = np.asarray(dx, dtype=np.float64)
    T, M = offsets.shape[0], offsets.shape[1] - 1
    g = np.zeros((T, rows, dim), dtype=np.float64)
    for t in range(T):
        for m in range(M):
            for i in range(offsets[t, m], offsets[t, m + 1]):
                g[t, indices[i]] += dx[m, n_dense + t * dim: n_dense + (t + 1) * dim]
    return g
