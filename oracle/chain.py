"""Matrix-chain products and their reordering (DLVM §3.1.2).

TEST INFRASTRUCTURE ONLY (see ``oracle/ir.py``).

§3.1.2 lists matrix multiplication reordering among the domain-specific
optimisations: by associativity, a chain of products of matrices of different
shapes can be evaluated in the order that needs the fewest elementary
operations. For ``A_0 A_1 ... A_{n-1}`` with ``A_i`` of shape
``dims[i] x dims[i+1]``, a product of a ``p x q`` by a ``q x r`` matrix costs
``p q r`` multiply-adds.

* ``chain_product(mats)`` is the plain definition: the product taken left to
  right with the IR's ``dot``, in float64. Every order gives the same exact
  result; that is what reordering relies on.
* ``chain_order(dims)`` is the classic dynamic programme over sub-chains
  (the optimal-parenthesisation recurrence of textbook algorithms courses):
  ``cost[i][j] = min over i <= k < j of cost[i][k] + cost[k+1][j] +
  dims[i] dims[k+1] dims[j+1]``, ties resolved towards the smallest k. It
  returns the minimal cost and the split table ``split[i][j] = k``.
* ``chain_product_in_order(mats, split)`` evaluates the product in a given
  order (for checking that an order computes the same matrix).
"""
from __future__ import annotations

import numpy as np

from .bf16 import round_to_bf16
from .ir import Function, evaluate


def _storage(a, dtype: str) -> np.ndarray:
    a32 = np.asarray(a, dtype=np.float32)
    return round_to_bf16(a32) if dtype == "bf16" else a32.astype(np.float64)


def chain_product(mats, dtype: str = "f32") -> np.ndarray:
    """A_0 A_1 ... A_{n-1}, left to right, float64 (inputs stored as ``dtype``)."""
    args = [_storage(m, dtype) for m in mats]
    f = Function("chain")
    vals = [f.arg(a.shape, name=f"A{i}") for i, a in enumerate(args)]
    acc = vals[0]
    for v in vals[1:]:
        acc = f.dot(acc, v)
    f.ret(acc)
    return evaluate(f, args)[0]


def chain_order(dims):
    """(minimal multiply-add count, split table) for the chain with shapes
    dims[i] x dims[i+1]; split[i][j] is the k of the outermost product
    (A_i..A_k)(A_{k+1}..A_j), -1 where i >= j."""
    n = len(dims) - 1
    assert n >= 1 and all(int(d) >= 1 for d in dims)
    d = [int(v) for v in dims]
    cost = [[0] * n for _ in range(n)]
    split = [[-1] * n for _ in range(n)]
    for length in range(2, n + 1):            # sub-chains of increasing length
        for i in range(0, n - length + 1):
            j = i + length - 1
            best = None
            for k in range(i, j):
                c = cost[i][k] + cost[k + 1][j] + d[i] * d[k + 1] * d[j + 1]
                if best is None or c < best:
                    best, split[i][j] = c, k
            cost[i][j] = best
    return cost[0][n - 1], split


def chain_product_in_order(mats, split, dtype: str = "f32") -> np.ndarray:
    """The chain product evaluated as the split table says, float64."""
    args = [_storage(m, dtype) for m in mats]
    f = Function("chain_ordered")
    vals = [f.arg(a.shape, name=f"A{i}") for i, a in enumerate(args)]

    def build(i, j):
        if i == j:
            return vals[i]
        k = split[i][j]
        return f.dot(build(i, k), build(k + 1, j))

    f.ret(build(0, len(args) - 1))
    return evaluate(f, args)[0]


def parenthesisation(split, i: int = 0, j: int | None = None) -> str:
    """The order of a split table as text, e.g. ``((A0(A1A2))((A3A4)A5))``."""
    if j is None:
        j = len(split) - 1
    if i == j:
        return f"A{i}"
    k = split[i][j]
    return "(" + parenthesisation(split, i, k) + parenthesisation(split, k + 1, j) + ")"
