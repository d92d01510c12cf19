"""The recurrent cell of DLVM §3.1.2, unrolled, in the oracle's IR.

TEST INFRASTRUCTURE ONLY (see ``oracle/ir.py``).

§3.1.2 gives the cell of a simple recurrent network,
``h_t = f(W x_{t-1} + U h_{t-1} + b)``: two matrix products and two
additions, which the linear-algebra fusion pass turns into one product. The
oracle writes the cell the unfused way, exactly as that formula reads, in the
row-major batch orientation used everywhere here (rows are batch entries,
``x_t`` is ``[B, Kx]``, ``W`` is ``[Kx, H]``, ``U`` is ``[H, H]``, ``b`` a row
broadcast over the batch):

    h_{t+1} = act(add(add(dot(x_t, W), dot(h_t, U)), b)),   t = 0 .. T-1

so the oracle never sees the concatenated operand the product uses.

* ``rnn(x_0, .., x_{T-1}, h0, W, U, b) -> (h_1, .., h_T)``.
* ``rnn_vjp``: the seedable gradient of all T outputs at once. With seeds
  ``s_t`` (the adjoints of ``h_{t+1}``) the vector-Jacobian product is the
  gradient of the scalar ``sum_t reduce_add(s_t * h_{t+1})`` in which the
  seeds are arguments that are not differentiated; ``ad.differentiate`` builds
  it (adjoint code generation, §3.1.3) with respect to W, U, b and, when
  asked, h0 and the x_t.

A bf16-storage network rounds its inputs and parameters to bf16 on the way in
and casts every stored hidden state to bf16 (Table 1's dataTypeCast), like
the dense networks of ``oracle/mlp.py``.
"""
from __future__ import annotations

from dataclasses import dataclass
from functools import lru_cache

import numpy as np

from .ad import differentiate
from .bf16 import round_to_bf16
from .ir import Function, evaluate
from .mlp import ACTS, _act


@dataclass(frozen=True)
class RnnSpec:
    """Static description of an unrolled recurrent cell."""

    steps: int
    in_width: int
    hidden: int
    act: str = "tanh"
    dtype: str = "f32"          # storage of x, h0, parameters and hidden states
    storage_casts: bool = True  # bf16: cast every stored hidden state to bf16

    def __post_init__(self):
        assert self.steps >= 1 and self.in_width >= 1 and self.hidden >= 1
        assert self.act in ACTS and self.dtype in ("f32", "bf16")


def _build(f: Function, spec: RnnSpec, batch: int):
    """Arguments and hidden states of the unrolled cell inside ``f``."""
    T, Kx, H = spec.steps, spec.in_width, spec.hidden
    xs = [f.arg((batch, Kx), name=f"x{t}") for t in range(T)]
    h0 = f.arg((batch, H), name="h0")
    W = f.arg((Kx, H), name="W")
    U = f.arg((H, H), name="U")
    b = f.arg((1, H), name="b")
    hs = []
    h = h0
    for t in range(T):
        z = f.add(f.add(f.dot(xs[t], W), f.dot(h, U)), b)
        h = _act(f, spec.act, z)
        if spec.dtype == "bf16" and spec.storage_casts:
            h = f.cast(h, "bf16")   # the hidden state is stored as bf16
        hs.append(h)
    return hs


@lru_cache(maxsize=32)
def build_rnn(spec: RnnSpec, batch: int) -> Function:
    """``rnn(x_0, .., x_{T-1}, h0, W, U, b) -> (h_1, .., h_T)``."""
    f = Function("rnn")
    f.ret(*_build(f, spec, batch))
    return f


@lru_cache(maxsize=32)
def build_rnn_vjp(spec: RnnSpec, batch: int, wrt_x: bool, wrt_h0: bool) -> Function:
    """Gradient of ``sum_t <s_t, h_{t+1}>`` wrt W, U, b [, h0] [, x_0 .. x_{T-1}]
    (arguments: the x_t, h0, W, U, b, then the seeds s_0 .. s_{T-1})."""
    T, H = spec.steps, spec.hidden
    f = Function("rnn_seeded")
    hs = _build(f, spec, batch)
    seeds = [f.arg((batch, H), name=f"s{t}") for t in range(T)]
    total = None
    for h, s in zip(hs, seeds):
        term = f.reduce("add", f.mul(s, h), None)
        total = term if total is None else f.add(total, term)
    f.ret(total)
    wrt = [T + 1, T + 2, T + 3]          # W, U, b
    if wrt_h0:
        wrt.append(T)
    if wrt_x:
        wrt += list(range(T))
    return differentiate(f, wrt=wrt, of=0)


def _storage(a, dtype: str) -> np.ndarray:
    a32 = np.asarray(a, dtype=np.float32)
    return round_to_bf16(a32) if dtype == "bf16" else a32.astype(np.float64)


def _args(spec: RnnSpec, xs, h0, W, U, b):
    xs = np.asarray(xs)
    assert xs.shape[0] == spec.steps
    args = [_storage(xs[t], spec.dtype) for t in range(spec.steps)]
    args += [_storage(h0, spec.dtype), _storage(W, spec.dtype), _storage(U, spec.dtype),
             _storage(np.reshape(b, (1, -1)), spec.dtype)]
    return args


def rnn_forward(spec: RnnSpec, xs, h0, W, U, b) -> np.ndarray:
    """All states [T + 1, B, H]: the stored h0, then h_1 .. h_T."""
    batch = np.shape(h0)[0]
    args = _args(spec, xs, h0, W, U, b)
    outs = evaluate(build_rnn(spec, batch), args)
    return np.stack([args[spec.steps]] + list(outs))


def rnn_vjp(spec: RnnSpec, xs, h0, W, U, b, dhs, wrt_x: bool = False, wrt_h0: bool = False):
    """(dW, dU, db, dxs or None, dh0 or None) for output adjoints dhs [T, B, H]
    (dhs[t] is the adjoint of h_{t+1})."""
    batch = np.shape(h0)[0]
    g = build_rnn_vjp(spec, batch, bool(wrt_x), bool(wrt_h0))
    seeds = [np.asarray(dhs[t], np.float64) for t in range(spec.steps)]
    res = evaluate(g, _args(spec, xs, h0, W, U, b) + seeds)
    dW, dU, db = res[0], res[1], res[2].reshape(-1)
    rest = list(res[3:])
    dh0 = rest.pop(0) if wrt_h0 else None
    dxs = np.stack(rest) if wrt_x else None
    return dW, dU, db, dxs, dh0
