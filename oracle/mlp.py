"""The hot-path functions written in the oracle's IR, and their gradients.

TEST INFRASTRUCTURE ONLY (see ``oracle/ir.py``).

Each front-end builder writes one straight-line IR function out of the
primitives of Table 1, the way a DSL lowering would (§3.4 lowering phase),
and ``ad.differentiate`` turns a gradient declaration for it into a gradient
function (§3.1.3). Everything is evaluated in float64.

Functions written here:

* ``mlp_loss(x, W1, b1, ..., WL, bL, y) -> (loss, logits)``: dense layers
  ``H_l = act_l(H_{l-1} . W_l + b_l)`` (Fig. 3 orientation: ``x`` is
  ``[batch, in]``, ``W`` is ``[in, out]``, the bias is a row broadcast over the
  batch), the last layer without activation, then softmax cross-entropy with
  natural log, averaged over the batch. Softmax is composed from primitives
  (§3.1.1): the row maximum is subtracted, then exp, reduce-add, log; the label
  column is picked with a one-hot mask built by an integer compare of the label
  against ``iota`` and a select.
* ``chain_loss(x, W, b) -> (loss, e)``: one dense layer without bias, then the
  eight-operator element-wise chain ``add bias, tanh, x0.5, +1, sigmoid,
  x x_skip, square, mean`` with ``x_skip = x``.
* ``mlp(x, W1, b1, ..., WL, bL) -> logits``: the same layers without the loss;
  ``mlp_vjp`` evaluates its seedable gradient declaration (the adjoint of the
  logits given as the seed, Fig. 3).
* ``softmax_xent(z, y)`` and ``chain8(z, b, x_skip)`` are the same losses on a
  given pre-activation tensor, for testing the loss kernels on their own.

Activations are composites: sigmoid = 1 / (1 + exp(-v)); relu =
select(v > 0, v, 0); tanh is a primitive.

A bf16-storage network stores its inputs, parameters and hidden activations
in bf16: x and the parameters are rounded on the way in, and each hidden
activation goes through a dataTypeCast to bf16 (Table 1) before the next layer
reads it. The logits stay float32 (their rounding to float32 is not modelled).
``MlpSpec(storage_casts=False)`` gives the same network without the
activation casts, i.e. the exact function of the rounded inputs.

Order sensitivity. With storage casts the network is a discontinuous function
of its pre-activations: a change far below float32 resolution can move a value
across a bf16 rounding boundary, the resulting one-ulp change grows through
later layers and can flip ReLU masks of pre-activations near zero, and a
flipped mask switches a whole gradient path on or off. The gradient of a deep
bf16 ReLU network is therefore only defined up to the accumulation order of
its dot products. ``MlpSpec(accumulate="f32")`` evaluates the same network with
float32 accumulation in the forward dots (what a bf16-storage, float32-
accumulate evaluator does); the distance between the two oracle evaluations
measures that intrinsic ambiguity.
"""
from __future__ import annotations

from dataclasses import dataclass
from functools import lru_cache

import numpy as np

from .ad import differentiate, simplify_algebra
from .bf16 import round_to_bf16
from .ir import I64, Function, evaluate

ACTS = ("none", "sigmoid", "tanh", "relu")
LOSSES = ("softmax_ce", "chain8")


@dataclass(frozen=True)
class MlpSpec:
    """Static description of a network (widths, activations, loss, storage type)."""

    widths: tuple
    acts: tuple          # one per layer; names from ACTS
    loss: str = "softmax_ce"
    dtype: str = "f32"   # storage type of x, params and hidden activations: "f32" or "bf16"
    storage_casts: bool = True  # bf16: cast every stored hidden activation to bf16
    accumulate: str = "f64"     # forward dots: "f64", or "f32" to measure order sensitivity

    @property
    def n_layers(self) -> int:
        return len(self.widths) - 1

    def __post_init__(self):
        assert len(self.acts) == self.n_layers
        assert all(a in ACTS for a in self.acts)
        assert self.loss in LOSSES and self.dtype in ("f32", "bf16")
        if self.loss == "softmax_ce":
            assert self.acts[-1] == "none", "the output layer has no activation"
        else:
            assert self.n_layers == 1 and self.acts[0] == "none"
            assert self.widths[0] == self.widths[1], "x_skip = x needs in == out"


def _act(f: Function, name: str, v: int) -> int:
    if name == "none":
        return v
    if name == "sigmoid":
        return f.sigmoid(v)
    if name == "tanh":
        return f.tanh(v)
    if name == "relu":
        return f.relu(v)
    raise ValueError(name)


def _softmax_xent_ir(f: Function, z: int, y: int, batch: int, classes: int) -> int:
    """Mean softmax cross-entropy of logits ``z`` [B, C] against labels ``y`` [B, 1]."""
    m = f.reduce("max", z, 1)                       # row maximum (the shift)
    e = f.exp(f.sub(z, m))
    s = f.reduce("add", e, 1)
    lse = f.add(m, f.log(s))                        # log-sum-exp per row
    onehot = f.select(f.compare("eq", y, f.iota(classes)), f.const(1.0), f.const(0.0))
    zy = f.reduce("add", f.mul(z, onehot), 1)       # logit of the label
    per_row = f.sub(lse, zy)
    return f.mul(f.reduce("add", per_row, None), f.const(1.0 / batch))


def _chain_ir(f: Function, z: int, b: int, xs: int, rows: int, cols: int):
    """The eight-operator chain on pre-activation ``z``: returns (loss, e)."""
    zb = f.add(z, b)                                # add bias
    a = f.tanh(zb)                                  # tanh
    c = f.mul(a, f.const(0.5))                      # x 0.5
    d = f.add(c, f.const(1.0))                      # + 1
    s = f.sigmoid(d)                                # sigmoid
    e = f.mul(s, xs)                                # x x_skip
    sq = f.power(e, 2.0)                            # square
    loss = f.mul(f.reduce("add", sq, None), f.const(1.0 / (rows * cols)))  # mean
    return loss, e


@lru_cache(maxsize=64)
def build_mlp_loss(spec: MlpSpec, batch: int) -> Function:
    """``mlp_loss`` (CE) or ``chain_loss`` (chain8) for a fixed batch size."""
    f = Function("mlp_loss" if spec.loss == "softmax_ce" else "chain_loss")
    x = f.arg((batch, spec.widths[0]), name="x")
    ws = []
    for l in range(spec.n_layers):
        W = f.arg((spec.widths[l], spec.widths[l + 1]), name=f"W{l + 1}")
        b = f.arg((1, spec.widths[l + 1]), name=f"b{l + 1}")
        ws.append((W, b))
    if spec.loss == "softmax_ce":
        y = f.arg((batch, 1), I64, name="y")
        h = x
        for l, ((W, b), act) in enumerate(zip(ws, spec.acts)):
            h = _act(f, act, f.add(f.dot(h, W, spec.accumulate), b))
            if spec.dtype == "bf16" and spec.storage_casts and l < spec.n_layers - 1:
                h = f.cast(h, "bf16")   # the hidden activation is stored as bf16
        loss = _softmax_xent_ir(f, h, y, batch, spec.widths[-1])
        f.ret(loss, h)
    else:
        (W, b), = ws
        z = f.dot(x, W)
        loss, e = _chain_ir(f, z, b, x, batch, spec.widths[1])
        f.ret(loss, e)
    return f


@lru_cache(maxsize=64)
def build_mlp_gradient(spec: MlpSpec, batch: int, wrt_x: bool) -> Function:
    """Gradient declaration ``[gradient @mlp_loss wrt params (, x) keeping 0]``."""
    f = build_mlp_loss(spec, batch)
    n_params = 2 * spec.n_layers
    wrt = list(range(1, 1 + n_params))
    if wrt_x:
        wrt = [0] + wrt
    return differentiate(f, wrt=wrt, keeping=(0,), of=0)


@lru_cache(maxsize=64)
def build_mlp_logits(spec: MlpSpec, batch: int) -> Function:
    """``mlp(x, W1, b1, ..., WL, bL) -> logits``: the dense layers of ``mlp_loss``
    without the loss (softmax cross-entropy networks only)."""
    assert spec.loss == "softmax_ce"
    f = Function("mlp")
    x = f.arg((batch, spec.widths[0]), name="x")
    h = x
    for l, act in enumerate(spec.acts):
        W = f.arg((spec.widths[l], spec.widths[l + 1]), name=f"W{l + 1}")
        b = f.arg((1, spec.widths[l + 1]), name=f"b{l + 1}")
        h = _act(f, act, f.add(f.dot(h, W, spec.accumulate), b))
        if spec.dtype == "bf16" and spec.storage_casts and l < spec.n_layers - 1:
            h = f.cast(h, "bf16")
    f.ret(h)
    return f


@lru_cache(maxsize=64)
def build_mlp_vjp(spec: MlpSpec, batch: int, wrt_x: bool) -> Function:
    """Gradient declaration ``[gradient @mlp wrt params (, x) seedable]`` (Fig. 3's
    seedable form): the seed, the adjoint of the logits, is the last argument."""
    f = build_mlp_logits(spec, batch)
    wrt = list(range(1, 1 + 2 * spec.n_layers))
    if wrt_x:
        wrt = [0] + wrt
    return differentiate(f, wrt=wrt, seedable=True, of=0)


def _storage(a, dtype: str) -> np.ndarray:
    """Values as the GPU stores them: float32, or float32 rounded to bf16."""
    a32 = np.asarray(a, dtype=np.float32)
    if dtype == "bf16":
        return round_to_bf16(a32)
    return a32.astype(np.float64)


def _args(spec: MlpSpec, x, params, y=None):
    assert len(params) == spec.n_layers
    args = [_storage(x, spec.dtype)]
    for W, b in params:
        args.append(_storage(W, spec.dtype))
        args.append(_storage(np.reshape(b, (1, -1)), spec.dtype))
    if spec.loss == "softmax_ce" and y is not None:
        y = np.asarray(y, dtype=np.int64).reshape(-1, 1)
        C = spec.widths[-1]
        assert y.min() >= 0 and y.max() < C, "labels must lie in [0, C)"
        args.append(y)
    return args


def mlp_forward(spec: MlpSpec, x, params, y=None):
    """Evaluate ``mlp_loss``; return (loss, out) with out = logits (CE) or e (chain8).

    For the CE loss ``y`` may be omitted; then only the logits are meaningful
    (labels of zero are used to fill the signature).
    """
    batch = np.shape(x)[0]
    if spec.loss == "softmax_ce" and y is None:
        y = np.zeros(batch, dtype=np.int64)
    f = build_mlp_loss(spec, batch)
    loss, out = evaluate(f, _args(spec, x, params, y))
    return float(loss), out


def mlp_vjp(spec: MlpSpec, x, params, seed, wrt_x: bool = False):
    """Evaluate the seedable gradient of the logits: ([(dW, db)...], dx or None)
    for the given adjoint ``seed`` [batch, classes] of the logits."""
    batch = np.shape(x)[0]
    g = build_mlp_vjp(spec, batch, bool(wrt_x))
    args = _args(spec, x, params)
    res = evaluate(g, args + [np.asarray(seed, np.float64)])
    dx = None
    if wrt_x:
        dx, res = res[0], res[1:]
    grads = [(res[2 * l], res[2 * l + 1].reshape(-1)) for l in range(spec.n_layers)]
    return grads, dx


def mlp_gradient(spec: MlpSpec, x, params, y=None, wrt_x: bool = False):
    """Evaluate the gradient function; return (loss, [(dW, db)...], dx or None)."""
    batch = np.shape(x)[0]
    g = build_mlp_gradient(spec, batch, bool(wrt_x))
    res = evaluate(g, _args(spec, x, params, y))
    dx = None
    if wrt_x:
        dx, res = res[0], res[1:]
    grads = [(res[2 * l], res[2 * l + 1].reshape(-1)) for l in range(spec.n_layers)]
    loss = float(res[-1])
    return loss, grads, dx


@lru_cache(maxsize=16)
def _xent_grad_fn(batch: int, classes: int) -> Function:
    f = Function("softmax_xent")
    z = f.arg((batch, classes), name="z")
    y = f.arg((batch, 1), I64, name="y")
    f.ret(_softmax_xent_ir(f, z, y, batch, classes))
    return differentiate(f, wrt=[0], keeping=(0,))


def softmax_xent(z, y):
    """Mean softmax cross-entropy of logits z [B, C] and its gradient w.r.t. z."""
    z = np.asarray(z, dtype=np.float64)
    B, C = z.shape
    y = np.asarray(y, dtype=np.int64).reshape(-1, 1)
    assert y.min() >= 0 and y.max() < C
    dz, loss = evaluate(_xent_grad_fn(B, C), [z, y])
    return float(loss), dz


@lru_cache(maxsize=16)
def _chain_grad_fn(rows: int, cols: int, simplified: bool) -> Function:
    f = Function("chain8")
    z = f.arg((rows, cols), name="z")
    b = f.arg((1, cols), name="b")
    xs = f.arg((rows, cols), name="x_skip")
    loss, e = _chain_ir(f, z, b, xs, rows, cols)
    f.ret(loss, e)
    if simplified:
        f = simplify_algebra(f)
    return differentiate(f, wrt=[0, 1, 2], keeping=(0, 1))


def chain8(z, b, x_skip, simplified: bool = False):
    """The chain on a given z: returns (loss, dz, db, dx_skip, e)."""
    z = np.asarray(z, dtype=np.float64)
    rows, cols = z.shape
    g = _chain_grad_fn(rows, cols, simplified)
    dz, db, dxs, loss, e = evaluate(
        g, [z, np.asarray(b, dtype=np.float64).reshape(1, -1),
            np.asarray(x_skip, dtype=np.float64)])
    return float(loss), dz, db.reshape(-1), dxs, e


def sgd_f32(param, grad, lr: float) -> np.ndarray:
    """Plain SGD on float32 storage: ``W <- W - lr * dW``, rounded to float32.

    The update rule is not part of the paper; it is the usual one (no momentum,
    no weight decay; biases are updated like weights).
    """
    lr64 = float(np.float32(lr))
    p = np.asarray(param, dtype=np.float32).astype(np.float64)
    g = np.asarray(grad, dtype=np.float32).astype(np.float64)
    return (p - lr64 * g).astype(np.float32)


def sgd_bf16(master, grad, lr: float):
    """SGD on a float32 master copy plus its bf16 shadow: returns (master', shadow')."""
    m = sgd_f32(master, grad, lr)
    return m, round_to_bf16(m)


def gemm(a, b) -> np.ndarray:
    """The ``dot`` instruction: a plain float64 matrix product."""
    return np.asarray(a, dtype=np.float64) @ np.asarray(b, dtype=np.float64)


# ---------------------------------------------------------------------------
# Single dense-layer steps (for checking each fused kernel on its own)
# ---------------------------------------------------------------------------
@lru_cache(maxsize=64)
def _dense_fn(M: int, N: int, K: int, act: str, alpha: float) -> Function:
    """dense(x, W, b) = act(alpha * x.W + b)."""
    f = Function("dense")
    x = f.arg((M, K), name="x")
    W = f.arg((K, N), name="W")
    b = f.arg((1, N), name="b")
    f.ret(_act(f, act, f.add(f.mul(f.dot(x, W), f.const(alpha)), b)))
    return f


def dense_forward(x, W, b, act: str = "none", alpha: float = 1.0) -> np.ndarray:
    """act(alpha * x.W + b) in float64 (b may be None for no bias)."""
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    M, K = x.shape
    N = W.shape[1]
    b = np.zeros((1, N)) if b is None else np.asarray(b, np.float64).reshape(1, N)
    out, = evaluate(_dense_fn(M, N, K, act, float(alpha)), [x, W, b])
    return out


@lru_cache(maxsize=64)
def _act_dot_vjp_fn(M: int, N: int, K: int, act: str) -> Function:
    """[gradient @g wrt 0 seedable] for g(u, W) = dot(act(u), W).

    g maps the previous layer's pre-activation u [M, K] through its activation
    and the next layer's weights W [K, N]: g(u) = dot(act(u), W). Its
    vector-Jacobian product with seed dY [M, N] is (dY.W^T) * act'(u).
    """
    f = Function("act_dot")
    u = f.arg((M, K), name="u")
    W = f.arg((K, N), name="W")
    f.ret(f.dot(_act(f, act, u), W))
    return differentiate(f, wrt=[0], seedable=True)


def dense_vjp_input(u, W, dY, act_prev: str = "none") -> np.ndarray:
    """Adjoint with respect to the previous pre-activation u: (dY.W^T) * act'(u)."""
    u = np.asarray(u, np.float64)
    W = np.asarray(W, np.float64)
    M, K = u.shape
    N = W.shape[1]
    du, = evaluate(_act_dot_vjp_fn(M, N, K, act_prev), [u, W, np.asarray(dY, np.float64)])
    return du


@lru_cache(maxsize=64)
def _linear_params_vjp_fn(M: int, N: int, K: int) -> Function:
    """Fig. 3's declaration 'wrt 1, 2 seedable' of foo(x, W, b) = dot(x, W) + b."""
    f = Function("foo")
    x = f.arg((M, K), name="x")
    W = f.arg((K, N), name="W")
    b = f.arg((1, N), name="b")
    f.ret(f.add(f.dot(x, W), b))
    return differentiate(f, wrt=[1, 2], seedable=True)


def dense_vjp_params(x, dY):
    """(dW, db) = (x^T.dY, column sums of dY), via the seedable gradient of foo."""
    x = np.asarray(x, np.float64)
    dY = np.asarray(dY, np.float64)
    M, K = x.shape
    N = dY.shape[1]
    dW, db = evaluate(_linear_params_vjp_fn(M, N, K),
                      [x, np.zeros((K, N)), np.zeros((1, N)), dY])
    return dW, db.reshape(-1)


def apply_act(u, act: str) -> np.ndarray:
    """act(u) in float64, through the same IR composites as the network."""
    u = np.asarray(u, np.float64)
    f = Function("act")
    a = f.arg(u.shape)
    f.ret(_act(f, act, a))
    out, = evaluate(f, [u])
    return out
