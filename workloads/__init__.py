"""Seeded synthetic workloads for the MLP hot path: shapes and input generators.

This module only draws random inputs and describes the five workload shapes;
it holds none of the method's arithmetic, so both the GPU path's tests and the
oracle may use it.

Every tensor has its own NumPy PCG64 stream seeded with ``(seed, tensor_id)``,
so any tensor can be regenerated on its own. Values are drawn in float32
(float32 is the storage type the inputs are handed over in; bf16 workloads
round them on each side independently).

Initialisers:
* Xavier-uniform: U(-a, a), a = sqrt(6 / (fan_in + fan_out));
* Kaiming-normal: N(0, 2 / fan_in);
* ``normal_var=v``: N(0, v) (the second parameter is a variance);
* biases are zero unless a test asks for U(-s, s) biases to exercise the bias path.
Labels are uniform integers in [0, classes).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 0x1711_03016


@dataclass(frozen=True)
class Workload:
    name: str
    title: str
    widths: tuple
    acts: tuple
    loss: str            # "softmax_ce" or "chain8"
    dtype: str           # storage type: "f32" or "bf16"
    batch: int
    x_init: tuple        # ("uniform", lo, hi) or ("normal_var", var)
    w_init: tuple        # ("xavier_uniform",), ("kaiming_normal",) or ("normal_var", var)
    sgd: bool = False
    lr: float = 0.01
    wrt_x: bool = False
    notes: str = field(default="", compare=False)

    @property
    def n_layers(self) -> int:
        return len(self.widths) - 1

    @property
    def classes(self) -> int:
        return self.widths[-1]

    def flops(self, batch: int | None = None) -> int:
        """Algorithmic GEMM flops of one forward + gradient: 2*M*N*K per GEMM.

        Counts the forward GEMM of every layer, the weight-gradient GEMM of
        every layer and the input-gradient GEMM of every layer but the first
        (the first is counted only when x is differentiated).
        """
        B = self.batch if batch is None else batch
        fl = 0
        for l in range(self.n_layers):
            k, n = self.widths[l], self.widths[l + 1]
            fl += 2 * B * n * k          # forward
            fl += 2 * k * n * B          # dW
            if l > 0 or self.wrt_x:
                fl += 2 * B * k * n      # dX
        return fl

    def param_count(self) -> int:
        return sum(self.widths[l] * self.widths[l + 1] + self.widths[l + 1]
                   for l in range(self.n_layers))


WORKLOADS = {
    "c1": Workload(
        "c1", "tiny MLP f32 64-32(sigmoid)-10, softmax-CE, batch 16",
        (64, 32, 10), ("sigmoid", "none"), "softmax_ce", "f32", 16,
        ("uniform", -1.0, 1.0), ("xavier_uniform",)),
    "c2": Workload(
        "c2", "MLP f32 784-512(tanh)-512(tanh)-10, softmax-CE, batch 256, SGD lr 0.01",
        (784, 512, 512, 10), ("tanh", "tanh", "none"), "softmax_ce", "f32", 256,
        ("uniform", 0.0, 1.0), ("xavier_uniform",), sgd=True, lr=0.01),
    "c3": Workload(
        "c3", "MLP bf16 784-1024(relu)-1024(relu)-10, softmax-CE, batch 4096",
        (784, 1024, 1024, 10), ("relu", "relu", "none"), "softmax_ce", "bf16", 4096,
        ("normal_var", 1.0), ("kaiming_normal",)),
    "c4": Workload(
        "c4", "f32 dense 4096-4096 + 8-op element-wise chain, batch 8192",
        (4096, 4096), ("none",), "chain8", "f32", 8192,
        ("normal_var", 1.0 / 4096), ("normal_var", 1.0 / 4096), wrt_x=True),
    "c5": Workload(
        "c5", "deep MLP bf16 4096-8x4096(relu)-1000, softmax-CE, batch 16384, SGD",
        (4096,) + (4096,) * 8 + (1000,), ("relu",) * 8 + ("none",), "softmax_ce",
        "bf16", 16384, ("normal_var", 1.0), ("kaiming_normal",), sgd=True, lr=0.01),
}


def _rng(seed: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng([int(seed) & 0xFFFFFFFFFFFF, int(tensor_id)])


def _draw(rng: np.random.Generator, shape, init: tuple, fan_in: int = 1,
          fan_out: int = 1) -> np.ndarray:
    kind = init[0]
    if kind == "uniform":
        return rng.uniform(init[1], init[2], size=shape).astype(np.float32)
    if kind == "normal_var":
        return (rng.standard_normal(size=shape, dtype=np.float32)
                * np.float32(np.sqrt(init[1])))
    if kind == "xavier_uniform":
        a = np.sqrt(6.0 / (fan_in + fan_out))
        return rng.uniform(-a, a, size=shape).astype(np.float32)
    if kind == "kaiming_normal":
        return (rng.standard_normal(size=shape, dtype=np.float32)
                * np.float32(np.sqrt(2.0 / fan_in)))
    raise ValueError(kind)


def make_params(wl: Workload, seed: int | None = None, bias_scale: float = 0.0):
    """Weights [in, out] and biases [out] of every layer, float32."""
    seed = SEED_BASE if seed is None else seed
    params = []
    for l in range(wl.n_layers):
        k, n = wl.widths[l], wl.widths[l + 1]
        W = _draw(_rng(seed, 100 + 2 * l), (k, n), wl.w_init, k, n)
        if bias_scale > 0:
            b = _rng(seed, 101 + 2 * l).uniform(-bias_scale, bias_scale, n).astype(np.float32)
        else:
            b = np.zeros(n, dtype=np.float32)
        params.append((W, b))
    return params


def make_x(wl: Workload, batch: int | None = None, seed: int | None = None) -> np.ndarray:
    seed = SEED_BASE if seed is None else seed
    B = wl.batch if batch is None else batch
    return _draw(_rng(seed, 1), (B, wl.widths[0]), wl.x_init)


def make_labels(wl: Workload, batch: int | None = None, seed: int | None = None):
    """Uniform class labels in [0, classes) as int32 (None for the chain workload)."""
    if wl.loss != "softmax_ce":
        return None
    seed = SEED_BASE if seed is None else seed
    B = wl.batch if batch is None else batch
    return _rng(seed, 2).integers(0, wl.classes, size=B, dtype=np.int64).astype(np.int32)


def make_inputs(wl: Workload, batch: int | None = None, seed: int | None = None,
                bias_scale: float = 0.0):
    """(x, params, labels) for a workload, optionally at another batch size."""
    return (make_x(wl, batch, seed), make_params(wl, seed, bias_scale),
            make_labels(wl, batch, seed))


def repeat_rows(base_x: np.ndarray, base_y, batch: int, seed: int = 7):
    """A batch made of the rows of ``base_x`` each repeated ``batch/len(base_x)`` times.

    The rows are placed in a seeded random order. Every base row occurs the
    same number of times, so any quantity that is a mean over the batch of a
    per-row quantity (a mean loss and its gradient) equals the same mean over
    the base rows alone. Returns (x, y, idx) with ``x = base_x[idx]``.
    """
    nb = base_x.shape[0]
    assert batch % nb == 0
    idx = np.tile(np.arange(nb), batch // nb)
    idx = _rng(seed, 3).permutation(idx)
    x = np.ascontiguousarray(base_x[idx])
    y = None if base_y is None else np.ascontiguousarray(np.asarray(base_y)[idx])
    return x, y, idx


def scaled(wl: Workload, width_div: int = 1, batch: int | None = None) -> Workload:
    """The same network family with hidden widths divided by ``width_div``.

    Input and output widths are kept (the input width fixes x's features and
    the output width the class count) unless the chain workload needs
    in == out, in which case both shrink.
    """
    w = list(wl.widths)
    if wl.loss == "chain8":
        w = [max(1, v // width_div) for v in w]
    else:
        for i in range(1, len(w) - 1):
            w[i] = max(1, w[i] // width_div)
    from dataclasses import replace
    return replace(wl, widths=tuple(w), batch=wl.batch if batch is None else batch)


# ---------------------------------------------------------------------------
# Recurrent cell (the RNN example of linear-algebra fusion): seeded inputs.
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class RnnWorkload:
    """T steps of hs[t+1] = act(xs[t] . W + hs[t] . U + b) and their seeded
    backward pass. Inputs x ~ N(0, 1), h0 ~ U(-0.5, 0.5); the stacked [W; U]
    has fan-in Kx + H and is drawn N(0, 1 / (Kx + H)) (pre-activations of
    unit variance); b ~ U(-0.1, 0.1); the output adjoints dhs ~ N(0, 1) / B
    (what a loss averaged over the batch hands back)."""

    name: str
    title: str
    steps: int
    in_width: int
    hidden: int
    act: str
    dtype: str
    batch: int
    sgd: bool = True
    lr: float = 0.01
    wrt_x: bool = True
    wrt_h0: bool = True

    def flops(self, batch: int | None = None) -> int:
        """Algorithmic GEMM flops of one forward + backward pass.

        Forward: T products [B, Kx + H] x [Kx + H, H]. Backward: T - 1
        recurrent products [B, H] x [H, H] (+1 for dh0), the weight gradient
        [Kx + H, T B] x [T B, H], and dxs [T B, H] x [H, Kx] when declared.
        """
        B = self.batch if batch is None else batch
        T, Kx, H = self.steps, self.in_width, self.hidden
        fl = T * 2 * B * H * (Kx + H)
        fl += (T - 1 + (1 if self.wrt_h0 else 0)) * 2 * B * H * H
        fl += 2 * (Kx + H) * H * T * B
        if self.wrt_x:
            fl += 2 * T * B * H * Kx
        return fl


RNN_WORKLOADS = {
    "r1": RnnWorkload(
        "r1", "RNN cell bf16 tanh, T=32 steps, x 1024 -> h 1024, batch 1024, BPTT + SGD",
        32, 1024, 1024, "tanh", "bf16", 1024),
}


def make_rnn_inputs(wl: RnnWorkload, batch: int | None = None, seed: int | None = None):
    """(xs [T, B, Kx], h0 [B, H], W [Kx, H], U [H, H], b [H], dhs [T, B, H]), float32."""
    seed = SEED_BASE if seed is None else seed
    B = wl.batch if batch is None else batch
    T, Kx, H = wl.steps, wl.in_width, wl.hidden
    xs = _draw(_rng(seed, 201), (T, B, Kx), ("normal_var", 1.0))
    h0 = _draw(_rng(seed, 202), (B, H), ("uniform", -0.5, 0.5))
    var = ("normal_var", 1.0 / (Kx + H))
    W = _draw(_rng(seed, 203), (Kx, H), var)
    U = _draw(_rng(seed, 204), (H, H), var)
    b = _draw(_rng(seed, 205), (H,), ("uniform", -0.1, 0.1))
    dhs = _draw(_rng(seed, 206), (T, B, H), ("normal_var", 1.0)) / np.float32(B)
    return xs, h0, W, U, b, dhs


# ---------------------------------------------------------------------------
# Matrix chains (the reordering row): seeded inputs.
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class ChainWorkload:
    """The product A_0 ... A_{n-1}, A_i of shape dims[i] x dims[i+1], entries
    N(0, 1 / dims[i]) (each product keeps unit-variance entries)."""

    name: str
    title: str
    dims: tuple
    dtype: str

    @property
    def n(self) -> int:
        return len(self.dims) - 1


CHAIN_WORKLOADS = {
    "m1": ChainWorkload(
        "m1", "bf16 chain 16384x4096 . 4096x64 . 64x4096 . 4096x64 . 64x1024 (low-rank factors)",
        (16384, 4096, 64, 4096, 64, 1024), "bf16"),
}


def make_chain_inputs(dims, seed: int | None = None):
    """The chain's matrices, float32."""
    seed = SEED_BASE if seed is None else seed
    return [_draw(_rng(seed, 300 + i), (dims[i], dims[i + 1]), ("normal_var", 1.0 / dims[i]))
            for i in range(len(dims) - 1)]
