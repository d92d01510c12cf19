"""A small SSA tensor IR and its float64 interpreter (the oracle's core).

TEST INFRASTRUCTURE ONLY. The oracle is a plain, slow, obviously correct CPU
reference for the hot path. Only the test suite, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import it; the product library
never does, and the two share no code.

What it follows (DLVM, arXiv 1711.03016):

* §3.1.1: a function is a list of instructions in static single assignment
  form; each instruction defines exactly one value and its operands are
  earlier values (function arguments or results of earlier instructions).
  The hot path is straight-line code, so a function here is one basic block.
* §3.1.1 / Table 1: the instruction kinds used here are the element-wise
  unary operators (``neg``, ``exp``, ``log``, ``tanh``), the element-wise
  binary operators with broadcasting (``add``, ``sub``, ``mul``, ``div``,
  ``power``), ``dot``, ``transpose``, ``reduce ... by add along <axis>``,
  compare (``gt``, ``eq``) and ``select``. Composite functions (sigmoid,
  softmax, ReLU) are *not* instructions; they are composed from these
  primitives (§3.1.1, last paragraph; §2 on min/max via compare and select).
* ``reduce_max`` is the "reduce by max" form of the reduce instruction. It is
  used only for the shift that keeps softmax finite; see ``oracle.ad`` for how
  its adjoint is treated.
* ``broadcast`` materialises a NumPy-style broadcast; it is the explicit form
  of the implicit broadcasting of element-wise binary operators and is what the
  adjoint of a reduction expands into.
* ``cast`` is Table 1's ``dataTypeCast``. Only the cast to bf16 is used: the
  value becomes the bf16 number nearest (round to nearest, ties to even) to the
  float32 rounding of the operand, kept as a float64. A network stored in bf16
  is the function with such a cast on every activation it stores.

Every value is a NumPy array. Floating-point values are float64 throughout;
``bool`` values come from compare instructions and ``int64`` values are
integer arguments (class labels) or integer constants (``iota``).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

F64 = "f64"
BOOL = "bool"
I64 = "i64"

_NP_DTYPE = {F64: np.float64, BOOL: np.bool_, I64: np.int64}

UNARY = ("neg", "exp", "log", "tanh")
BINARY = ("add", "sub", "mul", "div")
COMPARE = ("gt", "eq")


@dataclass
class Instr:
    """One SSA instruction: ``op`` applied to earlier values ``args``."""

    op: str
    args: tuple
    shape: tuple
    dtype: str
    attrs: dict = field(default_factory=dict)


def _broadcast_shape(a: tuple, b: tuple) -> tuple:
    return tuple(np.broadcast_shapes(a, b))


class Function:
    """A straight-line SSA function: arguments, instructions, returned values.

    Values are referred to by their integer index in ``self.instrs``; argument
    values are instructions of kind ``arg``.
    """

    def __init__(self, name: str):
        self.name = name
        self.instrs: list[Instr] = []
        self.arg_ids: list[int] = []
        self.returns: list[int] = []

    # -- construction -----------------------------------------------------
    def _add(self, ins: Instr) -> int:
        self.instrs.append(ins)
        return len(self.instrs) - 1

    def shape(self, v: int) -> tuple:
        return self.instrs[v].shape

    def dtype(self, v: int) -> str:
        return self.instrs[v].dtype

    def arg(self, shape, dtype: str = F64, name: str = "") -> int:
        v = self._add(Instr("arg", (), tuple(shape), dtype,
                            {"index": len(self.arg_ids), "name": name}))
        self.arg_ids.append(v)
        return v

    def const(self, value, shape=()) -> int:
        """A float64 constant, filled with ``value`` and of ``shape``."""
        return self._add(Instr("const", (), tuple(shape), F64,
                               {"value": float(value)}))

    def iota(self, n: int) -> int:
        """The integer row vector ``[[0, 1, ..., n-1]]``."""
        return self._add(Instr("iota", (), (1, n), I64, {"n": int(n)}))

    def unary(self, op: str, a: int) -> int:
        assert op in UNARY and self.dtype(a) == F64
        return self._add(Instr(op, (a,), self.shape(a), F64))

    def binary(self, op: str, a: int, b: int) -> int:
        assert op in BINARY and self.dtype(a) == F64 and self.dtype(b) == F64
        return self._add(Instr(op, (a, b),
                               _broadcast_shape(self.shape(a), self.shape(b)), F64))

    def power(self, a: int, k: float) -> int:
        """Element-wise ``a ** k`` for a scalar constant exponent ``k``."""
        return self._add(Instr("power", (a,), self.shape(a), F64, {"k": float(k)}))

    def compare(self, op: str, a: int, b: int) -> int:
        assert op in COMPARE
        return self._add(Instr(op, (a, b),
                               _broadcast_shape(self.shape(a), self.shape(b)), BOOL))

    def select(self, cond: int, a: int, b: int) -> int:
        """Element-wise ``cond ? a : b`` (with broadcasting)."""
        assert self.dtype(cond) == BOOL
        shp = _broadcast_shape(self.shape(cond),
                               _broadcast_shape(self.shape(a), self.shape(b)))
        return self._add(Instr("select", (cond, a, b), shp, F64))

    def dot(self, a: int, b: int, acc: str = "f64") -> int:
        """Matrix product; ``acc="f32"`` accumulates in float32 instead of float64.

        The float32 form exists only to measure how much a network's results
        depend on the accumulation order (see ``MlpSpec.accumulate``).
        """
        (m, k1), (k2, n) = self.shape(a), self.shape(b)
        assert k1 == k2, (self.shape(a), self.shape(b))
        assert acc in ("f64", "f32")
        attrs = {"acc": acc} if acc == "f32" else {}
        return self._add(Instr("dot", (a, b), (m, n), F64, attrs))

    def transpose(self, a: int) -> int:
        m, n = self.shape(a)
        return self._add(Instr("transpose", (a,), (n, m), F64))

    def reduce(self, kind: str, a: int, axis) -> int:
        """``reduce a by <kind> along axis`` keeping the reduced axis as size 1.

        ``axis=None`` reduces every axis and yields a scalar (shape ``()``).
        """
        assert kind in ("add", "max")
        shp = self.shape(a)
        if axis is None:
            out = ()
        else:
            out = tuple(1 if i == axis else s for i, s in enumerate(shp))
        return self._add(Instr("reduce_" + kind, (a,), out, F64, {"axis": axis}))

    def cast(self, a: int, to: str = "bf16") -> int:
        """``dataTypeCast a to <to>`` (only bf16 is used)."""
        assert to == "bf16" and self.dtype(a) == F64
        return self._add(Instr("cast", (a,), self.shape(a), F64, {"to": to}))

    def broadcast(self, a: int, shape) -> int:
        shape = tuple(shape)
        assert _broadcast_shape(self.shape(a), shape) == shape
        return self._add(Instr("broadcast", (a,), shape, self.dtype(a)))

    def ret(self, *values: int) -> None:
        self.returns = list(values)

    # -- convenience composites (built from primitives, never new opcodes) --
    def add(self, a, b):
        return self.binary("add", a, b)

    def sub(self, a, b):
        return self.binary("sub", a, b)

    def mul(self, a, b):
        return self.binary("mul", a, b)

    def div(self, a, b):
        return self.binary("div", a, b)

    def neg(self, a):
        return self.unary("neg", a)

    def exp(self, a):
        return self.unary("exp", a)

    def log(self, a):
        return self.unary("log", a)

    def tanh(self, a):
        return self.unary("tanh", a)

    def sigmoid(self, a: int) -> int:
        """sigmoid(a) = 1 / (1 + exp(-a)), composed from primitives."""
        one = self.const(1.0)
        return self.div(one, self.add(one, self.exp(self.neg(a))))

    def relu(self, a: int) -> int:
        """relu(a) = select(a > 0, a, 0), composed from compare and select."""
        zero = self.const(0.0)
        return self.select(self.compare("gt", a, zero), a, zero)

    def __len__(self):
        return len(self.instrs)

    def dump(self) -> str:
        """A readable listing (for debugging and for tests that inspect it)."""
        lines = [f"func @{self.name}"]
        for i, ins in enumerate(self.instrs):
            a = ", ".join(f"%{j}" for j in ins.args)
            extra = "" if not ins.attrs else " " + str(ins.attrs)
            lines.append(f"  %{i} = {ins.op} {a}{extra} : {ins.shape} {ins.dtype}")
        lines.append("  return " + ", ".join(f"%{j}" for j in self.returns))
        return "\n".join(lines)


def _eval_instr(ins: Instr, vals: list, args: list):
    op = ins.op
    if op == "arg":
        x = np.asarray(args[ins.attrs["index"]], dtype=_NP_DTYPE[ins.dtype])
        assert x.shape == ins.shape, (ins.attrs, x.shape, ins.shape)
        return x
    if op == "const":
        return np.full(ins.shape, ins.attrs["value"], dtype=np.float64)
    if op == "iota":
        return np.arange(ins.attrs["n"], dtype=np.int64)[None, :]
    a = [vals[j] for j in ins.args]
    if op == "neg":
        return -a[0]
    if op == "exp":
        return np.exp(a[0])
    if op == "log":
        return np.log(a[0])
    if op == "tanh":
        return np.tanh(a[0])
    if op == "add":
        return a[0] + a[1]
    if op == "sub":
        return a[0] - a[1]
    if op == "mul":
        return a[0] * a[1]
    if op == "div":
        return a[0] / a[1]
    if op == "power":
        return np.power(a[0], ins.attrs["k"])
    if op == "gt":
        return a[0] > a[1]
    if op == "eq":
        return a[0] == a[1]
    if op == "select":
        return np.where(a[0], a[1], a[2])
    if op == "dot":
        if ins.attrs.get("acc") == "f32":
            return (a[0].astype(np.float32) @ a[1].astype(np.float32)).astype(np.float64)
        return a[0] @ a[1]
    if op == "transpose":
        return a[0].T
    if op == "reduce_add":
        ax = ins.attrs["axis"]
        return a[0].sum() if ax is None else a[0].sum(axis=ax, keepdims=True)
    if op == "reduce_max":
        ax = ins.attrs["axis"]
        return a[0].max() if ax is None else a[0].max(axis=ax, keepdims=True)
    if op == "broadcast":
        return np.broadcast_to(a[0], ins.shape).copy()
    if op == "cast":
        from .bf16 import round_to_bf16
        return round_to_bf16(a[0].astype(np.float32))
    raise ValueError(f"unknown op {op}")


def evaluate(fn: Function, args, trace: bool = False):
    """Run ``fn`` on ``args`` in float64; return its results (and all values).

    Instructions are evaluated in program order; each instruction's value is
    stored so later instructions (and, when ``trace`` is set, the caller) can
    read it.
    """
    assert len(args) == len(fn.arg_ids), (len(args), len(fn.arg_ids))
    vals: list = [None] * len(fn.instrs)
    for i, ins in enumerate(fn.instrs):
        v = _eval_instr(ins, vals, args)
        v = np.asarray(v)
        assert v.shape == ins.shape, (i, ins.op, v.shape, ins.shape)
        vals[i] = v
    out = [vals[r] for r in fn.returns]
    return (out, vals) if trace else out
