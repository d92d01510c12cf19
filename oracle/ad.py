"""Reverse-mode AD by adjoint code generation, plus ADCE and algebra simplification.

TEST INFRASTRUCTURE ONLY (see ``oracle/ir.py``).

The differentiation pass follows DLVM §3.1.3: a gradient declaration is turned
into an ordinary function by first copying the instructions of the original
function into the new body and then appending adjoint code that walks the
copied instructions in reverse order. The result is a standalone function of
the original inputs that returns the requested partial derivatives followed by
any original outputs that the declaration keeps (Fig. 3, ``wrt ... keeping
... seedable``). With ``seedable`` the incoming adjoint (the seed) is an extra
last argument; otherwise the seed is all ones, so for a scalar output the
result is the gradient and for a tensor output it is the vector-Jacobian
product with a ones vector, which is what Fig. 3's ``@foo_grad`` returns.

Afterwards, aggressive dead code elimination (§3.1.4) removes every
instruction that no returned value depends on; this is what drops forward and
adjoint work that the declared derivatives do not need (§3.1.3).

The adjoint rules are the textbook ones for each primitive. Where an operand
was broadcast (all element-wise binary operators broadcast, §3.1.1), its
adjoint is summed over the broadcast axes.

``cast`` (dataTypeCast to bf16) is differentiated as the identity: its adjoint
is the incoming adjoint cast back to the operand's type, which in float64 is
the incoming adjoint itself. (Rounding is piecewise constant; the convention
used by every mixed-precision program is to pass the adjoint straight through.)

``reduce_max`` only ever appears as the shift inside log-sum-exp. Its adjoint
is routed to the positions that attain the maximum (compare + select); in the
shift-invariant composite the two contributions through the shift cancel, so
the result is the exact gradient up to rounding.
"""
from __future__ import annotations

from .ir import BOOL, F64, Function, Instr

# Instructions through which derivatives flow.
_DIFFERENTIABLE = {
    "neg", "exp", "log", "tanh", "add", "sub", "mul", "div", "power",
    "select", "dot", "transpose", "reduce_add", "reduce_max", "broadcast", "cast",
}


def _copy_into(src: Function, dst: Function) -> dict:
    """Copy every instruction of ``src`` into ``dst``; return the id mapping."""
    vmap = {}
    for i, ins in enumerate(src.instrs):
        if ins.op == "arg":
            vmap[i] = dst.arg(ins.shape, ins.dtype, ins.attrs.get("name", ""))
        else:
            vmap[i] = dst._add(Instr(ins.op, tuple(vmap[a] for a in ins.args),
                                     ins.shape, ins.dtype, dict(ins.attrs)))
    return vmap


def _unbroadcast(g: Function, v: int, shape: tuple) -> int:
    """Sum ``v`` over the axes along which an operand of ``shape`` was broadcast."""
    vs = g.shape(v)
    if vs == tuple(shape):
        return v
    if shape == ():
        return g.reduce("add", v, None)
    assert len(shape) == len(vs), (shape, vs)
    out = v
    for ax, (want, have) in enumerate(zip(shape, vs)):
        if want == 1 and have != 1:
            out = g.reduce("add", out, ax)
    assert g.shape(out) == tuple(shape), (g.shape(out), shape)
    return out


def differentiate(fn: Function, wrt, keeping=(), seedable: bool = False,
                  of: int = 0, name: str | None = None) -> Function:
    """Build the gradient function of ``fn`` (a gradient declaration, §3.1.3).

    ``wrt`` lists argument indices to differentiate with respect to, ``of``
    the index of the returned value being differentiated, ``keeping`` the
    indices of original returned values to append to the result, and
    ``seedable`` adds the seed as a trailing argument.
    Returns a new function whose results are ``(d/d arg_i for i in wrt) +
    (kept outputs)``.
    """
    g = Function(name or fn.name + "_grad")
    vmap = _copy_into(fn, g)
    n_fwd = len(g.instrs)
    y = vmap[fn.returns[of]]
    if seedable:
        seed = g.arg(g.shape(y), F64, "seed")
    else:
        seed = g.const(1.0, g.shape(y))

    wrt_vals = [vmap[fn.arg_ids[i]] for i in wrt]
    for w in wrt_vals:
        assert g.dtype(w) == F64, "cannot differentiate with respect to a non-float argument"

    # Activity: a value is active if it depends on a wrt argument through
    # differentiable instructions.
    active = set(wrt_vals)
    for v in range(n_fwd):
        ins = g.instrs[v]
        if ins.op in _DIFFERENTIABLE and any(a in active for a in ins.args):
            active.add(v)

    adj: dict[int, int] = {y: seed}

    def acc(target: int, contrib: int) -> None:
        if target not in active:
            return
        assert g.shape(contrib) == g.shape(target), (g.shape(contrib), g.shape(target))
        adj[target] = g.add(adj[target], contrib) if target in adj else contrib

    for v in reversed(range(n_fwd)):
        if v not in adj or v not in active:
            continue
        vb = adj[v]
        ins = g.instrs[v]
        op, a = ins.op, ins.args
        if op == "arg":
            continue
        if op == "neg":
            acc(a[0], g.neg(vb))
        elif op == "exp":
            acc(a[0], g.mul(vb, v))
        elif op == "log":
            acc(a[0], g.div(vb, a[0]))
        elif op == "tanh":
            one = g.const(1.0)
            acc(a[0], g.mul(vb, g.sub(one, g.mul(v, v))))
        elif op == "add":
            if a[0] in active:
                acc(a[0], _unbroadcast(g, vb, g.shape(a[0])))
            if a[1] in active:
                acc(a[1], _unbroadcast(g, vb, g.shape(a[1])))
        elif op == "sub":
            if a[0] in active:
                acc(a[0], _unbroadcast(g, vb, g.shape(a[0])))
            if a[1] in active:
                acc(a[1], _unbroadcast(g, g.neg(vb), g.shape(a[1])))
        elif op == "mul":
            if a[0] in active:
                acc(a[0], _unbroadcast(g, g.mul(vb, a[1]), g.shape(a[0])))
            if a[1] in active:
                acc(a[1], _unbroadcast(g, g.mul(vb, a[0]), g.shape(a[1])))
        elif op == "div":
            # v = a0 / a1;  d v / d a0 = 1 / a1;  d v / d a1 = -a0 / a1^2 = -v / a1
            if a[0] in active:
                acc(a[0], _unbroadcast(g, g.div(vb, a[1]), g.shape(a[0])))
            if a[1] in active:
                acc(a[1], _unbroadcast(g, g.neg(g.div(g.mul(vb, v), a[1])),
                                       g.shape(a[1])))
        elif op == "power":
            k = ins.attrs["k"]
            if k != 0.0:  # x^0 is the constant 1: no contribution
                acc(a[0], g.mul(vb, g.mul(g.const(k), g.power(a[0], k - 1.0))))
        elif op == "select":
            zero = g.const(0.0)
            if a[1] in active:
                acc(a[1], _unbroadcast(g, g.select(a[0], vb, zero), g.shape(a[1])))
            if a[2] in active:
                acc(a[2], _unbroadcast(g, g.select(a[0], zero, vb), g.shape(a[2])))
        elif op == "dot":
            # C = A B:  dA = dC B^T,  dB = A^T dC
            if a[0] in active:
                acc(a[0], g.dot(vb, g.transpose(a[1])))
            if a[1] in active:
                acc(a[1], g.dot(g.transpose(a[0]), vb))
        elif op == "transpose":
            acc(a[0], g.transpose(vb))
        elif op == "reduce_add":
            acc(a[0], g.broadcast(vb, g.shape(a[0])))
        elif op == "reduce_max":
            hit = g.compare("eq", a[0], g.broadcast(v, g.shape(a[0])))
            acc(a[0], g.select(hit, g.broadcast(vb, g.shape(a[0])), g.const(0.0)))
        elif op == "broadcast":
            acc(a[0], _unbroadcast(g, vb, g.shape(a[0])))
        elif op == "cast":
            acc(a[0], vb)
        else:  # compare, iota, const: no adjoint flows through these
            raise AssertionError(f"active value from non-differentiable op {op}")

    outs = []
    for w in wrt_vals:
        outs.append(adj[w] if w in adj else g.const(0.0, g.shape(w)))
    outs += [vmap[fn.returns[k]] for k in keeping]
    g.ret(*outs)
    return adce(g)


def adce(fn: Function) -> Function:
    """Aggressive dead code elimination (§3.1.4).

    Keeps the arguments (the signature) and every instruction that some
    returned value transitively depends on; removes everything else.
    """
    live = set(fn.returns)
    for v in reversed(range(len(fn.instrs))):
        if v in live:
            live.update(fn.instrs[v].args)
    out = Function(fn.name)
    vmap = {}
    for i, ins in enumerate(fn.instrs):
        if ins.op == "arg":
            vmap[i] = out.arg(ins.shape, ins.dtype, ins.attrs.get("name", ""))
        elif i in live:
            vmap[i] = out._add(Instr(ins.op, tuple(vmap[a] for a in ins.args),
                                     ins.shape, ins.dtype, dict(ins.attrs)))
    out.ret(*[vmap[r] for r in fn.returns])
    return out


def simplify_algebra(fn: Function) -> Function:
    """Algebra simplification (§3.1.2): ``x^2 -> x (.) x``, ``x^0 -> 1``, ``x^1 -> x``."""
    out = Function(fn.name)
    vmap = {}
    for i, ins in enumerate(fn.instrs):
        if ins.op == "arg":
            vmap[i] = out.arg(ins.shape, ins.dtype, ins.attrs.get("name", ""))
            continue
        args = tuple(vmap[a] for a in ins.args)
        if ins.op == "power" and ins.attrs["k"] == 2.0:
            vmap[i] = out.mul(args[0], args[0])
        elif ins.op == "power" and ins.attrs["k"] == 0.0:
            vmap[i] = out.const(1.0, ins.shape)
        elif ins.op == "power" and ins.attrs["k"] == 1.0:
            vmap[i] = args[0]
        else:
            vmap[i] = out._add(Instr(ins.op, args, ins.shape, ins.dtype, dict(ins.attrs)))
    out.ret(*[vmap[r] for r in fn.returns])
    return out


def count_ops(fn: Function, op: str) -> int:
    return sum(1 for ins in fn.instrs if ins.op == op)


__all__ = ["differentiate", "adce", "simplify_algebra", "count_ops", "BOOL"]
