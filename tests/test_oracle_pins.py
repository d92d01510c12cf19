"""Pins of the oracle against facts that do not come from the oracle itself.

Each test checks the float64 oracle against something the paper or the
mathematics fixes: central finite differences, closed-form derivatives
written in a different form from the oracle's adjoint rules, invariants,
special cases with known values, hand-worked values of Fig. 3, the
linear-algebra identities of §3.1.2, and an independent library autograd
(PyTorch float64 on the CPU). Planted mistakes in a copy of the oracle's
generated adjoint code must be caught by the finite-difference check.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import workloads
from oracle import MlpSpec
from oracle.ad import adce, count_ops, differentiate, simplify_algebra
from oracle.ir import I64, Function, Instr, evaluate
from oracle.mlp import build_mlp_gradient, build_mlp_logits, build_mlp_loss, build_mlp_vjp

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# helpers
# --------------------------------------------------------------------------
def _f64_args(spec, x, params, y=None):
    args = [np.asarray(x, np.float64)]
    for W, b in params:
        args += [np.asarray(W, np.float64), np.asarray(b, np.float64).reshape(1, -1)]
    if spec.loss == "softmax_ce":
        args.append(np.asarray(y, np.int64).reshape(-1, 1))
    return args


def _fd_check(f, g, args, wrt, rtol=1e-6, atol=1e-8, max_entries=None, rng=None,
              skip=None):
    """Central finite differences of output 0 of ``f`` against the gradient ``g``.

    Returns the largest violation ratio |fd - ad| / (atol + rtol |ad|); < 1 passes.
    """
    grads = evaluate(g, args)
    worst = 0.0
    for gi, ai in enumerate(wrt):
        base = args[ai]
        idxs = list(np.ndindex(base.shape))
        if max_entries is not None and len(idxs) > max_entries:
            sel = (rng or np.random.default_rng(0)).choice(len(idxs), max_entries, replace=False)
            idxs = [idxs[i] for i in sel]
        for idx in idxs:
            if skip is not None and skip(ai, idx):
                continue
            th = base[idx]
            h = 1e-6 * max(1.0, abs(th))
            pa = list(args)
            p = base.copy(); p[idx] = th + h; pa[ai] = p
            lp = float(evaluate(f, pa)[0])
            m = base.copy(); m[idx] = th - h; pa[ai] = m
            lm = float(evaluate(f, pa)[0])
            fd = (lp - lm) / (2 * h)
            ad = float(grads[gi][idx])
            worst = max(worst, abs(fd - ad) / (atol + rtol * abs(ad)))
    return worst


def _c1_setup(seed=None):
    wl = workloads.WORKLOADS["c1"]
    x, params, y = workloads.make_inputs(wl, seed=seed, bias_scale=0.1)
    spec = MlpSpec(wl.widths, wl.acts, wl.loss, "f32")
    return spec, x, params, y


# --------------------------------------------------------------------------
# finite differences
# --------------------------------------------------------------------------
def test_fd_c1_every_parameter_and_input():
    """C1 (64-32-10 sigmoid, batch 16): all 2,410 parameters and all 1,024 inputs."""
    spec, x, params, y = _c1_setup()
    f = build_mlp_loss(spec, 16)
    g = build_mlp_gradient(spec, 16, True)
    args = _f64_args(spec, x, params, y)
    wrt = [0, 1, 2, 3, 4]   # x, W1, b1, W2, b2
    assert _fd_check(f, g, args, wrt) < 1.0


def test_fd_chain8_small():
    """The eight-operator chain on a shrunken instance (batch 4, 8 -> 8), wrt W, b and x."""
    spec = MlpSpec((8, 8), ("none",), "chain8", "f32")
    rng = np.random.default_rng(5)
    x = rng.standard_normal((4, 8))
    W = rng.standard_normal((8, 8)) * 0.5
    b = rng.standard_normal(8) * 0.3
    f = build_mlp_loss(spec, 4)
    g = build_mlp_gradient(spec, 4, True)
    args = _f64_args(spec, x, [(W, b)])
    assert _fd_check(f, g, args, [0, 1, 2]) < 1.0


def test_fd_relu_and_tanh_mlp():
    """A small ReLU/tanh network; inputs are chosen so no pre-activation is near a kink."""
    spec = MlpSpec((6, 5, 4, 3), ("relu", "tanh", "none"), "softmax_ce", "f32")
    rng = np.random.default_rng(11)
    for _ in range(50):
        x = rng.standard_normal((5, 6))
        params = [(rng.standard_normal((6, 5)), rng.standard_normal(5) * 0.1),
                  (rng.standard_normal((5, 4)), rng.standard_normal(4) * 0.1),
                  (rng.standard_normal((4, 3)), rng.standard_normal(3) * 0.1)]
        v1 = x @ params[0][0] + params[0][1]
        if np.abs(v1).min() > 1e-3:
            break
    y = np.array([0, 2, 1, 1, 0])
    f = build_mlp_loss(spec, 5)
    g = build_mlp_gradient(spec, 5, True)
    assert _fd_check(f, g, _f64_args(spec, x, params, y), [0, 1, 2, 3, 4, 5, 6]) < 1.0


def test_fd_scaled_c3_c5_shapes():
    """Scaled-down C3 (ReLU, 10 classes) and C5-like deep ReLU nets, sampled entries."""
    rng = np.random.default_rng(3)
    for widths in [(20, 12, 12, 10), (16, 8, 8, 8, 8, 9)]:
        L = len(widths) - 1
        spec = MlpSpec(widths, ("relu",) * (L - 1) + ("none",), "softmax_ce", "f32")
        x = rng.standard_normal((7, widths[0]))
        params = [(rng.standard_normal((widths[l], widths[l + 1])) * math.sqrt(2 / widths[l]),
                   rng.standard_normal(widths[l + 1]) * 0.1) for l in range(L)]
        y = rng.integers(0, widths[-1], 7)
        # keep FD away from ReLU kinks: skip entries whose perturbation flips a mask
        f = build_mlp_loss(spec, 7)
        g = build_mlp_gradient(spec, 7, False)
        args = _f64_args(spec, x, params, y)
        _, vals = evaluate(f, args, trace=True)
        pre = [v for ins, v in zip(f.instrs, vals) if ins.op == "add" and v.ndim == 2
               and v.shape[0] == 7]
        margin = min(np.abs(p).min() for p in pre)
        assert margin > 1e-5
        wrt = list(range(1, 1 + 2 * L))
        assert _fd_check(f, g, args, wrt, max_entries=40) < 1.0


# --------------------------------------------------------------------------
# closed forms (written differently from the oracle's adjoint rules)
# --------------------------------------------------------------------------
def _elementwise_grad(build, v):
    f = Function("e")
    a = f.arg(v.shape)
    f.ret(f.reduce("add", build(f, a), None))
    g = differentiate(f, [0])
    return evaluate(g, [v])[0]


def test_sigmoid_derivative_closed_form():
    v = np.linspace(-30, 30, 601).reshape(1, -1)
    d = _elementwise_grad(lambda f, a: f.sigmoid(a), v)
    # s(1-s) written as sigmoid(v) * sigmoid(-v), which does not cancel for large v
    s_pos = 1.0 / (1.0 + np.exp(-v))
    s_neg = 1.0 / (1.0 + np.exp(v))
    np.testing.assert_allclose(d, s_pos * s_neg, rtol=1e-12, atol=1e-300)


def test_tanh_derivative_closed_form():
    v = np.linspace(-10, 10, 401).reshape(1, -1)
    d = _elementwise_grad(lambda f, a: f.tanh(a), v)
    # 1 - t^2 cancels when |t| -> 1: the oracle is accurate to a few ulp of 1 absolute
    np.testing.assert_allclose(d, 1.0 / np.cosh(v) ** 2, rtol=1e-12, atol=1e-15)


def test_relu_derivative_is_select_mask():
    v = np.array([[-2.0, -0.0, 0.0, 1e-300, 3.0]])
    d = _elementwise_grad(lambda f, a: f.relu(a), v)
    np.testing.assert_array_equal(d, [[0.0, 0.0, 0.0, 1.0, 1.0]])


def test_softmax_xent_closed_form():
    from scipy.special import logsumexp, softmax
    rng = np.random.default_rng(1)
    z = rng.standard_normal((33, 17)) * 4
    y = rng.integers(0, 17, 33)
    loss, dz = oracle.softmax_xent(z, y)
    onehot = np.zeros_like(z); onehot[np.arange(33), y] = 1
    ref = np.mean(logsumexp(z, axis=1) - z[np.arange(33), y])
    assert abs(loss - ref) < 1e-13 * abs(ref)
    np.testing.assert_allclose(dz, (softmax(z, axis=1) - onehot) / 33, rtol=1e-12, atol=1e-17)


def test_fig4_tanh_layer_gradient():
    """Fig. 4: g = tanh(x.w + b), gradient wrt (w, b) keeping g, returns (dg/dw, dg/db, g)."""
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 4)); w = rng.standard_normal((4, 3)); b = rng.standard_normal((1, 3))
    f = Function("g")
    xa, wa, ba = f.arg((5, 4)), f.arg((4, 3)), f.arg((1, 3))
    f.ret(f.tanh(f.add(f.dot(xa, wa), ba)))
    dg = differentiate(f, wrt=[1, 2], keeping=(0,))
    dw, db, gval = evaluate(dg, [x, w, b])
    sech2 = 1.0 / np.cosh(x @ w + b) ** 2
    np.testing.assert_allclose(gval, np.tanh(x @ w + b), rtol=1e-15)
    np.testing.assert_allclose(db, sech2.sum(axis=0, keepdims=True), rtol=1e-12)
    np.testing.assert_allclose(dw, x.T @ sech2, rtol=1e-12, atol=1e-14)


def test_fig3_golden_values():
    """Hand-worked values of Fig. 3's @foo and its two gradient declarations."""
    gd = json.load(open(os.path.join(GOLDEN, "fig3_foo.json")))
    x, w, b = (np.array(gd[k]) for k in ("x", "w", "b"))
    f = Function("foo")
    xa, wa, ba = f.arg(x.shape), f.arg(w.shape), f.arg(b.shape)
    f.ret(f.add(f.dot(xa, wa), ba))
    np.testing.assert_array_equal(evaluate(f, [x, w, b])[0], gd["foo"])
    dx, dw, db = evaluate(differentiate(f, wrt=[0, 1, 2]), [x, w, b])
    e = gd["foo_grad_all_ones_seed"]
    np.testing.assert_array_equal(dx, e["dx"])
    np.testing.assert_array_equal(dw, e["dw"])
    np.testing.assert_array_equal(db, e["db"])
    g3 = differentiate(f, wrt=[1, 2], keeping=(0,), seedable=True)
    assert len(g3.arg_ids) == 4          # (x, w, b, seed), as in @foo_grad_3
    dw3, db3, out = evaluate(g3, [x, w, b, np.array(gd["seed"])])
    e = gd["foo_grad_3_wrt_1_2_keeping_0"]
    np.testing.assert_array_equal(dw3, e["dw"])
    np.testing.assert_array_equal(db3, e["db"])
    np.testing.assert_array_equal(out, e["kept_output"])


def test_fig3_shapes():
    """Fig. 3 at its own shapes: x<1x784>, w<784x10>, b<1x10>; gradients are input-shaped."""
    f = Function("foo")
    xa, wa, ba = f.arg((1, 784)), f.arg((784, 10)), f.arg((1, 10))
    f.ret(f.add(f.dot(xa, wa), ba))
    g = differentiate(f, wrt=[0, 1, 2])
    assert [g.shape(r) for r in g.returns] == [(1, 784), (784, 10), (1, 10)]
    g3 = differentiate(f, wrt=[1, 2], keeping=(0,), seedable=True)
    assert [g3.shape(r) for r in g3.returns] == [(784, 10), (1, 10), (1, 10)]


# --------------------------------------------------------------------------
# invariants and special cases of softmax cross-entropy
# --------------------------------------------------------------------------
def test_softmax_rows_and_dlogits_rows():
    rng = np.random.default_rng(4)
    z = rng.standard_normal((64, 10)) * 3
    y = rng.integers(0, 10, 64)
    _, dz = oracle.softmax_xent(z, y)
    onehot = np.zeros_like(z); onehot[np.arange(64), y] = 1
    p = dz * 64 + onehot
    np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-14)
    np.testing.assert_allclose(dz.sum(axis=1), 0.0, atol=1e-16)
    assert (p > 0).all()
    # the only negative entry of each row sits at the label (an integer check)
    neg = dz < 0
    assert (neg.sum(axis=1) == 1).all()
    np.testing.assert_array_equal(np.argmax(neg, axis=1), y)


def test_zero_weights_give_log_classes():
    for C in (10, 1000):
        spec = MlpSpec((12, C), ("none",), "softmax_ce", "f32")
        x = np.random.default_rng(0).standard_normal((9, 12))
        params = [(np.zeros((12, C)), np.zeros(C))]
        y = np.arange(9) % C
        loss, _ = oracle.mlp_forward(spec, x, params, y)
        assert abs(loss - math.log(C)) < 1e-14 * math.log(C)


def test_distinct_biases_expose_label_index():
    C = 10
    spec = MlpSpec((5, C), ("none",), "softmax_ce", "f32")
    b = np.arange(C) / 10.0
    x = np.ones((C, 5))
    y = np.arange(C)[::-1].copy()
    loss, _ = oracle.mlp_forward(spec, x, [(np.zeros((5, C)), b)], y)
    lse = math.log(sum(math.exp(float(np.float32(v))) for v in b))
    ref = np.mean([lse - float(np.float32(b[c])) for c in y])
    assert abs(loss - ref) < 1e-13


def test_shift_invariance():
    rng = np.random.default_rng(6)
    z = rng.standard_normal((8, 7))
    y = rng.integers(0, 7, 8)
    l1, d1 = oracle.softmax_xent(z, y)
    l2, d2 = oracle.softmax_xent(z + rng.standard_normal((8, 1)) * 50, y)
    assert abs(l1 - l2) < 1e-12
    np.testing.assert_allclose(d1, d2, atol=1e-15)


# --------------------------------------------------------------------------
# algebra simplification and linear-algebra fusion identities (§3.1.2)
# --------------------------------------------------------------------------
def test_power_two_simplifies_to_product():
    rng = np.random.default_rng(8)
    z = rng.standard_normal((6, 5)); b = rng.standard_normal(5); xs = rng.standard_normal((6, 5))
    r0 = oracle.chain8(z, b, xs, simplified=False)
    r1 = oracle.chain8(z, b, xs, simplified=True)
    assert abs(r0[0] - r1[0]) <= 1e-15 * abs(r0[0])
    for a0, a1 in zip(r0[1:], r1[1:]):
        np.testing.assert_allclose(a0, a1, rtol=1e-14, atol=1e-18)
    from oracle.mlp import _chain_grad_fn
    assert count_ops(_chain_grad_fn(6, 5, True), "power") == 0
    assert count_ops(_chain_grad_fn(6, 5, False), "power") > 0


def test_power_zero_simplifies_to_one():
    f = Function("p0")
    a = f.arg((3, 4))
    f.ret(f.reduce("add", f.mul(f.power(a, 0.0), a), None))
    x = np.random.default_rng(9).standard_normal((3, 4))
    x[0, 0] = 0.0
    for fn in (f, simplify_algebra(f)):
        val, = evaluate(fn, [x])
        grad, = evaluate(differentiate(fn, [0]), [x])
        assert abs(val - x.sum()) < 1e-14
        np.testing.assert_array_equal(grad, np.ones_like(x))


def test_linear_algebra_fusion_padded_identity():
    """[X 1].[W; b] = X.W + b, and [X 1]^T.dZ = [dW; db]."""
    rng = np.random.default_rng(10)
    X = rng.standard_normal((7, 5)); W = rng.standard_normal((5, 3)); b = rng.standard_normal((1, 3))
    Xp = np.hstack([X, np.ones((7, 1))]); Wp = np.vstack([W, b])
    f = Function("plain"); xa, wa, ba = f.arg((7, 5)), f.arg((5, 3)), f.arg((1, 3))
    f.ret(f.reduce("add", f.tanh(f.add(f.dot(xa, wa), ba)), None))
    fp = Function("padded"); xpa, wpa = fp.arg((7, 6)), fp.arg((6, 3))
    fp.ret(fp.reduce("add", fp.tanh(fp.dot(xpa, wpa)), None))
    v0, = evaluate(f, [X, W, b]); v1, = evaluate(fp, [Xp, Wp])
    assert abs(v0 - v1) < 1e-12
    dW, db = evaluate(differentiate(f, [1, 2]), [X, W, b])
    dWp, = evaluate(differentiate(fp, [1]), [Xp, Wp])
    np.testing.assert_allclose(dWp, np.vstack([dW, db]), rtol=1e-12, atol=1e-14)


# --------------------------------------------------------------------------
# batch linearity (justifies reduced-batch and repeated-row parity cases)
# --------------------------------------------------------------------------
def test_batch_linearity_and_repeated_rows():
    wl = workloads.scaled(workloads.WORKLOADS["c2"], 16, batch=32)
    x, params, y = workloads.make_inputs(wl, bias_scale=0.05)
    spec = MlpSpec(wl.widths, wl.acts, wl.loss, "f32")
    l, g, _ = oracle.mlp_gradient(spec, x, params, y)
    l1, g1, _ = oracle.mlp_gradient(spec, x[:16], params, y[:16])
    l2, g2, _ = oracle.mlp_gradient(spec, x[16:], params, y[16:])
    assert abs(l - (l1 + l2) / 2) < 1e-13
    for (a, b), (a1, b1), (a2, b2) in zip(g, g1, g2):
        np.testing.assert_allclose(a, (a1 + a2) / 2, rtol=1e-11, atol=1e-16)
        np.testing.assert_allclose(b, (b1 + b2) / 2, rtol=1e-11, atol=1e-16)
    xr, yr, _ = workloads.repeat_rows(x, y, 128)
    lr_, gr, _ = oracle.mlp_gradient(spec, xr, params, yr)
    assert abs(lr_ - l) < 1e-13
    for (a, b), (ar, br) in zip(g, gr):
        np.testing.assert_allclose(ar, a, rtol=1e-11, atol=1e-16)
        np.testing.assert_allclose(br, b, rtol=1e-11, atol=1e-16)


# --------------------------------------------------------------------------
# an independent library autograd (test only): PyTorch float64 on the CPU
# --------------------------------------------------------------------------
def _torch_mlp(widths, acts, x, params, y, loss_kind):
    import torch
    xt = torch.tensor(np.asarray(x, np.float64), requires_grad=True)
    ps = [(torch.tensor(np.asarray(W, np.float64), requires_grad=True),
           torch.tensor(np.asarray(b, np.float64), requires_grad=True)) for W, b in params]
    h = xt
    for (W, b), a in zip(ps, acts):
        h = h @ W + b
        h = {"none": lambda t: t, "sigmoid": torch.sigmoid, "tanh": torch.tanh,
             "relu": torch.relu}[a](h)
    assert loss_kind == "softmax_ce"
    loss = torch.nn.functional.cross_entropy(h, torch.tensor(np.asarray(y, np.int64)))
    out = h
    loss.backward()
    return (float(loss.detach()), [(W.grad.numpy(), b.grad.numpy()) for W, b in ps],
            xt.grad.numpy(), out.detach().numpy())


@pytest.mark.parametrize("name,div", [("c1", 1), ("c2", 16), ("c3", 32), ("c5", 128)])
def test_against_torch_float64_autograd(name, div):
    wl = workloads.scaled(workloads.WORKLOADS[name], div, batch=24)
    x, params, y = workloads.make_inputs(wl, bias_scale=0.1)
    spec = MlpSpec(wl.widths, wl.acts, wl.loss, "f32")
    loss, grads, dx = oracle.mlp_gradient(spec, x, params, y, wrt_x=True)
    tl, tg, tdx, tout = _torch_mlp(wl.widths, wl.acts, x, params, y, wl.loss)
    _, out = oracle.mlp_forward(spec, x, params, y)
    assert abs(loss - tl) < 1e-12 * abs(tl)
    np.testing.assert_allclose(out, tout, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(dx, tdx, rtol=1e-9, atol=1e-15)
    for (a, b), (ta, tb) in zip(grads, tg):
        np.testing.assert_allclose(a, ta, rtol=1e-9, atol=1e-15)
        np.testing.assert_allclose(b, tb, rtol=1e-9, atol=1e-15)


def test_chain8_against_torch_float64_autograd():
    import torch
    rng = np.random.default_rng(12)
    # float32-representable inputs: the oracle's entry takes float32 storage values
    x = (rng.standard_normal((9, 16)) / 4).astype(np.float32).astype(np.float64)
    W = (rng.standard_normal((16, 16)) / 4).astype(np.float32).astype(np.float64)
    b = (rng.standard_normal(16) * 0.1).astype(np.float32).astype(np.float64)
    spec = MlpSpec((16, 16), ("none",), "chain8", "f32")
    loss, grads, dx = oracle.mlp_gradient(spec, x, [(W, b)], wrt_x=True)
    xt = torch.tensor(x, requires_grad=True); Wt = torch.tensor(W, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    e = torch.sigmoid(0.5 * torch.tanh(xt @ Wt + bt) + 1.0) * xt
    tl = (e * e).mean(); tl.backward()
    assert abs(loss - tl.item()) < 1e-13 * tl.item()
    np.testing.assert_allclose(grads[0][0], Wt.grad.numpy(), rtol=1e-10, atol=1e-18)
    np.testing.assert_allclose(grads[0][1], bt.grad.numpy(), rtol=1e-10, atol=1e-18)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-18)


def test_chain8_closed_form_adjoint():
    """Hand-derived adjoint of the chain: with L = mean(e^2), e = s x_skip,
    s = sigmoid(0.5 tanh(z + b) + 1): dL/de = 2e/(BN), dL/dx_skip = dL/de * s,
    dL/dz = dL/de * x_skip * s(1-s) * 0.5 * sech^2(z + b)."""
    rng = np.random.default_rng(13)
    z = rng.standard_normal((5, 7)); b = rng.standard_normal(7); xs = rng.standard_normal((5, 7))
    loss, dz, db, dxs, e = oracle.chain8(z, b, xs)
    s = 1 / (1 + np.exp(-(0.5 * np.tanh(z + b) + 1)))
    de = 2 * s * xs / 35
    np.testing.assert_allclose(e, s * xs, rtol=1e-14)
    assert abs(loss - np.mean((s * xs) ** 2)) < 1e-15
    np.testing.assert_allclose(dxs, de * s, rtol=1e-13)
    dz_ref = de * xs * s * (1 - s) * 0.5 / np.cosh(z + b) ** 2
    np.testing.assert_allclose(dz, dz_ref, rtol=1e-12)
    np.testing.assert_allclose(db, dz_ref.sum(axis=0), rtol=1e-12)


# --------------------------------------------------------------------------
# planted mistakes must be caught by the finite-difference check
# --------------------------------------------------------------------------
def _mutants(g: Function):
    """Copies of a gradient function, each with one plausible mistake planted."""
    n_fwd_guess = len(g.instrs)
    out = []
    # (1) flip the first subtraction emitted after the forward part into an addition
    #     (a wrong sign, e.g. 1 + t^2 instead of 1 - t^2)
    # (2) drop one accumulated contribution (a dropped term)
    # (3) swap the operands of one dot product in the adjoint (a transposed operand)
    for kind in ("flip_sub", "drop_term", "swap_dot"):
        m = Function(g.name + "_" + kind)
        m.instrs = [Instr(i.op, i.args, i.shape, i.dtype, dict(i.attrs)) for i in g.instrs]
        m.arg_ids = list(g.arg_ids)
        m.returns = list(g.returns)
        done = False
        for k in range(n_fwd_guess - 1, -1, -1):
            ins = m.instrs[k]
            if kind == "flip_sub" and ins.op == "sub" and ins.shape != () and \
                    m.instrs[ins.args[0]].op == "const":
                ins.op = "add"; done = True; break
            if kind == "drop_term" and ins.op == "add" and \
                    m.instrs[ins.args[0]].shape == m.instrs[ins.args[1]].shape and \
                    m.instrs[ins.args[0]].op in ("dot", "mul", "select", "div"):
                # keep only the first operand: an identity broadcast of it
                m.instrs[k] = Instr("broadcast", (ins.args[0],), ins.shape, ins.dtype)
                done = True; break
            if kind == "swap_dot" and ins.op == "dot":
                a0, a1 = ins.args
                if m.instrs[a0].shape == m.instrs[a1].shape and m.instrs[a0].shape[0] == m.instrs[a0].shape[1]:
                    ins.args = (a1, a0); done = True; break
        if done:
            out.append((kind, m))
    return out


def test_planted_mistakes_are_caught():
    rng = np.random.default_rng(14)
    spec = MlpSpec((6, 6, 6, 4), ("tanh", "sigmoid", "none"), "softmax_ce", "f32")
    x = rng.standard_normal((6, 6))
    params = [(rng.standard_normal((6, 6)) * 0.7, rng.standard_normal(6) * 0.1),
              (rng.standard_normal((6, 6)) * 0.7, rng.standard_normal(6) * 0.1),
              (rng.standard_normal((6, 4)) * 0.7, rng.standard_normal(4) * 0.1)]
    y = rng.integers(0, 4, 6)
    f = build_mlp_loss(spec, 6)
    g = build_mlp_gradient(spec, 6, True)
    args = _f64_args(spec, x, params, y)
    wrt = list(range(7))
    assert _fd_check(f, g, args, wrt) < 1.0
    mutants = _mutants(g)
    assert {k for k, _ in mutants} == {"flip_sub", "drop_term", "swap_dot"}
    for kind, m in mutants:
        assert _fd_check(f, adce(m), args, wrt) > 10.0, kind


# --------------------------------------------------------------------------
# bf16 rounding and SGD
# --------------------------------------------------------------------------
def test_bf16_rounding_matches_library_conversion():
    import torch
    rng = np.random.default_rng(15)
    v = np.concatenate([
        rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-40, 38, 100000),
        np.array([0.0, -0.0, np.inf, -np.inf, 3.4028235e38, 1e-45, -1e-45, 1.0, 1.00390625,
                  1.01171875, 1.0078125, 65504.0], np.float32),
        # exact ties between two bf16 values: low 16 bits == 0x8000
        (rng.integers(0, 2**31, 1000).astype(np.uint32) & np.uint32(0xFFFF0000) |
         np.uint32(0x8000)).view(np.float32),
    ]).astype(np.float32)
    v = v[np.isfinite(v) | np.isinf(v)]
    ours = oracle.round_to_bf16(v)
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)
    assert np.isnan(oracle.round_to_bf16(np.array([np.nan], np.float32))).all()


def test_sgd_descends_the_oracle_loss():
    """A small step along -gradient lowers the loss (ties SGD to the gradient)."""
    spec, x, params, y = _c1_setup()
    loss, grads, _ = oracle.mlp_gradient(spec, x, params, y)
    new = [(oracle.sgd_f32(W, dW, 0.01), oracle.sgd_f32(b, db, 0.01))
           for (W, b), (dW, db) in zip(params, grads)]
    loss2, _ = oracle.mlp_forward(spec, x, new, y)
    gn = sum(float((dW ** 2).sum() + (db ** 2).sum()) for dW, db in grads)
    assert loss2 < loss
    assert abs((loss - loss2) - 0.01 * gn) < 0.05 * 0.01 * gn   # first-order prediction


def test_sgd_f32_is_correctly_rounded():
    rng = np.random.default_rng(16)
    p = rng.standard_normal(10000).astype(np.float32)
    g = rng.standard_normal(10000).astype(np.float32)
    out = oracle.sgd_f32(p, g, 0.01)
    exact = p.astype(np.float64) - float(np.float32(0.01)) * g.astype(np.float64)
    err = np.abs(out.astype(np.float64) - exact)
    ulp = np.spacing(np.abs(out)).astype(np.float64)
    assert (err <= 0.5 * ulp + 1e-45).all()
    m, shadow = oracle.sgd_bf16(p, g, 0.01)
    np.testing.assert_array_equal(m, out)
    np.testing.assert_array_equal(shadow, oracle.round_to_bf16(out))


def test_bf16_storage_quantises_inputs():
    wl = workloads.scaled(workloads.WORKLOADS["c3"], 64, batch=8)
    x, params, y = workloads.make_inputs(wl)
    spec = MlpSpec(wl.widths, wl.acts, wl.loss, "bf16", storage_casts=False)
    spec32 = MlpSpec(wl.widths, wl.acts, wl.loss, "f32")
    xq = oracle.round_to_bf16(x)
    pq = [(oracle.round_to_bf16(W), oracle.round_to_bf16(b)) for W, b in params]
    l_bf, _ = oracle.mlp_forward(spec, x, params, y)
    l_q, _ = oracle.mlp_forward(spec32, xq.astype(np.float32), [(W.astype(np.float32), b.astype(np.float32)) for W, b in pq], y)
    assert l_bf == l_q


# --------------------------------------------------------------------------
# dataTypeCast to bf16 (Table 1): value rounding and straight-through adjoint
# --------------------------------------------------------------------------
def test_cast_value_matches_library_rounding():
    import torch
    v = np.random.default_rng(20).standard_normal((7, 9)) * 100
    f = Function("c"); a = f.arg((7, 9)); f.ret(f.cast(a, "bf16"))
    got, = evaluate(f, [v])
    ref = torch.from_numpy(v.astype(np.float32)).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(got, ref)


def test_cast_adjoint_passes_straight_through():
    rng = np.random.default_rng(21)
    a0 = rng.standard_normal((4, 5)); w = rng.standard_normal((4, 5))
    f = Function("c"); a = f.arg((4, 5)); wa = f.arg((4, 5))
    f.ret(f.reduce("add", f.mul(f.cast(a, "bf16"), wa), None))
    da, = evaluate(differentiate(f, [0]), [a0, w])
    np.testing.assert_array_equal(da, w)


def test_casts_vanish_on_bf16_representable_networks():
    """Integer-valued ReLU network: every activation is exact in bf16, so the
    network with storage casts and the one without compute the same values and
    the same gradients, bit for bit."""
    rng = np.random.default_rng(22)
    spec_c = MlpSpec((6, 5, 4, 3), ("relu", "relu", "none"), "softmax_ce", "bf16")
    spec_n = MlpSpec((6, 5, 4, 3), ("relu", "relu", "none"), "softmax_ce", "bf16",
                     storage_casts=False)
    x = rng.integers(-3, 4, (5, 6)).astype(np.float32)
    params = [(rng.integers(-2, 3, (6, 5)).astype(np.float32), rng.integers(-1, 2, 5).astype(np.float32)),
              (rng.integers(-2, 3, (5, 4)).astype(np.float32), rng.integers(-1, 2, 4).astype(np.float32)),
              (rng.integers(-1, 2, (4, 3)).astype(np.float32) / 4, np.zeros(3, np.float32))]
    y = np.array([0, 1, 2, 1, 0])
    lc, gc, dxc = oracle.mlp_gradient(spec_c, x, params, y, wrt_x=True)
    ln, gn, dxn = oracle.mlp_gradient(spec_n, x, params, y, wrt_x=True)
    assert lc == ln
    np.testing.assert_array_equal(dxc, dxn)
    for (a, b), (c, d) in zip(gc, gn):
        np.testing.assert_array_equal(a, c)
        np.testing.assert_array_equal(b, d)


def test_bf16_storage_network_against_torch_straight_through():
    """torch float64 autograd with a straight-through bf16 rounding of each
    hidden activation (h + (round(h) - h).detach()) computes the same function."""
    import torch
    wl = workloads.scaled(workloads.WORKLOADS["c5"], 64, batch=12)
    x, params, y = workloads.make_inputs(wl, bias_scale=0.1)
    spec = MlpSpec(wl.widths, wl.acts, wl.loss, "bf16")
    loss, grads, dx = oracle.mlp_gradient(spec, x, params, y, wrt_x=True)

    def q(a):
        return torch.from_numpy(oracle.round_to_bf16(np.asarray(a, np.float32)))
    xt = q(x).requires_grad_(True)
    ps = [(q(W).requires_grad_(True), q(b).requires_grad_(True)) for W, b in params]
    h = xt
    for l, (W, b) in enumerate(ps):
        h = h @ W + b
        if l < len(ps) - 1:
            h = torch.relu(h)
            hr = h.detach().float().to(torch.bfloat16).double()
            h = h + (hr - h).detach()
    tl = torch.nn.functional.cross_entropy(h, torch.from_numpy(y.astype(np.int64)))
    tl.backward()
    assert abs(loss - tl.item()) < 1e-12 * abs(loss)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-9, atol=1e-15)
    for (a, b), (W, bb) in zip(grads, ps):
        np.testing.assert_allclose(a, W.grad.numpy(), rtol=1e-9, atol=1e-15)
        np.testing.assert_allclose(b, bb.grad.numpy(), rtol=1e-9, atol=1e-15)


def test_float32_accumulation_mode():
    """accumulate="f32" changes only the accumulation precision of the forward dots:
    on a float32 network (no casts) the two evaluations agree to float32 accuracy,
    and the float32 dot equals a float32 library product."""
    from dataclasses import replace
    wl = workloads.scaled(workloads.WORKLOADS["c2"], 8, batch=16)
    x, params, y = workloads.make_inputs(wl, bias_scale=0.1)
    s64 = MlpSpec(wl.widths, wl.acts, wl.loss, "f32")
    l64, g64, _ = oracle.mlp_gradient(s64, x, params, y)
    l32, g32, _ = oracle.mlp_gradient(replace(s64, accumulate="f32"), x, params, y)
    assert abs(l64 - l32) < 1e-5 * l64
    for (a, b), (c, d) in zip(g64, g32):
        assert np.linalg.norm(a - c) <= 1e-5 * np.linalg.norm(a)
    f = Function("d"); A = f.arg((5, 7)); B = f.arg((7, 3)); f.ret(f.dot(A, B, "f32"))
    rng = np.random.default_rng(23)
    a, b = rng.standard_normal((5, 7)), rng.standard_normal((7, 3))
    got, = evaluate(f, [a, b])
    np.testing.assert_array_equal(got, (a.astype(np.float32) @ b.astype(np.float32)).astype(np.float64))


# ---------------------------------------------------------------------------
# The seedable gradient of the logits (Fig. 3's seedable declaration)
# ---------------------------------------------------------------------------
def _vjp_case(seed=31):
    spec = MlpSpec((7, 6, 5, 4), ("tanh", "sigmoid", "none"))
    r = np.random.default_rng(seed)
    x = r.standard_normal((3, 7))
    params = [(r.standard_normal((spec.widths[l], spec.widths[l + 1])) * 0.6,
               r.standard_normal(spec.widths[l + 1]) * 0.3) for l in range(3)]
    return spec, x, params, r


def test_vjp_adjoint_identity_by_finite_differences():
    """<seed, J v> = <VJP(seed), v> for a random direction v over x and every
    parameter, J v taken by central finite differences of the logits."""
    spec, x, params, r = _vjp_case()
    S = r.standard_normal((3, 4))
    vx = r.standard_normal(x.shape)
    vp = [(r.standard_normal(W.shape), r.standard_normal(b.shape)) for W, b in params]
    h = 1e-5

    # float64 arguments straight into the IR functions (no storage rounding)
    f = build_mlp_logits(spec, 3)
    g = build_mlp_vjp(spec, 3, True)

    def flat(t):
        a = [x + t * vx]
        for (W, b), (dW, db) in zip(params, vp):
            a += [W + t * dW, (b + t * db).reshape(1, -1)]
        return a

    jv = (evaluate(f, flat(h))[0] - evaluate(f, flat(-h))[0]) / (2 * h)
    lhs = float(np.sum(S * jv))
    res = evaluate(g, flat(0.0) + [S])
    dx, grads = res[0], [(res[1 + 2 * l], res[2 + 2 * l].reshape(-1)) for l in range(3)]
    rhs = float(np.sum(dx * vx)) + sum(float(np.sum(gW * dW) + np.sum(gb * db))
                                       for (gW, gb), (dW, db) in zip(grads, vp))
    assert abs(lhs - rhs) <= 1e-7 * max(1.0, abs(lhs)), (lhs, rhs)


def test_vjp_is_linear_in_the_seed():
    spec, x, params, r = _vjp_case(32)
    S1, S2 = r.standard_normal((3, 4)), r.standard_normal((3, 4))
    g1, d1 = oracle.mlp_vjp(spec, x, params, S1, wrt_x=True)
    g2, d2 = oracle.mlp_vjp(spec, x, params, S2, wrt_x=True)
    g3, d3 = oracle.mlp_vjp(spec, x, params, 2.0 * S1 - 0.5 * S2, wrt_x=True)
    np.testing.assert_allclose(d3, 2.0 * d1 - 0.5 * d2, rtol=1e-12, atol=1e-14)
    for (a1, b1), (a2, b2), (a3, b3) in zip(g1, g2, g3):
        np.testing.assert_allclose(a3, 2.0 * a1 - 0.5 * a2, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(b3, 2.0 * b1 - 0.5 * b2, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_vjp_with_the_loss_adjoint_is_the_loss_gradient(dtype):
    """Chain rule: the seed (softmax(z) - onehot(y)) / B, written from its closed
    form, turns the logits' gradient into the loss gradient."""
    spec = MlpSpec((8, 6, 5), ("relu", "none"), dtype=dtype)
    r = np.random.default_rng(33)
    x = r.standard_normal((4, 8)).astype(np.float32)
    params = [(r.standard_normal((8, 6)).astype(np.float32), r.uniform(-.3, .3, 6).astype(np.float32)),
              (r.standard_normal((6, 5)).astype(np.float32), r.uniform(-.3, .3, 5).astype(np.float32))]
    y = np.array([0, 4, 2, 2])
    _, z = oracle.mlp_forward(spec, x, params, y)
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    seed = (p - np.eye(5)[y]) / 4
    gv, _ = oracle.mlp_vjp(spec, x, params, seed)
    _, gl, _ = oracle.mlp_gradient(spec, x, params, y)
    for (a, b), (c, d) in zip(gv, gl):
        np.testing.assert_allclose(a, c, rtol=1e-10, atol=1e-13)
        np.testing.assert_allclose(b, d, rtol=1e-10, atol=1e-13)


# --------------------------------------------------------------------------
# The recurrent cell (§3.1.2): oracle.rnn_forward / oracle.rnn_vjp
# --------------------------------------------------------------------------
def _rnn_case(T, Kx, H, B, seed=3):
    from dataclasses import replace
    wl = replace(workloads.RNN_WORKLOADS["r1"], steps=T, in_width=Kx, hidden=H, dtype="f32")
    return workloads.make_rnn_inputs(wl, batch=B, seed=seed)


@pytest.mark.parametrize("act", ["tanh", "relu"])
def test_rnn_against_torch_rnn(act):
    """torch.nn.RNN (float64, CPU) computes h_t = act(x_t W_ih^T + b_ih + h_{t-1}
    W_hh^T + b_hh): an independent implementation of the same recurrence and of
    its gradient (library autograd)."""
    import torch
    T, Kx, H, B = 5, 7, 6, 4
    xs, h0, W, U, b, dhs = _rnn_case(T, Kx, H, B)
    spec = oracle.RnnSpec(T, Kx, H, act, "f32")
    hs = oracle.rnn_forward(spec, xs, h0, W, U, b)
    dW, dU, db, dxs, dh0 = oracle.rnn_vjp(spec, xs, h0, W, U, b, dhs, wrt_x=True, wrt_h0=True)
    f64 = lambda a: torch.from_numpy(np.asarray(a, np.float64))  # noqa: E731
    rnn = torch.nn.RNN(Kx, H, nonlinearity=act, bias=True).double()
    with torch.no_grad():
        rnn.weight_ih_l0.copy_(f64(W).T)
        rnn.weight_hh_l0.copy_(f64(U).T)
        rnn.bias_ih_l0.copy_(f64(b))
        rnn.bias_hh_l0.zero_()
    x = f64(xs).requires_grad_()
    h = f64(h0)[None].clone().requires_grad_()
    out, _ = rnn(x, h)
    np.testing.assert_allclose(hs[1:], out.detach().numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_array_equal(hs[0], np.asarray(h0, np.float64))
    (out * f64(dhs)).sum().backward()
    np.testing.assert_allclose(dW, rnn.weight_ih_l0.grad.numpy().T, rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(dU, rnn.weight_hh_l0.grad.numpy().T, rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(db, rnn.bias_ih_l0.grad.numpy(), rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(dxs, x.grad.numpy(), rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(dh0, h.grad.numpy()[0], rtol=1e-10, atol=1e-13)


def test_rnn_linear_scalar_closed_form():
    """act = none, Kx = H = 1: h_T = u^T h0 + sum_t u^(T-1-t) (x_t w + b), and with
    the seed on h_T alone dL/du = T u^(T-1) h0 + sum_t (T-1-t) u^(T-2-t) c_t,
    dL/dw = sum_t u^(T-1-t) x_t, dL/db = sum_t u^(T-1-t), dL/dh0 = u^T."""
    T, B = 6, 3
    rng = np.random.default_rng(11)
    xs = rng.standard_normal((T, B, 1)).astype(np.float32)
    h0 = rng.standard_normal((B, 1)).astype(np.float32)
    w, u, bb = np.float32(0.7), np.float32(-0.8), np.float32(0.3)
    dhs = np.zeros((T, B, 1), np.float32)
    dhs[-1] = 1.0
    spec = oracle.RnnSpec(T, 1, 1, "none", "f32")
    W, U, b = np.array([[w]]), np.array([[u]]), np.array([bb])
    hs = oracle.rnn_forward(spec, xs, h0, W, U, b)
    u64, w64, b64 = float(u), float(w), float(bb)
    x64, h64 = xs[:, :, 0].astype(np.float64), h0[:, 0].astype(np.float64)
    c = x64 * w64 + b64                                               # c_t [T, B]
    hT = u64 ** T * h64 + sum(u64 ** (T - 1 - t) * c[t] for t in range(T))
    np.testing.assert_allclose(hs[-1][:, 0], hT, rtol=1e-13)
    dW, dU, db, dxs, dh0 = oracle.rnn_vjp(spec, xs, h0, W, U, b, dhs, wrt_x=True, wrt_h0=True)
    du = np.sum(T * u64 ** (T - 1) * h64 +
                sum((T - 1 - t) * u64 ** (T - 2 - t) * c[t] for t in range(T - 1)))
    dw = np.sum(sum(u64 ** (T - 1 - t) * x64[t] for t in range(T)))
    np.testing.assert_allclose(dU[0, 0], du, rtol=1e-12)
    np.testing.assert_allclose(dW[0, 0], dw, rtol=1e-12)
    np.testing.assert_allclose(db[0], B * sum(u64 ** (T - 1 - t) for t in range(T)), rtol=1e-12)
    np.testing.assert_allclose(dh0[:, 0], np.full(B, u64 ** T), rtol=1e-12)
    np.testing.assert_allclose(dxs[:, :, 0], np.array([[w64 * u64 ** (T - 1 - t)] * B
                                                       for t in range(T)]), rtol=1e-12)


def test_rnn_sigmoid_single_step_and_adjoint_identity():
    """Sigmoid cells (not in torch.nn.RNN): one step from h0 = 0 is the dense
    layer sigmoid(x W + b) (library sigmoid), and the VJP satisfies the adjoint
    identity <vjp(s), v> = d/de <s, h(theta + e v)> against central differences
    of the forward."""
    import torch
    T, Kx, H, B = 4, 5, 6, 3
    xs, h0, W, U, b, dhs = _rnn_case(T, Kx, H, B, seed=9)
    spec1 = oracle.RnnSpec(1, Kx, H, "sigmoid", "f32")
    hs1 = oracle.rnn_forward(spec1, xs[:1], np.zeros_like(h0), W, U, b)
    ref = torch.sigmoid(torch.from_numpy(xs[0].astype(np.float64)) @
                        torch.from_numpy(W.astype(np.float64)) + torch.from_numpy(b.astype(np.float64)))
    np.testing.assert_allclose(hs1[1], ref.numpy(), rtol=1e-13)

    spec = oracle.RnnSpec(T, Kx, H, "sigmoid", "f32")
    dW, dU, db, dxs, dh0 = oracle.rnn_vjp(spec, xs, h0, W, U, b, dhs, wrt_x=True, wrt_h0=True)
    rng = np.random.default_rng(4)
    # float64 perturbations: evaluate the IR directly on float64 arguments
    f = oracle.rnn.build_rnn(spec, B)
    base = [np.asarray(xs[t], np.float64) for t in range(T)] + \
        [np.asarray(a, np.float64) for a in (h0, W, U, np.reshape(b, (1, -1)))]
    vs = [rng.standard_normal(a.shape) for a in base]

    def L(e):
        outs = evaluate(f, [a + e * v for a, v in zip(base, vs)])
        return sum(float(np.sum(np.asarray(dhs[t], np.float64) * outs[t])) for t in range(T))

    eps = 1e-5
    fd = (L(eps) - L(-eps)) / (2 * eps)
    grads = [dxs[t] for t in range(T)] + [dh0, dW, dU, db.reshape(1, -1)]
    ad = sum(float(np.sum(g * v)) for g, v in zip(grads, vs))
    assert abs(fd - ad) <= 1e-7 * max(1.0, abs(ad)), (fd, ad)


def test_rnn_bf16_states_are_stored_as_bf16():
    """With bf16 storage every state the oracle returns is a bf16 number, and
    without the casts it is the exact function of the rounded inputs."""
    T, Kx, H, B = 3, 8, 8, 4
    xs, h0, W, U, b, dhs = _rnn_case(T, Kx, H, B)
    hs = oracle.rnn_forward(oracle.RnnSpec(T, Kx, H, "tanh", "bf16"), xs, h0, W, U, b)
    np.testing.assert_array_equal(oracle.round_to_bf16(hs.astype(np.float32)), hs)
    exact = oracle.rnn_forward(oracle.RnnSpec(T, Kx, H, "tanh", "bf16", storage_casts=False),
                               xs, h0, W, U, b)
    assert not np.array_equal(exact, hs)
    assert np.max(np.abs(exact - hs)) < 0.05


# --------------------------------------------------------------------------
# Matrix multiplication reordering (§3.1.2): oracle.chain_order / chain_product
# --------------------------------------------------------------------------
def _brute_force_chain(d, i, j):
    """Minimal multiply-add count of A_i..A_j over every parenthesisation."""
    if i == j:
        return 0
    return min(_brute_force_chain(d, i, k) + _brute_force_chain(d, k + 1, j) + d[i] * d[k + 1] * d[j + 1]
               for k in range(i, j))


def test_chain_order_textbook_example():
    """The textbook's six-matrix example (tests/golden/matrix_chain_textbook.json)."""
    g = json.load(open(os.path.join(GOLDEN, "matrix_chain_textbook.json")))
    cost, split = oracle.chain_order(g["dims"])
    assert cost == g["min_cost"]
    assert oracle.parenthesisation(split) == g["order"]
    sub, _ = oracle.chain_order(g["dims"][1:6])    # A1..A4 of the example's 0-based names
    assert sub == g["cost_2_5"]


@pytest.mark.parametrize("seed", range(12))
def test_chain_order_against_brute_force(seed):
    """The dynamic programme's cost is the minimum over all parenthesisations
    (enumerated), and the order it returns achieves that cost."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 8))
    d = [int(v) for v in rng.integers(1, 60, size=n + 1)]
    cost, split = oracle.chain_order(d)
    assert cost == _brute_force_chain(d, 0, n - 1)

    def order_cost(i, j):
        if i == j:
            return 0
        k = split[i][j]
        return order_cost(i, k) + order_cost(k + 1, j) + d[i] * d[k + 1] * d[j + 1]

    assert order_cost(0, n - 1) == cost


def test_chain_products_agree_with_library_and_every_order():
    """The left-to-right product equals numpy's multi_dot (a library routine
    that picks its own order), and the product in the optimal order equals it
    too (associativity), in float64."""
    rng = np.random.default_rng(3)
    d = [7, 33, 4, 19, 2, 25]
    mats = [rng.standard_normal((d[i], d[i + 1])).astype(np.float32) for i in range(len(d) - 1)]
    ref = np.linalg.multi_dot([m.astype(np.float64) for m in mats])
    got = oracle.chain_product(mats)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    _, split = oracle.chain_order(d)
    np.testing.assert_allclose(oracle.chain_product_in_order(mats, split), ref, rtol=1e-12, atol=1e-12)
    single = oracle.chain_product(mats[:1])
    np.testing.assert_array_equal(single, mats[0].astype(np.float64))
