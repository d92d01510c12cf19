"""The deep bf16 network (4096 -> 8 x 4096 relu -> 1000, softmax cross-entropy,
batch 16384) checked one product at a time, at its full batch and in the launch
configuration the benchmark times (the planner's own choices, nothing forced).

Why per product. With bf16 storage every hidden output and adjoint is rounded
before the next product reads it, so the end-to-end gradient of eight ReLU
layers depends on the accumulation order of every product before it (a
rounding boundary crossed in layer 1 flips ReLU masks further on; see the
oracle's note on order sensitivity). Each product on its own is well
conditioned: here the oracle receives exactly the bf16 operands the GPU used
-- the inputs and parameters, and the layer outputs and adjoints the gradient
call kept in its workspace (read through ``dlvm_workspace_tensor``) -- so what
is left is the GPU's float32 accumulation and the final rounding of its
output. Every product is then held to the stated bounds: 2e-2 relative for
bf16 outputs and 1e-5 for float32 outputs of bf16 operands, over the tensor
and, per row, 2e-2 and 1e-4 (a single wrong row fails).

Rows of a product are independent, so the forward and input-adjoint products
are checked on a seeded sample of rows; each column of a product w.r.t. the
weights is a full contraction over the 16384 rows, so those are checked on a
seeded sample of columns (the bias gradients on every column). Samples include
the first and last rows and columns and the 256-element tile edges. The loss
adjoint is checked on every row, with the labels bit for bit.
"""
import numpy as np
import pytest

import oracle
import paper_1711_03016_amd as dl
import workloads
from helpers import assert_close, device, quant, to_dev

pytestmark = pytest.mark.gpu

WL = workloads.WORKLOADS["c5"]
L = WL.n_layers          # 9: eight hidden layers and the output layer
B = WL.batch             # 16384
BF16_TOL = 2e-2          # bf16 outputs (tensor and per row)
F32_TOL, F32_ROW_TOL = 1e-5, 1e-4   # float32 outputs of bf16 operands


def _sample(n, k, seed):
    """k seeded indices of range(n) plus the edges 0, 255, 256, n - 1."""
    rng = np.random.default_rng([1711, 3016, seed])
    idx = set(int(v) for v in rng.choice(n, size=min(k, n), replace=False))
    idx |= {0, min(255, n - 1), min(256, n - 1), n - 1}
    return np.array(sorted(idx))


def _f64(t):
    import torch
    return t.to(torch.float64).numpy()


@pytest.fixture(scope="module")
def c5():
    """One gradient call of the full network; everything it kept, on the host."""
    import torch
    x, params, y = workloads.make_inputs(WL, bias_scale=0.05)
    dev = device()
    m = dl.Model(WL.widths, WL.acts, WL.dtype, WL.loss, False, B)
    plan = [e["name"] for e in m.plan(B)]
    print("c5 plan:", plan, flush=True)
    P = m.pack(params, dev, torch.bfloat16)
    yd = torch.from_numpy(y).to(dev)
    ws = torch.empty(m.workspace_bytes(B), dtype=torch.uint8, device=dev)
    loss = torch.empty(1, device=dev)
    dP = torch.full((m.param_count(),), float("nan"), device=dev)
    m.gradient(P, to_dev(x, "bf16"), yd, B, loss, dP, None, ws)
    torch.cuda.synchronize()
    status = m.check(ws)
    out = {
        "x": x, "y": y, "status": status, "loss": loss.item(),
        "W": [quant(W, "bf16") for W, _ in params],
        "b": [quant(b, "bf16") for _, b in params],
        "H": {l: m.workspace_tensor(ws, B, dl.WS_HIDDEN, l).cpu() for l in range(1, L)},
        "dZ": {l: m.workspace_tensor(ws, B, dl.WS_ADJOINT, l).cpu() for l in range(1, L + 1)},
        "logits": m.workspace_tensor(ws, B, dl.WS_LOGITS).cpu(),
        "grads": [(gW.cpu(), gb.cpu()) for gW, gb in m.unpack(dP)],
        "nan": bool(torch.isnan(dP).any().item()),
    }
    del P, ws, dP
    torch.cuda.empty_cache()
    return out


def _layer_input(c5, l, rows=None):
    """H_{l-1} (H_0 = x) as the GPU read it, float64."""
    if l == 1:
        x = c5["x"] if rows is None else c5["x"][rows]
        return quant(x, "bf16")
    h = c5["H"][l - 1]
    return _f64(h if rows is None else h[rows])


def test_call_status(c5):
    assert c5["status"] == dl.OK
    assert not c5["nan"]
    for l in range(1, L):
        assert c5["H"][l].shape == (B, 4096)
    assert c5["dZ"][L].shape == (B, 1000) and c5["logits"].shape == (B, 1000)


@pytest.mark.parametrize("l", range(1, L))
def test_hidden_forward_product(c5, l):
    """H_l = relu(H_{l-1} . W_l + b_l) (16384 x 4096 x 4096, bf16 out) on sampled rows."""
    R = _sample(B, 508, l)
    ref = oracle.dense_forward(_layer_input(c5, l, R), c5["W"][l - 1], c5["b"][l - 1], "relu")
    got = _f64(c5["H"][l][R])
    assert_close(got, ref, BF16_TOL, ("H", l))


def test_output_layer_product(c5):
    """logits = H_8 . W_9 + b_9 (16384 x 1000 x 4096, float32 out) on sampled rows."""
    R = _sample(B, 1020, 100)
    ref = oracle.dense_forward(_layer_input(c5, L, R), c5["W"][L - 1], c5["b"][L - 1], "none")
    got = c5["logits"][R].numpy().astype(np.float64)
    assert_close(got, ref, F32_TOL, "logits", row_tol=F32_ROW_TOL)


def test_loss_and_its_adjoint_on_every_row(c5):
    """Softmax cross-entropy of the GPU's own logits: the loss, the adjoint
    (softmax - onehot) / B in bf16 on all 16384 rows, and the labels exactly:
    each row's one negative entry sits at its label."""
    z = c5["logits"].numpy().astype(np.float64)
    y = c5["y"]
    rl, rdz = oracle.softmax_xent(z, y)
    assert abs(c5["loss"] - rl) <= 1e-5 * abs(rl), (c5["loss"], rl)
    got = _f64(c5["dZ"][L])
    assert_close(got, rdz, BF16_TOL, "dZ_L")
    neg = got < 0
    assert (neg.sum(axis=1) == 1).all()
    np.testing.assert_array_equal(np.argmax(neg, axis=1), y)


@pytest.mark.parametrize("l", range(L, 1, -1))
def test_input_adjoint_product(c5, l):
    """dZ_{l-1} = (dZ_l . W_l^T) * relu'(H_{l-1}) (16384 x 4096 x N_l, bf16 out)
    on sampled rows; relu' is taken from the saved output, as the kernel does."""
    R = _sample(B, 508, 200 + l)
    u = _layer_input(c5, l, R)          # relu'(u) = [u > 0] = [H_{l-1} > 0]
    ref = oracle.dense_vjp_input(u, c5["W"][l - 1], _f64(c5["dZ"][l][R]), "relu")
    got = _f64(c5["dZ"][l - 1][R])
    assert_close(got, ref, BF16_TOL, ("dZ", l - 1))


@pytest.mark.parametrize("l", range(1, L + 1))
def test_weight_adjoint_product(c5, l):
    """dW_l = H_{l-1}^T . dZ_l (4096 x N_l x 16384, float32) on sampled columns,
    and db_l = column sums of dZ_l on every column."""
    N = WL.widths[l]
    S = _sample(N, 124, 300 + l)
    inp = _layer_input(c5, l)
    dz = c5["dZ"][l]
    rdW, _ = oracle.dense_vjp_params(inp, _f64(dz[:, S]))
    gW, gb = c5["grads"][l - 1]
    # one row per sampled column: a whole contraction over the batch
    assert_close(gW[:, S].numpy().T.astype(np.float64), rdW.T, F32_TOL, ("dW", l),
                 row_tol=F32_ROW_TOL)
    _, rdb = oracle.dense_vjp_params(inp[:, :1], _f64(dz[:, :N]))
    assert_close(gb.numpy().astype(np.float64), rdb, F32_TOL, ("db", l), row_tol=F32_ROW_TOL)
