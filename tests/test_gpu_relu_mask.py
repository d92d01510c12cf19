"""Rectifier masks: the forward product of a rectified bf16 layer writes the
derivative's bits (output > 0) in accumulator order and the product wrt the
input of the next layer reads them instead of the saved output (section 3.1.3:
the rectifier's adjoint needs only the sign of its saved output).

The masked path must give bitwise the results of the saved-output path
(DLVM_RELU_MASK=0), on ragged shapes, through the gradient, the seedable
gradient and the checkpointed plan, and agree with the oracle, on both tile
configurations that write masks (10: 256 x 256, 16: 64 x 128).
"""
from dataclasses import replace

import numpy as np
import pytest

import oracle
import paper_1711_03016_amd as dl
import workloads
from helpers import TOL, assert_close, device, rel_l2, to_dev, to_np, torch_dtype

BASE = workloads.WORKLOADS["c3"]


def _wl(widths, batch):
    acts = ("relu",) * (len(widths) - 2) + ("none",)
    return replace(BASE, widths=widths, acts=acts, batch=batch, wrt_x=True)


def _mask_bytes(M, N):
    return max(-(-M // 256) * -(-N // 256) * 8192, -(-M // 64) * -(-N // 128) * 1024)


@pytest.mark.parametrize("masks", ["on", "off"])
def test_workspace_reserves_masks_for_the_deep_network(masks, monkeypatch):
    """At the deep network's shape every hidden output gets a mask (its forward
    and its input-adjoint products run on the 256 x 256 tile unsplit); turning
    the masks off gives the workspace without them."""
    if masks == "off":
        monkeypatch.setenv("DLVM_RELU_MASK", "0")
    wl = workloads.WORKLOADS["c5"]
    m = dl.Model(wl.widths, wl.acts, wl.dtype, wl.loss, False, wl.batch)
    with_masks = m.workspace_bytes(wl.batch)
    monkeypatch.setenv("DLVM_RELU_MASK", "0")
    without = m.workspace_bytes(wl.batch)
    extra = sum(_mask_bytes(wl.batch, w) for w in wl.widths[1:-1])
    assert with_masks - without == (extra if masks == "on" else 0)


@pytest.mark.parametrize("widths,acts,dtype", [
    ((784, 512, 512, 10), ("relu", "relu", "none"), "f32"),         # float32 network
    ((4096, 4096, 4096, 10), ("tanh", "sigmoid", "none"), "bf16"),  # not rectified
    ((784, 2048, 2048, 10), ("relu", "relu", "none"), "bf16"),      # products on 256 x 128 tiles
])
def test_no_masks_where_products_do_not_qualify(widths, acts, dtype, monkeypatch):
    m = dl.Model(widths, acts, dtype, "softmax_ce", False, 4096)
    with_masks = m.workspace_bytes(4096)
    monkeypatch.setenv("DLVM_RELU_MASK", "0")
    assert m.workspace_bytes(4096) == with_masks


def test_operands_beyond_2gib_leave_the_256_tiles(monkeypatch):
    """The 256 x 256 tiles load through buffer descriptors, whose extents are
    32-bit: a product reading an operand of 2 GiB or more is planned on
    another tile (here the 16384 x 4096 bf16 input grows to 2.46 GB at a batch
    of 300000), and then its output gets no rectifier mask."""
    widths, acts = (4096, 4096, 4096, 10), ("relu", "relu", "none")
    m = dl.Model(widths, acts, "bf16", "softmax_ce", False, 300000)
    plan = m.plan(300000)
    for p in plan:
        if p["name"].startswith(("gemm_nn", "gemm_nt", "gemm_tn", "gemm_pair")):
            # bytes of the operands it reads through descriptors: A is M x K or K x M
            big = p["M"] * p["K"] * 2 >= 2 ** 31 or p["N"] * p["K"] * 2 >= 2 ** 31
            if big:
                assert "c10" not in p["name"] and "c13" not in p["name"], p
    assert plan[0]["name"].startswith("gemm_nn") and "c10" not in plan[0]["name"]
    with_masks = m.workspace_bytes(300000)
    monkeypatch.setenv("DLVM_RELU_MASK", "0")
    assert m.workspace_bytes(300000) == with_masks
    # below the limit the same network keeps the 256 x 256 tile and its masks
    monkeypatch.delenv("DLVM_RELU_MASK")
    m2 = dl.Model(widths, acts, "bf16", "softmax_ce", False, 200000)
    assert m2.plan(200000)[0]["name"].endswith("c10")
    masked = m2.workspace_bytes(200000)
    monkeypatch.setenv("DLVM_RELU_MASK", "0")
    assert masked - m2.workspace_bytes(200000) == 2 * _mask_bytes(200000, 4096)


def _gradient(wl, x, params, y, ckpt=1, seed=None):
    import torch
    B = x.shape[0]
    dev = device()
    m = dl.Model(wl.widths, wl.acts, wl.dtype, wl.loss, True, B, checkpoint_every=ckpt)
    P = m.pack(params, dev, torch_dtype(wl.dtype))
    ws = torch.full((m.workspace_bytes(B),), 0xFF, dtype=torch.uint8, device=dev)
    dP = torch.full((m.param_count(),), float("nan"), device=dev)
    dx = torch.empty((B, wl.widths[0]), device=dev)
    loss = torch.zeros(1, device=dev)
    if seed is None:
        yd = torch.from_numpy(np.asarray(y, np.int32)).to(dev)
        m.gradient(P, to_dev(x, wl.dtype), yd, B, loss, dP, dx, ws)
    else:
        m.vjp(P, to_dev(x, wl.dtype), to_dev(seed), B, dP, dx, ws)
    torch.cuda.synchronize()
    if seed is None:
        assert m.check(ws) == dl.OK
    return m, loss.cpu(), dP.cpu(), dx.cpu(), m.workspace_bytes(B)


@pytest.mark.gpu
@pytest.mark.parametrize("cfg", ["10", "16"])
@pytest.mark.parametrize("widths,batch", [
    ((264, 520, 296, 10), 1000),     # ragged rows and columns, several tiles
    ((264, 520, 296, 10), 7),        # one partial tile row
    ((520, 256, 512, 264, 40), 512), # whole tiles, three rectified outputs
])
@pytest.mark.parametrize("entry", ["gradient", "vjp"])
def test_masked_path_is_bitwise_the_saved_output_path(widths, batch, entry, cfg, monkeypatch):
    import torch
    monkeypatch.setenv("DLVM_GEMM_CONFIG", cfg)    # the tile on every product that can run it
    wl = _wl(widths, batch)
    x, params, y = workloads.make_inputs(wl, bias_scale=0.1)
    seed = None
    if entry == "vjp":
        seed = (np.random.default_rng(7).standard_normal((batch, widths[-1])) / batch).astype(np.float32)
    m, *on = _gradient(wl, x, params, y, seed=seed)
    monkeypatch.setenv("DLVM_RELU_MASK", "0")
    _, *off = _gradient(wl, x, params, y, seed=seed)
    assert on[3] > off[3]                            # masks were in use
    assert not torch.isnan(on[1]).any()
    for a, b in zip(on[:3], off[:3]):
        assert torch.equal(a, b)


@pytest.mark.gpu
@pytest.mark.parametrize("cfg", ["10", "16"])
def test_masked_path_with_checkpointing(cfg, monkeypatch):
    """Recomputed segments rewrite their masks: every segment length gives
    bitwise the keep-everything result."""
    import torch
    monkeypatch.setenv("DLVM_GEMM_CONFIG", cfg)
    wl = _wl((264,) + (296,) * 6 + (10,), 600)
    x, params, y = workloads.make_inputs(wl, bias_scale=0.1)
    _, *ref = _gradient(wl, x, params, y)
    for k in (2, 3, 7):
        _, *got = _gradient(wl, x, params, y, ckpt=k)
        for a, b in zip(got[:3], ref[:3]):
            assert torch.equal(a, b), k


@pytest.mark.gpu
@pytest.mark.parametrize("cfg", ["10", "16"])
def test_masked_path_against_oracle(cfg, monkeypatch):
    monkeypatch.setenv("DLVM_GEMM_CONFIG", cfg)
    wl = _wl((264, 520, 296, 10), 1000)
    x, params, y = workloads.make_inputs(wl, bias_scale=0.1)
    m, loss, dP, dx, _ = _gradient(wl, x, params, y)
    spec = oracle.MlpSpec(wl.widths, wl.acts, wl.loss, wl.dtype)
    rl, rg, rdx = oracle.mlp_gradient(spec, x, params, y, wrt_x=True)
    tol = TOL["bf16"]
    assert abs(loss.item() - rl) <= tol * abs(rl)
    for (gw, gb), (rw, rb) in zip(m.unpack(dP), rg):
        assert_close(to_np(gw), rw, tol, "dW")
        assert_close(to_np(gb), rb, tol, "db")
    assert rel_l2(to_np(dx), rdx) <= tol
