"""The C-ABI library on the host: it loads, exports every declared symbol, and
its host-side logic (validation, layouts, plans, error paths) works without a
device. No call here launches a kernel: every call either only computes on the
host or fails validation before any HIP call.
"""
import ctypes
import os

import pytest

import paper_1711_03016_amd as dl
import workloads


@pytest.fixture(scope="module", autouse=True)
def built_library():
    if not os.path.exists(dl.LIB_PATH):
        from paper_1711_03016_amd import build
        build.build()
    dl.lib()


def test_every_declared_function_is_exported():
    names = dl.header_functions()
    assert len(names) >= 20
    missing = [n for n in names if not hasattr(dl.lib(), n)]
    assert missing == []
    for n in ("dlvm_forward", "dlvm_gradient", "dlvm_sgd_step"):
        assert n in names


def _desc(widths, acts, dtype=0, loss=0, wrt_x=0, batch_max=8, ckpt=1):
    L = len(widths) - 1
    w = (ctypes.c_int32 * len(widths))(*widths)
    a = (ctypes.c_int32 * max(L, 1))(*acts)
    return dl._Desc(L, w, a, dtype, loss, wrt_x, batch_max, ckpt, 0), (w, a)


@pytest.mark.parametrize("widths,acts,dtype,loss,wrt_x,batch_max,status", [
    ((4, 3), (0,), 0, 0, 0, 8, dl.OK),
    ((4, 3), (3,), 0, 0, 0, 8, dl.ERR_INVALID_ARG),        # last layer has an activation
    ((4,), (), 0, 0, 0, 8, dl.ERR_INVALID_ARG),            # no layer
    ((4, 0), (0,), 0, 0, 0, 8, dl.ERR_INVALID_ARG),        # zero width
    ((4, 3), (0,), 7, 0, 0, 8, dl.ERR_INVALID_ARG),        # unknown dtype
    ((4, 3), (0,), 0, 5, 0, 8, dl.ERR_INVALID_ARG),        # unknown loss
    ((4, 3), (9,), 0, 0, 0, 8, dl.ERR_INVALID_ARG),        # unknown activation
    ((4, 3), (0,), 0, 0, 0, 0, dl.ERR_INVALID_ARG),        # batch_max 0
    ((4, 3), (0,), 0, 1, 1, 8, dl.ERR_UNSUPPORTED),        # chain needs in == out
    ((4, 4), (0,), 1, 1, 1, 8, dl.ERR_UNSUPPORTED),        # chain is float32
    ((4, 4), (0,), 0, 1, 0, 8, dl.ERR_UNSUPPORTED),        # chain differentiates x
    ((4, 4, 4), (0, 0), 0, 1, 1, 8, dl.ERR_UNSUPPORTED),   # chain is one layer
    ((4, 4), (0,), 0, 1, 1, 8, dl.OK),
])
def test_create_validates(widths, acts, dtype, loss, wrt_x, batch_max, status):
    d, keep = _desc(widths, acts, dtype, loss, wrt_x, batch_max)
    h = ctypes.c_void_p()
    assert dl.lib().dlvm_create(ctypes.byref(d), ctypes.byref(h)) == status
    if status == dl.OK:
        dl.lib().dlvm_destroy(h)
    else:
        assert h.value is None
        assert dl.lib().dlvm_last_error()


@pytest.mark.parametrize("name", sorted(workloads.WORKLOADS))
def test_layout_and_plan(name):
    wl = workloads.WORKLOADS[name]
    m = dl.Model(wl.widths, wl.acts, wl.dtype, wl.loss, wl.wrt_x, wl.batch)
    offs, lds = m.param_layout_lds()
    total = m.param_count()
    es = 2 if wl.dtype == "bf16" else 4
    prev_end = 0
    for l in range(wl.n_layers):
        K, N = wl.widths[l], wl.widths[l + 1]
        ld = lds[l]
        if wl.loss == "softmax_ce" and l == wl.n_layers - 1:
            assert ld == (N + 7) // 8 * 8
        else:
            assert ld == N
        for off, size in ((offs[2 * l], K * ld), (offs[2 * l + 1], N)):
            assert off % 128 == 0 and (off * es) % 256 == 0   # 256-byte aligned tensors
            assert off >= prev_end
            prev_end = off + size
    assert prev_end <= total
    assert total - sum(wl.widths[l] * lds[l] + wl.widths[l + 1] for l in range(wl.n_layers)) < 128 * 2 * wl.n_layers
    assert m.workspace_bytes(wl.batch) > 0
    assert m.workspace_bytes(0) == 0
    assert m.workspace_bytes(wl.batch + 1) == 0
    plan = m.plan(wl.batch)
    assert plan[-1]["name"].startswith("sgd")
    # the launch plan's matrix work is exactly the workload's algorithmic flops
    assert sum(p["flops"] for p in plan) == wl.flops()
    # dead-code elimination: no input-gradient product for layer 1 unless x is
    # differentiated (a paired launch holds one product wrt the weights and one
    # wrt the input)
    if plan[0]["name"].startswith("small_step"):
        # a small float32 network: the whole gradient is one launch
        assert wl.dtype == "f32" and len(plan) == 2
        return
    pair = [p for p in plan if p["name"].startswith("gemm_pair")]
    nt = [p for p in plan if p["name"].startswith("gemm_nt")]
    tn = [p for p in plan if p["name"].startswith("gemm_tn")]
    assert len(nt) + len(pair) == wl.n_layers - 1 + (1 if wl.wrt_x else 0)
    assert len(tn) + len(pair) == wl.n_layers


def test_k_group_tiles_where_the_planner_takes_them():
    """The k-group tiles (configurations 18 and 19) run the products they were
    measured on: the recurrent step's cell products and adjoints in two
    k-slices on 18, the batch-4096 network's large weight adjoints in four
    k-slices on 19; the forward and input-adjoint products of a whole batch
    keep configuration 16, and the deep network keeps its 256 x 256 tiles."""
    wl = workloads.RNN_WORKLOADS["r1"]
    rnn = dl.Rnn(wl.steps, wl.in_width, wl.hidden, wl.act, wl.dtype, wl.wrt_x, wl.wrt_h0, wl.batch)
    names = [p["name"] for p in rnn.plan(wl.batch)]
    assert names.count("gemm_nn_bf16_64x128c18s2") == wl.steps
    assert names.count("gemm_nt_bf16_64x128c18s2") == wl.steps - 1
    assert names.count("split_epilogue") == 2 * wl.steps - 1
    wl = workloads.WORKLOADS["c3"]
    plan = dl.Model(wl.widths, wl.acts, wl.dtype, wl.loss, wl.wrt_x, wl.batch).plan(wl.batch)
    big_tn = [p["name"] for p in plan if p["name"].startswith("gemm_tn") and p["N"] == 1024]
    assert big_tn == ["gemm_tn_bf16_128x128c19s4"] * 2, big_tn
    wide = [p["name"] for p in plan
            if p["name"].startswith(("gemm_nn", "gemm_nt")) and p["M"] == 4096 and p["N"] == 1024]
    assert wide and all(n.endswith("c16") for n in wide), wide
    wl = workloads.WORKLOADS["c5"]
    plan = dl.Model(wl.widths, wl.acts, wl.dtype, wl.loss, wl.wrt_x, wl.batch).plan(wl.batch)
    assert all("c10" in p["name"] for p in plan if p["name"].startswith("gemm")), plan


@pytest.mark.parametrize("name", sorted(workloads.WORKLOADS))
def test_workspace_tensors(name):
    """dlvm_workspace_tensor (host only): the saved layer outputs, logits and
    adjoints lie inside the workspace, do not overlap, have the documented
    strides and types, and invalid requests are refused."""
    wl = workloads.WORKLOADS[name]
    B = wl.batch
    m = dl.Model(wl.widths, wl.acts, wl.dtype, wl.loss, wl.wrt_x, B)
    if m.plan(B)[0]["name"] == "small_step_f32":
        with pytest.raises(dl.DlvmError) as e:       # c1: everything stays in LDS
            m.workspace_tensor_info(B, dl.WS_ADJOINT, 1)
        assert e.value.status == dl.ERR_UNSUPPORTED
        return
    total = m.workspace_bytes(B)
    _, lds = m.param_layout_lds()
    L = wl.n_layers
    chain = wl.loss == "chain8"
    spans = []
    for l in range(1, L):
        off, ld, dt = m.workspace_tensor_info(B, dl.WS_HIDDEN, l)
        assert ld == wl.widths[l] and dt == dl.DTYPES[wl.dtype]
        spans.append((off, off + B * ld * (2 if dt == dl.BF16 else 4)))
    for l in range(1, L + 1):
        off, ld, dt = m.workspace_tensor_info(B, dl.WS_ADJOINT, l)
        assert ld == lds[l - 1]
        assert dt == (dl.F32 if chain else dl.DTYPES[wl.dtype])
        spans.append((off, off + B * ld * (2 if dt == dl.BF16 else 4)))
    split_head = any(e["name"] == "split_softmax_xent" for e in m.plan(B))
    if split_head:
        with pytest.raises(dl.DlvmError) as e:
            m.workspace_tensor_info(B, dl.WS_LOGITS)
        assert e.value.status == dl.ERR_UNSUPPORTED
    else:
        off, ld, dt = m.workspace_tensor_info(B, dl.WS_LOGITS)
        assert ld == wl.widths[L] and dt == dl.F32
        spans.append((off, off + B * ld * 4))
    spans.sort()
    assert all(a % 16 == 0 for a, _ in spans)
    assert all(b <= c for (_, b), (c, _) in zip(spans, spans[1:]))   # disjoint
    assert spans[-1][1] <= total
    for kind, layer in ((dl.WS_HIDDEN, 0), (dl.WS_HIDDEN, L), (dl.WS_ADJOINT, 0),
                        (dl.WS_ADJOINT, L + 1), (7, 1)):
        with pytest.raises(dl.DlvmError) as e:
            m.workspace_tensor_info(B, kind, layer)
        assert e.value.status == dl.ERR_INVALID_ARG
    with pytest.raises(dl.DlvmError):
        m.workspace_tensor_info(B + 1, dl.WS_ADJOINT, 1)


@pytest.mark.parametrize("ckpt,status", [(0, dl.OK), (1, dl.OK), (3, dl.OK), (4, dl.OK),
                                         (5, dl.ERR_INVALID_ARG), (-1, dl.ERR_INVALID_ARG)])
def test_checkpoint_every_is_validated(ckpt, status):
    d, keep = _desc((8, 8, 8, 8, 4), (3, 3, 3, 0), ckpt=ckpt)
    h = ctypes.c_void_p()
    assert dl.lib().dlvm_create(ctypes.byref(d), ctypes.byref(h)) == status
    if status == dl.OK:
        dl.lib().dlvm_destroy(h)


@pytest.mark.parametrize("k", [2, 3, 4, 8])
def test_checkpoint_plan(k):
    """Checkpointing (section 3.1.3): the sweep recomputes the hidden layer
    outputs that are not kept, once per segment; the workspace holds the
    checkpoints plus k-1 segment slots."""
    wl = workloads.WORKLOADS["c5"]
    L, B = wl.n_layers, 256
    full = dl.Model(wl.widths, wl.acts, wl.dtype, wl.loss, wl.wrt_x, B)
    ck = dl.Model(wl.widths, wl.acts, wl.dtype, wl.loss, wl.wrt_x, B, checkpoint_every=k)
    p_full, p_ck = full.plan(B), ck.plan(B)
    nn_full = [p for p in p_full if p["name"].startswith("gemm_nn")]
    nn_ck = [p for p in p_ck if p["name"].startswith("gemm_nn")]
    # hidden outputs H_1 .. H_{L-1}; the resident (last) segment is not redone
    hidden = list(range(1, L))
    last_seg = max(l - l % k for l in hidden if l % k) if any(l % k for l in hidden) else None
    redo = 0
    for l in hidden:
        if l % k == 0:
            continue
        c = l - l % k
        if c != last_seg and (l + 1 >= L or (l + 1) % k == 0):
            redo += l - c   # the segment's layers c .. l-1, once
    assert len(nn_ck) - len(nn_full) == redo
    w = wl.widths
    extra = sum(p["flops"] for p in nn_ck[len(nn_full):])
    assert sum(p["flops"] for p in p_ck) - sum(p["flops"] for p in p_full) == extra
    kept = sum(1 for l in hidden if l % k == 0)
    slots = (k - 1) if any(l % k for l in hidden) else 0
    saved = len(hidden) - kept - slots
    es = 2
    assert full.workspace_bytes(B) - ck.workspace_bytes(B) >= saved * B * w[1] * es
    if saved > 0:
        assert ck.workspace_bytes(B) < full.workspace_bytes(B)


def test_gradient_argument_errors_are_host_side():
    L = dl.lib()
    m = dl.Model((64, 32, 10), ("sigmoid", "none"), batch_max=16)
    h = m._h
    ws = m.workspace_bytes(16)
    A = 0x100000  # never dereferenced: validation fails before any HIP call
    # null pointers
    assert L.dlvm_gradient(h, None, A, A, 16, A, A, None, A, ws, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_gradient(h, A, A, None, 16, A, A, None, A, ws, None) == dl.ERR_INVALID_ARG
    # misaligned
    assert L.dlvm_gradient(h, A + 4, A, A, 16, A, A, None, A, ws, None) == dl.ERR_MISALIGNED
    # batch out of range
    assert L.dlvm_gradient(h, A, A, A, 17, A, A, None, A, ws, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_gradient(h, A, A, A, 0, A, A, None, A, ws, None) == dl.ERR_INVALID_ARG
    # workspace
    assert L.dlvm_gradient(h, A, A, A, 16, A, A, None, A, ws - 1, None) == dl.ERR_WORKSPACE
    assert L.dlvm_gradient(h, A, A, A, 16, A, A, None, None, ws, None) == dl.ERR_WORKSPACE
    assert b"workspace" in L.dlvm_last_error()
    # forward
    assert L.dlvm_forward(h, A, A, 16, None, A, ws, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_forward(h, A, A, 16, A, A, 0, None) == dl.ERR_WORKSPACE
    # sgd
    assert L.dlvm_sgd_step(h, None, None, A, 0.1, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_sgd_step(h, A + 2, None, A, 0.1, None) == dl.ERR_MISALIGNED
    mb = dl.Model((8, 8), ("none",), "bf16", batch_max=4)
    assert L.dlvm_sgd_step(mb._h, A, None, A, 0.1, None) == dl.ERR_INVALID_ARG  # master needed
    # wrt_x requires dx; the chain requires no labels but dx
    mx = dl.Model((8, 8), ("none",), wrt_x=True, batch_max=4)
    w2 = mx.workspace_bytes(4)
    assert L.dlvm_gradient(mx._h, A, A, A, 4, A, A, None, A, w2, None) == dl.ERR_INVALID_ARG
    mc = dl.Model((8, 8), ("none",), "f32", "chain8", True, 4)
    w3 = mc.workspace_bytes(4)
    assert L.dlvm_gradient(mc._h, A, A, None, 4, A, A, None, A, w3, None) == dl.ERR_INVALID_ARG


def test_step_level_errors_are_host_side():
    L = dl.lib()
    A = 0x100000
    assert L.dlvm_dense_forward(0, 1, 0, 4, 4, 4, 1.0, A, A, None, A, None) == dl.ERR_UNSUPPORTED
    assert L.dlvm_dense_forward(0, 0, 0, 0, 4, 4, 1.0, A, A, None, A, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_dense_forward(0, 0, 0, 4, 4, 4, 1.0, A + 8, A, None, A, None) == dl.ERR_MISALIGNED
    assert L.dlvm_dense_backward_data(0, 0, 1, 4, 4, 4, A, A, None, None, A, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_dense_backward_params(3, 4, 4, 4, A, A, A, None, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_softmax_xent(0, 4, 10, A, A, 0.25, A, A, A, 0, None) == dl.ERR_WORKSPACE
    assert L.dlvm_chain8(4, 4, A, A, A, A, None, A, A, 1 << 20, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_sgd(1, 16, A, None, A, 0.1, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_softmax_xent_ws_bytes(0) == 0 and L.dlvm_softmax_xent_ws_bytes(5) > 0
    assert L.dlvm_chain8_ws_bytes(3, 0) == 0 and L.dlvm_chain8_ws_bytes(3, 5) > 0
    # the allocation-free loss refuses rows beyond its static scratch, and bad
    # arguments, before touching the device
    nf = L.dlvm_softmax_xent_noalloc
    assert nf(0, (1 << 20) + 1, 10, A, A, 1.0, A, A, None, None) == dl.ERR_INVALID_ARG
    assert b"1048576" in L.dlvm_last_error()
    assert nf(0, 4, 10, A, A, 1.0, A, None, None, None) == dl.ERR_INVALID_ARG
    assert nf(2, 4, 10, A, A, 1.0, A, A, None, None) == dl.ERR_INVALID_ARG
    assert nf(0, 4, 10, A, A, 1.0, A, A, A + 4, None) == dl.ERR_MISALIGNED


def test_probe_arguments_are_validated():
    L = dl.lib()
    m = dl.Model((8, 8), ("none",), batch_max=4)
    assert L.dlvm_probe_arm(m._h, -2, 4) == dl.ERR_INVALID_ARG
    assert L.dlvm_probe_arm(m._h, 0, 0) == dl.ERR_INVALID_ARG
    n = ctypes.c_int64()
    t = ctypes.c_double()
    assert L.dlvm_probe_read(m._h, 0, ctypes.byref(n), ctypes.byref(t)) == dl.OK
    assert n.value == 0
    assert L.dlvm_probe_disarm(m._h) == dl.OK
    info = dl.LaunchInfo()
    assert L.dlvm_plan_entry(m._h, 4, 99, ctypes.byref(info)) == dl.ERR_INVALID_ARG
    assert L.dlvm_plan_size(m._h, 5) == 0


def test_rnn_handle_plan_and_errors():
    """A recurrent model: T fused cell products (contraction Kx + H), the
    adjoint sweep, one weight-gradient contraction over all T * B rows, and the
    update; the dense-network entry points refuse it; errors are host-side."""
    L = dl.lib()
    wl = workloads.RNN_WORKLOADS["r1"]
    m = dl.Rnn(wl.steps, wl.in_width, wl.hidden, wl.act, wl.dtype, wl.wrt_x, wl.wrt_h0, wl.batch)
    offs, lds = m.param_layout_lds()
    assert offs[0] == 0 and lds == [wl.hidden]
    assert offs[1] >= (wl.in_width + wl.hidden) * wl.hidden and offs[1] % 128 == 0
    plan = m.plan(wl.batch)
    nn = [p for p in plan if p["name"].startswith("gemm_nn")]
    assert len(nn) == wl.steps
    assert all(p["K"] == wl.in_width + wl.hidden and p["M"] == wl.batch for p in nn)
    # every cell is a two-phase product, the first too (its h0 block has a
    # null address in the description, whose bases are null): one tile for all
    assert len({p["name"] for p in nn}) == 1
    assert plan[-1]["name"].startswith("sgd")
    assert sum(p["flops"] for p in plan) == wl.flops()
    ws = m.workspace_bytes(wl.batch)
    assert ws >= wl.steps * wl.batch * wl.hidden * 2
    A = 0x100000
    B = wl.batch
    # dense entry points refuse a recurrent handle
    assert L.dlvm_forward(m._h, A, A, B, A, A, ws, None) == dl.ERR_UNSUPPORTED
    assert L.dlvm_gradient(m._h, A, A, A, B, A, A, A, A, ws, None) == dl.ERR_UNSUPPORTED
    assert L.dlvm_vjp(m._h, A, A, A, B, A, A, A, ws, None) == dl.ERR_UNSUPPORTED
    # recurrent entry points: nulls, declared outputs, alignment, batch, workspace
    assert L.dlvm_rnn_forward(m._h, None, A, B, A, None, 0, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_rnn_forward(m._h, A, A + 2, B, A, None, 0, None) == dl.ERR_MISALIGNED
    assert L.dlvm_rnn_forward(m._h, A, A, B + 1, A, None, 0, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_rnn_forward(m._h, A, A, B, A, A, ws - 1, None) == dl.ERR_WORKSPACE
    assert L.dlvm_rnn_backward(m._h, A, A, A, A, B, A, None, A, A, ws, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_rnn_backward(m._h, A, A, A, A, B, A, A, None, A, ws, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_rnn_backward(m._h, A, A, A, A, B, A, A, A, A, ws - 1, None) == dl.ERR_WORKSPACE
    mlp = dl.Model((8, 8), ("none",), batch_max=4)
    assert L.dlvm_rnn_forward(mlp._h, A, A, 4, A, None, 0, None) == dl.ERR_UNSUPPORTED
    # create validation
    for bad in (dict(steps=0), dict(in_width=0), dict(hidden=0), dict(batch_max=0)):
        args = dict(steps=4, in_width=8, hidden=8, batch_max=4)
        args.update(bad)
        d = dl._RnnDesc(0, 2, args["steps"], args["in_width"], args["hidden"], args["batch_max"], 0, 0)
        h = ctypes.c_void_p()
        assert L.dlvm_rnn_create(ctypes.byref(d), ctypes.byref(h)) == dl.ERR_INVALID_ARG
    assert L.dlvm_rnn_cell_forward(0, 2, 4, 0, 4, 4, A, A, A, None, A, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_rnn_cell_forward(0, 2, 4, 4, 4, 4, A, A + 4, A, None, A, None) == dl.ERR_MISALIGNED


def test_rnn_dead_outputs_are_not_computed():
    """Without wrt_x / wrt_h0 the products that only feed dxs / dh0 are absent."""
    full = dl.Rnn(4, 64, 32, "tanh", "f32", True, True, 16).plan(16)
    lean = dl.Rnn(4, 64, 32, "tanh", "f32", False, False, 16).plan(16)
    nt = lambda p: sum(1 for e in p if "nt" in e["name"].split("_")[1])  # noqa: E731
    pairs = lambda p: sum(1 for e in p if e["name"].startswith("gemm_pair"))  # noqa: E731
    assert nt(full) + pairs(full) == nt(lean) + 2
    assert sum(e["flops"] for e in full) - sum(e["flops"] for e in lean) == \
        2 * 16 * 32 * 32 + 2 * 4 * 16 * 32 * 64


def test_chain_order_matches_oracle():
    """The library's host-side order (its own recurrence) against the oracle's:
    the same least cost and the same cuts (smallest cut among equal costs)."""
    import numpy as np
    import oracle
    rng = np.random.default_rng(17)
    for _ in range(300):
        n = int(rng.integers(1, 10))
        d = [int(v) for v in rng.integers(1, 200, size=n + 1)]
        assert dl.chain_order(d) == oracle.chain_order(d)
    assert dl.chain_order([30, 35, 15, 5, 10, 20, 25])[0] == 15125
    # large dimensions: the cost stays exact in 64 bits here
    d = [1 << 20, 1 << 20, 1 << 10, 1 << 20]
    assert dl.chain_order(d) == oracle.chain_order(d)


def test_matrix_chain_errors_are_host_side():
    L = dl.lib()
    A = 0x100000
    n = 3
    dims = (ctypes.c_int64 * 4)(8, 16, 4, 8)
    mats = (ctypes.c_void_p * 3)(A, A, A)
    assert L.dlvm_chain_order(0, dims, None) == -1
    assert L.dlvm_chain_order(n, (ctypes.c_int64 * 4)(8, 0, 4, 8), None) == -1
    assert L.dlvm_matrix_chain(0, 1, dims, mats, None, A, A, 1 << 20, None) == dl.ERR_INVALID_ARG
    bad = (ctypes.c_int32 * 9)(-1, 0, 2, -1, -1, 1, -1, -1, -1)   # cut of (0,2) outside [0, 2)
    assert L.dlvm_matrix_chain(0, n, dims, mats, bad, A, A, 1 << 20, None) == dl.ERR_INVALID_ARG
    assert L.dlvm_matrix_chain_ws_bytes(0, n, dims, bad) == 0
    mis = (ctypes.c_void_p * 3)(A, A + 4, A)
    assert L.dlvm_matrix_chain(0, n, dims, mis, None, A, A, 1 << 20, None) == dl.ERR_MISALIGNED
    need = L.dlvm_matrix_chain_ws_bytes(0, n, dims, None)
    assert need >= 8 * 4 * 4 or need >= 16 * 8 * 4
    assert L.dlvm_matrix_chain(0, n, dims, mats, None, A, A, need - 1, None) == dl.ERR_WORKSPACE


def test_handle_kinds_refuse_calls_that_do_not_apply():
    L = dl.lib()
    A = 0x100000
    r = dl.Rnn(2, 8, 8, "tanh", "f32", False, False, 4)
    c = dl.Chain("f32", [8, 4, 8])
    assert L.dlvm_check(r._h, A, None) == dl.ERR_UNSUPPORTED
    assert L.dlvm_check(c._h, A, None) == dl.ERR_UNSUPPORTED
    assert L.dlvm_sgd_step(c._h, A, None, A, 0.1, None) == dl.ERR_UNSUPPORTED
    assert L.dlvm_chain_run(r._h, (ctypes.c_void_p * 2)(A, A), A, A, 1 << 20, None) == dl.ERR_UNSUPPORTED
    assert L.dlvm_rnn_backward(c._h, A, A, A, A, 1, A, None, None, A, 1 << 20, None) == dl.ERR_UNSUPPORTED
    assert c.workspace_bytes(1) >= 16 and c.workspace_bytes(2) == 0
    plan = c.plan(1)
    assert [p["name"].split("_")[0] for p in plan[:-1]] == ["gemm"]


def test_small_network_plan(monkeypatch):
    """Small float32 softmax networks take the one-workgroup gradient; larger
    ones, bf16 ones and the chain keep the general plan; DLVM_SMALL_STEP=0
    turns it off."""
    small = dl.Model((64, 32, 10), ("sigmoid", "none"), batch_max=16)
    assert [p["name"] for p in small.plan(16)] == ["small_step_f32", "sgd_f32"]
    assert not dl.Model((784, 512, 512, 10), ("tanh", "tanh", "none"), batch_max=256) \
        .plan(256)[0]["name"].startswith("small")
    assert not dl.Model((64, 32, 10), ("sigmoid", "none"), "bf16", batch_max=16) \
        .plan(16)[0]["name"].startswith("small")
    # at the limits: LDS (the batch), the layer count
    assert dl.Model((6, 3), ("none",), batch_max=600).plan(600)[0]["name"] == "small_step_f32"
    assert dl.Model((6, 3), ("none",), batch_max=1000).plan(1000)[0]["name"].startswith("gemm")
    deep = (12,) * 8 + (10,)
    assert dl.Model(deep, ("tanh",) * 7 + ("none",), batch_max=8).plan(8)[0]["name"] == "small_step_f32"
    deeper = (12,) * 9 + (10,)
    assert dl.Model(deeper, ("tanh",) * 8 + ("none",), batch_max=8).plan(8)[0]["name"].startswith("gemm")
    monkeypatch.setenv("DLVM_SMALL_STEP", "0")
    assert small.plan(16)[0]["name"].startswith("gemm_nn")


def test_one_hip_runtime_whatever_the_import_order():
    """The library loaded before the caller imports torch still binds to
    torch's HIP runtime: one libamdhip64 mapped in the process (a second one
    would be a second HIP/HSA runtime, whose launches cannot find the
    device)."""
    import subprocess
    import sys
    code = (
        "import paper_1711_03016_amd as dl\n"
        "dl.lib()\n"
        "import torch\n"
        "paths = {l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}\n"
        "print(len(paths))\n"
    )
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True,
                         timeout=300)
    assert out.returncode == 0, out.stderr[-2000:]
    assert out.stdout.strip().splitlines()[-1] == "1"
