"""Python binding of ``libdlvm.so``, the gfx950 hot path of a DLVM-compiled network.

Argument marshalling only: every step of the forward, the gradient and the
update runs in the library's HIP kernels. PyTorch supplies device memory and
streams; tensors are passed as raw device pointers. The library must have
been built (``python -m paper_1711_03016_amd.build``); importing the binding
on a machine without it raises at first use, there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdlvm.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "dlvm.h")

# Constants mirrored from include/dlvm.h.
OK, ERR_INVALID_ARG, ERR_MISALIGNED, ERR_WORKSPACE = 0, -1, -2, -3
ERR_UNSUPPORTED, ERR_HIP, ERR_LABEL_RANGE, ERR_NONFINITE = -4, -5, -6, -7
F32, BF16 = 0, 1
ACTS = {"none": 0, "sigmoid": 1, "tanh": 2, "relu": 3}
DTYPES = {"f32": F32, "bf16": BF16}
LOSSES = {"softmax_ce": 0, "chain8": 1}
WS_HIDDEN, WS_LOGITS, WS_ADJOINT = 0, 1, 2


class DlvmError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"dlvm status {status}: {message}")
        self.status = status


class _Desc(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32),
        ("widths", ctypes.POINTER(ctypes.c_int32)),
        ("acts", ctypes.POINTER(ctypes.c_int32)),
        ("dtype", ctypes.c_int32),
        ("loss", ctypes.c_int32),
        ("wrt_x", ctypes.c_int32),
        ("batch_max", ctypes.c_int64),
        ("checkpoint_every", ctypes.c_int32),
        ("chain_in_epilogue", ctypes.c_int32),
    ]


class _RnnDesc(ctypes.Structure):
    _fields_ = [
        ("dtype", ctypes.c_int32),
        ("act", ctypes.c_int32),
        ("steps", ctypes.c_int64),
        ("in_width", ctypes.c_int64),
        ("hidden", ctypes.c_int64),
        ("batch_max", ctypes.c_int64),
        ("wrt_x", ctypes.c_int32),
        ("wrt_h0", ctypes.c_int32),
    ]


class LaunchInfo(ctypes.Structure):
    _fields_ = [
        ("name", ctypes.c_char * 48),
        ("M", ctypes.c_int64),
        ("N", ctypes.c_int64),
        ("K", ctypes.c_int64),
        ("flops", ctypes.c_double),
        ("bytes", ctypes.c_double),
    ]


_lib = None
_P = ctypes.c_void_p
_I32, _I64, _F = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
_SIGS = {
    "dlvm_create": (_I32, [ctypes.POINTER(_Desc), ctypes.POINTER(_P)]),
    "dlvm_destroy": (None, [_P]),
    "dlvm_param_count": (_I64, [_P]),
    "dlvm_param_layout": (_I32, [_P, ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "dlvm_workspace_bytes": (ctypes.c_size_t, [_P, _I64]),
    "dlvm_workspace_tensor": (_I32, [_P, _I64, _I32, _I32, ctypes.POINTER(ctypes.c_size_t),
                                     ctypes.POINTER(_I64), ctypes.POINTER(_I32)]),
    "dlvm_forward": (_I32, [_P, _P, _P, _I64, _P, _P, ctypes.c_size_t, _P]),
    "dlvm_gradient": (_I32, [_P, _P, _P, _P, _I64, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "dlvm_sgd_step": (_I32, [_P, _P, _P, _P, _F, _P]),
    "dlvm_vjp": (_I32, [_P, _P, _P, _P, _I64, _P, _P, _P, ctypes.c_size_t, _P]),
    "dlvm_check": (_I32, [_P, _P, _P]),
    "dlvm_last_error": (ctypes.c_char_p, []),
    "dlvm_dense_forward": (_I32, [_I32, _I32, _I32, _I64, _I64, _I64, _F, _P, _P, _P, _P, _P]),
    "dlvm_dense_backward_data": (_I32, [_I32, _I32, _I32, _I64, _I64, _I64, _P, _P, _P, _P, _P, _P]),
    "dlvm_dense_backward_params": (_I32, [_I32, _I64, _I64, _I64, _P, _P, _P, _P, _P]),
    "dlvm_softmax_xent_ws_bytes": (ctypes.c_size_t, [_I64]),
    "dlvm_softmax_xent": (_I32, [_I32, _I64, _I64, _P, _P, _F, _P, _P, _P, ctypes.c_size_t, _P]),
    "dlvm_softmax_xent_noalloc": (_I32, [_I32, _I64, _I64, _P, _P, _F, _P, _P, _P, _P]),
    "dlvm_chain8_ws_bytes": (ctypes.c_size_t, [_I64, _I64]),
    "dlvm_chain8": (_I32, [_I64, _I64, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "dlvm_sgd": (_I32, [_I32, _I64, _P, _P, _P, _F, _P]),
    "dlvm_plan_size": (_I32, [_P, _I64]),
    "dlvm_plan_entry": (_I32, [_P, _I64, _I32, ctypes.POINTER(LaunchInfo)]),
    "dlvm_probe_arm": (_I32, [_P, _I32, _I32]),
    "dlvm_probe_read": (_I32, [_P, _I32, ctypes.POINTER(_I64), ctypes.POINTER(ctypes.c_double)]),
    "dlvm_probe_disarm": (_I32, [_P]),
    "dlvm_step_graph_create": (_I32, [_P, _P, _P, _P, _P, _I64, _P, _P, _P, _P, ctypes.c_size_t,
                                      _I32, _F, ctypes.POINTER(_P)]),
    "dlvm_rnn_create": (_I32, [ctypes.POINTER(_RnnDesc), ctypes.POINTER(_P)]),
    "dlvm_rnn_forward": (_I32, [_P, _P, _P, _I64, _P, _P, ctypes.c_size_t, _P]),
    "dlvm_rnn_backward": (_I32, [_P, _P, _P, _P, _P, _I64, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "dlvm_rnn_cell_forward": (_I32, [_I32, _I32, _I64, _I64, _I64, _I64, _P, _P, _P, _P, _P, _P]),
    "dlvm_chain_order": (_I64, [_I32, ctypes.POINTER(_I64), ctypes.POINTER(_I32)]),
    "dlvm_matrix_chain_ws_bytes": (ctypes.c_size_t, [_I32, _I32, ctypes.POINTER(_I64),
                                                     ctypes.POINTER(_I32)]),
    "dlvm_matrix_chain": (_I32, [_I32, _I32, ctypes.POINTER(_I64), ctypes.POINTER(_P),
                                 ctypes.POINTER(_I32), _P, _P, ctypes.c_size_t, _P]),
    "dlvm_chain_create": (_I32, [_I32, _I32, ctypes.POINTER(_I64), ctypes.POINTER(_I32),
                                 ctypes.POINTER(_P)]),
    "dlvm_chain_run": (_I32, [_P, ctypes.POINTER(_P), _P, _P, ctypes.c_size_t, _P]),
    "dlvm_graph_launch": (_I32, [_P, _P]),
    "dlvm_graph_destroy": (None, [_P]),
}


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_1711_03016_amd.build`")
        # torch brings its own HIP runtime (libamdhip64 with the same soname).
        # Loaded first, it is the one the library binds to; loaded after the
        # library, it would be a second HIP/HSA runtime in the process, and
        # the library's launches would then fail to find the device.
        import torch  # noqa: F401
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _lib = h
    return _lib


def header_functions() -> list[str]:
    """Names of every function the C header declares."""
    text = open(HEADER_PATH).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dlvm_[a-z0-9_]+)\s*\(", text)))


def _check(status: int) -> None:
    if status != OK:
        msg = lib().dlvm_last_error()
        raise DlvmError(status, msg.decode() if msg else "")


def _ptr(t) -> int | None:
    """Device address of a tensor (or an int address, or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Model:
    """A handle on one shape-specialised network (see ``dlvm_create``)."""

    def __init__(self, widths, acts, dtype: str = "f32", loss: str = "softmax_ce",
                 wrt_x: bool = False, batch_max: int = 1, checkpoint_every: int = 1,
                 chain_in_epilogue: bool = False):
        self.widths = tuple(int(w) for w in widths)
        self.acts = tuple(acts)
        self.dtype = dtype
        self.loss = loss
        self.wrt_x = bool(wrt_x)
        self.batch_max = int(batch_max)
        self.checkpoint_every = int(checkpoint_every)
        self.chain_in_epilogue = bool(chain_in_epilogue)
        L = len(self.widths) - 1
        self._w = (ctypes.c_int32 * (L + 1))(*self.widths)
        self._a = (ctypes.c_int32 * max(L, 1))(*[ACTS[a] for a in self.acts])
        desc = _Desc(L, self._w, self._a, DTYPES[dtype], LOSSES[loss], int(self.wrt_x),
                     self.batch_max, self.checkpoint_every, int(self.chain_in_epilogue))
        h = _P()
        _check(lib().dlvm_create(ctypes.byref(desc), ctypes.byref(h)))
        self._h = h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.dlvm_destroy(h)
            self._h = None

    @property
    def n_layers(self) -> int:
        return len(self.widths) - 1

    def param_count(self) -> int:
        return int(lib().dlvm_param_count(self._h))

    def param_layout(self) -> list[int]:
        """Element offsets [W_1, b_1, ..., W_L, b_L] of the flat buffer."""
        return self.param_layout_lds()[0]

    def param_layout_lds(self) -> tuple[list[int], list[int]]:
        """(offsets, row stride of each W) of the flat buffer."""
        arr = (_I64 * (2 * self.n_layers))()
        lds = (_I64 * self.n_layers)()
        _check(lib().dlvm_param_layout(self._h, arr, lds))
        return list(arr), list(lds)

    def pack(self, params, device, torch_dtype):
        """A flat parameter tensor (zero padding) holding [(W [K,N], b [N]), ...]."""
        import torch
        flat = torch.zeros(self.param_count(), dtype=torch_dtype, device=device)
        for (Wv, bv), (W, b) in zip(self.unpack(flat), params):
            Wv.copy_(torch.as_tensor(W).to(device=device, dtype=torch_dtype))
            bv.copy_(torch.as_tensor(b).reshape(-1).to(device=device, dtype=torch_dtype))
        return flat

    def unpack(self, flat, padded: bool = False):
        """Views [(W [K,N], b [N]), ...] into a flat parameter or gradient tensor.

        With padded=True the weight views include the padding columns [K, ld].
        """
        offs, lds = self.param_layout_lds()
        out = []
        for l in range(self.n_layers):
            K, N, ld = self.widths[l], self.widths[l + 1], lds[l]
            Wp = flat[offs[2 * l]:offs[2 * l] + K * ld].view(K, ld)
            out.append((Wp if padded else Wp[:, :N], flat[offs[2 * l + 1]:offs[2 * l + 1] + N]))
        return out

    def workspace_bytes(self, batch: int) -> int:
        return int(lib().dlvm_workspace_bytes(self._h, int(batch)))

    def workspace_tensor_info(self, batch: int, kind: int, layer: int = 0) -> tuple[int, int, int]:
        """(byte offset, row stride, dtype code) of a tensor a gradient call
        keeps in its workspace (``dlvm_workspace_tensor``)."""
        off, ld, dt = ctypes.c_size_t(), _I64(), _I32()
        _check(lib().dlvm_workspace_tensor(self._h, int(batch), int(kind), int(layer),
                                           ctypes.byref(off), ctypes.byref(ld), ctypes.byref(dt)))
        return int(off.value), int(ld.value), int(dt.value)

    def workspace_tensor(self, ws, batch: int, kind: int, layer: int = 0):
        """A [batch, ld] view into the byte tensor `ws` of the saved layer
        output (WS_HIDDEN), the logits (WS_LOGITS) or a layer's adjoint
        (WS_ADJOINT) that the last gradient call on `ws` wrote."""
        import torch
        off, ld, dt = self.workspace_tensor_info(batch, kind, layer)
        tdt, es = (torch.float32, 4) if dt == F32 else (torch.bfloat16, 2)
        return ws[off:off + int(batch) * ld * es].view(tdt).view(int(batch), ld)

    def forward(self, params, x, batch, out, ws, stream=None) -> None:
        _check(lib().dlvm_forward(self._h, _ptr(params), _ptr(x), int(batch), _ptr(out),
                                  _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))

    def gradient(self, params, x, labels, batch, loss, dparams, dx, ws, stream=None) -> None:
        _check(lib().dlvm_gradient(self._h, _ptr(params), _ptr(x), _ptr(labels), int(batch),
                                   _ptr(loss), _ptr(dparams), _ptr(dx), _ptr(ws),
                                   ws.numel() * ws.element_size(), _stream(stream)))

    def vjp(self, params, x, seed, batch, dparams, dx, ws, stream=None) -> None:
        """Seedable gradient of the logits (``dlvm_vjp``)."""
        _check(lib().dlvm_vjp(self._h, _ptr(params), _ptr(x), _ptr(seed), int(batch),
                              _ptr(dparams), _ptr(dx), _ptr(ws), ws.numel() * ws.element_size(),
                              _stream(stream)))

    def sgd_step(self, params, master, dparams, lr: float, stream=None) -> None:
        _check(lib().dlvm_sgd_step(self._h, _ptr(params), _ptr(master), _ptr(dparams),
                                   float(lr), _stream(stream)))

    def plan(self, batch: int) -> list[dict]:
        """The launches of one training step (gradient call, then SGD call)."""
        n = int(lib().dlvm_plan_size(self._h, int(batch)))
        out = []
        for i in range(n):
            info = LaunchInfo()
            _check(lib().dlvm_plan_entry(self._h, int(batch), i, ctypes.byref(info)))
            out.append({"index": i, "name": info.name.decode(), "M": info.M, "N": info.N,
                        "K": info.K, "flops": info.flops, "bytes": info.bytes})
        return out

    def probe_arm(self, index: int, capacity: int) -> None:
        _check(lib().dlvm_probe_arm(self._h, int(index), int(capacity)))

    def probe_read(self, index: int) -> tuple[int, float]:
        """(launches recorded at position `index`, their summed milliseconds)."""
        n = _I64()
        ms = ctypes.c_double()
        _check(lib().dlvm_probe_read(self._h, int(index), ctypes.byref(n), ctypes.byref(ms)))
        return int(n.value), float(ms.value)

    def probe_disarm(self) -> None:
        _check(lib().dlvm_probe_disarm(self._h))

    def step_graph(self, params, master, x, labels, batch, loss, dparams, dx, ws,
                   update: bool = False, lr: float = 0.0) -> "StepGraph":
        """Capture one training step (gradient [+ SGD]) for replay (``dlvm_step_graph_create``)."""
        g = _P()
        _check(lib().dlvm_step_graph_create(self._h, _ptr(params), _ptr(master), _ptr(x),
                                            _ptr(labels), int(batch), _ptr(loss), _ptr(dparams),
                                            _ptr(dx), _ptr(ws), ws.numel() * ws.element_size(),
                                            int(bool(update)), float(lr), ctypes.byref(g)))
        return StepGraph(g, self)

    def check(self, ws, stream=None) -> int:
        """Status of the device flags (0, ERR_LABEL_RANGE or ERR_NONFINITE)."""
        return int(lib().dlvm_check(self._h, _ptr(ws), _stream(stream)))


class Rnn(Model):
    """A handle on a recurrent network (see ``dlvm_rnn_create``): T steps of the
    cell ``hs[t+1] = act(xs[t] . W + hs[t] . U + b)``, one fused product each.

    The flat parameter buffer holds the stacked ``[W; U]`` ([Kx + H, H]) and
    ``b``; ``pack_cell`` / ``split_cell`` convert from and to (W, U, b).
    """

    def __init__(self, steps: int, in_width: int, hidden: int, act: str = "tanh",
                 dtype: str = "f32", wrt_x: bool = False, wrt_h0: bool = False,
                 batch_max: int = 1):
        self.steps, self.in_width, self.hidden = int(steps), int(in_width), int(hidden)
        self.widths = (self.in_width + self.hidden, self.hidden)
        self.acts = (act,)
        self.dtype = dtype
        self.loss = None
        self.wrt_x, self.wrt_h0 = bool(wrt_x), bool(wrt_h0)
        self.batch_max = int(batch_max)
        self.checkpoint_every = 1
        desc = _RnnDesc(DTYPES[dtype], ACTS[act], self.steps, self.in_width, self.hidden,
                        self.batch_max, int(self.wrt_x), int(self.wrt_h0))
        h = _P()
        _check(lib().dlvm_rnn_create(ctypes.byref(desc), ctypes.byref(h)))
        self._h = h

    def pack_cell(self, W, U, b, device, torch_dtype):
        """A flat parameter tensor holding [W; U] and b."""
        import numpy as np
        WU = np.concatenate([np.asarray(W), np.asarray(U)], axis=0)
        return self.pack([(WU, np.asarray(b))], device, torch_dtype)

    def split_cell(self, flat):
        """Views (W [Kx, H], U [H, H], b [H]) into a flat parameter or gradient tensor."""
        (WU, b), = self.unpack(flat)
        return WU[:self.in_width], WU[self.in_width:], b

    def forward(self, params, xs, batch, hs, ws=None, stream=None) -> None:
        """hs[1..T] from xs [T, batch, Kx] and hs[0] ([T + 1, batch, H] buffer);
        `ws` (optional) lets the planner split the cell products."""
        nb = 0 if ws is None else ws.numel() * ws.element_size()
        _check(lib().dlvm_rnn_forward(self._h, _ptr(params), _ptr(xs), int(batch), _ptr(hs),
                                      _ptr(ws), nb, _stream(stream)))

    def backward(self, params, xs, hs, dhs, batch, dparams, dxs, dh0, ws, stream=None) -> None:
        """d[W; U], db (and dxs, dh0 when declared) for the output adjoints dhs."""
        _check(lib().dlvm_rnn_backward(self._h, _ptr(params), _ptr(xs), _ptr(hs), _ptr(dhs),
                                       int(batch), _ptr(dparams), _ptr(dxs), _ptr(dh0),
                                       _ptr(ws), ws.numel() * ws.element_size(),
                                       _stream(stream)))


class StepGraph:
    """A captured training step; ``launch()`` enqueues one replay."""

    def __init__(self, handle, model):
        self._g = handle
        self._model = model  # the graph must not outlive the model

    def launch(self, stream=None) -> None:
        _check(lib().dlvm_graph_launch(self._g, _stream(stream)))

    def __del__(self):
        g = getattr(self, "_g", None)
        if g is not None and g.value and _lib is not None:
            _lib.dlvm_graph_destroy(g)
            self._g = None


# ---------------------------------------------------------------------------
# step-level entry points
# ---------------------------------------------------------------------------
def dense_forward(dtype, out_dtype, act, M, N, K, alpha, X, W, bias, H, stream=None):
    _check(lib().dlvm_dense_forward(DTYPES[dtype], DTYPES[out_dtype], ACTS[act], M, N, K,
                                    float(alpha), _ptr(X), _ptr(W), _ptr(bias), _ptr(H),
                                    _stream(stream)))


def rnn_cell_forward(dtype, act, M, Kx, Kh, N, X, H, WU, bias, Hout, stream=None):
    _check(lib().dlvm_rnn_cell_forward(DTYPES[dtype], ACTS[act], M, Kx, Kh, N, _ptr(X), _ptr(H),
                                       _ptr(WU), _ptr(bias), _ptr(Hout), _stream(stream)))


def dense_backward_data(dtype, out_dtype, act_prev, M, N, K, dY, W, Hprev, R, dX, stream=None):
    _check(lib().dlvm_dense_backward_data(DTYPES[dtype], DTYPES[out_dtype], ACTS[act_prev],
                                          M, N, K, _ptr(dY), _ptr(W), _ptr(Hprev), _ptr(R),
                                          _ptr(dX), _stream(stream)))


def dense_backward_params(dtype, M, N, K, X, dY, dW, db, stream=None):
    _check(lib().dlvm_dense_backward_params(DTYPES[dtype], M, N, K, _ptr(X), _ptr(dY),
                                            _ptr(dW), _ptr(db), _stream(stream)))


def softmax_xent_ws_bytes(rows: int) -> int:
    return int(lib().dlvm_softmax_xent_ws_bytes(int(rows)))


def softmax_xent(dtype, rows, classes, logits, labels, scale, dlogits, loss, ws, stream=None):
    _check(lib().dlvm_softmax_xent(DTYPES[dtype], rows, classes, _ptr(logits), _ptr(labels),
                                   float(scale), _ptr(dlogits), _ptr(loss), _ptr(ws),
                                   ws.numel() * ws.element_size(), _stream(stream)))


def softmax_xent_noalloc(dtype, rows, classes, logits, labels, scale, dlogits, loss, flags=None,
                         stream=None):
    """dlvm_softmax_xent without a workspace (the library's static scratch)."""
    _check(lib().dlvm_softmax_xent_noalloc(DTYPES[dtype], rows, classes, _ptr(logits),
                                           _ptr(labels), float(scale), _ptr(dlogits), _ptr(loss),
                                           _ptr(flags), _stream(stream)))


def chain8_ws_bytes(rows: int, cols: int) -> int:
    return int(lib().dlvm_chain8_ws_bytes(int(rows), int(cols)))


def chain8(rows, cols, z, bias, x_skip, zbar, xbar, loss, ws, stream=None):
    _check(lib().dlvm_chain8(rows, cols, _ptr(z), _ptr(bias), _ptr(x_skip), _ptr(zbar),
                             _ptr(xbar), _ptr(loss), _ptr(ws), ws.numel() * ws.element_size(),
                             _stream(stream)))


def sgd(dtype, n, params, master, grads, lr, stream=None):
    _check(lib().dlvm_sgd(DTYPES[dtype], int(n), _ptr(params), _ptr(master), _ptr(grads),
                          float(lr), _stream(stream)))


# ---------------------------------------------------------------------------
# matrix multiplication reordering
# ---------------------------------------------------------------------------
def _split_arg(split, n):
    if split is None:
        return None
    flat = [int(v) for row in split for v in row]
    assert len(flat) == n * n
    return (_I32 * (n * n))(*flat)


def chain_order(dims) -> tuple[int, list[list[int]]]:
    """(multiply-add count of the best order, n x n split table) for a chain
    with shapes dims[i] x dims[i+1] (``dlvm_chain_order``)."""
    n = len(dims) - 1
    d = (_I64 * (n + 1))(*[int(v) for v in dims])
    sp = (_I32 * (n * n))()
    cost = int(lib().dlvm_chain_order(n, d, sp))
    if cost < 0:
        raise DlvmError(ERR_INVALID_ARG, "invalid chain")
    return cost, [list(sp[i * n:(i + 1) * n]) for i in range(n)]


def matrix_chain_ws_bytes(dtype, dims, split=None) -> int:
    n = len(dims) - 1
    d = (_I64 * (n + 1))(*[int(v) for v in dims])
    return int(lib().dlvm_matrix_chain_ws_bytes(DTYPES[dtype], n, d, _split_arg(split, n)))


def matrix_chain(dtype, dims, mats, out, ws, split=None, stream=None) -> None:
    """out = mats[0] @ ... @ mats[-1] in the given (or the optimal) order."""
    n = len(dims) - 1
    d = (_I64 * (n + 1))(*[int(v) for v in dims])
    ptrs = (_P * n)(*[_ptr(m) for m in mats])
    nb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().dlvm_matrix_chain(DTYPES[dtype], n, d, ptrs, _split_arg(split, n), _ptr(out),
                                   _ptr(ws), nb, _stream(stream)))


class Chain(Model):
    """A matrix chain of fixed shapes and order (``dlvm_chain_create``)."""

    def __init__(self, dtype, dims, split=None):
        self.dims = tuple(int(v) for v in dims)
        n = len(self.dims) - 1
        self.dtype, self.n = dtype, n
        self.widths, self.acts, self.loss, self.batch_max = (), (), None, 1
        d = (_I64 * (n + 1))(*self.dims)
        h = _P()
        _check(lib().dlvm_chain_create(DTYPES[dtype], n, d, _split_arg(split, n), ctypes.byref(h)))
        self._h = h

    @property
    def n_layers(self) -> int:
        return 0

    def run(self, mats, out, ws, stream=None) -> None:
        ptrs = (_P * self.n)(*[_ptr(m) for m in mats])
        _check(lib().dlvm_chain_run(self._h, ptrs, _ptr(out), _ptr(ws),
                                    ws.numel() * ws.element_size(), _stream(stream)))
