"""Shared test utilities: tolerances, device transfer, error measures."""
import numpy as np

# Relative L2 error bounds per output tensor: float32 storage, and bf16
# storage with float32 accumulation.
TOL = {"f32": 1e-4, "bf16": 2e-2}


def rel_l2(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(got - ref)
    return float(num / den) if den > 0 else float(num)


def rel_rows(got, ref, floor: float = 0.05) -> float:
    """The largest relative error of one row: max_i ||g_i - o_i|| / ||o_i||.

    A whole-tensor norm hides a single wrong row (one row of 4096 left at zero
    moves the tensor's relative error by 1/64); this measure does not. A row
    whose norm is below `floor` times the root-mean-square row norm is
    measured against that floor instead, so rows that are nearly zero (a ReLU
    output with few active units) are not judged on their rounding noise
    alone. One-dimensional arrays are taken one element per row.
    """
    g = np.asarray(got, np.float64)
    o = np.asarray(ref, np.float64)
    assert g.shape == o.shape, (g.shape, o.shape)
    if g.size == 0:
        return 0.0
    if g.ndim == 1:
        g, o = g[:, None], o[:, None]
    g = g.reshape(g.shape[0], -1)
    o = o.reshape(o.shape[0], -1)
    num = np.linalg.norm(g - o, axis=1)
    den = np.linalg.norm(o, axis=1)
    rms = float(np.sqrt(np.mean(den ** 2)))
    if rms == 0.0:
        return float(num.max())
    return float((num / np.maximum(den, floor * rms)).max())


def assert_close(got, ref, tol: float, what="", row_tol: float | None = None,
                 floor: float | None = None) -> None:
    """Whole-tensor relative L2 error within `tol` and every row's relative
    error (rel_rows) within `row_tol` (default: `tol`). Vectors are checked
    element by element against their root-mean-square (floor 1) unless a
    floor is given."""
    row_tol = tol if row_tol is None else row_tol
    if floor is None:
        floor = 1.0 if np.ndim(ref) == 1 else 0.05
    e = rel_l2(got, ref)
    r = rel_rows(got, ref, floor)
    assert e <= tol, (what, "rel_l2", e, tol)
    assert r <= row_tol, (what, "worst row", r, row_tol)


def device():
    import torch
    assert torch.cuda.is_available(), "this test needs a GPU"
    return torch.device("cuda:0")


def torch_dtype(dtype: str):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]


def to_dev(a, dtype: str = "f32"):
    """A float32 host array as a device tensor of the storage type (bf16: RNE)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.float32)))
    return t.to(device()).to(torch_dtype(dtype)).contiguous()


def to_np(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float64).cpu().numpy()


def quant(a, dtype: str) -> np.ndarray:
    """The value the oracle sees for a float32 input stored as `dtype`."""
    import oracle
    a32 = np.asarray(a, np.float32)
    return oracle.round_to_bf16(a32) if dtype == "bf16" else a32.astype(np.float64)
