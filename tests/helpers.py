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
