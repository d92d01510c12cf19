"""The allocation-free softmax cross-entropy (dlvm_softmax_xent_noalloc), for
callers that cannot allocate: its loss partials live in the library's static
device array. Checked through the C ABI against the workspace entry point
(dlvm_softmax_xent, the same kernels): loss and dlogits bit for bit, on two
calls in a row whose second has fewer rows (the array keeps the first call's
contents), plus the label flags and the row limit."""
import numpy as np
import pytest

import paper_1711_03016_amd as dl
from helpers import device, to_dev

pytestmark = pytest.mark.gpu


def _inputs(rows, classes, seed):
    r = np.random.default_rng([77, rows, classes, seed])
    z = (r.standard_normal((rows, classes)) * 3).astype(np.float32)
    y = r.integers(0, classes, rows).astype(np.int32)
    return z, y


def _both(dtype, z, y):
    import torch
    rows, classes = z.shape
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    zd, yd = to_dev(z), torch.from_numpy(y).to(device())
    ws = torch.zeros(dl.softmax_xent_ws_bytes(rows), dtype=torch.uint8, device=device())
    d0 = torch.full((rows, classes), float("nan"), dtype=tdt, device=device())
    l0 = torch.full((1,), float("nan"), device=device())
    dl.softmax_xent(dtype, rows, classes, zd, yd, 1.0 / rows, d0, l0, ws)
    d1 = torch.full((rows, classes), float("nan"), dtype=tdt, device=device())
    l1 = torch.full((1,), float("nan"), device=device())
    flags = torch.full((4,), -1, dtype=torch.int32, device=device())
    dl.softmax_xent_noalloc(dtype, rows, classes, zd, yd, 1.0 / rows, d1, l1, flags)
    torch.cuda.synchronize()
    return (l0, d0), (l1, d1), flags.cpu().numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_noalloc_matches_workspace_entry_point(dtype):
    import torch
    # the second call has fewer rows: the static array still holds the first
    # call's partials beyond them, which must not leak into the loss
    for rows, classes in ((20000, 1000), (333, 10)):
        z, y = _inputs(rows, classes, 1)
        (l0, d0), (l1, d1), flags = _both(dtype, z, y)
        assert torch.equal(l1, l0), (rows, l1.item(), l0.item())
        assert torch.equal(d1, d0), rows
        assert flags[0] == 0 and flags[1] == 0 and flags[2] == -1
        assert np.isfinite(l1.item())


def test_noalloc_flags_and_limits():
    import torch
    z, y = _inputs(64, 10, 2)
    y[5] = 10
    (l0, _), (l1, _), flags = _both("f32", z, y)
    assert np.isnan(l1.item()) and np.isnan(l0.item())
    assert flags[0] == 1 and flags[1] == 1
    zd = to_dev(np.zeros((1, 4), np.float32))
    yd = torch.zeros(1, dtype=torch.int32, device=device())
    out = torch.empty((1, 4), device=device())
    loss = torch.empty(1, device=device())
    with pytest.raises(dl.DlvmError) as e:      # beyond the static scratch: refused on the host
        dl.softmax_xent_noalloc("f32", (1 << 20) + 1, 4, zd, yd, 1.0, out, loss)
    assert e.value.status == dl.ERR_INVALID_ARG
    # the largest batch it takes, with no flags output
    rows = 1 << 20
    z = torch.randn((rows, 4), device=device())
    yb = torch.randint(0, 4, (rows,), dtype=torch.int32, device=device())
    d = torch.empty((rows, 4), device=device())
    dl.softmax_xent_noalloc("f32", rows, 4, z, yb, 1.0 / rows, d, loss)
    ws = torch.zeros(dl.softmax_xent_ws_bytes(rows), dtype=torch.uint8, device=device())
    d0 = torch.empty_like(d)
    l0 = torch.empty(1, device=device())
    dl.softmax_xent("f32", rows, 4, z, yb, 1.0 / rows, d0, l0, ws)
    torch.cuda.synchronize()
    assert torch.equal(loss, l0) and torch.equal(d, d0)
