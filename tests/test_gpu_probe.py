"""The row-gather measurement aid (libcold_probe.so) on the GPU: every row
of its output is the indexed table row, bit for bit, with indices outside
the table reading row 0, over counts that leave a partial last workgroup
(two threads per row, 128 rows per workgroup)."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def _probe():
    from paper_2007_16122_amd import build as hip_build
    L = ctypes.CDLL(hip_build.PROBE_LIB)
    f = L.cold_probe_row_gather
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                  ctypes.c_void_p]
    return f


@pytest.mark.parametrize("n", [1, 3, 128, 1021, 128 * 24 + 5])
def test_probe_rows_equal_the_indexed_rows(n):
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(1234 + n)
    rows = 5000
    table = torch.from_numpy(rng.integers(-2**31, 2**31, size=(rows, 8), dtype=np.int64)
                             .astype(np.int32)).to(dev)
    idx_np = rng.integers(-3, rows + 3, size=n).astype(np.int64)
    idx = torch.from_numpy(idx_np).to(dev)
    out = torch.full((n, 8), 7, dtype=torch.int32, device=dev)
    print(f"probe n={n}", flush=True)
    rc = _probe()(table.data_ptr(), rows, idx.data_ptr(), out.data_ptr(), n,
                  torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert rc == 0
    want_idx = np.where((idx_np >= 0) & (idx_np < rows), idx_np, 0)
    assert np.array_equal(out.cpu().numpy(), table.cpu().numpy()[want_idx])
