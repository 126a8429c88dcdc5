"""rac_recon_error_noalloc (the allocation-free variant of the error
reduction) against rac_recon_error with a caller workspace, through the C
ABI: bit-identical sums on two calls in a row, the second one smaller (so a
larger earlier call's partials left in the library's array must not leak in),
then again after the workspace variant ran in between; sizes beyond the
array's capacity are rejected before any launch."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

import paper_2608_04991_amd as rac
from paper_2608_04991_amd import workloads as wl
from tests.gpu_util import say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    L = rac.library()
    L.rac_recon_error_noalloc.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    L.rac_recon_error_noalloc.restype = ctypes.c_int
    return L


def _inputs(T, d, seed, bf16=False):
    import torch
    xb, rb, _ = wl.prefill_uplink(seed, rows=(0, T), hidden=d)
    flags = rac.RAC_FLAG_XHAT_BF16 if bf16 else 0
    cfg = rac.RacConfig(T, d, 128, 128, 4, 8, flags)
    x = to_dev(xb)
    xh = torch.empty((T, d), dtype=torch.int16 if bf16 else torch.float32, device="cuda")
    w = torch.empty(rac.rac_wire_size(cfg), dtype=torch.uint8, device="cuda")
    rac.rac_encode(cfg, x, to_dev(rb), None, w, xh)
    return x, xh, flags


def _with_workspace(T, d, x, xh, flags):
    import torch
    st = torch.full((3,), -7.0, dtype=torch.float64, device="cuda")
    ws = torch.full((max(rac.rac_recon_error_workspace(T), 8),), 0x7F, dtype=torch.uint8, device="cuda")
    rac.rac_recon_error(T, d, x, xh, st, ws, flags)
    torch.cuda.synchronize()
    return st.cpu().numpy()


def _noalloc(lib, T, d, x, xh, flags):
    import torch
    st = torch.full((3,), -7.0, dtype=torch.float64, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    assert lib.rac_recon_error_noalloc(T, d, flags, x.data_ptr(), xh.data_ptr(), st.data_ptr(), s) == 0
    torch.cuda.synchronize()
    return st.cpu().numpy()


def test_noalloc_matches_the_workspace_call_on_two_calls_in_a_row(lib):
    big = (4096, 4096, 0, False)
    small = (37, 1024, 1, True)
    runs = []
    for T, d, seed, bf16 in (big, small, big, small):
        say(f"[gpu] noalloc error reduction {T}x{d} bf16={bf16}")
        x, xh, flags = _inputs(T, d, seed, bf16)
        a = _noalloc(lib, T, d, x, xh, flags)
        b = _with_workspace(T, d, x, xh, flags)
        assert np.array_equal(a.view(np.uint64), b.view(np.uint64)), (T, a, b)
        assert a[0] > 0 and a[1] > 0 and a[2] > 0
        runs.append(a)
    assert np.array_equal(runs[0], runs[2]) and np.array_equal(runs[1], runs[3])


def test_noalloc_rejects_sizes_beyond_its_array(lib):
    # 131072 rows fit (16384 partials of 8 rows); one more does not; the
    # rejection comes before anything touches the pointers
    fake = 1 << 40
    assert lib.rac_recon_error_noalloc(131073, 64, 0, fake, fake, fake, 0) == 3
    assert lib.rac_recon_error_noalloc(16, 60, 0, fake, fake, fake, 0) == 1
