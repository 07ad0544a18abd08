"""wise_select_support_noalloc (selection on the library's own per-device
scratch array, for callers that cannot allocate) against
wise_select_support with a caller workspace, through the C ABI: identical
row_ptr, col_idx and row order, bit for bit, and both equal to the oracle's
selection of the same host fp32 masses.  Two calls in a row, the second on a
smaller input, so the second runs over the first call's leftover scratch
contents; then a size past the scratch limit is refused."""

import numpy as np
import pytest
import torch

from oracle import wise_oracle as O
from parity_util import say, synthetic_masses

pytestmark = pytest.mark.gpu


def run_both(w, shape, acc_host, tau, flags):
    acc = torch.from_numpy(acc_host).cuda()
    ref = w.Schedule(shape)
    ref.select(acc, tau, flags)
    rows = ref.row_ptr.numel() - 1
    row_ptr = torch.full((rows + 1,), -7, dtype=torch.int32, device="cuda")
    col_idx = torch.full((ref.col_idx.numel(),), -7, dtype=torch.int32, device="cuda")
    order = torch.full((rows,), -7, dtype=torch.int32, device="cuda")
    w.wise_select_support_noalloc(shape, acc, tau, flags, row_ptr, col_idx, order)
    torch.cuda.synchronize()
    nnz = int(ref.row_ptr[-1].item())
    assert torch.equal(row_ptr, ref.row_ptr), "row_ptr"
    assert torch.equal(col_idx[:nnz], ref.col_idx[:nnz]), "col_idx"
    assert torch.equal(order, ref.row_order), "row_order"
    rp_o, ci_o = O.select_support(acc_host.astype(np.float64), tau, flags)
    nb = acc_host.shape[-1]
    assert np.array_equal(row_ptr.cpu().numpy(), rp_o)
    assert np.array_equal(col_idx[:nnz].cpu().numpy(), ci_o)
    assert np.array_equal(order.cpu().numpy(), O.schedule_order(rp_o, nb))
    return rows, nnz


def test_noalloc_matches_workspace_entry_point(gpu_lib):
    w = gpu_lib
    # first call: the 220-head, 32-key-block geometry (28160 rows of up to
    # 128 blocks, 0.56 MiB of the 4 MiB scratch); second call: a smaller one
    cases = [((1, 220, 4096, 96, 32), 0.95, 3), ((2, 3, 1024, 64, 64), 0.8, 1)]
    for i, ((bt, h, n, d, B), tau, flags) in enumerate(cases):
        shape = w.make_shape(bt, h, n, d, B)
        nb = n // B
        acc_host = synthetic_masses((bt, h, nb, nb), seed=40 + i)
        tau = float(np.float32(tau))
        rows, nnz = run_both(w, shape, acc_host, tau, flags)
        say(f"noalloc call {i + 1}: {rows} rows, nnz {nnz}, scratch need "
            f"{w.wise_select_workspace_bytes(shape)} bytes: bit-exact")


def test_noalloc_refuses_sizes_past_the_scratch(gpu_lib):
    w = gpu_lib
    # 16 x 64 heads x 1024 blocks: 1024 rows per head, 16 mask words each
    shape = w.make_shape(16, 64, 1024 * 32, 64, 32)
    assert w.wise_select_workspace_bytes(shape) > w.NOALLOC_SCRATCH_BYTES
    dummy = torch.empty(256, dtype=torch.int32, device="cuda")
    status = w._lib().wise_select_support_noalloc(
        w.ctypes.byref(shape), w.ctypes.c_void_p(dummy.data_ptr()), w.ctypes.c_float(0.9),
        w.ctypes.c_uint32(3), w.ctypes.c_void_p(dummy.data_ptr()),
        w.ctypes.c_void_p(dummy.data_ptr()), None, None)
    assert status == 5, status        # WISE_ERR_WORKSPACE, nothing launched
