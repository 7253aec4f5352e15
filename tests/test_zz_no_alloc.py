"""The allocation-free time-gradient entry point against the workspace one, through the C ABI.

mtgnn_build_messages_bwd_noalloc runs the kernels of mtgnn_build_messages_bwd with the library's device
scratch in place of a caller workspace, so its sums must equal that call's bit for bit: checked on two
calls in a row, the second with fewer rows (the scratch keeps the first call's partials), with the row
count both on the device and as the host maximum, and with the size limit rejected before any launch.
"""

import numpy as np
import pytest
import torch

from paper_2608_16305_amd import mtgnn as M
from tests._gpu import log, needs_gpu

pytestmark = [pytest.mark.gpu, needs_gpu]


def _case(rows, d_time, seed):
    g = torch.Generator().manual_seed(seed)
    dphi = torch.randn(rows, d_time, generator=g).cuda()
    dt = (torch.rand(rows, generator=g) * 1e4).cuda()
    tw = (10.0 ** (-9.0 * torch.arange(d_time) / max(d_time - 1, 1))).float().cuda()
    tb = (torch.rand(d_time, generator=g) * 2 - 1).cuda()
    start_w = torch.randn(d_time, generator=g).cuda()
    start_b = torch.randn(d_time, generator=g).cuda()
    return dphi, dt, tw, tb, start_w, start_b


def _both(d, dphi, dt, n_rows, max_rows, tw, tb, start_w, start_b):
    ws = M.alloc_bytes(M.workspace_bytes(M.OP_BUILD_MESSAGES_BWD, d, max_rows, 0))
    gw_ref, gb_ref = start_w.clone(), start_b.clone()
    M.mtgnn_build_messages_bwd(dphi, dt, n_rows, max_rows, tw, tb, d, gw_ref, gb_ref, ws)
    gw, gb = start_w.clone(), start_b.clone()
    M.mtgnn_build_messages_bwd_noalloc(dphi, dt, n_rows, max_rows, tw, tb, d, gw, gb)
    torch.cuda.synchronize()
    return (gw_ref.cpu().numpy(), gb_ref.cpu().numpy()), (gw.cpu().numpy(), gb.cpu().numpy())


def test_noalloc_time_gradient_equals_workspace_call():
    d_time = 100
    d = M.dims(1000, 100, d_time, 0, 100, 2, 10, M.F32)
    log("[noalloc] two calls in a row: 120,000 rows, then 7,001 of a 50,000-row maximum (device count)")
    for rows, n_dev, seed in ((120_000, None, 1), (50_000, 7_001, 2)):
        dphi, dt, tw, tb, sw, sb = _case(rows, d_time, seed)
        n_rows = torch.tensor([n_dev], dtype=torch.int32, device="cuda") if n_dev is not None else None
        ref, got = _both(d, dphi, dt, n_rows, rows, tw, tb, sw, sb)
        for a, b in zip(ref, got):
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
        assert np.abs(ref[0] - sw.cpu().numpy()).max() > 0   # the call accumulated something


def test_noalloc_rejects_requests_beyond_the_scratch():
    d = M.dims(1000, 100, 100, 0, 100, 2, 10, M.F32)
    x = torch.zeros(8, 100, device="cuda")
    v = torch.zeros(100, device="cuda")
    with pytest.raises(M.MtgnnError, match="workspace too small"):
        M.mtgnn_build_messages_bwd_noalloc(x, torch.zeros(8, device="cuda"), None, 200_000, v, v, d, v, v)
