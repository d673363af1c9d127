"""The library's calls only enqueue kernels (no allocation, no memset, no host synchronisation),
so a forward/backward pair can be captured in a HIP graph. Each replay must give the same bits as
the eager calls, also with other GPU work and synchronisations between replays."""
import numpy as np
import pytest

from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U

pytestmark = pytest.mark.gpu


def _bits(x):
    import torch
    return x.contiguous().view(torch.uint8).cpu().numpy().copy()


@pytest.mark.parametrize("reuse", [False, True])
def test_lce_forward_backward_graph_replays_match_eager(reuse):
    import torch
    from paper_2605_21442_amd import binding as B
    inp = WL.custom(600, 128, 9000, seed=12, mask_frac=0.2, sigma_w=0.3)
    h, w, t = U.to_device(inp)
    n, d = h.shape
    v = w.shape[0]
    p = B.problem(n, d, v)
    # the backward may take the forward's valid-row list and gathered rows from the workspace
    pb = B.problem(n, d, v, flags=B.LCE_FLAG_REUSE_FORWARD if reuse else 0)
    fwd_bytes, bwd_bytes = B.lce_workspace_size(p)
    dev = h.device
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    grad = torch.full((1,), 0.5, dtype=torch.float32, device=dev)
    dh = torch.empty((n, d), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((v, d), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(max(fwd_bytes, bwd_bytes), dtype=torch.uint8, device=dev)
    outs = (loss, lse, nv, status, dh, dw)

    def step():
        s = torch.cuda.current_stream().cuda_stream
        B.lce_forward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), loss.data_ptr(), lse.data_ptr(), nv.data_ptr(),
                      status.data_ptr(), ws.data_ptr(), fwd_bytes, s)
        B.lce_backward(pb, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse.data_ptr(), nv.data_ptr(), grad.data_ptr(),
                       dh.data_ptr(), dw.data_ptr(), ws.data_ptr(), bwd_bytes, s)

    step()
    torch.cuda.synchronize()
    ref = [_bits(x) for x in outs]
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()                                         # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        for x in outs:
            x.view(torch.uint8).fill_(0xA5)            # poison, with a fill kernel
        _ = (torch.randn(2048, 2048, device=dev) @ torch.randn(2048, 2048, device=dev)).sum().item()
        g.replay()
        torch.cuda.synchronize()
        for k, (x, r) in enumerate(zip(outs, ref)):
            assert np.array_equal(_bits(x), r), (rep, k)


def test_kd_forward_backward_graph_replays_match_eager():
    import torch
    from paper_2605_21442_amd import binding as B
    inp = WL.kd_custom(300, 64, 96, 2000, seed=2)
    to = lambda b: torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).view(torch.bfloat16).to("cuda:0")
    hs, ws_, ht, wt = to(inp.hs_bits), to(inp.ws_bits), to(inp.ht_bits), to(inp.wt_bits)
    t = torch.from_numpy(inp.targets).to("cuda:0")
    n, ds = hs.shape
    v, dt = wt.shape[0], ht.shape[1]
    p = B.kd_problem(n, ds, dt, v, temperature=2.0)
    fwd_bytes, bwd_bytes = B.lce_kd_workspace_size(p)
    dev = hs.device
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    lse_s = torch.empty(n, dtype=torch.float32, device=dev)
    lse_t = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    grad = torch.ones(1, dtype=torch.float32, device=dev)
    dh = torch.empty((n, ds), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((v, ds), dtype=torch.bfloat16, device=dev)
    wsp = torch.empty(max(fwd_bytes, bwd_bytes), dtype=torch.uint8, device=dev)
    outs = (loss, lse_s, lse_t, nv, dh, dw)

    def step():
        s = torch.cuda.current_stream().cuda_stream
        B.lce_kd_forward(p, hs.data_ptr(), ws_.data_ptr(), ht.data_ptr(), wt.data_ptr(), t.data_ptr(),
                         loss.data_ptr(), lse_s.data_ptr(), lse_t.data_ptr(), nv.data_ptr(), status.data_ptr(),
                         wsp.data_ptr(), fwd_bytes, s)
        B.lce_kd_backward(p, hs.data_ptr(), ws_.data_ptr(), ht.data_ptr(), wt.data_ptr(), t.data_ptr(),
                          lse_s.data_ptr(), lse_t.data_ptr(), nv.data_ptr(), grad.data_ptr(), dh.data_ptr(),
                          dw.data_ptr(), wsp.data_ptr(), bwd_bytes, s)

    step()
    torch.cuda.synchronize()
    ref = [_bits(x) for x in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        for x in outs:
            x.view(torch.uint8).fill_(0x5A)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, (x, r) in enumerate(zip(outs, ref)):
            assert np.array_equal(_bits(x), r), (rep, k)
