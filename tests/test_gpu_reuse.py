"""The backward with LCE_FLAG_REUSE_FORWARD (it takes the valid-row list and gathered rows of H that
the preceding forward left in the shared workspace) gives the same bits as the backward that forms
them itself, for the plain, vocabulary-shard and in-backward AdamW calls, at widths where the
forward gathers the rows (D % 64 == 0) and where it does not."""
import numpy as np
import pytest

from oracle import lce_oracle as O
from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U

pytestmark = pytest.mark.gpu


def _bits(x):
    return x.contiguous().view(__import__("torch").uint8).cpu().numpy().copy()


def _run(inp, reuse, reduction="mean"):
    import torch
    from paper_2605_21442_amd import binding as B
    h, w, t = U.to_device(inp)
    n, d = h.shape
    v = w.shape[0]
    p = B.problem(n, d, v, reduction=reduction)
    pb = B.problem(n, d, v, reduction=reduction, flags=B.LCE_FLAG_REUSE_FORWARD if reuse else 0)
    fb, bb = B.lce_workspace_size(p)
    dev = h.device
    loss = torch.empty(n if reduction == "none" else 1, dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    st = torch.empty(1, dtype=torch.int32, device=dev)
    g = torch.full((n if reduction == "none" else 1,), 0.75, dtype=torch.float32, device=dev)
    dh = torch.empty((n, d), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((v, d), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(max(fb, bb), dtype=torch.uint8, device=dev)
    s = torch.cuda.current_stream().cuda_stream
    B.lce_forward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), loss.data_ptr(), lse.data_ptr(), nv.data_ptr(),
                  st.data_ptr(), ws.data_ptr(), fb, s)
    if not reuse:
        ws.fill_(0xFF)          # nothing of the forward's survives: the backward forms everything itself
    B.lce_backward(pb, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse.data_ptr(), nv.data_ptr(), g.data_ptr(),
                   dh.data_ptr(), dw.data_ptr(), ws.data_ptr(), bb, s)
    torch.cuda.synchronize()
    return _bits(dh), _bits(dw), dh.float().cpu().numpy(), dw.float().cpu().numpy()


@pytest.mark.parametrize("n,d,v,mask", [(700, 128, 5000, 0.2), (300, 264, 1000, 0.15), (520, 64, 40000, 0.3),
                                        (257, 72, 3000, 0.0), (64, 64, 800, 1.0), (1, 8, 5, 0.0)])
def test_reuse_gives_the_bits_of_the_full_backward(n, d, v, mask):
    inp = WL.custom(n, d, v, seed=n + d, mask_frac=mask, sigma_w=0.3)
    print(f"case n={n} d={d} v={v} mask={mask}", flush=True)
    a = _run(inp, reuse=True)
    b = _run(inp, reuse=False)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets, grad=0.75)
    if mask < 1.0:
        assert U.rel_fro(a[2], ref["dH"]) <= U.GRAD_REL_TOL and U.rel_fro(a[3], ref["dW"]) <= U.GRAD_REL_TOL
    else:
        assert np.all(a[2] == 0) and np.all(a[3] == 0)


def test_reuse_with_per_token_reduction():
    inp = WL.custom(400, 128, 3000, seed=5, mask_frac=0.25, sigma_w=0.3)
    a = _run(inp, reuse=True, reduction="none")
    b = _run(inp, reuse=False, reduction="none")
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_reuse_in_the_shard_calls():
    import torch
    from paper_2605_21442_amd import binding as B
    inp = WL.custom(600, 128, 7000, seed=9, mask_frac=0.2, sigma_w=0.3)
    h, w, t = U.to_device(inp)
    n, d = h.shape
    v = w.shape[0]
    lo, hi = 2000, 5000
    ws_ = w[lo:hi].contiguous()
    out = []
    for reuse in (True, False):
        p = B.problem(n, d, hi - lo)
        pf = B.problem(n, d, v)
        pb = B.problem(n, d, hi - lo, flags=B.LCE_FLAG_REUSE_FORWARD if reuse else 0)
        fb, bb = B.lce_workspace_size(p)
        cb, _ = B.lce_workspace_size(pf)
        ws = torch.empty(max(fb, bb, cb), dtype=torch.uint8, device=h.device)
        sh = B.LceShard(v, lo)
        lp = torch.empty(n, dtype=torch.float32, device=h.device)
        tp = torch.empty(n, dtype=torch.float32, device=h.device)
        nv = torch.empty(1, dtype=torch.int32, device=h.device)
        st = torch.empty(1, dtype=torch.int32, device=h.device)
        s = torch.cuda.current_stream().cuda_stream
        B.lce_forward_shard(p, sh, h.data_ptr(), ws_.data_ptr(), t.data_ptr(), lp.data_ptr(), tp.data_ptr(),
                            nv.data_ptr(), st.data_ptr(), ws.data_ptr(), fb, s)
        # one shard stands in for all: the combine of one row gives this shard's own lse
        loss = torch.empty(1, dtype=torch.float32, device=h.device)
        lse = torch.empty(n, dtype=torch.float32, device=h.device)
        B.lce_combine_shards(pf, 1, lp.data_ptr(), tp.data_ptr(), t.data_ptr(), loss.data_ptr(), lse.data_ptr(),
                             nv.data_ptr(), st.data_ptr(), ws.data_ptr(), cb, s)
        if not reuse:
            ws.fill_(0xFF)
        g = torch.ones(1, dtype=torch.float32, device=h.device)
        dhp = torch.empty((n, d), dtype=torch.float32, device=h.device)
        dw = torch.empty((hi - lo, d), dtype=torch.bfloat16, device=h.device)
        B.lce_backward_shard(pb, sh, h.data_ptr(), ws_.data_ptr(), t.data_ptr(), lse.data_ptr(), nv.data_ptr(),
                             g.data_ptr(), dhp.data_ptr(), dw.data_ptr(), ws.data_ptr(), bb, s)
        torch.cuda.synchronize()
        out.append((_bits(dhp), _bits(dw)))
    assert np.array_equal(out[0][0], out[1][0]) and np.array_equal(out[0][1], out[1][1])


def test_reuse_in_the_fused_adamw_backward():
    import torch
    from paper_2605_21442_amd import autograd as A
    inp = WL.custom(500, 128, 4000, seed=21, mask_frac=0.2, sigma_w=0.3)
    h, w, t = U.to_device(inp)
    res = []
    for reuse in (True, False):
        w1 = w.clone()
        state = A.AdamWState(w1, lr=1e-2, master_weights=True)
        loss, lse, nv, _, ws = A.forward(h, w1, t, keep_workspace=True)
        g = torch.ones(1, dtype=torch.float32, device=h.device)
        dh = A.backward_adamw(h, t, lse, nv, g, state, workspace=ws if reuse else None)
        torch.cuda.synchronize()
        res.append((_bits(dh), _bits(w1), _bits(state.exp_avg), _bits(state.master)))
    for x, y in zip(*res):
        assert np.array_equal(x, y)
