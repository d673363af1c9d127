"""lce_forward_noalloc (workspace in the library's own device array, nothing allocated by the call)
gives lce_forward's bits, on two calls in a row of which the second is smaller, and a third, larger
call after them; the oracle holds both to the method's tolerances."""
import numpy as np
import pytest

from oracle import lce_oracle as O
from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U

pytestmark = pytest.mark.gpu


def _outs(n, dev):
    import torch
    return (torch.full((1,), float("nan"), dtype=torch.float32, device=dev),
            torch.full((n,), float("nan"), dtype=torch.float32, device=dev),
            torch.full((1,), -1, dtype=torch.int32, device=dev), torch.full((1,), -1, dtype=torch.int32, device=dev))


def _both(inp):
    import torch
    from paper_2605_21442_amd import binding as B
    h, w, t = U.to_device(inp)
    n, d = h.shape
    v = w.shape[0]
    p = B.problem(n, d, v)
    fb, _ = B.lce_workspace_size(p)
    assert fb <= B.LCE_NOALLOC_SCRATCH_BYTES
    s = torch.cuda.current_stream().cuda_stream
    a = _outs(n, h.device)
    before = torch.cuda.memory_allocated()
    B.lce_forward_noalloc(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), *[x.data_ptr() for x in a], s)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == before
    b = _outs(n, h.device)
    ws = torch.empty(fb, dtype=torch.uint8, device=h.device)
    B.lce_forward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), *[x.data_ptr() for x in b], ws.data_ptr(), fb, s)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets)
    assert abs(float(a[0].item()) - ref["loss"]) <= U.LOSS_ABS_TOL
    assert np.max(np.abs(a[1].cpu().numpy() - ref["lse"])) <= U.LSE_ABS_TOL
    assert int(a[2].item()) == ref["n_valid"]


def test_two_calls_in_a_row_the_second_smaller_then_a_larger_one():
    print("case noalloc 2000x1024x40000, then 300x264x1000, then 4096x512x60000", flush=True)
    _both(WL.custom(2000, 1024, 40000, seed=31, mask_frac=0.2, sigma_w=0.1))
    _both(WL.custom(300, 264, 1000, seed=32, mask_frac=0.15, sigma_w=0.3))
    _both(WL.custom(4096, 512, 60000, seed=33, mask_frac=0.25, sigma_w=0.1))


def test_problem_beyond_the_array_is_rejected_before_any_launch():
    import torch
    from paper_2605_21442_amd import binding as B
    p = B.problem(32768, 3584, 152064)
    assert B.lce_workspace_size(p)[0] > B.LCE_NOALLOC_SCRATCH_BYTES
    with pytest.raises(B.LceError) as e:
        B.lce_forward_noalloc(p, 16, 16, 16, 16, 16, 16, 0, torch.cuda.current_stream().cuda_stream)
    assert e.value.code == B.LCE_ERR_WORKSPACE


def test_the_largest_workspace_the_array_holds():
    # the Llama-3.1-8B head: its 170 MiB forward workspace fits the 256 MiB array; bits as lce_forward
    import torch
    from paper_2605_21442_amd import binding as B
    n, d, v = 16384, 4096, 128256
    print(f"case noalloc {n}x{d}x{v}", flush=True)
    g = torch.Generator(device="cuda:0").manual_seed(5)
    h = torch.randn(n, d, device="cuda:0", generator=g).to(torch.bfloat16)
    w = (0.02 * torch.randn(v, d, device="cuda:0", generator=g)).to(torch.bfloat16)
    t = torch.randint(0, v, (n,), device="cuda:0", generator=g, dtype=torch.int32)
    t[::4] = -100
    p = B.problem(n, d, v)
    fb, _ = B.lce_workspace_size(p)
    s = torch.cuda.current_stream().cuda_stream
    a, b = _outs(n, h.device), _outs(n, h.device)
    B.lce_forward_noalloc(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), *[x.data_ptr() for x in a], s)
    ws = torch.empty(fb, dtype=torch.uint8, device=h.device)
    B.lce_forward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), *[x.data_ptr() for x in b], ws.data_ptr(), fb, s)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))
    assert int(a[2].item()) == n - n // 4
