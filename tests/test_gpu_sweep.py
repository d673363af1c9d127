"""Seeded random sweeps through the C ABI and the KD / vocabulary-shard entry points.

The LCE sweeps draw shapes across tile and slab boundaries (one of them 40 shapes of any width, up
to 5000 tokens and 40000 ids) and, in the strided one, per case row strides on both H
and W whose padding columns hold NaN (a kernel that read them would poison the results), int32 or
int64 targets, an ignore_index that may lie inside [0, V), and a few out-of-range targets (the
device status bit and the ignored-row treatment are checked against the oracle). The KD and
shard sweeps draw shapes, temperatures, reductions and vocabulary cuts. Tolerances as elsewhere:
loss 1e-3 absolute (plus one fp32 spacing for a summed loss; per token for "none"), lse 1e-3,
relative Frobenius 1e-2 on the gradients.
"""
import numpy as np
import pytest

from oracle import kd_oracle as K
from oracle import lce_oracle as O
from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U
from tests.test_gpu_kd import _check as kd_check
from tests.test_gpu_kd import _run as kd_run
from tests.test_gpu_shard import _run_shards

pytestmark = pytest.mark.gpu

BF16_NAN = np.int16(0x7FC0)


def _padded(bits, ld):
    """bf16 rows of `bits` in a [rows, ld] device buffer whose extra columns hold NaN."""
    import torch
    rows, d = bits.shape
    buf = np.full((rows, ld), BF16_NAN, dtype=np.int16)
    buf[:, :d] = bits.view(np.int16)
    return torch.from_numpy(buf).view(torch.bfloat16).to("cuda:0")


@pytest.mark.parametrize("case", range(10))
def test_c_abi_strided_sweep(case):
    import torch
    from paper_2605_21442_amd import binding as B
    rng = np.random.default_rng(2000 + case)
    n = int(rng.integers(1, 700))
    d = int(rng.integers(1, 70)) * 8
    v = int(rng.choice([int(rng.integers(1, 700)), int(rng.integers(4000, 12000))]))
    ld_h = d + 8 * int(rng.integers(0, 5))
    ld_w = d + 8 * int(rng.integers(0, 5))
    wide = case % 2 == 1
    ignore = int(rng.choice([-100, -1, 0, v + 3]))
    reduction = ["mean", "sum", "none"][case % 3]
    inp = WL.custom(n, d, v, seed=case, mask_frac=float(rng.uniform(0, 0.4)), sigma_w=0.3, ignore_index=ignore,
                    case_id=50)
    t = inp.targets.astype(np.int64)
    for r in rng.choice(n, size=min(n, 3), replace=False):      # out-of-range targets
        if t[r] != ignore:
            t[r] = int(rng.choice([v, v + 7, -5]))
            if t[r] == ignore:
                t[r] = v + 11
    grad = rng.standard_normal(n).astype(np.float32) if reduction == "none" else np.float32([rng.uniform(0.2, 2)])
    print(f"sweep {case}: n={n} d={d} v={v} ld_h={ld_h} ld_w={ld_w} int64={wide} ignore={ignore} {reduction}",
          flush=True)

    dev = torch.device("cuda:0")
    h = _padded(inp.h_bits, ld_h)
    w = _padded(inp.w_bits, ld_w)
    tt = torch.from_numpy(t if wide else t.astype(np.int32)).to(dev)
    p = B.problem(n, d, v, ld_h=ld_h, ld_w=ld_w, ignore_index=ignore, reduction=reduction,
                  target_bytes=8 if wide else 4)
    fwd_b, bwd_b = B.lce_workspace_size(p)
    ws = torch.empty(max(fwd_b, bwd_b, 1), dtype=torch.uint8, device=dev)
    loss = torch.empty(n if reduction == "none" else 1, dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    g = torch.from_numpy(grad).to(dev)
    dh = torch.empty((n, d), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((v, d), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    B.lce_forward(p, h.data_ptr(), w.data_ptr(), tt.data_ptr(), loss.data_ptr(), lse.data_ptr(), nv.data_ptr(),
                  status.data_ptr(), ws.data_ptr(), fwd_b, stream)
    B.lce_backward(p, h.data_ptr(), w.data_ptr(), tt.data_ptr(), lse.data_ptr(), nv.data_ptr(), g.data_ptr(),
                   dh.data_ptr(), dw.data_ptr(), ws.data_ptr(), bwd_b, stream)
    torch.cuda.synchronize()
    gpu = dict(loss=(loss.cpu().numpy().astype(np.float64) if reduction == "none" else float(loss.item())),
               lse=lse.cpu().numpy().astype(np.float64), n_valid=int(nv.item()), status=int(status.item()),
               dH=dh.float().cpu().numpy().astype(np.float64), dW=dw.float().cpu().numpy().astype(np.float64))
    ref = O.lce(inp.h_bits, inp.w_bits, t, ignore, reduction,
                grad.astype(np.float64) if reduction == "none" else float(grad[0]))
    U.assert_parity(gpu, ref)
    assert ref["status"] == (1 if np.any((t != ignore) & ((t < 0) | (t >= v))) else 0)


@pytest.mark.parametrize("case", range(40))
def test_random_shape_sweep(case):
    # any hidden width that is a multiple of 8 (both tile forms), token counts from 1 to 5000,
    # vocabularies from 1 to 40000 ids, all three reductions, 0-60 % masked, three weight scales
    rng = np.random.default_rng([4000, case])
    while True:
        n = int(rng.integers(1, 5000))
        d = int(rng.integers(1, 129)) * 8
        v = int(rng.integers(1, 40000))
        if n * v * d <= 3e9:                      # the oracle finishes in well under a second
            break
    reduction = ["mean", "sum", "none"][case % 3]
    inp = WL.custom(n, d, v, seed=case, mask_frac=float(rng.uniform(0, 0.6)),
                    sigma_w=float(rng.choice([0.02, 0.3, 1.0])), case_id=52)
    grad = rng.standard_normal(n).astype(np.float32) if reduction == "none" else 1.0
    print(f"random sweep {case}: n={n} d={d} v={v} {reduction}", flush=True)
    h, w, t = U.to_device(inp)
    gpu = U.run_gpu(h, w, t, inp.ignore_index, reduction, grad)
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets, inp.ignore_index, reduction,
                grad.astype(np.float64) if reduction == "none" else 1.0)
    U.assert_parity(gpu, ref)


@pytest.mark.parametrize("case", range(6))
def test_many_token_tiles_sweep(case):
    # more token tiles than the strided sweep (8 to 17 of 256): the forward and G launches deal the
    # vocabulary tiles past the last multiple of 8 to the XCDs by token tile, and the dW and dH
    # launches cut their tiles into per-XCD shares of several rounds
    rng = np.random.default_rng(3000 + case)
    n = int(rng.integers(1800, 4300))
    d = int(rng.choice([64, 128, 192, 256]))
    v = int(rng.integers(5000, 30000))
    reduction = ["mean", "sum"][case % 2]
    inp = WL.custom(n, d, v, seed=case, mask_frac=float(rng.uniform(0, 0.4)), sigma_w=0.3, case_id=51)
    print(f"token-tile sweep {case}: n={n} d={d} v={v} {reduction}", flush=True)
    h, w, t = U.to_device(inp)
    gpu = U.run_gpu(h, w, t, inp.ignore_index, reduction, 1.0)
    U.assert_parity(gpu, O.lce(inp.h_bits, inp.w_bits, inp.targets, inp.ignore_index, reduction, 1.0))


@pytest.mark.parametrize("case", range(6))
def test_kd_random_sweep(case):
    rng = np.random.default_rng(3000 + case)
    n = int(rng.integers(1, 600))
    ds = int(rng.integers(1, 50)) * 8
    dt = int(rng.integers(1, 70)) * 8
    v = int(rng.choice([int(rng.integers(2, 600)), int(rng.integers(4000, 10000))]))
    temperature = float(rng.choice([0.5, 1.0, 2.0, 3.7]))
    reduction = ["mean", "sum", "none"][case % 3]
    inp = WL.kd_custom(n, ds, dt, v, seed=40 + case, mask_frac=float(rng.uniform(0, 0.4)))
    grad = rng.standard_normal(n).astype(np.float32) if reduction == "none" else np.float32([rng.uniform(0.2, 2)])
    print(f"kd sweep {case}: n={n} ds={ds} dt={dt} v={v} T={temperature} {reduction}", flush=True)
    gpu = kd_run(inp, temperature, reduction, grad)
    ref = K.kd_bits(inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits, inp.targets, temperature=temperature,
                    ignore_index=inp.ignore_index, reduction=reduction,
                    grad=grad.astype(np.float64) if reduction == "none" else float(grad[0]))
    kd_check(gpu, ref)


@pytest.mark.parametrize("case", range(6))
def test_shard_random_sweep(case):
    rng = np.random.default_rng(4000 + case)
    n = int(rng.integers(1, 600))
    d = int(rng.integers(1, 50)) * 8
    v = int(rng.integers(2, 9000))
    k = int(rng.integers(1, min(6, v)))
    cuts = [0] + sorted(int(c) for c in rng.choice(np.arange(1, v), size=k - 1, replace=False)) + [v] if k > 1 \
        else [0, v]
    reduction = ["mean", "sum", "none"][case % 3]
    inp = WL.custom(n, d, v, seed=70 + case, mask_frac=float(rng.uniform(0, 0.4)), sigma_w=0.3, case_id=51)
    grad = rng.standard_normal(n).astype(np.float32) if reduction == "none" else np.float32([rng.uniform(0.2, 2)])
    print(f"shard sweep {case}: n={n} d={d} v={v} cuts={cuts} {reduction}", flush=True)
    gpu = _run_shards(inp, cuts, reduction, grad)
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets, inp.ignore_index, reduction,
                grad.astype(np.float64) if reduction == "none" else float(grad[0]))
    U.assert_parity(gpu, ref)
