"""The dH launches that split the K range of each XCD's last, partial round on the device (and the
launch status check).

With T live 384 x 256 output tiles, XCD x takes a balanced share of them; the tail of its share
(fewer tiles than its 32 CUs) is split along K into up to 8 parts whose fp32 blocks live in the
accumulator rows past the valid ones, and the finalise adds them in order. These cases pick Nv so
that the tails take 8, 3 and 2 parts, and one case where the tails do not fit the free rows (no
split). dH is compared with the oracle on every 384 x 256 block of the compacted valid rows, so
that a missing or doubled part of a single tail tile fails, and the result is bitwise the same
run to run.
"""
import numpy as np
import pytest

from oracle import lce_oracle as O
from paper_2605_21442_amd import binding as B
from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U
from tests.test_bounds_cpu import dh_tail_parts

pytestmark = pytest.mark.gpu

V = 1000


def _inputs(n, d, nv, seed):
    rng = np.random.default_rng([seed, n, d, nv])
    t = np.full(n, -100, dtype=np.int32)
    valid = np.sort(rng.choice(n, size=nv, replace=False))
    t[valid] = rng.integers(0, V, size=nv, dtype=np.int32)
    return WL.custom(n, d, V, seed=seed, sigma_w=0.3, target_override=t), valid


@pytest.mark.parametrize("n,d,nv,parts", [(12288, 2048, 300, 8), (12288, 2048, 1400, 8), (12288, 2048, 3686, 3),
                                          (12288, 2048, 4423, 2), (8192, 4096, 6209, 1)])
def test_dh_with_split_tails_matches_the_oracle_blockwise(n, d, nv, parts):
    info = B.lce_plan_info(B.problem(n, d, V))
    assert info["dh_kz"] == 1                      # the host did not split these launches
    split = dh_tail_parts(nv, d, info["rows_g"])
    assert max((p[3] for p in split), default=1) == parts
    inp, valid = _inputs(n, d, nv, seed=3)
    h, w, t = U.to_device(inp)
    print(f"case n={n} d={d} nv={nv} tail parts={parts}", flush=True)
    gpu = U.run_gpu(h, w, t, inp.ignore_index, "mean", 1.0)
    again = U.run_gpu(h, w, t, inp.ignore_index, "mean", 1.0)
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets, inp.ignore_index, "mean", 1.0)
    U.assert_parity(gpu, ref)
    assert np.array_equal(gpu["dH"], again["dH"]), "dH differs between two runs"
    dh, dh_ref = gpu["dH"][valid], ref["dH"][valid]
    for m0 in range(0, nv, 384):
        for d0 in range(0, d, 256):
            blk, rb = dh[m0:m0 + 384, d0:d0 + 256], dh_ref[m0:m0 + 384, d0:d0 + 256]
            e = np.linalg.norm(blk - rb) / np.linalg.norm(rb)
            assert e <= U.GRAD_REL_TOL, (m0, d0, e)
    assert np.all(gpu["dH"][inp.targets == inp.ignore_index] == 0.0)


def test_a_stale_hip_error_of_another_call_neither_fails_the_launches_nor_is_consumed():
    # a failed runtime call earlier on the thread leaves its status in HIP's last-error slot: the
    # library's launches report only their own status and leave that slot to its owner
    import ctypes
    import torch
    inp = WL.custom(300, 264, 1000, seed=1, sigma_w=0.3)
    h, w, t = U.to_device(inp)
    n, d, v = 300, 264, 1000
    p = B.problem(n, d, v, ignore_index=inp.ignore_index, reduction="mean", target_bytes=4)
    fb, bb = B.lce_workspace_size(p)
    dev = h.device
    ws = torch.empty(max(fb, bb), dtype=torch.uint8, device=dev)
    loss = torch.empty((), dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    st = torch.empty(1, dtype=torch.int32, device=dev)
    grad = torch.ones(1, dtype=torch.float32, device=dev)
    dh = torch.empty((n, d), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((v, d), dtype=torch.bfloat16, device=dev)
    s = torch.cuda.current_stream(dev).cuda_stream
    torch.cuda.synchronize()
    # the HIP runtime already in the process (torch's, which the library also uses)
    maps = open("/proc/self/maps").read()
    path = sorted({l.split()[-1] for l in maps.splitlines() if "libamdhip64" in l})
    assert len(path) == 1, path
    hip = ctypes.CDLL(path[0])
    bad = hip.hipSetDevice(ctypes.c_int(1 << 20))           # invalid device: an error, no effect
    assert bad != 0
    B.lce_forward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), loss.data_ptr(), lse.data_ptr(), nv.data_ptr(),
                  st.data_ptr(), ws.data_ptr(), fb, s)
    B.lce_backward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse.data_ptr(), nv.data_ptr(), grad.data_ptr(),
                   dh.data_ptr(), dw.data_ptr(), ws.data_ptr(), bb, s)
    assert hip.hipGetLastError() == bad                       # still there for its owner (and now cleared)
    torch.cuda.synchronize()
    gpu = {"loss": float(loss.item()), "lse": lse.cpu().numpy().astype(np.float64), "n_valid": int(nv.item()),
           "status": int(st.item()), "dH": dh.float().cpu().numpy().astype(np.float64),
           "dW": dw.float().cpu().numpy().astype(np.float64)}
    U.assert_parity(gpu, O.lce(inp.h_bits, inp.w_bits, inp.targets, inp.ignore_index, "mean", 1.0))


def test_vocabulary_shards_with_split_tails_reproduce_the_oracle():
    # the shard backward returns fp32 dH terms through the same finalise, here with tail parts
    from tests.test_gpu_shard import _run_shards
    n, d, nv = 12288, 2048, 1400
    info = B.lce_plan_info(B.problem(n, d, 500))
    assert info["dh_kz"] == 1 and dh_tail_parts(nv, d, info["rows_g"])
    inp, valid = _inputs(n, d, nv, seed=5)
    gpu = _run_shards(inp, [0, 500, V])
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets, inp.ignore_index, "mean", 1.0)
    U.assert_parity(gpu, ref)
    for m0 in range(0, nv, 384):
        blk, rb = gpu["dH"][valid][m0:m0 + 384], ref["dH"][valid][m0:m0 + 384]
        assert np.linalg.norm(blk - rb) / np.linalg.norm(rb) <= U.GRAD_REL_TOL, m0
