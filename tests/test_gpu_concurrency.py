"""Calls are reentrant: two independent problems run at the same time on two streams (each with
its own workspace), from one host thread and from two host threads, and each gives the same bits
as when it runs alone. Both streams keep the default priority."""
import threading

import numpy as np
import pytest

from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U

pytestmark = pytest.mark.gpu


def _bits(x):
    import torch
    return x.contiguous().view(torch.uint8).cpu().numpy().copy()


class _Job:
    def __init__(self, n, d, v, seed):
        import torch
        from paper_2605_21442_amd import binding as B
        self.B = B
        inp = WL.custom(n, d, v, seed=seed, mask_frac=0.2, sigma_w=0.3, case_id=60 + seed)
        self.h, self.w, self.t = U.to_device(inp)
        dev = self.h.device
        self.p = B.problem(n, d, v)
        self.fb, self.bb = B.lce_workspace_size(self.p)
        self.ws = torch.empty(max(self.fb, self.bb), dtype=torch.uint8, device=dev)
        self.loss = torch.empty(1, dtype=torch.float32, device=dev)
        self.lse = torch.empty(n, dtype=torch.float32, device=dev)
        self.nv = torch.empty(1, dtype=torch.int32, device=dev)
        self.status = torch.empty(1, dtype=torch.int32, device=dev)
        self.grad = torch.full((1,), 0.75, dtype=torch.float32, device=dev)
        self.dh = torch.empty((n, d), dtype=torch.bfloat16, device=dev)
        self.dw = torch.empty((v, d), dtype=torch.bfloat16, device=dev)

    def enqueue(self, stream):
        B = self.B
        s = stream.cuda_stream
        B.lce_forward(self.p, self.h.data_ptr(), self.w.data_ptr(), self.t.data_ptr(), self.loss.data_ptr(),
                      self.lse.data_ptr(), self.nv.data_ptr(), self.status.data_ptr(), self.ws.data_ptr(), self.fb, s)
        B.lce_backward(self.p, self.h.data_ptr(), self.w.data_ptr(), self.t.data_ptr(), self.lse.data_ptr(),
                       self.nv.data_ptr(), self.grad.data_ptr(), self.dh.data_ptr(), self.dw.data_ptr(),
                       self.ws.data_ptr(), self.bb, s)

    def outputs(self):
        return [_bits(x) for x in (self.loss, self.lse, self.nv, self.status, self.dh, self.dw)]

    def clear(self):
        for x in (self.loss, self.lse, self.nv, self.status, self.dh, self.dw):
            x.zero_()


def _same(a, b):
    return all(np.array_equal(x, y) for x, y in zip(a, b))


@pytest.mark.parametrize("threads", [False, True])
def test_two_streams_at_once_match_each_job_alone(threads):
    import torch
    jobs = [_Job(700, 136, 9000, 1), _Job(513, 264, 4097, 2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    alone = []
    for j, s in zip(jobs, streams):
        j.enqueue(s)
        torch.cuda.synchronize()
        alone.append(j.outputs())
    for rep in range(3):
        for j in jobs:
            j.clear()
        torch.cuda.synchronize()
        if threads:
            ts = [threading.Thread(target=j.enqueue, args=(s,)) for j, s in zip(jobs, streams)]
            for th in ts:
                th.start()
            for th in ts:
                th.join()
        else:
            for j, s in zip(jobs, streams):
                j.enqueue(s)
        torch.cuda.synchronize()
        for k, j in enumerate(jobs):
            assert _same(j.outputs(), alone[k]), (rep, k)
