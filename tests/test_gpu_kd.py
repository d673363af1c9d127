"""Fused linear knowledge-distillation loss on the GPU against the CPU oracle.

Student and teacher heads of different hidden sizes over one vocabulary, ragged tiles, several
vocabulary slabs, temperatures 1 and 2, every reduction, empty and fully masked batches. The
heads' statistics run on 12-wave tiles (D % 64 == 0), 8-wave tiles, or one of each, and with
D = 64 and 9000 ids in one launch per group of tiles (the student's layout serves both heads).
Tolerances as for LCE: loss 1e-3 absolute (per token for "none"), lse 1e-3, relative Frobenius
1e-2 on dHs and dWs.
"""
import numpy as np
import pytest

from oracle import kd_oracle as K
from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U

pytestmark = pytest.mark.gpu


def _dev(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda:0")


def _run(inp, temperature=1.0, reduction="mean", grad=None, target_dtype=None):
    import torch
    from paper_2605_21442_amd import autograd as AG
    hs, ws, ht, wt = (_dev(x) for x in (inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits))
    t = torch.from_numpy(inp.targets).to("cuda:0")
    if target_dtype is not None:
        t = t.to(target_dtype)
    n = hs.shape[0]
    loss, lse_s, lse_t, nv, status = AG.kd_forward(hs, ws, ht, wt, t, temperature, inp.ignore_index, reduction)
    if grad is None:
        grad = np.ones(n if reduction == "none" else 1, np.float32)
    g = torch.from_numpy(np.asarray(grad, np.float32).reshape(-1)).to("cuda:0")
    dh, dw = AG.kd_backward(hs, ws, ht, wt, t, lse_s, lse_t, nv, g, temperature, inp.ignore_index, reduction)
    torch.cuda.synchronize()
    return dict(loss=(loss.cpu().numpy().astype(np.float64) if reduction == "none" else float(loss.item())),
                lse_s=lse_s.cpu().numpy().astype(np.float64), lse_t=lse_t.cpu().numpy().astype(np.float64),
                n_valid=int(nv.item()), status=int(status.item()),
                dHs=dh.float().cpu().numpy().astype(np.float64), dWs=dw.float().cpu().numpy().astype(np.float64))


def _check(gpu, ref):
    assert gpu["n_valid"] == ref["n_valid"] and gpu["status"] == ref["status"]
    if isinstance(ref["loss"], np.ndarray):
        assert np.max(np.abs(gpu["loss"] - ref["loss"]), initial=0.0) <= U.LSE_ABS_TOL
    else:
        assert abs(gpu["loss"] - ref["loss"]) <= U.LOSS_ABS_TOL, (gpu["loss"], ref["loss"])
    for k in ("lse_s", "lse_t"):
        assert np.max(np.abs(gpu[k] - ref[k]), initial=0.0) <= U.LSE_ABS_TOL, k
    for k in ("dHs", "dWs"):
        assert np.all(np.isfinite(gpu[k]))
        if np.linalg.norm(ref[k]) > 0:
            assert U.rel_fro(gpu[k], ref[k]) <= U.GRAD_REL_TOL, (k, U.rel_fro(gpu[k], ref[k]))
        else:
            assert np.linalg.norm(gpu[k]) <= 1e-6, k


@pytest.mark.parametrize("n,ds,dt,v", [(300, 264, 136, 1000), (600, 128, 256, 9000), (1, 8, 16, 5),
                                       (257, 64, 72, 300), (513, 96, 520, 4097), (300, 64, 128, 9000),
                                       (300, 64, 128, 20000)])       # two slabs of the narrow KD width
@pytest.mark.parametrize("temperature", [1.0, 2.0])
def test_kd_matches_oracle(n, ds, dt, v, temperature):
    print(f"kd n={n} ds={ds} dt={dt} v={v} T={temperature}", flush=True)
    inp = WL.kd_custom(n, ds, dt, v, seed=n + v, mask_frac=0.2)
    gpu = _run(inp, temperature)
    ref = K.kd_bits(inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits, inp.targets, temperature=temperature)
    _check(gpu, ref)
    ignored = inp.targets == -100
    assert np.all(gpu["dHs"][ignored] == 0.0)


@pytest.mark.parametrize("reduction", ["sum", "none"])
def test_kd_reductions(reduction):
    inp = WL.kd_custom(700, 136, 200, 2000, seed=3, mask_frac=0.25)
    g = np.random.default_rng(4).standard_normal(700).astype(np.float32) if reduction == "none" else np.float32([0.6])
    gpu = _run(inp, 1.5, reduction, g)
    ref = K.kd_bits(inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits, inp.targets, temperature=1.5,
                    reduction=reduction, grad=(g.astype(np.float64) if reduction == "none" else 0.6))
    _check(gpu, ref)


def test_kd_tiny_workload_int64_labels():
    import torch
    inp = WL.kd_generate("kd_tiny", 0)
    gpu = _run(inp, target_dtype=torch.int64)
    ref = K.kd_bits(inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits, inp.targets)
    _check(gpu, ref)


@pytest.mark.parametrize("case", ["all_masked", "no_tokens"])
def test_kd_without_valid_tokens(case):
    n = 0 if case == "no_tokens" else 40
    inp = WL.kd_custom(n, 32, 48, 300, seed=1, target_override=np.full(n, -100, np.int32))
    gpu = _run(inp)
    assert gpu["n_valid"] == 0 and gpu["loss"] == 0.0
    assert np.all(gpu["dWs"] == 0.0) and np.all(gpu["dHs"] == 0.0)


def test_student_equal_to_teacher_has_zero_gradient():
    inp = WL.kd_custom(300, 64, 64, 1000, seed=6)
    inp.ht_bits, inp.wt_bits = inp.hs_bits.copy(), inp.ws_bits.copy()
    gpu = _run(inp, 1.0)
    ref = K.kd_bits(inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits, inp.targets)
    assert abs(gpu["loss"] - ref["loss"]) <= U.LOSS_ABS_TOL
    # G = c (p_s - p_t) vanishes up to the fp32 arithmetic of the two passes
    assert np.abs(gpu["dWs"]).max() <= 1e-6 and np.abs(gpu["dHs"]).max() <= 1e-6


def test_kd_autograd_function():
    import torch
    from paper_2605_21442_amd import linear_kd_loss
    inp = WL.kd_custom(2 * 150, 96, 128, 700, seed=7)
    hs = _dev(inp.hs_bits).view(2, 150, 96).clone().requires_grad_(True)
    ws = _dev(inp.ws_bits).clone().requires_grad_(True)
    ht, wt = _dev(inp.ht_bits).view(2, 150, 128), _dev(inp.wt_bits)
    t = torch.from_numpy(inp.targets).to("cuda:0").view(2, 150)
    loss = linear_kd_loss(hs, ws, ht, wt, t, temperature=2.0)
    (3.0 * loss).backward()
    ref = K.kd_bits(inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits, inp.targets, temperature=2.0, grad=3.0)
    assert abs(loss.item() - ref["loss"]) <= U.LOSS_ABS_TOL
    assert U.rel_fro(hs.grad.view(300, 96).float().cpu().numpy(), ref["dHs"]) <= U.GRAD_REL_TOL
    assert U.rel_fro(ws.grad.float().cpu().numpy(), ref["dWs"]) <= U.GRAD_REL_TOL


@pytest.mark.parametrize("n,ds,dt,v,reduction", [(600, 128, 256, 9000, "mean"), (300, 264, 136, 1000, "none"),
                                                 (1, 8, 16, 5, "sum"), (40, 16, 32, 300, "mean"),
                                                 (300, 64, 128, 9000, "mean"), (300, 64, 128, 20000, "mean")])
def test_fused_forward_backward_is_bitwise_the_two_calls(n, ds, dt, v, reduction):
    import torch
    from paper_2605_21442_amd import autograd as AG
    inp = WL.kd_custom(n, ds, dt, v, seed=n + 1, mask_frac=0.2)
    hs, ws, ht, wt = (_dev(x) for x in (inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits))
    t = torch.from_numpy(inp.targets).to("cuda:0")
    g = torch.from_numpy(np.random.default_rng(n).standard_normal(n if reduction == "none" else 1)
                         .astype(np.float32)).to("cuda:0")
    loss, lse_s, lse_t, nv, _ = AG.kd_forward(hs, ws, ht, wt, t, 1.5, -100, reduction)
    dh, dw = AG.kd_backward(hs, ws, ht, wt, t, lse_s, lse_t, nv, g, 1.5, -100, reduction)
    f = AG.kd_forward_backward(hs, ws, ht, wt, t, g, 1.5, -100, reduction)
    torch.cuda.synchronize()
    for a, b in ((loss, f[0]), (lse_s, f[1]), (lse_t, f[2]), (nv, f[3]), (dh, f[5]), (dw, f[6])):
        assert torch.equal(a.view(-1).view(torch.int8) if a.dtype != torch.int32 else a,
                           b.view(-1).view(torch.int8) if b.dtype != torch.int32 else b)


def test_fused_without_tokens():
    import torch
    from paper_2605_21442_amd import autograd as AG
    inp = WL.kd_custom(0, 32, 48, 300, seed=1, target_override=np.zeros(0, np.int32))
    hs, ws, ht, wt = (_dev(x) for x in (inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits))
    t = torch.from_numpy(inp.targets).to("cuda:0")
    f = AG.kd_forward_backward(hs, ws, ht, wt, t, torch.ones(1, device="cuda:0"))
    torch.cuda.synchronize()
    assert float(f[0].item()) == 0.0 and int(f[3].item()) == 0 and not f[6].float().abs().sum().item()
