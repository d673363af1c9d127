"""Helpers shared by the GPU tests: move drawn inputs to the GPU, run the library, compare."""
from __future__ import annotations

import numpy as np

LOSS_ABS_TOL = 1e-3      # mean-loss absolute error bound
GRAD_REL_TOL = 1e-2      # relative Frobenius error bound on dH and dW
LSE_ABS_TOL = 1e-3       # per-row lse absolute error bound


def to_device(inp, dev="cuda:0", target_dtype=None):
    import torch
    h = torch.from_numpy(inp.h_bits.view(np.int16)).view(torch.bfloat16).to(dev)
    w = torch.from_numpy(inp.w_bits.view(np.int16)).view(torch.bfloat16).to(dev)
    t = torch.from_numpy(inp.targets).to(dev)
    if target_dtype is not None:
        t = t.to(target_dtype)
    return h, w, t


def run_gpu(h, w, t, ignore_index=-100, reduction="mean", grad=1.0, backward=True):
    """Run lce_forward (+ lce_backward) through the C ABI; returns numpy results."""
    import torch
    from paper_2605_21442_amd import autograd as A
    loss, lse, nv, status = A.forward(h, w, t, ignore_index, reduction)
    out = {"loss_t": loss, "lse_t": lse, "nv_t": nv}
    if backward:
        if reduction == "none":
            g = torch.as_tensor(np.asarray(grad, dtype=np.float32), device=h.device)
        else:
            g = torch.tensor([grad], dtype=torch.float32, device=h.device)
        dh, dw = A.backward(h, w, t, lse, nv, g, ignore_index, reduction)
        out["dH_t"], out["dW_t"] = dh, dw
    torch.cuda.synchronize()
    out["loss"] = loss.cpu().numpy().astype(np.float64) if reduction == "none" else float(loss.item())
    out["lse"] = lse.cpu().numpy().astype(np.float64)
    out["n_valid"] = int(nv.item())
    out["status"] = int(status.item())
    if backward:
        out["dH"] = out["dH_t"].float().cpu().numpy().astype(np.float64)
        out["dW"] = out["dW_t"].float().cpu().numpy().astype(np.float64)
    return out


def rel_fro(x, ref):
    nr = np.linalg.norm(ref)
    return np.linalg.norm(x - ref) / nr if nr > 0 else np.linalg.norm(x)


def assert_parity(gpu, ref, *, grads=True, abs_zero_tol=1e-6):
    assert gpu["n_valid"] == ref["n_valid"], (gpu["n_valid"], ref["n_valid"])
    assert gpu["status"] == ref["status"]
    if isinstance(ref["loss"], np.ndarray):      # per-token losses
        assert np.max(np.abs(gpu["loss"] - ref["loss"]), initial=0.0) <= LSE_ABS_TOL
    else:
        # the bar is on the mean loss; a summed loss comes back as one fp32 number, whose spacing
        # exceeds the bar once |L| passes 8192: the bar plus one fp32 spacing of the reference
        tol = LOSS_ABS_TOL + float(np.spacing(np.float32(abs(ref["loss"]))))
        assert abs(gpu["loss"] - ref["loss"]) <= tol, (gpu["loss"], ref["loss"])
    assert np.max(np.abs(gpu["lse"] - ref["lse"]), initial=0.0) <= LSE_ABS_TOL
    if grads:
        for k in ("dH", "dW"):
            assert np.all(np.isfinite(gpu[k])), k
            if np.linalg.norm(ref[k]) > 0:
                e = rel_fro(gpu[k], ref[k])
                assert e <= GRAD_REL_TOL, (k, e)
            else:
                assert np.linalg.norm(gpu[k]) <= abs_zero_tol, k
