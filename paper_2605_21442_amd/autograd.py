"""torch front end of the LCE library: tensors in, tensors out, work in liblce.so.

``linear_cross_entropy(hidden, weight, targets)`` is the one-line replacement of
``cross_entropy(hidden @ weight.T, targets)`` that the paper's recipes switch on
(Sec. 3.3, Sec. 4.2): the library fuses the projection with the loss and never
materialises the logits. torch supplies device memory (outputs and workspace,
through its caching allocator) and the current stream; everything else runs in
the library's kernels.
"""
from __future__ import annotations

import torch

from . import binding as B


def _as_rows(x: torch.Tensor, name: str) -> tuple[torch.Tensor, int]:
    if x.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be bfloat16, got {x.dtype}")
    if not x.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    x2 = x.reshape(-1, x.shape[-1]) if x.dim() != 2 else x
    if x2.stride(-1) != 1 or x2.data_ptr() % 16 or x2.stride(0) % 8:
        x2 = x2.contiguous()
    return x2, (x2.stride(0) if x2.shape[0] > 1 else x2.shape[1])


def _targets(t: torch.Tensor, n: int) -> tuple[torch.Tensor, int]:
    if t.dtype not in (torch.int32, torch.int64):
        raise TypeError(f"targets must be int32 or int64, got {t.dtype}")
    t1 = t.reshape(-1)
    if t1.numel() != n:
        raise ValueError(f"targets has {t1.numel()} entries for {n} hidden rows")
    if not t1.is_contiguous():
        t1 = t1.contiguous()
    return t1, t1.element_size()


def _stream(dev: torch.device) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def forward(hidden: torch.Tensor, weight: torch.Tensor, targets: torch.Tensor,
            ignore_index: int = -100, reduction: str = "mean"):
    """(loss, lse fp32 [N], n_valid int32 [1], status int32 [1]) computed by lce_forward; loss is
    a fp32 scalar for "mean" / "sum" and the fp32 per-token losses [N] for "none"."""
    h, ldh = _as_rows(hidden, "hidden")
    w, ldw = _as_rows(weight, "weight")
    n, d = h.shape
    v = w.shape[0]
    if w.shape[1] != d:
        raise ValueError(f"weight is {tuple(w.shape)}, hidden size is {d}")
    t, tb = _targets(targets, n)
    p = B.problem(n, d, v, ld_h=ldh, ld_w=ldw, ignore_index=ignore_index, reduction=reduction,
                  target_bytes=tb)
    fwd_bytes, _ = B.lce_workspace_size(p)
    dev = h.device
    loss = torch.empty((n,) if reduction == "none" else (), dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(max(fwd_bytes, 1), dtype=torch.uint8, device=dev)
    B.lce_forward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), loss.data_ptr(), lse.data_ptr(),
                  nv.data_ptr(), status.data_ptr(), ws.data_ptr(), fwd_bytes, _stream(dev))
    return loss, lse, nv, status


def backward(hidden: torch.Tensor, weight: torch.Tensor, targets: torch.Tensor, lse: torch.Tensor,
             n_valid: torch.Tensor, grad_loss: torch.Tensor, ignore_index: int = -100,
             reduction: str = "mean"):
    """(dH bf16 [N, D], dW bf16 [V, D]) computed by lce_backward."""
    h, ldh = _as_rows(hidden, "hidden")
    w, ldw = _as_rows(weight, "weight")
    n, d = h.shape
    v = w.shape[0]
    t, tb = _targets(targets, n)
    p = B.problem(n, d, v, ld_h=ldh, ld_w=ldw, ignore_index=ignore_index, reduction=reduction,
                  target_bytes=tb)
    _, bwd_bytes = B.lce_workspace_size(p)
    dev = h.device
    want = n if reduction == "none" else 1
    if grad_loss.dtype != torch.float32 or grad_loss.numel() != want or not grad_loss.is_cuda:
        raise ValueError(f"grad_loss must be a {want}-element float32 GPU tensor")
    grad_loss = grad_loss.contiguous()
    if lse.dtype != torch.float32 or lse.numel() != n or not lse.is_contiguous():
        raise ValueError("lse must be the contiguous float32 [N] tensor from forward")
    dh = torch.empty((n, d), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((v, d), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(max(bwd_bytes, 1), dtype=torch.uint8, device=dev)
    B.lce_backward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse.data_ptr(), n_valid.data_ptr(),
                   grad_loss.data_ptr(), dh.data_ptr(), dw.data_ptr(), ws.data_ptr(), bwd_bytes,
                   _stream(dev))
    return dh, dw


class LinearCrossEntropy(torch.autograd.Function):
    """Fused projection + cross-entropy; backward returns gradients for hidden and weight."""

    @staticmethod
    def forward(ctx, hidden, weight, targets, ignore_index=-100, reduction="mean"):
        loss, lse, nv, _ = forward(hidden, weight, targets, ignore_index, reduction)
        ctx.save_for_backward(hidden, weight, targets, lse, nv)
        ctx.ignore_index = ignore_index
        ctx.reduction = reduction
        return loss.view(targets.shape) if reduction == "none" else loss

    @staticmethod
    def backward(ctx, grad):
        hidden, weight, targets, lse, nv = ctx.saved_tensors
        g = grad.reshape(-1)
        if g.dtype != torch.float32:
            g = g.float()
        dh, dw = backward(hidden, weight, targets, lse, nv, g, ctx.ignore_index, ctx.reduction)
        return dh.view(hidden.shape), dw, None, None, None


def linear_cross_entropy(hidden: torch.Tensor, weight: torch.Tensor, targets: torch.Tensor,
                         ignore_index: int = -100, reduction: str = "mean") -> torch.Tensor:
    """Cross-entropy of ``hidden @ weight.T`` against ``targets`` without the logits: the mean over
    valid tokens, their sum, or (``reduction="none"``) the per-token losses, shaped like targets."""
    return LinearCrossEntropy.apply(hidden, weight, targets, ignore_index, reduction)
