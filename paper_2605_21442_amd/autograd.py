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


def _rows_usable(shape, strides, data_ptr: int) -> bool:
    """Whether a 2-D bf16 view can be handed to the library as it is: unit column stride, 16-byte
    aligned start, a row stride that is a multiple of 8 and rows that do not overlap. A row stride
    below the row length (0 for an expand()ed tensor) would be read by the library as rows the
    allocation does not hold."""
    rows, cols = shape
    if rows > 1 and strides[0] < cols:
        return False
    return strides[1] == 1 and data_ptr % 16 == 0 and strides[0] % 8 == 0


def _as_rows(x: torch.Tensor, name: str) -> tuple[torch.Tensor, int]:
    if x.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be bfloat16, got {x.dtype}")
    if not x.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    x2 = x.reshape(-1, x.shape[-1]) if x.dim() != 2 else x
    if not _rows_usable(tuple(x2.shape), x2.stride(), x2.data_ptr()):
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
            ignore_index: int = -100, reduction: str = "mean", keep_workspace: bool = False):
    """(loss, lse fp32 [N], n_valid int32 [1], status int32 [1]) computed by lce_forward; loss is
    a fp32 scalar for "mean" / "sum" and the fp32 per-token losses [N] for "none". With
    ``keep_workspace`` a fifth element is the workspace, sized for the backward too, which a
    following ``backward(..., workspace=...)`` reuses (the valid-row list and gathered rows the
    forward left in it)."""
    h, ldh = _as_rows(hidden, "hidden")
    w, ldw = _as_rows(weight, "weight")
    n, d = h.shape
    v = w.shape[0]
    if w.shape[1] != d:
        raise ValueError(f"weight is {tuple(w.shape)}, hidden size is {d}")
    t, tb = _targets(targets, n)
    p = B.problem(n, d, v, ld_h=ldh, ld_w=ldw, ignore_index=ignore_index, reduction=reduction,
                  target_bytes=tb)
    fwd_bytes, bwd_bytes = B.lce_workspace_size(p)
    dev = h.device
    loss = torch.empty((n,) if reduction == "none" else (), dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(max(fwd_bytes, bwd_bytes if keep_workspace else 0, 1), dtype=torch.uint8, device=dev)
    B.lce_forward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), loss.data_ptr(), lse.data_ptr(),
                  nv.data_ptr(), status.data_ptr(), ws.data_ptr(), fwd_bytes, _stream(dev))
    if keep_workspace:
        return loss, lse, nv, status, ws
    return loss, lse, nv, status


def _backward_args(hidden, weight, targets, lse, grad_loss, ignore_index, reduction, flags=0):
    h, ldh = _as_rows(hidden, "hidden")
    w, ldw = _as_rows(weight, "weight")
    n, d = h.shape
    v = w.shape[0]
    t, tb = _targets(targets, n)
    p = B.problem(n, d, v, ld_h=ldh, ld_w=ldw, ignore_index=ignore_index, reduction=reduction,
                  target_bytes=tb, flags=flags)
    want = n if reduction == "none" else 1
    if grad_loss.dtype != torch.float32 or grad_loss.numel() != want or not grad_loss.is_cuda:
        raise ValueError(f"grad_loss must be a {want}-element float32 GPU tensor")
    if lse.dtype != torch.float32 or lse.numel() != n or not lse.is_contiguous():
        raise ValueError("lse must be the contiguous float32 [N] tensor from forward")
    return p, h, w, t, grad_loss.contiguous()


def _workspace(workspace, nbytes, dev):
    """The caller's workspace (from ``forward(..., keep_workspace=True)``) or a new one."""
    if workspace is None:
        return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    if workspace.dtype != torch.uint8 or workspace.numel() < nbytes or not workspace.is_contiguous():
        raise ValueError("workspace is not the one forward(..., keep_workspace=True) returned for this problem")
    return workspace


def backward(hidden: torch.Tensor, weight: torch.Tensor, targets: torch.Tensor, lse: torch.Tensor,
             n_valid: torch.Tensor, grad_loss: torch.Tensor, ignore_index: int = -100,
             reduction: str = "mean", accumulate_into: torch.Tensor | None = None,
             workspace: torch.Tensor | None = None):
    """(dH bf16 [N, D], dW bf16 [V, D]) computed by lce_backward. With ``accumulate_into`` (a
    dense bf16 [V, D] tensor) this call's dW is added to it in place and it is returned as dW.
    ``workspace`` is the one the forward of the same inputs kept (``keep_workspace=True``), untouched
    since: the backward then reuses what that forward left in it (LCE_FLAG_REUSE_FORWARD)."""
    flags = B.LCE_FLAG_ACCUMULATE_DW if accumulate_into is not None else 0
    if workspace is not None:
        flags |= B.LCE_FLAG_REUSE_FORWARD
    p, h, w, t, g = _backward_args(hidden, weight, targets, lse, grad_loss, ignore_index, reduction, flags)
    _, bwd_bytes = B.lce_workspace_size(p)
    dev = h.device
    dh = torch.empty((p.n, p.d), dtype=torch.bfloat16, device=dev)
    if accumulate_into is None:
        dw = torch.empty((p.v, p.d), dtype=torch.bfloat16, device=dev)
    else:
        dw = accumulate_into
        if dw.dtype != torch.bfloat16 or tuple(dw.shape) != (p.v, p.d) or not dw.is_contiguous():
            raise ValueError("accumulate_into must be a contiguous bf16 [V, D] tensor")
    ws = _workspace(workspace, bwd_bytes, dev)
    B.lce_backward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse.data_ptr(), n_valid.data_ptr(),
                   g.data_ptr(), dh.data_ptr(), dw.data_ptr(), ws.data_ptr(), bwd_bytes, _stream(dev))
    return dh, dw


class AdamWState:
    """AdamW state of one bf16 weight [V, D] (paper Sec. 4.1): fp32 moments, an optional fp32
    master copy, the hyper-parameters and the step count. ``step_with(dW)`` is the two-phase
    optimizer step (lce_adamw_step); passed as ``optimizer=`` to ``linear_cross_entropy`` it
    is instead applied inside the backward pass (lce_backward_adamw), which never forms dW."""

    def __init__(self, weight: torch.Tensor, lr: float = 1e-3, betas=(0.9, 0.999), eps: float = 1e-8,
                 weight_decay: float = 0.01, master_weights: bool = False):
        if weight.dtype != torch.bfloat16 or weight.dim() != 2 or not weight.is_cuda:
            raise ValueError("weight must be a 2-D bf16 GPU tensor")
        if (weight.stride(-1) != 1 or weight.stride(0) % 8 or weight.data_ptr() % 16
                or (weight.shape[0] > 1 and weight.stride(0) < weight.shape[1])):
            raise ValueError("weight must have unit column stride, rows that do not overlap, a row "
                             "stride divisible by 8 and 16-byte alignment, since it is updated in place")
        self.weight = weight
        self.lr, self.betas, self.eps, self.weight_decay = lr, tuple(betas), eps, weight_decay
        self.exp_avg = torch.zeros(weight.shape, dtype=torch.float32, device=weight.device)
        self.exp_avg_sq = torch.zeros_like(self.exp_avg)
        self.master = weight.float().contiguous() if master_weights else None
        self.step = 0

    def state_dict(self) -> dict:
        """Per-parameter state for checkpointing (tensors are shared, not copied)."""
        return {"step": self.step, "exp_avg": self.exp_avg, "exp_avg_sq": self.exp_avg_sq,
                "master": self.master, "lr": self.lr, "betas": self.betas, "eps": self.eps,
                "weight_decay": self.weight_decay}

    def load_state_dict(self, sd: dict) -> None:
        """Restore a state_dict: moments (and master copy) are copied into this state's tensors."""
        self.exp_avg.copy_(sd["exp_avg"])
        self.exp_avg_sq.copy_(sd["exp_avg_sq"])
        if (sd.get("master") is None) != (self.master is None):
            raise ValueError("master-weight setting differs from the checkpoint")
        if self.master is not None:
            self.master.copy_(sd["master"])
        self.step = int(sd["step"])
        for k in ("lr", "betas", "eps", "weight_decay"):
            if k in sd:
                setattr(self, k, tuple(sd[k]) if k == "betas" else sd[k])

    def next_opt(self) -> B.LceAdamW:
        return B.adamw(self.lr, self.betas[0], self.betas[1], self.eps, self.weight_decay, self.step + 1)

    def _ptrs(self):
        m = self.master.data_ptr() if self.master is not None else 0
        return self.exp_avg.data_ptr(), self.exp_avg_sq.data_ptr(), m

    def step_with(self, dW: torch.Tensor | None) -> None:
        """Two-phase step: one AdamW update of the weight with the bf16 gradient dW [V, D]."""
        w = self.weight
        if dW is not None and (dW.dtype != torch.bfloat16 or dW.shape != w.shape or not dW.is_contiguous()):
            raise ValueError("dW must be a contiguous bf16 tensor shaped like the weight")
        opt = self.next_opt()
        B.lce_adamw_step(w.shape[0], w.shape[1], w.stride(0), w.data_ptr(), dW.data_ptr() if dW is not None else 0,
                         *self._ptrs(), opt, _stream(w.device))
        self.step += 1


def backward_adamw(hidden: torch.Tensor, targets: torch.Tensor, lse: torch.Tensor, n_valid: torch.Tensor,
                   grad_loss: torch.Tensor, state: AdamWState, ignore_index: int = -100,
                   reduction: str = "mean", workspace: torch.Tensor | None = None) -> torch.Tensor:
    """dH bf16 [N, D] from lce_backward_adamw; the weight of ``state`` takes one AdamW step
    with its gradient inside the call. ``workspace`` as for ``backward``."""
    flags = B.LCE_FLAG_REUSE_FORWARD if workspace is not None else 0
    p, h, w, t, g = _backward_args(hidden, state.weight, targets, lse, grad_loss, ignore_index, reduction, flags)
    if w.data_ptr() != state.weight.data_ptr():
        raise ValueError("the weight must be usable in place")
    _, bwd_bytes = B.lce_workspace_size(p)
    dev = h.device
    dh = torch.empty((p.n, p.d), dtype=torch.bfloat16, device=dev)
    ws = _workspace(workspace, bwd_bytes, dev)
    B.lce_backward_adamw(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse.data_ptr(), n_valid.data_ptr(),
                         g.data_ptr(), dh.data_ptr(), *state._ptrs(), state.next_opt(), ws.data_ptr(),
                         bwd_bytes, _stream(dev))
    state.step += 1
    return dh


# ---- vocabulary-parallel (loss-parallel) pieces ---------------------------------------------
# Each function runs one library call for one vocabulary shard; moving the [N] partials and the
# dH terms between devices (all-gather, all-reduce) is the caller's collective.

def forward_shard(hidden, weight_shard, targets, v_begin: int, v_total: int, ignore_index: int = -100):
    """(lse_part fp32 [N], tgt_part fp32 [N], n_valid, status) of the shard holding ids
    [v_begin, v_begin + rows of weight_shard) of a v_total-id vocabulary (lce_forward_shard)."""
    h, ldh = _as_rows(hidden, "hidden")
    w, ldw = _as_rows(weight_shard, "weight")
    n, d = h.shape
    t, tb = _targets(targets, n)
    p = B.problem(n, d, w.shape[0], ld_h=ldh, ld_w=ldw, ignore_index=ignore_index, target_bytes=tb)
    fwd_bytes, _ = B.lce_workspace_size(p)
    dev = h.device
    lse_part = torch.empty(n, dtype=torch.float32, device=dev)
    tgt_part = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(max(fwd_bytes, 1), dtype=torch.uint8, device=dev)
    B.lce_forward_shard(p, B.LceShard(v_total, v_begin), h.data_ptr(), w.data_ptr(), t.data_ptr(),
                        lse_part.data_ptr(), tgt_part.data_ptr(), nv.data_ptr(), status.data_ptr(),
                        ws.data_ptr(), fwd_bytes, _stream(dev))
    return lse_part, tgt_part, nv, status


def combine_shards(lse_parts: torch.Tensor, tgt_parts: torch.Tensor, targets: torch.Tensor, v_total: int,
                   d: int, ignore_index: int = -100, reduction: str = "mean"):
    """(loss, lse [N], n_valid, status) of the whole vocabulary from [G, N] shard partials."""
    g, n = lse_parts.shape
    for x in (lse_parts, tgt_parts):
        if x.dtype != torch.float32 or not x.is_contiguous() or tuple(x.shape) != (g, n):
            raise ValueError("partials must be contiguous float32 [G, N] tensors")
    t, tb = _targets(targets, n)
    p = B.problem(n, d, v_total, ignore_index=ignore_index, reduction=reduction, target_bytes=tb)
    fwd_bytes, _ = B.lce_workspace_size(p)
    dev = lse_parts.device
    loss = torch.empty((n,) if reduction == "none" else (), dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(max(fwd_bytes, 1), dtype=torch.uint8, device=dev)
    B.lce_combine_shards(p, g, lse_parts.data_ptr(), tgt_parts.data_ptr(), t.data_ptr(), loss.data_ptr(),
                         lse.data_ptr(), nv.data_ptr(), status.data_ptr(), ws.data_ptr(), fwd_bytes, _stream(dev))
    return loss, lse, nv, status


def backward_shard(hidden, weight_shard, targets, lse, n_valid, grad_loss, v_begin: int, v_total: int,
                   ignore_index: int = -100, reduction: str = "mean"):
    """(dH term fp32 [N, D], dW rows bf16 [V_shard, D]) of one shard, given the global lse
    (lce_backward_shard); the dH terms of all shards sum to dH."""
    p, h, w, t, g = _backward_args(hidden, weight_shard, targets, lse, grad_loss, ignore_index, reduction)
    _, bwd_bytes = B.lce_workspace_size(p)
    dev = h.device
    dh = torch.empty((p.n, p.d), dtype=torch.float32, device=dev)
    dw = torch.empty((p.v, p.d), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(max(bwd_bytes, 1), dtype=torch.uint8, device=dev)
    B.lce_backward_shard(p, B.LceShard(v_total, v_begin), h.data_ptr(), w.data_ptr(), t.data_ptr(),
                         lse.data_ptr(), n_valid.data_ptr(), g.data_ptr(), dh.data_ptr(), dw.data_ptr(),
                         ws.data_ptr(), bwd_bytes, _stream(dev))
    return dh, dw


class LinearCrossEntropy(torch.autograd.Function):
    """Fused projection + cross-entropy; backward returns gradients for hidden and weight."""

    @staticmethod
    def forward(ctx, hidden, weight, targets, ignore_index=-100, reduction="mean"):
        # when a gradient will be taken, the workspace (sized for both passes) is kept for the
        # backward, which then skips the compaction and row gather the forward already did
        keep = any(ctx.needs_input_grad[:2])
        loss, lse, nv, _, *ws = forward(hidden, weight, targets, ignore_index, reduction, keep_workspace=keep)
        ctx.save_for_backward(hidden, weight, targets, lse, nv)
        ctx.ws = ws[0] if keep else None
        ctx.ignore_index = ignore_index
        ctx.reduction = reduction
        return loss.view(targets.shape) if reduction == "none" else loss

    @staticmethod
    def backward(ctx, grad):
        hidden, weight, targets, lse, nv = ctx.saved_tensors
        g = grad.reshape(-1)
        if g.dtype != torch.float32:
            g = g.float()
        ws, ctx.ws = ctx.ws, None     # used once: a second backward through the graph forms its own
        dh, dw = backward(hidden, weight, targets, lse, nv, g, ctx.ignore_index, ctx.reduction, workspace=ws)
        return dh.view(hidden.shape), dw, None, None, None


class LinearCrossEntropyAdamW(torch.autograd.Function):
    """As LinearCrossEntropy, but the backward steps the weight with AdamW in place (paper
    Sec. 4.1) and returns no weight gradient."""

    @staticmethod
    def forward(ctx, hidden, weight, targets, state, ignore_index=-100, reduction="mean"):
        loss, lse, nv, _, ws = forward(hidden, weight, targets, ignore_index, reduction, keep_workspace=True)
        ctx.save_for_backward(hidden, targets, lse, nv)
        ctx.ws = ws
        ctx.state = state
        ctx.ignore_index = ignore_index
        ctx.reduction = reduction
        return loss.view(targets.shape) if reduction == "none" else loss

    @staticmethod
    def backward(ctx, grad):
        hidden, targets, lse, nv = ctx.saved_tensors
        g = grad.reshape(-1)
        if g.dtype != torch.float32:
            g = g.float()
        ws, ctx.ws = ctx.ws, None
        dh = backward_adamw(hidden, targets, lse, nv, g, ctx.state, ctx.ignore_index, ctx.reduction, workspace=ws)
        return dh.view(hidden.shape), None, None, None, None, None


def linear_cross_entropy(hidden: torch.Tensor, weight: torch.Tensor, targets: torch.Tensor,
                         ignore_index: int = -100, reduction: str = "mean",
                         optimizer: AdamWState | None = None) -> torch.Tensor:
    """Cross-entropy of ``hidden @ weight.T`` against ``targets`` without the logits: the mean over
    valid tokens, their sum, or (``reduction="none"``) the per-token losses, shaped like targets.
    With ``optimizer`` (an AdamWState of this weight) the backward pass applies the AdamW step
    to the weight itself instead of producing its gradient."""
    if optimizer is not None:
        if optimizer.weight.data_ptr() != weight.data_ptr() or optimizer.weight.shape != weight.shape:
            raise ValueError("optimizer state belongs to another weight")
        return LinearCrossEntropyAdamW.apply(hidden, weight, targets, optimizer, ignore_index, reduction)
    return LinearCrossEntropy.apply(hidden, weight, targets, ignore_index, reduction)


# ---- fused linear knowledge distillation ------------------------------------------------------

def _kd_problem(hs, ws, ht, wt, targets, temperature, ignore_index, reduction, flags=0):
    h_s, ldhs = _as_rows(hs, "student hidden")
    w_s, ldws = _as_rows(ws, "student weight")
    h_t, ldht = _as_rows(ht, "teacher hidden")
    w_t, ldwt = _as_rows(wt, "teacher weight")
    n, ds = h_s.shape
    dt = h_t.shape[1]
    v = w_s.shape[0]
    if h_t.shape[0] != n or w_s.shape[1] != ds or w_t.shape != (v, dt):
        raise ValueError("student/teacher shapes disagree")
    t, tb = _targets(targets, n)
    p = B.kd_problem(n, ds, dt, v, ld_hs=ldhs, ld_ws=ldws, ld_ht=ldht, ld_wt=ldwt, temperature=temperature,
                     ignore_index=ignore_index, reduction=reduction, target_bytes=tb, flags=flags)
    return p, h_s, w_s, h_t, w_t, t


def kd_forward(hs, ws, ht, wt, targets, temperature: float = 1.0, ignore_index: int = -100,
               reduction: str = "mean"):
    """(loss, lse_s [N], lse_t [N], n_valid, status) from lce_kd_forward."""
    p, h_s, w_s, h_t, w_t, t = _kd_problem(hs, ws, ht, wt, targets, temperature, ignore_index, reduction)
    fwd_bytes, _ = B.lce_kd_workspace_size(p)
    dev = h_s.device
    n = p.n
    loss = torch.empty((n,) if reduction == "none" else (), dtype=torch.float32, device=dev)
    lse_s = torch.empty(n, dtype=torch.float32, device=dev)
    lse_t = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    ws_ = torch.empty(max(fwd_bytes, 1), dtype=torch.uint8, device=dev)
    B.lce_kd_forward(p, h_s.data_ptr(), w_s.data_ptr(), h_t.data_ptr(), w_t.data_ptr(), t.data_ptr(),
                     loss.data_ptr(), lse_s.data_ptr(), lse_t.data_ptr(), nv.data_ptr(), status.data_ptr(),
                     ws_.data_ptr(), fwd_bytes, _stream(dev))
    return loss, lse_s, lse_t, nv, status


def kd_backward(hs, ws, ht, wt, targets, lse_s, lse_t, n_valid, grad_loss, temperature: float = 1.0,
                ignore_index: int = -100, reduction: str = "mean", accumulate_into: torch.Tensor | None = None):
    """(dHs bf16 [N, Ds], dWs bf16 [V, Ds]) from lce_kd_backward."""
    flags = B.LCE_FLAG_ACCUMULATE_DW if accumulate_into is not None else 0
    p, h_s, w_s, h_t, w_t, t = _kd_problem(hs, ws, ht, wt, targets, temperature, ignore_index, reduction, flags)
    n, ds, v = p.n, p.ds, p.v
    want = n if reduction == "none" else 1
    if grad_loss.dtype != torch.float32 or grad_loss.numel() != want or not grad_loss.is_cuda:
        raise ValueError(f"grad_loss must be a {want}-element float32 GPU tensor")
    for x in (lse_s, lse_t):
        if x.dtype != torch.float32 or x.numel() != n or not x.is_contiguous():
            raise ValueError("lse_s / lse_t must be the contiguous float32 [N] tensors from kd_forward")
    _, bwd_bytes = B.lce_kd_workspace_size(p)
    dev = h_s.device
    dh = torch.empty((n, ds), dtype=torch.bfloat16, device=dev)
    if accumulate_into is None:
        dw = torch.empty((v, ds), dtype=torch.bfloat16, device=dev)
    else:
        dw = accumulate_into
        if dw.dtype != torch.bfloat16 or tuple(dw.shape) != (v, ds) or not dw.is_contiguous():
            raise ValueError("accumulate_into must be a contiguous bf16 [V, Ds] tensor")
    g = grad_loss.contiguous()
    ws_ = torch.empty(max(bwd_bytes, 1), dtype=torch.uint8, device=dev)
    B.lce_kd_backward(p, h_s.data_ptr(), w_s.data_ptr(), h_t.data_ptr(), w_t.data_ptr(), t.data_ptr(),
                      lse_s.data_ptr(), lse_t.data_ptr(), n_valid.data_ptr(), g.data_ptr(), dh.data_ptr(),
                      dw.data_ptr(), ws_.data_ptr(), bwd_bytes, _stream(dev))
    return dh, dw


def kd_forward_backward(hs, ws, ht, wt, targets, grad_loss, temperature: float = 1.0, ignore_index: int = -100,
                        reduction: str = "mean"):
    """(loss, lse_s, lse_t, n_valid, status, dHs, dWs) from lce_kd_forward_backward: the KD loss
    and the student's gradients in one call, ``grad_loss`` being the upstream gradient."""
    p, h_s, w_s, h_t, w_t, t = _kd_problem(hs, ws, ht, wt, targets, temperature, ignore_index, reduction)
    n, ds, v = p.n, p.ds, p.v
    want = n if reduction == "none" else 1
    if grad_loss.dtype != torch.float32 or grad_loss.numel() != want or not grad_loss.is_cuda:
        raise ValueError(f"grad_loss must be a {want}-element float32 GPU tensor")
    g = grad_loss.contiguous()
    nbytes = B.lce_kd_workspace_size_fused(p)
    dev = h_s.device
    loss = torch.empty((n,) if reduction == "none" else (), dtype=torch.float32, device=dev)
    lse_s = torch.empty(n, dtype=torch.float32, device=dev)
    lse_t = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    dh = torch.empty((n, ds), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((v, ds), dtype=torch.bfloat16, device=dev)
    ws_ = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    B.lce_kd_forward_backward(p, h_s.data_ptr(), w_s.data_ptr(), h_t.data_ptr(), w_t.data_ptr(), t.data_ptr(),
                              g.data_ptr(), loss.data_ptr(), lse_s.data_ptr(), lse_t.data_ptr(), nv.data_ptr(),
                              status.data_ptr(), dh.data_ptr(), dw.data_ptr(), ws_.data_ptr(), nbytes, _stream(dev))
    return loss, lse_s, lse_t, nv, status, dh, dw


class LinearKD(torch.autograd.Function):
    """Soft-target cross-entropy of a student head against a teacher head; gradients for the
    student's hidden states and weight only."""

    @staticmethod
    def forward(ctx, hs, ws, ht, wt, targets, temperature=1.0, ignore_index=-100, reduction="mean"):
        loss, lse_s, lse_t, nv, _ = kd_forward(hs, ws, ht, wt, targets, temperature, ignore_index, reduction)
        ctx.save_for_backward(hs, ws, ht, wt, targets, lse_s, lse_t, nv)
        ctx.opts = (temperature, ignore_index, reduction)
        return loss.view(targets.shape) if reduction == "none" else loss

    @staticmethod
    def backward(ctx, grad):
        hs, ws, ht, wt, targets, lse_s, lse_t, nv = ctx.saved_tensors
        temperature, ignore_index, reduction = ctx.opts
        g = grad.reshape(-1)
        if g.dtype != torch.float32:
            g = g.float()
        dh, dw = kd_backward(hs, ws, ht, wt, targets, lse_s, lse_t, nv, g, temperature, ignore_index, reduction)
        return dh.view(hs.shape), dw, None, None, None, None, None, None


def linear_kd_loss(student_hidden, student_weight, teacher_hidden, teacher_weight, targets,
                   temperature: float = 1.0, ignore_index: int = -100, reduction: str = "mean"):
    """Knowledge-distillation loss between two output heads without either logit matrix: the
    soft-target cross-entropy of softmax(student / T) against softmax(teacher / T), averaged (or
    summed, or per token) over the tokens whose label is not ignored."""
    return LinearKD.apply(student_hidden, student_weight, teacher_hidden, teacher_weight, targets,
                          temperature, ignore_index, reduction)
