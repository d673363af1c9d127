"""Plain CPU oracle of the linear-cross-entropy (LCE) objective.

TEST INFRASTRUCTURE ONLY. Only the tests, the package's ``smoke()`` check and
the benchmark's CPU-baseline leg may import this module. The product path (the
HIP library and its Python binding) never calls it and shares no code with it.

What it computes (paper Sec. 4.2 and Sec. 3.3): LCE fuses the model's final
output projection with the cross-entropy over the whole vocabulary, drops the
ignored target positions before the projection, and is a drop-in for the
standard cross-entropy objective -- it reaches the same value, only without
holding the [tokens, vocab] logit matrix at once. The oracle therefore is the
textbook cross-entropy written out in float64 from the bf16 inputs (exactly
representable in float64), materialising each row's full-vocabulary logits:

  valid set        M = {n : t_n != ignore_index and 0 <= t_n < V},  Nv = |M|
  logits           s[n, v] = sum_d H[n, d] * W[v, d]
  log-sum-exp      lse_n = m_n + ln sum_v exp(s[n, v] - m_n),  m_n = max_v s[n, v]
  per-row loss     l_n = lse_n - s[n, t_n]                        (n in M)
  reduction        L = (1 / Nv) sum_{n in M} l_n   ("mean"),  sum_{n in M} l_n  ("sum"),
                   or the vector of l_n with 0 on rows outside M ("none": per-token losses, i.e.
                   minus the per-token log-probabilities of the targets)
  softmax grad     G[n, v] = c_n * (exp(s[n, v] - lse_n) - [v == t_n])  (n in M; 0 otherwise)
                   c_n = g / Nv for "mean", c_n = g for "sum" (g = upstream gradient of L),
                   c_n = g_n for "none" (g = vector of upstream gradients of the l_n)
  gradients        dH = G W,  dW = G^T H

Readings where the paper is silent (each is also listed in the design notes):
* "mean" divides by the valid-token count of this call; Nv = 0 gives L = 0 and
  zero gradients (not NaN);
* a target outside [0, V) that is not ignore_index is treated as ignored and
  raises status bit 0;
* lse is reported for valid rows only and is 0.0 on every other row;
* targets are already aligned with H (no next-token shift inside the loss).

Pins: the oracle is checked (``tests/test_oracle.py``) against closed forms
(zero weights give L = ln V; a geometric-series vocabulary; V = 1 and V = 2),
central finite differences, an independent library routine (torch CPU float64
cross-entropy with autograd), and invariants (softmax-grad rows sum to zero,
masked rows contribute nothing, shift and permutation invariance). The vocabulary-parallel
helpers at the end are pinned by recombining their per-shard results over several partitions of
the vocabulary into the full-vocabulary results above.
"""
from __future__ import annotations

import numpy as np

STATUS_TARGET_OUT_OF_RANGE = 1


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Decode bf16 bit patterns (uint16) to float64; every bf16 value is exact in float64."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def valid_rows(targets: np.ndarray, v: int, ignore_index: int = -100):
    """Valid-row mask and status word (bit 0: some target outside [0, V) that is not ignored)."""
    t = np.asarray(targets, dtype=np.int64)
    ignored = t == ignore_index
    bad = (~ignored) & ((t < 0) | (t >= v))
    status = STATUS_TARGET_OUT_OF_RANGE if bad.any() else 0
    return (~ignored) & (~bad), status


def row_lse(h_rows: np.ndarray, w: np.ndarray) -> np.ndarray:
    """lse_n = m_n + ln sum_v exp(s[n, v] - m_n) for the given float64 rows of H."""
    s = h_rows @ w.T
    m = s.max(axis=1)
    return m + np.log(np.exp(s - m[:, None]).sum(axis=1))


def scale_c(n_valid: int, reduction: str, grad):
    """Scale of the softmax gradient: g / Nv for "mean", g for "sum" (0 when Nv = 0), and the
    per-row upstream gradients for "none" (an array, returned as float64)."""
    if reduction == "none":
        return np.asarray(grad, dtype=np.float64)
    if reduction not in ("mean", "sum"):
        raise ValueError(f"unknown reduction {reduction!r}")
    if n_valid == 0:
        return 0.0
    return grad / n_valid if reduction == "mean" else grad


def forward(h, w, targets, ignore_index=-100, reduction="mean", block=512):
    """Loss, per-row lse (0 on non-valid rows), Nv and status, from float64 H [N, D] and W [V, D]."""
    n, v = h.shape[0], w.shape[0]
    ok, status = valid_rows(targets, v, ignore_index)
    rows = np.nonzero(ok)[0]
    t = np.asarray(targets, dtype=np.int64)
    lse = np.zeros(n, dtype=np.float64)
    per_row = np.zeros(n, dtype=np.float64)
    for s0 in range(0, rows.size, block):
        r = rows[s0:s0 + block]
        s = h[r] @ w.T                                  # full-vocabulary logits of these rows
        m = s.max(axis=1)
        lse_r = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
        lse[r] = lse_r
        per_row[r] = lse_r - s[np.arange(r.size), t[r]]
    nv = int(rows.size)
    if reduction == "none":
        loss = per_row.copy()
    elif nv == 0:
        loss = 0.0
    elif reduction == "mean":
        loss = float(per_row[rows].sum() / nv)
    elif reduction == "sum":
        loss = float(per_row[rows].sum())
    else:
        raise ValueError(f"unknown reduction {reduction!r}")
    return {"loss": loss, "lse": lse, "per_row": per_row, "n_valid": nv, "status": status}


def softmax_grad_rows(h_rows, w, t_rows, c):
    """G rows c * (softmax(s) - onehot(t)) for valid float64 rows of H (c scalar or per row)."""
    s = h_rows @ w.T
    m = s.max(axis=1)
    lse = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
    g = np.exp(s - lse[:, None])
    g[np.arange(len(t_rows)), t_rows] -= 1.0
    c = np.asarray(c, dtype=np.float64)
    return (c[:, None] if c.ndim == 1 else c) * g


def backward(h, w, targets, ignore_index=-100, reduction="mean", grad=1.0, block=512, progress=None):
    """dH = G W and dW = G^T H with G the scaled softmax-minus-onehot of the valid rows.
    ``progress(done, total)``, if given, is called after each block of valid rows."""
    n, v = h.shape[0], w.shape[0]
    ok, _ = valid_rows(targets, v, ignore_index)
    rows = np.nonzero(ok)[0]
    t = np.asarray(targets, dtype=np.int64)
    c = scale_c(int(rows.size), reduction, grad)
    dh = np.zeros_like(h)
    dw = np.zeros_like(w)
    for s0 in range(0, rows.size, block):
        r = rows[s0:s0 + block]
        g = softmax_grad_rows(h[r], w, t[r], c[r] if reduction == "none" else c)
        dh[r] = g @ w
        dw += g.T @ h[r]
        if progress is not None:
            progress(s0 + r.size, rows.size)
    return {"dH": dh, "dW": dw}


def backward_by_vocab_chunks(h_bits, w_bits, targets, lse, on_dw_chunk, ignore_index=-100,
                             reduction="mean", grad=1.0, chunk=16384, block=4096, progress=None):
    """The backward above (dH = G W, dW = G^T H, G the scaled softmax-minus-onehot of the valid
    rows) for sizes whose whole dW does not fit beside the inputs in host memory: with each valid
    row's lse given (the forward's), the columns of G for a chunk of vocabulary ids need only that
    chunk's logits, exp(s[n, v] - lse_n) - [v == t_n]. The ids are taken chunk by chunk and the
    valid rows block by block within a chunk; dH accumulates over the chunks and each chunk's
    finished rows of dW go to ``on_dw_chunk(v0, dw_rows)`` (ids v0 ..). Host memory stays
    O(Nv D + chunk D + block chunk). Returns (valid row ids, dH of those rows) in float64;
    ``progress(done, total)`` is called after each chunk."""
    v = w_bits.shape[0]
    ok, _ = valid_rows(targets, v, ignore_index)
    rows = np.nonzero(ok)[0]
    c = scale_c(int(rows.size), reduction, grad)
    t = np.asarray(targets, dtype=np.int64)
    hv = bf16_to_f64(h_bits[rows])                             # [Nv, D]
    dh = np.zeros_like(hv)
    lse_v = np.asarray(lse, dtype=np.float64)[rows]
    t_v = t[rows]
    c_v = c[rows] if reduction == "none" else c
    for v0 in range(0, v, chunk):
        v1 = min(v0 + chunk, v)
        wc = bf16_to_f64(w_bits[v0:v1])                        # [k, D]
        dwc = np.zeros_like(wc)
        for s0 in range(0, rows.size, block):
            s1 = min(s0 + block, rows.size)
            g = np.exp(hv[s0:s1] @ wc.T - lse_v[s0:s1, None])  # softmax columns v0 .. v1 of these rows
            hit = np.nonzero((t_v[s0:s1] >= v0) & (t_v[s0:s1] < v1))[0]
            g[hit, t_v[s0:s1][hit] - v0] -= 1.0
            g *= c_v[s0:s1, None] if reduction == "none" else c_v
            dh[s0:s1] += g @ wc
            dwc += g.T @ hv[s0:s1]
        on_dw_chunk(v0, dwc)
        if progress is not None:
            progress(v1, v)
    return rows, dh


def lce(h_bits, w_bits, targets, ignore_index=-100, reduction="mean", grad=1.0):
    """Whole objective from bf16 bit patterns: loss, lse, Nv, status, dH, dW (all float64)."""
    h = bf16_to_f64(h_bits)
    w = bf16_to_f64(w_bits)
    out = forward(h, w, targets, ignore_index, reduction)
    out.update(backward(h, w, targets, ignore_index, reduction, grad))
    return out


# ---- sampled outputs for full-size workloads -------------------------------------------------

def lse_of_rows(h_bits, w_bits, rows, block=64):
    """lse_n of the given rows (no masking logic: rows are taken as they are)."""
    w = bf16_to_f64(w_bits)
    out = np.empty(len(rows), dtype=np.float64)
    for s0 in range(0, len(rows), block):
        r = np.asarray(rows[s0:s0 + block])
        out[s0:s0 + block] = row_lse(bf16_to_f64(h_bits[r]), w)
    return out


def dh_of_rows(h_bits, w_bits, targets, rows, n_valid, ignore_index=-100,
               reduction="mean", grad=1.0):
    """Rows of dH = G W; rows whose target is ignored or out of range are zero."""
    w = bf16_to_f64(w_bits)
    v = w.shape[0]
    ok, _ = valid_rows(targets, v, ignore_index)
    c = scale_c(n_valid, reduction, grad)
    t = np.asarray(targets, dtype=np.int64)
    out = np.zeros((len(rows), w.shape[1]), dtype=np.float64)
    for i, r in enumerate(rows):
        if ok[r]:
            g = softmax_grad_rows(bf16_to_f64(h_bits[r:r + 1]), w, t[r:r + 1],
                                  c[r:r + 1] if reduction == "none" else c)
            out[i] = (g @ w)[0]
    return out


def dw_of_rows(h_bits, w_bits, targets, vrows, lse_valid, ignore_index=-100,
               reduction="mean", grad=1.0, block=4096):
    """Rows of dW = G^T H for vocabulary ids ``vrows``; ``lse_valid`` is the oracle's lse vector."""
    v = w_bits.shape[0]
    ok, _ = valid_rows(targets, v, ignore_index)
    rows = np.nonzero(ok)[0]
    c = scale_c(int(rows.size), reduction, grad)
    t = np.asarray(targets, dtype=np.int64)
    wv = bf16_to_f64(w_bits[np.asarray(vrows)])                 # [k, D]
    out = np.zeros((len(vrows), w_bits.shape[1]), dtype=np.float64)
    for s0 in range(0, rows.size, block):
        r = rows[s0:s0 + block]
        hr = bf16_to_f64(h_bits[r])                            # [b, D]
        p = np.exp(hr @ wv.T - lse_valid[r][:, None])          # softmax columns of these ids
        p -= (t[r][:, None] == np.asarray(vrows)[None, :])
        out += ((c[r][:, None] if reduction == "none" else c) * p).T @ hr
    return out


# ---- vocabulary-parallel (loss-parallel) decomposition --------------------------------------
# With W split by rows (vocabulary ids) over shards, the softmax normaliser is a log-sum-exp of
# the shards' log-sum-exps and the target logit is held by exactly one shard (paper Sec. 4.2 and
# Sec. 5: the loss composes with loss-parallel sharding of the output projection).

def shard_forward(h, w_shard, targets, v_begin, v_total, ignore_index=-100):
    """Partials of one shard holding ids [v_begin, v_begin + rows of w_shard): per valid row the
    log-sum-exp over the shard's ids and the target logit if the shard holds the target (else 0);
    both 0 on rows that are not valid for the full vocabulary ``v_total``."""
    n = h.shape[0]
    ok, status = valid_rows(targets, v_total, ignore_index)
    rows = np.nonzero(ok)[0]
    t = np.asarray(targets, dtype=np.int64)
    lse_part = np.zeros(n, dtype=np.float64)
    tgt_part = np.zeros(n, dtype=np.float64)
    if rows.size:
        s = h[rows] @ w_shard.T
        m = s.max(axis=1)
        lse_part[rows] = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
        local = t[rows] - v_begin
        own = (local >= 0) & (local < w_shard.shape[0])
        tgt_part[rows[own]] = s[np.nonzero(own)[0], local[own]]
    return {"lse_part": lse_part, "tgt_part": tgt_part, "n_valid": int(rows.size), "status": status}


def combine_shards(lse_parts, tgt_parts, targets, v_total, ignore_index=-100, reduction="mean"):
    """Full-vocabulary lse and loss from the shards' partials ([G, N] each)."""
    ok, status = valid_rows(targets, v_total, ignore_index)
    lp = np.asarray(lse_parts, dtype=np.float64)
    m = lp.max(axis=0)
    lse = np.where(ok, m + np.log(np.exp(lp - m[None, :]).sum(axis=0)), 0.0)
    per_row = np.where(ok, lse - np.asarray(tgt_parts, dtype=np.float64).sum(axis=0), 0.0)
    nv = int(ok.sum())
    if reduction == "none":
        loss = per_row
    elif nv == 0:
        loss = 0.0
    else:
        loss = float(per_row.sum() / nv) if reduction == "mean" else float(per_row.sum())
    return {"loss": loss, "lse": lse, "per_row": per_row, "n_valid": nv, "status": status}


def shard_backward(h, w_shard, targets, lse, v_begin, v_total, n_valid, ignore_index=-100,
                   reduction="mean", grad=1.0):
    """One shard's terms of the gradients, given the full-vocabulary lse: dH_part = G_s W_s (the
    shards' parts sum to dH) and dW_s = G_s^T H (the shard's rows of dW), with
    G_s = c (exp(s - lse) - onehot) over the shard's ids (the onehot only where the shard holds
    the target)."""
    ok, _ = valid_rows(targets, v_total, ignore_index)
    rows = np.nonzero(ok)[0]
    t = np.asarray(targets, dtype=np.int64)
    c = scale_c(n_valid, reduction, grad)
    dh = np.zeros((h.shape[0], w_shard.shape[1]), dtype=np.float64)
    dw = np.zeros_like(w_shard, dtype=np.float64)
    if rows.size:
        s = h[rows] @ w_shard.T
        g = np.exp(s - np.asarray(lse, dtype=np.float64)[rows][:, None])
        local = t[rows] - v_begin
        own = np.nonzero((local >= 0) & (local < w_shard.shape[0]))[0]
        g[own, local[own]] -= 1.0
        cr = (c[rows][:, None] if reduction == "none" else c)
        g = cr * g
        dh[rows] = g @ w_shard
        dw = g.T @ h[rows]
    return {"dH_part": dh, "dW": dw}
