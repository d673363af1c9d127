"""Plain CPU oracle of the fused linear knowledge-distillation (KD) loss.

TEST INFRASTRUCTURE ONLY. Only the tests, the package's ``smoke()`` check and
the benchmark's CPU-baseline leg may import this module. The product path never
calls it and shares no code with it.

What it computes: the paper's recipes include knowledge distillation with
dedicated KD losses (Sec. 3.2) and cite Hinton et al. (2015) for it (Sec. 2); the loss
there is the cross-entropy of the student's softened predictions against the
teacher's softened predictions. Applied to the two models' output heads, the
same way LCE applies the hard-label cross-entropy to one head (Sec. 4.2):

  valid set   M = {n : t_n != ignore_index and 0 <= t_n < V},  Nv = |M|   (labels only mask)
  logits      zs = Hs Ws^T / T,  zt = Ht Wt^T / T        (student [N, Ds], [V, Ds]; teacher [N, Dt], [V, Dt])
  soft target p_t = softmax(zt),  p_s = softmax(zs)
  per token   l_n = - sum_v p_t(v) log p_s(v) = lse(zs_n) - sum_v p_t(v) zs_n(v)          (n in M)
  reduction   mean over M, sum over M, or the per-token vector (0 outside M)
  gradient    dL/dzs = c (p_s - p_t),  with dzs/d(Hs Ws^T) = 1/T:
              G = c (p_s - p_t) / T,  dHs = G Ws,  dWs = G^T Hs       (the teacher gets none)
  c           g / Nv (mean), g (sum), g_n (none)

Readings where the paper is silent: T is a parameter (default 1) and the loss is not
multiplied by T^2 (a caller that wants Hinton's T^2 weighting scales g); the loss is the
soft-target cross-entropy, which differs from KL(p_t || p_s) by the teacher's entropy (a
constant for the student, so the gradients agree); labels act only as the mask.

Pins (``tests/test_kd_oracle.py``): torch's cross-entropy with probability targets and
autograd (an independent library routine), torch's KL divergence plus the teacher entropy,
central finite differences, and closed forms (a zero student head gives ln V; a student
identical to the teacher has zero gradient and loss equal to the teacher's entropy).
"""
from __future__ import annotations

import numpy as np

from .lce_oracle import bf16_to_f64, scale_c, valid_rows


def _lse(z):
    m = z.max(axis=1)
    return m + np.log(np.exp(z - m[:, None]).sum(axis=1))


def kd(hs, ws, ht, wt, targets, temperature=1.0, ignore_index=-100, reduction="mean", grad=1.0,
       block=512, grads=True):
    """Loss, lse of both heads (0 outside M), Nv, status, dHs and dWs (unless grads=False), all
    float64."""
    n, v = hs.shape[0], ws.shape[0]
    ok, status = valid_rows(targets, v, ignore_index)
    rows = np.nonzero(ok)[0]
    nv = int(rows.size)
    c = scale_c(nv, reduction, grad)
    if reduction == "none":
        c = np.broadcast_to(c, (n,))
    lse_s = np.zeros(n)
    lse_t = np.zeros(n)
    per_row = np.zeros(n)
    dhs = np.zeros_like(hs)
    dws = np.zeros_like(ws)
    for s0 in range(0, nv, block):
        r = rows[s0:s0 + block]
        zs = hs[r] @ ws.T / temperature
        zt = ht[r] @ wt.T / temperature
        ls, lt = _lse(zs), _lse(zt)
        lse_s[r], lse_t[r] = ls, lt
        pt = np.exp(zt - lt[:, None])
        ps = np.exp(zs - ls[:, None])
        per_row[r] = ls - (pt * zs).sum(axis=1)
        if not grads:
            continue
        cr = c[r][:, None] if reduction == "none" else c
        g = cr * (ps - pt) / temperature
        dhs[r] = g @ ws
        dws += g.T @ hs[r]
    if reduction == "none":
        loss = per_row.copy()
    elif nv == 0:
        loss = 0.0
    else:
        loss = float(per_row[rows].sum() / nv) if reduction == "mean" else float(per_row[rows].sum())
    return {"loss": loss, "per_row": per_row, "lse_s": lse_s, "lse_t": lse_t, "n_valid": nv,
            "status": status, "dHs": dhs, "dWs": dws}


def kd_bits(hs_bits, ws_bits, ht_bits, wt_bits, targets, **kw):
    """``kd`` from bf16 bit patterns."""
    return kd(bf16_to_f64(hs_bits), bf16_to_f64(ws_bits), bf16_to_f64(ht_bits), bf16_to_f64(wt_bits),
              targets, **kw)


def kd_rows(hs_bits, ws_bits, ht_bits, wt_bits, targets, rows, temperature=1.0, ignore_index=-100):
    """Per-token loss, lse_s and lse_t of the given rows only (sampling at full size)."""
    v = ws_bits.shape[0]
    ok, _ = valid_rows(targets, v, ignore_index)
    ws = bf16_to_f64(ws_bits)
    wt = bf16_to_f64(wt_bits)
    out = {"per_row": np.zeros(len(rows)), "lse_s": np.zeros(len(rows)), "lse_t": np.zeros(len(rows))}
    for i, r in enumerate(rows):
        if not ok[r]:
            continue
        zs = bf16_to_f64(hs_bits[r:r + 1]) @ ws.T / temperature
        zt = bf16_to_f64(ht_bits[r:r + 1]) @ wt.T / temperature
        ls, lt = _lse(zs)[0], _lse(zt)[0]
        pt = np.exp(zt[0] - lt)
        out["per_row"][i] = ls - float(pt @ zs[0])
        out["lse_s"][i], out["lse_t"][i] = ls, lt
    return out


def kd_dh_rows(hs_bits, ws_bits, ht_bits, wt_bits, targets, rows, n_valid, temperature=1.0,
               ignore_index=-100, grad=1.0):
    """Rows of dHs = G Ws for the mean reduction (zero for rows outside M)."""
    v = ws_bits.shape[0]
    ok, _ = valid_rows(targets, v, ignore_index)
    ws = bf16_to_f64(ws_bits)
    wt = bf16_to_f64(wt_bits)
    c = scale_c(n_valid, "mean", grad)
    out = np.zeros((len(rows), ws.shape[1]))
    for i, r in enumerate(rows):
        if not ok[r]:
            continue
        zs = bf16_to_f64(hs_bits[r:r + 1]) @ ws.T / temperature
        zt = bf16_to_f64(ht_bits[r:r + 1]) @ wt.T / temperature
        ps = np.exp(zs - _lse(zs)[:, None])
        pt = np.exp(zt - _lse(zt)[:, None])
        out[i] = ((c * (ps - pt) / temperature) @ ws)[0]
    return out


def kd_dw_rows(hs_bits, ws_bits, ht_bits, wt_bits, targets, vrows, lse_s, lse_t, temperature=1.0,
               ignore_index=-100, grad=1.0, block=4096):
    """Rows of dWs = G^T Hs (mean reduction) for vocabulary ids ``vrows``, given the oracle's lse of
    both heads for every row."""
    v = ws_bits.shape[0]
    ok, _ = valid_rows(targets, v, ignore_index)
    rows = np.nonzero(ok)[0]
    c = scale_c(int(rows.size), "mean", grad)
    wsv = bf16_to_f64(ws_bits[np.asarray(vrows)])
    wtv = bf16_to_f64(wt_bits[np.asarray(vrows)])
    out = np.zeros((len(vrows), ws_bits.shape[1]))
    for s0 in range(0, rows.size, block):
        r = rows[s0:s0 + block]
        hs = bf16_to_f64(hs_bits[r])
        ps = np.exp(hs @ wsv.T / temperature - lse_s[r][:, None])
        pt = np.exp(bf16_to_f64(ht_bits[r]) @ wtv.T / temperature - lse_t[r][:, None])
        out += (c * (ps - pt) / temperature).T @ hs
    return out
