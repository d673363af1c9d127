"""Pins of the KD oracle (soft-target cross-entropy of two heads) -- no GPU needed.

Checked against torch's cross-entropy with probability targets and autograd, torch's KL
divergence plus the teacher entropy, central finite differences, and closed forms; a
dropped 1/T, a swapped student/teacher or a missing mask fails at least one of them.
"""
import numpy as np
import pytest
import torch

from oracle import kd_oracle as K


def _heads(n=13, ds=6, dt=9, v=21, seed=0, sw=0.7, tw=0.9):
    rng = np.random.default_rng(seed)
    hs, ht = rng.standard_normal((n, ds)), rng.standard_normal((n, dt))
    ws, wt = sw * rng.standard_normal((v, ds)), tw * rng.standard_normal((v, dt))
    t = rng.integers(0, v, n)
    t[[1, 4]] = -100
    return hs, ws, ht, wt, t


@pytest.mark.parametrize("reduction", ["mean", "sum", "none"])
@pytest.mark.parametrize("temperature", [1.0, 2.5])
def test_matches_torch_soft_target_cross_entropy(reduction, temperature):
    hs, ws, ht, wt, t = _heads()
    n = hs.shape[0]
    g = np.linspace(-1, 1, n) if reduction == "none" else 0.8
    ours = K.kd(hs, ws, ht, wt, t, temperature=temperature, reduction=reduction, grad=g)
    Hs, Ws = torch.tensor(hs, requires_grad=True), torch.tensor(ws, requires_grad=True)
    valid = torch.tensor(t != -100)
    zs = (Hs @ Ws.T) / temperature
    pt = torch.softmax(torch.tensor(ht @ wt.T) / temperature, dim=1)
    per = torch.nn.functional.cross_entropy(zs, pt, reduction="none") * valid
    if reduction == "mean":
        loss = per.sum() / valid.sum()
    elif reduction == "sum":
        loss = per.sum()
    else:
        loss = per
    (loss * torch.tensor(g, dtype=torch.float64)).sum().backward()
    np.testing.assert_allclose(ours["loss"], loss.detach().numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(ours["dHs"], Hs.grad.numpy(), rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(ours["dWs"], Ws.grad.numpy(), rtol=1e-10, atol=1e-13)


def test_kl_divergence_plus_teacher_entropy():
    hs, ws, ht, wt, t = _heads(seed=3)
    out = K.kd(hs, ws, ht, wt, t, reduction="none")
    logps = torch.log_softmax(torch.tensor(hs @ ws.T), dim=1)
    pt = torch.softmax(torch.tensor(ht @ wt.T), dim=1)
    kl = torch.nn.functional.kl_div(logps, pt, reduction="none").sum(1).numpy()
    ent = -(pt * torch.log(pt)).sum(1).numpy()
    valid = t != -100
    np.testing.assert_allclose(out["loss"][valid], (kl + ent)[valid], rtol=1e-12)
    assert np.all(out["loss"][~valid] == 0.0)


def test_finite_differences():
    hs, ws, ht, wt, t = _heads(n=5, ds=4, dt=3, v=7, seed=5)
    T = 1.7
    out = K.kd(hs, ws, ht, wt, t, temperature=T)
    eps = 1e-6
    for arr, grad in ((hs, out["dHs"]), (ws, out["dWs"])):
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            up = K.kd(hs, ws, ht, wt, t, temperature=T)["loss"]
            arr[idx] = old - eps
            dn = K.kd(hs, ws, ht, wt, t, temperature=T)["loss"]
            arr[idx] = old
            assert abs((up - dn) / (2 * eps) - grad[idx]) <= 1e-7 * max(1.0, abs(grad[idx]))


def test_zero_student_head_gives_log_v():
    hs, ws, ht, wt, t = _heads(v=33, seed=7)
    out = K.kd(hs, 0 * ws, ht, wt, t)
    assert abs(out["loss"] - np.log(33)) <= 1e-12


def test_student_equal_to_teacher():
    hs, ws, _, _, t = _heads(ds=6, dt=6, seed=8)
    out = K.kd(hs, ws, hs.copy(), ws.copy(), t, temperature=1.3, reduction="none")
    z = hs @ ws.T / 1.3
    p = np.exp(z - z.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    ent = -(p * np.log(p)).sum(1)
    valid = t != -100
    np.testing.assert_allclose(out["loss"][valid], ent[valid], rtol=1e-12)
    assert np.abs(out["dHs"]).max() <= 1e-14 and np.abs(out["dWs"]).max() <= 1e-14


def test_sampled_rows_helper_matches_whole_oracle():
    from oracle import lce_oracle as O
    rng = np.random.default_rng(2)
    bits = lambda a: (np.asarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    hs, ws, ht, wt, t = _heads(seed=9)
    hs_b, ws_b, ht_b, wt_b = bits(hs), bits(ws), bits(ht), bits(wt)
    whole = K.kd_bits(hs_b, ws_b, ht_b, wt_b, t, temperature=2.0, reduction="none")
    rows = np.array([0, 1, 5, 12])
    part = K.kd_rows(hs_b, ws_b, ht_b, wt_b, t, rows, temperature=2.0)
    np.testing.assert_allclose(part["per_row"], whole["loss"][rows], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(part["lse_t"], whole["lse_t"][rows], rtol=1e-13, atol=1e-15)


def test_sampled_gradient_rows_match_whole_oracle():
    bits = lambda a: (np.asarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    hs, ws, ht, wt, t = _heads(n=40, v=50, seed=10)
    hs_b, ws_b, ht_b, wt_b = bits(hs), bits(ws), bits(ht), bits(wt)
    whole = K.kd_bits(hs_b, ws_b, ht_b, wt_b, t, temperature=2.0, grad=1.5)
    rows = np.array([0, 1, 4, 39])
    dh = K.kd_dh_rows(hs_b, ws_b, ht_b, wt_b, t, rows, whole["n_valid"], temperature=2.0, grad=1.5)
    np.testing.assert_allclose(dh, whole["dHs"][rows], rtol=1e-11, atol=1e-15)
    ids = np.array([0, 7, 49])
    dw = K.kd_dw_rows(hs_b, ws_b, ht_b, wt_b, t, ids, whole["lse_s"], whole["lse_t"], temperature=2.0, grad=1.5,
                      block=16)
    np.testing.assert_allclose(dw, whole["dWs"][ids], rtol=1e-11, atol=1e-15)
