"""Pins of the CPU oracle against what the mathematics fixes (no GPU needed).

The objective is the standard cross-entropy over the full vocabulary (paper
Sec. 3.3: LCE swaps in for the standard CE with a one-line edit; Sec. 4.2: it
fuses the output projection, masks ignored tokens before it and never holds
the dense logits). Every pin below checks the oracle against something other
than itself: an independent library routine, finite differences, closed forms,
or invariants; each is chosen so that a dropped term, a wrong sign or scale, or
a transposed operand fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch

from oracle import lce_oracle as O
from paper_2605_21442_amd import workloads as WL

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _f64(n, d, v, seed=0, sigma_w=0.5, mask=None, ignore=-100):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((n, d))
    w = sigma_w * rng.standard_normal((v, d))
    t = rng.integers(0, v, size=n)
    if mask is not None:
        t[mask] = ignore
    return h, w, t


def _oracle_f64(h, w, t, reduction="mean", grad=1.0, ignore=-100):
    out = O.forward(h, w, t, ignore, reduction)
    out.update(O.backward(h, w, t, ignore, reduction, grad))
    return out


# ---- independent library routine ------------------------------------------------------------

@pytest.mark.parametrize("reduction", ["mean", "sum"])
@pytest.mark.parametrize("shape", [(37, 24, 53), (5, 8, 3), (64, 16, 1000)])
def test_matches_torch_cross_entropy(reduction, shape):
    n, d, v = shape
    h, w, t = _f64(n, d, v, seed=n + v, mask=np.arange(0, n, 4))
    g = 0.75
    ours = _oracle_f64(h, w, t, reduction, grad=g)
    H = torch.tensor(h, requires_grad=True)
    W = torch.tensor(w, requires_grad=True)
    loss = torch.nn.functional.cross_entropy(H @ W.T, torch.tensor(t), ignore_index=-100,
                                             reduction=reduction)
    (loss * g).backward()
    assert abs(ours["loss"] - loss.item()) <= 1e-12 * max(1.0, abs(loss.item()))
    np.testing.assert_allclose(ours["dH"], H.grad.numpy(), rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(ours["dW"], W.grad.numpy(), rtol=1e-11, atol=1e-14)
    lse_ref = torch.logsumexp(H.detach() @ W.detach().T, dim=1).numpy()
    valid = t != -100
    np.testing.assert_allclose(ours["lse"][valid], lse_ref[valid], rtol=1e-13)
    assert np.all(ours["lse"][~valid] == 0.0)
    assert ours["n_valid"] == int(valid.sum())


# ---- central finite differences ---------------------------------------------------------------

@pytest.mark.parametrize("reduction", ["mean", "sum"])
def test_gradients_match_central_differences(reduction):
    n, d, v = 6, 8, 16
    h, w, t = _f64(n, d, v, seed=3, mask=[2])
    g = 1.3
    out = _oracle_f64(h, w, t, reduction, grad=g)
    eps = 1e-6

    def loss_at(hh, ww):
        return g * O.forward(hh, ww, t, -100, reduction)["loss"]

    num_dh = np.zeros_like(h)
    for i in range(n):
        for j in range(d):
            hp, hm = h.copy(), h.copy()
            hp[i, j] += eps
            hm[i, j] -= eps
            num_dh[i, j] = (loss_at(hp, w) - loss_at(hm, w)) / (2 * eps)
    num_dw = np.zeros_like(w)
    for i in range(v):
        for j in range(d):
            wp, wm = w.copy(), w.copy()
            wp[i, j] += eps
            wm[i, j] -= eps
            num_dw[i, j] = (loss_at(h, wp) - loss_at(h, wm)) / (2 * eps)
    scale_h = np.abs(out["dH"]).max()
    scale_w = np.abs(out["dW"]).max()
    assert np.abs(num_dh - out["dH"]).max() <= 1e-7 * scale_h + 1e-10
    assert np.abs(num_dw - out["dW"]).max() <= 1e-7 * scale_w + 1e-10
    assert np.all(out["dH"][2] == 0.0)          # the ignored row gets exactly nothing


# ---- closed forms ------------------------------------------------------------------------------

def test_zero_weight_gives_log_v_and_closed_form_grads():
    n, d, v = 40, 16, 50
    h, _, t = _f64(n, d, v, seed=5, mask=[0, 7, 9])
    w = np.zeros((v, d))
    g = 2.0
    out = _oracle_f64(h, w, t, "mean", grad=g)
    valid = t != -100
    nv = int(valid.sum())
    assert out["loss"] == pytest.approx(math.log(v), abs=1e-13)
    np.testing.assert_allclose(out["lse"][valid], math.log(v), atol=1e-13)
    # dW[v,:] = (g/Nv) * [(1/V) sum_{n in M} H_n - sum_{n in M, t_n = v} H_n]
    ref = np.tile(h[valid].sum(0) / v, (v, 1))
    for i in np.nonzero(valid)[0]:
        ref[t[i]] -= h[i]
    np.testing.assert_allclose(out["dW"], g / nv * ref, atol=1e-13)
    assert np.all(out["dH"] == 0.0)


def test_zero_hidden_closed_form_dh():
    n, d, v = 12, 8, 30
    _, w, t = _f64(n, d, v, seed=6, mask=[4])
    h = np.zeros((n, d))
    out = _oracle_f64(h, w, t, "mean")
    valid = t != -100
    nv = int(valid.sum())
    assert out["loss"] == pytest.approx(math.log(v), abs=1e-13)
    # dH[n,:] = (1/Nv) * [(1/V) sum_v W_v - W_{t_n}] for valid n, 0 otherwise
    for i in range(n):
        ref = (w.mean(0) - w[t[i]]) / nv if valid[i] else np.zeros(d)
        np.testing.assert_allclose(out["dH"][i], ref, atol=1e-14)
    assert np.all(out["dW"] == 0.0)


def test_single_class_vocabulary_is_zero_loss():
    h, w, t = _f64(9, 8, 1, seed=7)
    out = _oracle_f64(h, w, t)
    assert out["loss"] == 0.0
    assert np.all(out["dH"] == 0.0) and np.all(out["dW"] == 0.0)


def test_two_class_vocabulary_is_logistic_loss():
    h, w, t = _f64(20, 8, 2, seed=8)
    out = _oracle_f64(h, w, t, "sum")
    s = h @ w.T
    other = 1 - t
    margin = s[np.arange(20), other] - s[np.arange(20), t]
    softplus = np.logaddexp(0.0, margin)
    assert out["loss"] == pytest.approx(softplus.sum(), rel=1e-13)


def test_geometric_series_vocabulary_pins_every_target_id():
    # H = e_0 and W[v, 0] = v / 64 give s[n, v] = v / 64 exactly in bf16;
    # lse = ln sum_v e^{v/64} = ln((e^4 - 1) / (e^{1/64} - 1)) and l_n = lse - t_n / 64.
    v, d = 256, 8
    one = np.uint16(0x3F80)
    h_bits = np.zeros((v, d), np.uint16)
    h_bits[:, 0] = one
    w32 = np.zeros((v, d), np.float32)
    w32[:, 0] = np.arange(v, dtype=np.float32) / 64.0
    w_bits = WL.f32_to_bf16_bits(w32)
    assert np.array_equal(WL.bf16_bits_to_f32(w_bits)[:, 0], w32[:, 0])   # exact in bf16
    t = np.arange(v, dtype=np.int32)                                       # every id once
    out = O.lce(h_bits, w_bits, t, reduction="sum")
    lse = math.log(math.expm1(4.0) / math.expm1(1.0 / 64.0))
    np.testing.assert_allclose(out["lse"], lse, rtol=1e-14)
    np.testing.assert_allclose(out["per_row"], lse - t / 64.0, rtol=1e-13, atol=1e-13)


# ---- invariants -------------------------------------------------------------------------------

def test_softmax_grad_rows_sum_to_zero():
    h, w, t = _f64(30, 12, 70, seed=9, mask=[1, 2])
    out = _oracle_f64(h, w, t)
    assert np.abs(out["dW"].sum(axis=0)).max() <= 1e-15 * 70 * 30
    # G has exactly one negative entry per valid row, at its target
    r = np.nonzero(t != -100)[0][:5]
    g = O.softmax_grad_rows(h[r], w, t[r], 1.0)
    for i in range(5):
        neg = np.nonzero(g[i] < 0)[0]
        assert neg.size == 1 and neg[0] == t[r[i]]


def test_masked_rows_change_nothing():
    n, d, v = 25, 10, 40
    mask = [0, 3, 11, 24]
    h, w, t = _f64(n, d, v, seed=10, mask=mask)
    a = _oracle_f64(h, w, t)
    h2 = h.copy()
    h2[mask] = 1e3 * np.random.default_rng(1).standard_normal((len(mask), d))
    b = _oracle_f64(h2, w, t)
    assert a["loss"] == b["loss"]
    np.testing.assert_array_equal(a["dW"], b["dW"])
    np.testing.assert_array_equal(a["dH"][mask], 0.0)
    np.testing.assert_array_equal(b["dH"][mask], 0.0)
    valid = np.setdiff1d(np.arange(n), mask)
    np.testing.assert_array_equal(a["lse"][valid], b["lse"][valid])


def test_sum_is_nv_times_mean_and_duplication_keeps_mean():
    h, w, t = _f64(17, 6, 23, seed=11, mask=[5])
    mean = _oracle_f64(h, w, t, "mean")
    tot = _oracle_f64(h, w, t, "sum")
    assert tot["loss"] == pytest.approx(mean["n_valid"] * mean["loss"], rel=1e-14)
    np.testing.assert_allclose(tot["dW"], mean["n_valid"] * mean["dW"], rtol=1e-12, atol=1e-15)
    dup = _oracle_f64(np.vstack([h, h]), w, np.concatenate([t, t]), "mean")
    assert dup["loss"] == pytest.approx(mean["loss"], rel=1e-13)


def test_shift_of_weight_rows_leaves_everything_unchanged():
    h, w, t = _f64(15, 6, 19, seed=12)
    c = np.random.default_rng(2).standard_normal(6)
    a = _oracle_f64(h, w, t)
    b = _oracle_f64(h, w + c[None, :], t)
    assert b["loss"] == pytest.approx(a["loss"], rel=1e-12)
    np.testing.assert_allclose(b["dH"], a["dH"], atol=1e-12)
    np.testing.assert_allclose(b["dW"], a["dW"], atol=1e-12)


def test_vocab_and_token_permutations_are_equivariant():
    h, w, t = _f64(14, 6, 21, seed=13, mask=[3])
    a = _oracle_f64(h, w, t)
    rng = np.random.default_rng(4)
    pv = rng.permutation(21)            # new id j holds old id pv[j]
    inv = np.argsort(pv)
    t2 = np.where(t == -100, -100, inv[np.where(t == -100, 0, t)])
    b = _oracle_f64(h, w[pv], t2)
    assert b["loss"] == pytest.approx(a["loss"], rel=1e-13)
    np.testing.assert_allclose(b["dW"], a["dW"][pv], atol=1e-14)
    pn = rng.permutation(14)
    c = _oracle_f64(h[pn], w, t[pn])
    np.testing.assert_allclose(c["dH"], a["dH"][pn], atol=1e-14)


def test_all_masked_is_zero_not_nan():
    h, w, t = _f64(8, 4, 5, seed=14, mask=np.arange(8))
    out = _oracle_f64(h, w, t)
    assert out["n_valid"] == 0 and out["loss"] == 0.0
    assert np.all(out["dH"] == 0.0) and np.all(out["dW"] == 0.0)
    assert np.all(out["lse"] == 0.0)


def test_out_of_range_targets_are_flagged_and_ignored():
    h, w, t = _f64(10, 4, 7, seed=15)
    t_bad = t.copy()
    t_bad[2] = 7
    t_bad[5] = -3
    out = _oracle_f64(h, w, t_bad)
    assert out["status"] == O.STATUS_TARGET_OUT_OF_RANGE
    t_ign = t.copy()
    t_ign[[2, 5]] = -100
    ref = _oracle_f64(h, w, t_ign)
    assert out["loss"] == ref["loss"] and out["n_valid"] == 8
    np.testing.assert_array_equal(out["dW"], ref["dW"])
    assert _oracle_f64(h, w, t)["status"] == 0


def test_custom_ignore_index():
    h, w, t = _f64(10, 4, 7, seed=16)
    t[[1, 4]] = 3
    a = O.forward(h, w, t, ignore_index=3)
    assert a["n_valid"] == 10 - int((t == 3).sum())


# ---- sampled-output helpers agree with the whole oracle -------------------------------------

def test_sampled_helpers_match_full_oracle():
    inp = WL.custom(48, 32, 300, seed=3, mask_frac=0.25)
    full = O.lce(inp.h_bits, inp.w_bits, inp.targets)
    valid = np.nonzero(inp.targets != -100)[0]
    rows = np.array([0, 5, 17, 47])
    lse_r = O.lse_of_rows(inp.h_bits, inp.w_bits, valid[:6])
    np.testing.assert_allclose(lse_r, full["lse"][valid[:6]], rtol=1e-14)
    dh = O.dh_of_rows(inp.h_bits, inp.w_bits, inp.targets, rows, full["n_valid"])
    np.testing.assert_allclose(dh, full["dH"][rows], rtol=1e-12, atol=1e-16)
    vrows = np.array([0, 1, 150, 299])
    dw = O.dw_of_rows(inp.h_bits, inp.w_bits, inp.targets, vrows, full["lse"], block=7)
    np.testing.assert_allclose(dw, full["dW"][vrows], rtol=1e-11, atol=1e-16)


# ---- statistical sanity (gross-error detector, not parity) ----------------------------------

def test_expected_loss_of_random_head():
    wl = WL.WORKLOADS["tiny"]
    inp = WL.generate(wl, seed=0)
    out = O.lce(inp.h_bits, inp.w_bits, inp.targets)
    expect = math.log(wl.v) + wl.sigma_w ** 2 * wl.d / 2
    assert abs(out["loss"] - expect) < 0.05
    assert out["n_valid"] == wl.n_valid()


# ---- per-token losses (reduction "none") ------------------------------------------------------

def test_none_reduction_matches_torch_per_token_losses():
    n, d, v = 41, 16, 77
    h, w, t = _f64(n, d, v, seed=21, mask=np.arange(0, n, 5))
    g = np.random.default_rng(3).standard_normal(n)
    ours = _oracle_f64(h, w, t, "none", grad=g)
    H = torch.tensor(h, requires_grad=True)
    W = torch.tensor(w, requires_grad=True)
    per = torch.nn.functional.cross_entropy(H @ W.T, torch.tensor(t), ignore_index=-100,
                                            reduction="none")
    (per * torch.tensor(g)).sum().backward()
    np.testing.assert_allclose(ours["loss"], per.detach().numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(ours["dH"], H.grad.numpy(), rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(ours["dW"], W.grad.numpy(), rtol=1e-11, atol=1e-14)
    assert np.all(ours["loss"][t == -100] == 0.0)


def test_none_reduction_sums_to_sum_reduction():
    h, w, t = _f64(30, 12, 50, seed=22, mask=[3, 4])
    per = _oracle_f64(h, w, t, "none", grad=np.ones(30))
    tot = _oracle_f64(h, w, t, "sum", grad=1.0)
    assert per["loss"].sum() == pytest.approx(tot["loss"], rel=1e-13)
    np.testing.assert_allclose(per["dW"], tot["dW"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(per["dH"], tot["dH"], rtol=1e-12, atol=1e-15)


def test_none_reduction_gradient_of_one_token_is_central_difference():
    n, d, v = 5, 6, 9
    h, w, t = _f64(n, d, v, seed=23)
    g = np.zeros(n)
    g[2] = 1.0                                    # gradient of token 2's loss alone
    out = _oracle_f64(h, w, t, "none", grad=g)
    eps = 1e-6
    num = np.zeros_like(w)
    for i in range(v):
        for j in range(d):
            wp, wm = w.copy(), w.copy()
            wp[i, j] += eps
            wm[i, j] -= eps
            num[i, j] = (O.forward(h, wp, t, -100, "none")["loss"][2]
                         - O.forward(h, wm, t, -100, "none")["loss"][2]) / (2 * eps)
    assert np.abs(num - out["dW"]).max() <= 1e-7 * np.abs(out["dW"]).max() + 1e-10
    assert np.all(out["dH"][[0, 1, 3, 4]] == 0.0)


# ---- vocabulary-parallel decomposition ----------------------------------------------------------

@pytest.mark.parametrize("reduction", ["mean", "sum", "none"])
@pytest.mark.parametrize("cuts", [[0, 53], [0, 1, 20, 52, 53], [0, 52, 53]])
def test_shard_partials_combine_to_the_full_objective(reduction, cuts):
    n, d, v = 19, 7, 53
    h, w, t = _f64(n, d, v, seed=11, mask=np.array([2, 5]))
    t[7] = v + 3                                      # out of range: ignored and flagged
    g = np.linspace(-1, 2, n) if reduction == "none" else 0.5
    full = _oracle_f64(h, w, t, reduction, grad=g)
    parts = [O.shard_forward(h, w[a:b], t, a, v) for a, b in zip(cuts[:-1], cuts[1:])]
    comb = O.combine_shards(np.stack([p["lse_part"] for p in parts]),
                            np.stack([p["tgt_part"] for p in parts]), t, v, reduction=reduction)
    assert comb["n_valid"] == full["n_valid"] and comb["status"] == full["status"] == 1
    np.testing.assert_allclose(comb["lse"], full["lse"], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(comb["loss"], full["loss"], rtol=1e-12, atol=1e-13)
    # exactly one shard holds each valid target
    owners = sum((t - a >= 0) & (t - a < b - a) for a, b in zip(cuts[:-1], cuts[1:]))
    valid = (t != -100) & (t >= 0) & (t < v)
    assert np.all(owners[valid] == 1)
    bw = [O.shard_backward(h, w[a:b], t, comb["lse"], a, v, comb["n_valid"], reduction=reduction, grad=g)
          for a, b in zip(cuts[:-1], cuts[1:])]
    np.testing.assert_allclose(sum(b["dH_part"] for b in bw), full["dH"], rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(np.concatenate([b["dW"] for b in bw]), full["dW"], rtol=1e-11, atol=1e-14)


# ---- the backward by vocabulary chunks (full-size checks) -------------------------------------

@pytest.mark.parametrize("reduction", ["mean", "sum", "none"])
@pytest.mark.parametrize("chunk,block", [(7, 5), (53, 64), (20, 1)])
def test_backward_by_vocab_chunks_matches_torch_autograd(reduction, chunk, block):
    inp = WL.custom(37, 24, 53, seed=41, mask_frac=0.25, sigma_w=0.5)
    h, w = O.bf16_to_f64(inp.h_bits), O.bf16_to_f64(inp.w_bits)
    t = inp.targets.astype(np.int64)
    g = np.linspace(0.5, 1.5, 37) if reduction == "none" else 0.75
    H = torch.tensor(h, requires_grad=True)
    W = torch.tensor(w, requires_grad=True)
    loss = torch.nn.functional.cross_entropy(H @ W.T, torch.tensor(t), ignore_index=-100, reduction=reduction)
    (loss * torch.tensor(g)).sum().backward()
    lse = O.forward(h, w, t, -100, reduction)["lse"]
    got = {}
    rows, dh = O.backward_by_vocab_chunks(inp.h_bits, inp.w_bits, inp.targets, lse,
                                          lambda v0, dw: got.__setitem__(v0, dw), reduction=reduction,
                                          grad=g, chunk=chunk, block=block)
    dw = np.concatenate([got[k] for k in sorted(got)])
    assert sorted(got) == list(range(0, 53, chunk))
    full_dh = np.zeros_like(h)
    full_dh[rows] = dh
    np.testing.assert_allclose(full_dh, H.grad.numpy(), rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(dw, W.grad.numpy(), rtol=1e-11, atol=1e-14)
    assert np.array_equal(rows, np.nonzero(inp.targets != -100)[0])


def test_backward_by_vocab_chunks_matches_the_whole_oracle():
    inp = WL.custom(300, 64, 1000, seed=42, mask_frac=0.3, sigma_w=0.2, targets="zipf")
    full = O.lce(inp.h_bits, inp.w_bits, inp.targets)
    parts = []
    rows, dh = O.backward_by_vocab_chunks(inp.h_bits, inp.w_bits, inp.targets, full["lse"],
                                          lambda v0, dw: parts.append((v0, dw)), chunk=384, block=100)
    np.testing.assert_allclose(dh, full["dH"][rows], rtol=1e-12, atol=1e-17)
    np.testing.assert_allclose(np.concatenate([p for _, p in parts]), full["dW"], rtol=1e-11, atol=1e-17)
    assert np.all(full["dH"][np.setdiff1d(np.arange(300), rows)] == 0.0)
