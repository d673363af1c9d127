"""HIP path vs the CPU oracle, element by element, at sizes the oracle finishes in seconds.

Cases span several 256-wide tiles with ragged tails in every dimension, the
degenerate shapes of the objective (one token, one class, no valid token, no
masked token), both target widths, both reductions, a non-unit upstream
gradient, a strided hidden-state view and several backward vocabulary slabs.
Tolerances (mean-loss absolute error <= 1e-3, relative Frobenius error <= 1e-2
on dH and dW) are the ones the method is held to; lse is held to 1e-3 per row.
"""
import math

import numpy as np
import pytest

from oracle import lce_oracle as O
from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U

pytestmark = pytest.mark.gpu


def _case(inp, reduction="mean", grad=1.0, target_dtype=None):
    import torch
    h, w, t = U.to_device(inp, target_dtype=target_dtype)
    print(f"case n={inp.h_bits.shape[0]} d={inp.h_bits.shape[1]} v={inp.w_bits.shape[0]} "
          f"red={reduction} g={grad}", flush=True)
    gpu = U.run_gpu(h, w, t, inp.ignore_index, reduction, grad)
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets, inp.ignore_index, reduction, grad)
    U.assert_parity(gpu, ref)
    return gpu, ref


def test_tiny_workload():
    gpu, ref = _case(WL.generate(WL.WORKLOADS["tiny"], seed=0))
    ignored = WL.generate(WL.WORKLOADS["tiny"], seed=0).targets == -100
    assert np.all(gpu["dH"][ignored] == 0.0)


@pytest.mark.parametrize("n,d,v", [(300, 264, 1000), (700, 136, 4097), (257, 64, 9000),
                                   (1, 8, 5), (33, 72, 1), (40, 16, 2), (513, 520, 300)])
def test_ragged_shapes(n, d, v):
    _case(WL.custom(n, d, v, seed=n + v, mask_frac=0.15, sigma_w=0.3))


@pytest.mark.parametrize("n,d,v", [(768, 128, 1536), (512, 256, 768), (1152, 64, 3072)])
def test_tile_exact_shapes(n, d, v):
    # every count a whole number of tiles (no ragged tile anywhere): N and V multiples of 384 and
    # 256, no masked token, so Nv = N
    _case(WL.custom(n, d, v, seed=n + d, mask_frac=0.0, sigma_w=0.3))


@pytest.mark.parametrize("n,d,v", [(300, 64, 24588), (200, 128, 24577)])
def test_last_slab_shorter_than_one_k_slice(n, d, v):
    # 24576-id slabs at these widths: the last slab holds 12 ids (1 id), less than one 64-wide K
    # slice, so in the split dH launches (fewer output tiles than CUs: eight K parts) every part
    # past the first is empty and only writes zeros into its accumulator
    _case(WL.custom(n, d, v, seed=n + v, mask_frac=0.2, sigma_w=0.3))


@pytest.mark.parametrize("n,d,v", [(300, 64, 40000), (270, 128, 60000), (520, 64, 90000)])
def test_forward_vocabulary_groups(n, d, v):
    # with D % 64 == 0 the forward runs one launch per group of 384-id tiles as wide as a backward
    # slab (24576 ids at these widths): 2, 3 and 4 groups, a ragged last group, both partial row
    # sets and the running pair
    _case(WL.custom(n, d, v, seed=n + d, mask_frac=0.2, sigma_w=0.3))


def test_sum_reduction_and_upstream_gradient():
    _case(WL.custom(300, 128, 2000, seed=2, mask_frac=0.3), reduction="sum", grad=0.37)
    _case(WL.custom(300, 128, 2000, seed=2, mask_frac=0.3), reduction="mean", grad=-2.5)


def test_int64_targets():
    import torch
    _case(WL.custom(260, 96, 777, seed=4, mask_frac=0.2), target_dtype=torch.int64)


def test_no_masked_tokens_and_all_masked():
    _case(WL.custom(270, 64, 600, seed=5, mask_frac=0.0))
    inp = WL.custom(270, 64, 600, seed=6, mask_frac=1.0)
    assert np.all(inp.targets == -100)
    gpu, _ = _case(inp)
    assert gpu["loss"] == 0.0 and gpu["n_valid"] == 0
    assert np.all(gpu["dH"] == 0.0) and np.all(gpu["dW"] == 0.0) and np.all(gpu["lse"] == 0.0)


def test_targets_at_tile_edges():
    v = 4097
    edges = np.array([0, 1, 255, 256, 257, 511, 512, 4095, 4096, 2048, 4094, 3], dtype=np.int32)
    t = np.resize(edges, 300)
    _case(WL.custom(300, 64, v, seed=7, target_override=t, sigma_w=0.5))


def test_out_of_range_targets_are_flagged_and_ignored():
    inp = WL.custom(200, 64, 500, seed=8, mask_frac=0.1)
    inp.targets[[3, 50, 199]] = [500, -7, 100000]
    gpu, ref = _case(inp)
    assert gpu["status"] == O.STATUS_TARGET_OUT_OF_RANGE
    assert np.all(gpu["dH"][[3, 50, 199]] == 0.0)


def test_custom_ignore_index():
    inp = WL.custom(200, 64, 500, seed=9, mask_frac=0.0)
    inp.targets[::5] = 7
    inp.ignore_index = 7
    gpu, ref = _case(inp)
    assert gpu["n_valid"] == 200 - int((inp.targets == 7).sum())


def test_zero_weight_closed_form():
    inp = WL.custom(300, 128, 3000, seed=10, mask_frac=0.1)
    inp.w_bits[:] = 0
    gpu, ref = _case(inp)
    assert abs(gpu["loss"] - math.log(3000)) <= 1e-5
    valid = inp.targets != -100
    assert np.max(np.abs(gpu["lse"][valid] - math.log(3000))) <= 1e-5
    assert np.all(gpu["dH"] == 0.0)


def test_strided_hidden_view():
    import torch
    from paper_2605_21442_amd import autograd as A
    inp = WL.custom(280, 96, 900, seed=11, mask_frac=0.2)
    h, w, t = U.to_device(inp)
    wide = torch.zeros((280, 160), dtype=torch.bfloat16, device=h.device)
    wide[:, 32:128] = h
    hv = wide[:, 32:128]
    assert hv.stride(0) == 160
    gpu = U.run_gpu(hv, w, t)
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets)
    U.assert_parity(gpu, ref)


def test_expanded_hidden_matches_its_contiguous_copy():
    # an expand()ed hidden (row stride 0) must be made dense before the call, not passed as ld 0
    import torch
    inp = WL.custom(300, 128, 1000, seed=15, mask_frac=0.2)
    h, w, t = U.to_device(inp)
    he = h[:1].expand(300, 128)
    assert he.stride(0) == 0
    a = U.run_gpu(he, w, t)
    b = U.run_gpu(he.contiguous(), w, t)
    assert a["loss"] == b["loss"]
    assert torch.equal(a["dH_t"], b["dH_t"]) and torch.equal(a["dW_t"], b["dW_t"])
    rows = np.repeat(inp.h_bits[:1], 300, axis=0)
    U.assert_parity(a, O.lce(rows, inp.w_bits, inp.targets))


def test_softmax_grad_rows_sum_to_zero_on_gpu():
    inp = WL.custom(600, 256, 5000, seed=12, mask_frac=0.2, sigma_w=0.1)
    h, w, t = U.to_device(inp)
    gpu = U.run_gpu(h, w, t)
    col = gpu["dW"].sum(axis=0)
    # exact arithmetic gives 0; bf16 rounding of G and of dW bounds each column by ~2^-8 sum|dW|
    budget = 4 * 2.0 ** -8 * np.abs(gpu["dW"]).sum(axis=0)
    assert np.all(np.abs(col) <= budget)


def test_deterministic_bits():
    import torch
    inp = WL.custom(520, 200, 3000, seed=13, mask_frac=0.25)
    h, w, t = U.to_device(inp)
    a = U.run_gpu(h, w, t)
    b = U.run_gpu(h, w, t)
    assert a["loss"] == b["loss"]
    assert torch.equal(a["lse_t"], b["lse_t"])
    assert torch.equal(a["dH_t"], b["dH_t"]) and torch.equal(a["dW_t"], b["dW_t"])


def test_autograd_function_matches_oracle():
    import torch
    from paper_2605_21442_amd import linear_cross_entropy
    inp = WL.custom(3 * 100, 128, 1500, seed=14, mask_frac=0.2)
    h, w, t = U.to_device(inp)
    h3 = h.view(3, 100, 128).clone().requires_grad_(True)
    w1 = w.clone().requires_grad_(True)
    loss = linear_cross_entropy(h3, w1, t.view(3, 100).long())
    (2.0 * loss).backward()
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets, grad=2.0)
    assert abs(loss.item() - ref["loss"]) <= U.LOSS_ABS_TOL
    assert U.rel_fro(h3.grad.view(300, 128).float().cpu().numpy(), ref["dH"]) <= U.GRAD_REL_TOL
    assert U.rel_fro(w1.grad.float().cpu().numpy(), ref["dW"]) <= U.GRAD_REL_TOL


@pytest.mark.parametrize("n,d,v", [(300, 264, 1000), (600, 128, 9000), (1, 8, 5)])
def test_per_token_losses_and_gradients(n, d, v):
    inp = WL.custom(n, d, v, seed=n + 3, mask_frac=0.2, sigma_w=0.3)
    g = np.random.default_rng(n).standard_normal(n).astype(np.float32)
    gpu, ref = _case(inp, reduction="none", grad=g)
    assert np.all(gpu["loss"][inp.targets == -100] == 0.0)


def test_per_token_autograd_shape():
    import torch
    from paper_2605_21442_amd import linear_cross_entropy
    inp = WL.custom(2 * 150, 96, 700, seed=31, mask_frac=0.1)
    h, w, t = U.to_device(inp)
    h3 = h.view(2, 150, 96).clone().requires_grad_(True)
    w1 = w.clone().requires_grad_(True)
    per = linear_cross_entropy(h3, w1, t.view(2, 150), reduction="none")
    assert per.shape == (2, 150)
    g = torch.linspace(-1, 1, 300, device=h.device).view(2, 150)
    (per * g).sum().backward()
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets, reduction="none",
                grad=g.view(-1).cpu().numpy().astype(np.float64))
    assert np.max(np.abs(per.detach().view(-1).cpu().numpy() - ref["loss"])) <= U.LSE_ABS_TOL
    assert U.rel_fro(h3.grad.view(300, 96).float().cpu().numpy(), ref["dH"]) <= U.GRAD_REL_TOL
    assert U.rel_fro(w1.grad.float().cpu().numpy(), ref["dW"]) <= U.GRAD_REL_TOL


@pytest.mark.parametrize("case", range(12))
def test_random_shapes_sweep(case):
    """Seeded random shapes across tile, slab and partition boundaries (D multiple of 8)."""
    rng = np.random.default_rng(1000 + case)
    n = int(rng.integers(1, 900))
    d = int(rng.integers(1, 80)) * 8
    v = int(rng.choice([int(rng.integers(1, 600)), int(rng.integers(8000, 34000))]))
    reduction = ["mean", "sum", "none"][case % 3]
    grad = (rng.standard_normal(n).astype(np.float32) if reduction == "none" else float(rng.uniform(0.2, 2.0)))
    inp = WL.custom(n, d, v, seed=case, mask_frac=float(rng.uniform(0, 0.5)), sigma_w=0.3)
    print(f"sweep case {case}: n={n} d={d} v={v} {reduction}", flush=True)
    _case(inp, reduction=reduction, grad=grad)
