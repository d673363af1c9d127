"""Pins of the AdamW oracle (in-backward optimizer fusion, paper Sec. 4.1) -- no GPU needed.

Each pin checks the oracle against something other than itself: torch's own
AdamW (an independent library routine), the closed form of the first step, and
properties of the update; a dropped bias correction, a coupled weight decay or
a swapped beta fails at least one of them.
"""
import numpy as np
import pytest
import torch

from oracle import adamw_oracle as A
from oracle import lce_oracle as O
from paper_2605_21442_amd import workloads as WL

HP = dict(lr=3e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


@pytest.mark.parametrize("hp", [HP, dict(lr=1e-2, beta1=0.8, beta2=0.999, eps=1e-6, weight_decay=0.0)])
def test_matches_torch_adamw_over_steps(hp):
    rng = np.random.default_rng(5)
    theta0 = rng.standard_normal((7, 12))
    grads = [rng.standard_normal((7, 12)) * s for s in (1.0, 0.3, 2.0, 1e-3)]
    p = torch.nn.Parameter(torch.tensor(theta0))
    opt = torch.optim.AdamW([p], lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]), eps=hp["eps"],
                            weight_decay=hp["weight_decay"], foreach=False)
    theta, m, v = theta0, np.zeros_like(theta0), np.zeros_like(theta0)
    for t, g in enumerate(grads, start=1):
        p.grad = torch.tensor(g)
        opt.step()
        theta, m, v = A.adamw_step(theta, g, m, v, step=t, **hp)
        st = opt.state[p]
        np.testing.assert_allclose(theta, p.detach().numpy(), rtol=1e-13, atol=1e-15)
        np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-13, atol=1e-16)
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-13, atol=1e-18)


def test_first_step_closed_form():
    rng = np.random.default_rng(1)
    theta0, g = rng.standard_normal(50), rng.standard_normal(50)
    theta, m, v = A.adamw_step(theta0, g, 0 * g, 0 * g, step=1, **HP)
    # bias correction turns the first moments into g and g^2 exactly
    expect = theta0 * (1 - HP["lr"] * HP["weight_decay"]) - HP["lr"] * g / (np.abs(g) + HP["eps"])
    np.testing.assert_allclose(theta, expect, rtol=1e-14)
    np.testing.assert_allclose(m, (1 - HP["beta1"]) * g, rtol=1e-15)
    np.testing.assert_allclose(v, (1 - HP["beta2"]) * g * g, rtol=1e-15)


def test_zero_gradient_only_decays():
    theta0 = np.linspace(-1, 1, 9)
    m0 = np.linspace(0.1, 0.5, 9)
    v0 = np.linspace(0.2, 0.9, 9)
    theta, m, v = A.adamw_step(theta0, np.zeros(9), m0, v0, step=3, **HP)
    np.testing.assert_allclose(m, HP["beta1"] * m0, rtol=1e-15)
    np.testing.assert_allclose(v, HP["beta2"] * v0, rtol=1e-15)
    mh = m / (1 - HP["beta1"] ** 3)
    vh = v / (1 - HP["beta2"] ** 3)
    np.testing.assert_allclose(theta, theta0 * (1 - HP["lr"] * HP["weight_decay"])
                               - HP["lr"] * mh / (np.sqrt(vh) + HP["eps"]), rtol=1e-14)


def test_memoryless_betas_forget_history():
    rng = np.random.default_rng(2)
    hp = dict(HP, beta1=0.0, beta2=0.0, weight_decay=0.0)
    g = rng.standard_normal(20)
    a, _, _ = A.adamw_step(np.zeros(20), g, rng.standard_normal(20), rng.random(20), step=7, **hp)
    np.testing.assert_allclose(a, -hp["lr"] * g / (np.abs(g) + hp["eps"]), rtol=1e-14)


def test_update_is_scale_invariant_without_eps():
    rng = np.random.default_rng(3)
    hp = dict(HP, eps=0.0, weight_decay=0.0)
    g1, g2 = rng.standard_normal(30), rng.standard_normal(30)

    def two_steps(scale):
        z = np.zeros(30)
        t, m, v = A.adamw_step(z, scale * g1, z, z, step=1, **hp)
        return A.adamw_step(t, scale * g2, m, v, step=2, **hp)[0]

    # scaling the whole gradient history leaves the parameters where they were
    np.testing.assert_allclose(two_steps(1e3), two_steps(1.0), rtol=1e-12)
    assert not np.allclose(two_steps(1.0), 0.0)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(4)
    x32 = (rng.standard_normal(4000) * np.exp(rng.uniform(-30, 30, 4000))).astype(np.float32)
    # exact ties: a bf16 value plus half its spacing
    base = rng.standard_normal(200).astype(np.float32)
    bits = base.view(np.uint32) & np.uint32(0xFFFF0000)
    ties = (bits | np.uint32(0x8000)).view(np.float32)
    x = np.concatenate([x32, ties, np.float32([0.0, -0.0, 1e-40, -3e-39])])
    ours = A.f64_to_bf16_bits(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


def test_fused_objective_is_backward_then_step():
    inp = WL.custom(40, 16, 70, seed=9, mask_frac=0.2, sigma_w=0.5)
    rng = np.random.default_rng(0)
    m0 = 1e-3 * rng.standard_normal((70, 16))
    v0 = 1e-6 * rng.random((70, 16))
    out = A.lce_adamw(inp.h_bits, inp.w_bits, inp.targets, m0, v0, step=4, **HP)
    h, w = O.bf16_to_f64(inp.h_bits), O.bf16_to_f64(inp.w_bits)
    H = torch.tensor(h, requires_grad=True)
    W = torch.nn.Parameter(torch.tensor(w))
    opt = torch.optim.AdamW([W], lr=HP["lr"], betas=(HP["beta1"], HP["beta2"]), eps=HP["eps"],
                            weight_decay=HP["weight_decay"], foreach=False)
    torch.nn.functional.cross_entropy(H @ W.T, torch.tensor(inp.targets.astype(np.int64)),
                                      ignore_index=-100).backward()
    opt.state[W] = {"step": torch.tensor(3.0, dtype=torch.float64), "exp_avg": torch.tensor(m0),
                    "exp_avg_sq": torch.tensor(v0)}
    opt.step()
    np.testing.assert_allclose(out["theta"], W.detach().numpy(), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(out["dH"], H.grad.numpy(), rtol=1e-10, atol=1e-14)
