"""AdamW inside the LCE backward (paper Sec. 4.1 on the Sec. 4.2 weight) and gradient accumulation.

* the standalone step (lce_adamw_step) against the float64 AdamW oracle;
* the fused backward (lce_backward_adamw) against the two-phase path (lce_backward, then
  lce_adamw_step): the paper states that with one update per backward pass the trajectory
  is bitwise that of the standard optimizer, so the comparison is bit for bit;
* the fused backward against the oracle of "LCE backward, then AdamW" end to end;
* the accumulate-into-dW flag against oracle dW0 + dW.
"""
import numpy as np
import pytest

from oracle import adamw_oracle as A
from oracle import lce_oracle as O
from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U

pytestmark = pytest.mark.gpu

HP = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


def _t(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")


def _bf16(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda:0")


def _bits(t):
    import torch
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _state(w_bits, master, cold=False, seed=0):
    """Device copies of a drawn optimizer state: (m, v, master or None)."""
    s = WL.opt_state(w_bits, seed=seed, cold=cold)
    return _t(s.m), _t(s.v), (_t(s.master) if master else None), s


def _step(W, dW, m, v, mst, step, hp=HP):
    import torch
    from paper_2605_21442_amd import binding as B
    B.lce_adamw_step(W.shape[0], W.shape[1], W.stride(0), W.data_ptr(), dW.data_ptr() if dW is not None else 0,
                     m.data_ptr(), v.data_ptr(), mst.data_ptr() if mst is not None else 0,
                     B.adamw(step=step, **hp), torch.cuda.current_stream().cuda_stream)


def _ulp_close(gpu_bits, ref_theta, atol=0.0, min_exact=0.99):
    """bf16 results vs the float64 parameter: the nearest bf16 of it or a neighbour of that (or,
    for values so small that fp32 rounding of the update matters more, within ``atol``), and
    nearly all exactly the nearest bf16."""
    ref_bits = A.f64_to_bf16_bits(ref_theta)
    a = gpu_bits.astype(np.int32)
    b = ref_bits.astype(np.int32)
    same_sign = (a >> 15) == (b >> 15)
    diff = np.abs(a - b)
    near = np.abs(O.bf16_to_f64(gpu_bits) - ref_theta) <= atol
    ok = (same_sign & (diff <= 1)) | near | ((a & 0x7FFF) == 0) & ((b & 0x7FFF) <= 1)
    assert ok.all(), (np.argwhere(~ok)[:5], a[~ok][:5], b[~ok][:5])
    assert (diff == 0).mean() >= min_exact, (diff == 0).mean()


# ---- standalone step vs the oracle -----------------------------------------------------------

@pytest.mark.parametrize("v,d", [(300, 264), (1, 8), (1000, 72)])
def test_standalone_step_with_master_matches_oracle_over_steps(v, d):
    import torch
    w_bits = WL.custom(1, d, v, seed=v).w_bits
    m, vv, mst, s = _state(w_bits, master=True)
    W = _bf16(w_bits)
    theta, mo, vo = s.master.astype(np.float64), s.m.astype(np.float64), s.v.astype(np.float64)
    print(f"adamw standalone master v={v} d={d}", flush=True)
    for t in (1, 2, 3):
        g_bits = WL.gradient_bits(v, d, seed=t)
        _step(W, _bf16(g_bits), m, vv, mst, t)
        torch.cuda.synchronize()
        theta, mo, vo = A.adamw_step(theta, O.bf16_to_f64(g_bits), mo, vo, step=t, **HP)
        np.testing.assert_allclose(m.cpu().numpy(), mo, rtol=1e-6, atol=1e-9)
        np.testing.assert_allclose(vv.cpu().numpy(), vo, rtol=1e-6, atol=1e-15)
        np.testing.assert_allclose(mst.cpu().numpy(), theta, rtol=1e-6, atol=1e-5 * HP["lr"])
        _ulp_close(_bits(W), mst.cpu().numpy().astype(np.float64), min_exact=1.0)
        _ulp_close(_bits(W), theta, atol=1e-5 * HP["lr"])


@pytest.mark.parametrize("cold", [True, False])
def test_standalone_step_on_bf16_weight_matches_oracle(cold):
    import torch
    v, d = 513, 136
    w_bits = WL.custom(1, d, v, seed=3, sigma_w=0.02).w_bits
    m, vv, _, s = _state(w_bits, master=False, cold=cold)
    W = _bf16(w_bits)
    g_bits = WL.gradient_bits(v, d, seed=11)
    # a large rate so that the step moves bf16 weights by several units in the last place
    hp = dict(HP, lr=2e-2)
    _step(W, _bf16(g_bits), m, vv, None, 1 if cold else 5, hp)
    torch.cuda.synchronize()
    theta, mo, vo = A.adamw_step(O.bf16_to_f64(w_bits), O.bf16_to_f64(g_bits), s.m, s.v,
                                 step=1 if cold else 5, **hp)
    np.testing.assert_allclose(m.cpu().numpy(), mo, rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(vv.cpu().numpy(), vo, rtol=1e-6, atol=1e-15)
    _ulp_close(_bits(W), theta, atol=1e-5 * hp["lr"])
    assert (_bits(W) != w_bits).mean() > 0.5            # the step did move the weights


def test_zero_gradient_step_matches_oracle():
    import torch
    v, d = 70, 64
    w_bits = WL.custom(1, d, v, seed=4).w_bits
    m, vv, mst, s = _state(w_bits, master=True)
    W = _bf16(w_bits)
    _step(W, None, m, vv, mst, 4)
    torch.cuda.synchronize()
    theta, mo, vo = A.adamw_step(s.master, np.zeros((v, d)), s.m, s.v, step=4, **HP)
    np.testing.assert_allclose(m.cpu().numpy(), mo, rtol=1e-6, atol=1e-12)
    np.testing.assert_allclose(mst.cpu().numpy(), theta, rtol=1e-6, atol=1e-5 * HP["lr"])


# ---- fused backward vs the two-phase path (bit for bit) --------------------------------------

def _two_paths(inp, master, reduction="mean", cold=False, ld_pad=0, grad=None):
    """Run (a) forward, lce_backward, lce_adamw_step and (b) forward, lce_backward_adamw from the
    same drawn inputs and state; returns both results as host arrays."""
    import torch
    from paper_2605_21442_amd import autograd as AG
    n, d = inp.h_bits.shape
    v = inp.w_bits.shape[0]
    h, _, t = U.to_device(inp)
    if grad is None:
        grad = np.ones(n if reduction == "none" else 1, np.float32)
    g = _t(np.asarray(grad, np.float32).reshape(-1))
    out = []
    for fused in (False, True):
        wfull = torch.zeros((v, d + ld_pad), dtype=torch.bfloat16, device="cuda:0")
        wfull[:, :d] = _bf16(inp.w_bits)
        if ld_pad:
            wfull[:, d:] = -1.5                            # untouched padding columns
        W = wfull[:, :d]
        m, vv, mst, _ = _state(inp.w_bits, master, cold=cold)
        loss, lse, nv, _ = AG.forward(h, W, t, inp.ignore_index, reduction)
        st = AG.AdamWState(W, lr=HP["lr"], betas=(HP["beta1"], HP["beta2"]), eps=HP["eps"],
                           weight_decay=HP["weight_decay"], master_weights=master)
        st.load_state_dict({"exp_avg": m, "exp_avg_sq": vv, "master": mst, "step": 0 if cold else 6})
        m, vv, mst = st.exp_avg, st.exp_avg_sq, st.master
        if fused:
            dh = AG.backward_adamw(h, t, lse, nv, g, st, inp.ignore_index, reduction)
        else:
            dh, dw = AG.backward(h, W, t, lse, nv, g, inp.ignore_index, reduction)
            st.step_with(dw)
        torch.cuda.synchronize()
        out.append(dict(W=_bits(wfull), m=m.cpu().numpy().view(np.uint32), v=vv.cpu().numpy().view(np.uint32),
                        master=(mst.cpu().numpy().view(np.uint32) if mst is not None else None),
                        dH=_bits(dh), step=st.step, wfull=wfull))
    return out


@pytest.mark.parametrize("n,d,v", [(600, 128, 9000), (300, 264, 1000), (257, 64, 9000), (1, 8, 5),
                                   (40, 16, 2), (513, 520, 300)])
@pytest.mark.parametrize("master", [False, True])
def test_fused_backward_is_bitwise_the_two_phase_path(n, d, v, master):
    print(f"fused vs two-phase n={n} d={d} v={v} master={master}", flush=True)
    inp = WL.custom(n, d, v, seed=n + d, mask_frac=0.2, sigma_w=0.3)
    a, b = _two_paths(inp, master)
    for k in ("W", "m", "v", "master", "dH"):
        if a[k] is not None:
            np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    assert a["step"] == b["step"] == 7


def test_fused_backward_bitwise_cold_start_none_reduction_and_strided_weight():
    inp = WL.custom(700, 136, 9100, seed=8, mask_frac=0.25, sigma_w=0.3)
    g = np.random.default_rng(1).standard_normal(700).astype(np.float32)
    a, b = _two_paths(inp, master=True, reduction="none", cold=True, ld_pad=8, grad=g)
    for k in ("W", "m", "v", "master", "dH"):
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    pad = a["W"][:, 136:]
    assert np.all(pad == np.float32(-1.5).view(np.uint32) >> 16)


@pytest.mark.parametrize("case", ["all_masked", "no_tokens"])
def test_fused_backward_without_valid_tokens_is_a_zero_gradient_step(case):
    import torch
    from paper_2605_21442_amd import autograd as AG
    n = 0 if case == "no_tokens" else 50
    inp = WL.custom(n, 64, 700, seed=2, mask_frac=0.0,
                    target_override=np.full(n, -100, np.int32))
    a, b = _two_paths(inp, master=True)
    for k in ("W", "m", "v", "master"):
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    s = WL.opt_state(inp.w_bits)
    theta, mo, _ = A.adamw_step(s.master, np.zeros(s.m.shape), s.m, s.v, step=7, **HP)
    np.testing.assert_allclose(b["master"].view(np.float32), theta, rtol=1e-6, atol=1e-5 * HP["lr"])


# ---- fused backward vs the oracle, end to end ------------------------------------------------

@pytest.mark.parametrize("n,d,v", [(300, 264, 1000), (600, 128, 9000)])
def test_fused_backward_matches_oracle(n, d, v):
    print(f"fused vs oracle n={n} d={d} v={v}", flush=True)
    inp = WL.custom(n, d, v, seed=5, mask_frac=0.2, sigma_w=0.3)
    a, b = _two_paths(inp, master=True)
    s = WL.opt_state(inp.w_bits)
    ref = A.lce_adamw(inp.h_bits, inp.w_bits, inp.targets, s.m, s.v, s.master, step=7, **HP)
    upd_gpu = b["master"].view(np.float32).astype(np.float64) - s.master
    upd_ref = ref["theta"] - s.master
    assert U.rel_fro(upd_gpu, upd_ref) <= U.GRAD_REL_TOL
    assert U.rel_fro(b["m"].view(np.float32).astype(np.float64), ref["m"]) <= U.GRAD_REL_TOL
    assert U.rel_fro(b["v"].view(np.float32).astype(np.float64), ref["v"]) <= U.GRAD_REL_TOL
    assert U.rel_fro(O.bf16_to_f64(b["dH"]), ref["dH"]) <= U.GRAD_REL_TOL


def test_in_backward_optimizer_trajectory_equals_two_phase_training():
    """Two training steps through the autograd front end: optimizer inside the backward vs
    backward producing weight.grad followed by the standalone step."""
    import torch
    from paper_2605_21442_amd import linear_cross_entropy, AdamWState
    n, d, v = 384, 96, 2000
    ws = []
    for fused in (False, True):
        inp0 = WL.custom(n, d, v, seed=0, mask_frac=0.1, sigma_w=0.3)
        W = torch.nn.Parameter(_bf16(inp0.w_bits))
        st = AdamWState(W.data, lr=5e-3, betas=(0.9, 0.99), eps=1e-8, weight_decay=0.05,
                        master_weights=True)
        for it in range(2):
            inp = WL.custom(n, d, v, seed=10 + it, mask_frac=0.1)
            h, _, t = U.to_device(inp)
            h.requires_grad_(True)
            if fused:
                loss = linear_cross_entropy(h, W, t, optimizer=st)
                loss.backward()
                assert W.grad is None
            else:
                loss = linear_cross_entropy(h, W, t)
                loss.backward()
                st.step_with(W.grad)
                W.grad = None
        torch.cuda.synchronize()
        ws.append((_bits(W.data), st.master.cpu().numpy().view(np.uint32), st.step))
    np.testing.assert_array_equal(ws[0][0], ws[1][0])
    np.testing.assert_array_equal(ws[0][1], ws[1][1])
    assert ws[0][2] == ws[1][2] == 2


# ---- gradient accumulation -------------------------------------------------------------------

@pytest.mark.parametrize("n,d,v", [(300, 264, 1000), (257, 64, 9000)])
def test_accumulate_into_dw_matches_oracle(n, d, v):
    import torch
    from paper_2605_21442_amd import autograd as AG
    inp = WL.custom(n, d, v, seed=6, mask_frac=0.2, sigma_w=0.3)
    h, w, t = U.to_device(inp)
    loss, lse, nv, _ = AG.forward(h, w, t)
    g = torch.ones(1, dtype=torch.float32, device="cuda:0")
    _, dw_plain = AG.backward(h, w, t, lse, nv, g)
    # previous micro-batches' gradient, of the same order as this one's
    scale = float(dw_plain.float().abs().mean())
    dw0_bits = WL.gradient_bits(v, d, seed=7, g_scale=scale)
    acc = _bf16(dw0_bits)
    _, out = AG.backward(h, w, t, lse, nv, g, accumulate_into=acc)
    torch.cuda.synchronize()
    assert out.data_ptr() == acc.data_ptr()
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets)
    expect = O.bf16_to_f64(dw0_bits) + ref["dW"]
    assert U.rel_fro(out.float().cpu().numpy().astype(np.float64), expect) <= U.GRAD_REL_TOL
    # accumulating onto zeros gives the plain gradient's values
    z = torch.zeros_like(dw_plain)
    AG.backward(h, w, t, lse, nv, g, accumulate_into=z)
    torch.cuda.synchronize()
    assert torch.equal(z.float(), dw_plain.float())
