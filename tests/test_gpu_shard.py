"""Vocabulary-parallel (loss-parallel) mode on one GPU (paper Sec. 4.2 with the loss-parallel
sharding of Sec. 5): W is split into shards by vocabulary rows, every shard runs
lce_forward_shard, the [N] partials are stacked (standing in for the all-gather between
devices) and combined by lce_combine_shards, every shard runs lce_backward_shard with the
global lse, and the fp32 dH terms are summed (standing in for the all-reduce). The combined
results must reproduce the full-vocabulary oracle; the per-shard partials must match the
oracle's shard partials.
"""
import numpy as np
import pytest

from oracle import lce_oracle as O
from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U

pytestmark = pytest.mark.gpu


def _run_shards(inp, cuts, reduction="mean", grad=None):
    import torch
    from paper_2605_21442_amd import autograd as AG
    n, d = inp.h_bits.shape
    v = inp.w_bits.shape[0]
    h, w, t = U.to_device(inp)
    parts = [AG.forward_shard(h, w[a:b], t, a, v, inp.ignore_index) for a, b in zip(cuts[:-1], cuts[1:])]
    lse_parts = torch.stack([q[0] for q in parts]).contiguous()
    tgt_parts = torch.stack([q[1] for q in parts]).contiguous()
    loss, lse, nv, status = AG.combine_shards(lse_parts, tgt_parts, t, v, d, inp.ignore_index, reduction)
    if grad is None:
        grad = np.ones(n if reduction == "none" else 1, np.float32)
    g = torch.from_numpy(np.asarray(grad, np.float32).reshape(-1)).to(h.device)
    bw = [AG.backward_shard(h, w[a:b], t, lse, nv, g, a, v, inp.ignore_index, reduction)
          for a, b in zip(cuts[:-1], cuts[1:])]
    dh = torch.stack([q[0] for q in bw]).sum(0)
    dw = torch.cat([q[1] for q in bw])
    torch.cuda.synchronize()
    return dict(loss=(loss.cpu().numpy().astype(np.float64) if reduction == "none" else float(loss.item())),
                lse=lse.cpu().numpy().astype(np.float64), n_valid=int(nv.item()), status=int(status.item()),
                dH=dh.cpu().numpy().astype(np.float64), dW=dw.float().cpu().numpy().astype(np.float64),
                parts=[(q[0].cpu().numpy(), q[1].cpu().numpy(), int(q[2].item()), int(q[3].item())) for q in parts],
                dh_terms=[q[0].cpu().numpy() for q in bw])


@pytest.mark.parametrize("n,d,v,cuts", [
    (300, 264, 1000, [0, 500, 1000]),
    (600, 128, 9000, [0, 2048, 2049, 5000, 9000]),           # a one-id shard, uneven shards
    (257, 64, 9000, [0, 9000]),                               # one shard holding everything
    (700, 136, 4097, [0, 1000, 2000, 3000, 4097]),
])
@pytest.mark.parametrize("reduction", ["mean", "sum", "none"])
def test_shards_reproduce_the_full_vocabulary_oracle(n, d, v, cuts, reduction):
    print(f"shards n={n} d={d} v={v} cuts={cuts} red={reduction}", flush=True)
    inp = WL.custom(n, d, v, seed=n + len(cuts), mask_frac=0.2, sigma_w=0.3)
    grad = np.random.default_rng(2).standard_normal(n).astype(np.float32) if reduction == "none" else 0.7
    gpu = _run_shards(inp, cuts, reduction, grad if reduction == "none" else np.float32([grad]))
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets, inp.ignore_index, reduction, grad)
    U.assert_parity(gpu, ref)


def test_shard_partials_match_oracle_partials():
    n, d, v = 400, 96, 3000
    cuts = [0, 700, 2999, 3000]
    inp = WL.custom(n, d, v, seed=4, mask_frac=0.25, sigma_w=0.3)
    t = inp.targets.copy()
    t[5] = v + 10                                             # flagged, ignored on every shard
    inp = WL.custom(n, d, v, seed=4, mask_frac=0.25, sigma_w=0.3, target_override=t)
    gpu = _run_shards(inp, cuts)
    h, w = O.bf16_to_f64(inp.h_bits), O.bf16_to_f64(inp.w_bits)
    full = O.lce(inp.h_bits, inp.w_bits, inp.targets)
    for (a, b), (lp, tp, nv, status), dh_term in zip(zip(cuts[:-1], cuts[1:]), gpu["parts"], gpu["dh_terms"]):
        ref = O.shard_forward(h, w[a:b], inp.targets, a, v)
        assert nv == ref["n_valid"] and status == ref["status"] == 1
        assert np.max(np.abs(lp - ref["lse_part"])) <= U.LSE_ABS_TOL
        assert np.max(np.abs(tp - ref["tgt_part"])) <= 1e-3 * max(1.0, np.abs(ref["tgt_part"]).max())
        rb = O.shard_backward(h, w[a:b], inp.targets, full["lse"], a, v, full["n_valid"])
        assert U.rel_fro(dh_term.astype(np.float64), rb["dH_part"]) <= U.GRAD_REL_TOL
    assert gpu["status"] == 1


def test_single_shard_equals_the_unsharded_path_bitwise_on_the_loss():
    import torch
    from paper_2605_21442_amd import autograd as AG
    inp = WL.custom(513, 520, 300, seed=9, mask_frac=0.1, sigma_w=0.3)
    h, w, t = U.to_device(inp)
    loss_a, lse_a, _, _ = AG.forward(h, w, t)
    lp, tp, _, _ = AG.forward_shard(h, w, t, 0, 300)
    loss_b, lse_b, _, _ = AG.combine_shards(lp.view(1, -1).contiguous(), tp.view(1, -1).contiguous(), t, 300, 520)
    torch.cuda.synchronize()
    assert torch.equal(lse_a, lse_b)
    assert torch.equal(loss_a, loss_b)


def test_shard_holding_no_target_has_no_onehot_term():
    """Every target lies in the first shard: the second shard's G is the plain softmax block, so
    its dW rows are c * softmax^T H and its target logits are all zero."""
    n, d, v = 200, 64, 1000
    t = np.random.default_rng(0).integers(0, 100, n).astype(np.int32)
    inp = WL.custom(n, d, v, seed=3, sigma_w=0.3, target_override=t)
    gpu = _run_shards(inp, [0, 100, 1000])
    assert np.all(gpu["parts"][1][1] == 0.0)
    ref = O.lce(inp.h_bits, inp.w_bits, inp.targets)
    U.assert_parity(gpu, ref)
