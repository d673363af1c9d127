"""HIP path vs the CPU oracle at the full workload sizes, in the launch configuration the
benchmark times (same library calls, same shapes: the forward keeps its workspace and the backward
reuses what the forward left in it).

The oracle's forward (loss and every row's lse) for seed 0 is stored under tests/golden/ by
``tests/golden/make_golden.py`` (oracle only). Every head is checked on every row's lse and on
every element of dH and dW: the oracle's backward runs by vocabulary chunks from the stored lse
(``backward_by_vocab_chunks``), each chunk of dW compared with the same rows of the GPU's dW as it
is finished, so that neither a float64 dW nor a float64 copy of the GPU's is held whole. The
case with spread logits (the 8B head with sigma_w = 0.125) makes the softmax part of G carry more
than half of both gradients in the 8B launch plan. Whole-output properties (ignored dH rows are
exactly zero, dW columns sum to ~0, everything finite) are checked on the GPU outputs.
"""
import os

import numpy as np
import pytest

from oracle import lce_oracle as O
from paper_2605_21442_amd import workloads as WL
from tests import lce_testutil as U
from tests.golden import make_golden as MG

pytestmark = pytest.mark.gpu

NAMES = ["llama1b", "llama8b", "qwen7b", "llama70b", "llama8b_spread"]


_CAPSYS = []


def _say(msg):
    # progress of the long oracle passes and the measured errors: past pytest's output capture
    # where the test has the capsys fixture, else captured like any print
    if _CAPSYS:
        with _CAPSYS[0].disabled():
            print(msg, flush=True)
    else:
        print(msg, flush=True)


@pytest.mark.parametrize("name", NAMES)
def test_full_size_against_oracle(name, capsys):
    import torch
    from paper_2605_21442_amd import autograd as A
    _CAPSYS[:] = [capsys]
    path = MG.path_for(name, 0)
    if not os.path.exists(path):
        pytest.skip(f"{path} missing: run tests/golden/make_golden.py")
    gold = np.load(path, allow_pickle=False)
    wl = WL.WORKLOADS[name]
    _say(f"[{name}] drawing inputs")
    inp = WL.generate(wl, 0)
    assert str(gold["fingerprint"]) == MG.fingerprint(inp), "golden file is stale"
    h, w, t = U.to_device(inp)
    _say(f"[{name}] lce_forward + lce_backward (reusing the forward's workspace)")
    loss, lse, nv, status, ws = A.forward(h, w, t, keep_workspace=True)
    g = torch.ones(1, dtype=torch.float32, device=h.device)
    dh_t, dw_t = A.backward(h, w, t, lse, nv, g, workspace=ws)
    del ws, w
    torch.cuda.synchronize()

    # forward: exact count, loss, every lse
    assert int(nv.item()) == int(gold["n_valid"]) == wl.n_valid()
    assert int(status.item()) == 0
    assert abs(float(loss.item()) - float(gold["loss"])) <= U.LOSS_ABS_TOL, (float(loss.item()), float(gold["loss"]))
    valid = inp.targets != inp.ignore_index
    lse_np = lse.cpu().numpy().astype(np.float64)
    lse_err = np.max(np.abs(lse_np[valid] - gold["lse"][valid]))
    assert lse_err <= U.LSE_ABS_TOL, lse_err
    assert np.all(lse_np[~valid] == 0.0)

    # whole-output properties on the GPU
    ign = torch.from_numpy(~valid).to(h.device)
    assert torch.count_nonzero(dh_t[ign]).item() == 0
    assert torch.isfinite(dh_t.float()).all().item() and torch.isfinite(dw_t.float()).all().item()
    col = dw_t.float().sum(0)
    budget = 4 * 2.0 ** -8 * dw_t.float().abs().sum(0)
    assert bool((col.abs() <= budget).all().item())

    # every element of dW (chunk by chunk) and of dH against the oracle's float64 backward
    nvalid = int(gold["n_valid"])
    c = 1.0 / nvalid
    t64 = inp.targets.astype(np.int64)
    vrows = np.nonzero(valid)[0]
    acc = dict(dw_err=0.0, dw_ref=0.0, dw_soft=0.0)

    def on_chunk(v0, ref):
        got = dw_t[v0:v0 + ref.shape[0]].double().cpu().numpy()
        acc["dw_err"] += float(np.sum((got - ref) ** 2))
        acc["dw_ref"] += float(np.sum(ref ** 2))
        # softmax part of the chunk: the reference plus the one-hot part c * (rows whose target is here)
        onehot = np.zeros_like(ref)
        sel = vrows[(t64[vrows] >= v0) & (t64[vrows] < v0 + ref.shape[0])]
        np.add.at(onehot, t64[sel] - v0, O.bf16_to_f64(inp.h_bits[sel]))
        acc["dw_soft"] += float(np.sum((ref + c * onehot) ** 2))

    def progress(done, total):
        _say(f"[{name}]   oracle vocabulary ids {done}/{total}")

    _say(f"[{name}] oracle backward over {nvalid} valid rows by vocabulary chunks")
    rows, ref_dh = O.backward_by_vocab_chunks(inp.h_bits, inp.w_bits, inp.targets, gold["lse"], on_chunk,
                                              progress=progress)
    got_dh = dh_t[torch.from_numpy(rows).to(h.device)].double().cpu().numpy()
    e_dh = U.rel_fro(got_dh, ref_dh)
    e_dw = np.sqrt(acc["dw_err"] / acc["dw_ref"])
    share_dw = np.sqrt(acc["dw_soft"] / acc["dw_ref"])
    # softmax part of dH: the reference plus the one-hot part c * W[t_n]
    share_dh = np.linalg.norm(ref_dh + c * O.bf16_to_f64(inp.w_bits[t64[rows]])) / np.linalg.norm(ref_dh)
    _say(f"[{name}] every element: dH rel Frobenius {e_dh:.2e}, dW rel Frobenius {e_dw:.2e}; "
         f"softmax share of dH {share_dh:.3f}, of dW {share_dw:.3f}; loss {float(loss.item()):.6f} "
         f"(oracle {float(gold['loss']):.6f}), lse err {lse_err:.2e}")
    assert e_dh <= U.GRAD_REL_TOL and e_dw <= U.GRAD_REL_TOL, (e_dh, e_dw)
    if name == "llama8b_spread":
        assert share_dh >= 0.5 and share_dw >= 0.5, (share_dh, share_dw)


def test_full_size_fused_adamw_llama8b():
    """lce_backward_adamw at the 8B head size, in the launch configuration the benchmark's
    fused variant times: bit for bit the two-phase path (lce_backward, then lce_adamw_step), and
    sampled rows of the updated parameter and moments against the oracle."""
    import torch
    from oracle import adamw_oracle as A
    from paper_2605_21442_amd import autograd as AG
    name = "llama8b"
    path = MG.path_for(name, 0)
    if not os.path.exists(path):
        pytest.skip(f"{path} missing: run tests/golden/make_golden.py")
    gold = np.load(path, allow_pickle=False)
    wl = WL.WORKLOADS[name]
    inp = WL.generate(wl, 0)
    h, _, t = U.to_device(inp)
    hp = dict(lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
    g_scale = 2e-5                                   # typical |dW| of this head
    results = []
    for fused in (False, True):
        _say(f"[{name}] {'fused' if fused else 'two-phase'} backward + AdamW")
        w = torch.from_numpy(inp.w_bits.view(np.int16)).view(torch.bfloat16).to(h.device)
        st = AG.AdamWState(w, lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]), eps=hp["eps"],
                           weight_decay=hp["weight_decay"], master_weights=True)
        st.exp_avg_sq.fill_(g_scale * g_scale)       # a warm, uniform second moment
        st.step = 9
        loss, lse, nv, _ = AG.forward(h, w, t)
        g = torch.ones(1, dtype=torch.float32, device=h.device)
        if fused:
            AG.backward_adamw(h, t, lse, nv, g, st)
        else:
            _, dw = AG.backward(h, w, t, lse, nv, g)
            st.step_with(dw)
            del dw
        torch.cuda.synchronize()
        results.append((w, st))
    (wa, sa), (wb, sb) = results
    assert torch.equal(wa.view(torch.int16), wb.view(torch.int16))
    for x, y in ((sa.exp_avg, sb.exp_avg), (sa.exp_avg_sq, sb.exp_avg_sq), (sa.master, sb.master)):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))

    rng = np.random.default_rng(3)
    v = wl.v
    ids = np.array(sorted(set([0, 1, 255, 256, 16383, 16384, v - 1] + rng.integers(2, v, 3).tolist())))
    _say(f"[{name}] oracle AdamW rows {ids.tolist()}")
    ref_dw = O.dw_of_rows(inp.h_bits, inp.w_bits, inp.targets, ids, gold["lse"])
    w0 = O.bf16_to_f64(inp.w_bits[ids])
    theta, m1, v1 = A.adamw_step(w0, ref_dw, np.zeros_like(w0), np.full(w0.shape, np.float32(g_scale * g_scale)),
                                 step=10, **hp)
    sel = torch.from_numpy(ids).to(h.device)
    got_theta = sb.master[sel].cpu().numpy().astype(np.float64)
    got_m = sb.exp_avg[sel].cpu().numpy().astype(np.float64)
    got_v = sb.exp_avg_sq[sel].cpu().numpy().astype(np.float64)
    assert U.rel_fro(got_theta - w0, theta - w0) <= U.GRAD_REL_TOL
    assert U.rel_fro(got_m, m1) <= U.GRAD_REL_TOL
    assert U.rel_fro(got_v, v1) <= U.GRAD_REL_TOL
    _say(f"[{name}] fused AdamW ok")


def test_full_size_vocabulary_shards_llama8b():
    """The 8B head split into 8 vocabulary shards (each the per-device shape of 8-way loss
    parallelism, N tokens x V/8 ids), combined on the one GPU: loss and every lse against the
    stored oracle forward, sampled dH rows (sum of the shards' fp32 terms) and dW rows against
    the oracle."""
    import torch
    from paper_2605_21442_amd import autograd as AG
    name = "llama8b"
    path = MG.path_for(name, 0)
    if not os.path.exists(path):
        pytest.skip(f"{path} missing: run tests/golden/make_golden.py")
    gold = np.load(path, allow_pickle=False)
    wl = WL.WORKLOADS[name]
    inp = WL.generate(wl, 0)
    h, w, t = U.to_device(inp)
    v, g_count = wl.v, 8
    cuts = [round(i * v / g_count) for i in range(g_count + 1)]
    _say(f"[{name}] {g_count} vocabulary shards, cuts {cuts}")
    parts = [AG.forward_shard(h, w[a:b], t, a, v) for a, b in zip(cuts[:-1], cuts[1:])]
    lse_parts = torch.stack([q[0] for q in parts]).contiguous()
    tgt_parts = torch.stack([q[1] for q in parts]).contiguous()
    del parts
    loss, lse, nv, status = AG.combine_shards(lse_parts, tgt_parts, t, v, wl.d)
    assert int(nv.item()) == int(gold["n_valid"]) and int(status.item()) == 0
    assert abs(float(loss.item()) - float(gold["loss"])) <= U.LOSS_ABS_TOL
    valid = inp.targets != inp.ignore_index
    lse_err = np.max(np.abs(lse.cpu().numpy()[valid] - gold["lse"][valid]))
    assert lse_err <= U.LSE_ABS_TOL, lse_err

    g = torch.ones(1, dtype=torch.float32, device=h.device)
    dh = torch.zeros((wl.n, wl.d), dtype=torch.float32, device=h.device)
    dws = []
    for a, b in zip(cuts[:-1], cuts[1:]):
        term, dw = AG.backward_shard(h, w[a:b], t, lse, nv, g, a, v)
        dh += term
        dws.append(dw)
        del term
    dw = torch.cat(dws)
    rng = np.random.default_rng(11)
    vrows = np.nonzero(valid)[0]
    rows = np.concatenate([rng.choice(vrows, 5, replace=False), np.nonzero(~valid)[0][:1]])
    ref_dh = O.dh_of_rows(inp.h_bits, inp.w_bits, inp.targets, rows, int(gold["n_valid"]))
    got_dh = dh[torch.from_numpy(rows).to(h.device)].cpu().numpy().astype(np.float64)
    assert U.rel_fro(got_dh, ref_dh) <= U.GRAD_REL_TOL
    assert np.all(got_dh[-1] == 0.0)
    ids = np.array(sorted(set([0, 1, cuts[1] - 1, cuts[1], cuts[4], v - 1] + rng.integers(2, v, 3).tolist())))
    ref_dw = O.dw_of_rows(inp.h_bits, inp.w_bits, inp.targets, ids, gold["lse"])
    got_dw = dw[torch.from_numpy(ids).to(h.device)].float().cpu().numpy().astype(np.float64)
    assert U.rel_fro(got_dw, ref_dw) <= U.GRAD_REL_TOL
    _say(f"[{name}] shards ok: loss {float(loss.item()):.6f} (oracle {float(gold['loss']):.6f})")


def test_full_size_kd_8b_to_1b():
    """Distilling the 8B head into the 1B head (N = 16384, Ds = 2048, Dt = 4096, V = 128256, T = 2)
    in the launch configuration the benchmark's KD variant times: loss and every row's lse of both
    heads against the stored oracle forward, sampled dHs / dWs rows against the oracle."""
    import torch
    from oracle import kd_oracle as K
    from paper_2605_21442_amd import autograd as AG
    name = "kd_8b_to_1b"
    path = MG.path_for(name, 0)
    if not os.path.exists(path):
        pytest.skip(f"{path} missing: run tests/golden/make_golden.py")
    gold = np.load(path, allow_pickle=False)
    inp = WL.kd_generate(name, 0)
    assert str(gold["fingerprint"]) == MG.kd_fingerprint(inp), "golden file is stale"
    T = float(gold["temperature"])
    dev = "cuda:0"
    to = lambda b: torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).to(dev)
    hs, ws, ht, wt = to(inp.hs_bits), to(inp.ws_bits), to(inp.ht_bits), to(inp.wt_bits)
    t = torch.from_numpy(inp.targets).to(dev)
    _say(f"[{name}] kd forward + backward")
    loss, lse_s, lse_t, nv, status = AG.kd_forward(hs, ws, ht, wt, t, T)
    g = torch.ones(1, dtype=torch.float32, device=dev)
    dh, dw = AG.kd_backward(hs, ws, ht, wt, t, lse_s, lse_t, nv, g, T)
    torch.cuda.synchronize()
    assert int(nv.item()) == int(gold["n_valid"]) and int(status.item()) == 0
    assert abs(float(loss.item()) - float(gold["loss"])) <= U.LOSS_ABS_TOL, (float(loss.item()), float(gold["loss"]))
    valid = inp.targets != inp.ignore_index
    for k, got in (("lse_s", lse_s), ("lse_t", lse_t)):
        err = np.max(np.abs(got.cpu().numpy()[valid] - gold[k][valid]))
        assert err <= U.LSE_ABS_TOL, (k, err)
    rng = np.random.default_rng(5)
    vrows = np.nonzero(valid)[0]
    rows = np.concatenate([rng.choice(vrows, 4, replace=False), np.nonzero(~valid)[0][:1]])
    _say(f"[{name}] oracle dHs rows {rows.tolist()}")
    ref = K.kd_dh_rows(inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits, inp.targets, rows,
                       int(gold["n_valid"]), temperature=T)
    got = dh[torch.from_numpy(rows).to(dev)].float().cpu().numpy().astype(np.float64)
    assert U.rel_fro(got, ref) <= U.GRAD_REL_TOL
    assert np.all(got[-1] == 0.0)
    v = inp.ws_bits.shape[0]
    ids = np.array(sorted(set([0, 1, 8191, 8192, v - 1] + rng.integers(2, v, 3).tolist())))
    _say(f"[{name}] oracle dWs rows {ids.tolist()}")
    ref = K.kd_dw_rows(inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits, inp.targets, ids, gold["lse_s"],
                       gold["lse_t"], temperature=T)
    got = dw[torch.from_numpy(ids).to(dev)].float().cpu().numpy().astype(np.float64)
    assert U.rel_fro(got, ref) <= U.GRAD_REL_TOL
    _say(f"[{name}] ok: loss {float(loss.item()):.6f} (oracle {float(gold['loss']):.6f})")


def test_full_size_allocates_nothing_beyond_the_workspace():
    """8B head: the library makes no allocation of its own (the driver's free memory is unchanged
    across the calls), the caller-sized workspace stays below half a bf16 copy of the logits, and
    no buffer of the path comes near the [N, V] size the method avoids."""
    import torch
    from paper_2605_21442_amd import binding as B
    wl = WL.WORKLOADS["llama8b"]
    inp = WL.generate(wl, 0)
    h, w, t = U.to_device(inp)
    dev = h.device
    n, d, v = wl.n, wl.d, wl.v
    p = B.problem(n, d, v, ignore_index=inp.ignore_index, reduction="mean", target_bytes=4)
    fwd_bytes, bwd_bytes = B.lce_workspace_size(p)
    ws = torch.empty(max(fwd_bytes, bwd_bytes), dtype=torch.uint8, device=dev)
    loss = torch.empty((), dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    grad = torch.ones(1, dtype=torch.float32, device=dev)
    dh = torch.empty((n, d), dtype=torch.bfloat16, device=dev)
    dw = torch.empty((v, d), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream

    def step():
        B.lce_forward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), loss.data_ptr(), lse.data_ptr(),
                      nv.data_ptr(), status.data_ptr(), ws.data_ptr(), fwd_bytes, stream)
        B.lce_backward(p, h.data_ptr(), w.data_ptr(), t.data_ptr(), lse.data_ptr(), nv.data_ptr(),
                       grad.data_ptr(), dh.data_ptr(), dw.data_ptr(), ws.data_ptr(), bwd_bytes, stream)

    step()                                   # first call loads the code objects
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info(dev)[0]
    alloc0 = torch.cuda.memory_allocated(dev)
    torch.cuda.reset_peak_memory_stats(dev)
    _say("[llama8b] second forward + backward, watching device memory")
    step()
    torch.cuda.synchronize()
    free1 = torch.cuda.mem_get_info(dev)[0]
    assert torch.cuda.max_memory_allocated(dev) == alloc0       # nothing through torch's allocator
    assert abs(free1 - free0) <= (2 << 20), (free0, free1)      # nothing through the driver either
    logits_bf16 = n * v * 2
    assert max(fwd_bytes, bwd_bytes) < logits_bf16 // 2
    for x in (h, w, dh, dw, ws):
        assert x.numel() * x.element_size() < logits_bf16 // 2
    assert int(nv.item()) == wl.n_valid() and int(status.item()) == 0
