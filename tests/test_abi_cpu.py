"""The C ABI without a GPU: the library loads, exports what include/lce.h declares, sizes its
workspace as documented and rejects bad arguments before launching anything."""
import ctypes
import os
import re

import pytest

from paper_2605_21442_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH), reason="liblce.so not built")


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "lce.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lce_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    lib = B.load()
    declared = _declared_functions()
    assert set(declared) == set(B.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings():
    for code in range(8):
        assert B.lce_status_string(code) and B.lce_status_string(code) != "unknown status"
    assert B.lce_status_string(99) == "unknown status"


def test_workspace_is_linear_in_tokens_and_never_tokens_times_vocab():
    f1, b1 = B.lce_workspace_size(B.problem(16384, 4096, 128256))
    f2, b2 = B.lce_workspace_size(B.problem(32768, 4096, 128256))
    assert f2 < 2.1 * f1 and b2 < 2.1 * b1
    n, d, v = 16384, 4096, 128256
    assert b1 < n * v * 2 // 2                              # below half a bf16 copy of the logits
    slab = max(8192, 4 * d)
    bound = 4 * n * 4 + 2 * d * n + 2 * 2 * n * slab + 2 * d * slab + 4 * n * d + 4096
    assert b1 <= bound
    # the backward workspace does not depend on V; the forward's partial rows (8 bytes per token and
    # 384-id tile) are capped at 2 D bytes per token, beyond which it switches to a fixed row count
    fwd = {}
    for vv in (128256, 256512, 393216, 393600, 1 << 20, 1 << 22):
        fv, bv = B.lce_workspace_size(B.problem(n, d, vv))
        assert bv == b1
        fwd[vv] = fv
    assert fwd[393216] - fwd[128256] == 8 * n * (1024 - 334)     # one row per tile up to D / 4 tiles
    assert fwd[393600] < fwd[393216] and fwd[1 << 20] == fwd[1 << 22] == fwd[393600]
    assert max(fwd.values()) <= f1 + 8 * n * (d // 4)


@pytest.mark.parametrize("kw,code", [
    (dict(n=-1, d=64, v=10), B.LCE_ERR_SHAPE),
    (dict(n=4, d=0, v=10), B.LCE_ERR_SHAPE),
    (dict(n=4, d=64, v=0), B.LCE_ERR_SHAPE),
    (dict(n=4, d=60, v=10), B.LCE_ERR_UNSUPPORTED),
    (dict(n=4, d=64, v=10, ld_h=32), B.LCE_ERR_SHAPE),
    (dict(n=4, d=64, v=10, ld_w=68), B.LCE_ERR_ALIGN),
    (dict(n=4, d=64, v=10, reduction=7), B.LCE_ERR_UNSUPPORTED),
    (dict(n=4, d=64, v=10, reduction=3), B.LCE_ERR_UNSUPPORTED),
    (dict(n=4, d=64, v=10, target_bytes=2), B.LCE_ERR_UNSUPPORTED),
    (dict(n=1 << 22, d=1024, v=10), B.LCE_ERR_SHAPE),       # H beyond 32-bit byte offsets
])
def test_bad_problems_are_rejected(kw, code):
    with pytest.raises(B.LceError) as e:
        B.lce_workspace_size(B.problem(**kw))
    assert e.value.code == code


@pytest.mark.parametrize("flags", [4, 8, 1 << 30, -1])
def test_unknown_flag_bits_are_rejected(flags):
    p = B.problem(4, 64, 10, flags=flags)
    with pytest.raises(B.LceError) as e:
        B.lce_workspace_size(p)
    assert e.value.code == B.LCE_ERR_ARG
    B.lce_workspace_size(B.problem(4, 64, 10, flags=B.LCE_FLAG_ACCUMULATE_DW))
    B.lce_workspace_size(B.problem(4, 64, 10, flags=B.LCE_FLAG_REUSE_FORWARD))
    B.lce_workspace_size(B.problem(4, 64, 10, flags=B.LCE_FLAG_REUSE_FORWARD | B.LCE_FLAG_ACCUMULATE_DW))


def test_reuse_flag_is_rejected_by_the_distillation_calls():
    # the KD calls lay out their workspace differently from lce_forward
    with pytest.raises(B.LceError) as e:
        B.lce_kd_workspace_size(B.kd_problem(8, 64, 64, 100, flags=B.LCE_FLAG_REUSE_FORWARD))
    assert e.value.code == B.LCE_ERR_ARG


@pytest.mark.parametrize("n,d,v", [(16384, 4096, 128256), (300, 264, 1000), (1, 8, 5), (8192, 2048, 128256)])
def test_the_forward_and_backward_share_the_prefix_the_reuse_flag_relies_on(n, d, v):
    # idx, pos, Nv and the gathered rows sit at the same offsets in both passes' layouts, and the
    # forward's own regions (partials, terms) start after them, so a backward reusing the
    # forward's workspace finds its list and rows untouched
    info = B.lce_plan_info(B.problem(n, d, v))
    assert info["o_idx"] < info["o_pos"] < info["o_nv"] < info["o_hv"]
    prefix_end = info["o_hv"] + 2 * d * info["npad"]
    assert info["o_pm"] >= prefix_end and info["o_g"] >= prefix_end
    assert info["fwd_gathers"] == (1 if d % 64 == 0 else 0)


def _fake(addr=0x100000):
    return addr


def test_forward_argument_checks_run_before_any_launch():
    p = B.problem(8, 64, 10)
    fwd, _ = B.lce_workspace_size(p)
    ok = dict(H=_fake(), W=_fake(0x200000), targets=_fake(0x300000), loss=_fake(0x400000),
              lse=_fake(0x500000), n_valid=_fake(0x600000), dev_status=0,
              workspace=_fake(0x700000), workspace_bytes=fwd, stream=0)
    cases = [
        (dict(H=0), B.LCE_ERR_NULL), (dict(loss=0), B.LCE_ERR_NULL), (dict(lse=0), B.LCE_ERR_NULL),
        (dict(W=0x200008), B.LCE_ERR_ALIGN), (dict(workspace=0x700010), B.LCE_ERR_ALIGN),
        (dict(workspace_bytes=fwd - 1), B.LCE_ERR_WORKSPACE),
    ]
    for change, code in cases:
        args = dict(ok, **change)
        with pytest.raises(B.LceError) as e:
            B.lce_forward(p, **args)
        assert e.value.code == code, change


def test_backward_argument_checks_run_before_any_launch():
    p = B.problem(8, 64, 10)
    _, bwd = B.lce_workspace_size(p)
    ok = dict(H=_fake(), W=_fake(0x200000), targets=_fake(0x300000), lse=_fake(0x400000),
              n_valid=_fake(0x500000), grad_loss=_fake(0x600000), dH=_fake(0x700000),
              dW=_fake(0x800000), workspace=_fake(0x900000), workspace_bytes=bwd, stream=0)
    cases = [
        (dict(dW=0), B.LCE_ERR_NULL), (dict(grad_loss=0), B.LCE_ERR_NULL),
        (dict(dH=0x700004), B.LCE_ERR_ALIGN), (dict(workspace_bytes=16), B.LCE_ERR_WORKSPACE),
    ]
    for change, code in cases:
        args = dict(ok, **change)
        with pytest.raises(B.LceError) as e:
            B.lce_backward(p, **args)
        assert e.value.code == code, change


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "liblce.so"))
    with pytest.raises(RuntimeError, match="not built"):
        B.load()


HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, step=1)


def test_adamw_step_argument_checks_run_before_any_launch():
    ok = dict(v=10, d=64, ld_w=0, W=_fake(0x200000), dW=_fake(0x300000), exp_avg=_fake(0x400000),
              exp_avg_sq=_fake(0x500000), W_master=0, stream=0)
    cases = [
        (dict(W=0), {}, B.LCE_ERR_NULL), (dict(exp_avg=0), {}, B.LCE_ERR_NULL),
        (dict(exp_avg_sq=0x500004), {}, B.LCE_ERR_ALIGN), (dict(W_master=0x600008), {}, B.LCE_ERR_ALIGN),
        (dict(d=60), {}, B.LCE_ERR_UNSUPPORTED), (dict(v=0), {}, B.LCE_ERR_SHAPE),
        (dict(ld_w=32), {}, B.LCE_ERR_SHAPE), (dict(ld_w=68), {}, B.LCE_ERR_ALIGN),
        ({}, dict(step=0), B.LCE_ERR_ARG), ({}, dict(beta1=1.0), B.LCE_ERR_ARG),
        ({}, dict(beta2=-0.1), B.LCE_ERR_ARG), ({}, dict(lr=float("nan")), B.LCE_ERR_ARG),
        ({}, dict(eps=-1.0), B.LCE_ERR_ARG), ({}, dict(weight_decay=float("inf")), B.LCE_ERR_ARG),
    ]
    for change, hp, code in cases:
        with pytest.raises(B.LceError) as e:
            B.lce_adamw_step(**dict(ok, **change), opt=B.adamw(**dict(HP, **hp)))
        assert e.value.code == code, (change, hp)
    opt = B.adamw(**HP)
    opt.reserved = 3
    with pytest.raises(B.LceError) as e:
        B.lce_adamw_step(**ok, opt=opt)
    assert e.value.code == B.LCE_ERR_ARG


def test_backward_adamw_argument_checks_run_before_any_launch():
    p = B.problem(8, 64, 10)
    _, bwd = B.lce_workspace_size(p)
    ok = dict(H=_fake(), W=_fake(0x200000), targets=_fake(0x300000), lse=_fake(0x400000),
              n_valid=_fake(0x500000), grad_loss=_fake(0x600000), dH=_fake(0x700000),
              exp_avg=_fake(0x800000), exp_avg_sq=_fake(0x880000), W_master=0,
              workspace=_fake(0x900000), workspace_bytes=bwd, stream=0)
    cases = [
        (dict(W=0), B.LCE_ERR_NULL), (dict(exp_avg=0), B.LCE_ERR_NULL),
        (dict(exp_avg_sq=0x880008), B.LCE_ERR_ALIGN), (dict(dH=0x700004), B.LCE_ERR_ALIGN),
        (dict(workspace_bytes=16), B.LCE_ERR_WORKSPACE),
    ]
    for change, code in cases:
        with pytest.raises(B.LceError) as e:
            B.lce_backward_adamw(p, **dict(ok, **change), opt=B.adamw(**HP))
        assert e.value.code == code, change
    # one update per backward pass: accumulation cannot be combined with the fused step
    with pytest.raises(B.LceError) as e:
        B.lce_backward_adamw(B.problem(8, 64, 10, flags=B.LCE_FLAG_ACCUMULATE_DW), **ok, opt=B.adamw(**HP))
    assert e.value.code == B.LCE_ERR_ARG
    with pytest.raises(B.LceError) as e:
        B.lce_backward_adamw(p, **ok, opt=B.adamw(**dict(HP, step=-2)))
    assert e.value.code == B.LCE_ERR_ARG


def test_shard_argument_checks_run_before_any_launch():
    p = B.problem(8, 64, 10)
    fwd, bwd = B.lce_workspace_size(p)
    fok = dict(H=_fake(), W=_fake(0x200000), targets=_fake(0x300000), lse_part=_fake(0x400000),
               tgt_part=_fake(0x500000), n_valid=_fake(0x600000), dev_status=0,
               workspace=_fake(0x700000), workspace_bytes=fwd, stream=0)
    for shard, code in [(B.LceShard(20, 11), B.LCE_ERR_SHAPE),     # rows 11..20 leave [0, 20)
                        (B.LceShard(20, -1), B.LCE_ERR_SHAPE),
                        (B.LceShard(1 << 30, 0), B.LCE_ERR_SHAPE),
                        (B.LceShard(9, 0), B.LCE_ERR_SHAPE)]:
        with pytest.raises(B.LceError) as e:
            B.lce_forward_shard(p, shard, **fok)
        assert e.value.code == code, (shard.v_total, shard.v_begin)
    with pytest.raises(B.LceError) as e:
        B.lce_forward_shard(p, B.LceShard(20, 10), **dict(fok, tgt_part=0))
    assert e.value.code == B.LCE_ERR_NULL
    cok = dict(lse_parts=_fake(0x200000), tgt_parts=_fake(0x300000), targets=_fake(0x400000),
               loss=_fake(0x500000), lse=_fake(0x600000), n_valid=_fake(0x700000), dev_status=0,
               workspace=_fake(0x800000), workspace_bytes=fwd, stream=0)
    for n_shards, change, code in [(0, {}, B.LCE_ERR_ARG), (5000, {}, B.LCE_ERR_ARG),
                                   (2, dict(tgt_parts=0), B.LCE_ERR_NULL),
                                   (2, dict(workspace_bytes=64), B.LCE_ERR_WORKSPACE)]:
        with pytest.raises(B.LceError) as e:
            B.lce_combine_shards(p, n_shards, **dict(cok, **change))
        assert e.value.code == code, (n_shards, change)
    bok = dict(H=_fake(), W=_fake(0x200000), targets=_fake(0x300000), lse=_fake(0x400000),
               n_valid=_fake(0x500000), grad_loss=_fake(0x600000), dH_part=_fake(0x700000),
               dW=_fake(0x800000), workspace=_fake(0x900000), workspace_bytes=bwd, stream=0)
    for change, code in [(dict(dH_part=0), B.LCE_ERR_NULL), (dict(dW=0x800008), B.LCE_ERR_ALIGN),
                         (dict(workspace_bytes=16), B.LCE_ERR_WORKSPACE)]:
        with pytest.raises(B.LceError) as e:
            B.lce_backward_shard(p, B.LceShard(20, 10), **dict(bok, **change))
        assert e.value.code == code, change


def test_kd_argument_checks_run_before_any_launch():
    p = B.kd_problem(8, 64, 96, 10)
    fwd, bwd = B.lce_kd_workspace_size(p)
    assert fwd > 0 and bwd > 0
    for kw, code in [(dict(temperature=0.0), B.LCE_ERR_ARG), (dict(temperature=float("nan")), B.LCE_ERR_ARG),
                     (dict(flags=4), B.LCE_ERR_ARG)]:
        with pytest.raises(B.LceError) as e:
            B.lce_kd_workspace_size(B.kd_problem(8, 64, 96, 10, **kw))
        assert e.value.code == code, kw
    with pytest.raises(B.LceError) as e:
        B.lce_kd_workspace_size(B.kd_problem(8, 64, 90, 10))            # teacher width not a multiple of 8
    assert e.value.code == B.LCE_ERR_UNSUPPORTED
    q = B.kd_problem(8, 64, 96, 10)
    q.reserved = 1
    with pytest.raises(B.LceError) as e:
        B.lce_kd_workspace_size(q)
    assert e.value.code == B.LCE_ERR_ARG
    fok = dict(Hs=_fake(), Ws=_fake(0x200000), Ht=_fake(0x300000), Wt=_fake(0x400000), targets=_fake(0x500000),
               loss=_fake(0x600000), lse_s=_fake(0x700000), lse_t=_fake(0x800000), n_valid=_fake(0x900000),
               dev_status=0, workspace=_fake(0xA00000), workspace_bytes=fwd, stream=0)
    for change, code in [(dict(Ht=0), B.LCE_ERR_NULL), (dict(lse_t=0), B.LCE_ERR_NULL),
                         (dict(Wt=0x400008), B.LCE_ERR_ALIGN), (dict(workspace_bytes=fwd - 1), B.LCE_ERR_WORKSPACE)]:
        with pytest.raises(B.LceError) as e:
            B.lce_kd_forward(p, **dict(fok, **change))
        assert e.value.code == code, change
    bok = dict(Hs=_fake(), Ws=_fake(0x200000), Ht=_fake(0x300000), Wt=_fake(0x400000), targets=_fake(0x500000),
               lse_s=_fake(0x600000), lse_t=_fake(0x700000), n_valid=_fake(0x800000), grad_loss=_fake(0x900000),
               dHs=_fake(0xA00000), dWs=_fake(0xB00000), workspace=_fake(0xC00000), workspace_bytes=bwd, stream=0)
    for change, code in [(dict(dWs=0), B.LCE_ERR_NULL), (dict(lse_t=0), B.LCE_ERR_NULL),
                         (dict(Ht=0x300004), B.LCE_ERR_ALIGN), (dict(workspace_bytes=bwd - 1), B.LCE_ERR_WORKSPACE)]:
        with pytest.raises(B.LceError) as e:
            B.lce_kd_backward(p, **dict(bok, **change))
        assert e.value.code == code, change


def test_overlapping_rows_are_copied_before_the_call():
    # an expand()ed tensor has row stride 0, which the library would read as "dense" rows
    from paper_2605_21442_amd.autograd import _rows_usable
    assert not _rows_usable((4, 64), (0, 1), 0)          # expand() of one row
    assert not _rows_usable((4, 64), (32, 1), 0)         # rows overlapping by half
    assert not _rows_usable((4, 64), (64, 2), 0)         # non-unit column stride
    assert not _rows_usable((4, 64), (72, 1), 8)         # misaligned start
    assert not _rows_usable((4, 64), (68, 1), 0)         # row stride not a multiple of 8
    assert _rows_usable((4, 64), (64, 1), 0)             # dense
    assert _rows_usable((4, 64), (160, 1), 64)           # strided view of wider rows
    assert _rows_usable((1, 64), (0, 1), 0)              # one row: its stride is never used


def test_noalloc_forward_rejects_problems_beyond_its_array_before_any_launch():
    # the Qwen2.5-7B head's forward workspace is larger than the library's fixed array: rejected
    # before any HIP call, so this runs without a GPU
    p = B.problem(32768, 3584, 152064)
    assert B.lce_workspace_size(p)[0] > B.LCE_NOALLOC_SCRATCH_BYTES
    with pytest.raises(B.LceError) as e:
        B.lce_forward_noalloc(p, _fake(), _fake(), _fake(), _fake(), _fake(), _fake(), 0, 0)
    assert e.value.code == B.LCE_ERR_WORKSPACE
    with pytest.raises(B.LceError) as e:
        B.lce_forward_noalloc(B.problem(4, 60, 10), _fake(), _fake(), _fake(), _fake(), _fake(), _fake(), 0, 0)
    assert e.value.code == B.LCE_ERR_UNSUPPORTED


def test_loading_the_library_first_keeps_one_hip_runtime_in_the_process():
    # torch carries its own HIP runtime; the library must bind to it even when it is loaded before
    # torch is imported (two runtimes in one process leave the library's launches without a device)
    import subprocess
    import sys
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2605_21442_amd import binding as B\n"
            "B.load()\n"
            "import torch\n"
            "maps = open('/proc/self/maps').read()\n"
            "print(sorted({l.split()[-1] for l in maps.splitlines() if 'libamdhip64' in l}))\n") % ROOT
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    libs = eval(r.stdout.strip().splitlines()[-1])
    assert len(libs) == 1, libs

