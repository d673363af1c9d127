"""The seeded input generator: determinism, exact mask counts, bf16 rounding."""
import numpy as np
import pytest
import torch

from paper_2605_21442_amd import workloads as WL


def test_same_seed_same_bytes_and_different_seed_differs():
    wl = WL.WORKLOADS["tiny"]
    a, b, c = WL.generate(wl, 0), WL.generate(wl, 0), WL.generate(wl, 1)
    assert np.array_equal(a.h_bits, b.h_bits) and np.array_equal(a.w_bits, b.w_bits)
    assert np.array_equal(a.targets, b.targets)
    assert not np.array_equal(a.h_bits, c.h_bits)


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 3.0
    x[:4] = [0.0, -0.0, 1e-40, 3.4e38]
    ours = WL.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = WL.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


@pytest.mark.parametrize("name", ["tiny", "llama1b"])
def test_mask_counts_and_target_ranges(name):
    wl = WL.WORKLOADS[name]
    inp = WL.generate(wl, 0, draw_w=False)
    t = inp.targets
    assert t.dtype == np.int32 and t.shape == (wl.n,)
    assert int((t == -100).sum()) == wl.masked_count()
    valid = t[t != -100]
    assert valid.min() >= 0 and valid.max() < wl.v


def test_prefix_masks_cover_the_start_of_each_sequence():
    wl = WL.Workload("p", n=64, d=8, v=100, batch=4, seq=16, mask_frac=0.25,
                     mask_kind="prefix", case_id=7)
    t = WL.generate(wl, 0).targets.reshape(4, 16)
    assert np.all(t[:, :4] == -100) and np.all(t[:, 4:] != -100)


def test_zipf_targets_favour_low_ids():
    t = WL.draw_targets(np.random.default_rng(0), 200000, 128256, "zipf", 1.1)
    # P(id = 0) = 1 / H_{V,1.1}; generalised harmonic number of 128256 terms
    k = np.arange(1, 128257, dtype=np.float64)
    p0 = 1.0 / np.sum(k ** -1.1)
    assert abs(np.mean(t == 0) - p0) < 4 * np.sqrt(p0 / 200000)
    assert t.max() < 128256


def test_named_workload_sizes():
    sizes = {k: (w.n, w.d, w.v, w.n_valid()) for k, w in WL.WORKLOADS.items()}
    assert sizes["tiny"] == (256, 512, 4096, 230)
    assert sizes["llama1b"] == (8192, 2048, 128256, 6144)
    assert sizes["llama8b"] == (16384, 4096, 128256, 12288)
    assert sizes["qwen7b"] == (32768, 3584, 152064, 22936)
    assert sizes["llama70b"] == (16384, 8192, 128256, 13107)
