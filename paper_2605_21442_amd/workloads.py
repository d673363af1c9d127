"""Seeded synthetic inputs for the linear-cross-entropy (LCE) hot path.

This module only *draws* inputs: hidden states H, the output-projection weight
W and the target ids. It holds none of the objective's arithmetic, so both the
HIP path and the CPU oracle can be fed from it without sharing any of the
method's code.

The five named workloads are vocabulary-head shapes of the models the paper
fine-tunes (Sec. 3.2 model zoo, Tab. 1-2 and App. D): a tiny case that the
oracle finishes in seconds, and Llama-3.2-1B, Llama-3.1-8B, Qwen2.5-7B
(long sequence) and Llama-3.1-70B heads. The paper measures on Alpaca-style
SFT data with real checkpoints (Sec. 5.1); neither is available here, and the
LCE kernels only see shapes and value statistics, so seeded synthetic tensors
with the same shapes stand in for them:

* H ~ N(0, 1) rounded to bf16 (round-to-nearest-even), shape [N, D], row
  n = b * seq + s;
* W ~ N(0, sigma_w) rounded to bf16, shape [V, D] (``nn.Linear(D, V).weight``);
* targets: uniform ids (tiny case) or a truncated Zipf law
  P(id = k) ~ (k + 1)^-1.1 over the vocabulary (frequent ids low, as in BPE
  vocabularies), drawn by inverse CDF;
* a masked share of positions set to ``ignore_index`` (-100), standing in for
  the prompt tokens that SFT masks: an exact count drawn uniformly without
  replacement, or a contiguous prompt span at the start of every sequence.

Every stream uses ``numpy.random.Generator(PCG64(SeedSequence([seed, case,
stream])))`` so a (workload, seed) pair always gives the same bytes.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

IGNORE_INDEX = -100

# RNG stream ids
_S_H, _S_W, _S_T, _S_MASK, _S_OPT, _S_GRAD = 0, 1, 2, 3, 4, 5


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and value recipe of one LCE input set."""

    name: str
    n: int                      # tokens = batch * seq
    d: int                      # hidden size
    v: int                      # vocabulary size
    batch: int = 1
    seq: int = 0                # 0 means n
    sigma_w: float = 0.02
    targets: str = "zipf"       # "zipf" | "uniform"
    zipf_s: float = 1.1
    mask_frac: float = 0.0      # share of positions set to ignore_index
    mask_kind: str = "random"   # "random" | "prefix" (contiguous prompt span per sequence)
    case_id: int = 0            # RNG domain separator

    @property
    def seq_len(self) -> int:
        return self.seq if self.seq else self.n

    def masked_count(self) -> int:
        if self.mask_kind == "prefix":
            return self.batch * int(round(self.mask_frac * self.seq_len))
        return int(round(self.mask_frac * self.n))

    def n_valid(self) -> int:
        return self.n - self.masked_count()

    def flops(self) -> float:
        """Algorithmic multiply-add work of one fwd+bwd: 8 * Nv * D * V."""
        return 8.0 * self.n_valid() * self.d * self.v


# The five workloads, in order: tiny, Llama-3.2-1B, Llama-3.1-8B, Qwen2.5-7B, Llama-3.1-70B.
WORKLOADS = {
    "tiny": Workload("tiny", n=256, d=512, v=4096, targets="uniform",
                     mask_frac=0.10, case_id=1),
    "llama1b": Workload("llama1b", n=8192, d=2048, v=128256, batch=4, seq=2048,
                        mask_frac=0.25, case_id=2),
    "llama8b": Workload("llama8b", n=16384, d=4096, v=128256, batch=8, seq=2048,
                        mask_frac=0.25, case_id=3),
    "qwen7b": Workload("qwen7b", n=32768, d=3584, v=152064, batch=4, seq=8192,
                       mask_frac=0.30, mask_kind="prefix", case_id=4),
    "llama70b": Workload("llama70b", n=16384, d=8192, v=128256, batch=2, seq=8192,
                         sigma_w=0.015, mask_frac=0.20, case_id=5),
    # A check case, not a benchmark workload: the 8B head's tokens, targets, mask and weight draws
    # (same case id) with the weights scaled up (sigma_w = 0.125), so that each row's softmax is
    # peaked and the softmax part of G carries more than half of dH and dW (at 0.02 the logits are
    # nearly flat and the one-hot part dominates both); same shapes, so the same launch plan.
    "llama8b_spread": Workload("llama8b_spread", n=16384, d=4096, v=128256, batch=8, seq=2048,
                               sigma_w=0.125, mask_frac=0.25, case_id=3),
}


def _rng(seed: int, case: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, case, stream])))


_SLAB = 1 << 22


def f32_to_bf16_bits(x: np.ndarray, scale: Optional[float] = None) -> np.ndarray:
    """Round float32 values (times ``scale`` in float32, if given) to bfloat16 (nearest, ties to
    even); returns uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    # in slabs through temporaries allocated once (fresh large allocations cost a page fault per
    # page, which dominates for billion-element weights); 32-bit arithmetic wraps only for NaN
    # patterns, which are replaced (quiet NaN with the payload's top bits)
    flat_x, flat_o = x.reshape(-1), out.reshape(-1)
    m = min(_SLAB, flat_x.size)
    f = np.empty(m, dtype=np.float32)
    r = np.empty(m, dtype=np.uint32)
    t = np.empty(m, dtype=np.uint32)
    for s in range(0, flat_x.size, _SLAB):
        k = min(_SLAB, flat_x.size - s)
        fb, rb, tb = f[:k], r[:k], t[:k]
        if scale is None:
            fb[...] = flat_x[s:s + k]
        else:
            np.multiply(flat_x[s:s + k], np.float32(scale), out=fb)
        b = fb.view(np.uint32)
        np.right_shift(b, 16, out=rb)
        np.bitwise_and(rb, 1, out=rb)
        np.add(rb, b, out=rb)
        np.add(rb, 0x7FFF, out=rb)
        np.right_shift(rb, 16, out=rb)
        np.bitwise_and(b, 0x7FFFFFFF, out=tb)
        nan = tb > 0x7F800000
        if nan.any():
            rb[nan] = (b[nan] >> 16) | 0x40
        flat_o[s:s + k] = rb
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def draw_normal_bf16(rng: np.random.Generator, shape, sigma: float) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    return f32_to_bf16_bits(x, None if sigma == 1.0 else sigma)


def draw_targets(rng: np.random.Generator, n: int, v: int, kind: str, zipf_s: float) -> np.ndarray:
    if kind == "uniform":
        return rng.integers(0, v, size=n, dtype=np.int64).astype(np.int32)
    if kind == "zipf":
        p = np.arange(1, v + 1, dtype=np.float64) ** (-zipf_s)
        cdf = np.cumsum(p)
        cdf /= cdf[-1]
        u = rng.random(n)
        t = np.searchsorted(cdf, u, side="right")
        return np.minimum(t, v - 1).astype(np.int32)
    raise ValueError(f"unknown target distribution {kind!r}")


def apply_mask(rng: np.random.Generator, t: np.ndarray, w: Workload,
               ignore_index: int = IGNORE_INDEX) -> np.ndarray:
    t = t.copy()
    if w.mask_frac <= 0:
        return t
    if w.mask_kind == "prefix":
        span = int(round(w.mask_frac * w.seq_len))
        for b in range(w.batch):
            t[b * w.seq_len: b * w.seq_len + span] = ignore_index
    elif w.mask_kind == "random":
        k = w.masked_count()
        pos = rng.choice(w.n, size=k, replace=False)
        t[pos] = ignore_index
    else:
        raise ValueError(f"unknown mask kind {w.mask_kind!r}")
    return t


@dataclasses.dataclass
class Inputs:
    """One drawn input set: bf16 bit patterns for H and W, int32 targets."""

    workload: Workload
    seed: int
    h_bits: np.ndarray          # uint16 [N, D]
    w_bits: np.ndarray          # uint16 [V, D]
    targets: np.ndarray         # int32 [N]
    ignore_index: int = IGNORE_INDEX


def weight_normals(w: Workload, seed: int = 0) -> np.ndarray:
    """The standard normal draws [V, D] (float32) behind workload ``w``'s weight: W is their bf16
    rounding after scaling by sigma_w, so workloads that share a case id share these draws."""
    return _rng(seed, w.case_id, _S_W).standard_normal((w.v, w.d), dtype=np.float32)


def weight_bits(z: np.ndarray, sigma: float) -> np.ndarray:
    """bf16 bit patterns of the weight ``sigma * z`` (z from weight_normals; the product in float32)."""
    return f32_to_bf16_bits(z, sigma)


def generate(w: Workload, seed: int = 0, *, draw_w: bool = True,
             ignore_index: int = IGNORE_INDEX) -> Inputs:
    """Draw the inputs of workload ``w``; ``draw_w=False`` leaves W empty (for callers that only need H and targets)."""
    h = draw_normal_bf16(_rng(seed, w.case_id, _S_H), (w.n, w.d), 1.0)
    wb = weight_bits(weight_normals(w, seed), w.sigma_w) if draw_w else np.empty((0, w.d), np.uint16)
    t = draw_targets(_rng(seed, w.case_id, _S_T), w.n, w.v, w.targets, w.zipf_s)
    t = apply_mask(_rng(seed, w.case_id, _S_MASK), t, w, ignore_index)
    return Inputs(w, seed, h, wb, t, ignore_index)


def custom(n: int, d: int, v: int, *, seed: int = 0, sigma_w: float = 0.02,
           sigma_h: float = 1.0, targets: str = "uniform", mask_frac: float = 0.1,
           mask_kind: str = "random", batch: int = 1, case_id: int = 99,
           ignore_index: int = IGNORE_INDEX, target_override: Optional[np.ndarray] = None) -> Inputs:
    """Small ad-hoc input sets for edge cases (ragged tiles, tiny V, all-masked ...)."""
    w = Workload(f"custom_{n}x{d}x{v}", n=n, d=d, v=v, batch=batch,
                 seq=(n // batch if batch > 1 else 0), sigma_w=sigma_w,
                 targets=targets, mask_frac=mask_frac, mask_kind=mask_kind, case_id=case_id)
    h = draw_normal_bf16(_rng(seed, case_id, _S_H), (n, d), sigma_h)
    wb = draw_normal_bf16(_rng(seed, case_id, _S_W), (v, d), sigma_w)
    if target_override is not None:
        t = np.asarray(target_override, dtype=np.int32).copy()
    else:
        t = draw_targets(_rng(seed, case_id, _S_T), n, v, targets, 1.1)
        t = apply_mask(_rng(seed, case_id, _S_MASK), t, w, ignore_index)
    return Inputs(w, seed, h, wb, t, ignore_index)


@dataclasses.dataclass
class OptState:
    """AdamW state of a [V, D] weight as a run would have left it (all float32)."""

    m: np.ndarray               # first moments
    v: np.ndarray               # second moments, >= 0
    master: np.ndarray          # full-precision copy of the weight


def opt_state(w_bits: np.ndarray, *, seed: int = 0, case_id: int = 99, g_scale: float = 1e-3,
              cold: bool = False) -> OptState:
    """Optimizer state for the bf16 weight ``w_bits``: zero moments (``cold``, a first step) or
    moments of gradient scale ``g_scale`` (m ~ N(0, g_scale), v ~ g_scale^2 U(0.5, 1.5)); the master
    copy is the weight plus a small float32 offset (below half a bf16 spacing of typical entries)."""
    rng = _rng(seed, case_id, _S_OPT)
    shape = w_bits.shape
    if cold:
        m = np.zeros(shape, np.float32)
        v = np.zeros(shape, np.float32)
    else:
        m = (g_scale * rng.standard_normal(shape)).astype(np.float32)
        v = ((g_scale * g_scale) * rng.uniform(0.5, 1.5, shape)).astype(np.float32)
    master = bf16_bits_to_f32(w_bits) + (1e-5 * rng.standard_normal(shape)).astype(np.float32)
    return OptState(m, v, master.astype(np.float32))


def gradient_bits(v: int, d: int, *, seed: int = 0, case_id: int = 99, g_scale: float = 1e-3) -> np.ndarray:
    """A bf16 gradient matrix [V, D] ~ N(0, g_scale) (input of a standalone optimizer step)."""
    return draw_normal_bf16(_rng(seed, case_id, _S_GRAD), (v, d), g_scale)


# ---- knowledge distillation: a student head and a teacher head over the same tokens -----------

_S_HT, _S_WT = 6, 7


@dataclasses.dataclass
class KdInputs:
    """Student (hs, ws) and teacher (ht, wt) bf16 bit patterns and int32 labels (mask only)."""

    name: str
    hs_bits: np.ndarray         # uint16 [N, Ds]
    ws_bits: np.ndarray         # uint16 [V, Ds]
    ht_bits: np.ndarray         # uint16 [N, Dt]
    wt_bits: np.ndarray         # uint16 [V, Dt]
    targets: np.ndarray         # int32 [N]
    ignore_index: int = IGNORE_INDEX


# Distilling a Llama-3.1-8B head (teacher) into a Llama-3.2-1B head (student): same 128256-id
# vocabulary, 8 x 2048 tokens, 25 % of positions masked as prompt.
KD_WORKLOADS = {
    "kd_tiny": dict(n=256, ds=256, dt=512, v=4096, batch=1, seq=256, sigma_s=0.02, sigma_t=0.02,
                    mask_frac=0.10, targets="uniform", case_id=11),
    "kd_8b_to_1b": dict(n=16384, ds=2048, dt=4096, v=128256, batch=8, seq=2048, sigma_s=0.02,
                        sigma_t=0.02, mask_frac=0.25, targets="zipf", case_id=12),
}


def kd_generate(name: str, seed: int = 0, **over) -> KdInputs:
    """Draw the inputs of a KD workload (KD_WORKLOADS entry, fields overridable)."""
    k = dict(KD_WORKLOADS[name], **over)
    n, v, cid = k["n"], k["v"], k["case_id"]
    w = Workload(name, n=n, d=k["ds"], v=v, batch=k["batch"], seq=k["seq"], sigma_w=k["sigma_s"],
                 targets=k["targets"], mask_frac=k["mask_frac"], case_id=cid)
    hs = draw_normal_bf16(_rng(seed, cid, _S_H), (n, k["ds"]), 1.0)
    ws = draw_normal_bf16(_rng(seed, cid, _S_W), (v, k["ds"]), k["sigma_s"])
    ht = draw_normal_bf16(_rng(seed, cid, _S_HT), (n, k["dt"]), 1.0)
    wt = draw_normal_bf16(_rng(seed, cid, _S_WT), (v, k["dt"]), k["sigma_t"])
    t = draw_targets(_rng(seed, cid, _S_T), n, v, k["targets"], 1.1)
    t = apply_mask(_rng(seed, cid, _S_MASK), t, w)
    return KdInputs(name, hs, ws, ht, wt, t)


def kd_custom(n: int, ds: int, dt: int, v: int, *, seed: int = 0, sigma_s: float = 0.3,
              sigma_t: float = 0.3, mask_frac: float = 0.1, target_override=None) -> KdInputs:
    """Small ad-hoc KD inputs (ragged shapes, edge cases)."""
    over = dict(n=n, ds=ds, dt=dt, v=v, batch=1, seq=n, sigma_s=sigma_s, sigma_t=sigma_t,
                mask_frac=mask_frac, targets="uniform", case_id=13)
    inp = kd_generate("kd_tiny", seed, **over)
    if target_override is not None:
        inp.targets = np.asarray(target_override, dtype=np.int32).copy()
    return inp
