"""Plain CPU oracle of the AdamW update applied inside the LCE backward.

TEST INFRASTRUCTURE ONLY. Only the tests, the package's ``smoke()`` check and
the benchmark's CPU-baseline leg may import this module. The product path never
calls it and shares no code with it.

What it computes (paper Sec. 4.1, in-backward optimizer fusion, combined with
the LCE loss of Sec. 4.2): as soon as the gradient of a parameter exists, an
AdamW step consumes it and the gradient is dropped. For the output projection
W of the LCE loss the gradient is dW = G^T H (the LCE oracle's backward), so
the fused operation is "LCE backward, then one AdamW step on W with dW"; with
one update per backward pass the result is the same as the two-phase
"backward, then optimizer step". The update is AdamW with decoupled weight
decay (Loshchilov & Hutter) and bias-corrected moments (Kingma & Ba); the
paper names it only as the standard optimizer it swaps for, so the oracle is
that textbook step in float64:

  theta <- theta * (1 - lr * weight_decay)
  m     <- beta1 * m + (1 - beta1) * g
  v     <- beta2 * v + (1 - beta2) * g^2
  theta <- theta - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)

with t the 1-based index of the step. When the parameter is stored in bf16
without a float32 master copy, the new value is rounded to the nearest bf16
(ties to even); the moments are float32 state on the GPU and float64 here.

Pins (``tests/test_adamw_oracle.py``): torch.optim.AdamW on CPU float64 over
several steps (an independent library routine), the closed form of the first
step, zero-gradient decay, the beta = 0 memoryless case and the scale
invariance of the update.
"""
from __future__ import annotations

import numpy as np

from .lce_oracle import backward, bf16_to_f64


def adamw_step(theta, grad, m, v, *, lr, beta1, beta2, eps, weight_decay, step):
    """One AdamW step in float64; returns new (theta, m, v) without touching the inputs."""
    if step < 1:
        raise ValueError("step is 1-based")
    theta = np.asarray(theta, dtype=np.float64) * (1.0 - lr * weight_decay)
    g = np.asarray(grad, dtype=np.float64)
    m = beta1 * np.asarray(m, dtype=np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, dtype=np.float64) + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** step)
    v_hat = v / (1.0 - beta2 ** step)
    theta = theta - lr * m_hat / (np.sqrt(v_hat) + eps)
    return theta, m, v


def f64_to_bf16_bits(x) -> np.ndarray:
    """Nearest bf16 (ties to even) of float64 values, as uint16 bit patterns (finite inputs).

    The rounding is done on the float64 value directly: the bf16 grid near x has spacing
    2^(e - 7) for x in [2^e, 2^(e+1)); rint rounds half to even, and an even multiple of the
    spacing is exactly a bf16 with an even last mantissa bit.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros(x.shape, dtype=np.float64)
    nz = x != 0
    e = np.floor(np.log2(np.abs(x[nz])))
    e = np.maximum(e, -126.0)                         # subnormal bf16 share the 2^-133 spacing
    q = np.ldexp(1.0, (e - 7).astype(np.int64))
    out[nz] = np.rint(x[nz] / q) * q
    out[~nz] = x[~nz]                                 # keep the sign of zero
    f32 = out.astype(np.float32)                      # exact: every bf16 value is a float32
    return (f32.view(np.uint32) >> 16).astype(np.uint16)


def lce_adamw(h_bits, w_bits, targets, m, v, master=None, *, lr, beta1, beta2, eps,
              weight_decay, step, ignore_index=-100, reduction="mean", grad=1.0):
    """LCE backward followed by one AdamW step on W (Sec. 4.1 with Sec. 4.2).

    ``master`` (float array [V, D] or None) is the parameter's full-precision copy; without it
    the parameter is the bf16 W itself. Returns dH and the new W (float64 and its bf16 bits), m,
    v and master.
    """
    h = bf16_to_f64(h_bits)
    w = bf16_to_f64(w_bits)
    bw = backward(h, w, targets, ignore_index, reduction, grad)
    theta0 = w if master is None else np.asarray(master, dtype=np.float64)
    theta, m1, v1 = adamw_step(theta0, bw["dW"], m, v, lr=lr, beta1=beta1, beta2=beta2, eps=eps,
                               weight_decay=weight_decay, step=step)
    return {"dH": bw["dH"], "dW": bw["dW"], "theta": theta, "W_bits": f64_to_bf16_bits(theta),
            "m": m1, "v": v1}

