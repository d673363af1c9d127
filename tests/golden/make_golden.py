"""Write the oracle's forward results for the full-size named workloads.

Run from the repository root:  ``python tests/golden/make_golden.py [name ...]``

For each workload this draws the seeded inputs (seed 0) and stores, from the
CPU oracle only, the mean loss, Nv, the status word and lse for every row, plus
a fingerprint of the drawn inputs so a test can tell when the generator has
changed and the file is stale. The parity tests on the GPU compare against
these values and compute sampled dH / dW rows with the oracle on the fly.
"""
import hashlib
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import kd_oracle as K  # noqa: E402
from oracle import lce_oracle as O  # noqa: E402
from paper_2605_21442_amd import workloads as WL  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


def fingerprint(inp: WL.Inputs) -> str:
    h = hashlib.sha256()
    for a in (inp.h_bits[:2], inp.h_bits[-2:], inp.w_bits[:2], inp.w_bits[-2:], inp.targets):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def path_for(name: str, seed: int = 0) -> str:
    return os.path.join(HERE, f"oracle_fwd_{name}_seed{seed}.npz")


def make(name: str, seed: int = 0) -> None:
    wl = WL.WORKLOADS[name]
    t0 = time.time()
    inp = WL.generate(wl, seed)
    h = O.bf16_to_f64(inp.h_bits)
    w = O.bf16_to_f64(inp.w_bits)
    out = O.forward(h, w, inp.targets, inp.ignore_index, "mean")
    np.savez_compressed(path_for(name, seed), loss=np.float64(out["loss"]),
                        lse=out["lse"], n_valid=np.int64(out["n_valid"]),
                        status=np.int64(out["status"]), fingerprint=np.array(fingerprint(inp)),
                        workload=np.array(name), seed=np.int64(seed))
    print(f"{name}: loss={out['loss']:.9f} Nv={out['n_valid']} ({time.time() - t0:.0f} s)",
          flush=True)


def kd_fingerprint(inp: WL.KdInputs) -> str:
    h = hashlib.sha256()
    for a in (inp.hs_bits[:2], inp.ws_bits[-2:], inp.ht_bits[:2], inp.wt_bits[-2:], inp.targets):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


KD_TEMPERATURE = 2.0


def make_kd(name: str, seed: int = 0) -> None:
    """KD forward of a full-size distillation workload at temperature 2."""
    t0 = time.time()
    inp = WL.kd_generate(name, seed)
    out = K.kd_bits(inp.hs_bits, inp.ws_bits, inp.ht_bits, inp.wt_bits, inp.targets,
                    temperature=KD_TEMPERATURE, grads=False)
    np.savez_compressed(path_for(name, seed), loss=np.float64(out["loss"]), lse_s=out["lse_s"],
                        lse_t=out["lse_t"], n_valid=np.int64(out["n_valid"]), status=np.int64(out["status"]),
                        temperature=np.float64(KD_TEMPERATURE), fingerprint=np.array(kd_fingerprint(inp)),
                        workload=np.array(name), seed=np.int64(seed))
    print(f"{name}: loss={out['loss']:.9f} Nv={out['n_valid']} ({time.time() - t0:.0f} s)", flush=True)


if __name__ == "__main__":
    names = sys.argv[1:] or [k for k in WL.WORKLOADS if k != "tiny"] + ["kd_8b_to_1b"]
    for k in names:
        make_kd(k) if k in WL.KD_WORKLOADS else make(k)
