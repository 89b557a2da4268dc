"""Writes tests/golden/ternary_envelope.txt: the rounding-noise envelope of
the 24-layer W2A8 workload, computed with the CPU oracle only.

The W2A8 stack quantises every projection input to int8 per token; on these
random weights most activation codes are small, so any rounding difference
upstream of a quantiser (fp32 vs fp64 accumulation order, bf16 storage)
flips codes and the flips compound over the layers.  Two equally valid
evaluations therefore differ by the stack's own quantisation noise.  This
script measures that spread: the plain fp64 oracle is re-run with
every quantiser input multiplied by (1 + 1e-5 * N(0,1)) for several seeds,
and the largest max|d| and mean|d| against the unperturbed run are recorded.

Usage: python tests/golden/make_ternary_envelope.py
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402
from oracle import vla_oracle as O  # noqa: E402

JITTER = 1e-5
SEEDS = 4


def main():
    cfg = wl.TERNARY_W2A8
    W = wl.make_weights(cfg)
    inp = wl.make_batch(cfg, 1)
    tau = wl.uniform_schedule(cfg.n_steps)
    cache = O.prefix_kv_build(cfg, W, inp["prefix"])
    ref = O.denoise(cfg, W, cache, inp["noise"], inp["state"], tau)
    orig = O.quantize_int8_rows
    maxes, means = [], []
    for seed in range(SEEDS):
        rng = np.random.default_rng(seed)

        def jittered(u, rng=rng):
            u = np.asarray(u, np.float32)
            return orig((u * (1 + JITTER * rng.standard_normal(u.shape))).astype(np.float32))

        O.quantize_int8_rows = jittered
        try:
            out = O.denoise(cfg, W, cache, inp["noise"], inp["state"], tau)
        finally:
            O.quantize_int8_rows = orig
        d = np.abs(out - ref)
        maxes.append(float(d.max()))
        means.append(float(d.mean()))
        print(f"seed {seed}: max {maxes[-1]:.4f} mean {means[-1]:.5f}", flush=True)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "ternary_envelope.txt")
    with open(path, "w") as f:
        f.write("# Rounding-noise envelope of the 24-layer W2A8 workload (ternary_w2a8),\n")
        f.write("# written by tests/golden/make_ternary_envelope.py from the CPU oracle only.\n")
        f.write(f"# {SEEDS} runs with quantiser inputs jittered by 1 + {JITTER} N(0,1) vs the exact run.\n")
        f.write("# columns: envelope_max_abs envelope_mean_abs rms_of_reference\n")
        f.write(f"{max(maxes):.6f} {max(means):.6f} {float(np.sqrt(np.mean(ref ** 2))):.6f}\n")
    print("wrote", path)


if __name__ == "__main__":
    main()
