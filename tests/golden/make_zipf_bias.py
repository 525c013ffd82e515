"""Calibrate the router bias of the skewed many-small-experts workload.

Writes tests/golden/zipf_bias_many_small_zipf.txt, which the input generator
(paper_2601_05296_amd/synth.py) reads in place of its analytic bias.

The expert loads of this workload are meant to follow Zipf(1.2) popularity,
water-filled at 1/k (an expert takes every token at most once, so the two
most popular experts saturate at T choices and the excess goes down the
ranks). A bias b_e is added to the router logits before the softmax. It is
found by fixed-point steps

    b_e += 0.5 * (log target_e - log observed_e)

on a calibration draw of x (its own seed, not the workload's x), with the
workload's own router weights and rank permutation. The observed loads come
from the oracle's routing (oracle.route: fp64 logits, top-k with ties to the
lower id). This script calls nothing but the oracle and the input generator.

    python tests/golden/make_zipf_bias.py
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import oracle  # noqa: E402
from paper_2601_05296_amd import synth  # noqa: E402

NAME = "many_small_zipf"
T_CAL = 65536
STEPS = 60
CAL_SEED = 0xCA1B


def main():
    cfg = synth.CONFIGS[NAME]
    E, k, d = cfg.E, cfg.k, cfg.d
    wg = synth.make_inputs(cfg, T=1, with_dy=False).vals["w_gate"].astype(np.float64)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, CAL_SEED])))
    x = synth.bf16_to_f32(synth.bf16_round(rng.standard_normal((T_CAL, d), dtype=np.float32)))
    x = x.astype(np.float64)
    rank = synth.zipf_ranks(cfg)
    target = synth.zipf_targets(E, k, cfg.zipf_s)[rank - 1] * T_CAL * k
    # start from the analytic bias (Gumbel-scale Zipf weights)
    sigma = 0.02 * np.sqrt(d)
    bias = -cfg.zipf_s * sigma * np.sqrt(6.0) / np.pi * np.log(rank.astype(np.float64))
    for step in range(STEPS):
        ids, _, _, _ = oracle.route(x, wg, bias.astype(np.float32), k, False)
        obs = np.bincount(ids.reshape(-1), minlength=E).astype(np.float64)
        err = np.abs(np.log(np.maximum(obs, 0.5) / target))
        print("step %2d: max |log(observed/target)| = %.4f" % (step, err.max()), flush=True)
        bias = (bias + 0.5 * (np.log(target) - np.log(np.maximum(obs, 0.5)))).astype(np.float32)
        bias = bias.astype(np.float64)
    ids, _, _, _ = oracle.route(x, wg, bias.astype(np.float32), k, False)
    obs = np.bincount(ids.reshape(-1), minlength=E)
    out = os.path.join(ROOT, "tests", "golden", "zipf_bias_%s.txt" % NAME)
    order = np.argsort(rank)
    with open(out, "w") as fh:
        fh.write("# router bias of the %s workload, calibrated by tests/golden/make_zipf_bias.py\n"
                 % NAME)
        fh.write("# targets: Zipf(%g) shares water-filled at 1/k; calibration draw of %d tokens "
                 "(seed [%d, %d]); %d fixed-point steps\n" % (cfg.zipf_s, T_CAL, cfg.seed, CAL_SEED,
                                                            STEPS))
        fh.write("# loads of the calibration draw, most popular first: %s ... %s\n"
                 % (" ".join(str(int(obs[e])) for e in order[:6]),
                    " ".join(str(int(obs[e])) for e in order[-3:])))
        fh.write("d %d\nE %d\nk %d\nzipf_s %g\n" % (d, E, k, cfg.zipf_s))
        fh.write("# bias <expert> <value> <rank> <target> <calibration load>\n")
        for e in range(E):
            fh.write("bias %d %.9g %d %.1f %d\n" % (e, np.float32(bias[e]), rank[e], target[e],
                                                  obs[e]))
    print("wrote", out)


if __name__ == "__main__":
    main()
