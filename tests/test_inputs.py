"""The synthetic input recipe (CPU): the water-filled Zipf targets of the
skewed workload and the calibrated router bias that produces them."""
import numpy as np

from oracle import oracle
from paper_2601_05296_amd import synth


def test_zipf_targets_water_filling():
    E, k, s = 128, 8, 1.2
    t = synth.zipf_targets(E, k, s)
    assert abs(t.sum() - 1.0) < 1e-12
    assert np.all(t <= 1.0 / k + 1e-15) and np.all(np.diff(t) <= 0)
    capped = t >= 1.0 / k - 1e-15
    assert capped.sum() == 2                       # the first two ranks saturate
    # below the cap the shares keep the Zipf ratios r^-s
    r = np.arange(1, E + 1, dtype=np.float64)
    free = ~capped
    ratio = t[free] / r[free] ** -s
    assert np.allclose(ratio, ratio[0], rtol=1e-12)
    # no cap binds: plain Zipf
    t1 = synth.zipf_targets(8, 1, 1.2)
    w = np.arange(1, 9, dtype=np.float64) ** -1.2
    assert np.allclose(t1, w / w.sum(), rtol=1e-12)


def test_calibrated_bias_table():
    cfg = synth.CONFIGS["many_small_zipf"]
    b = synth.load_calibrated_bias(cfg)
    assert b is not None and b.shape == (cfg.E,) and np.all(np.isfinite(b))
    inp = synth.make_inputs(cfg, T=1, with_dy=False, experts=False)
    assert np.array_equal(inp.vals["bias"], b)
    # more popular ranks get larger biases (in blocks of ranks: single tail
    # experts differ by their own router weights)
    by_rank = b[np.argsort(synth.zipf_ranks(cfg))]
    blocks = [by_rank[:2].mean(), by_rank[2:8].mean(), by_rank[8:32].mean(), by_rank[32:].mean()]
    assert all(x > y for x, y in zip(blocks, blocks[1:]))
    # a table made for other sizes is not used
    assert synth.load_calibrated_bias(cfg.with_(d=cfg.d * 2)) is None


def test_calibrated_loads_on_a_sample():
    """Routing the workload's first 8192 tokens with the calibrated bias puts
    every expert's load near its water-filled target."""
    cfg = synth.CONFIGS["many_small_zipf"]
    T = 8192
    inp = synth.make_inputs(cfg, T=T, with_dy=False, experts=False)
    ids, _, _, _ = oracle.route(inp.vals["x"], inp.vals["w_gate"], inp.vals["bias"], cfg.k, False)
    obs = np.bincount(ids.reshape(-1), minlength=cfg.E).astype(np.float64)
    tgt = synth.zipf_targets(cfg.E, cfg.k, cfg.zipf_s)[synth.zipf_ranks(cfg) - 1] * T * cfg.k
    head = tgt >= T - 0.5
    assert np.all(obs[head] >= 0.97 * T)
    rel = np.abs(obs - tgt) / tgt
    # sampling noise of about 1/sqrt(64) at the smallest targets of this sample
    assert np.all(rel < 0.45) and np.median(rel) < 0.1
