"""Seeded synthetic inputs for one MoE layer (forward + backward).

This module only draws random numbers and rounds them to the storage format.
It holds none of the layer's arithmetic: routing, dispatch, the expert FFN and
the combine live in the HIP library (product path) and in ``oracle/`` (test
infrastructure), and both receive the arrays made here.

Workloads follow the paper's setting (a single MoE layer, token-choice top-k
routing, SwiGLU experts; Sections 2 and 5.1); the paper trains on synthetic
shapes, so no dataset is involved. Shapes and distributions:

* ``x ~ N(0, 1)``            ``[T, d]``
* ``w_gate ~ N(0, 0.02)``    ``[E, d]``   (router, Section 2.1)
* ``w1, w3 ~ N(0, 1/sqrt(d))`` ``[E, d, f]`` (SiLU branch, linear branch)
* ``w2 ~ N(0, 1/sqrt(f))``   ``[E, f, d]`` (down projection)
* ``dy ~ N(0, 1)``           ``[T, d]``   (upstream gradient)

The second argument of N is the standard deviation. Independent streams are
spawned from one ``SeedSequence`` in the fixed order x, w_gate, w1, w3, w2, dy,
bias, perm, so that changing one tensor's size never changes another's values.

For the skewed many-small-experts workload a per-expert bias is added to the
router logits before the softmax. Expert ``e`` has popularity rank ``r(e)``
(a seeded permutation). The target loads are Zipf(1.2) shares of the T*k
choices water-filled at 1/k (``zipf_targets``: an expert takes every token at
most once, so the two most popular experts saturate at T and the excess goes
down the ranks). The bias that produces them is read from
``tests/golden/zipf_bias_<workload>.txt``, written once by
``tests/golden/make_zipf_bias.py`` (fixed-point steps on a calibration draw of
x with its own seed). Any other shape with ``zipf_s > 0`` takes the analytic
bias ``-s * c * log(r(e))`` with ``c = sigma * sqrt(6) / pi``, where ``sigma =
0.02 * sqrt(d)`` is the standard deviation of one router logit: with Gumbel
noise of that scale top-k selection would be Plackett-Luce sampling with
weights ``r**-s``; the Gaussian router noise makes the shares Zipf-like.
"""
from __future__ import annotations

import math
import os
from dataclasses import dataclass, field

import numpy as np

DTYPES = ("f32", "bf16")
_ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@dataclass(frozen=True)
class MoEConfig:
    name: str
    T: int
    d: int
    f: int
    E: int
    k: int
    dtype: str = "bf16"
    renorm: bool = False
    zipf_s: float = 0.0          # > 0: per-expert Zipf-shaped router bias
    n_dead: int = 0              # experts whose bias is -inf (never chosen)
    seed: int = 0
    act: str = "swiglu"          # expert: "swiglu" (gated) or non-gated "silu" / "relu"

    @property
    def S(self) -> int:
        return self.T * self.k

    def with_(self, **kw) -> "MoEConfig":
        d = dict(self.__dict__)
        d.update(kw)
        return MoEConfig(**d)


# The five layer workloads this library is measured on.
CONFIGS = {
    "tiny_f32": MoEConfig("tiny_f32", T=1024, d=256, f=512, E=8, k=2, dtype="f32"),
    "mid_e64k6": MoEConfig("mid_e64k6", T=16384, d=2048, f=1408, E=64, k=6,
                           dtype="bf16", renorm=True),
    "few_large_e8k2": MoEConfig("few_large_e8k2", T=32768, d=4096, f=14336, E=8,
                                k=2, dtype="bf16"),
    "many_small_zipf": MoEConfig("many_small_zipf", T=65536, d=2048, f=768, E=128,
                                 k=8, dtype="bf16", zipf_s=1.2),
    "mem_sweep_e64k8": MoEConfig("mem_sweep_e64k8", T=16384, d=4096, f=2048, E=64,
                                 k=8, dtype="bf16"),
    # widths that are multiples of 64 but not of 128 (partial column tiles in
    # every GEMM), at the shape of a current 128-expert top-4 model layer
    "d2880_e128k4": MoEConfig("d2880_e128k4", T=16384, d=2880, f=2880, E=128, k=4,
                              dtype="bf16"),
}

# The seven configurations of the paper's Table 1 (Section 6.1): input width
# d, experts E, top-k, batch x sequence length tokens, FFN hidden width 4d,
# with the non-gated SiLU expert of its SiLU experiments (select another
# expert with MoEConfig.with_(act=...)).
TABLE1 = {  # name: (d, E, k, batch, seq_len)
    "conf1": (512, 4, 1, 32, 2048),
    "conf2": (1024, 8, 2, 32, 2048),
    "conf3": (1024, 16, 4, 32, 2048),
    "conf4": (2048, 16, 4, 32, 1024),
    "conf5": (512, 16, 4, 32, 1024),
    "conf6": (1024, 16, 4, 16, 1024),
    "conf7": (2048, 8, 4, 16, 512),
}
for _n, (_d, _E, _k, _b, _l) in TABLE1.items():
    CONFIGS["table1_" + _n] = MoEConfig("table1_" + _n, T=_b * _l, d=_d, f=4 * _d, E=_E, k=_k,
                                        dtype="bf16", act="silu")


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns the
    16-bit patterns as uint16."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns (uint16) to float32 exactly."""
    return (b.astype(np.uint32) << 16).view(np.float32)


@dataclass
class LayerInputs:
    """Host copies of one layer's inputs.

    ``vals`` holds float32 arrays of exactly the values the device sees (for
    bf16 workloads: the bf16-rounded values, widened). ``store`` holds what is
    uploaded: uint16 bf16 patterns, or float32 for the f32 workload. ``bias``
    stays float32 in both.
    """
    cfg: MoEConfig
    vals: dict = field(default_factory=dict)
    store: dict = field(default_factory=dict)


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


def zipf_targets(E: int, k: int, s: float) -> np.ndarray:
    """Zipf(s) shares of the T*k expert choices by popularity rank (rank 1
    first), water-filled at 1/k: an expert can take at most every token once,
    so shares above 1/k are capped there and the excess is spread over the
    other ranks in proportion to their Zipf weights, until none exceeds the
    cap. Returns float64 [E] summing to 1."""
    w = np.arange(1, E + 1, dtype=np.float64) ** -s
    cap = 1.0 / k
    capped = np.zeros(E, dtype=bool)
    while True:
        free = 1.0 - cap * capped.sum()
        share = np.where(capped, cap, free * w / w[~capped].sum())
        over = (share > cap) & ~capped
        if not over.any():
            return share
        capped |= over


def zipf_ranks(cfg: MoEConfig) -> np.ndarray:
    """Popularity rank (1 = most popular) of every expert: a permutation drawn
    from the workload's own stream."""
    ss = np.random.SeedSequence(cfg.seed)
    s_perm = ss.spawn(8)[7]
    return np.random.Generator(np.random.PCG64(s_perm)).permutation(cfg.E) + 1


def calibrated_bias_path(cfg: MoEConfig) -> str:
    return os.path.join(_ROOT, "tests", "golden", "zipf_bias_%s.txt" % cfg.name)


def load_calibrated_bias(cfg: MoEConfig):
    """The calibrated router bias of a named workload (float32 [E]), or None
    when no table exists for it or the table was made for other sizes."""
    p = calibrated_bias_path(cfg)
    if not os.path.exists(p):
        return None
    head, vals = {}, []
    for line in open(p):
        parts = line.split()
        if not parts:
            continue
        if parts[0] == "#":
            continue
        if parts[0] == "bias":
            vals.append(float(parts[2]))
        else:
            head[parts[0]] = parts[1]
    if (int(head.get("d", -1)), int(head.get("E", -1)), int(head.get("k", -1)),
            float(head.get("zipf_s", -1))) != (cfg.d, cfg.E, cfg.k, cfg.zipf_s):
        return None
    assert len(vals) == cfg.E
    return np.array(vals, dtype=np.float32)


def zipf_bias(cfg: MoEConfig, rng_bias: np.random.Generator, rng_perm: np.random.Generator):
    """Per-expert router bias (float32 [E]) or None; see the module docstring."""
    if cfg.zipf_s <= 0.0 and cfg.n_dead == 0:
        return None
    E = cfg.E
    bias = np.zeros(E, dtype=np.float64)
    rank = rng_perm.permutation(E) + 1          # rank 1 = most popular
    if cfg.zipf_s > 0.0:
        table = load_calibrated_bias(cfg)
        if table is not None:
            bias = table.astype(np.float64)
        else:
            sigma = 0.02 * math.sqrt(cfg.d)
            c = sigma * math.sqrt(6.0) / math.pi
            bias = -cfg.zipf_s * c * np.log(rank.astype(np.float64))
    if cfg.n_dead > 0:
        dead = rng_bias.choice(E, size=cfg.n_dead, replace=False)
        bias[dead] = -np.inf
    return bias.astype(np.float32)


def make_inputs(cfg: MoEConfig, T: int | None = None, with_dy: bool = True,
                experts: bool = True) -> LayerInputs:
    """Draw one layer's inputs. ``T`` overrides the token count (the first T
    rows of x and dy are the same for every T, because each row is drawn from
    the same stream in order). ``experts=False`` leaves out w1, w3 and w2
    (None); the other tensors keep their values, each having its own stream."""
    T = cfg.T if T is None else T
    ss = np.random.SeedSequence(cfg.seed)
    s_x, s_g, s_w1, s_w3, s_w2, s_dy, s_bias, s_perm = ss.spawn(8)
    rng = lambda s: np.random.Generator(np.random.PCG64(s))
    d, f, E = cfg.d, cfg.f, cfg.E
    raw = {
        "x": _normal(rng(s_x), (T, d), 1.0),
        "w_gate": _normal(rng(s_g), (E, d), 0.02),
        "w1": _normal(rng(s_w1), (E, d, f), 1.0 / math.sqrt(d)) if experts else None,
        # (the W3 stream is spawned for every expert type, so the other
        # draws do not depend on it)
        "w3": (_normal(rng(s_w3), (E, d, f), 1.0 / math.sqrt(d))
               if experts and cfg.act == "swiglu" else None),
        "w2": _normal(rng(s_w2), (E, f, d), 1.0 / math.sqrt(f)) if experts else None,
    }
    if with_dy:
        raw["dy"] = _normal(rng(s_dy), (T, d), 1.0)
    out = LayerInputs(cfg.with_(T=T))
    for name, a in raw.items():
        if a is None:
            out.store[name] = out.vals[name] = None
        elif cfg.dtype == "bf16":
            b = bf16_round(a)
            out.store[name] = b
            out.vals[name] = bf16_to_f32(b)
        else:
            out.store[name] = a
            out.vals[name] = a
    bias = zipf_bias(cfg, rng(s_bias), rng(s_perm))
    out.vals["bias"] = bias
    out.store["bias"] = bias
    return out


def device_inputs(cfg: MoEConfig, device, T: int | None = None, with_dy: bool = True) -> dict:
    """Draw one layer's inputs directly on the GPU (for token counts whose host
    copies would be too large to draw and upload): a torch generator seeded
    with ``cfg.seed`` draws, in this fixed order, w_gate, w1, w3 (gated
    experts only), w2, x and dy with the distributions of the module
    docstring, each rounded to bfloat16 (round to nearest even). The values
    differ from ``make_inputs``'s (another generator); the recipe is the same.
    The Zipf bias of the skewed workload is not drawn here (None)."""
    import torch
    assert cfg.dtype == "bf16" and cfg.zipf_s == 0.0 and cfg.n_dead == 0
    T = cfg.T if T is None else T
    gen = torch.Generator(device=device)
    gen.manual_seed(cfg.seed)
    d, f, E = cfg.d, cfg.f, cfg.E

    def normal(shape, std):
        return (torch.randn(shape, generator=gen, device=device) * std).to(torch.bfloat16)

    out = {"w_gate": normal((E, d), 0.02), "w1": normal((E, d, f), d ** -0.5)}
    out["w3"] = normal((E, d, f), d ** -0.5) if cfg.act == "swiglu" else None
    out["w2"] = normal((E, f, d), f ** -0.5)
    out["x"] = normal((T, d), 1.0)
    out["dy"] = normal((T, d), 1.0) if with_dy else None
    out["bias"] = None
    return out


def random_ids(T: int, E: int, k: int, seed: int = 0, popularity=None) -> np.ndarray:
    """Random top-k expert choices [T, k] int32 with distinct ids per row.
    ``popularity`` (length E, nonnegative) skews the draw (Plackett-Luce)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if popularity is None:
        keys = rng.random((T, E))
    else:
        w = np.asarray(popularity, dtype=np.float64)
        g = rng.gumbel(size=(T, E))
        with np.errstate(divide="ignore"):
            keys = np.log(w)[None, :] + g
    ids = np.argsort(-keys, axis=1, kind="stable")[:, :k]
    return np.ascontiguousarray(ids.astype(np.int32))
