"""Pins for the CPU oracle: each test checks the oracle against something other
than itself (a printed example, a closed form, an invariant, a brute-force
dense evaluation, torch autograd, finite differences).

Section references are to the MoEBlaze paper (arXiv 2601.05296).
"""
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

from oracle import oracle
from paper_2601_05296_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            out[key] = [int(v) for v in vals]
    return out


def _tiny_layer(T=12, d=16, f=24, E=4, k=2, seed=0, zipf=0.0):
    cfg = synth.MoEConfig("t", T=T, d=d, f=f, E=E, k=k, dtype="f32", zipf_s=zipf, seed=seed)
    inp = synth.make_inputs(cfg)
    v = {n: (None if a is None else a.astype(np.float64)) for n, a in inp.vals.items()}
    # widen the router so that its logits are far apart (no near-ties under FD)
    v["w_gate"] = v["w_gate"] * 50.0
    return v


# --------------------------------------------------------------------------
# Dispatch maps (Section 4)
# --------------------------------------------------------------------------

def test_worked_example_section_4_1():
    g = _read_golden("worked_example.txt")
    E, k = g["E"][0], g["k"][0]
    ids = np.array(g["ids"], np.int32).reshape(-1, k)
    ix = oracle.build_index(ids, E)
    assert ix.eti.tolist() == g["expert_token_indices"]
    assert ix.offsets.tolist() == g["expert_token_offsets"]
    assert ix.tim.reshape(-1).tolist() == g["token_index_map"]
    assert ix.counts.tolist() == [3, 2, 2, 3]


def _check_index_invariants(ids, E, ix):
    T, k = ids.shape
    S = T * k
    assert ix.counts.sum() == S
    assert ix.offsets[0] == 0 and ix.offsets[E] == S
    assert np.all(np.diff(ix.offsets) == ix.counts)
    # every token has exactly k slots, the map is a bijection onto [0, S)
    assert np.array_equal(np.sort(ix.tim.reshape(-1)), np.arange(S))
    # eti[tim[t, j]] == t and the slot lies in its expert's segment
    t_of = np.repeat(np.arange(T), k).reshape(T, k)
    assert np.array_equal(ix.eti[ix.tim], t_of)
    seg_lo = ix.offsets[ids]
    seg_hi = ix.offsets[ids + 1]
    assert np.all((ix.tim >= seg_lo) & (ix.tim < seg_hi))
    # token ids ascend strictly inside every expert segment
    for e in range(E):
        seg = ix.eti[ix.offsets[e]:ix.offsets[e + 1]]
        assert np.all(np.diff(seg) > 0)
    # slot_src is the inverse of tim
    assert np.array_equal(ix.slot_src[ix.tim.reshape(-1)], np.arange(S))


@pytest.mark.parametrize("T,E,k,skew", [(1, 4, 1, None), (7, 4, 4, None), (100, 8, 2, None),
                                        (333, 16, 4, "zipf"), (256, 32, 8, "dead"),
                                        (0, 8, 2, None)])
def test_index_invariants(T, E, k, skew):
    pop = None
    if skew == "zipf":
        pop = np.arange(1, E + 1, dtype=np.float64) ** -1.2
    elif skew == "dead":
        pop = np.ones(E)
        pop[: E // 2] = 0.0
    ids = synth.random_ids(T, E, k, seed=T + E, popularity=pop)
    ix = oracle.build_index(ids, E)
    _check_index_invariants(ids, E, ix)
    if skew == "dead":
        assert np.all(ix.counts[: E // 2] == 0)


def test_index_matches_stable_sort():
    # Section 4.2 describes the sort-based construction the method replaces:
    # sorting the flattened (expert, token) pairs by expert with a stable sort
    # gives the same maps.
    T, E, k = 500, 16, 4
    ids = synth.random_ids(T, E, k, seed=3)
    ix = oracle.build_index(ids, E)
    order = np.argsort(ids.reshape(-1), kind="stable")
    assert np.array_equal(ix.slot_src, order)
    assert np.array_equal(ix.eti, order // k)
    assert np.array_equal(ix.counts, np.bincount(ids.reshape(-1), minlength=E))


# --------------------------------------------------------------------------
# Gating (Section 2.1)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("renorm", [False, True])
def test_route_against_library_softmax_and_sort(renorm):
    v = _tiny_layer(T=40, d=32, E=8, k=3)
    ids, gates, logits, probs = oracle.route(v["x"], v["w_gate"], None, 3, renorm)
    ref_logits = v["x"] @ v["w_gate"].T
    np.testing.assert_allclose(logits, ref_logits, rtol=1e-12, atol=1e-12)
    ref_p = scipy.special.softmax(ref_logits, axis=1)
    np.testing.assert_allclose(probs, ref_p, rtol=1e-12, atol=1e-15)
    ref_ids = np.argsort(-ref_logits.astype(np.float32), axis=1, kind="stable")[:, :3]
    assert np.array_equal(ids, ref_ids)
    ref_g = np.take_along_axis(ref_p, ref_ids, axis=1)
    if renorm:
        ref_g = ref_g / ref_g.sum(axis=1, keepdims=True)
        np.testing.assert_allclose(gates.sum(axis=1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(gates, ref_g, rtol=1e-12)


def test_route_ties_go_to_lower_id_and_bias_applies():
    T, d, E, k = 5, 8, 6, 3
    rng = np.random.default_rng(1)
    x = rng.standard_normal((T, d))
    wg = rng.standard_normal((E, d))
    wg[4] = wg[1]            # experts 1 and 4 always tie
    wg[5] = wg[1]            # and 5
    bias = np.zeros(E)
    bias[[1, 4, 5]] = 100.0  # ... and always win
    ids, gates, logits, _ = oracle.route(x, wg, bias, k, False)
    assert np.all(ids == np.array([1, 4, 5]))
    np.testing.assert_allclose(gates, np.full((T, 3), gates[:, :1]), rtol=1e-15)
    bias[0] = -np.inf        # an expert that can never be chosen
    ids, gates, logits, probs = oracle.route(x, wg, bias, k, False)
    assert np.all(probs[:, 0] == 0.0) and np.all(ids != 0)


# --------------------------------------------------------------------------
# Forward (Sections 2.2, 2.3, 3.1, 5.1)
# --------------------------------------------------------------------------

def _silu(u):
    return u / (1.0 + np.exp(-u))


def _dense_forward(v, ids, gates):
    """Brute force: every expert on every token, weighted by the dense [T,E]
    gate matrix that is zero outside each token's top-k."""
    x = v["x"]
    T = x.shape[0]
    E = v["w1"].shape[0]
    G = np.zeros((T, E))
    np.put_along_axis(G, ids, gates, axis=1)
    y = np.zeros_like(x)
    for e in range(E):
        ffn = (_silu(x @ v["w1"][e]) * (x @ v["w3"][e])) @ v["w2"][e]
        y += G[:, e:e + 1] * ffn
    return y


@pytest.mark.parametrize("renorm,zipf", [(False, 0.0), (True, 0.0), (False, 1.2)])
def test_forward_matches_dense_bruteforce(renorm, zipf):
    v = _tiny_layer(T=30, d=16, f=24, E=6, k=3, zipf=zipf)
    fw = oracle.layer_forward(v["x"], v["w_gate"], v["bias"], v["w1"], v["w3"], v["w2"], 3, renorm)
    y_ref = _dense_forward(v, fw["ids"], fw["gates"])
    np.testing.assert_allclose(fw["y"], y_ref, rtol=1e-11, atol=1e-12)


def test_single_expert_is_textbook_swiglu_ffn():
    # E = 1, k = 1: the only gate is softmax of one logit = 1, so the layer is
    # a plain SwiGLU FFN (Section 5.1 definition).
    v = _tiny_layer(T=9, d=16, f=20, E=1, k=1)
    fw = oracle.layer_forward(v["x"], v["w_gate"], None, v["w1"], v["w3"], v["w2"], 1, False)
    x = v["x"]
    ref = (_silu(x @ v["w1"][0]) * (x @ v["w3"][0])) @ v["w2"][0]
    np.testing.assert_allclose(fw["gates"], 1.0, rtol=1e-15)
    np.testing.assert_allclose(fw["y"], ref, rtol=1e-12, atol=1e-13)
    assert np.array_equal(fw["ix"].eti, np.arange(9))


@pytest.mark.parametrize("renorm", [False, True])
def test_identity_experts_combine(renorm):
    # With O[s] = x[eti[s]] (identity experts) the combine returns x * sum_j g.
    v = _tiny_layer(T=20, d=8, E=5, k=3)
    ids, gates, _, _ = oracle.route(v["x"], v["w_gate"], None, 3, renorm)
    ix = oracle.build_index(ids, 5)
    y = oracle.combine(v["x"][ix.eti], gates, ix.tim)
    np.testing.assert_allclose(y, v["x"] * gates.sum(axis=1, keepdims=True), rtol=1e-14)
    if renorm:
        np.testing.assert_allclose(y, v["x"], rtol=1e-14)
    # unit weights: each token's row comes back k times
    y1 = oracle.combine(v["x"][ix.eti], None, ix.tim)
    np.testing.assert_allclose(y1, 3.0 * v["x"], rtol=1e-15)


# --------------------------------------------------------------------------
# Backward (Section 3.2, Algorithm 1, router closed form)
# --------------------------------------------------------------------------

def _torch_dense_grads(v, ids, renorm, dy):
    """Independent backward: torch float64 autograd through a dense
    formulation (all experts on all tokens) with the routing decision fixed."""
    t = {n: torch.tensor(a, dtype=torch.float64, requires_grad=True)
         for n, a in v.items() if a is not None and n in ("x", "w_gate", "w1", "w3", "w2")}
    logits = t["x"] @ t["w_gate"].T
    if v.get("bias") is not None:
        logits = logits + torch.tensor(v["bias"], dtype=torch.float64)
    p = torch.softmax(logits, dim=1)
    idx = torch.tensor(ids, dtype=torch.int64)
    g = torch.gather(p, 1, idx)
    if renorm:
        g = g / g.sum(dim=1, keepdim=True)
    G = torch.zeros_like(p).scatter(1, idx, g)
    y = torch.zeros_like(t["x"])
    for e in range(v["w1"].shape[0]):
        a = t["x"] @ t["w1"][e]
        b = t["x"] @ t["w3"][e]
        y = y + G[:, e:e + 1] * ((torch.nn.functional.silu(a) * b) @ t["w2"][e])
    (y * torch.tensor(dy)).sum().backward()
    return {n: tt.grad.numpy() for n, tt in t.items()}


@pytest.mark.parametrize("renorm,zipf", [(False, 0.0), (True, 0.0), (False, 1.2)])
def test_backward_matches_torch_autograd_dense(renorm, zipf):
    v = _tiny_layer(T=14, d=12, f=16, E=5, k=2, zipf=zipf)
    dy = v["dy"]
    fw = oracle.layer_forward(v["x"], v["w_gate"], v["bias"], v["w1"], v["w3"], v["w2"], 2, renorm)
    bw = oracle.layer_backward(fw, dy, v["x"], v["w_gate"], v["w1"], v["w3"], v["w2"], renorm)
    ref = _torch_dense_grads(v, fw["ids"], renorm, dy)
    for mine, theirs in (("dx", "x"), ("dw_gate", "w_gate"), ("dw1", "w1"), ("dw3", "w3"),
                         ("dw2", "w2")):
        np.testing.assert_allclose(bw[mine], ref[theirs], rtol=1e-10, atol=1e-12, err_msg=mine)


def _loss(v, dy, k, renorm, ids):
    fw = oracle.layer_forward(v["x"], v["w_gate"], v["bias"], v["w1"], v["w3"], v["w2"], k,
                              renorm, ids=ids)
    return float((fw["y"] * dy).sum())


@pytest.mark.parametrize("renorm", [False, True])
def test_backward_central_finite_differences(renorm):
    k = 2
    v = _tiny_layer(T=10, d=8, f=12, E=4, k=k, seed=5)
    dy = v["dy"]
    fw = oracle.layer_forward(v["x"], v["w_gate"], None, v["w1"], v["w3"], v["w2"], k, renorm)
    bw = oracle.layer_backward(fw, dy, v["x"], v["w_gate"], v["w1"], v["w3"], v["w2"], renorm)
    ids = fw["ids"]
    rng = np.random.default_rng(0)
    h = 1e-6
    for name, gname in (("x", "dx"), ("w_gate", "dw_gate"), ("w1", "dw1"), ("w3", "dw3"),
                        ("w2", "dw2")):
        for _ in range(6):
            idx = tuple(rng.integers(0, s) for s in v[name].shape)
            vp = dict(v); vm = dict(v)
            vp[name] = v[name].copy(); vm[name] = v[name].copy()
            vp[name][idx] += h
            vm[name][idx] -= h
            fd = (_loss(vp, dy, k, renorm, ids) - _loss(vm, dy, k, renorm, ids)) / (2 * h)
            an = bw[gname][idx]
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, idx, fd, an)
    # gate gradient: y is linear in the gates, so d<dy, y>/dg[t,j] = <dy[t], O[tim[t,j]]>
    gp = fw["gates"].copy()
    t, j = 3, 1
    gp[t, j] += 1.0
    y2 = oracle.combine(fw["O"], gp, fw["ix"].tim)
    assert abs(float((y2 * dy).sum() - (fw["y"] * dy).sum()) - bw["d_gates"][t, j]) < 1e-9


def test_full_softmax_jacobian_when_all_experts_selected():
    # k = E with renorm: g = softmax(logits) permuted by ids, so the router
    # backward is the textbook softmax Jacobian (diag(p) - p p^T) applied to dg.
    T, d, E = 6, 8, 5
    rng = np.random.default_rng(2)
    x = rng.standard_normal((T, d))
    wg = rng.standard_normal((E, d))
    dg = rng.standard_normal((T, E))
    for renorm in (False, True):
        ids, gates, logits, probs = oracle.route(x, wg, None, E, renorm)
        dl, dwg, dxr = oracle.route_bwd(dg, logits, ids, x, wg, renorm)
        for t in range(T):
            p = probs[t]
            J = np.diag(p) - np.outer(p, p)
            dp = np.zeros(E)
            dp[ids[t]] = dg[t]
            np.testing.assert_allclose(dl[t], J @ dp, rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(dwg, dl.T @ x, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(dxr, dl @ wg, rtol=1e-12, atol=1e-14)


def test_swiglu_derivative_closed_form():
    # The derivative used for dA (Algorithm 1, backward): SiLU'(u) =
    # sigmoid(u) (1 + u (1 - sigmoid(u))), checked through a 1x1x1 layer where
    # dA = dh * B * SiLU'(A) with dh = g * dy * w2.
    x = np.array([[0.7]]); w1 = np.array([[[1.3]]]); w3 = np.array([[[-0.4]]])
    w2 = np.array([[[2.0]]]); dy = np.array([[0.5]])
    ix = oracle.build_index(np.zeros((1, 1), np.int32), 1)
    A, B, O = oracle.ffn_fwd(x, w1, w3, w2, ix, 1)
    bw = oracle.ffn_bwd(dy, x, w1, w3, w2, np.ones((1, 1)), ix, A, B)
    a = 0.7 * 1.3
    sg = 1.0 / (1.0 + math.exp(-a))
    assert A[0, 0] == pytest.approx(a, rel=1e-15)
    dh = 0.5 * 2.0
    assert bw["dA"][0, 0] == pytest.approx(dh * (-0.28) * sg * (1 + a * (1 - sg)), rel=1e-14)
    assert bw["dB"][0, 0] == pytest.approx(dh * a * sg, rel=1e-14)
    assert O[0, 0] == pytest.approx(a * sg * (-0.28) * 2.0, rel=1e-14)


# --------------------------------------------------------------------------
# Non-gated experts (Section 2.2: E(x) = W2 act(W1 x); ReLU and SiLU as in the
# experiments of Section 6)
# --------------------------------------------------------------------------

_TORCH_ACT = {"silu": torch.nn.functional.silu, "relu": torch.relu}


def _torch_dense_act(v, ids, renorm, act, dy=None):
    """Dense all-experts evaluation in float64 torch (routing fixed by ids);
    returns y, and the input/weight gradients when dy is given."""
    t = {n: torch.tensor(v[n], dtype=torch.float64, requires_grad=dy is not None)
         for n in ("x", "w_gate", "w1", "w2")}
    logits = t["x"] @ t["w_gate"].T
    if v.get("bias") is not None:
        logits = logits + torch.tensor(v["bias"], dtype=torch.float64)
    p = torch.softmax(logits, dim=1)
    idx = torch.tensor(ids, dtype=torch.int64)
    g = torch.gather(p, 1, idx)
    if renorm:
        g = g / g.sum(dim=1, keepdim=True)
    G = torch.zeros_like(p).scatter(1, idx, g)
    y = torch.zeros_like(t["x"])
    for e in range(v["w1"].shape[0]):
        y = y + G[:, e:e + 1] * (_TORCH_ACT[act](t["x"] @ t["w1"][e]) @ t["w2"][e])
    if dy is None:
        return y.detach().numpy(), None
    (y * torch.tensor(dy)).sum().backward()
    return y.detach().numpy(), {n: tt.grad.numpy() for n, tt in t.items()}


@pytest.mark.parametrize("act", ["silu", "relu"])
@pytest.mark.parametrize("renorm,zipf", [(False, 0.0), (True, 0.0), (False, 1.2)])
def test_nongated_forward_matches_dense_bruteforce(act, renorm, zipf):
    v = _tiny_layer(T=30, d=16, f=24, E=6, k=3, zipf=zipf)
    fw = oracle.layer_forward(v["x"], v["w_gate"], v["bias"], v["w1"], None, v["w2"], 3, renorm,
                              act=act)
    assert fw["B"] is None
    y_ref, _ = _torch_dense_act(v, fw["ids"], renorm, act)
    np.testing.assert_allclose(fw["y"], y_ref, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("act", ["silu", "relu"])
def test_single_expert_is_textbook_mlp(act):
    # E = 1, k = 1: a plain two-layer MLP W2 act(W1 x) (Section 2.2).
    v = _tiny_layer(T=9, d=16, f=20, E=1, k=1)
    fw = oracle.layer_forward(v["x"], v["w_gate"], None, v["w1"], None, v["w2"], 1, False, act=act)
    a = v["x"] @ v["w1"][0]
    h = np.maximum(a, 0.0) if act == "relu" else _silu(a)
    np.testing.assert_allclose(fw["A"], a, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(fw["y"], h @ v["w2"][0], rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("act", ["silu", "relu"])
@pytest.mark.parametrize("renorm,zipf", [(False, 0.0), (True, 0.0), (False, 1.2)])
def test_nongated_backward_matches_torch_autograd_dense(act, renorm, zipf):
    v = _tiny_layer(T=14, d=12, f=16, E=5, k=2, zipf=zipf)
    dy = v["dy"]
    fw = oracle.layer_forward(v["x"], v["w_gate"], v["bias"], v["w1"], None, v["w2"], 2, renorm,
                              act=act)
    assert np.abs(fw["A"]).min() > 1e-9   # no pre-activation at the ReLU kink
    bw = oracle.layer_backward(fw, dy, v["x"], v["w_gate"], v["w1"], None, v["w2"], renorm)
    _, ref = _torch_dense_act(v, fw["ids"], renorm, act, dy)
    for mine, theirs in (("dx", "x"), ("dw_gate", "w_gate"), ("dw1", "w1"), ("dw2", "w2")):
        np.testing.assert_allclose(bw[mine], ref[theirs], rtol=1e-10, atol=1e-12, err_msg=mine)
    assert "dw3" not in bw and "dB" not in bw


@pytest.mark.parametrize("act", ["silu", "relu"])
def test_nongated_backward_central_finite_differences(act):
    k = 2
    v = _tiny_layer(T=10, d=8, f=12, E=4, k=k, seed=5)
    dy = v["dy"]
    fw = oracle.layer_forward(v["x"], v["w_gate"], None, v["w1"], None, v["w2"], k, False, act=act)
    bw = oracle.layer_backward(fw, dy, v["x"], v["w_gate"], v["w1"], None, v["w2"], False)
    ids = fw["ids"]
    h = 1e-6
    assert np.abs(fw["A"]).min() > 1e3 * h   # steps never cross the ReLU kink

    def loss(vv):
        f2 = oracle.layer_forward(vv["x"], vv["w_gate"], None, vv["w1"], None, vv["w2"], k, False,
                                  ids=ids, act=act)
        return float((f2["y"] * dy).sum())

    rng = np.random.default_rng(1)
    for name, gname in (("x", "dx"), ("w_gate", "dw_gate"), ("w1", "dw1"), ("w2", "dw2")):
        for _ in range(6):
            idx = tuple(rng.integers(0, s) for s in v[name].shape)
            vp = dict(v); vm = dict(v)
            vp[name] = v[name].copy(); vm[name] = v[name].copy()
            vp[name][idx] += h
            vm[name][idx] -= h
            fd = (loss(vp) - loss(vm)) / (2 * h)
            an = bw[gname][idx]
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, idx, fd, an)


def test_relu_derivative_closed_form():
    # 1x1 expert: dA = dh * [a > 0] with dh = g dy w2; at a = 0 exactly the
    # derivative is taken as 0 (h = 0 there, so dW2 and d_gate vanish too).
    w2 = np.array([[[2.0]]]); dy = np.array([[0.5]])
    ix = oracle.build_index(np.zeros((1, 1), np.int32), 1)
    for xv, w1v, want in ((0.7, 1.3, 1.0), (0.7, -1.3, 0.0), (0.0, 1.3, 0.0)):
        x = np.array([[xv]]); w1 = np.array([[[w1v]]])
        A, O = oracle.ffn_fwd_act(x, w1, w2, ix, 1, "relu")
        bw = oracle.ffn_bwd_act(dy, x, w1, w2, np.ones((1, 1)), ix, A, "relu")
        a = xv * w1v
        assert A[0, 0] == a and O[0, 0] == max(a, 0.0) * 2.0
        assert bw["dA"][0, 0] == 0.5 * 2.0 * want
        assert bw["dw2"][0, 0, 0] == max(a, 0.0) * 0.5
        assert bw["dw1"][0, 0, 0] == xv * 0.5 * 2.0 * want
        assert bw["d_gates"][0, 0] == 0.5 * O[0, 0]
