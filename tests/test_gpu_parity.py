"""GPU parity: every C-ABI entry point against the CPU oracle on the same
seeded inputs, at sizes the oracle finishes in seconds (several tiles per
expert plus ragged tails), and the edge cases of the method."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2601_05296_amd import binding as B
from paper_2601_05296_amd import layer, synth
from tests.parity import TOL, assert_close, dev, host, near_tie_ok, rel_err

pytestmark = pytest.mark.gpu


def _ids_case(T, E, k, pattern, seed=0):
    pop = None
    if pattern == "zipf":
        pop = np.arange(1, E + 1, dtype=np.float64) ** -1.2
    elif pattern == "dead":
        pop = np.ones(E)
        pop[::2] = 0.0
    elif pattern == "one":
        pop = np.full(E, 1e-9)
        pop[: k] = 1.0
    return synth.random_ids(T, E, k, seed=seed, popularity=pop)


def _gpu_index(ids, E):
    T, k = ids.shape
    S = T * k
    i32 = dict(dtype=torch.int32, device="cuda")
    out = dict(counts=torch.empty(E, **i32), offsets=torch.empty(E + 1, **i32),
               eti=torch.empty(S, **i32), tim=torch.empty((T, k), **i32),
               slot_src=torch.empty(S, **i32))
    wsb = B.moe_build_index_workspace_size(T, E, k)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    B.moe_build_index(dev(ids), T, E, k, out["counts"], out["offsets"], out["eti"], out["tim"],
                      out["slot_src"], ws, wsb)
    torch.cuda.synchronize()
    return {n: t.cpu().numpy() for n, t in out.items()}


# ---------------------------------------------------------------------------
# moe_build_index: bit-exact
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T,E,k,pattern", [
    (5, 4, 2, "worked"), (1, 4, 1, None), (1000, 8, 2, None), (4097, 64, 6, None),
    (3000, 128, 8, "zipf"), (2000, 32, 4, "dead"), (777, 256, 16, None), (513, 16, 4, "one"),
    (300000, 64, 8, None), (65536, 128, 8, "zipf")])
def test_build_index_bit_exact(T, E, k, pattern):
    if pattern == "worked":
        ids = np.array([[2, 3], [0, 1], [0, 3], [1, 2], [0, 3]], np.int32)
    else:
        ids = _ids_case(T, E, k, pattern, seed=T)
    ref = oracle.build_index(ids, E)
    got = _gpu_index(ids, E)
    assert np.array_equal(got["counts"], ref.counts)
    assert np.array_equal(got["offsets"], ref.offsets)
    assert np.array_equal(got["eti"], ref.eti)
    assert np.array_equal(got["tim"], ref.tim)
    assert np.array_equal(got["slot_src"], ref.slot_src)


def test_build_index_deterministic():
    ids = _ids_case(50000, 64, 6, "zipf", seed=1)
    a = _gpu_index(ids, 64)
    b = _gpu_index(ids, 64)
    for n in a:
        assert np.array_equal(a[n], b[n])


# ---------------------------------------------------------------------------
# ids top-k never produces (outside [0, E), or repeated within a row): the
# index build rejects such a choice and every later call stays in bounds.
# Expected values come from the oracle with each rejected choice sent to an
# extra, last expert whose weights are zero: its slots come after all others
# and it adds exactly nothing.
# ---------------------------------------------------------------------------

def _corrupt_ids(T, E, k, seed, frac):
    ids = _ids_case(T, E, k, None, seed=seed)
    rng = np.random.default_rng(seed + 1)
    bad = [-1, E, 1 << 30, -(1 << 31)]
    for t in np.nonzero(rng.random(T) < frac)[0]:
        j = int(rng.integers(k))
        kind = int(rng.integers(5))
        ids[t, j] = ids[t, int(rng.integers(j))] if (kind == 4 and j > 0) else bad[kind % 4]
    return ids


def _rejected(ids, E):
    """Brute force: a choice is rejected when its id is outside [0, E) or
    equals an earlier id of its row."""
    T, k = ids.shape
    rej = np.zeros((T, k), bool)
    for t in range(T):
        for j in range(k):
            e = int(ids[t, j])
            rej[t, j] = not 0 <= e < E or e in ids[t, :j].tolist()
    return rej


def _sink_index(ids, rej, E):
    return oracle.build_index(np.where(rej, E, ids), E + 1)


@pytest.mark.parametrize("T,E,k,frac", [
    (300, 8, 2, 0.2), (1000, 64, 6, 0.3), (777, 256, 16, 0.5), (513, 16, 4, 1.0), (1, 4, 2, 1.0),
    (200, 8, 3, None)])
def test_build_index_rejects_invalid_ids(T, E, k, frac):
    if frac is None:   # every choice rejected
        ids = np.full((T, k), -1, np.int32)
    else:
        ids = _corrupt_ids(T, E, k, seed=T, frac=frac)
    rej = _rejected(ids, E)
    assert rej.any()
    ref = _sink_index(ids, rej, E)
    got = _gpu_index(ids, E)
    n = int(ref.offsets[E])
    assert n == T * k - int(rej.sum())
    assert np.array_equal(got["counts"], ref.counts[:E])
    assert np.array_equal(got["offsets"], ref.offsets[:E + 1])
    assert np.array_equal(got["eti"][:n], ref.eti[:n])
    assert np.array_equal(got["slot_src"][:n], ref.slot_src[:n])
    assert np.array_equal(got["tim"], np.where(rej, -1, ref.tim))


@pytest.mark.parametrize("dtype,act,h_on_load,combined", [
    ("bf16", "swiglu", False, True), ("bf16", "swiglu", True, True), ("bf16", "swiglu", False, False),
    ("bf16", "relu", False, True), ("f32", "swiglu", False, False),
    ("bf16", "swiglu", True, "atomic"), ("bf16", "silu", False, "atomic")])
def test_ffn_with_rejected_choices(dtype, act, h_on_load, combined):
    T, d, f, E, k = 300, 256, 384, 8, 3
    inp, _, g = _layer_case(dtype, T, d, f, E, k, False, None)
    ids = _corrupt_ids(T, E, k, seed=3, frac=0.3)
    ids[:5] = -1                      # tokens with no valid choice at all
    rej = _rejected(ids, E)
    v, st = inp.vals, inp.store
    gated = act == "swiglu"
    S = T * k
    # oracle with the rejected choices on a zero-weight last expert
    ix = _sink_index(ids, rej, E)

    def z(w):
        return np.concatenate([w, np.zeros((1,) + w.shape[1:])])

    if gated:
        A_r, B_r, O_r = oracle.ffn_fwd(v["x"], z(v["w1"]), z(v["w3"]), z(v["w2"]), ix, k)
        bw = oracle.ffn_bwd(v["dy"], v["x"], z(v["w1"]), z(v["w3"]), z(v["w2"]), g, ix, A_r, B_r)
    else:
        A_r, O_r = oracle.ffn_fwd_act(v["x"], z(v["w1"]), z(v["w2"]), ix, k, act)
        bw = oracle.ffn_bwd_act(v["dy"], v["x"], z(v["w1"]), z(v["w2"]), g, ix, A_r, act)
    y_r = oracle.combine(O_r, g, ix.tim)
    dx_r = oracle.combine(bw["dX_slot"], None, ix.tim)
    # device, on the ids as they are
    gi = _gpu_index(ids, E)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x, w1, w2, dy = (dev(st[n]) for n in ("x", "w1", "w2", "dy"))
    w3 = dev(st["w3"]) if gated else None
    offsets, eti, tim, ss = (dev(gi[n]) for n in ("offsets", "eti", "tim", "slot_src"))
    gates = dev(g)
    flags = B.dtype_flag(x) | B.ACT_FLAG[act] | (B.MOE_H_ON_LOAD if h_on_load else 0)
    nan = float("nan")
    A = torch.full((S, f), nan, dtype=tdt, device="cuda")
    Bm = torch.full((S, f), nan, dtype=tdt, device="cuda") if gated else None
    y = torch.empty((T, d), dtype=tdt, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    dw1 = torch.full((E, d, f), nan, **f32)
    dw3 = torch.full((E, d, f), nan, **f32) if gated else None
    dw2 = torch.full((E, f, d), nan, **f32)
    dg = torch.full((T, k), nan, **f32)
    dx = torch.empty((T, d), dtype=tdt, device="cuda")
    if combined:
        if combined == "atomic":   # y and dx start as NaN: the call clears them
            flags |= B.MOE_ATOMIC_COMBINE
            y.fill_(nan)
            dx.fill_(nan)
        wsb = B.moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, flags)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        B.moe_ffn_fwd_combine(x, w1, w3, w2, offsets, eti, gates, tim, T, d, f, E, k, flags,
                              A, Bm, y, ws, wsb)
        wsb = B.moe_ffn_bwd_combine_workspace_size(T, d, f, E, k, flags)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        B.moe_ffn_bwd_combine(dy, x, w1, w3, w2, gates, offsets, eti, ss, tim, A, Bm, T, d, f,
                              E, k, flags, dw1, dw3, dw2, dg, dx, ws, wsb)
    else:
        # rows of O and dX_slot past offsets[E] are never written: NaN there
        # would reach y or dx if the combine read them
        O = torch.full((S, d), nan, dtype=tdt, device="cuda")
        wsb = B.moe_ffn_fwd_workspace_size(T, d, f, E, k, flags)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        B.moe_ffn_fwd(x, w1, w3, w2, offsets, eti, T, d, f, E, k, flags, A, Bm, O, ws, wsb)
        B.moe_combine(O, gates, tim, T, d, k, B.dtype_flag(x), y)
        dX = torch.full((S, d), nan, dtype=tdt, device="cuda")
        wsb = B.moe_ffn_bwd_workspace_size(T, d, f, E, k, flags)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        B.moe_ffn_bwd(dy, x, w1, w3, w2, gates, offsets, eti, ss, A, Bm, T, d, f, E, k, flags,
                      dw1, dw3, dw2, dg, dX, ws, wsb)
        B.moe_combine(dX, None, tim, T, d, k, B.dtype_flag(x), dx)
    torch.cuda.synchronize()
    assert_close("y", host(y), y_r, dtype)
    assert np.all(host(y)[:5] == 0)
    assert_close("dx", host(dx), dx_r, dtype)
    assert_close("dw1", host(dw1), bw["dw1"][:E], dtype)
    assert_close("dw2", host(dw2), bw["dw2"][:E], dtype)
    if gated:
        assert_close("dw3", host(dw3), bw["dw3"][:E], dtype)
    got_dg = host(dg)
    assert_close("d_gates", got_dg[~rej], bw["d_gates"][~rej], dtype)
    assert np.all(np.isnan(got_dg[rej]))     # not written


@pytest.mark.parametrize("renorm", [False, True])
def test_route_bwd_ignores_invalid_ids(renorm):
    T, d, E, k = 500, 256, 64, 6
    cfg = synth.MoEConfig("rb", T=T, d=d, f=128, E=E, k=k, dtype="bf16", renorm=renorm)
    inp = synth.make_inputs(cfg)
    v = inp.vals
    ids, gates, logits, _ = oracle.route(v["x"], v["w_gate"], None, k, renorm)
    rng = np.random.default_rng(9)
    bad_rows = rng.random(T) < 0.3
    bad_ids = ids.copy()
    for t in np.nonzero(bad_rows)[0]:
        bad_ids[t, int(rng.integers(k))] = [-1, E, 1 << 30, -(1 << 31)][int(rng.integers(4))]
    dgates = rng.standard_normal((T, k))
    clean = ~bad_rows
    _, _, dx_r = oracle.route_bwd(dgates[clean], logits[clean], ids[clean], v["x"][clean],
                                  v["w_gate"], renorm)
    x, wg = dev(inp.store["x"]), dev(inp.store["w_gate"])
    flags = B.dtype_flag(x) | (B.MOE_RENORM if renorm else 0)
    dwg = torch.empty((E, d), dtype=torch.float32, device="cuda")
    dx = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    wsb = B.moe_route_bwd_workspace_size(T, d, E, k, flags)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    B.moe_route_bwd(dev(dgates.astype(np.float32)), dev(logits.astype(np.float32)), dev(bad_ids),
                    dev(gates.astype(np.float32)), x, wg, T, d, E, k, flags, dwg, dx, ws, wsb)
    torch.cuda.synchronize()
    assert np.all(np.isfinite(host(dwg))) and np.all(np.isfinite(host(dx)))
    assert_close("dx (clean tokens)", host(dx)[clean], dx_r, "bf16")


# ---------------------------------------------------------------------------
# moe_route
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,T,d,E,k,renorm,bias", [
    ("bf16", 1000, 256, 8, 2, False, None), ("bf16", 1000, 512, 64, 6, True, None),
    ("bf16", 777, 256, 128, 8, False, "zipf"), ("bf16", 300, 384, 200, 16, False, "dead"),
    ("f32", 1000, 256, 8, 2, False, None), ("f32", 500, 256, 64, 6, True, "dead"),
    ("bf16", 700, 320, 64, 6, True, None),
    ("bf16", 100, 64, 1, 1, False, None), ("bf16", 100, 64, 3, 3, True, None),
    ("bf16", 500, 128, 256, 16, False, None), ("bf16", 400, 192, 256, 16, True, "zipf"),
    # 128-token workgroups (E > 64, T >= 65536), ragged last workgroup
    ("bf16", 70000, 256, 128, 8, False, "zipf"), ("bf16", 65601, 128, 256, 16, True, None)])
def test_route_parity(dtype, T, d, E, k, renorm, bias):
    cfg = synth.MoEConfig("r", T=T, d=d, f=128, E=E, k=k, dtype=dtype, renorm=renorm,
                          zipf_s=1.2 if bias == "zipf" else 0.0,
                          n_dead=E // 4 if bias == "dead" else 0)
    inp = synth.make_inputs(cfg, with_dy=False)
    v = inp.vals
    ids_r, gates_r, logits_r, _ = oracle.route(v["x"], v["w_gate"], v["bias"], k, renorm)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x, wg = dev(inp.store["x"]), dev(inp.store["w_gate"])
    bias_t = dev(v["bias"]) if v["bias"] is not None else None
    ids = torch.empty((T, k), dtype=torch.int32, device="cuda")
    gates = torch.empty((T, k), dtype=torch.float32, device="cuda")
    logits = torch.empty((T, E), dtype=torch.float32, device="cuda")
    flags = B.dtype_flag(x) | (B.MOE_RENORM if renorm else 0)
    B.moe_route(x, wg, bias_t, T, d, E, k, flags, ids, gates, logits)
    torch.cuda.synchronize()
    assert x.dtype == tdt
    ids_g = ids.cpu().numpy()
    lg = host(logits)
    fin = np.isfinite(logits_r)
    assert np.array_equal(np.isfinite(lg), fin)
    assert_close("logits", lg[fin], logits_r[fin], "f32")
    nflip = near_tie_ok(ids_g, ids_r, logits_r)
    assert nflip <= max(1, T // 200)
    same = np.all(ids_g == ids_r, axis=1)
    assert_close("gates", host(gates)[same], gates_r[same], "f32" if dtype == "f32" else "bf16")
    # ids are distinct per row and in range
    assert np.all(np.sort(ids_g, axis=1)[:, 1:] != np.sort(ids_g, axis=1)[:, :-1])
    assert ids_g.min() >= 0 and ids_g.max() < E


# ---------------------------------------------------------------------------
# moe_combine
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,T,d,k,weighted,accumulate", [
    ("bf16", 1000, 256, 2, True, False), ("bf16", 333, 2048, 6, True, True),
    ("bf16", 257, 512, 8, False, False), ("f32", 1000, 256, 2, True, False),
    ("f32", 100, 128, 16, False, True),
    # per-token array bounds 4 / 8 / 16 (the kernel is sized by the smallest
    # bound >= k): both sides of each edge, and bf16 rows wider than 256 chunks
    ("bf16", 129, 256, 4, True, False), ("bf16", 200, 4096, 5, False, True),
    ("bf16", 300, 1024, 12, True, True), ("f32", 150, 512, 3, True, False)])
def test_combine_parity(dtype, T, d, k, weighted, accumulate):
    rng = np.random.default_rng(T + d + k)
    E = max(k, 8)
    ids = _ids_case(T, E, k, None, seed=3)
    ix = oracle.build_index(ids, E)
    src = rng.standard_normal((T * k, d)).astype(np.float32)
    base = rng.standard_normal((T, d)).astype(np.float32)
    w = rng.random((T, k)).astype(np.float32) if weighted else None
    if dtype == "bf16":
        src_s, base_s = synth.bf16_round(src), synth.bf16_round(base)
        src, base = synth.bf16_to_f32(src_s), synth.bf16_to_f32(base_s)
    else:
        src_s, base_s = src, base
    out = dev(base_s)
    flags = (B.MOE_F32 if dtype == "f32" else 0) | (B.MOE_ACCUMULATE if accumulate else 0)
    B.moe_combine(dev(src_s), dev(w), dev(ix.tim), T, d, k, flags, out)
    torch.cuda.synchronize()
    ref = oracle.combine(src, w, ix.tim) + (base if accumulate else 0.0)
    assert_close("combine", host(out), ref, dtype)


# ---------------------------------------------------------------------------
# moe_ffn_fwd / moe_ffn_bwd / moe_route_bwd on one layer
# ---------------------------------------------------------------------------

FFN_CASES = [
    # dtype, T, d, f, E, k, renorm, ids pattern
    ("bf16", 300, 256, 384, 8, 2, False, None),
    ("bf16", 700, 256, 256, 16, 4, True, "zipf"),
    ("bf16", 500, 384, 128, 12, 3, False, "dead"),
    ("f32", 300, 256, 384, 8, 2, False, None),
    ("f32", 257, 128, 256, 16, 4, True, "dead"),
    # d and f odd multiples of 64: partial column tiles in every GEMM
    ("bf16", 300, 320, 192, 8, 2, False, None),
    ("f32", 200, 192, 320, 8, 3, False, None),
    # the smallest shapes the ABI accepts: d = f = 64 (one or two K slices),
    # a single expert, top-1
    ("bf16", 100, 64, 64, 1, 1, False, None),
    ("bf16", 37, 64, 192, 3, 2, True, None),
    ("f32", 50, 64, 64, 2, 2, False, None),
    # the largest E and k: 256 experts of about 19 slots each, many empty
    ("bf16", 300, 128, 128, 256, 16, True, None),
]


def _layer_case(dtype, T, d, f, E, k, renorm, pattern, seed=0):
    cfg = synth.MoEConfig("l", T=T, d=d, f=f, E=E, k=k, dtype=dtype, renorm=renorm, seed=seed)
    inp = synth.make_inputs(cfg)
    ids = _ids_case(T, E, k, pattern, seed=seed + 11)
    rng = np.random.default_rng(seed + 5)
    g = rng.random((T, k)).astype(np.float32)
    return inp, ids, g


@pytest.mark.parametrize("dtype,T,d,f,E,k,renorm,pattern", FFN_CASES)
def test_ffn_fwd_bwd_parity(dtype, T, d, f, E, k, renorm, pattern):
    inp, ids, g = _layer_case(dtype, T, d, f, E, k, renorm, pattern)
    v, st = inp.vals, inp.store
    S = T * k
    # oracle
    ix = oracle.build_index(ids, E)
    A_r, B_r, O_r = oracle.ffn_fwd(v["x"], v["w1"], v["w3"], v["w2"], ix, k)
    y_r = oracle.combine(O_r, g, ix.tim)
    bw = oracle.ffn_bwd(v["dy"], v["x"], v["w1"], v["w3"], v["w2"], g, ix, A_r, B_r)
    dx_r = oracle.combine(bw["dX_slot"], None, ix.tim)
    # device
    gi = _gpu_index(ids, E)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x, w1, w3, w2, dy = (dev(st[n]) for n in ("x", "w1", "w3", "w2", "dy"))
    offsets, eti, tim, ss = (dev(gi[n]) for n in ("offsets", "eti", "tim", "slot_src"))
    gates = dev(g)
    flags = B.dtype_flag(x)
    A = torch.empty((S, f), dtype=tdt, device="cuda")
    Bm = torch.empty((S, f), dtype=tdt, device="cuda")
    O = torch.empty((S, d), dtype=tdt, device="cuda")
    wsf = B.moe_ffn_fwd_workspace_size(T, d, f, E, k, flags)
    wsf_t = torch.empty(max(wsf, 16), dtype=torch.uint8, device="cuda")
    B.moe_ffn_fwd(x, w1, w3, w2, offsets, eti, T, d, f, E, k, flags, A, Bm, O, wsf_t, wsf)
    y = torch.empty((T, d), dtype=tdt, device="cuda")
    B.moe_combine(O, gates, tim, T, d, k, flags, y)
    torch.cuda.synchronize()
    assert_close("A", host(A), A_r, dtype)
    assert_close("B", host(Bm), B_r, dtype)
    assert_close("O", host(O), O_r, dtype)
    assert_close("y", host(y), y_r, dtype)
    f32 = dict(dtype=torch.float32, device="cuda")
    dw1 = torch.full((E, d, f), float("nan"), **f32)
    dw3 = torch.full((E, d, f), float("nan"), **f32)
    dw2 = torch.full((E, f, d), float("nan"), **f32)
    dg = torch.full((T, k), float("nan"), **f32)
    dX = torch.empty((S, d), dtype=tdt, device="cuda")
    wsb = B.moe_ffn_bwd_workspace_size(T, d, f, E, k, flags)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    B.moe_ffn_bwd(dy, x, w1, w3, w2, gates, offsets, eti, ss, A, Bm, T, d, f, E, k, flags,
                  dw1, dw3, dw2, dg, dX, ws, wsb)
    dx = torch.empty((T, d), dtype=tdt, device="cuda")
    B.moe_combine(dX, None, tim, T, d, k, flags, dx)
    torch.cuda.synchronize()
    assert_close("dA", host(A), bw["dA"], dtype)
    assert_close("dB", host(Bm), bw["dB"], dtype)
    assert_close("dw2", host(dw2), bw["dw2"], dtype)
    assert_close("dw1", host(dw1), bw["dw1"], dtype)
    assert_close("dw3", host(dw3), bw["dw3"], dtype)
    assert_close("d_gates", host(dg), bw["d_gates"], dtype)
    assert_close("dX_slot", host(dX), bw["dX_slot"], dtype)
    assert_close("dx_ffn", host(dx), dx_r, dtype)
    if pattern == "dead":  # experts without tokens get exact zero gradients
        empty = np.nonzero(gi["counts"] == 0)[0]
        assert empty.size > 0
        assert np.all(host(dw1)[empty] == 0) and np.all(host(dw2)[empty] == 0)


@pytest.mark.parametrize("dtype,T,d,E,k,renorm,accumulate", [
    ("bf16", 1000, 256, 8, 2, False, False), ("bf16", 2500, 512, 64, 6, True, True),
    ("bf16", 1500, 256, 128, 8, False, True), ("bf16", 777, 384, 200, 16, True, False),
    ("f32", 1000, 256, 8, 2, False, False),
    ("f32", 700, 128, 32, 4, True, True),
    ("bf16", 900, 192, 64, 6, False, True), ("bf16", 600, 320, 256, 8, True, False),
    ("bf16", 100, 64, 1, 1, True, False), ("bf16", 300, 64, 4, 3, False, True),
    ("bf16", 500, 128, 256, 16, False, True), ("bf16", 400, 192, 256, 16, True, False),
    # more tokens than 128 splits of 512 (bf16) / 1024 (f32): longer, capped splits
    ("bf16", 150001, 128, 16, 2, False, True), ("f32", 140001, 64, 8, 2, True, False)])
def test_route_bwd_parity(dtype, T, d, E, k, renorm, accumulate):
    cfg = synth.MoEConfig("rb", T=T, d=d, f=128, E=E, k=k, dtype=dtype, renorm=renorm)
    inp = synth.make_inputs(cfg)
    v = inp.vals
    ids, gates, logits, _ = oracle.route(v["x"], v["w_gate"], None, k, renorm)
    rng = np.random.default_rng(7)
    dgates = rng.standard_normal((T, k))
    dl, dwg_r, dxr_r = oracle.route_bwd(dgates, logits, ids, v["x"], v["w_gate"], renorm)
    base = synth.bf16_to_f32(synth.bf16_round(v["dy"])) if dtype == "bf16" else v["dy"]
    base_store = synth.bf16_round(v["dy"]) if dtype == "bf16" else v["dy"]
    x, wg = dev(inp.store["x"]), dev(inp.store["w_gate"])
    flags = B.dtype_flag(x) | (B.MOE_RENORM if renorm else 0) | (B.MOE_ACCUMULATE if accumulate else 0)
    dwg = torch.empty((E, d), dtype=torch.float32, device="cuda")
    dx = dev(base_store)
    wsb = B.moe_route_bwd_workspace_size(T, d, E, k, flags)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    B.moe_route_bwd(dev(dgates.astype(np.float32)), dev(logits.astype(np.float32)), dev(ids),
                    dev(gates.astype(np.float32)), x, wg, T, d, E, k, flags, dwg, dx, ws, wsb)
    torch.cuda.synchronize()
    assert_close("dw_gate", host(dwg), dwg_r, "f32" if dtype == "f32" else "bf16")
    ref_dx = dxr_r + (base if accumulate else 0.0)
    got = host(dx)
    if accumulate:  # compare the router part, which is small next to the base
        got = got - base
        ref_dx = dxr_r
    tol = "f32" if dtype == "f32" else "bf16"
    e = rel_err(got, ref_dx)
    lim = TOL[tol] if not (accumulate and dtype == "bf16") else 2e-2 * np.abs(base).max() / np.abs(dxr_r).max()
    assert e <= max(lim, TOL[tol]), e


# ---------------------------------------------------------------------------
NONGATED_CASES = [
    # dtype, T, d, f, E, k, renorm, ids pattern, activation
    ("bf16", 300, 256, 384, 8, 2, False, None, "silu"),
    ("bf16", 700, 256, 256, 16, 4, True, "zipf", "relu"),
    ("bf16", 500, 384, 128, 12, 3, False, "dead", "silu"),
    ("f32", 300, 256, 384, 8, 2, False, None, "relu"),
    ("f32", 257, 128, 256, 16, 4, True, "dead", "silu"),
    ("bf16", 400, 192, 320, 8, 2, False, "zipf", "relu"),
]


@pytest.mark.parametrize("dtype,T,d,f,E,k,renorm,pattern,act", NONGATED_CASES)
def test_ffn_nongated_parity(dtype, T, d, f, E, k, renorm, pattern, act):
    """Non-gated SiLU / ReLU experts (MOE_ACT_SILU / MOE_ACT_RELU): w3, B and
    dw3 are passed as NULL."""
    inp, ids, g = _layer_case(dtype, T, d, f, E, k, renorm, pattern)
    v, st = inp.vals, inp.store
    S = T * k
    ix = oracle.build_index(ids, E)
    A_r, O_r = oracle.ffn_fwd_act(v["x"], v["w1"], v["w2"], ix, k, act)
    y_r = oracle.combine(O_r, g, ix.tim)
    bw = oracle.ffn_bwd_act(v["dy"], v["x"], v["w1"], v["w2"], g, ix, A_r, act)
    dx_r = oracle.combine(bw["dX_slot"], None, ix.tim)
    gi = _gpu_index(ids, E)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x, w1, w2, dy = (dev(st[n]) for n in ("x", "w1", "w2", "dy"))
    offsets, eti, tim, ss = (dev(gi[n]) for n in ("offsets", "eti", "tim", "slot_src"))
    gates = dev(g)
    flags = B.dtype_flag(x) | B.ACT_FLAG[act]
    A = torch.empty((S, f), dtype=tdt, device="cuda")
    O = torch.empty((S, d), dtype=tdt, device="cuda")
    wsf = B.moe_ffn_fwd_workspace_size(T, d, f, E, k, flags)
    wsf_t = torch.empty(max(wsf, 16), dtype=torch.uint8, device="cuda")
    B.moe_ffn_fwd(x, w1, None, w2, offsets, eti, T, d, f, E, k, flags, A, None, O, wsf_t, wsf)
    y = torch.empty((T, d), dtype=tdt, device="cuda")
    B.moe_combine(O, gates, tim, T, d, k, B.dtype_flag(x), y)
    torch.cuda.synchronize()
    assert_close("A", host(A), A_r, dtype)
    assert_close("O", host(O), O_r, dtype)
    assert_close("y", host(y), y_r, dtype)
    f32 = dict(dtype=torch.float32, device="cuda")
    dw1 = torch.full((E, d, f), float("nan"), **f32)
    dw2 = torch.full((E, f, d), float("nan"), **f32)
    dg = torch.full((T, k), float("nan"), **f32)
    dX = torch.empty((S, d), dtype=tdt, device="cuda")
    wsb = B.moe_ffn_bwd_workspace_size(T, d, f, E, k, flags)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    B.moe_ffn_bwd(dy, x, w1, None, w2, gates, offsets, eti, ss, A, None, T, d, f, E, k, flags,
                  dw1, None, dw2, dg, dX, ws, wsb)
    dx = torch.empty((T, d), dtype=tdt, device="cuda")
    B.moe_combine(dX, None, tim, T, d, k, B.dtype_flag(x), dx)
    torch.cuda.synchronize()
    dA = host(A)
    if act == "relu":
        # the derivative is a decision on the sign of A; where A is within the
        # device's accumulation error of 0 either decision is valid
        tie = np.abs(A_r) < 1e-4 * np.abs(A_r).max()
        assert tie.mean() < 1e-3
        assert_close("dA", np.where(tie, 0, dA), np.where(tie, 0, bw["dA"]), dtype)
    else:
        assert_close("dA", dA, bw["dA"], dtype)
    assert_close("dw2", host(dw2), bw["dw2"], dtype)
    assert_close("dw1", host(dw1), bw["dw1"], dtype)
    assert_close("d_gates", host(dg), bw["d_gates"], dtype)
    assert_close("dX_slot", host(dX), bw["dX_slot"], dtype)
    assert_close("dx_ffn", host(dx), dx_r, dtype)
    if pattern == "dead":
        empty = np.nonzero(gi["counts"] == 0)[0]
        assert empty.size > 0
        assert np.all(host(dw1)[empty] == 0) and np.all(host(dw2)[empty] == 0)


@pytest.mark.parametrize("act", ["silu", "relu"])
def test_layer_nongated_end_to_end(act):
    """Whole layer through layer.forward / layer.backward with a non-gated
    expert, routing included, on a small bf16 problem."""
    cfg = synth.MoEConfig("ng", T=600, d=256, f=512, E=8, k=2, dtype="bf16", renorm=False)
    inp = synth.make_inputs(cfg)
    v, st = inp.vals, inp.store
    fw_r = oracle.layer_forward(v["x"], v["w_gate"], None, v["w1"], None, v["w2"], cfg.k, False,
                                act=act)
    bw_r = oracle.layer_backward(fw_r, v["dy"], v["x"], v["w_gate"], v["w1"], None, v["w2"], False)
    x, wg, w1, w2, dy = (dev(st[n]) for n in ("x", "w_gate", "w1", "w2", "dy"))
    y, saved = layer.forward(x, wg, None, w1, None, w2, cfg.k, False, act=act)
    assert saved.B is None
    assert saved.nbytes() == pytest.approx(
        layer.saved_bytes_per_token(cfg.d, cfg.f, cfg.E, cfg.k, 2, cfg.T, act) * cfg.T)
    ids_g = saved.ids.cpu().numpy()
    assert np.array_equal(ids_g, fw_r["ids"])
    g = layer.backward(saved, dy, x, wg, w1, None, w2)
    torch.cuda.synchronize()
    assert g["dw3"] is None
    assert_close("y", host(y), fw_r["y"], "bf16")
    for n in ("dw1", "dw2", "dw_gate", "dx", "d_gates"):
        assert_close(n, host(g[n]), bw_r[n], "bf16")


COMBINED_CASES = [
    # dtype, T, d, f, E, k, ids pattern, activation
    ("bf16", 400, 1280, 256, 8, 2, None, "swiglu"),
    ("bf16", 333, 384, 256, 12, 3, "dead", "silu"),
    ("bf16", 500, 640, 384, 16, 4, "zipf", "relu"),
    ("f32", 257, 256, 256, 8, 2, None, "swiglu"),
    ("bf16", 500, 576, 448, 16, 4, None, "swiglu"),
    ("bf16", 100, 64, 64, 2, 2, None, "swiglu"),
    # 393k slots: three strips of 256 columns (bit-exactness only; the
    # full-size tests check multi-strip workloads against the oracle)
    ("bf16", 49152, 768, 256, 16, 8, None, "swiglu"),
]


@pytest.mark.parametrize("dtype,T,d,f,E,k,pattern,act", COMBINED_CASES)
def test_ffn_combined_equals_separate(dtype, T, d, f, E, k, pattern, act):
    """moe_ffn_fwd_combine / moe_ffn_bwd_combine against moe_ffn_fwd / moe_ffn_bwd
    followed by moe_combine: the same kernels in the same order, so the results
    are bit-identical; and against the oracle."""
    inp, ids, g = _layer_case(dtype, T, d, f, E, k, False, pattern)
    v, st = inp.vals, inp.store
    gated = act == "swiglu"
    S = T * k
    gi = _gpu_index(ids, E)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x, w1, w2, dy = (dev(st[n]) for n in ("x", "w1", "w2", "dy"))
    w3 = dev(st["w3"]) if gated else None
    offsets, eti, tim, ss = (dev(gi[n]) for n in ("offsets", "eti", "tim", "slot_src"))
    gates = dev(g)
    flags = B.dtype_flag(x) | B.ACT_FLAG[act]
    f32 = dict(dtype=torch.float32, device="cuda")

    def fwd(combined):
        A = torch.empty((S, f), dtype=tdt, device="cuda")
        Bm = torch.empty((S, f), dtype=tdt, device="cuda") if gated else None
        y = torch.empty((T, d), dtype=tdt, device="cuda")
        if combined:
            wsb = B.moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, flags)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
            B.moe_ffn_fwd_combine(x, w1, w3, w2, offsets, eti, gates, tim, T, d, f, E, k, flags,
                                  A, Bm, y, ws, wsb)
        else:
            O = torch.empty((S, d), dtype=tdt, device="cuda")
            wsb = B.moe_ffn_fwd_workspace_size(T, d, f, E, k, flags)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
            B.moe_ffn_fwd(x, w1, w3, w2, offsets, eti, T, d, f, E, k, flags, A, Bm, O, ws, wsb)
            B.moe_combine(O, gates, tim, T, d, k, B.dtype_flag(x), y)
        return A, Bm, y

    def bwd(A, Bm, combined, dx0=None):
        dw1 = torch.empty((E, d, f), **f32)
        dw3 = torch.empty((E, d, f), **f32) if gated else None
        dw2 = torch.empty((E, f, d), **f32)
        dg = torch.empty((T, k), **f32)
        dx = torch.empty((T, d), dtype=tdt, device="cuda") if dx0 is None else dx0.clone()
        if combined:
            fl = flags | (B.MOE_ACCUMULATE if dx0 is not None else 0)
            wsb = B.moe_ffn_bwd_combine_workspace_size(T, d, f, E, k, flags)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
            B.moe_ffn_bwd_combine(dy, x, w1, w3, w2, gates, offsets, eti, ss, tim, A, Bm, T, d, f,
                                  E, k, fl, dw1, dw3, dw2, dg, dx, ws, wsb)
        else:
            dX = torch.empty((S, d), dtype=tdt, device="cuda")
            wsb = B.moe_ffn_bwd_workspace_size(T, d, f, E, k, flags)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
            B.moe_ffn_bwd(dy, x, w1, w3, w2, gates, offsets, eti, ss, A, Bm, T, d, f, E, k, flags,
                          dw1, dw3, dw2, dg, dX, ws, wsb)
            B.moe_combine(dX, None, tim, T, d, k,
                          B.dtype_flag(x) | (B.MOE_ACCUMULATE if dx0 is not None else 0), dx)
        return dict(dw1=dw1, dw3=dw3, dw2=dw2, d_gates=dg, dx=dx)

    res = {}
    for combined in (False, True):
        A, Bm, y = fwd(combined)
        A0 = A.clone()
        Bm0 = Bm.clone() if gated else None
        r = bwd(A, Bm, combined)
        r2 = bwd(A0, Bm0, combined, dx0=y)   # MOE_ACCUMULATE: dx = y + token gradient
        torch.cuda.synchronize()
        res[combined] = (A0, y, r, r2)
    (A_s, y_s, r_s, r2_s), (A_c, y_c, r_c, r2_c) = res[False], res[True]
    assert torch.equal(A_s, A_c) and torch.equal(y_s, y_c)
    for n in ("dw1", "dw2", "d_gates", "dx") + (("dw3",) if gated else ()):
        assert torch.equal(r_s[n], r_c[n]), n
    assert torch.equal(r2_s["dx"], r2_c["dx"])
    if S > 20000:
        return
    # and the oracle
    ix = oracle.build_index(ids, E)
    if gated:
        A_r, B_r, O_r = oracle.ffn_fwd(v["x"], v["w1"], v["w3"], v["w2"], ix, k)
        bw = oracle.ffn_bwd(v["dy"], v["x"], v["w1"], v["w3"], v["w2"], g, ix, A_r, B_r)
    else:
        A_r, O_r = oracle.ffn_fwd_act(v["x"], v["w1"], v["w2"], ix, k, act)
        bw = oracle.ffn_bwd_act(v["dy"], v["x"], v["w1"], v["w2"], g, ix, A_r, act)
    assert_close("y", host(y_c), oracle.combine(O_r, g, ix.tim), dtype)
    assert_close("dx", host(r_c["dx"]), oracle.combine(bw["dX_slot"], None, ix.tim), dtype)
    assert_close("dw1", host(r_c["dw1"]), bw["dw1"], dtype)


ATOMIC_CASES = [
    # T, d, f, E, k, ids pattern, activation, h on load
    (400, 1280, 256, 8, 2, None, "swiglu", True),
    (333, 384, 256, 12, 3, "dead", "silu", True),
    (500, 640, 384, 16, 4, "zipf", "relu", False),
    (500, 576, 448, 16, 4, None, "swiglu", False),
    (100, 64, 64, 2, 2, None, "swiglu", True),
    (1000, 512, 320, 64, 8, None, "swiglu", True),
    (3000, 256, 128, 32, 6, "zipf", "swiglu", True),
    # a single expert with top-1; 256 experts with top-16 (16 adds into each row)
    (100, 64, 64, 1, 1, None, "swiglu", True),
    (300, 128, 128, 256, 16, None, "swiglu", False),
]


@pytest.mark.parametrize("T,d,f,E,k,pattern,act,hol", ATOMIC_CASES)
def test_ffn_atomic_combine(T, d, f, E, k, pattern, act, hol):
    """MOE_ATOMIC_COMBINE: the second GEMM and the dX GEMM add their slot rows
    into y and dx by atomics. A, B and every weight and gate gradient are those
    of the strip path bit for bit (the same kernels); y and dx match the
    oracle (each term rounded to bf16 before it is added, each add rounded
    again), with and without MOE_ACCUMULATE; with k <= 2 the atomic result is
    deterministic, which a second run checks."""
    inp, ids, g = _layer_case("bf16", T, d, f, E, k, False, pattern)
    v, st = inp.vals, inp.store
    gated = act == "swiglu"
    S = T * k
    gi = _gpu_index(ids, E)
    x, w1, w2, dy = (dev(st[n]) for n in ("x", "w1", "w2", "dy"))
    w3 = dev(st["w3"]) if gated else None
    offsets, eti, tim, ss = (dev(gi[n]) for n in ("offsets", "eti", "tim", "slot_src"))
    gates = dev(g)
    base = B.dtype_flag(x) | B.ACT_FLAG[act] | (B.MOE_H_ON_LOAD if hol else 0)
    f32 = dict(dtype=torch.float32, device="cuda")
    bf = dict(dtype=torch.bfloat16, device="cuda")

    def run(atomic, dx0=None):
        flags = base | (B.MOE_ATOMIC_COMBINE if atomic else 0)
        A = torch.empty((S, f), **bf)
        Bm = torch.empty((S, f), **bf) if gated else None
        y = torch.full((T, d), float("nan"), **bf)
        wsb = B.moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, flags)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        B.moe_ffn_fwd_combine(x, w1, w3, w2, offsets, eti, gates, tim, T, d, f, E, k, flags,
                              A, Bm, y, ws, wsb)
        A0 = A.clone()
        Bm0 = Bm.clone() if gated else None
        out = dict(A=A0, B=Bm0, y=y)
        dw1 = torch.empty((E, d, f), **f32)
        dw3 = torch.empty((E, d, f), **f32) if gated else None
        dw2 = torch.empty((E, f, d), **f32)
        dg = torch.empty((T, k), **f32)
        dx = torch.full((T, d), float("nan"), **bf) if dx0 is None else dx0.clone()
        fl = flags | (B.MOE_ACCUMULATE if dx0 is not None else 0)
        wsb = B.moe_ffn_bwd_combine_workspace_size(T, d, f, E, k, flags)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        B.moe_ffn_bwd_combine(dy, x, w1, w3, w2, gates, offsets, eti, ss, tim, A, Bm, T, d, f, E,
                              k, fl, dw1, dw3, dw2, dg, dx, ws, wsb)
        torch.cuda.synchronize()
        out.update(dw1=dw1, dw3=dw3, dw2=dw2, d_gates=dg, dx=dx)
        return out

    ref = run(False)
    at = run(True)
    dx1 = dev(synth.bf16_round(np.random.default_rng(9).standard_normal((T, d),
                                                                        dtype=np.float32)))
    at_acc = run(True, dx0=dx1)
    for n in ("A", "dw1", "dw2", "d_gates") + (("B", "dw3") if gated else ()):
        assert torch.equal(at[n], ref[n]), n
    if k <= 2:
        again = run(True)
        assert torch.equal(again["y"], at["y"]) and torch.equal(again["dx"], at["dx"])
    ix = oracle.build_index(ids, E)
    if gated:
        A_r, B_r, O_r = oracle.ffn_fwd(v["x"], v["w1"], v["w3"], v["w2"], ix, k)
        bw = oracle.ffn_bwd(v["dy"], v["x"], v["w1"], v["w3"], v["w2"], g, ix, A_r, B_r)
    else:
        A_r, O_r = oracle.ffn_fwd_act(v["x"], v["w1"], v["w2"], ix, k, act)
        bw = oracle.ffn_bwd_act(v["dy"], v["x"], v["w1"], v["w2"], g, ix, A_r, act)
    dx_r = oracle.combine(bw["dX_slot"], None, ix.tim)
    assert_close("y", host(at["y"]), oracle.combine(O_r, g, ix.tim), "bf16")
    assert_close("dx", host(at["dx"]), dx_r, "bf16")
    assert_close("dx accumulated", host(at_acc["dx"]), host(dx1) + dx_r, "bf16")


@pytest.mark.parametrize("dtype,T,d,f,E,k,pattern,act", [c for c in COMBINED_CASES if c[0] == "bf16"])
def test_ffn_h_on_load_bit_identical(dtype, T, d, f, E, k, pattern, act):
    """MOE_H_ON_LOAD: the second GEMM forms h from A (and B) as it loads them,
    with G1's arithmetic, and the dW2 GEMM forms g*h from A, B and the gates
    before G4 overwrites them, with G4's arithmetic; so A, B, O, y and every
    gradient are bit-identical to the buffered path, and the workspaces drop
    the S x f bf16 h and g*h buffers."""
    inp, ids, g = _layer_case(dtype, T, d, f, E, k, False, pattern)
    st = inp.store
    gated = act == "swiglu"
    S = T * k
    gi = _gpu_index(ids, E)
    x, w1, w2 = (dev(st[n]) for n in ("x", "w1", "w2"))
    w3 = dev(st["w3"]) if gated else None
    offsets, eti, tim = (dev(gi[n]) for n in ("offsets", "eti", "tim"))
    gates = dev(g)
    base = B.dtype_flag(x) | B.ACT_FLAG[act]

    def fwd(flags, combined):
        A = torch.empty((S, f), dtype=torch.bfloat16, device="cuda")
        Bm = torch.empty((S, f), dtype=torch.bfloat16, device="cuda") if gated else None
        if combined:
            out = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
            wsb = B.moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, flags)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
            B.moe_ffn_fwd_combine(x, w1, w3, w2, offsets, eti, gates, tim, T, d, f, E, k, flags,
                                  A, Bm, out, ws, wsb)
        else:
            out = torch.empty((S, d), dtype=torch.bfloat16, device="cuda")
            wsb = B.moe_ffn_fwd_workspace_size(T, d, f, E, k, flags)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
            B.moe_ffn_fwd(x, w1, w3, w2, offsets, eti, T, d, f, E, k, flags, A, Bm, out, ws, wsb)
        torch.cuda.synchronize()
        return A, Bm, out, wsb

    dy, ss = dev(st["dy"]), dev(gi["slot_src"])
    f32 = dict(dtype=torch.float32, device="cuda")

    def bwd(flags, combined, A, Bm, dx0):
        dw1 = torch.empty((E, d, f), **f32)
        dw3 = torch.empty((E, d, f), **f32) if gated else None
        dw2 = torch.empty((E, f, d), **f32)
        dg = torch.empty((T, k), **f32)
        if combined:
            dx = dx0.clone()
            wsb = B.moe_ffn_bwd_combine_workspace_size(T, d, f, E, k, flags)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
            B.moe_ffn_bwd_combine(dy, x, w1, w3, w2, gates, offsets, eti, ss, tim, A, Bm, T, d, f,
                                  E, k, flags | B.MOE_ACCUMULATE, dw1, dw3, dw2, dg, dx, ws, wsb)
        else:
            dx = torch.empty((S, d), dtype=torch.bfloat16, device="cuda")
            wsb = B.moe_ffn_bwd_workspace_size(T, d, f, E, k, flags)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
            B.moe_ffn_bwd(dy, x, w1, w3, w2, gates, offsets, eti, ss, A, Bm, T, d, f, E, k, flags,
                          dw1, dw3, dw2, dg, dx, ws, wsb)
        torch.cuda.synchronize()
        return dict(dw1=dw1, dw3=dw3, dw2=dw2, d_gates=dg, dx=dx, dA=A, dB=Bm), wsb

    for combined in (False, True):
        A0, B0, out0, ws0 = fwd(base, combined)
        A1, B1, out1, ws1 = fwd(base | B.MOE_H_ON_LOAD, combined)
        assert torch.equal(A0, A1)
        if gated:
            assert torch.equal(B0, B1)
        assert torch.equal(out0, out1), "combined" if combined else "O"
        if combined:
            # the h buffer is gone; the strip of the h-on-load GEMM is rounded
            # to its 512-column tiles (at most one 256-column tile wider)
            assert ws0 - ws1 >= (S * f * 2 + 255) // 256 * 256 - S * 256 * 2 - 256
        else:
            assert ws0 - ws1 == (S * f * 2 + 255) // 256 * 256
        dx0 = out0 if combined else None          # combined: accumulate onto y
        r0, wb0 = bwd(base, combined, A0, B0, dx0)
        r1, wb1 = bwd(base | B.MOE_H_ON_LOAD, combined, A1, B1, dx0)
        for n in ("dw1", "dw2", "d_gates", "dx", "dA") + (("dw3", "dB") if gated else ()):
            assert torch.equal(r0[n], r1[n]), (n, combined)
        assert wb1 <= wb0 if combined else wb0 - wb1 >= S * f * 2 - S * 4 - 256


# whole layer (routing included) on the tiny float32 workload
# ---------------------------------------------------------------------------

def test_layer_end_to_end_tiny_f32():
    cfg = synth.CONFIGS["tiny_f32"]
    inp = synth.make_inputs(cfg)
    v, st = inp.vals, inp.store
    fw_r = oracle.layer_forward(v["x"], v["w_gate"], None, v["w1"], v["w3"], v["w2"], cfg.k, cfg.renorm)
    bw_r = oracle.layer_backward(fw_r, v["dy"], v["x"], v["w_gate"], v["w1"], v["w3"], v["w2"], cfg.renorm)
    x, wg, w1, w3, w2, dy = (dev(st[n]) for n in ("x", "w_gate", "w1", "w3", "w2", "dy"))
    y, saved = layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm)
    ids_g = saved.ids.cpu().numpy()
    assert near_tie_ok(ids_g, fw_r["ids"], fw_r["logits"]) == 0
    assert saved.nbytes() == pytest.approx(
        layer.saved_bytes_per_token(cfg.d, cfg.f, cfg.E, cfg.k, 4, cfg.T) * cfg.T)
    g = layer.backward(saved, dy, x, wg, w1, w3, w2)
    torch.cuda.synchronize()
    assert_close("y", host(y), fw_r["y"], "f32")
    for n in ("dw1", "dw3", "dw2", "dw_gate", "dx", "d_gates"):
        assert_close(n, host(g[n]), bw_r[n], "f32")


@pytest.mark.parametrize("act", ["swiglu", "silu"])
def test_layer_recompute_policy_bit_identical(act):
    """Full-recompute policy (moe_ffn_recompute in the backward) against the
    default policy that saves A and B: identical outputs and gradients, and
    only the routing decision and maps saved."""
    cfg = synth.MoEConfig("rc", T=1500, d=256, f=384, E=16, k=4, dtype="bf16", renorm=True,
                          act=act)
    inp = synth.make_inputs(cfg)
    st = inp.store
    x, wg, w1, w2, dy = (dev(st[n]) for n in ("x", "w_gate", "w1", "w2", "dy"))
    w3 = dev(st["w3"]) if act == "swiglu" else None
    outs = []
    # (recompute, h_on_load): default, full recompute, no h / g*h buffers, both
    for rc, hol in ((False, False), (True, False), (False, True), (True, True)):
        y, saved = layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm, act=act, recompute=rc,
                                 h_on_load=hol)
        assert (saved.A is None) == rc
        assert saved.nbytes() == pytest.approx(layer.saved_bytes_per_token(
            cfg.d, cfg.f, cfg.E, cfg.k, 2, cfg.T, act, recompute=rc) * cfg.T)
        g = layer.backward(saved, dy, x, wg, w1, w3, w2)
        torch.cuda.synchronize()
        outs.append([y] + [g[n] for n in ("dx", "dw1", "dw2", "dw_gate", "d_gates")])
    for other in outs[1:]:
        for a, b in zip(outs[0], other):
            assert torch.equal(a, b)


@pytest.mark.parametrize("act,hol", [("swiglu", True), ("swiglu", False), ("relu", True)])
def test_layer_recompute_chunked_vs_oracle(act, hol):
    """Full recompute over several token chunks (the last one ragged): every
    output and gradient against the oracle; y, dx, d_gates and dw_gate
    bit-identical to the policy that saves A and B (they are per-token
    results), and the weight gradients equal to float32 summation order (each
    chunk's are added into the layer's)."""
    cfg = synth.MoEConfig("rcc", T=1500, d=256, f=384, E=16, k=4, dtype="bf16", renorm=True,
                          act=act)
    inp = synth.make_inputs(cfg)
    v, st = inp.vals, inp.store
    x, wg, w1, w2, dy = (dev(st[n]) for n in ("x", "w_gate", "w1", "w2", "dy"))
    gated = act == "swiglu"
    w3 = dev(st["w3"]) if gated else None
    y0, s0 = layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm, act=act, h_on_load=hol)
    g0 = layer.backward(s0, dy, x, wg, w1, w3, w2)
    y1, s1 = layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm, act=act, h_on_load=hol,
                           recompute=True, chunk_tokens=400)
    assert s1.chunk == 400 and s1.A is None and s1.eti is None
    assert s1.nbytes() == layer.saved_bytes_per_token(cfg.d, cfg.f, cfg.E, cfg.k, 2, cfg.T, act,
                                                      recompute=True) * cfg.T
    g1 = layer.backward(s1, dy, x, wg, w1, w3, w2)
    torch.cuda.synchronize()
    assert torch.equal(y0, y1)
    for n in ("dx", "d_gates", "dw_gate"):
        assert torch.equal(g0[n], g1[n]), n
    for n in ("dw1", "dw2") + (("dw3",) if gated else ()):
        err = float((g0[n] - g1[n]).abs().max() / g0[n].abs().max())
        assert err <= 1e-5, (n, err)
    fw = oracle.layer_forward(v["x"], v["w_gate"], None, v["w1"], v["w3"], v["w2"], cfg.k,
                              cfg.renorm, act=act)
    assert np.array_equal(fw["ids"], s1.ids.cpu().numpy())
    bw = oracle.layer_backward(fw, v["dy"], v["x"], v["w_gate"], v["w1"], v["w3"], v["w2"],
                               cfg.renorm)
    assert_close("y", host(y1), fw["y"], "bf16")
    for n in ("dx", "d_gates", "dw_gate", "dw1", "dw2") + (("dw3",) if gated else ()):
        assert_close(n, host(g1[n]), bw[n], "bf16")


@pytest.mark.parametrize("recompute", [False, True])
def test_layer_atomic_combine_vs_oracle(recompute):
    """The layer with the combine folded into the GEMM epilogues
    (atomic_combine), saving A and B or fully recomputing them: y and every
    gradient against the oracle; the routing and the weight and gate gradients
    equal to the strip path's (per-token dx and y differ by bf16 rounding)."""
    cfg = synth.MoEConfig("atc", T=1500, d=256, f=384, E=16, k=4, dtype="bf16", renorm=True)
    inp = synth.make_inputs(cfg)
    v, st = inp.vals, inp.store
    x, wg, w1, w3, w2, dy = (dev(st[n]) for n in ("x", "w_gate", "w1", "w3", "w2", "dy"))
    kw = dict(recompute=True, chunk_tokens=400) if recompute else {}
    y0, s0 = layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm, **kw)
    g0 = layer.backward(s0, dy, x, wg, w1, w3, w2)
    y1, s1 = layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm, atomic_combine=True, **kw)
    assert s1.atomic_combine
    g1 = layer.backward(s1, dy, x, wg, w1, w3, w2)
    torch.cuda.synchronize()
    assert torch.equal(s0.ids, s1.ids)
    for n in ("d_gates", "dw1", "dw3", "dw2"):
        assert torch.equal(g0[n], g1[n]), n
    fw = oracle.layer_forward(v["x"], v["w_gate"], None, v["w1"], v["w3"], v["w2"], cfg.k,
                              cfg.renorm)
    assert np.array_equal(fw["ids"], s1.ids.cpu().numpy())
    bw = oracle.layer_backward(fw, v["dy"], v["x"], v["w_gate"], v["w1"], v["w3"], v["w2"],
                               cfg.renorm)
    assert_close("y", host(y1), fw["y"], "bf16")
    for n in ("dx", "d_gates", "dw_gate", "dw1", "dw3", "dw2"):
        assert_close(n, host(g1[n]), bw[n], "bf16")
    with pytest.raises(ValueError):
        layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm, atomic_combine=True,
                      separate=True)


def _random_layer_cases(n=16, seed=2601, tmax=700, wmax=8, emax=32, kmax=8, i0=0, modes=False):
    """Seeded random shapes over the whole option space: T, d, f (multiples
    of 64 up to 64 wmax), E, k, activation, h policy, combine mode, renorm."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(i0, i0 + n):
        E = int(rng.integers(1, emax + 1))
        k = int(rng.integers(1, min(E, kmax) + 1))
        cases.append(dict(i=i, T=int(rng.integers(1, tmax)), d=64 * int(rng.integers(1, wmax + 1)),
                          f=64 * int(rng.integers(1, wmax + 1)), E=E, k=k,
                          act=("swiglu", "silu", "relu")[int(rng.integers(3))],
                          hol=bool(rng.integers(2)), atomic=bool(rng.integers(2)),
                          renorm=bool(rng.integers(2))))
        if modes:   # also the calling mode, the chunking and the element type
            mode = ("combined", "separate", "recompute")[int(rng.integers(3))]
            dtype = "f32" if rng.random() < 0.25 else "bf16"
            cases[-1].update(mode=mode, dtype=dtype,
                             chunk=int(rng.integers(1, cases[-1]["T"] + 1)),
                             zipf=float(rng.choice([0.0, 1.2])),
                             dead=int(rng.integers(0, (E - k) // 2 + 1)))
            if mode == "separate" or dtype == "f32":
                cases[-1]["atomic"] = False
    return cases


@pytest.mark.parametrize("c", _random_layer_cases() +
                         _random_layer_cases(n=16, seed=2602, tmax=2500, wmax=16, emax=256,
                                             kmax=16, i0=16) +
                         _random_layer_cases(n=16, seed=2603, tmax=1500, wmax=8, emax=64,
                                             kmax=8, i0=32, modes=True),
                         ids=lambda c: "r%d" % c["i"])
def test_layer_random_shapes_vs_oracle(c):
    """The layer on seeded random small shapes against the oracle: y and every
    gradient within the bf16 tolerance, the routing equal up to near-ties
    (the oracle is then run on the device's choices)."""
    dtype, mode = c.get("dtype", "bf16"), c.get("mode", "combined")
    cfg = synth.MoEConfig("rnd%d" % c["i"], T=c["T"], d=c["d"], f=c["f"], E=c["E"], k=c["k"],
                          dtype=dtype, renorm=c["renorm"], act=c["act"], seed=300 + c["i"],
                          zipf_s=c.get("zipf", 0.0), n_dead=c.get("dead", 0))
    inp = synth.make_inputs(cfg)
    v, st = inp.vals, inp.store
    bias = dev(st["bias"]) if st["bias"] is not None else None
    gated = c["act"] == "swiglu"
    x, wg, w1, w2, dy = (dev(st[n]) for n in ("x", "w_gate", "w1", "w2", "dy"))
    w3 = dev(st["w3"]) if gated else None
    extra = dict(separate=True) if mode == "separate" else \
        dict(recompute=True, chunk_tokens=c["chunk"]) if mode == "recompute" else {}
    y, s = layer.forward(x, wg, bias, w1, w3, w2, cfg.k, cfg.renorm, act=cfg.act,
                         h_on_load=c["hol"], atomic_combine=c["atomic"], **extra)
    g = layer.backward(s, dy, x, wg, w1, w3, w2, separate=mode == "separate")
    torch.cuda.synchronize()
    ids_g = s.ids.cpu().numpy()
    ids_r, _, logits_r, _ = oracle.route(v["x"], v["w_gate"], v["bias"], cfg.k, cfg.renorm)
    near_tie_ok(ids_g, ids_r, logits_r)
    fw = oracle.layer_forward(v["x"], v["w_gate"], v["bias"], v["w1"], v["w3"], v["w2"], cfg.k,
                              cfg.renorm, ids=ids_g, act=cfg.act)
    bw = oracle.layer_backward(fw, v["dy"], v["x"], v["w_gate"], v["w1"], v["w3"], v["w2"],
                               cfg.renorm)
    assert_close("y", host(y), fw["y"], dtype)
    keep_dx = np.ones(cfg.T, dtype=bool)
    keep_dw1 = np.ones(bw["dw1"].shape, dtype=bool)
    if cfg.act == "relu":
        # ReLU'(A) is decided on the device's bf16 A: where the oracle's A is
        # within 1e-4 max|A| of zero either decision is valid (as in the other
        # ReLU tests), and a flipped one moves a whole term of the token's dx
        # and of its expert's dW1 column; those are left out, found from the
        # oracle's A alone
        A_r, ix = fw["A"], fw["ix"]
        tie = np.abs(A_r) < 1e-4 * np.abs(A_r).max()
        assert tie.mean() < 1e-3
        tok_of_slot = ix.eti[: A_r.shape[0]]
        keep_dx[np.unique(tok_of_slot[tie.any(axis=1)])] = False
        for e in range(cfg.E):
            lo, hi = ix.offsets[e], ix.offsets[e + 1]
            keep_dw1[e][:, tie[lo:hi].any(axis=0)] = False
    assert_close("dx", host(g["dx"])[keep_dx], bw["dx"][keep_dx], dtype)
    assert_close("dw1", np.where(keep_dw1, host(g["dw1"]), 0), np.where(keep_dw1, bw["dw1"], 0),
                 dtype)
    for n in ("d_gates", "dw_gate", "dw2") + (("dw3",) if gated else ()):
        assert_close(n, host(g[n]), bw[n], dtype)


def test_layer_deterministic_bf16():
    cfg = synth.MoEConfig("det", T=2000, d=256, f=256, E=16, k=4, dtype="bf16", renorm=True)
    inp = synth.make_inputs(cfg)
    st = inp.store
    x, wg, w1, w3, w2, dy = (dev(st[n]) for n in ("x", "w_gate", "w1", "w3", "w2", "dy"))
    outs = []
    for _ in range(2):
        y, saved = layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm)
        g = layer.backward(saved, dy, x, wg, w1, w3, w2)
        torch.cuda.synchronize()
        outs.append([y.cpu()] + [g[n].cpu() for n in ("dx", "dw1", "dw3", "dw2", "dw_gate")])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_layer_on_a_side_stream():
    """The layer driven on a second stream (default priority) while the
    current stream is busy with other work: the same bits as on the current
    stream."""
    cfg = synth.MoEConfig("st", T=1500, d=256, f=384, E=16, k=4, dtype="bf16", renorm=True)
    inp = synth.make_inputs(cfg)
    st = inp.store
    x, wg, w1, w3, w2, dy = (dev(st[n]) for n in ("x", "w_gate", "w1", "w3", "w2", "dy"))
    y0, s0 = layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm)
    g0 = layer.backward(s0, dy, x, wg, w1, w3, w2)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    busy = torch.randn(2048, 2048, device="cuda")
    for _ in range(4):
        busy = busy @ busy.T / 2048.0     # unrelated work on the current stream
    y1, s1 = layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm, stream=side)
    g1 = layer.backward(s1, dy, x, wg, w1, w3, w2, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert torch.equal(y0, y1)
    for n in ("dx", "dw1", "dw3", "dw2", "dw_gate", "d_gates"):
        assert torch.equal(g0[n], g1[n]), n
    with pytest.raises(TypeError):
        layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm, stream=side.cuda_stream)


@pytest.mark.parametrize("k", [2, 4])
def test_layer_graph_replay(k):
    """The whole layer step, forward and backward through every entry point,
    captured in a HIP graph (the library allocates nothing, clears memory with
    kernels rather than memsets, and never synchronises): every replay, with
    eager steps between the replays, gives the eager step's bits. k = 2 runs
    the combine folded into the GEMM epilogues, k = 4 the strips."""
    cfg = synth.MoEConfig("gr", T=1500, d=256, f=384, E=16, k=k, dtype="bf16", renorm=True)
    inp = synth.make_inputs(cfg)
    st = inp.store
    x, wg, w1, w3, w2, dy = (dev(st[n]) for n in ("x", "w_gate", "w1", "w3", "w2", "dy"))
    names = ("dx", "dw1", "dw3", "dw2", "dw_gate", "d_gates")

    def step():
        y, s = layer.forward(x, wg, None, w1, w3, w2, cfg.k, cfg.renorm)
        return y, s, layer.backward(s, dy, x, wg, w1, w3, w2)

    y0, s0, g0 = step()
    torch.cuda.synchronize()
    assert s0.atomic_combine == (k <= 2)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):        # warm-up on a side stream before the capture
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        y1, _, g1 = step()
    for r in range(3):
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y1, y0), r
        for n in names:
            assert torch.equal(g1[n], g0[n]), (r, n)
        y2, _, g2 = step()               # eager work between the replays
        torch.cuda.synchronize()
        assert torch.equal(y2, y0) and torch.equal(g2["dx"], g0["dx"]), r
    del graph


def test_error_codes_launch_nothing():
    """The library's own validation, reached with raw device addresses (the
    binding checks tensor sizes and dtypes, not raw addresses)."""
    xt = torch.zeros((4, 128), dtype=torch.bfloat16, device="cuda")
    x = xt.data_ptr()
    with pytest.raises(B.MoEError) as ei:
        B.moe_route(x, x, None, 4, 128, 2, 3, 0, x, x, None)
    assert ei.value.status == B.MOE_ERR_INVALID_ARG
    with pytest.raises(B.MoEError) as ei:
        B.moe_build_index(x, 4, 8, 2, x, x, x, x, x, x, 0)
    assert ei.value.status == B.MOE_ERR_WORKSPACE
    # activation flags: both at once, or on a call other than the FFN
    with pytest.raises(B.MoEError) as ei:
        B.moe_ffn_fwd(x, x, None, x, x, x, 4, 128, 128, 2, 1,
                      B.MOE_ACT_SILU | B.MOE_ACT_RELU, x, None, x, x, 1 << 20)
    assert ei.value.status == B.MOE_ERR_INVALID_ARG
    with pytest.raises(B.MoEError) as ei:
        B.moe_combine(x, None, x, 4, 128, 2, B.MOE_ACT_SILU, x)
    assert ei.value.status == B.MOE_ERR_INVALID_ARG
    # SwiGLU needs w3 and B
    with pytest.raises(B.MoEError) as ei:
        B.moe_ffn_fwd(x, x, None, x, x, x, 4, 128, 128, 2, 1, 0, x, None, x, x, 1 << 20)
    assert ei.value.status == B.MOE_ERR_INVALID_ARG
    # T == 0 is a no-op
    B.moe_combine(x, None, x, 0, 128, 2, 0, x)
