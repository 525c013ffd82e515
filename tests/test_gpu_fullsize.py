"""GPU parity at the full sizes of the benchmarked workloads, in the launch
configuration bench.py times (layer.forward / layer.backward).

The oracle cannot run a whole layer of these sizes, so the checks are:
  * routing for every token (oracle route is cheap): ids equal up to
    near-ties, logits and gates within tolerance;
  * the index build, fed the oracle's ids, bit-exact for every token;
  * y, dx, d_gates, A, B, dA, dB at sampled tokens (half of them those with
    the highest slots), from an oracle run on just those tokens (each of these
    depends on its own token only);
  * dw1, dw3, dw2 at sampled hidden columns (some in the last f-tile) of the
    most- and the least-loaded expert, from an oracle run on a sub-problem
    holding that expert's tokens and those columns of its weights (SwiGLU
    columns are independent);
  * the router backward at full size on the oracle's logits and seeded gate
    gradients, against the oracle's router backward for every token.
No oracle input is taken from the device.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2601_05296_amd import binding as B
from paper_2601_05296_amd import layer, synth
from tests.parity import assert_close, dev, host, near_tie_ok

pytestmark = pytest.mark.gpu

# "_atomic": the combine folded into the GEMM epilogues where the layer would
# otherwise use the ordered strips (k > 2)
CASES = ["mid_e64k6", "few_large_e8k2", "many_small_zipf", "mem_sweep_e64k8", "zipf_empty",
         "table1_conf4", "table1_conf1_relu", "d2880_e128k4", "mid_e64k6_atomic",
         "many_small_zipf_atomic"]
NTOK = 24      # sampled tokens (half of them holding the highest slots)
NCOL = 8       # sampled hidden columns


def _cfg(name):
    if name.endswith("_atomic"):   # the same workload and inputs
        return _cfg(name[:-len("_atomic")])
    if name == "zipf_empty":
        return synth.CONFIGS["many_small_zipf"].with_(name="zipf_empty", n_dead=16)
    if name == "table1_conf1_relu":
        return synth.CONFIGS["table1_conf1"].with_(name=name, act="relu")
    return synth.CONFIGS[name]


def _f64(a):
    return None if a is None else a.astype(np.float64)


@pytest.mark.parametrize("name", CASES)
def test_full_size_layer(name):
    cfg = _cfg(name)
    T, d, f, E, k = cfg.T, cfg.d, cfg.f, cfg.E, cfg.k
    gated = cfg.act == "swiglu"
    print("full-size case %s: T=%d d=%d f=%d E=%d k=%d act=%s" % (name, T, d, f, E, k, cfg.act),
          flush=True)
    inp = synth.make_inputs(cfg)
    v = {n: _f64(a) for n, a in inp.vals.items()}
    st = inp.store
    x, wg, w1, w3, w2, dy = (dev(st[n]) if st[n] is not None else None
                             for n in ("x", "w_gate", "w1", "w3", "w2", "dy"))
    bias = dev(st["bias"]) if st["bias"] is not None else None

    # ---- device: the benchmarked forward + backward --------------------------
    atomic = True if name.endswith("_atomic") else None
    y, saved = layer.forward(x, wg, bias, w1, w3, w2, k, cfg.renorm, act=cfg.act,
                             atomic_combine=atomic)
    assert saved.atomic_combine == (k <= 2 or atomic is True)
    A_fwd = saved.A.clone()
    B_fwd = saved.B.clone() if gated else None
    g = layer.backward(saved, dy, x, wg, w1, w3, w2)
    torch.cuda.synchronize()
    ids_g = saved.ids.cpu().numpy()

    # ---- routing, every token --------------------------------------------------
    ids_r, gates_r, logits_r, _ = oracle.route(v["x"], v["w_gate"], v["bias"], k, cfg.renorm)
    nflip = near_tie_ok(ids_g, ids_r, logits_r)
    assert nflip <= max(2, T // 5000), nflip
    same_tok = np.all(ids_g == ids_r, axis=1)
    fin = np.isfinite(logits_r)
    assert_close("logits", host(saved.logits)[fin], logits_r[fin], "f32", case=name)
    assert_close("gates", host(saved.gates)[same_tok], gates_r[same_tok], "bf16", case=name)
    if cfg.n_dead:
        dead = np.nonzero(~np.isfinite(v["bias"]))[0]
        assert np.all(saved.counts.cpu().numpy()[dead] == 0)

    # ---- index build on the oracle's ids, bit-exact ------------------------------
    ix_r = oracle.build_index(ids_r, E)
    S = T * k
    i32 = dict(dtype=torch.int32, device="cuda")
    o = [torch.empty(E, **i32), torch.empty(E + 1, **i32), torch.empty(S, **i32),
         torch.empty((T, k), **i32), torch.empty(S, **i32)]
    wsb = B.moe_build_index_workspace_size(T, E, k)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    B.moe_build_index(dev(ids_r), T, E, k, *o, ws, wsb)
    torch.cuda.synchronize()
    for got, ref in zip(o, (ix_r.counts, ix_r.offsets, ix_r.eti, ix_r.tim, ix_r.slot_src)):
        assert np.array_equal(got.cpu().numpy(), ref)

    # ---- sampled tokens: forward and backward rows -------------------------------
    rng = np.random.default_rng(1234)
    cand = np.nonzero(same_tok)[0]
    tim_all = saved.tim.cpu().numpy()
    # random tokens, and the tokens holding the highest slots (the tail of the
    # last experts' segments, where slot-row offsets are largest)
    top = cand[np.argsort(-tim_all[cand].max(axis=1), kind="stable")[:NTOK // 2]]
    rest = np.setdiff1d(cand, top)
    toks = np.sort(np.concatenate([top, rng.choice(rest, size=min(NTOK - top.size, rest.size),
                                                   replace=False)]))
    sub = lambda a: None if a is None else a[toks]
    fw = oracle.layer_forward(v["x"][toks], v["w_gate"], v["bias"], v["w1"], v["w3"], v["w2"], k,
                              cfg.renorm, act=cfg.act)
    assert np.array_equal(fw["ids"], ids_g[toks])
    bw = oracle.layer_backward(fw, v["dy"][toks], v["x"][toks], v["w_gate"], v["w1"], v["w3"],
                               v["w2"], cfg.renorm)
    assert_close("y", host(y)[toks], fw["y"], "bf16", case=name)
    assert_close("dx", host(g["dx"])[toks], bw["dx"], "bf16", case=name)
    assert_close("d_gates", host(g["d_gates"])[toks], bw["d_gates"], "bf16", case=name)
    tim_g = saved.tim.cpu().numpy()
    slots_g = tim_g[toks].reshape(-1)                 # device slots, (t, j) order
    slots_r = fw["ix"].tim.reshape(-1)                # oracle sub-run slots, same order
    sl = torch.from_numpy(slots_g).long().cuda()
    A_r = fw["A"][slots_r]
    assert_close("A", host(A_fwd[sl]), A_r, "bf16", case=name)
    dA_g, dA_r = host(saved.A[sl]), bw["dA"][slots_r]
    if cfg.act == "relu":   # sign decisions within the accumulation error of 0 may differ
        tie = np.abs(A_r) < 1e-4 * np.abs(A_r).max()
        dA_g, dA_r = np.where(tie, 0, dA_g), np.where(tie, 0, dA_r)
    assert_close("dA", dA_g, dA_r, "bf16", case=name)
    if gated:
        assert_close("B", host(B_fwd[sl]), fw["B"][slots_r], "bf16", case=name)
        assert_close("dB", host(saved.B[sl]), bw["dB"][slots_r], "bf16", case=name)
    del A_fwd, B_fwd

    # ---- weight gradients: sampled columns of the most- and the least-loaded
    # expert (whose token sets agree), including columns of the last f-tile ----
    counts_r = ix_r.counts
    off_g = saved.offsets.cpu().numpy()
    eti_g = saved.eti.cpu().numpy()

    def agrees(e):
        seg_r = ix_r.eti[ix_r.offsets[e]:ix_r.offsets[e + 1]]
        seg_g = eti_g[off_g[e]:off_g[e + 1]]
        return counts_r[e] > 0 and np.array_equal(seg_r, seg_g)

    order = np.argsort(-counts_r, kind="stable")
    heavy = next(int(e) for e in order if agrees(e))
    light = next(int(e) for e in order[::-1] if agrees(e))
    cols = np.unique(np.concatenate([rng.choice(f, size=NCOL // 2, replace=False),
                                     f - 1 - rng.choice(min(f, 256), size=NCOL // 2, replace=False)]))
    for e, tag in ((heavy, "most-loaded"), (light, "least-loaded")):
        seg = ix_r.eti[ix_r.offsets[e]:ix_r.offsets[e + 1]]
        jsel = np.argmax(ids_r[seg] == e, axis=1)
        g_e = gates_r[seg, jsel][:, None]
        sub_ix = oracle.build_index(np.zeros((seg.size, 1), np.int32), 1)
        xw = v["x"][seg]
        W1s = v["w1"][e][:, cols][None]
        W2s = v["w2"][e][cols, :][None]
        if gated:
            W3s = v["w3"][e][:, cols][None]
            As, Bs, _ = oracle.ffn_fwd(xw, W1s, W3s, W2s, sub_ix, 1)
            sbw = oracle.ffn_bwd(v["dy"][seg], xw, W1s, W3s, W2s, g_e, sub_ix, As, Bs)
            assert_close("dw3 %s" % tag, host(g["dw3"][e])[:, cols], sbw["dw3"][0], "bf16", case=name)
        else:
            As, _ = oracle.ffn_fwd_act(xw, W1s, W2s, sub_ix, 1, cfg.act)
            sbw = oracle.ffn_bwd_act(v["dy"][seg], xw, W1s, W2s, g_e, sub_ix, As, cfg.act)
        assert_close("dw1 %s" % tag, host(g["dw1"][e])[:, cols], sbw["dw1"][0], "bf16", case=name)
        assert_close("dw2 %s" % tag, host(g["dw2"][e])[cols, :], sbw["dw2"][0], "bf16", case=name)
    if cfg.n_dead:
        dead = np.nonzero(~np.isfinite(v["bias"]))[0]
        assert np.all(host(g["dw1"][dead[0]]) == 0) and np.all(host(g["dw2"][dead[0]]) == 0)
    del y, saved, g
    torch.cuda.empty_cache()

    # ---- router backward at full size, oracle logits and seeded gate gradients ----------
    dgates = rng.standard_normal((T, k))
    dl_r, dwg_r, dxr_r = oracle.route_bwd(dgates, logits_r, ids_r, v["x"], v["w_gate"], cfg.renorm)
    flags = B.MOE_BF16 | (B.MOE_RENORM if cfg.renorm else 0)
    dwg = torch.empty((E, d), dtype=torch.float32, device="cuda")
    dxr = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    wsb = B.moe_route_bwd_workspace_size(T, d, E, k, flags)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    lg = np.where(np.isfinite(logits_r), logits_r, -np.inf).astype(np.float32)
    B.moe_route_bwd(dev(dgates.astype(np.float32)), dev(lg), dev(ids_r),
                    dev(gates_r.astype(np.float32)), x, wg, T, d, E, k, flags, dwg, dxr, ws, wsb)
    torch.cuda.synchronize()
    assert_close("dw_gate", host(dwg), dwg_r, "bf16", case=name)
    assert_close("dx_router", host(dxr), dxr_r, "bf16", case=name)


@pytest.mark.parametrize("name", ["mid_e64k6", "table1_conf1_relu", "d2880_e128k4", "few_large_e8k2"])
def test_full_size_h_on_load_bit_identical(name):
    """MOE_H_ON_LOAD at full size, in the launch configuration bench.py times
    (multi-strip combined calls): outputs and every gradient bit-identical to
    the default policy that buffers h and g*h."""
    cfg = _cfg(name)
    print("full-size h-on-load case %s: T=%d d=%d f=%d E=%d k=%d act=%s"
          % (name, cfg.T, cfg.d, cfg.f, cfg.E, cfg.k, cfg.act), flush=True)
    inp = synth.make_inputs(cfg, with_dy=True)
    st = inp.store
    x, wg, w1, w3, w2, dy = (dev(st[n]) if st[n] is not None else None
                             for n in ("x", "w_gate", "w1", "w3", "w2", "dy"))
    bias = dev(st["bias"]) if st["bias"] is not None else None
    outs = []
    for hol in (False, True):
        y, saved = layer.forward(x, wg, bias, w1, w3, w2, cfg.k, cfg.renorm, act=cfg.act,
                                 h_on_load=hol)
        g = layer.backward(saved, dy, x, wg, w1, w3, w2)
        torch.cuda.synchronize()
        outs.append([y] + [g[n] for n in ("dx", "dw1", "dw3", "dw2", "dw_gate", "d_gates")])
    for n, a, b in zip(("y", "dx", "dw1", "dw3", "dw2", "dw_gate", "d_gates"), *outs):
        if a is None:
            assert b is None
            continue
        assert torch.equal(a, b), n
