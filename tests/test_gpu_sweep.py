"""GPU parity at the memory-sweep sizes (d=4096, f=2048, E=64, k=8): T = 2^20
tokens with the buffered h policy and T = 2^21 with h formed on load (with the
ordered strip combine, and with the combine folded into the GEMM epilogues), the
largest T each policy fits in one GPU's memory (paper Sections 3.1-3.2: the
method exists to run larger T in the same memory). Here S = T*k reaches 2^24
slots, and slot-row element offsets (slot * f) pass 2^31.

Inputs are drawn on the device by the seeded generator (synth.device_inputs);
the oracle receives the same values, downloaded. No oracle input comes from
the HIP path. Checks:
  * routing of every token by the oracle: ids equal up to near-ties;
  * the index build fed the oracle's ids, bit-exact against the oracle's;
  * the layer's own maps (built from the device ids) satisfy the defining
    invariants of Section 4.1, which leave exactly one set of maps for given
    ids: counts and offsets, each choice in its expert's segment, tokens
    ascending inside a segment, token_index_map a bijection, slot_src and
    expert_token_indices its inverse;
  * y, dx, d_gates, A, B, dA, dB of sampled tokens (half of them those holding
    the highest slots, in the last experts' tails) against the oracle run on
    those tokens alone;
  * dw1, dw3, dw2 of the last expert at sampled hidden columns (some in the
    last f-tile) against the oracle on that expert's sub-problem;
  * every weight gradient of the full run equals the sum of the two runs over
    the first and the second half of the tokens (the gradient is a sum over
    tokens), to float32 summation-order error.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2601_05296_amd import binding as B
from paper_2601_05296_amd import layer, synth
from tests.parity import assert_close, host, near_tie_ok

pytestmark = pytest.mark.gpu

# name, T, h on load, combine folded into the GEMM epilogues (atomics)
CASES = [("sweep_T2^20_buffered", 1 << 20, False, False),
         ("sweep_T2^21_h_on_load", 1 << 21, True, False),
         ("sweep_T2^21_h_on_load_atomic", 1 << 21, True, True)]
NTOK = 16
NCOL = 8
CHUNK = 1 << 17      # tokens per host chunk of the oracle's routing


def step(msg):
    print(msg, flush=True)


def f64(t):
    """Device bf16 / float32 tensor -> host float64 (bf16 widened exactly)."""
    return t.float().cpu().numpy().astype(np.float64)


def check_maps(ids, counts, offsets, eti, tim, slot_src, E):
    """The index-map invariants that fix the maps for given ids."""
    T, k = ids.shape
    S = T * k
    flat = ids.reshape(-1).astype(np.int64)
    assert flat.min() >= 0 and flat.max() < E
    assert np.array_equal(counts, np.bincount(flat, minlength=E))
    assert offsets[0] == 0 and np.array_equal(np.diff(offsets), counts) and offsets[E] == S
    slots = tim.reshape(-1).astype(np.int64)
    assert slots.min() >= 0 and slots.max() < S
    assert np.all(np.bincount(slots, minlength=S) == 1)                 # bijection
    expert_of_slot = np.repeat(np.arange(E), counts)
    assert np.array_equal(expert_of_slot[slots], flat)                  # own segment
    assert np.array_equal(eti[slots], np.repeat(np.arange(T), k))       # eti inverts tim
    assert np.array_equal(slot_src[slots], np.arange(S))                # slot_src too
    step_up = np.diff(eti.astype(np.int64))
    inner = np.ones(S - 1, dtype=bool)
    inner[offsets[1:E][(offsets[1:E] > 0) & (offsets[1:E] < S)] - 1] = False
    assert np.all(step_up[inner] > 0)                                   # ascending tokens


@pytest.mark.parametrize("name,T,hol,atomic", CASES)
def test_memory_sweep_size(name, T, hol, atomic):
    cfg = synth.CONFIGS["mem_sweep_e64k8"].with_(T=T)
    d, f, E, k = cfg.d, cfg.f, cfg.E, cfg.k
    S = T * k
    step("sweep case %s: T=%d d=%d f=%d E=%d k=%d h_on_load=%s atomic combine=%s "
         "(S*f = %d elements)" % (name, T, d, f, E, k, hol, atomic, S * f))
    inp = synth.device_inputs(cfg, "cuda")
    x, wg, w1, w3, w2, dy = (inp[n] for n in ("x", "w_gate", "w1", "w3", "w2", "dy"))

    # ---- oracle routing of every token, host chunks of x -----------------------
    step("  oracle routing of %d tokens" % T)
    wg64 = f64(wg)
    ids_r = np.empty((T, k), np.int32)
    gates_r = np.empty((T, k))
    logits_r = np.empty((T, E))
    for t0 in range(0, T, CHUNK):
        ir, gr, lr, _ = oracle.route(f64(x[t0:t0 + CHUNK]), wg64, None, k, cfg.renorm)
        ids_r[t0:t0 + CHUNK], gates_r[t0:t0 + CHUNK], logits_r[t0:t0 + CHUNK] = ir, gr, lr

    # ---- index build on the oracle's ids, bit-exact ------------------------------
    step("  index build on the oracle's ids")
    ix_r = oracle.build_index(ids_r, E)
    i32 = dict(dtype=torch.int32, device="cuda")
    o = [torch.empty(E, **i32), torch.empty(E + 1, **i32), torch.empty(S, **i32),
         torch.empty((T, k), **i32), torch.empty(S, **i32)]
    wsb = B.moe_build_index_workspace_size(T, E, k)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
    B.moe_build_index(torch.from_numpy(ids_r).cuda(), T, E, k, *o, ws, wsb)
    torch.cuda.synchronize()
    for got, ref in zip(o, (ix_r.counts, ix_r.offsets, ix_r.eti, ix_r.tim, ix_r.slot_src)):
        assert np.array_equal(got.cpu().numpy(), ref)
    del o, ws

    # ---- the layer, forward -------------------------------------------------------
    step("  layer forward")
    y, saved = layer.forward(x, wg, None, w1, w3, w2, k, cfg.renorm, h_on_load=hol,
                             atomic_combine=atomic)
    torch.cuda.synchronize()
    assert saved.atomic_combine == atomic
    ids_g = saved.ids.cpu().numpy()
    nflip = near_tie_ok(ids_g, ids_r, logits_r)
    assert nflip <= max(2, T // 5000), nflip
    assert_close("gates", host(saved.gates)[np.all(ids_g == ids_r, axis=1)],
                 gates_r[np.all(ids_g == ids_r, axis=1)], "bf16", case=name)
    step("  map invariants (%d flips)" % nflip)
    tim_g = saved.tim.cpu().numpy()
    eti_g = saved.eti.cpu().numpy()
    off_g = saved.offsets.cpu().numpy()
    check_maps(ids_g, saved.counts.cpu().numpy(), off_g, eti_g, tim_g, saved.slot_src.cpu().numpy(),
               E)

    # sampled tokens: the highest slots, and random ones, all with agreeing ids
    rng = np.random.default_rng(4321)
    agree = np.nonzero(np.all(ids_g == ids_r, axis=1))[0]
    top = agree[np.argsort(-tim_g[agree].max(axis=1), kind="stable")[:NTOK // 2]]
    rest = np.setdiff1d(agree, top)
    toks = np.sort(np.concatenate([top, rng.choice(rest, NTOK - top.size, replace=False)]))
    assert int(tim_g[toks].max()) * f > 2 ** 31
    sl = torch.from_numpy(tim_g[toks].reshape(-1)).long().cuda()
    A_fwd = saved.A[sl].clone()
    B_fwd = saved.B[sl].clone()
    y_s = host(y[torch.from_numpy(toks).cuda()])
    del y

    # ---- backward -------------------------------------------------------------------
    step("  layer backward")
    g = layer.backward(saved, dy, x, wg, w1, w3, w2)
    torch.cuda.synchronize()

    # ---- sampled tokens against the oracle --------------------------------------------
    step("  oracle on %d sampled tokens" % toks.size)
    tk = torch.from_numpy(toks).cuda()
    W1, W3, W2 = f64(w1), f64(w3), f64(w2)
    xs, dys = f64(x[tk]), f64(dy[tk])
    fw = oracle.layer_forward(xs, wg64, None, W1, W3, W2, k, cfg.renorm)
    assert np.array_equal(fw["ids"], ids_g[toks])
    bw = oracle.layer_backward(fw, dys, xs, wg64, W1, W3, W2, cfg.renorm)
    slots_r = fw["ix"].tim.reshape(-1)
    assert_close("y", y_s, fw["y"], "bf16", case=name)
    assert_close("dx", host(g["dx"][tk]), bw["dx"], "bf16", case=name)
    assert_close("d_gates", host(g["d_gates"][tk]), bw["d_gates"], "bf16", case=name)
    assert_close("A", host(A_fwd), fw["A"][slots_r], "bf16", case=name)
    assert_close("B", host(B_fwd), fw["B"][slots_r], "bf16", case=name)
    assert_close("dA", host(saved.A[sl]), bw["dA"][slots_r], "bf16", case=name)
    assert_close("dB", host(saved.B[sl]), bw["dB"][slots_r], "bf16", case=name)
    del A_fwd, B_fwd

    # ---- the last expert's weight gradients at sampled columns --------------------------
    e = E - 1
    seg = ix_r.eti[ix_r.offsets[e]:ix_r.offsets[e + 1]]
    assert np.array_equal(seg, eti_g[off_g[e]:off_g[e + 1]])
    step("  oracle sub-problem of expert %d (%d tokens)" % (e, seg.size))
    cols = np.unique(np.concatenate([rng.choice(f, NCOL // 2, replace=False),
                                     f - 1 - rng.choice(256, NCOL // 2, replace=False)]))
    jsel = np.argmax(ids_r[seg] == e, axis=1)
    g_e = gates_r[seg, jsel][:, None]
    sub_ix = oracle.build_index(np.zeros((seg.size, 1), np.int32), 1)
    sg = torch.from_numpy(seg.astype(np.int64)).cuda()
    xw, dyw = f64(x[sg]), f64(dy[sg])
    W1s, W3s, W2s = W1[e][:, cols][None], W3[e][:, cols][None], W2[e][cols, :][None]
    del W1, W3, W2
    As, Bs, _ = oracle.ffn_fwd(xw, W1s, W3s, W2s, sub_ix, 1)
    sbw = oracle.ffn_bwd(dyw, xw, W1s, W3s, W2s, g_e, sub_ix, As, Bs)
    assert_close("dw1 last expert", host(g["dw1"][e])[:, cols], sbw["dw1"][0], "bf16", case=name)
    assert_close("dw3 last expert", host(g["dw3"][e])[:, cols], sbw["dw3"][0], "bf16", case=name)
    assert_close("dw2 last expert", host(g["dw2"][e])[cols, :], sbw["dw2"][0], "bf16", case=name)
    del xw, dyw, saved

    # ---- gradients are sums over tokens: full run = first half + second half ------------
    step("  two-halves weight-gradient check")
    full = {n: g[n] for n in ("dw1", "dw3", "dw2", "dw_gate")}
    del g
    torch.cuda.empty_cache()
    acc = None
    for h0, h1 in ((0, T // 2), (T // 2, T)):
        yh, sh = layer.forward(x[h0:h1], wg, None, w1, w3, w2, k, cfg.renorm, h_on_load=hol,
                               atomic_combine=atomic)
        gh = layer.backward(sh, dy[h0:h1], x[h0:h1], wg, w1, w3, w2)
        del yh, sh
        part = {n: gh[n] for n in full}
        del gh
        if acc is None:
            acc = part
        else:
            for n in full:
                acc[n] += part[n]
            del part
        torch.cuda.empty_cache()
    torch.cuda.synchronize()
    for n in full:
        err = float((full[n] - acc[n]).abs().max() / full[n].abs().max())
        step("    %s: max|full - halves| / max|full| = %.2e" % (n, err))
        assert err <= 1e-3, (n, err)
