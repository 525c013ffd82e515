"""One MoE layer, forward and backward, driven through the C ABI.

This module only allocates device buffers with torch and calls the library's
entry points in order; every arithmetic step runs in the HIP kernels.

Forward (MoEBlaze paper, Sections 2-5):
  moe_route -> moe_build_index -> moe_ffn_fwd_combine
  (= moe_ffn_fwd + moe_combine, strip by strip, with no [T*k, d] output buffer)
Backward (Section 3.2):
  moe_ffn_bwd_combine (= moe_ffn_bwd + the unit-weight combine that sums the
  token gradient) -> moe_route_bwd (router gradient, added into dx)
``separate=True`` runs the four separate calls instead (same results).
``recompute=True`` is the full-recompute checkpoint policy (Section 5.2's
checkpoint carried one step further): the forward keeps only the routing
decision (ids, gates, logits). It runs the dispatch and the expert FFN over
chunks of tokens (``chunk_tokens``, rounded down to a multiple of 4 tokens;
by default as many tokens as keep a chunk's A and B within 4 GiB), so that
A, B and the maps of no more than one
chunk exist at a time. The backward rebuilds each chunk's maps, recomputes its
A and B with moe_ffn_recompute (bit-identical to the forward's), and adds the
chunk's weight gradients into the layer's (MOE_ACCUMULATE_DW). Per token, y,
dx and d_gates are bit-identical to the other policies; the weight gradients
differ only by the order of float32 sums over chunks.
``h_on_load=True`` (MOE_H_ON_LOAD, the default) buffers neither h in the
forward nor g*h in the backward: the second GEMM and the dW2 GEMM form them
again from A and B as they load them, so no SwiGLU intermediate is ever
written to HBM. ``h_on_load=False`` is the buffered policy: h passes from the
first GEMM to the second through a transient buffer, and g*h from the dh GEMM
to the dW2 GEMM (bit-identical results, more memory, less vector work).
``atomic_combine`` (MOE_ATOMIC_COMBINE, combined calls only) folds the
combine into the epilogues of the second GEMM and of the dX GEMM: their slot
rows are added into y and dx by packed-bf16 atomics, so no strip of the expert
output or of dX_slot is held, and no separate combine pass runs. Each add
rounds to bf16, and for k > 2 the result depends on the order in which the
tiles finish. The default (None) uses it where it is deterministic: bf16 and
k <= 2; otherwise the strips and the ordered gather-reduce.

What the forward keeps for the backward (the "saved activations"): the first
layer outputs A and B [S, f] (A alone for the non-gated SiLU / ReLU experts),
the routing decision (ids, gates, logits) and the dispatch maps (offsets,
expert_token_indices, token_index_map, slot_src). No permuted copy of x, no
SiLU(A), no h and no expert output O is kept.
"""
from __future__ import annotations

import contextlib
from dataclasses import dataclass

import torch

from . import binding as B

ELEM = {torch.bfloat16: 2, torch.float32: 4}


@dataclass
class Saved:
    T: int
    d: int
    f: int
    E: int
    k: int
    flags: int        # element type flag
    act: str          # "swiglu", "silu" or "relu"
    renorm: bool
    ids: torch.Tensor
    gates: torch.Tensor
    logits: torch.Tensor
    counts: torch.Tensor | None     # the maps and A, B: None under full recompute
    offsets: torch.Tensor | None
    eti: torch.Tensor | None
    tim: torch.Tensor | None
    slot_src: torch.Tensor | None
    A: torch.Tensor | None
    B: torch.Tensor | None
    h_on_load: bool = True
    chunk: int = 0                  # full recompute: tokens per chunk
    atomic_combine: bool = False

    @property
    def ffn_flags(self) -> int:
        return self.flags | B.ACT_FLAG[self.act] | (B.MOE_H_ON_LOAD if self.h_on_load else 0)

    @property
    def combine_flags(self) -> int:
        """Flags of the combined FFN calls."""
        return self.ffn_flags | (B.MOE_ATOMIC_COMBINE if self.atomic_combine else 0)

    def tensors(self):
        return [t for t in (self.ids, self.gates, self.logits, self.counts, self.offsets,
                            self.eti, self.tim, self.slot_src, self.A, self.B) if t is not None]

    def nbytes(self) -> int:
        return sum(t.numel() * t.element_size() for t in self.tensors())


def saved_bytes_per_token(d: int, f: int, E: int, k: int, elem: int, T: int,
                          act: str = "swiglu", recompute: bool = False) -> float:
    """Closed form of Saved.nbytes() / T: A and B (2 k f elem; A alone, k f elem,
    for a non-gated expert), ids, gates, token_index_map, expert_token_indices
    and slot_src (5 x 4k), logits (4E), counts and offsets (4(2E+1) per layer).
    Full recompute keeps the ids, gates and logits alone (8k + 4E)."""
    if recompute:
        return 8.0 * k + 4.0 * E
    n_first = 2 if act == "swiglu" else 1
    return n_first * k * f * elem + 20.0 * k + 4.0 * E + 4.0 * (2 * E + 1) / T


def default_chunk(T: int, k: int, f: int, gated: bool, elem: int) -> int:
    """Tokens per chunk of the full-recompute policy: A and B of one chunk
    within 4 GiB (at least 4096 tokens, at most T)."""
    per_token = k * f * elem * (2 if gated else 1)
    return int(max(1, min(T, max(4096, (4 << 30) // per_token))))


def aligned_chunk(chunk: int, T: int) -> int:
    """A chunk of T tokens as the chunked calls take it: all of T, or a
    multiple of 4 tokens (at least 4), so that every chunk's rows of the
    [T, k] routing arrays (4-byte elements) start 16-byte aligned, as the C
    ABI requires of its pointers."""
    if chunk >= T:
        return T
    return max(4, chunk - chunk % 4)


def _on(stream):
    """Run a layer call on `stream` (a torch.cuda.Stream; None: torch's current
    stream). The temporaries are allocated under it too, so the caching
    allocator never hands a freed workspace to other work while the library's
    kernels on that stream may still use it."""
    if stream is None:
        return contextlib.nullcontext()
    if not isinstance(stream, torch.cuda.Stream):
        raise TypeError("stream must be a torch.cuda.Stream or None")
    return torch.cuda.stream(stream)


def forward(x, w_gate, bias, w1, w3, w2, k: int, renorm: bool, stream=None, keep_O=False,
            act: str = "swiglu", separate: bool = False, recompute: bool = False,
            h_on_load: bool = True, chunk_tokens: int | None = None,
            atomic_combine: bool | None = None):
    """Returns (y, saved[, O]). ``act`` picks the expert: "swiglu" (gated, w3
    used) or the non-gated "silu" / "relu" (w3 ignored, may be None).
    ``keep_O`` (returns the expert outputs) implies ``separate``. Everything
    runs on ``stream`` (torch's current stream if None)."""
    if atomic_combine and (keep_O or separate):
        raise ValueError("atomic_combine applies to the combined calls only")
    if atomic_combine is None:   # where the atomic sum is deterministic
        atomic_combine = (not (keep_O or separate) and k <= 2 and
                          x.dtype == torch.bfloat16)
    with _on(stream):
        if recompute:
            if keep_O or separate:
                raise ValueError("the full-recompute policy runs the combined calls only")
            return _forward_recompute(x, w_gate, bias, w1, w3, w2, k, renorm, act, h_on_load,
                                      chunk_tokens, atomic_combine)
        return _forward(x, w_gate, bias, w1, w3, w2, k, renorm, keep_O, act, separate,
                        h_on_load, atomic_combine)


def _route(x, w_gate, bias, E, k, renorm, flags):
    T, d = x.shape
    i32 = dict(dtype=torch.int32, device=x.device)
    f32 = dict(dtype=torch.float32, device=x.device)
    ids = torch.empty((T, k), **i32)
    gates = torch.empty((T, k), **f32)
    logits = torch.empty((T, E), **f32)
    B.moe_route(x, w_gate, bias, T, d, E, k, flags | (B.MOE_RENORM if renorm else 0), ids, gates,
                logits, None)
    return ids, gates, logits


def _maps(ids, T, E, k):
    """The dispatch maps of ids [T, k]: counts, offsets, eti, tim, slot_src."""
    i32 = dict(dtype=torch.int32, device=ids.device)
    S = T * k
    m = (torch.empty(E, **i32), torch.empty(E + 1, **i32), torch.empty(S, **i32),
         torch.empty((T, k), **i32), torch.empty(S, **i32))
    wsb = B.moe_build_index_workspace_size(T, E, k)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=ids.device)
    B.moe_build_index(ids, T, E, k, *m, ws, wsb, None)
    del ws
    return m


def _chunks(T, chunk):
    for t0 in range(0, T, chunk):
        yield t0, min(T, t0 + chunk)


def _forward_recompute(x, w_gate, bias, w1, w3, w2, k, renorm, act, h_on_load, chunk_tokens,
                       atomic_combine):
    T, d = x.shape
    E, _, f = w1.shape
    flags = B.dtype_flag(x)
    gated = act == "swiglu"
    ids, gates, logits = _route(x, w_gate, bias, E, k, renorm, flags)
    chunk = aligned_chunk(chunk_tokens or default_chunk(T, k, f, gated, x.element_size()), T)
    fflags = (flags | B.ACT_FLAG[act] | (B.MOE_H_ON_LOAD if h_on_load else 0)
              | (B.MOE_ATOMIC_COMBINE if atomic_combine else 0))
    y = torch.empty((T, d), dtype=x.dtype, device=x.device)
    for t0, t1 in _chunks(T, chunk):
        Tc = t1 - t0
        counts, offsets, eti, tim, slot_src = _maps(ids[t0:t1], Tc, E, k)
        A = torch.empty((Tc * k, f), dtype=x.dtype, device=x.device)
        Bm = torch.empty((Tc * k, f), dtype=x.dtype, device=x.device) if gated else None
        wsb = B.moe_ffn_fwd_combine_workspace_size(Tc, d, f, E, k, fflags)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=x.device)
        B.moe_ffn_fwd_combine(x[t0:t1], w1, w3 if gated else None, w2, offsets, eti, gates[t0:t1],
                              tim, Tc, d, f, E, k, fflags, A, Bm, y[t0:t1], ws, wsb, None)
        del counts, offsets, eti, tim, slot_src, A, Bm, ws
    saved = Saved(T, d, f, E, k, flags, act, renorm, ids, gates, logits, None, None, None, None,
                  None, None, None, h_on_load, chunk, atomic_combine)
    return y, saved


def _forward(x, w_gate, bias, w1, w3, w2, k, renorm, keep_O, act, separate, h_on_load,
             atomic_combine):
    stream = None   # torch's current stream, set by forward()
    T, d = x.shape
    E, _, f = w1.shape
    dev = x.device
    flags = B.dtype_flag(x)
    S = T * k
    i32 = dict(dtype=torch.int32, device=dev)
    f32 = dict(dtype=torch.float32, device=dev)
    ids = torch.empty((T, k), **i32)
    gates = torch.empty((T, k), **f32)
    logits = torch.empty((T, E), **f32)
    B.moe_route(x, w_gate, bias, T, d, E, k, flags | (B.MOE_RENORM if renorm else 0), ids, gates,
                logits, stream)
    counts = torch.empty(E, **i32)
    offsets = torch.empty(E + 1, **i32)
    eti = torch.empty(S, **i32)
    tim = torch.empty((T, k), **i32)
    slot_src = torch.empty(S, **i32)
    wsb = B.moe_build_index_workspace_size(T, E, k)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
    B.moe_build_index(ids, T, E, k, counts, offsets, eti, tim, slot_src, ws, wsb, stream)
    del ws
    gated = act == "swiglu"
    fflags = flags | B.ACT_FLAG[act] | (B.MOE_H_ON_LOAD if h_on_load else 0)
    A = torch.empty((S, f), dtype=x.dtype, device=dev)
    Bm = torch.empty((S, f), dtype=x.dtype, device=dev) if gated else None
    y = torch.empty((T, d), dtype=x.dtype, device=dev)
    saved = Saved(T, d, f, E, k, flags, act, renorm, ids, gates, logits, counts, offsets, eti,
                  tim, slot_src, A, Bm, h_on_load, 0, atomic_combine)
    w3g = w3 if gated else None
    if not (separate or keep_O):
        cflags = saved.combine_flags
        wsb = B.moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, cflags)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
        B.moe_ffn_fwd_combine(x, w1, w3g, w2, offsets, eti, gates, tim, T, d, f, E, k, cflags, A,
                              Bm, y, ws, wsb, stream)
        del ws
        return y, saved
    O = torch.empty((S, d), dtype=x.dtype, device=dev)
    wsb = B.moe_ffn_fwd_workspace_size(T, d, f, E, k, fflags)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
    B.moe_ffn_fwd(x, w1, w3g, w2, offsets, eti, T, d, f, E, k, fflags, A, Bm, O, ws, wsb, stream)
    del ws
    B.moe_combine(O, gates, tim, T, d, k, flags, y, stream)
    if keep_O:
        return y, saved, O
    del O
    return y, saved


def backward(saved: Saved, dy, x, w_gate, w1, w3, w2, stream=None, keep=False,
             separate: bool = False):
    """Returns dict(dx, dw_gate, dw1, dw3, dw2, d_gates[, dX_slot]). Overwrites
    saved.A / saved.B with dA / dB. dw3 is None for a non-gated expert.
    ``keep`` (returns dX_slot and the FFN part of dx) implies ``separate``.
    Everything runs on ``stream`` (torch's current stream if None)."""
    with _on(stream):
        return _backward(saved, dy, x, w_gate, w1, w3, w2, keep, separate)


def _backward_recompute(s, dy, x, w_gate, w1, w3, w2):
    """Full recompute: per chunk, the maps and the first layer again, then the
    chunk's backward with its weight gradients added into the layer's."""
    T, d, f, E, k = s.T, s.d, s.f, s.E, s.k
    dev = dy.device
    f32 = dict(dtype=torch.float32, device=dev)
    gated = s.act == "swiglu"
    w3g = w3 if gated else None
    dw1 = torch.empty((E, d, f), **f32)
    dw3 = torch.empty((E, d, f), **f32) if gated else None
    dw2 = torch.empty((E, f, d), **f32)
    d_gates = torch.empty((T, k), **f32)
    dx = torch.empty((T, d), dtype=dy.dtype, device=dev)
    for i, (t0, t1) in enumerate(_chunks(T, s.chunk)):
        Tc = t1 - t0
        counts, offsets, eti, tim, slot_src = _maps(s.ids[t0:t1], Tc, E, k)
        A = torch.empty((Tc * k, f), dtype=dy.dtype, device=dev)
        Bm = torch.empty((Tc * k, f), dtype=dy.dtype, device=dev) if gated else None
        B.moe_ffn_recompute(x[t0:t1], w1, w3g, offsets, eti, Tc, d, f, E, k, s.ffn_flags, A, Bm,
                            None)
        fl = s.combine_flags | (B.MOE_ACCUMULATE_DW if i else 0)
        wsb = B.moe_ffn_bwd_combine_workspace_size(Tc, d, f, E, k, fl)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
        B.moe_ffn_bwd_combine(dy[t0:t1], x[t0:t1], w1, w3g, w2, s.gates[t0:t1], offsets, eti,
                              slot_src, tim, A, Bm, Tc, d, f, E, k, fl, dw1, dw3, dw2,
                              d_gates[t0:t1], dx[t0:t1], ws, wsb, None)
        del counts, offsets, eti, tim, slot_src, A, Bm, ws
    return dict(dw1=dw1, dw3=dw3, dw2=dw2, d_gates=d_gates), dx


def _backward(saved, dy, x, w_gate, w1, w3, w2, keep, separate):
    stream = None   # torch's current stream, set by backward()
    s = saved
    T, d, f, E, k = s.T, s.d, s.f, s.E, s.k
    dev = dy.device
    f32 = dict(dtype=torch.float32, device=dev)
    gated = s.act == "swiglu"
    if s.chunk:   # full recompute
        if keep or separate:
            raise ValueError("the full-recompute policy runs the combined calls only")
        out, dx = _backward_recompute(s, dy, x, w_gate, w1, w3, w2)
        return _router_backward(s, x, w_gate, out, dx)
    dw1 = torch.empty((E, d, f), **f32)
    dw3 = torch.empty((E, d, f), **f32) if gated else None
    dw2 = torch.empty((E, f, d), **f32)
    d_gates = torch.empty((T, k), **f32)
    dx = torch.empty((T, d), dtype=dy.dtype, device=dev)
    w3g = w3 if gated else None
    out = dict(dw1=dw1, dw3=dw3, dw2=dw2, d_gates=d_gates)
    if not (separate or keep):
        wsb = B.moe_ffn_bwd_combine_workspace_size(T, d, f, E, k, s.combine_flags)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
        B.moe_ffn_bwd_combine(dy, x, w1, w3g, w2, s.gates, s.offsets, s.eti, s.slot_src, s.tim,
                              s.A, s.B, T, d, f, E, k, s.combine_flags, dw1, dw3, dw2, d_gates, dx,
                              ws, wsb, stream)
        del ws
    else:
        dX = torch.empty((T * k, d), dtype=dy.dtype, device=dev)
        wsb = B.moe_ffn_bwd_workspace_size(T, d, f, E, k, s.ffn_flags)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
        B.moe_ffn_bwd(dy, x, w1, w3g, w2, s.gates, s.offsets, s.eti, s.slot_src, s.A, s.B, T, d,
                      f, E, k, s.ffn_flags, dw1, dw3, dw2, d_gates, dX, ws, wsb, stream)
        del ws
        B.moe_combine(dX, None, s.tim, T, d, k, s.flags, dx, stream)
        if keep:
            out["dX_slot"] = dX
            out["dx_ffn"] = dx.clone()
        del dX
    return _router_backward(s, x, w_gate, out, dx)


def _router_backward(s, x, w_gate, out, dx):
    """moe_route_bwd over all tokens: dW_g, and the router's part added into dx."""
    T, d, E, k = s.T, s.d, s.E, s.k
    dwg = torch.empty((E, d), dtype=torch.float32, device=dx.device)
    rflags = s.flags | B.MOE_ACCUMULATE | (B.MOE_RENORM if s.renorm else 0)
    wsb = B.moe_route_bwd_workspace_size(T, d, E, k, rflags)
    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dx.device)
    B.moe_route_bwd(out["d_gates"], s.logits, s.ids, s.gates, x, w_gate, T, d, E, k, rflags, dwg,
                    dx, ws, wsb, None)
    del ws
    out.update(dx=dx, dw_gate=dwg)
    return out
