"""Python front end of the CPU oracle (``moe_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the package smoke check
and the benchmark's CPU-baseline leg, never by the product path. It shares no
code with the HIP library. Every function takes and returns numpy arrays; all
floating point is float64.

Section references are to the MoEBlaze paper (arXiv 2601.05296).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile ``moe_oracle.c`` into ``liboracle.so`` with gcc and OpenMP."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        _lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        I64, I = ctypes.c_int64, ctypes.c_int
        _lib.oracle_route.argtypes = [P, P, P, I64, I, I, I, I, P, P, P, P]
        _lib.oracle_build_index.argtypes = [P, I64, I, I, P, P, P, P, P]
        _lib.oracle_ffn_fwd.argtypes = [P, P, P, P, P, P, I64, I, I, I, I, P, P, P]
        _lib.oracle_combine.argtypes = [P, P, P, I64, I, I, P]
        _lib.oracle_ffn_bwd.argtypes = [P] * 11 + [I64, I, I, I, I] + [P] * 7
        _lib.oracle_route_bwd.argtypes = [P, P, P, P, P, I64, I, I, I, I, P, P, P]
        _lib.oracle_ffn_fwd_act.argtypes = [P, P, P, P, P, I64, I, I, I, I, I, P, P]
        _lib.oracle_ffn_bwd_act.argtypes = [P] * 9 + [I64, I, I, I, I, I] + [P] * 5
        _lib.oracle_threads.argtypes = []
        _lib.oracle_threads.restype = ctypes.c_int
        for fn in ("oracle_route", "oracle_build_index", "oracle_ffn_fwd",
                   "oracle_combine", "oracle_ffn_bwd", "oracle_route_bwd"):
            getattr(_lib, fn).restype = None
    return _lib


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def threads() -> int:
    """Number of threads the oracle's OpenMP loops use."""
    return int(_load().oracle_threads())


def route(x, w_gate, bias, k: int, renorm: bool):
    """Top-k softmax gating (Section 2.1). Returns ids [T,k] int32, gates [T,k],
    logits [T,E], probs [T,E]."""
    x, w_gate, bias = _f64(x), _f64(w_gate), _f64(bias)
    T, d = x.shape
    E = w_gate.shape[0]
    ids = np.empty((T, k), np.int32)
    gates = np.empty((T, k))
    logits = np.empty((T, E))
    probs = np.empty((T, E))
    _load().oracle_route(_p(x), _p(w_gate), _p(bias), T, d, E, k, int(bool(renorm)),
                         _p(ids), _p(gates), _p(logits), _p(probs))
    return ids, gates, logits, probs


@dataclass
class Index:
    counts: np.ndarray
    offsets: np.ndarray
    eti: np.ndarray       # expert_token_indices [S]
    tim: np.ndarray       # token_index_map [T,k]
    slot_src: np.ndarray  # [S]


def build_index(ids, E: int) -> Index:
    """Dispatch maps (Section 4.1 definitions)."""
    ids = _i32(ids)
    T, k = ids.shape
    S = T * k
    ix = Index(np.empty(E, np.int32), np.empty(E + 1, np.int32), np.empty(S, np.int32),
               np.empty((T, k), np.int32), np.empty(S, np.int32))
    _load().oracle_build_index(_p(ids), T, E, k, _p(ix.counts), _p(ix.offsets), _p(ix.eti),
                               _p(ix.tim), _p(ix.slot_src))
    return ix


def ffn_fwd(x, w1, w3, w2, ix: Index, k: int):
    """Per-slot SwiGLU expert forward (Section 3.1, Algorithm 1). Returns A, B
    [S,f] and O [S,d]."""
    x, w1, w3, w2 = _f64(x), _f64(w1), _f64(w3), _f64(w2)
    T, d = x.shape
    E, _, f = w1.shape
    S = T * k
    A = np.empty((S, f)); B = np.empty((S, f)); O = np.empty((S, d))
    _load().oracle_ffn_fwd(_p(x), _p(w1), _p(w3), _p(w2), _p(ix.offsets), _p(ix.eti),
                           T, d, f, E, k, _p(A), _p(B), _p(O))
    return A, B, O


# expert activations: "swiglu" (Section 5.1, gated, W3 branch) or the non-gated
# "silu" / "relu" experts of Section 2.2 (E(x) = W2 act(W1 x))
ACTS = {"silu": 1, "relu": 2}


def ffn_fwd_act(x, w1, w2, ix: Index, k: int, act: str):
    """Per-slot non-gated expert forward (Section 2.2). Returns A [S,f] (the
    saved pre-activation) and O [S,d]."""
    x, w1, w2 = _f64(x), _f64(w1), _f64(w2)
    T, d = x.shape
    E, _, f = w1.shape
    S = T * k
    A = np.empty((S, f)); O = np.empty((S, d))
    _load().oracle_ffn_fwd_act(_p(x), _p(w1), _p(w2), _p(ix.offsets), _p(ix.eti), T, d, f, E, k,
                               ACTS[act], _p(A), _p(O))
    return A, O


def ffn_bwd_act(dy, x, w1, w2, gates, ix: Index, A, act: str):
    """Non-gated expert backward (Section 3.2 with the Section 2.2 expert).
    Returns dict with dA [S,f], dw1 [E,d,f], dw2 [E,f,d], d_gates [T,k],
    dX_slot [S,d]."""
    dy, x, w1, w2, gates, A = map(_f64, (dy, x, w1, w2, gates, A))
    T, d = x.shape
    E, _, f = w1.shape
    k = gates.shape[1]
    S = T * k
    out = dict(dA=np.empty((S, f)), dw1=np.empty((E, d, f)), dw2=np.empty((E, f, d)),
               d_gates=np.empty((T, k)), dX_slot=np.empty((S, d)))
    _load().oracle_ffn_bwd_act(_p(dy), _p(x), _p(w1), _p(w2), _p(gates), _p(ix.offsets),
                               _p(ix.eti), _p(ix.slot_src), _p(A), T, d, f, E, k, ACTS[act],
                               _p(out["dA"]), _p(out["dw1"]), _p(out["dw2"]),
                               _p(out["d_gates"]), _p(out["dX_slot"]))
    return out


def combine(src, weights, tim):
    """out[t] = sum_j w[t,j] src[tim[t,j]] (Section 2.3; weights None = 1)."""
    src, weights, tim = _f64(src), _f64(weights), _i32(tim)
    T, k = tim.shape
    d = src.shape[1]
    out = np.empty((T, d))
    _load().oracle_combine(_p(src), _p(weights), _p(tim), T, d, k, _p(out))
    return out


def ffn_bwd(dy, x, w1, w3, w2, gates, ix: Index, A, B):
    """Expert backward (Section 3.2, Algorithm 1). Returns dict with dA, dB
    [S,f], dw1, dw3 [E,d,f], dw2 [E,f,d], d_gates [T,k], dX_slot [S,d]."""
    dy, x, w1, w3, w2, gates, A, B = map(_f64, (dy, x, w1, w3, w2, gates, A, B))
    T, d = x.shape
    E, _, f = w1.shape
    k = gates.shape[1]
    S = T * k
    out = dict(dA=np.empty((S, f)), dB=np.empty((S, f)), dw1=np.empty((E, d, f)),
               dw3=np.empty((E, d, f)), dw2=np.empty((E, f, d)), d_gates=np.empty((T, k)),
               dX_slot=np.empty((S, d)))
    _load().oracle_ffn_bwd(_p(dy), _p(x), _p(w1), _p(w3), _p(w2), _p(gates), _p(ix.offsets),
                           _p(ix.eti), _p(ix.slot_src), _p(A), _p(B), T, d, f, E, k,
                           _p(out["dA"]), _p(out["dB"]), _p(out["dw1"]), _p(out["dw3"]),
                           _p(out["dw2"]), _p(out["d_gates"]), _p(out["dX_slot"]))
    return out


def route_bwd(d_gates, logits, ids, x, w_gate, renorm: bool):
    """Router backward (closed-form gating Jacobian). Returns dlogits [T,E],
    dw_gate [E,d], dx_router [T,d]."""
    d_gates, logits, x, w_gate = map(_f64, (d_gates, logits, x, w_gate))
    ids = _i32(ids)
    T, k = ids.shape
    E, d = w_gate.shape
    dl = np.empty((T, E)); dwg = np.empty((E, d)); dxr = np.empty((T, d))
    _load().oracle_route_bwd(_p(d_gates), _p(logits), _p(ids), _p(x), _p(w_gate), T, d, E, k,
                             int(bool(renorm)), _p(dl), _p(dwg), _p(dxr))
    return dl, dwg, dxr


def layer_forward(x, w_gate, bias, w1, w3, w2, k: int, renorm: bool, ids=None,
                  act: str = "swiglu"):
    """Whole layer forward. ``ids`` pins the routing decision (used when a
    caller compares against a device run that already routed). For a
    non-gated ``act`` w3 is unused and B is None."""
    r_ids, gates, logits, probs = route(x, w_gate, bias, k, renorm)
    if ids is not None:
        ids = _i32(ids)
        p_sel = np.take_along_axis(probs, ids, axis=1)
        gates = p_sel / p_sel.sum(axis=1, keepdims=True) if renorm else p_sel
    else:
        ids = r_ids
    E = w_gate.shape[0]
    ix = build_index(ids, E)
    if act == "swiglu":
        A, B, O = ffn_fwd(x, w1, w3, w2, ix, k)
    else:
        (A, O), B = ffn_fwd_act(x, w1, w2, ix, k, act), None
    y = combine(O, gates, ix.tim)
    return dict(ids=ids, gates=gates, logits=logits, probs=probs, ix=ix, A=A, B=B, O=O, y=y,
                act=act)


def layer_backward(fw: dict, dy, x, w_gate, w1, w3, w2, renorm: bool):
    """Whole layer backward from a ``layer_forward`` result: expert backward,
    token gradient accumulation (Section 3.2 step 3) and router backward."""
    act = fw.get("act", "swiglu")
    if act == "swiglu":
        bw = ffn_bwd(dy, x, w1, w3, w2, fw["gates"], fw["ix"], fw["A"], fw["B"])
    else:
        bw = ffn_bwd_act(dy, x, w1, w2, fw["gates"], fw["ix"], fw["A"], act)
    dx_ffn = combine(bw["dX_slot"], None, fw["ix"].tim)
    dl, dwg, dxr = route_bwd(bw["d_gates"], fw["logits"], fw["ids"], x, w_gate, renorm)
    bw.update(dx_ffn=dx_ffn, dlogits=dl, dw_gate=dwg, dx_router=dxr, dx=dx_ffn + dxr)
    return bw
