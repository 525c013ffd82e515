"""ctypes binding of libmoeblaze.so: one Python function per C entry point,
same names, argument marshalling only.

Tensors are torch tensors on the GPU (PyTorch supplies device memory and
streams); every computation runs in the library's HIP kernels. If the library
is not built, or no GPU is present when a call is made, the call raises: there
is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

from .build import LIB

MOE_OK = 0
MOE_ERR_INVALID_ARG = -1
MOE_ERR_UNSUPPORTED = -2
MOE_ERR_WORKSPACE = -3
MOE_ERR_HIP = -4

MOE_BF16 = 0
MOE_F32 = 1
MOE_RENORM = 2
MOE_ACCUMULATE = 4
MOE_ACT_SILU = 8
MOE_ACT_RELU = 16
MOE_H_ON_LOAD = 32
MOE_ACCUMULATE_DW = 64
MOE_ATOMIC_COMBINE = 128
ACT_FLAG = {"swiglu": 0, "silu": MOE_ACT_SILU, "relu": MOE_ACT_RELU}

# Every symbol declared in include/moeblaze.h.
EXPORTS = ("moe_strerror", "moe_last_error", "moe_route", "moe_build_index_workspace_size",
           "moe_build_index", "moe_build_index_noalloc", "moe_ffn_fwd_workspace_size", "moe_ffn_fwd", "moe_combine", "moe_ffn_bwd_workspace_size",
           "moe_ffn_bwd", "moe_ffn_recompute", "moe_ffn_fwd_combine_workspace_size",
           "moe_ffn_fwd_combine",
           "moe_ffn_bwd_combine_workspace_size", "moe_ffn_bwd_combine",
           "moe_route_bwd_workspace_size", "moe_route_bwd", "moe_probe_enable",
           "moe_probe_disable", "moe_probe_count", "moe_probe_dropped", "moe_probe_get")


class MoEError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__("%s: %s" % (_status_name(status), detail))
        self.status = status


_lib = None


def _status_name(s: int) -> str:
    return {0: "MOE_OK", -1: "MOE_ERR_INVALID_ARG", -2: "MOE_ERR_UNSUPPORTED",
            -3: "MOE_ERR_WORKSPACE", -4: "MOE_ERR_HIP"}.get(s, "status %d" % s)


def load_library(path: str = LIB):
    """Load libmoeblaze.so and declare the C signatures. Raises if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError("libmoeblaze.so is not built (%s); run "
                          "`python -m paper_2601_05296_amd.build`" % path)
    lib = ctypes.CDLL(path)
    P, I64, I, U, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_uint, ctypes.c_size_t
    sig = {
        "moe_strerror": (ctypes.c_char_p, [I]),
        "moe_last_error": (ctypes.c_char_p, []),
        "moe_route": (I, [P, P, P, I64, I, I, I, U, P, P, P, P]),
        "moe_build_index_workspace_size": (SZ, [I64, I, I]),
        "moe_build_index": (I, [P, I64, I, I, P, P, P, P, P, P, SZ, P]),
        "moe_build_index_noalloc": (I, [P, I64, I, I, P, P, P, P, P, P]),
        "moe_ffn_fwd_workspace_size": (SZ, [I64, I, I, I, I, U]),
        "moe_ffn_fwd": (I, [P, P, P, P, P, P, I64, I, I, I, I, U, P, P, P, P, SZ, P]),
        "moe_combine": (I, [P, P, P, I64, I, I, U, P, P]),
        "moe_ffn_bwd_workspace_size": (SZ, [I64, I, I, I, I, U]),
        "moe_ffn_bwd": (I, [P] * 11 + [I64, I, I, I, I, U] + [P] * 6 + [SZ, P]),
        "moe_ffn_recompute": (I, [P] * 5 + [I64, I, I, I, I, U, P, P, P]),
        "moe_ffn_fwd_combine_workspace_size": (SZ, [I64, I, I, I, I, U]),
        "moe_ffn_fwd_combine": (I, [P] * 8 + [I64, I, I, I, I, U] + [P] * 4 + [SZ, P]),
        "moe_ffn_bwd_combine_workspace_size": (SZ, [I64, I, I, I, I, U]),
        "moe_ffn_bwd_combine": (I, [P] * 12 + [I64, I, I, I, I, U] + [P] * 6 + [SZ, P]),
        "moe_route_bwd_workspace_size": (SZ, [I64, I, I, I, U]),
        "moe_route_bwd": (I, [P] * 6 + [I64, I, I, I, U, P, P, P, SZ, P]),
        "moe_probe_enable": (I, [I]),
        "moe_probe_disable": (None, []),
        "moe_probe_count": (I, []),
        "moe_probe_dropped": (I, []),
        "moe_probe_get": (I, [I, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_float)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _elt(flags: int):
    """Element type of the activation and weight tensors under `flags`."""
    return torch.float32 if flags & MOE_F32 else torch.bfloat16


def _gated(flags: int) -> bool:
    return not flags & (MOE_ACT_SILU | MOE_ACT_RELU)


def _need(t, n: int, name: str, dtype=None):
    """Check, before the library sees a bare pointer, that tensor `t` holds at
    least `n` elements of `dtype` (None or a raw address: not checked here)."""
    if t is None or isinstance(t, int):
        return
    if dtype is not None and t.dtype != dtype:
        raise ValueError("%s: dtype %s, expected %s" % (name, t.dtype, dtype))
    if t.numel() < n:
        raise ValueError("%s: %d elements, at least %d needed" % (name, t.numel(), n))


def _need_bytes(t, nbytes: int, name: str = "workspace"):
    if t is None or isinstance(t, int):
        return
    if t.numel() * t.element_size() < nbytes:
        raise ValueError("%s: %d bytes, workspace_bytes says %d" %
                         (name, t.numel() * t.element_size(), nbytes))


def _ffn_inputs(flags, T, d, f, E, k, x, w1, w3, w2, offsets, eti):
    el, S = _elt(flags), T * k
    _need(x, T * d, "x", el)
    _need(w1, E * d * f, "w1", el)
    if _gated(flags):
        _need(w3, E * d * f, "w3", el)
    if w2 is not None:
        _need(w2, E * f * d, "w2", el)
    _need(offsets, E + 1, "offsets", torch.int32)
    _need(eti, S, "expert_token_indices", torch.int32)


def _first_outputs(flags, T, f, k, A, B):
    _need(A, T * k * f, "A", _elt(flags))
    if _gated(flags):
        _need(B, T * k * f, "B", _elt(flags))


def _ffn_grads(flags, T, d, f, E, k, dy, gates, slot_src, dw1, dw3, dw2, d_gates):
    f32 = torch.float32
    _need(dy, T * d, "dy", _elt(flags))
    _need(gates, T * k, "gates", f32)
    _need(slot_src, T * k, "slot_src", torch.int32)
    _need(dw1, E * d * f, "dw1", f32)
    if _gated(flags):
        _need(dw3, E * d * f, "dw3", f32)
    _need(dw2, E * f * d, "dw2", f32)
    _need(d_gates, T * k, "d_gates", f32)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _check(status: int):
    if status != MOE_OK:
        raise MoEError(status, load_library().moe_last_error().decode())


def dtype_flag(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return MOE_BF16
    if t.dtype == torch.float32:
        return MOE_F32
    raise ValueError("unsupported dtype %s" % t.dtype)


def moe_route(x, w_gate, bias, T, d, E, k, flags, topk_ids, gates, logits, stream=None):
    _need(x, T * d, "x", _elt(flags))
    _need(w_gate, E * d, "w_gate", _elt(flags))
    _need(bias, E, "bias", torch.float32)
    _need(topk_ids, T * k, "topk_ids", torch.int32)
    _need(gates, T * k, "gates", torch.float32)
    _need(logits, T * E, "logits", torch.float32)
    _check(load_library().moe_route(_ptr(x), _ptr(w_gate), _ptr(bias), T, d, E, k, flags,
                                    _ptr(topk_ids), _ptr(gates), _ptr(logits), _stream(stream)))


def moe_build_index_workspace_size(T, E, k) -> int:
    return load_library().moe_build_index_workspace_size(T, E, k)


def moe_build_index(topk_ids, T, E, k, counts, offsets, expert_token_indices, token_index_map,
                    slot_src, workspace, workspace_bytes, stream=None):
    i32 = torch.int32
    _need(topk_ids, T * k, "topk_ids", i32)
    _need(counts, E, "counts", i32)
    _need(offsets, E + 1, "offsets", i32)
    _need(expert_token_indices, T * k, "expert_token_indices", i32)
    _need(token_index_map, T * k, "token_index_map", i32)
    _need(slot_src, T * k, "slot_src", i32)
    _need_bytes(workspace, workspace_bytes)
    _check(load_library().moe_build_index(_ptr(topk_ids), T, E, k, _ptr(counts), _ptr(offsets),
                                          _ptr(expert_token_indices), _ptr(token_index_map),
                                          _ptr(slot_src), _ptr(workspace), workspace_bytes,
                                          _stream(stream)))


def moe_build_index_noalloc(topk_ids, T, E, k, counts, offsets, expert_token_indices,
                            token_index_map, slot_src, stream=None):
    i32 = torch.int32
    _need(topk_ids, T * k, "topk_ids", i32)
    _need(counts, E, "counts", i32)
    _need(offsets, E + 1, "offsets", i32)
    _need(expert_token_indices, T * k, "expert_token_indices", i32)
    _need(token_index_map, T * k, "token_index_map", i32)
    _need(slot_src, T * k, "slot_src", i32)
    _check(load_library().moe_build_index_noalloc(_ptr(topk_ids), T, E, k, _ptr(counts),
                                                  _ptr(offsets), _ptr(expert_token_indices),
                                                  _ptr(token_index_map), _ptr(slot_src),
                                                  _stream(stream)))


def moe_ffn_fwd_workspace_size(T, d, f, E, k, flags) -> int:
    return load_library().moe_ffn_fwd_workspace_size(T, d, f, E, k, flags)


def moe_ffn_fwd(x, w1, w3, w2, offsets, expert_token_indices, T, d, f, E, k, flags, A, B, O,
                workspace, workspace_bytes, stream=None):
    _ffn_inputs(flags, T, d, f, E, k, x, w1, w3, w2, offsets, expert_token_indices)
    _first_outputs(flags, T, f, k, A, B)
    _need(O, T * k * d, "O", _elt(flags))
    _need_bytes(workspace, workspace_bytes)
    _check(load_library().moe_ffn_fwd(_ptr(x), _ptr(w1), _ptr(w3), _ptr(w2), _ptr(offsets),
                                      _ptr(expert_token_indices), T, d, f, E, k, flags, _ptr(A),
                                      _ptr(B), _ptr(O), _ptr(workspace), workspace_bytes,
                                      _stream(stream)))


def moe_ffn_recompute(x, w1, w3, offsets, expert_token_indices, T, d, f, E, k, flags, A, B,
                      stream=None):
    _ffn_inputs(flags, T, d, f, E, k, x, w1, w3, None, offsets, expert_token_indices)
    _first_outputs(flags, T, f, k, A, B)
    _check(load_library().moe_ffn_recompute(_ptr(x), _ptr(w1), _ptr(w3), _ptr(offsets),
                                            _ptr(expert_token_indices), T, d, f, E, k, flags,
                                            _ptr(A), _ptr(B), _stream(stream)))


def moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, flags) -> int:
    return load_library().moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, flags)


def moe_ffn_fwd_combine(x, w1, w3, w2, offsets, expert_token_indices, gates, token_index_map,
                        T, d, f, E, k, flags, A, B, y, workspace, workspace_bytes, stream=None):
    _ffn_inputs(flags, T, d, f, E, k, x, w1, w3, w2, offsets, expert_token_indices)
    _first_outputs(flags, T, f, k, A, B)
    _need(gates, T * k, "gates", torch.float32)
    _need(token_index_map, T * k, "token_index_map", torch.int32)
    _need(y, T * d, "y", _elt(flags))
    _need_bytes(workspace, workspace_bytes)
    _check(load_library().moe_ffn_fwd_combine(
        _ptr(x), _ptr(w1), _ptr(w3), _ptr(w2), _ptr(offsets), _ptr(expert_token_indices),
        _ptr(gates), _ptr(token_index_map), T, d, f, E, k, flags, _ptr(A), _ptr(B), _ptr(y),
        _ptr(workspace), workspace_bytes, _stream(stream)))


def moe_ffn_bwd_combine_workspace_size(T, d, f, E, k, flags) -> int:
    return load_library().moe_ffn_bwd_combine_workspace_size(T, d, f, E, k, flags)


def moe_ffn_bwd_combine(dy, x, w1, w3, w2, gates, offsets, expert_token_indices, slot_src,
                        token_index_map, A, B, T, d, f, E, k, flags, dw1, dw3, dw2, d_gates, dx,
                        workspace, workspace_bytes, stream=None):
    _ffn_inputs(flags, T, d, f, E, k, x, w1, w3, w2, offsets, expert_token_indices)
    _first_outputs(flags, T, f, k, A, B)
    _ffn_grads(flags, T, d, f, E, k, dy, gates, slot_src, dw1, dw3, dw2, d_gates)
    _need(token_index_map, T * k, "token_index_map", torch.int32)
    _need(dx, T * d, "dx", _elt(flags))
    _need_bytes(workspace, workspace_bytes)
    _check(load_library().moe_ffn_bwd_combine(
        _ptr(dy), _ptr(x), _ptr(w1), _ptr(w3), _ptr(w2), _ptr(gates), _ptr(offsets),
        _ptr(expert_token_indices), _ptr(slot_src), _ptr(token_index_map), _ptr(A), _ptr(B), T, d,
        f, E, k, flags, _ptr(dw1), _ptr(dw3), _ptr(dw2), _ptr(d_gates), _ptr(dx), _ptr(workspace),
        workspace_bytes, _stream(stream)))


def moe_combine(src, weights, token_index_map, T, d, k, flags, out, stream=None):
    _need(src, T * k * d, "src", _elt(flags))
    _need(weights, T * k, "weights", torch.float32)
    _need(token_index_map, T * k, "token_index_map", torch.int32)
    _need(out, T * d, "out", _elt(flags))
    _check(load_library().moe_combine(_ptr(src), _ptr(weights), _ptr(token_index_map), T, d, k,
                                      flags, _ptr(out), _stream(stream)))


def moe_ffn_bwd_workspace_size(T, d, f, E, k, flags) -> int:
    return load_library().moe_ffn_bwd_workspace_size(T, d, f, E, k, flags)


def moe_ffn_bwd(dy, x, w1, w3, w2, gates, offsets, expert_token_indices, slot_src, A, B, T, d,
                f, E, k, flags, dw1, dw3, dw2, d_gates, dX_slot, workspace, workspace_bytes,
                stream=None):
    _ffn_inputs(flags, T, d, f, E, k, x, w1, w3, w2, offsets, expert_token_indices)
    _first_outputs(flags, T, f, k, A, B)
    _ffn_grads(flags, T, d, f, E, k, dy, gates, slot_src, dw1, dw3, dw2, d_gates)
    _need(dX_slot, T * k * d, "dX_slot", _elt(flags))
    _need_bytes(workspace, workspace_bytes)
    _check(load_library().moe_ffn_bwd(_ptr(dy), _ptr(x), _ptr(w1), _ptr(w3), _ptr(w2),
                                      _ptr(gates), _ptr(offsets), _ptr(expert_token_indices),
                                      _ptr(slot_src), _ptr(A), _ptr(B), T, d, f, E, k, flags,
                                      _ptr(dw1), _ptr(dw3), _ptr(dw2), _ptr(d_gates),
                                      _ptr(dX_slot), _ptr(workspace), workspace_bytes,
                                      _stream(stream)))


def moe_route_bwd_workspace_size(T, d, E, k, flags) -> int:
    return load_library().moe_route_bwd_workspace_size(T, d, E, k, flags)


def moe_route_bwd(d_gates, logits, topk_ids, gates, x, w_gate, T, d, E, k, flags, dw_gate, dx,
                  workspace, workspace_bytes, stream=None):
    f32 = torch.float32
    _need(d_gates, T * k, "d_gates", f32)
    _need(logits, T * E, "logits", f32)
    _need(topk_ids, T * k, "topk_ids", torch.int32)
    _need(gates, T * k, "gates", f32)
    _need(x, T * d, "x", _elt(flags))
    _need(w_gate, E * d, "w_gate", _elt(flags))
    _need(dw_gate, E * d, "dw_gate", f32)
    _need(dx, T * d, "dx", _elt(flags))
    _need_bytes(workspace, workspace_bytes)
    _check(load_library().moe_route_bwd(_ptr(d_gates), _ptr(logits), _ptr(topk_ids),
                                        _ptr(gates), _ptr(x), _ptr(w_gate), T, d, E, k, flags,
                                        _ptr(dw_gate), _ptr(dx), _ptr(workspace),
                                        workspace_bytes, _stream(stream)))


def moe_probe_enable(capacity: int):
    _check(load_library().moe_probe_enable(capacity))


def moe_probe_disable():
    load_library().moe_probe_disable()


def moe_probe_count() -> int:
    return load_library().moe_probe_count()


def moe_probe_dropped() -> int:
    return load_library().moe_probe_dropped()


def moe_probe_get(index: int):
    """Returns (kernel name, milliseconds) of kernel record `index`."""
    name = ctypes.c_char_p()
    ms = ctypes.c_float()
    _check(load_library().moe_probe_get(index, ctypes.byref(name), ctypes.byref(ms)))
    return name.value.decode(), ms.value
