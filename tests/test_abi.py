"""CPU checks of the C ABI: the built library exports every function the
header declares, and argument validation rejects bad calls before touching
the GPU (no kernel is launched in these tests)."""
import os
import re

import pytest

from paper_2601_05296_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moeblaze.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_]+)\s*\(", src)))


def test_header_and_binding_agree():
    assert sorted(B.EXPORTS) == _declared()


def test_library_exports_every_declared_symbol():
    lib = B.load_library()
    for name in _declared():
        assert hasattr(lib, name), name


def test_status_strings():
    lib = B.load_library()
    for code, name in ((0, b"MOE_OK"), (-1, b"MOE_ERR_INVALID_ARG"), (-2, b"MOE_ERR_UNSUPPORTED"),
                       (-3, b"MOE_ERR_WORKSPACE"), (-4, b"MOE_ERR_HIP")):
        assert lib.moe_strerror(code) == name


FAKE = 1 << 20  # an aligned non-null address that is never dereferenced


@pytest.mark.parametrize("args,status", [
    (dict(T=10, d=128, E=8, k=9), B.MOE_ERR_INVALID_ARG),    # k > E
    (dict(T=10, d=128, E=8, k=0), B.MOE_ERR_INVALID_ARG),
    (dict(T=-1, d=128, E=8, k=2), B.MOE_ERR_INVALID_ARG),
    (dict(T=10, d=100, E=8, k=2), B.MOE_ERR_UNSUPPORTED),    # d % 64
    (dict(T=10, d=96, E=8, k=2), B.MOE_ERR_UNSUPPORTED),     # d % 64
    (dict(T=10, d=128, E=300, k=2), B.MOE_ERR_UNSUPPORTED),  # E > 256
    (dict(T=10, d=128, E=64, k=17), B.MOE_ERR_UNSUPPORTED),  # k > 16
    (dict(T=1 << 30, d=128, E=64, k=8), B.MOE_ERR_UNSUPPORTED),  # T*k >= 2^31
])
def test_route_validation(args, status):
    lib = B.load_library()
    r = lib.moe_route(FAKE, FAKE, None, args["T"], args["d"], args["E"], args["k"], 0, FAKE, FAKE,
                      None, None)
    assert r == status, lib.moe_last_error()


def test_null_and_misaligned_pointers():
    lib = B.load_library()
    assert lib.moe_route(None, FAKE, None, 10, 128, 8, 2, 0, FAKE, FAKE, None, None) == B.MOE_ERR_INVALID_ARG
    assert b"x is NULL" in lib.moe_last_error()
    assert lib.moe_route(FAKE + 2, FAKE, None, 10, 128, 8, 2, 0, FAKE, FAKE, None, None) == B.MOE_ERR_INVALID_ARG
    assert b"aligned" in lib.moe_last_error()
    assert lib.moe_combine(FAKE, None, FAKE, 10, 128, 2, B.MOE_RENORM, FAKE, None) == B.MOE_ERR_INVALID_ARG
    assert lib.moe_route(FAKE, FAKE, None, 10, 128, 8, 2, 0x100, FAKE, FAKE, None, None) == B.MOE_ERR_INVALID_ARG
    assert b"unknown flag" in lib.moe_last_error()


def test_workspace_checks_and_zero_tokens():
    lib = B.load_library()
    need = lib.moe_build_index_workspace_size(1000, 8, 2)
    assert need > 0
    r = lib.moe_build_index(FAKE, 1000, 8, 2, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need - 1, None)
    assert r == B.MOE_ERR_WORKSPACE
    r = lib.moe_ffn_bwd(*([FAKE] * 11), 1000, 128, 128, 8, 2, 0, *([FAKE] * 6), 0, None)
    assert r == B.MOE_ERR_WORKSPACE
    need = lib.moe_route_bwd_workspace_size(1000, 128, 8, 2, 0)
    r = lib.moe_route_bwd(*([FAKE] * 6), 1000, 128, 8, 2, 0, FAKE, FAKE, FAKE, need - 16, None)
    assert r == B.MOE_ERR_WORKSPACE
    # T == 0: no-op success, pointers not even inspected
    assert lib.moe_ffn_fwd(*([None] * 6), 0, 128, 128, 8, 2, 0, None, None, None, None, 0,
                           None) == B.MOE_OK
    need = lib.moe_ffn_fwd_workspace_size(1000, 128, 128, 8, 2, 0)
    r = lib.moe_ffn_fwd(*([FAKE] * 6), 1000, 128, 128, 8, 2, 0, FAKE, FAKE, FAKE, FAKE, need - 1, None)
    assert r == B.MOE_ERR_WORKSPACE
    assert lib.moe_build_index_workspace_size(0, 8, 2) == 0


def test_h_on_load_flag():
    lib = B.load_library()
    T, d, f, E, k = 1000, 256, 384, 8, 2
    S = T * k
    h = (S * f * 2 + 255) // 256 * 256
    for fl in (0, B.MOE_ACT_SILU, B.MOE_ACT_RELU):
        # the forward workspace drops exactly the bf16 h buffer
        assert lib.moe_ffn_fwd_workspace_size(T, d, f, E, k, fl) - \
            lib.moe_ffn_fwd_workspace_size(T, d, f, E, k, fl | B.MOE_H_ON_LOAD) == h
        assert lib.moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, fl) - \
            lib.moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, fl | B.MOE_H_ON_LOAD) == h
    # the backward drops g*h (the dX strip of the combined call may be larger)
    for fl in (0, B.MOE_ACT_SILU):
        assert lib.moe_ffn_bwd_workspace_size(T, d, f, E, k, fl) - \
            lib.moe_ffn_bwd_workspace_size(T, d, f, E, k, fl | B.MOE_H_ON_LOAD) >= h - (S + 64) * 4 - 256
        assert lib.moe_ffn_bwd_combine_workspace_size(T, d, f, E, k, fl | B.MOE_H_ON_LOAD) <= \
            lib.moe_ffn_bwd_combine_workspace_size(T, d, f, E, k, fl)
    # float32 debug mode buffers no h either way
    assert lib.moe_ffn_fwd_workspace_size(T, d, f, E, k, B.MOE_F32 | B.MOE_H_ON_LOAD) == \
        lib.moe_ffn_fwd_workspace_size(T, d, f, E, k, B.MOE_F32)
    # without h the separate forward needs no workspace at all
    assert lib.moe_ffn_fwd_workspace_size(T, d, f, E, k, B.MOE_H_ON_LOAD) == 0
    # the FFN calls accept it (here a short workspace stops the call before any launch)
    r = lib.moe_ffn_fwd_combine(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, T, d, f, E, k,
                                B.MOE_H_ON_LOAD, FAKE, FAKE, FAKE, FAKE, 16, None)
    assert r == B.MOE_ERR_WORKSPACE, lib.moe_last_error()
    # the other calls reject it
    assert lib.moe_combine(FAKE, None, FAKE, 10, 128, 2, B.MOE_H_ON_LOAD, FAKE, None) == \
        B.MOE_ERR_INVALID_ARG
    assert lib.moe_route(FAKE, FAKE, None, 10, 128, 8, 2, B.MOE_H_ON_LOAD, FAKE, FAKE, None,
                         None) == B.MOE_ERR_INVALID_ARG


def test_accumulate_dw_flag():
    lib = B.load_library()
    T, d, f, E, k = 1000, 256, 384, 8, 2
    fl = B.MOE_ACCUMULATE_DW
    # the backward calls accept it (a short workspace stops them before any launch)
    r = lib.moe_ffn_bwd(*([FAKE] * 11), T, d, f, E, k, fl, *([FAKE] * 6), 16, None)
    assert r == B.MOE_ERR_WORKSPACE, lib.moe_last_error()
    r = lib.moe_ffn_bwd_combine(*([FAKE] * 12), T, d, f, E, k, fl, *([FAKE] * 6), 16, None)
    assert r == B.MOE_ERR_WORKSPACE, lib.moe_last_error()
    # the forward, the recompute and the other calls reject it
    r = lib.moe_ffn_fwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, T, d, f, E, k, fl, FAKE, FAKE, FAKE,
                        FAKE, 1 << 40, None)
    assert r == B.MOE_ERR_INVALID_ARG
    assert lib.moe_ffn_recompute(FAKE, FAKE, FAKE, FAKE, FAKE, T, d, f, E, k, fl, FAKE, FAKE,
                                 None) == B.MOE_ERR_INVALID_ARG
    assert lib.moe_combine(FAKE, None, FAKE, 10, 128, 2, fl, FAKE, None) == B.MOE_ERR_INVALID_ARG
    assert lib.moe_route(FAKE, FAKE, None, 10, 128, 8, 2, fl, FAKE, FAKE, None,
                         None) == B.MOE_ERR_INVALID_ARG


def test_activation_flags():
    lib = B.load_library()
    S, f = 1000 * 2, 128
    # both activation flags at once
    r = lib.moe_ffn_fwd(FAKE, FAKE, None, FAKE, FAKE, FAKE, 1000, 128, f, 8, 2,
                        B.MOE_ACT_SILU | B.MOE_ACT_RELU, FAKE, None, FAKE, FAKE, 1 << 30, None)
    assert r == B.MOE_ERR_INVALID_ARG and b"both" in lib.moe_last_error()
    # the activation flags belong to the FFN calls only
    assert lib.moe_combine(FAKE, None, FAKE, 10, 128, 2, B.MOE_ACT_RELU, FAKE, None) == B.MOE_ERR_INVALID_ARG
    assert lib.moe_route(FAKE, FAKE, None, 10, 128, 8, 2, B.MOE_ACT_SILU, FAKE, FAKE, None,
                         None) == B.MOE_ERR_INVALID_ARG
    # SwiGLU needs w3 and B; a non-gated expert accepts NULL for them (a short
    # workspace then stops the call before any launch)
    r = lib.moe_ffn_fwd(FAKE, FAKE, None, FAKE, FAKE, FAKE, 1000, 128, f, 8, 2, 0, FAKE, FAKE,
                        FAKE, FAKE, 1 << 30, None)
    assert r == B.MOE_ERR_INVALID_ARG and b"w3 is NULL" in lib.moe_last_error()
    for act in (B.MOE_ACT_SILU, B.MOE_ACT_RELU):
        r = lib.moe_ffn_fwd(FAKE, FAKE, None, FAKE, FAKE, FAKE, 1000, 128, f, 8, 2, act, FAKE,
                            None, FAKE, FAKE, 16, None)
        assert r == B.MOE_ERR_WORKSPACE, lib.moe_last_error()
        r = lib.moe_ffn_bwd(*([FAKE] * 3), None, FAKE, *([FAKE] * 5), None, 1000, 128, f, 8, 2,
                            act, FAKE, None, FAKE, FAKE, FAKE, FAKE, 16, None)
        assert r == B.MOE_ERR_WORKSPACE, lib.moe_last_error()
    # the non-gated workspaces hold the same buffers (h; partials and g*h)
    assert lib.moe_ffn_fwd_workspace_size(1000, 128, f, 8, 2, B.MOE_ACT_SILU) == \
        lib.moe_ffn_fwd_workspace_size(1000, 128, f, 8, 2, 0) >= S * f * 2



def test_binding_checks_sizes_and_dtypes_before_the_library():
    """The C ABI takes bare pointers; the binding checks element counts and
    dtypes first (here on host tensors, so nothing reaches the library)."""
    import torch
    bf, f32, i32 = torch.bfloat16, torch.float32, torch.int32
    T, d, E, k, f = 10, 128, 8, 2, 256

    def z(n, dt):
        return torch.zeros(n, dtype=dt)

    with pytest.raises(ValueError, match="w_gate: 1016 elements"):
        B.moe_route(z(T * d, bf), z(E * d - 8, bf), None, T, d, E, k, 0, z(T * k, i32),
                    z(T * k, f32), None)
    with pytest.raises(ValueError, match="topk_ids: dtype torch.int64"):
        B.moe_route(z(T * d, bf), z(E * d, bf), None, T, d, E, k, 0,
                    z(T * k, torch.int64), z(T * k, f32), None)
    with pytest.raises(ValueError, match="x: dtype torch.bfloat16"):   # MOE_F32 wants float32
        B.moe_route(z(T * d, bf), z(E * d, bf), None, T, d, E, k, B.MOE_F32,
                    z(T * k, i32), z(T * k, f32), None)
    with pytest.raises(ValueError, match="src: 2559 elements"):
        B.moe_combine(z(T * k * d - 1, bf), None, z(T * k, i32), T, d, k, 0, z(T * d, bf))
    with pytest.raises(ValueError, match="workspace: 16 bytes"):
        B.moe_build_index(z(T * k, i32), T, E, k, z(E, i32), z(E + 1, i32), z(T * k, i32),
                          z(T * k, i32), z(T * k, i32), z(16, torch.uint8), 64)
    with pytest.raises(ValueError, match="B: 0 elements"):   # SwiGLU needs B
        B.moe_ffn_fwd(z(T * d, bf), z(E * d * f, bf), z(E * d * f, bf), z(E * f * d, bf),
                      z(E + 1, i32), z(T * k, i32), T, d, f, E, k, 0, z(T * k * f, bf),
                      z(0, bf), z(T * k * d, bf), None, 0)
    # non-gated: w3 and B are not needed; every size is right, so the next
    # check (device placement) is the one that fails
    with pytest.raises(ValueError, match="must be on the GPU"):
        B.moe_ffn_fwd(z(T * d, bf), z(E * d * f, bf), None, z(E * f * d, bf), z(E + 1, i32),
                      z(T * k, i32), T, d, f, E, k, B.MOE_ACT_RELU, z(T * k * f, bf), None,
                      z(T * k * d, bf), None, 0)


def test_atomic_combine_flag():
    lib = B.load_library()
    T, d, f, E, k = 1000, 256, 384, 8, 2
    S = T * k
    gs = (S * 4 + 255) // 256 * 256
    for fl in (0, B.MOE_H_ON_LOAD, B.MOE_ACT_SILU | B.MOE_H_ON_LOAD):
        # the forward holds the slot gates instead of a strip of the expert output
        plain = lib.moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, fl)
        atomic = lib.moe_ffn_fwd_combine_workspace_size(T, d, f, E, k, fl | B.MOE_ATOMIC_COMBINE)
        assert plain - atomic > 0
        assert atomic == lib.moe_ffn_fwd_workspace_size(T, d, f, E, k, fl) + gs
        # the backward drops its dX strip: what is left is the separate call's workspace
        assert lib.moe_ffn_bwd_combine_workspace_size(T, d, f, E, k, fl | B.MOE_ATOMIC_COMBINE) == \
            lib.moe_ffn_bwd_workspace_size(T, d, f, E, k, fl)
    fl = B.MOE_ATOMIC_COMBINE
    # the combined calls accept it (a short workspace stops them before any launch)
    r = lib.moe_ffn_fwd_combine(*([FAKE] * 8), T, d, f, E, k, fl, *([FAKE] * 4), 16, None)
    assert r == B.MOE_ERR_WORKSPACE, lib.moe_last_error()
    r = lib.moe_ffn_bwd_combine(*([FAKE] * 12), T, d, f, E, k, fl, *([FAKE] * 6), 16, None)
    assert r == B.MOE_ERR_WORKSPACE, lib.moe_last_error()
    # bf16 only
    r = lib.moe_ffn_fwd_combine(*([FAKE] * 8), T, d, f, E, k, fl | B.MOE_F32, *([FAKE] * 4),
                                1 << 40, None)
    assert r == B.MOE_ERR_UNSUPPORTED, lib.moe_last_error()
    r = lib.moe_ffn_bwd_combine(*([FAKE] * 12), T, d, f, E, k, fl | B.MOE_F32, *([FAKE] * 6),
                                1 << 40, None)
    assert r == B.MOE_ERR_UNSUPPORTED, lib.moe_last_error()
    # the separate FFN calls, the recompute and the other calls reject it
    r = lib.moe_ffn_fwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, T, d, f, E, k, fl, FAKE, FAKE, FAKE,
                        FAKE, 1 << 40, None)
    assert r == B.MOE_ERR_INVALID_ARG
    r = lib.moe_ffn_bwd(*([FAKE] * 11), T, d, f, E, k, fl, *([FAKE] * 6), 1 << 40, None)
    assert r == B.MOE_ERR_INVALID_ARG
    assert lib.moe_ffn_recompute(FAKE, FAKE, FAKE, FAKE, FAKE, T, d, f, E, k, fl, FAKE, FAKE,
                                 None) == B.MOE_ERR_INVALID_ARG
    assert lib.moe_combine(FAKE, None, FAKE, 10, 128, 2, fl, FAKE, None) == B.MOE_ERR_INVALID_ARG
    assert lib.moe_route(FAKE, FAKE, None, 10, 128, 8, 2, fl, FAKE, FAKE, None,
                         None) == B.MOE_ERR_INVALID_ARG
