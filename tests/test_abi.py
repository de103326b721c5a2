"""The C ABI without a GPU: libmoe.so loads, exports every function that
include/moe.h declares, and rejects bad arguments synchronously (these calls
return before any device work is enqueued)."""
import ctypes
import os
import re

import pytest

from paper_2205_01848_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe.h")

EINVAL, EWORKSPACE = 1, 4


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ["moe_gate_topk", "moe_dispatch", "moe_update_capacity", "moe_expert_ffn_fwd",
                     "moe_expert_ffn_bwd", "moe_combine", "moe_combine_bwd", "moe_gate_bwd",
                     "moe_dispatch_bwd", "moe_count"]:
        assert required in names


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert name in B.SIGNATURES, f"binding lacks {name}"
    assert lib.moe_abi_version() == B.ABI_VERSION == 7
    assert lib.moe_status_string(0) == b"MOE_OK"


def test_set_gemm_tiles_accepts_three_modes():
    for mode in (1, 2, 0):
        B.moe_set_gemm_tiles(mode)
    for bad in (-1, 3, 100):
        assert B.lib().moe_set_gemm_tiles(bad) == EINVAL
    B.moe_set_gemm_tiles(0)


def test_dx_weight_copy_modes_and_workspace():
    """The workspace query includes the transposed copy of [W1; W3] (E d F
    bf16 elements) exactly when the mode would make it: automatically from
    8192 rows per expert, never under mode 1, always under mode 2, and never
    for float32 layers."""
    BF16, F32, SWIGLU, RELU = 1, 0, 2, 0
    q = B.lib().moe_ffn_bwd_workspace_bytes
    E, d, f = 4, 256, 512
    try:
        for act, F in ((SWIGLU, 2 * f), (RELU, f)):
            copy = E * d * F * 2
            B.moe_set_dx_weight_copy(1)
            small, big = q(BF16, act, E, d, f, 8192 * E - 1), q(BF16, act, E, d, f, 8192 * E)
            B.moe_set_dx_weight_copy(0)
            assert q(BF16, act, E, d, f, 8192 * E - 1) == small
            assert copy <= q(BF16, act, E, d, f, 8192 * E) - big < copy + 512
            B.moe_set_dx_weight_copy(2)
            assert copy <= q(BF16, act, E, d, f, 8192 * E - 1) - small < copy + 512
            f32 = [q(F32, act, E, d, f, 8192 * E)]
            B.moe_set_dx_weight_copy(1)
            assert q(F32, act, E, d, f, 8192 * E) == f32[0]
        for bad in (-1, 3):
            assert B.lib().moe_set_dx_weight_copy(bad) == EINVAL
    finally:
        B.moe_set_dx_weight_copy(0)


def test_binding_refuses_a_library_of_another_abi(monkeypatch):
    # the binding sizes buffers for its own ABI: an older or newer library
    # must not be called through it
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "ABI_VERSION", B.ABI_VERSION - 1)
    with pytest.raises(B.MoEError, match="ABI version"):
        B.lib()
    monkeypatch.setattr(B, "_lib", None)


FAKE = ctypes.c_void_p(1 << 20)   # never dereferenced: every call below fails validation


@pytest.mark.parametrize("args", [
    (1, -1, 64, 4, 1, 0),      # T < 0
    (1, 16, 60, 4, 1, 0),      # d not a multiple of 8
    (1, 16, 64, 65, 1, 0),     # E > 64
    (1, 16, 64, 4, 5, 0),      # k > E
    (1, 16, 64, 16, 9, 0),     # k > 8
    (7, 16, 64, 4, 1, 0),      # bad dtype
])
def test_gate_rejects_bad_shapes(args):
    dt, T, d, E, k, renorm = args
    L = B.lib()
    st = L.moe_gate_topk(None, dt, T, d, E, k, renorm, FAKE, FAKE, None, FAKE, FAKE, FAKE)
    assert st == EINVAL


def test_gate_rejects_null_and_misaligned():
    L = B.lib()
    assert L.moe_gate_topk(None, 1, 16, 64, 4, 1, 0, None, FAKE, None, FAKE, FAKE, FAKE) == EINVAL
    odd = ctypes.c_void_p((1 << 20) + 2)
    assert L.moe_gate_topk(None, 1, 16, 64, 4, 1, 0, odd, FAKE, None, FAKE, FAKE, FAKE) == EINVAL


def test_capacity_and_count_reject_bad_arguments():
    L = B.lib()
    assert L.moe_update_capacity(None, 10, 1, 4, None, 0, 1, 0, 1, FAKE, FAKE) == EINVAL   # num < 1
    assert L.moe_update_capacity(None, 10, 1, 4, None, 1, 0, 0, 1, FAKE, FAKE) == EINVAL   # den < 1
    assert L.moe_update_capacity(None, 10, 1, 4, None, 1, 1, -1, 1, FAKE, FAKE) == EINVAL  # cap_min
    assert L.moe_update_capacity(None, 10, 1, 4, None, 1, 1, 0, 1, None, FAKE) == EINVAL
    assert L.moe_update_capacity(None, 10, 1, 4, None, 1, 1, 0, 0, FAKE, FAKE) == EINVAL   # row_align
    assert L.moe_update_capacity(None, 10, 1, 4, None, 1, 1, 0, 1025, FAKE, FAKE) == EINVAL
    assert L.moe_count(None, 10, 4, 1, FAKE, None, FAKE) == EINVAL


def test_dispatch_workspace_and_arguments():
    L = B.lib()
    need = L.moe_dispatch_workspace_bytes(1000, 8, 2)
    assert need > 0
    assert L.moe_dispatch_workspace_bytes(1000, 8, 9) == 0
    args = [None, 1, 1000, 64, 8, 2, FAKE, FAKE, FAKE, FAKE, 2000, FAKE, FAKE, FAKE, FAKE, FAKE,
            FAKE]
    assert L.moe_dispatch(*args, FAKE, need - 1) == EWORKSPACE
    assert L.moe_dispatch(*args, None, need) == EWORKSPACE
    bad_rows = list(args)
    bad_rows[10] = -5
    assert L.moe_dispatch(*bad_rows, FAKE, need) == EINVAL


def test_ffn_workspace_queries_and_arguments():
    L = B.lib()
    for act in (0, 1, 2):
        fw = L.moe_ffn_fwd_workspace_bytes(1, act, 8, 256, 512, 5000)
        bw = L.moe_ffn_bwd_workspace_bytes(1, act, 8, 256, 512, 5000)
        assert 0 < fw < bw
    assert L.moe_ffn_fwd_workspace_bytes(1, 3, 8, 256, 512, 5000) == 0          # bad act
    assert L.moe_ffn_fwd_workspace_bytes(1, 0, 8, 250, 512, 5000) == 0          # d % 8
    need = L.moe_ffn_fwd_workspace_bytes(1, 2, 8, 256, 512, 5000)
    base = [None, 1, 2, 8, 256, 512, FAKE, FAKE, 5000, FAKE, FAKE]
    # SwiGLU without w3
    assert L.moe_expert_ffn_fwd(*base, None, FAKE, None, FAKE, FAKE, need) == EINVAL
    assert L.moe_expert_ffn_fwd(*base, FAKE, FAKE, None, FAKE, FAKE, need - 1) == EWORKSPACE
    needb = L.moe_ffn_bwd_workspace_bytes(1, 0, 8, 256, 512, 5000)
    assert L.moe_expert_ffn_bwd(None, 1, 0, 8, 256, 512, FAKE, FAKE, 5000, FAKE, FAKE, FAKE, None,
                                FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, needb - 1) == EWORKSPACE


def test_combine_and_backward_reject_bad_arguments():
    L = B.lib()
    assert L.moe_combine(None, 1, 10, 64, 0, 100, FAKE, FAKE, FAKE, FAKE) == EINVAL      # k = 0
    assert L.moe_combine_bwd(None, 1, 10, 64, 2, 100, None, FAKE, FAKE, FAKE, FAKE,
                             FAKE) == EINVAL
    # dlogits without w_g
    assert L.moe_dispatch_bwd(None, 1, 10, 64, 4, 2, 100, FAKE, FAKE, FAKE, None, FAKE) == EINVAL
    assert L.moe_gate_bwd_workspace_bytes(100, 64, 4) > 0
    assert L.moe_gate_bwd(None, 1, 100, 64, 4, 2, 1, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE,
                          FAKE, 0) == EWORKSPACE


def test_loss_operators_reject_bad_arguments():
    L = B.lib()
    need = L.moe_balance_workspace_bytes(1000, 8)
    assert need >= 4 * 8 * 4       # four 256-token partials of 8 experts
    assert L.moe_balance_workspace_bytes(1000, 65) == 0
    assert L.moe_balance_fwd(None, 1000, 8, 2, ctypes.c_float(-0.1), FAKE, FAKE, FAKE, FAKE, FAKE,
                             need) == EINVAL
    assert L.moe_balance_fwd(None, 1000, 8, 2, ctypes.c_float(float("nan")), FAKE, FAKE, FAKE,
                             FAKE, FAKE, need) == EINVAL
    assert L.moe_balance_fwd(None, 1000, 8, 2, ctypes.c_float(float("inf")), FAKE, FAKE, FAKE,
                             FAKE, FAKE, need) == EINVAL
    assert L.moe_balance_fwd(None, 1000, 8, 2, ctypes.c_float(0.01), FAKE, FAKE, FAKE, FAKE, FAKE,
                             need - 1) == EWORKSPACE
    assert L.moe_aggregate_spec(None, 1, 10, 64, 0, FAKE, FAKE, 100, FAKE) == EINVAL      # k = 0
    assert L.moe_aggregate_spec(None, 1, 10, 60, 2, FAKE, FAKE, 100, FAKE) == EINVAL      # d % 8
    wsl = L.moe_spec_loss_workspace_bytes(10)
    assert L.moe_spec_loss(None, 1, 10, 64, 2, FAKE, FAKE, FAKE, FAKE, 100, FAKE, FAKE, FAKE,
                           FAKE, wsl - 1) == EWORKSPACE
    assert L.moe_spec_loss(None, 1, 10, 64, 2, FAKE, FAKE, FAKE, None, 100, FAKE, FAKE, FAKE,
                           FAKE, wsl) == EINVAL                                            # target


def test_cache_operators_reject_bad_arguments():
    L = B.lib()
    assert L.moe_cache_update(None, 10, 9, FAKE, FAKE, FAKE, FAKE) == EINVAL             # k > 8
    assert L.moe_cache_update(None, 10, 2, FAKE, FAKE, FAKE, None) == EINVAL
    assert L.moe_cached_weights(None, 10, 65, 2, 1, FAKE, FAKE, FAKE) == EINVAL           # E > 64
    assert L.moe_cached_weights(None, 10, 8, 2, 1, None, FAKE, FAKE) == EINVAL
    assert L.moe_caching_decision(0, 5, 4, 20, 96, 100, 90, 100, 10) == -1               # u > n
    assert L.moe_caching_decision(0, 5, 10, 20, 96, 0, 90, 100, 10) == -1                # den 0


def test_policy_rejects_bad_arguments():
    L = B.lib()
    init = (ctypes.c_int32 * 4)(5, 5, 5, 5)
    h = ctypes.c_void_p()
    # grow above shrink, negative delta, bad ratio, negative initial capacity
    assert L.moe_policy_create(100, 2, 4, 1, 14, 10, 13, 10, 0, 1, init, ctypes.byref(h)) == EINVAL
    assert L.moe_policy_create(100, 2, 4, -1, 11, 10, 13, 10, 0, 1, init, ctypes.byref(h)) == EINVAL
    assert L.moe_policy_create(100, 2, 4, 1, 0, 10, 13, 10, 0, 1, init, ctypes.byref(h)) == EINVAL
    neg = (ctypes.c_int32 * 4)(5, -1, 5, 5)
    assert L.moe_policy_create(100, 2, 4, 1, 11, 10, 13, 10, 0, 1, neg, ctypes.byref(h)) == EINVAL
    assert L.moe_policy_create(100, 2, 4, 1, 11, 10, 13, 10, 0, 0, init, ctypes.byref(h)) == EINVAL  # row_align
    assert not h.value
    assert L.moe_policy_begin(None, None, FAKE, FAKE, None, None) == EINVAL
    assert L.moe_policy_end(None, None, FAKE) == EINVAL
