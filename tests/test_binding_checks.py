"""The Python binding refuses, before any device call, a tensor smaller than
the buffer the C entry point reads or writes, or of the wrong element type.
The C ABI takes bare pointers, so an undersized tensor would otherwise be
accessed past its end on the device.  Runs on the CPU: the checks come before
any device access, so CPU tensors of the right size get past them and fail
only where the call first needs the device (its stream, or a device pointer)."""
import pytest
import torch

from paper_2205_01848_amd import binding as B

bf16, f32, i32 = torch.bfloat16, torch.float32, torch.int32


def z(n, dt):
    return torch.zeros(n, dtype=dt)


def passes_checks(fn, **kw):
    """fn(**kw) gets past the size and type checks: it fails only for want of
    a device."""
    with pytest.raises((B.MoEError, RuntimeError)) as e:
        fn(**kw)
    msg = str(e.value)
    assert "device memory" in msg or "GPU" in msg, msg


def _ffn_fwd_args(E=2, f=16, d=8, R=32, act=B.MOE_SWIGLU, planes=3):
    w1 = torch.zeros(E, f, d, dtype=bf16)
    return dict(act=act, offsets=z(E + 1, i32), rows=z(E, i32), x_disp=torch.zeros(R, d, dtype=bf16),
                w1=w1, w3=torch.zeros_like(w1), w2=torch.zeros(E, d, f, dtype=bf16),
                h_save=z(planes * R * f, bf16), y_disp=torch.zeros(R, d, dtype=bf16), ws=z(256, torch.uint8))


def test_sizes_that_fit_reach_the_device_check():
    passes_checks(B.moe_expert_ffn_fwd, **_ffn_fwd_args())


def test_swiglu_h_save_needs_three_planes():
    with pytest.raises(B.MoEError, match="h_save holds"):
        B.moe_expert_ffn_fwd(**_ffn_fwd_args(planes=2))
    # GELU keeps H and A, ReLU only A
    a = _ffn_fwd_args(act=B.MOE_GELU_TANH, planes=2)
    a["w3"] = None
    passes_checks(B.moe_expert_ffn_fwd, **a)
    with pytest.raises(B.MoEError, match="h_save holds"):
        B.moe_expert_ffn_fwd(**dict(a, h_save=z(1 * 32 * 16, bf16)))
    a = _ffn_fwd_args(act=B.MOE_RELU, planes=1)
    a["w3"] = None
    passes_checks(B.moe_expert_ffn_fwd, **a)


def test_required_and_optional_operands():
    a = _ffn_fwd_args()
    a["w3"] = None
    with pytest.raises(B.MoEError, match="w3 is required"):
        B.moe_expert_ffn_fwd(**a)
    a = _ffn_fwd_args()
    a["h_save"] = None                                   # inference: no saved planes
    passes_checks(B.moe_expert_ffn_fwd, **a)


def test_element_types():
    T, d, E, k = 10, 8, 4, 2
    x = torch.zeros(T, d, dtype=bf16)
    with pytest.raises(B.MoEError, match="ids: element type"):
        B.moe_gate_topk(x, torch.zeros(E, d, dtype=bf16), None, k, 1, z(T * E, f32),
                        torch.zeros(T, k, dtype=torch.int64), z(T * k, f32))
    with pytest.raises(B.MoEError, match="w_g: element type"):
        B.moe_gate_topk(x, torch.zeros(E, d, dtype=f32), None, k, 1, z(T * E, f32),
                        z(T * k, i32), z(T * k, f32))
    with pytest.raises(B.MoEError, match="y_disp: element type"):
        B.moe_combine(torch.zeros(5, d, dtype=f32), torch.zeros(T, k, dtype=i32), z(T * k, f32),
                      torch.zeros(T, d, dtype=bf16))


def test_undersized_outputs():
    T, d, E, k, R = 10, 8, 4, 2, 12
    x = torch.zeros(T, d, dtype=bf16)
    ids = torch.zeros(T, k, dtype=i32)
    good = dict(capacity=z(E, i32), offsets=z(E + 1, i32), rows_alloc=R, counts=z(E, i32),
                fill=z(E, i32), dest_row=z(T * k, i32), src=z(R, i32),
                x_disp=z(R * d, bf16), status=z(1, i32), ws=z(256, torch.uint8))
    passes_checks(B.moe_dispatch, x=x, ids=ids, E=E, **good)
    for name, short in (("x_disp", z(R * d - 1, bf16)), ("src", z(R - 1, i32)),
                        ("offsets", z(E, i32)), ("dest_row", z(T * k - 1, i32))):
        bad = dict(good, **{name: short})
        with pytest.raises(B.MoEError, match=f"{name} holds"):
            B.moe_dispatch(x, ids, E, **bad)


def test_backward_operands():
    E, f, d, R = 2, 16, 8, 32
    a = _ffn_fwd_args(E, f, d, R)
    kw = dict(act=a["act"], offsets=a["offsets"], rows=a["rows"], x_disp=a["x_disp"],
              h_save=a["h_save"], w1=a["w1"], w3=a["w3"], w2=a["w2"], dy_disp=a["y_disp"],
              dx_disp=torch.zeros(R, d, dtype=bf16), dw1=z(E * f * d, f32), dw3=z(E * f * d, f32),
              dw2=z(E * d * f, f32), ws=a["ws"])
    passes_checks(B.moe_expert_ffn_bwd, **kw)
    with pytest.raises(B.MoEError, match="dw3 is required"):
        B.moe_expert_ffn_bwd(**dict(kw, dw3=None))
    with pytest.raises(B.MoEError, match="dw2: element type"):
        B.moe_expert_ffn_bwd(**dict(kw, dw2=z(E * d * f, bf16)))
    with pytest.raises(B.MoEError, match="h_save is required"):
        B.moe_expert_ffn_bwd(**dict(kw, h_save=None))


def test_loss_and_cache_operands():
    T, d, E, k, R = 6, 8, 4, 2, 12
    with pytest.raises(B.MoEError, match="dprob_coef holds"):
        B.moe_balance_fwd(torch.zeros(T, E, dtype=f32), z(E, i32), k, 0.1, z(1, f32),
                          z(E - 1, f32), z(256, torch.uint8))
    with pytest.raises(B.MoEError, match="out holds"):
        B.moe_aggregate_spec(torch.zeros(R, d, dtype=bf16), torch.zeros(T, k, dtype=i32),
                             torch.zeros(T * k - 1, d, dtype=bf16))
    with pytest.raises(B.MoEError, match="cache_out holds"):
        B.moe_cache_update(torch.zeros(T, k, dtype=i32), z(T * k, i32), z(T * k - 1, i32),
                           z(1, i32))
    with pytest.raises(B.MoEError, match="weights holds"):
        B.moe_cached_weights(torch.zeros(T, E, dtype=f32), torch.zeros(T, k, dtype=i32), 1,
                             z(T * k - 1, f32))
