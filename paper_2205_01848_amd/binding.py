"""ctypes binding of libmoe.so: the same names as the C entry points in
include/moe.h, taking torch tensors (device memory) and ints.  This module
only marshals arguments; every step runs in the HIP kernels of libmoe.  If
the library is missing it raises - there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmoe.so")

MOE_F32, MOE_BF16 = 0, 1
MOE_RELU, MOE_GELU_TANH, MOE_SWIGLU = 0, 1, 2
ACTS = {"relu": MOE_RELU, "gelu_tanh": MOE_GELU_TANH, "swiglu": MOE_SWIGLU}
STATUS_BAD_ID, STATUS_DUP_ID, STATUS_REGION = 1, 2, 4

_c_int, _c_i64, _c_size, _p = ctypes.c_int, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p

# name -> (restype, argtypes)
SIGNATURES = {
    "moe_status_string": (ctypes.c_char_p, [_c_int]),
    "moe_abi_version": (_c_int, []),
    "moe_gate_topk": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                               _p, _p, _p, _p, _p, _p]),
    "moe_count": (_c_int, [_p, _c_int, _c_int, _c_int, _p, _p, _p]),
    "moe_update_capacity": (_c_int, [_p, _c_int, _c_int, _c_int, _p, _c_int, _c_int, _c_int,
                                     _c_int, _p, _p]),
    "moe_dispatch_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int]),
    "moe_dispatch": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_int, _p, _p, _p, _p,
                              _c_i64, _p, _p, _p, _p, _p, _p, _p, _c_size]),
    "moe_dispatch_noalloc": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_int, _p, _p, _p,
                                      _p, _c_i64, _p, _p, _p, _p, _p, _p]),
    "moe_dispatch_noalloc_max_assignments": (_c_size, []),
    "moe_ffn_fwd_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_i64]),
    "moe_ffn_bwd_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_i64]),
    "moe_expert_ffn_fwd": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_int, _p, _p,
                                    _c_i64, _p, _p, _p, _p, _p, _p, _p, _c_size]),
    "moe_zero_pad_rows": (_c_int, [_p, _c_int, _c_int, _c_int, _p, _p, _p, _c_i64, _p]),
    "moe_combine": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_i64, _p, _p, _p, _p]),
    "moe_combine_bwd": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_i64, _p, _p, _p,
                                 _p, _p, _p]),
    "moe_expert_ffn_bwd": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_int, _p, _p,
                                    _c_i64, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p,
                                    _c_size]),
    "moe_gate_bwd_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int]),
    "moe_gate_bwd": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _p, _p,
                              _p, _p, _p, _p, _p, _p, _c_size]),
    "moe_dispatch_bwd": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_int, _c_i64, _p,
                                  _p, _p, _p, _p]),
    "moe_balance_workspace_bytes": (_c_size, [_c_int, _c_int]),
    "moe_balance_fwd": (_c_int, [_p, _c_int, _c_int, _c_int, ctypes.c_float, _p, _p, _p, _p,
                                 _p, _c_size]),
    "moe_aggregate_spec": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _p, _p, _c_i64, _p]),
    "moe_spec_loss_workspace_bytes": (_c_size, [_c_int]),
    "moe_spec_loss": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _p, _p, _p, _p, _c_i64, _p,
                               _p, _p, _p, _c_size]),
    "moe_cache_update": (_c_int, [_p, _c_int, _c_int, _p, _p, _p, _p]),
    "moe_cached_weights": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _p, _p, _p]),
    "moe_caching_decision": (_c_int, [_c_int, _c_i64, _c_i64, _c_int, _c_int, _c_int, _c_int,
                                      _c_int, _c_int]),
    "moe_capacity_trigger": (_c_int, [_c_int, _c_int, _p, _p, _c_int, _c_int, _c_int, _c_int,
                                      _c_int]),
    "moe_policy_create": (_c_int, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                                   _c_int, _c_int, _c_int, _p, _p]),
    "moe_policy_destroy": (None, [_p]),
    "moe_policy_begin": (_c_int, [_p, _p, _p, _p, _p, _p]),
    "moe_policy_end": (_c_int, [_p, _p, _p]),
    "moe_policy_state": (_c_int, [_p, _p, _p, _p, _p]),
    "moe_timing_enable": (_c_int, [_c_int]),
    "moe_set_gemm_tiles": (_c_int, [_c_int]),
    "moe_set_dx_weight_copy": (_c_int, [_c_int]),
    "moe_timing_report": (_c_int, [ctypes.c_char_p, _c_size]),
}

_lib = None


ABI_VERSION = 7   # moe_abi_version() of the library this binding is written for


class MoEError(RuntimeError):
    pass


def lib():
    """The loaded libmoe.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise MoEError(f"{LIB_PATH} is not built (python -m paper_2205_01848_amd.build); "
                           "the HIP library is required, there is no fallback")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        # buffer sizes here follow this ABI (h_save planes, argument lists):
        # a library of another version would read and write past them
        if L.moe_abi_version() != ABI_VERSION:
            raise MoEError(f"{LIB_PATH} has ABI version {L.moe_abi_version()}, this binding "
                           f"expects {ABI_VERSION}: rebuild it (python -m paper_2205_01848_amd.build)")
        _lib = L
    return _lib


def _check(st: int, what: str):
    if st != 0:
        raise MoEError(f"{what}: {lib().moe_status_string(st).decode()}")


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise MoEError("tensor must live in device memory")
    if not t.is_contiguous():
        raise MoEError("tensor must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return MOE_BF16
    if t.dtype == torch.float32:
        return MOE_F32
    raise MoEError(f"unsupported layer dtype {t.dtype}")


_I32, _F32 = torch.int32, torch.float32


def _need(t: Optional[torch.Tensor], n: int, name: str, dtype=None, optional=False):
    """Refuse a tensor with fewer than the n elements the entry point reads or
    writes, or of the wrong element type.  The C ABI takes bare pointers and
    cannot check sizes; an undersized buffer would be accessed past its end."""
    if t is None:
        if optional:
            return
        raise MoEError(f"{name} is required")
    if dtype is not None and t.dtype != dtype:
        raise MoEError(f"{name}: element type {t.dtype}, expected {dtype}")
    if t.numel() < n:
        raise MoEError(f"{name} holds {t.numel()} elements, the call needs {n}")


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def h_save_planes(act: int) -> int:
    """[rows_alloc, f] planes of h_save: A for ReLU, H and A for GELU, H1, H3
    and A for SwiGLU."""
    return 3 if act == MOE_SWIGLU else 2 if act == MOE_GELU_TANH else 1


def workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


# ---- entry points -----------------------------------------------------------
def moe_gate_topk(x, w_g, bias, k, renorm, logits, ids, weights):
    T, d = x.shape
    E = w_g.shape[0]
    _need(w_g, E * d, "w_g", x.dtype)
    _need(bias, E, "bias", _F32, optional=True)
    _need(logits, T * E, "logits", _F32)
    _need(ids, T * k, "ids", _I32)
    _need(weights, T * k, "weights", _F32)
    _check(lib().moe_gate_topk(_stream(), _dt(x), T, d, E, k, int(renorm), _ptr(x), _ptr(w_g),
                               _ptr(bias), _ptr(logits), _ptr(ids), _ptr(weights)),
           "moe_gate_topk")


def moe_count(ids, E, counts, status):
    T, k = ids.shape
    _need(ids, T * k, "ids", _I32)
    _need(counts, E, "counts", _I32)
    _need(status, 1, "status", _I32)
    _check(lib().moe_count(_stream(), T, E, k, _ptr(ids), _ptr(counts), _ptr(status)),
           "moe_count")


def moe_update_capacity(T, k, E, counts, num, den, cap_min, capacity, offsets, row_align=1):
    _need(counts, E, "counts", _I32, optional=True)
    _need(capacity, E, "capacity", _I32)
    _need(offsets, E + 1, "offsets", _I32)
    _check(lib().moe_update_capacity(_stream(), T, k, E, _ptr(counts), num, den, cap_min,
                                     row_align, _ptr(capacity), _ptr(offsets)),
           "moe_update_capacity")


def moe_dispatch_workspace_bytes(T, E, k) -> int:
    return lib().moe_dispatch_workspace_bytes(T, E, k)


def moe_dispatch(x, ids, E, capacity, offsets, rows_alloc, counts, fill, dest_row, src, x_disp,
                 status, ws):
    T, d = x.shape
    k = ids.shape[1]
    _need(ids, T * k, "ids", _I32)
    for t, n, name in ((capacity, E, "capacity"), (offsets, E + 1, "offsets"),
                       (counts, E, "counts"), (fill, E, "fill"), (dest_row, T * k, "dest_row"),
                       (src, rows_alloc, "src"), (status, 1, "status")):
        _need(t, n, name, _I32)
    _need(x_disp, rows_alloc * d, "x_disp", x.dtype)
    _check(lib().moe_dispatch(_stream(), _dt(x), T, d, E, k, _ptr(x), _ptr(ids), _ptr(capacity),
                              _ptr(offsets), rows_alloc, _ptr(counts), _ptr(fill),
                              _ptr(dest_row), _ptr(src), _ptr(x_disp), _ptr(status), _ptr(ws),
                              _nbytes(ws)), "moe_dispatch")


def moe_dispatch_noalloc_max_assignments() -> int:
    return lib().moe_dispatch_noalloc_max_assignments()


def moe_dispatch_noalloc(x, ids, E, capacity, offsets, rows_alloc, counts, fill, dest_row, src,
                         x_disp, status):
    """moe_dispatch without a workspace (the library's fixed device scratch)."""
    T, d = x.shape
    k = ids.shape[1]
    _need(ids, T * k, "ids", _I32)
    for t, n, name in ((capacity, E, "capacity"), (offsets, E + 1, "offsets"),
                       (counts, E, "counts"), (fill, E, "fill"), (dest_row, T * k, "dest_row"),
                       (src, rows_alloc, "src"), (status, 1, "status")):
        _need(t, n, name, _I32)
    _need(x_disp, rows_alloc * d, "x_disp", x.dtype)
    _check(lib().moe_dispatch_noalloc(_stream(), _dt(x), T, d, E, k, _ptr(x), _ptr(ids),
                                      _ptr(capacity), _ptr(offsets), rows_alloc, _ptr(counts),
                                      _ptr(fill), _ptr(dest_row), _ptr(src), _ptr(x_disp),
                                      _ptr(status)), "moe_dispatch_noalloc")


def moe_ffn_fwd_workspace_bytes(dt, act, E, d, f, rows_alloc) -> int:
    return lib().moe_ffn_fwd_workspace_bytes(dt, act, E, d, f, rows_alloc)


def moe_ffn_bwd_workspace_bytes(dt, act, E, d, f, rows_alloc) -> int:
    return lib().moe_ffn_bwd_workspace_bytes(dt, act, E, d, f, rows_alloc)


def moe_expert_ffn_fwd(act, offsets, rows, x_disp, w1, w3, w2, h_save, y_disp, ws):
    E, f, d = w1.shape
    R, dt = x_disp.shape[0], w1.dtype
    _need(offsets, E + 1, "offsets", _I32)
    _need(rows, E, "rows", _I32)
    _need(x_disp, R * d, "x_disp", dt)
    _need(w3, E * f * d, "w3", dt, optional=act != MOE_SWIGLU)
    _need(w2, E * d * f, "w2", dt)
    _need(h_save, h_save_planes(act) * R * f, "h_save", dt, optional=True)
    _need(y_disp, R * d, "y_disp", dt)
    _check(lib().moe_expert_ffn_fwd(_stream(), _dt(w1), act, E, d, f, _ptr(offsets), _ptr(rows),
                                    x_disp.shape[0], _ptr(x_disp), _ptr(w1), _ptr(w3), _ptr(w2),
                                    _ptr(h_save), _ptr(y_disp), _ptr(ws), _nbytes(ws)),
           "moe_expert_ffn_fwd")


def moe_zero_pad_rows(offsets, fill, rows, buf):
    E = fill.shape[0]
    R, d = buf.shape
    _need(offsets, E + 1, "offsets", _I32)
    _need(fill, E, "fill", _I32)
    _need(rows, E, "rows", _I32)
    _check(lib().moe_zero_pad_rows(_stream(), _dt(buf), E, d, _ptr(offsets), _ptr(fill),
                                   _ptr(rows), R, _ptr(buf)), "moe_zero_pad_rows")


def moe_combine(y_disp, dest_row, weights, y):
    T, k = dest_row.shape
    d = y.shape[1]
    _need(y_disp, y_disp.shape[0] * d, "y_disp", y.dtype)
    _need(dest_row, T * k, "dest_row", _I32)
    _need(weights, T * k, "weights", _F32)
    _need(y, T * d, "y")
    _check(lib().moe_combine(_stream(), _dt(y), T, d, k, y_disp.shape[0], _ptr(y_disp),
                             _ptr(dest_row), _ptr(weights), _ptr(y)), "moe_combine")


def moe_combine_bwd(dy, y_disp, dest_row, weights, dy_disp, dweights):
    T, k = dest_row.shape
    d = dy.shape[1]
    R = y_disp.shape[0]
    _need(dy, T * d, "dy")
    _need(y_disp, R * d, "y_disp", dy.dtype)
    _need(dest_row, T * k, "dest_row", _I32)
    _need(weights, T * k, "weights", _F32)
    _need(dy_disp, R * d, "dy_disp", dy.dtype)
    _need(dweights, T * k, "dweights", _F32)
    _check(lib().moe_combine_bwd(_stream(), _dt(dy), T, d, k, y_disp.shape[0], _ptr(dy),
                                 _ptr(y_disp), _ptr(dest_row), _ptr(weights), _ptr(dy_disp),
                                 _ptr(dweights)), "moe_combine_bwd")


def moe_expert_ffn_bwd(act, offsets, rows, x_disp, h_save, w1, w3, w2, dy_disp, dx_disp, dw1,
                       dw3, dw2, ws):
    E, f, d = w1.shape
    R, dt, sw = x_disp.shape[0], w1.dtype, act == MOE_SWIGLU
    _need(offsets, E + 1, "offsets", _I32)
    _need(rows, E, "rows", _I32)
    _need(x_disp, R * d, "x_disp", dt)
    _need(h_save, h_save_planes(act) * R * f, "h_save", dt)
    _need(w3, E * f * d, "w3", dt, optional=not sw)
    _need(w2, E * d * f, "w2", dt)
    _need(dy_disp, R * d, "dy_disp", dt)
    _need(dx_disp, R * d, "dx_disp", dt)
    _need(dw1, E * f * d, "dw1", _F32)
    _need(dw3, E * f * d, "dw3", _F32, optional=not sw)
    _need(dw2, E * d * f, "dw2", _F32)
    _check(lib().moe_expert_ffn_bwd(_stream(), _dt(w1), act, E, d, f, _ptr(offsets), _ptr(rows),
                                    x_disp.shape[0], _ptr(x_disp), _ptr(h_save), _ptr(w1),
                                    _ptr(w3), _ptr(w2), _ptr(dy_disp), _ptr(dx_disp), _ptr(dw1),
                                    _ptr(dw3), _ptr(dw2), _ptr(ws), _nbytes(ws)),
           "moe_expert_ffn_bwd")


def moe_gate_bwd_workspace_bytes(T, d, E) -> int:
    return lib().moe_gate_bwd_workspace_bytes(T, d, E)


def moe_gate_bwd(x, logits, ids, dweights, renorm, dlogits, dw_g, ws, dprob_coef=None):
    T, d = x.shape
    E = logits.shape[1]
    k = ids.shape[1]
    _need(logits, T * E, "logits", _F32)
    _need(ids, T * k, "ids", _I32)
    _need(dweights, T * k, "dweights", _F32)
    _need(dprob_coef, E, "dprob_coef", _F32, optional=True)
    _need(dlogits, T * E, "dlogits", _F32)
    _need(dw_g, E * d, "dw_g", _F32)
    _check(lib().moe_gate_bwd(_stream(), _dt(x), T, d, E, k, int(renorm), _ptr(x), _ptr(logits),
                              _ptr(ids), _ptr(dweights), _ptr(dprob_coef), _ptr(dlogits),
                              _ptr(dw_g), _ptr(ws), _nbytes(ws)), "moe_gate_bwd")


def moe_dispatch_bwd(dx_disp, dest_row, E, dlogits, w_g, dx):
    T, k = dest_row.shape
    d = dx.shape[1]
    _need(dx_disp, dx_disp.shape[0] * d, "dx_disp", dx.dtype)
    _need(dest_row, T * k, "dest_row", _I32)
    _need(dlogits, T * E, "dlogits", _F32, optional=True)
    _need(w_g, E * d, "w_g", dx.dtype, optional=True)
    _need(dx, T * d, "dx")
    _check(lib().moe_dispatch_bwd(_stream(), _dt(dx), T, d, E, k, dx_disp.shape[0],
                                  _ptr(dx_disp), _ptr(dest_row), _ptr(dlogits), _ptr(w_g),
                                  _ptr(dx)), "moe_dispatch_bwd")


# ---- loss-side operators ------------------------------------------------------
def moe_balance_workspace_bytes(T, E) -> int:
    return lib().moe_balance_workspace_bytes(T, E)


def moe_balance_fwd(logits, counts, k, lam, loss, dprob_coef, ws):
    T, E = logits.shape
    _need(logits, T * E, "logits", _F32)
    _need(counts, E, "counts", _I32)
    _need(loss, 1, "loss", _F32)
    _need(dprob_coef, E, "dprob_coef", _F32)
    _check(lib().moe_balance_fwd(_stream(), T, E, k, float(lam), _ptr(logits), _ptr(counts),
                                 _ptr(loss), _ptr(dprob_coef), _ptr(ws), _nbytes(ws)),
           "moe_balance_fwd")


def moe_aggregate_spec(y_disp, dest_row, out):
    T, k = dest_row.shape
    d = out.shape[1]
    _need(y_disp, y_disp.shape[0] * d, "y_disp", out.dtype)
    _need(dest_row, T * k, "dest_row", _I32)
    _need(out, T * k * d, "out")
    _check(lib().moe_aggregate_spec(_stream(), _dt(out), T, d, k, _ptr(y_disp), _ptr(dest_row),
                                    y_disp.shape[0], _ptr(out)), "moe_aggregate_spec")


def moe_spec_loss_workspace_bytes(T) -> int:
    return lib().moe_spec_loss_workspace_bytes(T)


def moe_spec_loss(y_disp, dest_row, weights, target, dy_disp, dweights, loss, ws):
    T, k = dest_row.shape
    d = target.shape[1]
    R = y_disp.shape[0]
    _need(y_disp, R * d, "y_disp", target.dtype)
    _need(dest_row, T * k, "dest_row", _I32)
    _need(weights, T * k, "weights", _F32)
    _need(target, T * d, "target")
    _need(dy_disp, R * d, "dy_disp", target.dtype)
    _need(dweights, T * k, "dweights", _F32)
    _need(loss, 1, "loss", _F32)
    _check(lib().moe_spec_loss(_stream(), _dt(target), T, d, k, _ptr(y_disp), _ptr(dest_row),
                               _ptr(weights), _ptr(target), y_disp.shape[0], _ptr(dy_disp),
                               _ptr(dweights), _ptr(loss), _ptr(ws), _nbytes(ws)),
           "moe_spec_loss")


# ---- sample assignment caching ------------------------------------------------
def moe_cache_update(fresh_ids, cached, cache_out, unchanged):
    T, k = fresh_ids.shape
    for t, name in ((fresh_ids, "fresh_ids"), (cached, "cached"), (cache_out, "cache_out")):
        _need(t, T * k, name, _I32)
    _need(unchanged, 1, "unchanged", _I32)
    _check(lib().moe_cache_update(_stream(), T, k, _ptr(fresh_ids), _ptr(cached), _ptr(cache_out),
                                  _ptr(unchanged)), "moe_cache_update")


def moe_cached_weights(logits, ids, renorm, weights):
    T, E = logits.shape
    k = ids.shape[1]
    _need(logits, T * E, "logits", _F32)
    _need(ids, T * k, "ids", _I32)
    _need(weights, T * k, "weights", _F32)
    _check(lib().moe_cached_weights(_stream(), T, E, k, int(renorm), _ptr(logits), _ptr(ids),
                                    _ptr(weights)), "moe_cached_weights")


def moe_caching_decision(enabled, unchanged, samples, epoch, on=(96, 100), off=(90, 100),
                         min_epoch=10) -> bool:
    r = lib().moe_caching_decision(int(bool(enabled)), int(unchanged), int(samples), int(epoch),
                                   on[0], on[1], off[0], off[1], int(min_epoch))
    if r < 0:
        raise MoEError("moe_caching_decision: invalid arguments")
    return bool(r)


# ---- capacity policy at the launch frontier --------------------------------------
def moe_capacity_trigger(T, counts, cap, grow, shrink, cap_min=0):
    """Host trigger: returns (new capacities, recompiled)."""
    E = len(counts)
    c = (ctypes.c_int32 * E)(*[int(v) for v in counts])
    C = (ctypes.c_int32 * E)(*[int(v) for v in cap])
    r = lib().moe_capacity_trigger(T, E, c, C, grow[0], grow[1], shrink[0], shrink[1], cap_min)
    if r < 0:
        raise MoEError("moe_capacity_trigger: invalid arguments")
    return list(C), bool(r)


class CapacityPolicy:
    """Owner of one moe_capacity_policy object (see include/moe.h)."""

    def __init__(self, T, k, E, delta_launch, grow, shrink, init_cap, cap_min=0, row_align=1):
        init = (ctypes.c_int32 * E)(*[int(c) for c in init_cap])
        h = ctypes.c_void_p()
        _check(lib().moe_policy_create(T, k, E, delta_launch, grow[0], grow[1], shrink[0],
                                       shrink[1], cap_min, row_align, init, ctypes.byref(h)),
               "moe_policy_create")
        self._h, self.E = h, E

    def begin(self, capacity, offsets):
        """Enqueue the capacities for the next launch; returns (rows needed,
        whether the trigger recompiled)."""
        _need(capacity, self.E, "capacity", _I32)
        _need(offsets, self.E + 1, "offsets", _I32)
        rows = ctypes.c_int64()
        rec = ctypes.c_int()
        _check(lib().moe_policy_begin(self._h, _stream(), _ptr(capacity), _ptr(offsets),
                                      ctypes.byref(rows), ctypes.byref(rec)), "moe_policy_begin")
        return rows.value, bool(rec.value)

    def end(self, counts):
        _need(counts, self.E, "counts", _I32)
        _check(lib().moe_policy_end(self._h, _stream(), _ptr(counts)), "moe_policy_end")

    def state(self):
        cap = (ctypes.c_int32 * self.E)()
        n, c, r = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(lib().moe_policy_state(self._h, cap, ctypes.byref(n), ctypes.byref(c),
                                      ctypes.byref(r)), "moe_policy_state")
        return dict(cap=list(cap), launched=n.value, consumed=c.value, recompiles=r.value)

    def close(self):
        if self._h is not None and self._h.value:
            lib().moe_policy_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---- kernel timing (instrumentation) ----------------------------------------
def moe_timing_enable(on: bool):
    _check(lib().moe_timing_enable(1 if on else 0), "moe_timing_enable")


def moe_set_gemm_tiles(mode: int):
    """0: automatic tile choice; 1: 256x256 tiles only (bf16 and fp32); 2: 128x128 tiles
    only (bf16)."""
    _check(lib().moe_set_gemm_tiles(int(mode)), "moe_set_gemm_tiles")


def moe_set_dx_weight_copy(mode: int):
    """0: automatic; 1: dX reads W1/W3 K-major; 2: dX reads a transposed copy (bf16)."""
    _check(lib().moe_set_dx_weight_copy(int(mode)), "moe_set_dx_weight_copy")


def moe_timing_report() -> dict:
    """{kernel name: (launches, total ms)} since the last report."""
    buf = ctypes.create_string_buffer(1 << 16)
    lib().moe_timing_report(buf, len(buf))
    out = {}
    for line in buf.value.decode().splitlines():
        name, n, ms = line.split()
        out[name] = (int(n), float(ms))
    return out
