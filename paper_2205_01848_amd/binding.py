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
                                     _p, _p]),
    "moe_dispatch_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int]),
    "moe_dispatch": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_int, _p, _p, _p, _p,
                              _c_i64, _p, _p, _p, _p, _p, _p, _p, _c_size]),
    "moe_ffn_fwd_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_i64]),
    "moe_ffn_bwd_workspace_bytes": (_c_size, [_c_int, _c_int, _c_int, _c_int, _c_int, _c_i64]),
    "moe_expert_ffn_fwd": (_c_int, [_p, _c_int, _c_int, _c_int, _c_int, _c_int, _p, _p,
                                    _c_i64, _p, _p, _p, _p, _p, _p, _p, _c_size]),
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
                                   _c_int, _c_int, _p, _p]),
    "moe_policy_destroy": (None, [_p]),
    "moe_policy_begin": (_c_int, [_p, _p, _p, _p, _p, _p]),
    "moe_policy_end": (_c_int, [_p, _p, _p]),
    "moe_policy_state": (_c_int, [_p, _p, _p, _p, _p]),
    "moe_timing_enable": (_c_int, [_c_int]),
    "moe_timing_report": (_c_int, [ctypes.c_char_p, _c_size]),
}

_lib = None


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


def workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


# ---- entry points -----------------------------------------------------------
def moe_gate_topk(x, w_g, bias, k, renorm, logits, ids, weights):
    T, d = x.shape
    E = w_g.shape[0]
    _check(lib().moe_gate_topk(_stream(), _dt(x), T, d, E, k, int(renorm), _ptr(x), _ptr(w_g),
                               _ptr(bias), _ptr(logits), _ptr(ids), _ptr(weights)),
           "moe_gate_topk")


def moe_count(ids, E, counts, status):
    T, k = ids.shape
    _check(lib().moe_count(_stream(), T, E, k, _ptr(ids), _ptr(counts), _ptr(status)),
           "moe_count")


def moe_update_capacity(T, k, E, counts, num, den, cap_min, capacity, offsets):
    _check(lib().moe_update_capacity(_stream(), T, k, E, _ptr(counts), num, den, cap_min,
                                     _ptr(capacity), _ptr(offsets)), "moe_update_capacity")


def moe_dispatch_workspace_bytes(T, E, k) -> int:
    return lib().moe_dispatch_workspace_bytes(T, E, k)


def moe_dispatch(x, ids, E, capacity, offsets, rows_alloc, counts, fill, dest_row, src, x_disp,
                 status, ws):
    T, d = x.shape
    k = ids.shape[1]
    _check(lib().moe_dispatch(_stream(), _dt(x), T, d, E, k, _ptr(x), _ptr(ids), _ptr(capacity),
                              _ptr(offsets), rows_alloc, _ptr(counts), _ptr(fill),
                              _ptr(dest_row), _ptr(src), _ptr(x_disp), _ptr(status), _ptr(ws),
                              ws.numel()), "moe_dispatch")


def moe_ffn_fwd_workspace_bytes(dt, act, E, d, f, rows_alloc) -> int:
    return lib().moe_ffn_fwd_workspace_bytes(dt, act, E, d, f, rows_alloc)


def moe_ffn_bwd_workspace_bytes(dt, act, E, d, f, rows_alloc) -> int:
    return lib().moe_ffn_bwd_workspace_bytes(dt, act, E, d, f, rows_alloc)


def moe_expert_ffn_fwd(act, offsets, rows, x_disp, w1, w3, w2, h_save, y_disp, ws):
    E, f, d = w1.shape
    _check(lib().moe_expert_ffn_fwd(_stream(), _dt(w1), act, E, d, f, _ptr(offsets), _ptr(rows),
                                    x_disp.shape[0], _ptr(x_disp), _ptr(w1), _ptr(w3), _ptr(w2),
                                    _ptr(h_save), _ptr(y_disp), _ptr(ws), ws.numel()),
           "moe_expert_ffn_fwd")


def moe_combine(y_disp, dest_row, weights, y):
    T, k = dest_row.shape
    d = y.shape[1]
    _check(lib().moe_combine(_stream(), _dt(y), T, d, k, y_disp.shape[0], _ptr(y_disp),
                             _ptr(dest_row), _ptr(weights), _ptr(y)), "moe_combine")


def moe_combine_bwd(dy, y_disp, dest_row, weights, dy_disp, dweights):
    T, k = dest_row.shape
    d = dy.shape[1]
    _check(lib().moe_combine_bwd(_stream(), _dt(dy), T, d, k, y_disp.shape[0], _ptr(dy),
                                 _ptr(y_disp), _ptr(dest_row), _ptr(weights), _ptr(dy_disp),
                                 _ptr(dweights)), "moe_combine_bwd")


def moe_expert_ffn_bwd(act, offsets, rows, x_disp, h_save, w1, w3, w2, dy_disp, dx_disp, dw1,
                       dw3, dw2, ws):
    E, f, d = w1.shape
    _check(lib().moe_expert_ffn_bwd(_stream(), _dt(w1), act, E, d, f, _ptr(offsets), _ptr(rows),
                                    x_disp.shape[0], _ptr(x_disp), _ptr(h_save), _ptr(w1),
                                    _ptr(w3), _ptr(w2), _ptr(dy_disp), _ptr(dx_disp), _ptr(dw1),
                                    _ptr(dw3), _ptr(dw2), _ptr(ws), ws.numel()),
           "moe_expert_ffn_bwd")


def moe_gate_bwd_workspace_bytes(T, d, E) -> int:
    return lib().moe_gate_bwd_workspace_bytes(T, d, E)


def moe_gate_bwd(x, logits, ids, dweights, renorm, dlogits, dw_g, ws, dprob_coef=None):
    T, d = x.shape
    E = logits.shape[1]
    k = ids.shape[1]
    _check(lib().moe_gate_bwd(_stream(), _dt(x), T, d, E, k, int(renorm), _ptr(x), _ptr(logits),
                              _ptr(ids), _ptr(dweights), _ptr(dprob_coef), _ptr(dlogits),
                              _ptr(dw_g), _ptr(ws), ws.numel()), "moe_gate_bwd")


def moe_dispatch_bwd(dx_disp, dest_row, E, dlogits, w_g, dx):
    T, k = dest_row.shape
    d = dx.shape[1]
    _check(lib().moe_dispatch_bwd(_stream(), _dt(dx), T, d, E, k, dx_disp.shape[0],
                                  _ptr(dx_disp), _ptr(dest_row), _ptr(dlogits), _ptr(w_g),
                                  _ptr(dx)), "moe_dispatch_bwd")


# ---- loss-side operators ------------------------------------------------------
def moe_balance_workspace_bytes(T, E) -> int:
    return lib().moe_balance_workspace_bytes(T, E)


def moe_balance_fwd(logits, counts, k, lam, loss, dprob_coef, ws):
    T, E = logits.shape
    _check(lib().moe_balance_fwd(_stream(), T, E, k, float(lam), _ptr(logits), _ptr(counts),
                                 _ptr(loss), _ptr(dprob_coef), _ptr(ws), ws.numel()),
           "moe_balance_fwd")


def moe_aggregate_spec(y_disp, dest_row, out):
    T, k = dest_row.shape
    d = out.shape[1]
    _check(lib().moe_aggregate_spec(_stream(), _dt(out), T, d, k, _ptr(y_disp), _ptr(dest_row),
                                    y_disp.shape[0], _ptr(out)), "moe_aggregate_spec")


def moe_spec_loss_workspace_bytes(T) -> int:
    return lib().moe_spec_loss_workspace_bytes(T)


def moe_spec_loss(y_disp, dest_row, weights, target, dy_disp, dweights, loss, ws):
    T, k = dest_row.shape
    d = target.shape[1]
    _check(lib().moe_spec_loss(_stream(), _dt(target), T, d, k, _ptr(y_disp), _ptr(dest_row),
                               _ptr(weights), _ptr(target), y_disp.shape[0], _ptr(dy_disp),
                               _ptr(dweights), _ptr(loss), _ptr(ws), ws.numel()),
           "moe_spec_loss")


# ---- sample assignment caching ------------------------------------------------
def moe_cache_update(fresh_ids, cached, cache_out, unchanged):
    T, k = fresh_ids.shape
    _check(lib().moe_cache_update(_stream(), T, k, _ptr(fresh_ids), _ptr(cached), _ptr(cache_out),
                                  _ptr(unchanged)), "moe_cache_update")


def moe_cached_weights(logits, ids, renorm, weights):
    T, E = logits.shape
    k = ids.shape[1]
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

    def __init__(self, T, k, E, delta_launch, grow, shrink, init_cap, cap_min=0):
        init = (ctypes.c_int32 * E)(*[int(c) for c in init_cap])
        h = ctypes.c_void_p()
        _check(lib().moe_policy_create(T, k, E, delta_launch, grow[0], grow[1], shrink[0],
                                       shrink[1], cap_min, init, ctypes.byref(h)),
               "moe_policy_create")
        self._h, self.E = h, E

    def begin(self, capacity, offsets):
        """Enqueue the capacities for the next launch; returns (rows needed,
        whether the trigger recompiled)."""
        rows = ctypes.c_int64()
        rec = ctypes.c_int()
        _check(lib().moe_policy_begin(self._h, _stream(), _ptr(capacity), _ptr(offsets),
                                      ctypes.byref(rows), ctypes.byref(rec)), "moe_policy_begin")
        return rows.value, bool(rec.value)

    def end(self, counts):
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


def moe_timing_report() -> dict:
    """{kernel name: (launches, total ms)} since the last report."""
    buf = ctypes.create_string_buffer(1 << 16)
    lib().moe_timing_report(buf, len(buf))
    out = {}
    for line in buf.value.decode().splitlines():
        name, n, ms = line.split()
        out[name] = (int(n), float(ms))
    return out
