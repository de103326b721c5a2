"""One MoE layer on one GPU: device buffers plus the sequence of libmoe calls.

PyTorch only allocates device memory and provides the stream; every step of
the layer is a libmoe entry point (see include/moe.h).  Buffers are sized
once, on the host, with no device synchronisation:

* static capacity factor alpha = num/den:  rows_alloc = E * min(T, ceil(alpha*T*k/E))
* dynamic capacity with margin num/den:    rows_alloc = min(E*T, ceil(num*T*k/den) + E)
* exact capacity (margin 1):               rows_alloc = T*k
each plus, when the regions are aligned (row_align > 1), at most
row_align - 1 padding rows per expert.
"""
from __future__ import annotations

from typing import Optional

import torch

from . import binding as B


def _cdiv(a: int, b: int) -> int:
    return -(-a // b)


# Default alignment (rows) of the expert regions of the grouped buffers
# (moe_update_capacity's row_align).  1 packs them: regions aligned to the
# GEMMs' 256-row tiles measured the same step time on MI355X (within 0.5% on
# every workload), so the packed layout, which needs no padding rows, is kept.
ROW_ALIGN = 1


def rows_alloc_for(kind: str, T: int, k: int, E: int, num: int = 1, den: int = 1,
                   align: int = ROW_ALIGN) -> int:
    if kind == "static":
        return E * _cdiv(min(T, _cdiv(num * T * k, den * E)), align) * align
    pad = E * (align - 1)
    if kind == "dynamic":
        return min(E * T, _cdiv(num * T * k, den) + E) + pad
    if kind == "exact":
        return T * k + pad
    raise ValueError(kind)


class MoELayer:
    def __init__(self, T: int, d: int, E: int, k: int, f: int, act: str,
                 dtype: torch.dtype, rows_alloc: int, backward: bool = False,
                 gate: bool = True, device="cuda", row_align: int = ROW_ALIGN):
        self.T, self.d, self.E, self.k, self.f = T, d, E, k, f
        self.row_align = row_align
        self.act = B.ACTS[act]
        self.swiglu = act == "swiglu"
        self.dtype = dtype
        self.rows_alloc = int(rows_alloc)
        self.dev = torch.device(device)
        self.has_gate = gate
        dt = B.MOE_BF16 if dtype == torch.bfloat16 else B.MOE_F32
        i32, f32 = torch.int32, torch.float32
        e = lambda *s, t=dtype: torch.empty(*s, dtype=t, device=self.dev)
        R = self.rows_alloc
        self.logits = e(T, E, t=f32)
        self.ids = e(T, k, t=i32)
        self.weights = e(T, k, t=f32)
        self.counts = e(E, t=i32)
        self.fill = e(E, t=i32)
        self.capacity = e(E, t=i32)
        self.offsets = e(E + 1, t=i32)
        self.status = torch.zeros(1, dtype=i32, device=self.dev)
        self.dest_row = e(T, k, t=i32)
        self.src = e(max(R, 1), t=i32)
        self.x_disp = e(max(R, 1), d)
        self.y_disp = e(max(R, 1), d)
        self.y = e(T, d)
        self.ws_dispatch = B.workspace(B.moe_dispatch_workspace_bytes(T, E, k), self.dev)
        self.ws_fwd = B.workspace(B.moe_ffn_fwd_workspace_bytes(dt, self.act, E, d, f, R), self.dev)
        self.backward_enabled = backward
        self.h_save = None
        if backward:
            # A = act(H), after H (GELU) or H1, H3 (SwiGLU), kept for the backward
            self.h_save = e(B.h_save_planes(self.act) * max(R, 1) * f)
            self.dy_disp = e(max(R, 1), d)
            self.dx_disp = e(max(R, 1), d)
            self.dweights = e(T, k, t=f32)
            self.dw1 = e(E, f, d, t=f32)
            self.dw3 = e(E, f, d, t=f32) if self.swiglu else None
            self.dw2 = e(E, d, f, t=f32)
            self.dx = e(T, d)
            self.ws_bwd = B.workspace(B.moe_ffn_bwd_workspace_bytes(dt, self.act, E, d, f, R),
                                      self.dev)
            if gate:
                self.dlogits = e(T, E, t=f32)
                self.dw_g = e(E, d, t=f32)
                self.ws_gate_bwd = B.workspace(B.moe_gate_bwd_workspace_bytes(T, d, E), self.dev)
        # loss-side operators and caching: allocated on first use
        self.balance_loss = self.dprob_coef = self.ws_balance = None
        self._balance_on = False
        self.spec_loss_value = self.ws_spec = None
        self.cached_weights = None

    # ---- forward pieces ------------------------------------------------------
    def gate(self, x, w_g, bias, renorm: int):
        B.moe_gate_topk(x, w_g, bias, self.k, renorm, self.logits, self.ids, self.weights)

    def count(self, ids: Optional[torch.Tensor] = None):
        B.moe_count(self.ids if ids is None else ids, self.E, self.counts, self.status)

    def capacity_static(self, num: int, den: int, cap_min: int = 0):
        B.moe_update_capacity(self.T, self.k, self.E, None, num, den, cap_min, self.capacity,
                              self.offsets, row_align=self.row_align)

    def capacity_dynamic(self, num: int, den: int, counts: Optional[torch.Tensor] = None,
                         cap_min: int = 0):
        B.moe_update_capacity(self.T, self.k, self.E, self.counts if counts is None else counts,
                              num, den, cap_min, self.capacity, self.offsets,
                              row_align=self.row_align)

    def dispatch(self, x, ids: Optional[torch.Tensor] = None):
        B.moe_dispatch(x, self.ids if ids is None else ids, self.E, self.capacity, self.offsets,
                       self.rows_alloc, self.counts, self.fill, self.dest_row, self.src,
                       self.x_disp, self.status, self.ws_dispatch)

    def ffn_fwd(self, w1, w3, w2, rows: str = "fill"):
        """rows="fill": the method, each expert over its kept rows.
        rows="capacity": the padded static-shape baseline, each expert over
        its whole capacity with the unfilled rows of x_disp zeroed first."""
        if rows == "fill":
            r = self.fill
        else:
            r = self.capacity
            B.moe_zero_pad_rows(self.offsets, self.fill, r, self.x_disp)
        B.moe_expert_ffn_fwd(self.act, self.offsets, r, self.x_disp, w1, w3, w2, self.h_save,
                             self.y_disp, self.ws_fwd)

    def combine(self, weights: Optional[torch.Tensor] = None):
        B.moe_combine(self.y_disp, self.dest_row, self.weights if weights is None else weights,
                      self.y)

    # ---- loss-side operators ----------------------------------------------------
    def balance(self, lam: float):
        """Eq. 3 balance term of this batch from the gate logits and the
        demand counts of the last dispatch; keeps its dprobs coefficient for
        the gate backward.  Returns the [1] loss tensor."""
        if self.balance_loss is None:
            self.balance_loss = torch.empty(1, dtype=torch.float32, device=self.dev)
            self.dprob_coef = torch.empty(self.E, dtype=torch.float32, device=self.dev)
            self.ws_balance = B.workspace(B.moe_balance_workspace_bytes(self.T, self.E), self.dev)
        B.moe_balance_fwd(self.logits, self.counts, self.k, lam, self.balance_loss,
                          self.dprob_coef, self.ws_balance)
        self._balance_on = True
        return self.balance_loss

    def aggregate_spec(self, out: Optional[torch.Tensor] = None):
        """AggregateSpec: [T*k, d] predictions of every (token, choice)."""
        if out is None:
            out = torch.empty(self.T * self.k, self.d, dtype=self.dtype, device=self.dev)
        B.moe_aggregate_spec(self.y_disp, self.dest_row, out)
        return out

    def spec_loss(self, target, weights: Optional[torch.Tensor] = None):
        """Eq. 2 with squared error: the [1] loss, with dy_disp and dweights
        written for the backward (in place of combine_bwd)."""
        if self.spec_loss_value is None:
            self.spec_loss_value = torch.empty(1, dtype=torch.float32, device=self.dev)
            self.ws_spec = B.workspace(B.moe_spec_loss_workspace_bytes(self.T), self.dev)
        B.moe_spec_loss(self.y_disp, self.dest_row, self.weights if weights is None else weights,
                        target, self.dy_disp, self.dweights, self.spec_loss_value, self.ws_spec)
        return self.spec_loss_value

    # ---- backward pieces -----------------------------------------------------
    def combine_bwd(self, dy, weights: Optional[torch.Tensor] = None):
        B.moe_combine_bwd(dy, self.y_disp, self.dest_row,
                          self.weights if weights is None else weights, self.dy_disp,
                          self.dweights)

    def ffn_bwd(self, w1, w3, w2, rows: str = "fill"):
        """rows="capacity" zeroes the unfilled rows of dy_disp first, so the
        padding adds nothing to the weight gradients."""
        if rows == "fill":
            r = self.fill
        else:
            r = self.capacity
            B.moe_zero_pad_rows(self.offsets, self.fill, r, self.dy_disp)
        B.moe_expert_ffn_bwd(self.act, self.offsets, r, self.x_disp, self.h_save, w1, w3, w2,
                             self.dy_disp, self.dx_disp, self.dw1, self.dw3, self.dw2,
                             self.ws_bwd)

    def gate_bwd(self, x, renorm: int, ids: Optional[torch.Tensor] = None):
        B.moe_gate_bwd(x, self.logits, self.ids if ids is None else ids, self.dweights, renorm,
                       self.dlogits, self.dw_g, self.ws_gate_bwd,
                       dprob_coef=self.dprob_coef if self._balance_on else None)

    def dispatch_bwd(self, w_g=None):
        if w_g is not None:
            B.moe_dispatch_bwd(self.dx_disp, self.dest_row, self.E, self.dlogits, w_g, self.dx)
        else:
            B.moe_dispatch_bwd(self.dx_disp, self.dest_row, self.E, None, None, self.dx)

    # ---- whole layer ---------------------------------------------------------
    def _capacity(self, capacity, ids, counts_from_batch):
        kind, num, den = capacity
        if kind == "static":
            self.capacity_static(num, den)
        elif kind == "policy":
            pass            # capacity and offsets uploaded by a CapacityPolicy
        else:
            if counts_from_batch:
                self.count(ids)
            self.capacity_dynamic(num, den)

    def forward(self, x, w1, w3, w2, *, w_g=None, bias=None, renorm=0, ids=None, weights=None,
                capacity=("dynamic", 1, 1), counts_from_batch=True, rows="fill",
                balance: Optional[float] = None):
        """gate (or cached ids) -> [count ->] capacity -> dispatch -> FFN -> combine.

        capacity = ("static", num, den) | ("dynamic", num, den) | ("policy",
        1, 1); a dynamic rule uses this batch's counts when counts_from_batch,
        else the counts left in self.counts by the previous dispatch (a lagged
        capacity update); "policy" uses capacities a CapacityPolicy uploaded.
        balance = lambda adds the Eq. 3 balance term (self.balance_loss) and
        its gradient to the gate backward."""
        self._balance_on = False
        if ids is None:
            self.gate(x, w_g, bias, renorm)
            ids, weights = self.ids, self.weights
        self._capacity(capacity, ids, counts_from_batch)
        self.dispatch(x, ids)
        if balance is not None:
            self.balance(balance)
        self.ffn_fwd(w1, w3, w2, rows=rows)
        self.combine(weights)
        return self.y

    def forward_cached(self, x, w1, w3, w2, *, cached, cache_out, unchanged, w_g, bias=None,
                       renorm=0, capacity=("dynamic", 1, 1), gate_stream=None, rows="fill"):
        """Forward with sample assignment caching on (Section 4.2): the expert
        batches are built from the cached picks while the gate runs on
        gate_stream; the combine waits for the gate and weighs the cached
        picks with the fresh probabilities.  The Cache operator counts the
        samples whose picks did not change (added to `unchanged`) and writes
        the fresh picks to cache_out.  cache_out must not be `cached`: the
        dispatch reads the cached picks after the gate (on either stream),
        and the backward (ids=cached, weights=self.cached_weights) reads them
        again, so storing the fresh picks over them would route one set of
        picks and weigh or differentiate another."""
        main = torch.cuda.current_stream(self.dev)
        gs = gate_stream if gate_stream is not None else main
        if cache_out.data_ptr() == cached.data_ptr():
            raise ValueError("cache_out must be a different buffer from cached: the cached "
                             "picks are read by the dispatch and the backward of this step")
        if self.cached_weights is None:
            self.cached_weights = torch.empty(self.T, self.k, dtype=torch.float32,
                                              device=self.dev)
        self._balance_on = False
        ready = torch.cuda.Event()
        ready.record(main)
        with torch.cuda.stream(gs):
            gs.wait_event(ready)
            self.gate(x, w_g, bias, renorm)
            B.moe_cached_weights(self.logits, cached, renorm, self.cached_weights)
            B.moe_cache_update(self.ids, cached, cache_out, unchanged)
            gate_done = torch.cuda.Event()
            gate_done.record(gs)
        self._capacity(capacity, cached, True)
        self.dispatch(x, cached)
        self.ffn_fwd(w1, w3, w2, rows=rows)
        main.wait_event(gate_done)
        self.combine(self.cached_weights)
        return self.y

    def backward(self, x, dy, w1, w3, w2, *, w_g=None, renorm=0, ids=None, weights=None,
                 rows="fill", target=None):
        """combine_bwd (or, given target, the Eq. 2 specification loss in its
        place) -> gate backward -> FFN backward -> dispatch backward.  The
        gate backward needs only dweights, so it runs before the FFN
        backward, whose last product (dx_disp) the dispatch backward then
        reads straight after it was written."""
        if target is not None:
            self.spec_loss(target, self.weights if weights is None else weights)
        else:
            self.combine_bwd(dy, self.weights if weights is None else weights)
        if w_g is not None:
            self.gate_bwd(x, renorm, ids)
        self.ffn_bwd(w1, w3, w2, rows=rows)
        self.dispatch_bwd(w_g)
        return self.dx
