"""Plain, slow, step-by-step CPU definition of one capacity-bounded top-k MoE
layer, forward and backward.  TEST INFRASTRUCTURE ONLY (see the package
docstring): nothing in the product path imports this module.

Paper passages followed (Kossmann, Jia, Aiken, MLSys 2022):

* Algorithm 1 (MoE forward pass with top-k gating): gate scores, arg-top-k,
  normalised weights of the picks, weighted sum of the picked experts.
* Eq. 1 (cooperation loss): the layer output is the gate-weighted sum of
  expert outputs.
* Section 4.1 (dynamic capacity factors) with Eq. 4: capacity
  C = alpha * batch * k / n, samples beyond an expert's capacity are dropped
  (no forward contribution, zero gradient), the first entries of an expert's
  tensor are the ones filled; the per-expert assigned-sample count is the
  model metric that dynamic capacities are derived from.
* Section 4.2 (sample assignment caching): previously computed assignments
  replace the gate's output when building the expert batches.

Precision: every step is evaluated in float64.  For a bf16 layer the values
are rounded to bf16 (round to nearest even) at the points the kernels store
them: H (saved pre-activation, or H1/H3 for the gated FFN), A = act(H), Y,
the layer output y, dy_disp, dH (dH1/dH3) and dx_disp / dx.  Gate logits,
probabilities and combine weights are float32 values; every dW is float32.
For an fp32 layer nothing is rounded below float64 except the fp32 logits
that decide routing.

Readings of the paper taken here (each is stated where it is used):
R1 k=1 keeps the raw softmax probability as the weight, k>=2 renormalises
   the picked probabilities (the `renorm` flag); R2 top-k is taken on the
   fp32 logits, ties to the lower expert index; R3 capacity rounds up, in
   exact integer arithmetic, clamped to [cap_min, T]; R4 slot priority is
   all first choices in token order, then all second choices, ...;
R5 dropped assignments contribute nothing and get zero gradient, a token
   with nothing kept outputs 0; R6 no bias inside the expert FFN.

Parity pins for every function live in tests/test_oracle_*.py.
"""
from __future__ import annotations

import math
from typing import Dict, Optional, Tuple

import numpy as np

__all__ = [
    "STATUS_BAD_ID", "STATUS_DUP_ID", "STATUS_REGION",
    "bf16_to_f64", "round_bf16", "round_to", "as_f64",
    "gate_logits", "topk", "softmax", "gate_weights",
    "validate_assignments", "count_assignments",
    "capacity_static", "capacity_dynamic", "exclusive_offsets",
    "assign_slots", "dispatch_rows",
    "act_fwd", "act_grad", "ffn_rows_fwd", "ffn_rows_bwd", "ffn_dw_slices",
    "topk_alternatives",
    "combine", "combine_bwd", "gate_bwd", "dispatch_bwd",
    "route", "layer_forward", "layer_backward",
]

STATUS_BAD_ID = 1    # a cached expert id outside [0, E)
STATUS_DUP_ID = 2    # the same expert twice in one token's row
STATUS_REGION = 4    # an expert's capacity region does not fit its rows


# ----------------------------------------------------------------------------
# number formats
# ----------------------------------------------------------------------------
def bf16_to_f64(u16: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact float64 values."""
    u32 = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u32.view(np.float32).astype(np.float64)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even).

    bf16 keeps 8 significant bits: write a = m * 2**e with 0.5 <= |m| < 1,
    round m * 2**8 to the nearest integer (half to even) and scale back.
    Finite, normal-range inputs only (the layer never leaves that range)."""
    a = np.asarray(a, dtype=np.float64)
    m, e = np.frexp(a)
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def round_to(a: np.ndarray, dtype: str) -> np.ndarray:
    """Storage rounding of a layer tensor: bf16 layers round, fp32 layers
    are kept in float64 (the comparison tolerance covers fp32 storage)."""
    return round_bf16(a) if dtype == "bf16" else np.asarray(a, dtype=np.float64)


def as_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """A stored layer tensor (bf16 bits or float32) as float64 values."""
    if dtype == "bf16":
        return bf16_to_f64(a)
    return np.asarray(a, dtype=np.float64)


def _f32(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64).astype(np.float32)


# ----------------------------------------------------------------------------
# gate: Algorithm 1, steps score <- G(x), indices <- argmax_k, w <- normalize
# ----------------------------------------------------------------------------
def gate_logits(x: np.ndarray, w_g: np.ndarray, bias: Optional[np.ndarray]) -> np.ndarray:
    """G(x) for a linear gate: l[t,e] = sum_i x[t,i] w_g[e,i] + b[e].
    float64 accumulation, result rounded once to float32."""
    l = x @ w_g.T
    if bias is not None:
        l = l + np.asarray(bias, dtype=np.float64)[None, :]
    return _f32(l)


def topk(logits: np.ndarray, k: int) -> np.ndarray:
    """argmax_k of Algorithm 1 (reading R2): k rounds of 'take the largest
    remaining logit'; among equal logits the lower expert index wins.
    Logits are compared as the float32 values the kernels compare."""
    l = np.asarray(logits, dtype=np.float32).astype(np.float64)
    if np.isnan(l).any():
        raise ValueError("NaN logit")
    T, E = l.shape
    if not 1 <= k <= E:
        raise ValueError("k out of range")
    avail = np.ones((T, E), dtype=bool)
    ids = np.empty((T, k), dtype=np.int32)
    rows = np.arange(T)
    for j in range(k):
        best = np.where(avail, l, -np.inf).max(axis=1)
        cand = avail & (l == best[:, None])
        pick = np.argmax(cand, axis=1)            # first candidate = lowest index
        ids[:, j] = pick
        avail[rows, pick] = False
    return ids


def softmax(logits: np.ndarray) -> np.ndarray:
    """Gate probabilities p = exp(l - max l) / sum exp(l - max l), float64."""
    l = np.asarray(logits, dtype=np.float64)
    z = np.exp(l - l.max(axis=1, keepdims=True))
    return z / z.sum(axis=1, keepdims=True)


def gate_weights(p: np.ndarray, ids: np.ndarray, renorm: int) -> np.ndarray:
    """normalize(score[indices]) of Algorithm 1 (reading R1): with renorm the
    picked probabilities are divided by their sum, else the raw probability
    of each pick is its weight.  Weights are fixed before capacity, so a drop
    never re-normalises the survivors.  On the cached path (Section 4.2) an id
    outside [0, E) is not a pick: its weight is 0 and it is left out of the
    sum (the gate never produces one).  Returned as float32 values."""
    sel = _picked_probs(p, ids)
    if renorm:
        tot = sel.sum(axis=1, keepdims=True)
        sel = np.divide(sel, tot, out=np.zeros_like(sel), where=tot > 0)
    return _f32(sel)


def _picked_probs(p: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """p[t, ids[t,j]], and 0 where ids[t,j] is not an expert index."""
    idx = np.asarray(ids).astype(np.int64)
    ok = (idx >= 0) & (idx < p.shape[1])
    sel = np.take_along_axis(p, np.where(ok, idx, 0), axis=1)
    return np.where(ok, sel, 0.0)


# ----------------------------------------------------------------------------
# per-expert load (the Section 4.1 model metric) and capacities (Eq. 4)
# ----------------------------------------------------------------------------
def validate_assignments(ids: np.ndarray, E: int) -> Tuple[np.ndarray, int]:
    """Which (t, j) assignments are live, and the status bits.

    An id outside [0, E) is not an assignment (bit 1).  A token naming an
    expert it already named at a lower j gets it once: the later copy is not
    an assignment (bit 2).  The gate never produces either; cached ids can."""
    ids = np.asarray(ids)
    valid = (ids >= 0) & (ids < E)
    status = STATUS_BAD_ID if (~valid).any() else 0
    dup = np.zeros_like(valid)
    for j in range(1, ids.shape[1]):
        for jj in range(j):
            dup[:, j] |= valid[:, j] & valid[:, jj] & (ids[:, j] == ids[:, jj])
    if dup.any():
        status |= STATUS_DUP_ID
    return valid & ~dup, status


def count_assignments(ids: np.ndarray, E: int) -> np.ndarray:
    """counts[e] = number of live assignments to expert e, before capacity:
    how many samples the gate assigns to each expert (Section 4.1)."""
    live, _ = validate_assignments(ids, E)
    return np.bincount(np.asarray(ids)[live].astype(np.int64), minlength=E).astype(np.int64)


def _ceil_div(a: int, b: int) -> int:
    return -((-a) // b)


def capacity_static(T: int, k: int, E: int, num: int, den: int,
                    cap_min: int = 0) -> np.ndarray:
    """Eq. 4, C = alpha * batch * k / n with alpha = num/den, rounded up in
    exact integer arithmetic and clamped to [cap_min, T] (reading R3); the
    same C for every expert."""
    c = _ceil_div(num * T * k, den * E)
    c = min(T, max(cap_min, c))
    return np.full(E, c, dtype=np.int64)


def capacity_dynamic(counts: np.ndarray, T: int, num: int, den: int,
                     cap_min: int = 0) -> np.ndarray:
    """Dynamic capacity factors (Section 4.1): each expert's capacity follows
    its own observed load, C_e = ceil(num/den * counts[e]) in exact integer
    arithmetic, clamped to [cap_min, T].  num/den = 1 gives exact capacity."""
    out = np.empty(len(counts), dtype=np.int64)
    for e, c in enumerate(counts):
        v = _ceil_div(num * int(c), den)
        out[e] = min(T, max(cap_min, v))
    return out


def exclusive_offsets(capacity: np.ndarray, align: int = 1) -> np.ndarray:
    """Row layout of the grouped expert buffer (a storage choice, not part of
    the method): expert e's region starts at offsets[e] = the sum, over
    experts before e, of their capacities each rounded up to a multiple of
    `align` rows; offsets[E] = the rows the layout takes.  align = 1 packs
    the regions."""
    cap = np.asarray(capacity, dtype=np.int64)
    sizes = (cap + align - 1) // align * align
    off = np.zeros(len(cap) + 1, dtype=np.int64)
    off[1:] = np.cumsum(sizes)
    return off


# ----------------------------------------------------------------------------
# slot assignment and dispatch (GroupBy; Section 4.1 drop rule)
# ----------------------------------------------------------------------------
def assign_slots(ids: np.ndarray, E: int, capacity: np.ndarray,
                 offsets: np.ndarray, rows_alloc: int) -> Dict[str, np.ndarray]:
    """Place every live assignment in its expert's tensor.

    Expert e owns rows [offsets[e], offsets[e] + C_e) of the grouped buffer.
    The buffer is filled from its first entry (Section 4.1); priority is
    all first choices in token order, then all second choices, ... (R4).
    An assignment whose position is >= C_e is dropped (dest_row = -1).
    A capacity region that overlaps the next expert's or runs past rows_alloc
    is cut to what fits, with status bit 4.

    Returns counts (demand, before capacity), fill (kept per expert),
    dest_row [T,k] (row of the grouped buffer or -1), src [rows_alloc]
    (t*k + j of the row's assignment or -1), pos [T,k] (rank within the
    expert, -1 if not live), status."""
    ids = np.asarray(ids)
    T, k = ids.shape
    cap = np.asarray(capacity, dtype=np.int64)
    off = np.asarray(offsets, dtype=np.int64)
    live, status = validate_assignments(ids, E)
    cap_eff = np.zeros(E, dtype=np.int64)
    for e in range(E):
        if off[e] < 0:
            room = 0
        else:
            room = min(int(cap[e]), int(off[e + 1] - off[e]), int(rows_alloc - off[e]))
        cap_eff[e] = max(0, room)
        if cap_eff[e] < cap[e]:
            status |= STATUS_REGION
    ctr = np.zeros(E, dtype=np.int64)
    pos = np.full((T, k), -1, dtype=np.int64)
    dest = np.full((T, k), -1, dtype=np.int64)
    for j in range(k):                      # first choices before second ...
        col = ids[:, j].astype(np.int64)
        lv = live[:, j]
        tok = np.nonzero(lv)[0]             # ... and tokens in index order
        e_of = col[tok]
        order = np.argsort(e_of, kind="stable")
        e_sorted = e_of[order]
        start = np.searchsorted(e_sorted, np.arange(E), side="left")
        rank_sorted = np.arange(len(order)) - start[e_sorted]
        rank = np.empty(len(order), dtype=np.int64)
        rank[order] = rank_sorted
        p = ctr[e_of] + rank
        pos[tok, j] = p
        keep = p < cap_eff[e_of]
        dest[tok[keep], j] = off[e_of[keep]] + p[keep]
        ctr += np.bincount(e_of, minlength=E)
    counts = ctr
    fill = np.minimum(counts, cap_eff)
    src = np.full(rows_alloc, -1, dtype=np.int64)
    tt, jj = np.nonzero(dest >= 0)
    src[dest[tt, jj]] = tt * k + jj
    return dict(counts=counts, fill=fill, dest_row=dest, src=src, pos=pos,
                status=status, cap_eff=cap_eff)


def dispatch_rows(x: np.ndarray, dest_row: np.ndarray, rows_alloc: int) -> np.ndarray:
    """Grouped buffer x_disp[dest_row[t,j]] = x[t] (an exact copy); rows not
    written are NaN (unspecified in the kernels, never read)."""
    out = np.full((rows_alloc, x.shape[1]), np.nan)
    tt, jj = np.nonzero(dest_row >= 0)
    out[dest_row[tt, jj]] = x[tt]
    return out


# ----------------------------------------------------------------------------
# expert FFN (E_e(x) of Algorithm 1), forward and backward
# ----------------------------------------------------------------------------
_SQRT_2_OVER_PI = math.sqrt(2.0 / math.pi)


def act_fwd(h: np.ndarray, act: str) -> np.ndarray:
    """relu(h); gelu with the tanh approximation,
    0.5 h (1 + tanh(sqrt(2/pi) (h + 0.044715 h^3))); silu(h) = h sigmoid(h)."""
    if act == "relu":
        return np.maximum(h, 0.0)
    if act == "gelu_tanh":
        return 0.5 * h * (1.0 + np.tanh(_SQRT_2_OVER_PI * (h + 0.044715 * h ** 3)))
    if act == "silu":
        return h / (1.0 + np.exp(-h))
    raise ValueError(act)


def act_grad(h: np.ndarray, act: str) -> np.ndarray:
    """Derivative of act_fwd; relu'(0) = 0."""
    if act == "relu":
        return (h > 0).astype(np.float64)
    if act == "gelu_tanh":
        u = _SQRT_2_OVER_PI * (h + 0.044715 * h ** 3)
        th = np.tanh(u)
        du = _SQRT_2_OVER_PI * (1.0 + 3 * 0.044715 * h ** 2)
        return 0.5 * (1.0 + th) + 0.5 * h * (1.0 - th ** 2) * du
    if act == "silu":
        s = 1.0 / (1.0 + np.exp(-h))
        return s * (1.0 + h * (1.0 - s))
    raise ValueError(act)


def ffn_rows_fwd(X: np.ndarray, e_of_row: np.ndarray, w1: np.ndarray,
                 w3: Optional[np.ndarray], w2: np.ndarray, act: str,
                 dtype: str) -> Dict[str, np.ndarray]:
    """Expert FFN on rows X (float64 values of the stored inputs), row r
    through expert e_of_row[r].  Weights are float64 values,
    w1/w3 [E, f, d], w2 [E, d, f].

    relu / gelu:  H = X W1^T,  A = act(H),  Y = A W2^T
    swiglu:       H1 = X W1^T, H3 = X W3^T, A = silu(H1) * H3, Y = A W2^T
    Each of H (H1, H3), A and Y is rounded to the storage type; A is taken
    from the rounded H.  No bias (R6)."""
    R = X.shape[0]
    f = w1.shape[1]
    d = w2.shape[1]
    H = np.zeros((R, f))
    H3 = np.zeros((R, f)) if act == "swiglu" else None
    A = np.zeros((R, f))
    Y = np.zeros((R, d))
    for e in np.unique(e_of_row):
        m = e_of_row == e
        Xe = X[m]
        h = round_to(Xe @ w1[e].T, dtype)
        H[m] = h
        if act == "swiglu":
            h3 = round_to(Xe @ w3[e].T, dtype)
            H3[m] = h3
            a = round_to(act_fwd(h, "silu") * h3, dtype)
        else:
            a = round_to(act_fwd(h, act), dtype)
        A[m] = a
        Y[m] = round_to(a @ w2[e].T, dtype)
    return dict(H=H, H3=H3, A=A, Y=Y)


def ffn_rows_bwd(X: np.ndarray, e_of_row: np.ndarray, H: np.ndarray,
                 H3: Optional[np.ndarray], dY: np.ndarray, w1: np.ndarray,
                 w3: Optional[np.ndarray], w2: np.ndarray, act: str,
                 dtype: str, E: int) -> Dict[str, np.ndarray]:
    """Backward of ffn_rows_fwd given dY (the stored dy_disp rows) and the
    saved, rounded H (H1, H3).  A is recomputed from the saved values.

    dA = dY W2;  relu/gelu: dH = dA * act'(H);
    swiglu: dH1 = dA * H3 * silu'(H1), dH3 = dA * silu(H1);
    dW2_e = dY_e^T A_e, dW1_e = dH1_e^T X_e, dW3_e = dH3_e^T X_e (float32
    arrays: summed in float64, rounded once);
    dX = dH1 W1 + dH3 W3 (one rounding).  An expert with no rows has dW = 0."""
    f = w1.shape[1]
    d = w2.shape[1]
    R = X.shape[0]
    dX = np.zeros((R, d))
    dH = np.zeros((R, f))
    dH3 = np.zeros((R, f)) if act == "swiglu" else None
    # weight gradients are float32 values: each is summed in float64 and
    # rounded once to float32 (stored as float32 arrays)
    dW1 = np.zeros((E, f, d), dtype=np.float32)
    dW3 = np.zeros((E, f, d), dtype=np.float32) if act == "swiglu" else None
    dW2 = np.zeros((E, d, f), dtype=np.float32)
    for e in np.unique(e_of_row):
        m = e_of_row == e
        Xe, dYe, h = X[m], dY[m], H[m]
        dA = dYe @ w2[e]
        if act == "swiglu":
            h3 = H3[m]
            a = round_to(act_fwd(h, "silu") * h3, dtype)
            g1 = round_to(dA * h3 * act_grad(h, "silu"), dtype)
            g3 = round_to(dA * act_fwd(h, "silu"), dtype)
            dH[m], dH3[m] = g1, g3
            dW3[e] = _f32(g3.T @ Xe)
            dX[m] = round_to(g1 @ w1[e] + g3 @ w3[e], dtype)
        else:
            a = round_to(act_fwd(h, act), dtype)
            g1 = round_to(dA * act_grad(h, act), dtype)
            dH[m] = g1
            dX[m] = round_to(g1 @ w1[e], dtype)
        dW1[e] = _f32(g1.T @ Xe)
        dW2[e] = _f32(dYe.T @ a)
    return dict(dX=dX, dH=dH, dH3=dH3, dW1=dW1, dW2=dW2, dW3=dW3)


def ffn_dw_slices(X: np.ndarray, dY: np.ndarray, w1_e: np.ndarray,
                  w3_e: Optional[np.ndarray], w2_e: np.ndarray, act: str, dtype: str,
                  cols: np.ndarray) -> Dict[str, np.ndarray]:
    """Slices of one expert's weight gradients, by the same definitions as
    ffn_rows_bwd restricted to hidden units `cols` (for checks at sizes where
    the full gradient is too costly): dW2[:, cols] (d x n), dW1[cols, :] and
    dW3[cols, :] (n x d).  X, dY are all of the expert's rows."""
    J = np.asarray(cols, dtype=np.int64)
    h = round_to(X @ w1_e[J].T, dtype)
    dA = dY @ w2_e[:, J]
    if act == "swiglu":
        h3 = round_to(X @ w3_e[J].T, dtype)
        a = round_to(act_fwd(h, "silu") * h3, dtype)
        g1 = round_to(dA * h3 * act_grad(h, "silu"), dtype)
        g3 = round_to(dA * act_fwd(h, "silu"), dtype)
    else:
        a = round_to(act_fwd(h, act), dtype)
        g1 = round_to(dA * act_grad(h, act), dtype)
        g3 = None
    out = dict(dW2=_f32(dY.T @ a), dW1=_f32(g1.T @ X))
    out["dW3"] = None if g3 is None else _f32(g3.T @ X)
    return out


def topk_alternatives(logits: np.ndarray, k: int, tol: float) -> list:
    """Valid top-k lists of one token when logits closer than `tol` are taken
    as tied (their order is not decided by the arithmetic): start from the
    strict order (ties to the lower index) and apply every adjacent swap of
    near-tied logits among the positions that can reach the first k picks."""
    l = np.asarray(logits, dtype=np.float64)
    order = list(np.argsort(-l, kind="stable"))
    # positions that can reach the first k picks: the first k, extended
    # through any chain of near ties across the k-th / (k+1)-th boundary
    r = k
    while r < len(order) and abs(l[order[r - 1]] - l[order[r]]) <= tol:
        r += 1
    seen = {tuple(order)}
    frontier = [order]
    while frontier:
        nxt = []
        for o in frontier:
            for p in range(min(r, len(o)) - 1):
                if abs(l[o[p]] - l[o[p + 1]]) <= tol:
                    q = list(o)
                    q[p], q[p + 1] = q[p + 1], q[p]
                    if tuple(q) not in seen:
                        seen.add(tuple(q))
                        nxt.append(q)
        frontier = nxt
    return sorted({tuple(o[:k]) for o in seen})


# ----------------------------------------------------------------------------
# combine (Aggregate: Algorithm 1's weighted sum, Eq. 1) and its backward
# ----------------------------------------------------------------------------
def combine(Y_disp: np.ndarray, dest_row: np.ndarray, weights: np.ndarray,
            dtype: str) -> np.ndarray:
    """y[t] = sum over kept j, in order j = 0..k-1, of w[t,j] * Y[dest_row[t,j]];
    a token with nothing kept outputs 0 (R5).  One rounding at the end."""
    T, k = dest_row.shape
    y = np.zeros((T, Y_disp.shape[1]))
    w = np.asarray(weights, dtype=np.float64)
    for j in range(k):
        kept = dest_row[:, j] >= 0
        y[kept] += w[kept, j, None] * Y_disp[dest_row[kept, j]]
    return round_to(y, dtype)


def combine_bwd(dy: np.ndarray, Y_disp: np.ndarray, dest_row: np.ndarray,
                weights: np.ndarray, dtype: str) -> Tuple[np.ndarray, np.ndarray]:
    """dweights[t,j] = <dy[t], Y[dest_row[t,j]]> if kept else 0 (float32);
    dy_disp[dest_row[t,j]] = w[t,j] * dy[t] (rounded).  Rows of dy_disp with
    no kept assignment are NaN (never read)."""
    T, k = dest_row.shape
    dw = np.zeros((T, k))
    dy_disp = np.full_like(Y_disp, np.nan)
    w = np.asarray(weights, dtype=np.float64)
    for j in range(k):
        kept = dest_row[:, j] >= 0
        r = dest_row[kept, j]
        dw[kept, j] = np.einsum("td,td->t", dy[kept], Y_disp[r])
        dy_disp[r] = round_to(w[kept, j, None] * dy[kept], dtype)
    return _f32(dw).astype(np.float64), dy_disp


# ----------------------------------------------------------------------------
# gate backward and dispatch backward
# ----------------------------------------------------------------------------
def gate_bwd(logits: np.ndarray, ids: np.ndarray, dweights: np.ndarray,
             renorm: int, x: np.ndarray,
             dprob_coef: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Gradient through normalize(score[indices]) and the softmax to the gate
    logits, then to the gate weights.

    raw:    g_j = dw_j
    renorm: w_j = p_j / S with S = sum_j p_j, so g_j = (dw_j - sum_i dw_i w_i) / S
    dp[t,e] = sum_j [ids[t,j] = e] g_j (+ dprob_coef[e], a gradient that is
    the same for every token, such as Eq. 3's balance term);
    dl = p * (dp - <dp, p>);
    dW_g[e,i] = sum_t dl[t,e] x[t,i].  dl and dW_g are float32."""
    p = softmax(logits)
    T, E = p.shape
    idx = ids.astype(np.int64)
    ok = (idx >= 0) & (idx < E)          # an id outside [0, E) is no pick
    sel = _picked_probs(p, idx)
    dw = np.asarray(dweights, dtype=np.float64)
    if renorm:
        S = sel.sum(axis=1, keepdims=True)
        w = np.divide(sel, S, out=np.zeros_like(sel), where=S > 0)
        g = np.divide(dw - (dw * w).sum(axis=1, keepdims=True), S,
                      out=np.zeros_like(sel), where=S > 0)
    else:
        g = dw
    dp = np.zeros((T, E))
    for j in range(idx.shape[1]):
        rows = np.nonzero(ok[:, j])[0]
        dp[rows, idx[rows, j]] += g[rows, j]
    if dprob_coef is not None:
        dp += np.asarray(dprob_coef, dtype=np.float64)[None, :]
    dl = p * (dp - (dp * p).sum(axis=1, keepdims=True))
    dl32 = _f32(dl).astype(np.float64)
    dwg = _f32(dl32.T @ x).astype(np.float64)
    return dl32, dwg


def dispatch_bwd(dx_disp: np.ndarray, dest_row: np.ndarray,
                 dl: Optional[np.ndarray], w_g: Optional[np.ndarray],
                 dtype: str) -> np.ndarray:
    """dx[t] = sum over kept j of dx_disp[dest_row[t,j]] (+ dl[t] . W_g when
    the gate ran), one rounding at the end."""
    T, k = dest_row.shape
    dx = np.zeros((T, dx_disp.shape[1]))
    for j in range(k):
        kept = dest_row[:, j] >= 0
        dx[kept] += dx_disp[dest_row[kept, j]]
    if dl is not None:
        dx += dl @ w_g
    return round_to(dx, dtype)


# ----------------------------------------------------------------------------
# whole layer (the composition the kernels are tested against at small sizes)
# ----------------------------------------------------------------------------
def route(x, w_g, bias, k, renorm):
    """Gate part of Algorithm 1: logits, picks, probabilities, weights."""
    logits = gate_logits(x, w_g, bias)
    ids = topk(logits, k)
    p = softmax(logits)
    w = gate_weights(p, ids, renorm)
    return dict(logits=logits, ids=ids, p=p, weights=w)


def layer_forward(x, w1, w3, w2, act, dtype, ids, weights, capacity,
                  rows_alloc, E, align: int = 1) -> Dict[str, np.ndarray]:
    """Dispatch -> per-expert FFN -> combine for given ids/weights (gate
    output or cached) and capacities, in the row layout of
    exclusive_offsets(capacity, align).  All tensors are float64 values."""
    off = exclusive_offsets(capacity, align)
    s = assign_slots(ids, E, capacity, off, rows_alloc)
    x_disp = dispatch_rows(x, s["dest_row"], rows_alloc)
    f = w1.shape[1]
    d = w2.shape[1]
    H = np.full((rows_alloc, f), np.nan)
    H3 = np.full((rows_alloc, f), np.nan) if act == "swiglu" else None
    A = np.full((rows_alloc, f), np.nan)
    Y = np.full((rows_alloc, d), np.nan)
    rows = np.concatenate([np.arange(off[e], off[e] + s["fill"][e]) for e in range(E)]
                          ).astype(np.int64)
    e_of = np.concatenate([np.full(s["fill"][e], e) for e in range(E)]).astype(np.int64)
    if len(rows):
        r = ffn_rows_fwd(x_disp[rows], e_of, w1, w3, w2, act, dtype)
        H[rows], A[rows], Y[rows] = r["H"], r["A"], r["Y"]
        if H3 is not None:
            H3[rows] = r["H3"]
    y = combine(Y, s["dest_row"], weights, dtype)
    return dict(offsets=off, x_disp=x_disp, H=H, H3=H3, A=A, Y=Y, y=y,
                rows=rows, e_of=e_of, **s)


def layer_backward(fw, x, dy, w1, w3, w2, act, dtype, ids, weights, E,
                   logits=None, renorm=0, w_g=None, target=None,
                   dprob_coef=None) -> Dict[str, np.ndarray]:
    """combine_bwd -> FFN backward -> gate backward -> dispatch backward.

    With `target`, the specification loss of Eq. 2 (squared error) takes the
    place of combine_bwd and `dy` is not used; `dprob_coef` adds a dprobs
    term shared by every token (Eq. 3's balance term) to the gate backward."""
    spec = None
    if target is not None:
        from .losses import spec_loss
        spec, dw, dy_disp = spec_loss(fw["Y"], fw["dest_row"], weights, target, dtype)
    else:
        dw, dy_disp = combine_bwd(dy, fw["Y"], fw["dest_row"], weights, dtype)
    rows, e_of = fw["rows"], fw["e_of"]
    d = x.shape[1]
    dx_disp = np.full((fw["x_disp"].shape[0], d), np.nan)
    f = w1.shape[1]
    if len(rows):
        b = ffn_rows_bwd(fw["x_disp"][rows], e_of, fw["H"][rows],
                         None if fw["H3"] is None else fw["H3"][rows],
                         dy_disp[rows], w1, w3, w2, act, dtype, E)
        dx_disp[rows] = b["dX"]
        dW1, dW2, dW3 = b["dW1"], b["dW2"], b["dW3"]
    else:
        dW1 = np.zeros((E, f, d), dtype=np.float32)
        dW2 = np.zeros((E, d, f), dtype=np.float32)
        dW3 = np.zeros((E, f, d), dtype=np.float32) if act == "swiglu" else None
    dl = dwg = None
    if logits is not None:
        dl, dwg = gate_bwd(logits, ids, dw, renorm, x, dprob_coef)
    dx = dispatch_bwd(dx_disp, fw["dest_row"], dl, w_g, dtype)
    return dict(dweights=dw, dy_disp=dy_disp, dx_disp=dx_disp, dW1=dW1,
                dW2=dW2, dW3=dW3, dlogits=dl, dw_g=dwg, dx=dx, spec_loss=spec)
