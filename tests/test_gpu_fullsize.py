"""Full-size GPU parity on every workload, in the launch configuration
bench.py times (same buffers, same call sequence, same capacity rules).

Routing is compared bit-exactly with the oracle run over all tokens:
gate ids (where the oracle's fp32 logits put two candidates closer than
8 ulps of the largest |logit|, both orders are valid and the kernel's pick
must be one of the oracle's enumerated alternatives), counts, capacities,
fill, dest_row and src.

Float outputs, two ways:
* end to end on sampled tokens: at least two kept rows of every non-empty
  expert plus random tokens (x_disp, H, A, Y, y, dweights, dy_disp, dx_disp,
  dlogits, dx from the oracle's own forward of those rows), and four
  sampled hidden units of the weight gradients of every non-empty expert
  (dW1, dW2, dW3 slices from all of that expert's rows);
* stage-wise over all tokens: the oracle step fed the kernel's input to that
  step (itself checked on the samples above): y from the kernel's y_disp;
  dweights and dy_disp from the kernel's y_disp; dlogits and dW_g from the
  kernel's dweights; dx from the kernel's dx_disp.
Expert weights are converted to float64 one expert at a time and dropped
after use, so the largest layers fit in host memory."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import NEAR_TIE, RTOL, assert_close, dev, relu_kink_bound, to_dev, to_np, torch_dtype
from paper_2205_01848_amd import MoELayer, rows_alloc_for
from paper_2205_01848_amd.layer import ROW_ALIGN

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _ffn_rows_per_expert(Xr, e_of, I, dt, act):
    """O.ffn_rows_fwd on rows of several experts, one expert's weights in
    float64 at a time."""
    R, f, d = len(Xr), I.w1.shape[1], I.w1.shape[2]
    out = dict(H=np.zeros((R, f)), H3=np.zeros((R, f)) if act == "swiglu" else None,
               A=np.zeros((R, f)), Y=np.zeros((R, d)))
    for e in np.unique(e_of):
        m = e_of == e
        w1 = O.as_f64(I.w1[e], dt)[None]
        w3 = O.as_f64(I.w3[e], dt)[None] if act == "swiglu" else None
        w2 = O.as_f64(I.w2[e], dt)[None]
        fr = O.ffn_rows_fwd(Xr[m], np.zeros(int(m.sum()), np.int64), w1, w3, w2, act, dt)
        for n in out:
            if out[n] is not None:
                out[n][m] = fr[n]
    return out


def _ffn_rows_bwd_per_expert(Xr, e_of, fr, dYr, I, dt, act):
    """O.ffn_rows_bwd's dX on rows of several experts, one expert at a time."""
    dX = np.zeros_like(Xr)
    for e in np.unique(e_of):
        m = e_of == e
        w1 = O.as_f64(I.w1[e], dt)[None]
        w3 = O.as_f64(I.w3[e], dt)[None] if act == "swiglu" else None
        w2 = O.as_f64(I.w2[e], dt)[None]
        b = O.ffn_rows_bwd(Xr[m], np.zeros(int(m.sum()), np.int64), fr["H"][m],
                           None if fr["H3"] is None else fr["H3"][m], dYr[m], w1, w3, w2, act,
                           dt, 1)
        dX[m] = b["dX"]
    return dX


def _run_gpu(wl, I, rule):
    dt = wl.dtype
    kind, num, den = rule
    R = rows_alloc_for(kind, wl.T, wl.k, wl.E, num, den)
    L = MoELayer(wl.T, wl.d, wl.E, wl.k, wl.f, wl.act, torch_dtype(dt), R, backward=wl.backward,
                 gate=wl.gate == "linear")
    x, w1, w2 = to_dev(I.x, dt), to_dev(I.w1, dt), to_dev(I.w2, dt)
    w3 = to_dev(I.w3, dt) if I.w3 is not None else None
    if wl.gate == "linear":
        wg = to_dev(I.w_g, dt)
        bias = torch.from_numpy(I.bias).to(dev()) if I.bias is not None else None
        L.forward(x, w1, w3, w2, w_g=wg, bias=bias, renorm=wl.renorm, capacity=rule)
        if wl.backward:
            L.backward(x, to_dev(I.dy, dt), w1, w3, w2, w_g=wg, renorm=wl.renorm)
    else:
        ids = torch.from_numpy(I.ids).to(dev())
        cw = torch.from_numpy(I.cw).to(dev())
        L.forward(x, w1, w3, w2, ids=ids, weights=cw, capacity=rule)
        if wl.backward:
            L.backward(x, to_dev(I.dy, dt), w1, w3, w2, weights=cw)
    torch.cuda.synchronize()
    return L, R


def _rows(t, dt, idx):
    """Selected rows of a device tensor as float64 numpy."""
    return to_np(t[torch.from_numpy(np.asarray(idx, dtype=np.int64)).to(t.device)])


def _check(name, run):
    wl = W.config(name)
    I = W.make_inputs(wl)
    rule = wl.capacity[run]
    dt, rt = wl.dtype, RTOL[wl.dtype]
    L, R = _run_gpu(wl, I, rule)
    print(f"full size {name} run {run}: T={wl.T} d={wl.d} E={wl.E} k={wl.k} f={wl.f}", flush=True)
    X = O.as_f64(I.x, dt)

    # ---- routing: oracle over all tokens --------------------------------------
    gpu_ids = to_np(L.ids) if wl.gate == "linear" else I.ids.astype(np.int64)
    logits = None
    if wl.gate == "linear":
        logits = O.gate_logits(X, O.as_f64(I.w_g, dt), I.bias)
        ids = O.topk(logits, wl.k).astype(np.int64)
        tol = NEAR_TIE * float(np.abs(logits).max())
        diff = np.nonzero((gpu_ids != ids).any(axis=1))[0]
        for t in diff:   # only certified near ties may differ, and only to a valid pick
            alts = O.topk_alternatives(logits[t], wl.k, tol)
            assert tuple(int(v) for v in gpu_ids[t]) in alts, f"token {t}: {gpu_ids[t]} not in {alts}"
            ids[t] = gpu_ids[t]
        assert len(diff) <= 4, f"{len(diff)} near-tie tokens resolved differently"
        wts = O.gate_weights(O.softmax(logits), ids, wl.renorm)
        assert_close(to_np(L.logits), logits, 1e-5, "logits")
        assert_close(to_np(L.weights), wts, 1e-5, "weights")
    else:
        ids, wts = I.ids.astype(np.int64), I.cw.astype(np.float64)
    counts = O.count_assignments(ids, wl.E)
    kind, num, den = rule
    cap = (O.capacity_static(wl.T, wl.k, wl.E, num, den) if kind == "static"
           else O.capacity_dynamic(counts, wl.T, num, den))
    off = O.exclusive_offsets(cap, ROW_ALIGN)
    s = O.assign_slots(ids, wl.E, cap, off, R)
    np.testing.assert_array_equal(to_np(L.counts), s["counts"])
    np.testing.assert_array_equal(to_np(L.capacity), cap)
    np.testing.assert_array_equal(to_np(L.offsets), off)
    np.testing.assert_array_equal(to_np(L.fill), s["fill"])
    np.testing.assert_array_equal(to_np(L.dest_row), s["dest_row"])
    np.testing.assert_array_equal(to_np(L.src)[:R], s["src"])
    assert int(L.status.item()) == 0
    dest = s["dest_row"]

    # ---- sampled tokens: two kept rows of every non-empty expert + random ----
    fill = s["fill"]
    nonempty = [e for e in range(wl.E) if fill[e] > 0]
    rng = np.random.default_rng(7)
    picks = []
    for e in nonempty:
        erows = np.arange(off[e], off[e] + fill[e])
        picks.append(s["src"][rng.choice(erows, size=min(2, len(erows)), replace=False)] // wl.k)
    cand = np.nonzero((dest >= 0).any(axis=1))[0]
    picks.append(rng.choice(cand, size=min(24, len(cand)), replace=False))
    dropped = np.nonzero((dest < 0).all(axis=1))[0]
    picks.append(dropped[:4])
    toks = np.unique(np.concatenate(picks)).astype(np.int64)
    tt, jj = np.nonzero(dest[toks] >= 0)
    rows = dest[toks][tt, jj]
    rtok = toks[tt]
    e_of = ids[toks][tt, jj]
    assert set(int(e) for e in e_of) == set(int(e) for e in nonempty)
    Xr = X[rtok]
    # dispatched rows are exact copies
    np.testing.assert_array_equal(_rows(L.x_disp, dt, rows), Xr)
    fr = _ffn_rows_per_expert(Xr, e_of, I, dt, wl.act)
    assert_close(_rows(L.y_disp, dt, rows), fr["Y"], rt, "Y rows")
    # the layer output of the sampled tokens, end to end
    dsub = -np.ones_like(dest[toks])
    dsub[tt, jj] = np.arange(len(rows))
    assert_close(to_np(L.y)[toks], O.combine(fr["Y"], dsub, wts[toks], dt), rt,
                 "y (sampled tokens)")
    # stage-wise over all tokens: combine of the kernel's expert rows
    Yd = to_np(L.y_disp)
    assert_close(to_np(L.y), O.combine(Yd, dest, wts, dt), rt, "y (all tokens, stage-wise)")
    if len(dropped):
        assert (to_np(L.y)[dropped] == 0).all()
    if not wl.backward:
        return
    hs = L.h_save.view(-1, R, wl.f)   # H (GELU) or H1, H3 (SwiGLU), then A = act(H)
    if L.swiglu:
        assert_close(_rows(hs[0], dt, rows), fr["H"], rt, "H1 rows")
        assert_close(_rows(hs[1], dt, rows), fr["H3"], rt, "H3 rows")
    elif wl.act != "relu":
        assert_close(_rows(hs[0], dt, rows), fr["H"], rt, "H rows")
    assert_close(_rows(hs[-1], dt, rows), fr["A"], rt, "A rows")

    # ---- backward on the sampled tokens ----------------------------------------------
    dY = O.as_f64(I.dy, dt)
    dw_ref = np.zeros((len(toks), wl.k))
    dw_ref[tt, jj] = np.einsum("rd,rd->r", dY[rtok], fr["Y"])
    dw_ref = dw_ref.astype(np.float32).astype(np.float64)
    assert_close(to_np(L.dweights)[toks], dw_ref, rt, "dweights")
    dyd = O.round_to(wts[toks][tt, jj][:, None] * dY[rtok], dt)
    assert_close(_rows(L.dy_disp, dt, rows), dyd, rt, "dy_disp rows")
    dXr = _ffn_rows_bwd_per_expert(Xr, e_of, fr, dyd, I, dt, wl.act)
    ok = np.ones(len(rows), dtype=bool)
    if wl.act == "relu":   # relu'(H) is not decided by the arithmetic where H ~ 0
        ok = ~(np.abs(fr["H"]) < 1e-5 * np.sqrt(np.mean(fr["H"] ** 2))).any(axis=1)
        assert (~ok).sum() <= relu_kink_bound(len(rows) * wl.f)
    assert_close(_rows(L.dx_disp, dt, rows)[ok], dXr[ok], rt, "dx_disp rows")
    dl = None
    if wl.gate == "linear":
        dl, _ = O.gate_bwd(logits[toks], ids[toks], dw_ref, wl.renorm, X[toks])
        assert_close(to_np(L.dlogits)[toks], dl, rt, "dlogits")
    dxd = np.zeros((len(rows), wl.d))
    dxd[:] = dXr
    dx_ref = O.dispatch_bwd(dxd, dsub, dl, O.as_f64(I.w_g, dt) if dl is not None else None, dt)
    tok_ok = np.ones(len(toks), dtype=bool)
    tok_ok[tt[~ok]] = False
    assert_close(to_np(L.dx)[toks][tok_ok], dx_ref[tok_ok], rt, "dx (sampled tokens)")

    # ---- stage-wise over all tokens ----------------------------------------------------
    dw_all, dyd_all = O.combine_bwd(dY, Yd, dest, wts, dt)
    del Yd
    dw_gpu = to_np(L.dweights)
    assert_close(dw_gpu, dw_all, rt, "dweights (all tokens, stage-wise)")
    kept_rows = s["src"] >= 0
    assert_close(to_np(L.dy_disp)[:R][kept_rows], dyd_all[kept_rows], rt,
                 "dy_disp (all kept rows, stage-wise)")
    del dyd_all
    dl_all = None
    if wl.gate == "linear":
        dl_all, dwg_all = O.gate_bwd(logits, ids, dw_gpu, wl.renorm, X)
        assert_close(to_np(L.dlogits), dl_all, rt, "dlogits (all tokens, stage-wise)")
        assert_close(to_np(L.dw_g), dwg_all, rt, "dW_g (full, stage-wise)")
    dx_all = O.dispatch_bwd(to_np(L.dx_disp), dest, dl_all,
                            O.as_f64(I.w_g, dt) if dl_all is not None else None, dt)
    assert_close(to_np(L.dx), dx_all, rt, "dx (all tokens, stage-wise)")
    del dx_all

    # ---- weight-gradient slices of every non-empty expert --------------------------------
    for e in nonempty:
        erows = np.arange(off[e], off[e] + fill[e])
        src = s["src"][erows]
        et, ej = src // wl.k, src % wl.k
        Xe = X[et]
        dYe = O.round_to(wts[et, ej][:, None] * dY[et], dt)
        cols = np.sort(np.random.default_rng(100 + e).choice(wl.f, size=4, replace=False))
        w1s = O.as_f64(I.w1[e][cols], dt)                         # [4, d]
        w3s = O.as_f64(I.w3[e][cols], dt) if I.w3 is not None else None
        w2s = O.as_f64(I.w2[e][:, cols], dt)                      # [d, 4]
        sl = O.ffn_dw_slices(Xe, dYe, w1s, w3s, w2s, wl.act, dt, np.arange(4))
        J = torch.from_numpy(cols).to(dev())
        assert_close(to_np(L.dw2[e][:, J]), sl["dW2"], rt, f"dW2[{e}] slice")
        assert_close(to_np(L.dw1[e][J]), sl["dW1"], rt, f"dW1[{e}] slice")
        if L.swiglu:
            assert_close(to_np(L.dw3[e][J]), sl["dW3"], rt, f"dW3[{e}] slice")
    for e in range(wl.E):
        if fill[e] == 0:
            assert float(L.dw1[e].abs().max()) == 0.0 and float(L.dw2[e].abs().max()) == 0.0


@pytest.mark.parametrize("name,run", [("c2", 0), ("c2", 1), ("c3", 0), ("c3", 1), ("c4", 0),
                                      ("c5", 0)])
def test_full_size(name, run):
    _check(name, run)
    torch.cuda.empty_cache()
