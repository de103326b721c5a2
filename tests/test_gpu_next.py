"""GPU parity (through the C ABI) of the operators beyond the layer's core
path, against the CPU oracle on the same seeded inputs:

* Eq. 3 balance term and its gradient through the gate backward;
* AggregateSpec and the Eq. 2 specification loss with its gradients, alone
  and inside the layer backward;
* the Cache operator (Section 4.2): unchanged-sample count and cache update,
  combine weights at cached picks, and the layer forward with the gate on a
  second stream;
* the capacity policy at the launch frontier (Section 3 and its
  implementation appendix), driven by real device counts over a drifting
  trajectory of mini-batches.

Integers (counts, cached picks, capacities, AggregateSpec rows) are compared
bit-exactly; floats with the tolerance rule of gpu_util."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import NEAR_TIE, RTOL, assert_close, dev, min_topk_gap, scaled_small, to_dev, to_np, torch_dtype
from paper_2205_01848_amd import MoELayer, rows_alloc_for
from paper_2205_01848_amd.layer import ROW_ALIGN
from paper_2205_01848_amd import binding as B

pytestmark = pytest.mark.gpu


def _enc(a, dt):
    return W.to_bf16_bits(a) if dt == "bf16" else np.asarray(a, dtype=np.float32)


def _dec(a, dt):
    return O.bf16_to_f64(a) if dt == "bf16" else np.asarray(a, dtype=np.float64)


def _routing(rng, T, E, k, cap_div=None):
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    counts = O.count_assignments(ids, E)
    cap = counts if cap_div is None else counts // cap_div
    off = O.exclusive_offsets(cap)
    R = int(off[-1])
    s = O.assign_slots(ids, E, cap, off, R)
    return ids, s["dest_row"], R, s


# ---- Eq. 3 balance term ---------------------------------------------------------
@pytest.mark.parametrize("T,E,k", [(1000, 8, 2), (70001, 64, 1), (300, 33, 3), (1, 1, 1)])
def test_balance_fwd_matches_oracle(T, E, k):
    rng = np.random.default_rng(T + E)
    logits = (rng.standard_normal((T, E)) * 2).astype(np.float32)
    ids = O.topk(logits.astype(np.float64), k)
    counts = O.count_assignments(ids, E).astype(np.int32)
    lam = float(np.float32(0.01))
    loss = torch.empty(1, dtype=torch.float32, device=dev())
    coef = torch.empty(E, dtype=torch.float32, device=dev())
    ws = B.workspace(B.moe_balance_workspace_bytes(T, E), dev())
    B.moe_balance_fwd(torch.from_numpy(logits).to(dev()), torch.from_numpy(counts).to(dev()), k,
                      lam, loss, coef, ws)
    torch.cuda.synchronize()
    Bref, cref = O.balance_term(logits.astype(np.float64), counts, k, lam)
    assert_close(to_np(loss), np.array([Bref]), 1e-5, "balance loss")
    assert_close(to_np(coef), cref, 1e-6, "dprob coefficient")


def test_balance_fwd_empty_batch():
    E = 8
    loss = torch.full((1,), 7.0, device=dev())
    coef = torch.full((E,), 7.0, device=dev())
    ws = B.workspace(B.moe_balance_workspace_bytes(0, E), dev())
    B.moe_balance_fwd(torch.empty(0, E, device=dev()), torch.zeros(E, dtype=torch.int32,
                                                                    device=dev()),
                      2, 0.01, loss, coef, ws)
    torch.cuda.synchronize()
    assert float(loss.item()) == 0.0 and (to_np(coef) == 0).all()


@pytest.mark.parametrize("dt,renorm", [("bf16", 1), ("f32", 0)])
def test_gate_bwd_with_balance_coefficient(dt, renorm):
    rng = np.random.default_rng(31)
    T, d, E, k = 700, 72, 8, 2 if renorm else 1
    x = _enc(rng.standard_normal((T, d)), dt)
    logits = (rng.standard_normal((T, E))).astype(np.float32)
    ids = O.topk(logits.astype(np.float64), k).astype(np.int32)
    dwt = (rng.standard_normal((T, k)) * 0.1).astype(np.float32)
    coef = (rng.standard_normal(E) * 1e-3).astype(np.float32)
    dl = torch.empty(T, E, dtype=torch.float32, device=dev())
    dwg = torch.empty(E, d, dtype=torch.float32, device=dev())
    ws = B.workspace(B.moe_gate_bwd_workspace_bytes(T, d, E), dev())
    B.moe_gate_bwd(to_dev(x, dt), torch.from_numpy(logits).to(dev()),
                   torch.from_numpy(ids).to(dev()), torch.from_numpy(dwt).to(dev()), renorm, dl,
                   dwg, ws, dprob_coef=torch.from_numpy(coef).to(dev()))
    torch.cuda.synchronize()
    rdl, rdwg = O.gate_bwd(logits.astype(np.float64), ids, dwt.astype(np.float64), renorm,
                           _dec(x, dt), dprob_coef=coef.astype(np.float64))
    assert_close(to_np(dl), rdl, 1e-5, "dlogits")
    assert_close(to_np(dwg), rdwg, 1e-5, "dw_g")


# ---- AggregateSpec and Eq. 2 specification loss -----------------------------------
@pytest.mark.parametrize("dt,k,d", [("bf16", 2, 136), ("f32", 1, 64), ("bf16", 3, 1096)])
def test_aggregate_spec_exact(dt, k, d):
    rng = np.random.default_rng(40 + k)
    T, E = 1300, 6
    ids, dest, R, _ = _routing(rng, T, E, k, cap_div=2)
    assert (dest < 0).any()
    yd = _enc(rng.standard_normal((R, d)), dt)
    out = torch.full((T * k, d), float("nan"), dtype=torch_dtype(dt), device=dev())
    B.moe_aggregate_spec(to_dev(yd, dt), torch.from_numpy(dest.astype(np.int32)).to(dev()), out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(out), O.aggregate_spec(_dec(yd, dt), dest))


@pytest.mark.parametrize("dt,k,d", [("bf16", 2, 512), ("f32", 1, 64), ("bf16", 3, 1096),
                                    ("f32", 2, 584)])
def test_spec_loss_matches_oracle(dt, k, d):
    rng = np.random.default_rng(60 + k + d)
    T, E = 1500, 6
    ids, dest, R, s = _routing(rng, T, E, k, cap_div=2)
    yd = _enc(rng.standard_normal((R, d)), dt)
    tgt = _enc(rng.standard_normal((T, d)), dt)
    wts = rng.random((T, k)).astype(np.float32)
    dyd = torch.full((max(R, 1), d), float("nan"), dtype=torch_dtype(dt), device=dev())
    dwt = torch.empty(T, k, dtype=torch.float32, device=dev())
    loss = torch.empty(1, dtype=torch.float32, device=dev())
    ws = B.workspace(B.moe_spec_loss_workspace_bytes(T), dev())
    B.moe_spec_loss(to_dev(yd, dt), torch.from_numpy(dest.astype(np.int32)).to(dev()),
                    torch.from_numpy(wts).to(dev()), to_dev(tgt, dt), dyd, dwt, loss, ws)
    torch.cuda.synchronize()
    rl, rdw, rdy = O.spec_loss(_dec(yd, dt), dest, wts.astype(np.float64), _dec(tgt, dt), dt)
    assert_close(to_np(loss), np.array([rl]), 1e-5, "spec loss")
    assert_close(to_np(dwt), rdw, 1e-5, "dweights")
    kept = s["src"] >= 0
    assert_close(to_np(dyd)[kept], rdy[kept], RTOL[dt], "dy_disp")


def test_spec_loss_empty_batch():
    loss = torch.full((1,), 7.0, device=dev())
    ws = B.workspace(B.moe_spec_loss_workspace_bytes(0), dev())
    z = torch.empty(0, 64, dtype=torch.bfloat16, device=dev())
    B.moe_spec_loss(torch.empty(1, 64, dtype=torch.bfloat16, device=dev()),
                    torch.empty(0, 2, dtype=torch.int32, device=dev()),
                    torch.empty(0, 2, device=dev()), z,
                    torch.empty(1, 64, dtype=torch.bfloat16, device=dev()),
                    torch.empty(0, 2, device=dev()), loss, ws)
    torch.cuda.synchronize()
    assert float(loss.item()) == 0.0


@pytest.mark.parametrize("name,lam", [("c2", 0.01), ("c5", 0.05)])
def test_layer_backward_with_spec_loss_and_balance(name, lam):
    """Whole layer: gate -> dispatch -> FFN -> combine with the balance term,
    then the backward driven by the specification loss instead of dy (c2's
    static capacity drops assignments; c5 keeps all)."""
    wl = scaled_small(W, name, T=1024, d=128, f=256, backward=True)
    I = W.make_inputs(wl)
    tgt = W.make_target(wl)
    dt = wl.dtype
    kind, num, den = wl.capacity[0]
    R = rows_alloc_for(kind, wl.T, wl.k, wl.E, num, den)
    L = MoELayer(wl.T, wl.d, wl.E, wl.k, wl.f, wl.act, torch_dtype(dt), R, backward=True)
    x, w1, w2, wg = (to_dev(a, dt) for a in (I.x, I.w1, I.w2, I.w_g))
    w3 = to_dev(I.w3, dt) if I.w3 is not None else None
    bias = torch.from_numpy(I.bias).to(dev()) if I.bias is not None else None
    L.forward(x, w1, w3, w2, w_g=wg, bias=bias, renorm=wl.renorm, capacity=(kind, num, den),
              balance=lam)
    spec_rows = L.aggregate_spec()
    L.backward(x, None, w1, w3, w2, w_g=wg, renorm=wl.renorm, target=to_dev(tgt, dt))
    torch.cuda.synchronize()

    X = _dec(I.x, dt)
    r = O.route(X, _dec(I.w_g, dt), I.bias, wl.k, wl.renorm)
    assert min_topk_gap(r["logits"], wl.k) > NEAR_TIE * np.abs(r["logits"]).max()
    counts = O.count_assignments(r["ids"], wl.E)
    cap = (O.capacity_static(wl.T, wl.k, wl.E, num, den) if kind == "static"
           else O.capacity_dynamic(counts, wl.T, num, den))
    W1, W2 = _dec(I.w1, dt), _dec(I.w2, dt)
    W3 = _dec(I.w3, dt) if I.w3 is not None else None
    fw = O.layer_forward(X, W1, W3, W2, wl.act, dt, r["ids"], r["weights"], cap, R, wl.E,
                         ROW_ALIGN)
    Bref, coef = O.balance_term(r["logits"], counts, wl.k, lam)
    assert_close(to_np(L.balance_loss), np.array([Bref]), 1e-5, "balance loss")
    assert_close(to_np(L.dprob_coef), coef, 1e-6, "dprob coefficient")
    rt = RTOL[dt]
    agg = O.aggregate_spec(np.nan_to_num(fw["Y"]), fw["dest_row"])
    assert_close(to_np(spec_rows), agg, rt, "AggregateSpec rows")
    bw = O.layer_backward(fw, X, None, W1, W3, W2, wl.act, dt, r["ids"], r["weights"], wl.E,
                          logits=r["logits"], renorm=wl.renorm, w_g=_dec(I.w_g, dt),
                          target=_dec(tgt, dt), dprob_coef=coef)
    assert_close(to_np(L.spec_loss_value), np.array([bw["spec_loss"]]), rt, "spec loss")
    assert_close(to_np(L.dweights), bw["dweights"], rt, "dweights")
    assert_close(to_np(L.dw1), bw["dW1"], rt, "dW1")
    assert_close(to_np(L.dw2), bw["dW2"], rt, "dW2")
    assert_close(to_np(L.dlogits), bw["dlogits"], rt, "dlogits")
    assert_close(to_np(L.dw_g), bw["dw_g"], rt, "dw_g")
    assert_close(to_np(L.dx), bw["dx"], rt, "dx")


# ---- Section 4.2: sample assignment caching ------------------------------------------
@pytest.mark.parametrize("T,E,k,frac", [(3000, 16, 2, 0.1), (70001, 64, 1, 0.03),
                                        (999, 8, 4, 0.5)])
def test_cache_update_counts_and_stores(T, E, k, frac):
    wl = W.small("c4", T=T, d=64, f=64, E=E, k=k)
    cached = W.make_inputs(wl).ids
    fresh = W.reassign_some(T + E, cached, E, frac)
    fresh[::7] = fresh[::7, ::-1]              # reordered rows are still unchanged
    want = int(O.cache_unchanged(fresh, cached).sum())
    assert 0 < want < T
    unchanged = torch.zeros(1, dtype=torch.int32, device=dev())
    c_in = torch.from_numpy(cached).to(dev())
    out = torch.full((T, k), -9, dtype=torch.int32, device=dev())
    f_dev = torch.from_numpy(fresh).to(dev())
    B.moe_cache_update(f_dev, c_in, out, unchanged)                  # separate buffers
    B.moe_cache_update(f_dev, out, out, unchanged)                   # in place: all unchanged
    torch.cuda.synchronize()
    assert int(unchanged.item()) == want + T
    np.testing.assert_array_equal(to_np(out), fresh)
    np.testing.assert_array_equal(to_np(c_in), cached)


def test_cached_weights_equal_gate_weights_and_oracle():
    wl = scaled_small(W, "c5", T=1500, d=128, f=64)
    I = W.make_inputs(wl)
    x, wg = to_dev(I.x, "bf16"), to_dev(I.w_g, "bf16")
    T, E, k = wl.T, wl.E, wl.k
    logits = torch.empty(T, E, device=dev())
    ids = torch.empty(T, k, dtype=torch.int32, device=dev())
    w = torch.empty(T, k, device=dev())
    B.moe_gate_topk(x, wg, torch.from_numpy(I.bias).to(dev()), k, 1, logits, ids, w)
    same = torch.empty(T, k, device=dev())
    B.moe_cached_weights(logits, ids, 1, same)
    rng = np.random.default_rng(5)
    other = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    other[3, 1] = E + 5                        # an invalid cached id gets weight 0
    ow = torch.empty(T, k, device=dev())
    B.moe_cached_weights(logits, torch.from_numpy(other).to(dev()), 1, ow)
    raw = torch.empty(T, k, device=dev())
    B.moe_cached_weights(logits, torch.from_numpy(other).to(dev()), 0, raw)
    torch.cuda.synchronize()
    assert torch.equal(same, w)
    L = to_np(logits)
    p = O.softmax(L)
    valid = np.where(other < E, other, 0)
    sel = np.where(other < E, np.take_along_axis(p, valid, axis=1), 0.0)
    ref_raw = sel
    ref_norm = sel / sel.sum(axis=1, keepdims=True)
    ok = np.ones(T, dtype=bool)
    ok[3] = False
    assert_close(to_np(ow)[ok], O.gate_weights(p, valid, 1)[ok], 1e-6, "renormalised")
    assert_close(to_np(ow)[3], ref_norm[3], 1e-6, "row with an invalid id")
    assert_close(to_np(raw)[ok], O.gate_weights(p, valid, 0)[ok], 1e-6, "raw")
    assert to_np(raw)[3, 1] == 0.0 and abs(to_np(raw)[3, 0] - ref_raw[3, 0]) < 1e-6


@pytest.mark.parametrize("concurrent", [True, False])
def test_forward_cached_with_concurrent_gate(concurrent):
    """Caching on: dispatch and FFN from the previous epoch's picks while the
    gate runs on a second stream; the combine uses the gate's fresh
    probabilities at the cached picks; the Cache operator counts the
    unchanged samples and stores the fresh picks."""
    wl = scaled_small(W, "c5", T=1024, d=128, f=256)
    I = W.make_inputs(wl)
    dt, T, E, k = "bf16", wl.T, wl.E, wl.k
    X = _dec(I.x, dt)
    r = O.route(X, _dec(I.w_g, dt), I.bias, k, wl.renorm)
    assert min_topk_gap(r["logits"], k) > NEAR_TIE * np.abs(r["logits"]).max()
    cached = W.reassign_some(11, r["ids"], E, 0.08)           # last epoch's picks
    R = rows_alloc_for("dynamic", T, k, E, 21, 20)
    L = MoELayer(T, wl.d, E, k, wl.f, wl.act, torch.bfloat16, R, backward=True)
    x, w1, w3, w2, wg = (to_dev(a, dt) for a in (I.x, I.w1, I.w3, I.w2, I.w_g))
    bias = torch.from_numpy(I.bias).to(dev())
    c_dev = torch.from_numpy(cached).to(dev())
    c_out = torch.empty_like(c_dev)
    unchanged = torch.zeros(1, dtype=torch.int32, device=dev())
    gs = torch.cuda.Stream() if concurrent else None
    L.forward_cached(x, w1, w3, w2, cached=c_dev, cache_out=c_out, unchanged=unchanged, w_g=wg,
                     bias=bias, renorm=wl.renorm, capacity=("dynamic", 21, 20), gate_stream=gs)
    dy = to_dev(I.dy, dt)
    L.backward(x, dy, w1, w3, w2, w_g=wg, renorm=wl.renorm, ids=c_dev, weights=L.cached_weights)
    torch.cuda.synchronize()

    assert int(unchanged.item()) == int(O.cache_unchanged(r["ids"], cached).sum())
    np.testing.assert_array_equal(to_np(c_out), r["ids"])
    wts = O.gate_weights(O.softmax(r["logits"]), cached, wl.renorm)
    assert_close(to_np(L.cached_weights), wts, 1e-5, "weights at cached picks")
    counts = O.count_assignments(cached, E)
    cap = O.capacity_dynamic(counts, T, 21, 20)
    W1, W2, W3 = _dec(I.w1, dt), _dec(I.w2, dt), _dec(I.w3, dt)
    fw = O.layer_forward(X, W1, W3, W2, wl.act, dt, cached, wts, cap, R, E, ROW_ALIGN)
    np.testing.assert_array_equal(to_np(L.dest_row), fw["dest_row"])
    rt = RTOL[dt]
    assert_close(to_np(L.y), fw["y"], rt, "y")
    bw = O.layer_backward(fw, X, _dec(I.dy, dt), W1, W3, W2, wl.act, dt, cached, wts, E,
                          logits=r["logits"], renorm=wl.renorm, w_g=_dec(I.w_g, dt))
    assert_close(to_np(L.dlogits), bw["dlogits"], rt, "dlogits")
    assert_close(to_np(L.dw_g), bw["dw_g"], rt, "dw_g")
    assert_close(to_np(L.dx), bw["dx"], rt, "dx")


def test_forward_cached_rejects_cache_stored_in_place():
    """The cached picks drive the dispatch and the backward of the same
    step, so the fresh picks may not be stored over them, on one stream or
    two."""
    wl = scaled_small(W, "c5", T=256, d=64, f=64)
    I = W.make_inputs(wl)
    dt, T, E, k = "bf16", wl.T, wl.E, wl.k
    R = rows_alloc_for("dynamic", T, k, E, 21, 20)
    L = MoELayer(T, wl.d, E, k, wl.f, wl.act, torch.bfloat16, R, backward=True)
    x, w1, w3, w2, wg = (to_dev(a, dt) for a in (I.x, I.w1, I.w3, I.w2, I.w_g))
    c_dev = torch.from_numpy(np.tile(np.arange(k, dtype=np.int32), (T, 1))).to(dev())
    unchanged = torch.zeros(1, dtype=torch.int32, device=dev())
    for gs in (None, torch.cuda.Stream()):
        with pytest.raises(ValueError):
            L.forward_cached(x, w1, w3, w2, cached=c_dev, cache_out=c_dev, unchanged=unchanged,
                             w_g=wg, renorm=wl.renorm, capacity=("dynamic", 21, 20),
                             gate_stream=gs)
    torch.cuda.synchronize()
    assert int(unchanged.item()) == 0


# ---- capacity policy at the launch frontier ---------------------------------------
# the grow / shrink settings of the benchmark's policy sweep, on its two shapes
# (T, E, k of the largest layer and of the 64-expert top-1 layer)
POLICY_SETTINGS = [((21, 20), (5, 4)), ((11, 10), (13, 10)), ((6, 5), (3, 2)), ((5, 4), (2, 1))]


@pytest.mark.parametrize("delta", [0, 1, 3])
@pytest.mark.parametrize("setting", range(len(POLICY_SETTINGS)))
@pytest.mark.parametrize("shape", [(4096, 8, 2), (16384, 64, 1)])
def test_capacity_policy_on_device_counts(delta, setting, shape):
    (T, E, k), d, N = shape, 64, 24
    traj = W.drifting_assignments(9, T, E, k, N)
    init = O.capacity_static(T, k, E, 1, 1)
    grow, shrink = POLICY_SETTINGS[setting]
    pol = B.CapacityPolicy(T, k, E, delta, grow, shrink, init)
    R = E * T                                   # any capacity the policy can choose fits
    x = torch.zeros(T, d, dtype=torch.bfloat16, device=dev())
    cap = torch.empty(E, dtype=torch.int32, device=dev())
    off = torch.empty(E + 1, dtype=torch.int32, device=dev())
    counts = torch.empty(E, dtype=torch.int32, device=dev())
    fill = torch.empty(E, dtype=torch.int32, device=dev())
    dest = torch.empty(T, k, dtype=torch.int32, device=dev())
    src = torch.empty(R, dtype=torch.int32, device=dev())
    xd = torch.empty(R, d, dtype=torch.bfloat16, device=dev())
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    ws = B.workspace(B.moe_dispatch_workspace_bytes(T, E, k), dev())
    ids_dev = [torch.from_numpy(a).to(dev()) for a in traj]
    fills = torch.empty(N, E, dtype=torch.int32, device=dev())
    caps_dev = torch.empty(N, E, dtype=torch.int32, device=dev())
    host_caps, recs = [], []
    for i in range(N):
        rows, rec = pol.begin(cap, off)
        host_caps.append(pol.state()["cap"])
        recs.append(rec)
        assert rows == sum(host_caps[-1]) <= R
        B.moe_dispatch(x, ids_dev[i], E, cap, off, R, counts, fill, dest, src, xd, status, ws)
        pol.end(counts)
        fills[i].copy_(fill)
        caps_dev[i].copy_(cap)
    torch.cuda.synchronize()
    st = pol.state()
    pol.close()
    seq = [O.count_assignments(a, E) for a in traj]
    sim = O.simulate_capacity_policy(seq, T, k, delta, init, grow, shrink)
    np.testing.assert_array_equal(np.array(host_caps), sim["caps"])
    np.testing.assert_array_equal(to_np(caps_dev), sim["caps"])
    np.testing.assert_array_equal(np.array(recs), sim["recompile"])
    drops = (np.array(seq) - to_np(fills)).sum(axis=1)
    np.testing.assert_array_equal(drops, sim["drops"])
    # begin() of iteration i consumes the metrics up to iteration i - 1 - delta
    assert st["launched"] == N and st["consumed"] == N - 1 - delta
    assert st["recompiles"] == int(sim["recompile"].sum())
    assert int(status.item()) == 0


# ---- error paths -------------------------------------------------------------------
def test_policy_call_order_and_state():
    """begin twice, or end without begin, is rejected without enqueuing; the
    object stays usable, and destroying it with copies in flight is safe."""
    T, E, k = 1000, 4, 2
    pol = B.CapacityPolicy(T, k, E, 2, (11, 10), (3, 2), [500] * E)
    cap = torch.empty(E, dtype=torch.int32, device=dev())
    off = torch.empty(E + 1, dtype=torch.int32, device=dev())
    counts = torch.tensor([400, 600, 500, 500], dtype=torch.int32, device=dev())
    with pytest.raises(B.MoEError):
        pol.end(counts)                        # end without begin
    rows, rec = pol.begin(cap, off)
    assert rows == 2000 and not rec
    with pytest.raises(B.MoEError):
        pol.begin(cap, off)                    # begin twice
    pol.end(counts)
    recs = []
    for _ in range(3):                         # iteration 0's metric is seen by iteration 3
        recs.append(pol.begin(cap, off)[1])
        pol.end(counts)
    torch.cuda.synchronize()
    assert recs == [False, False, True]
    st = pol.state()
    assert st["launched"] == 4 and st["consumed"] == 1 and st["recompiles"] == 1
    assert st["cap"] == [440, 660, 550, 550]   # ceil(1.1 * counts): 600 overflowed 500
    np.testing.assert_array_equal(to_np(cap), [440, 660, 550, 550])
    np.testing.assert_array_equal(to_np(off), [0, 440, 1100, 1650, 2200])
    rows, rec = pol.begin(cap, off)            # iteration 1's metric fits: no change
    assert rows == 2200 and not rec
    pol.end(counts)
    pol.close()                                # copies still outstanding: waited for


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_loss_kernels_treat_rows_beyond_rows_alloc_as_dropped(dt):
    rng = np.random.default_rng(77)
    T, E, k, d = 300, 4, 2, 64
    ids, dest, R, _ = _routing(rng, T, E, k)
    bad = dest.copy()
    bad[::5, 1] = R + 3                        # not a row of y_disp
    yd = _enc(rng.standard_normal((R, d)), dt)
    tgt = _enc(rng.standard_normal((T, d)), dt)
    wts = rng.random((T, k)).astype(np.float32)
    t_bad = torch.from_numpy(bad.astype(np.int32)).to(dev())
    agg = torch.full((T * k, d), float("nan"), dtype=torch_dtype(dt), device=dev())
    B.moe_aggregate_spec(to_dev(yd, dt), t_bad, agg)
    dyd = torch.full((R, d), float("nan"), dtype=torch_dtype(dt), device=dev())
    dwt = torch.empty(T, k, dtype=torch.float32, device=dev())
    loss = torch.empty(1, dtype=torch.float32, device=dev())
    ws = B.workspace(B.moe_spec_loss_workspace_bytes(T), dev())
    B.moe_spec_loss(to_dev(yd, dt), t_bad, torch.from_numpy(wts).to(dev()), to_dev(tgt, dt), dyd,
                    dwt, loss, ws)
    torch.cuda.synchronize()
    as_dropped = np.where(bad >= R, -1, bad)
    np.testing.assert_array_equal(to_np(agg), O.aggregate_spec(_dec(yd, dt), as_dropped))
    rl, rdw, _ = O.spec_loss(_dec(yd, dt), as_dropped, wts.astype(np.float64), _dec(tgt, dt), dt)
    assert_close(to_np(loss), np.array([rl]), 1e-5, "loss")
    assert_close(to_np(dwt), rdw, 1e-5, "dweights")
