"""Pins of the oracle's expert FFN, combine and backward.

Forward: with capacity >= load the layer equals Eq. 1's dense weighted sum of
expert outputs (every expert evaluated on every token with torch, then
picked); E = 1 is a plain two-layer MLP; k = E with renormalisation is the
fully soft mixture; dropped assignments contribute nothing.
Backward: torch autograd in float64 on the same dense formulation with the
routing held fixed, and central finite differences of the oracle's own
forward.  The fp32 layer path (no bf16 rounding) is the one pinned exactly;
the bf16 path is pinned to it within bf16 rounding error."""
import numpy as np
import pytest
import torch

import oracle as O

F = torch.nn.functional


def _act_t(h, act):
    if act == "relu":
        return torch.relu(h)
    if act == "gelu_tanh":
        return F.gelu(h, approximate="tanh")
    raise ValueError(act)


def _dense_expert_outputs(x, w1, w3, w2, act):
    """[E, T, d]: expert e applied to every token (torch, float64)."""
    outs = []
    for e in range(w1.shape[0]):
        if act == "swiglu":
            a = F.silu(F.linear(x, w1[e])) * F.linear(x, w3[e])
        else:
            a = _act_t(F.linear(x, w1[e]), act)
        outs.append(F.linear(a, w2[e]))
    return torch.stack(outs)


def _params(seed, T, d, E, f, act, bias=True):
    rng = np.random.default_rng(seed)
    P = dict(
        x=rng.standard_normal((T, d)),
        w_g=rng.standard_normal((E, d)) * 0.3,
        b=(rng.standard_normal(E) * 0.2).astype(np.float32) if bias else None,
        w1=rng.standard_normal((E, f, d)) * 0.2,
        w3=rng.standard_normal((E, f, d)) * 0.2 if act == "swiglu" else None,
        w2=rng.standard_normal((E, d, f)) * 0.2,
        dy=rng.standard_normal((T, d)),
    )
    return P


def _forward(P, k, renorm, act, cap, dtype="f32"):
    E = P["w_g"].shape[0]
    r = O.route(P["x"], P["w_g"], P["b"], k, renorm)
    rows_alloc = int(np.sum(cap))
    fw = O.layer_forward(P["x"], P["w1"], P["w3"], P["w2"], act, dtype, r["ids"],
                         r["weights"], cap, rows_alloc, E)
    return r, fw


ACTS = ["relu", "gelu_tanh", "swiglu"]


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("k,renorm", [(1, 0), (2, 1), (3, 1)])
def test_infinite_capacity_is_dense_weighted_sum(act, k, renorm):
    T, d, E, f = 37, 12, 5, 20
    P = _params(11 + k, T, d, E, f, act)
    r, fw = _forward(P, k, renorm, act, np.full(E, T))
    tt = {n: (torch.tensor(v) if v is not None else None) for n, v in P.items()}
    dense = _dense_expert_outputs(tt["x"], tt["w1"], tt["w3"], tt["w2"], act)
    ref = torch.zeros(T, d, dtype=torch.float64)
    for j in range(k):
        ref += torch.tensor(r["weights"][:, j], dtype=torch.float64)[:, None] * \
            dense[torch.tensor(r["ids"][:, j].astype(np.int64)), torch.arange(T)]
    np.testing.assert_allclose(fw["y"], ref.numpy(), rtol=1e-12, atol=1e-13)
    assert (fw["dest_row"] >= 0).all()


def test_single_expert_is_plain_mlp():
    T, d, f = 23, 16, 24
    P = _params(21, T, d, 1, f, "gelu_tanh")
    r, fw = _forward(P, 1, 0, "gelu_tanh", np.array([T]))
    assert (r["weights"] == 1.0).all()
    x = torch.tensor(P["x"])
    ref = F.linear(F.gelu(F.linear(x, torch.tensor(P["w1"][0])), approximate="tanh"),
                   torch.tensor(P["w2"][0]))
    np.testing.assert_allclose(fw["y"], ref.numpy(), rtol=1e-12, atol=1e-13)


def test_k_equals_E_renormalised_is_soft_mixture():
    T, d, E, f = 19, 8, 4, 10
    P = _params(22, T, d, E, f, "relu")
    r, fw = _forward(P, E, 1, "relu", np.full(E, T))
    tt = {n: (torch.tensor(v) if v is not None else None) for n, v in P.items()}
    dense = _dense_expert_outputs(tt["x"], tt["w1"], None, tt["w2"], "relu")
    p = torch.softmax(torch.tensor(r["logits"], dtype=torch.float64), dim=1)
    ref = (p.T[:, :, None] * dense).sum(0)
    np.testing.assert_allclose(fw["y"], ref.numpy(), rtol=2e-7, atol=1e-7 * np.abs(ref.numpy()).max())


def test_drops_contribute_nothing_and_combine_is_linear():
    T, d, E, f = 60, 8, 3, 12
    P = _params(23, T, d, E, f, "relu")
    cap = np.array([5, 30, 0])
    r, fw = _forward(P, 2, 1, "relu", cap)
    dest = fw["dest_row"]
    assert (dest == -1).any() and (dest >= 0).any()
    tt = {n: (torch.tensor(v) if v is not None else None) for n, v in P.items()}
    dense = _dense_expert_outputs(tt["x"], tt["w1"], None, tt["w2"], "relu").numpy()
    ref = np.zeros((T, d))
    for t in range(T):
        for j in range(2):
            if dest[t, j] >= 0:
                ref[t] += r["weights"][t, j] * dense[r["ids"][t, j], t]
    np.testing.assert_allclose(fw["y"], ref, rtol=1e-12, atol=1e-13)
    nothing = (dest < 0).all(axis=1)
    assert nothing.any() and (fw["y"][nothing] == 0).all()
    w_a = np.abs(np.random.default_rng(1).standard_normal((T, 2)))
    w_b = np.abs(np.random.default_rng(2).standard_normal((T, 2)))
    ya = O.combine(fw["Y"], dest, w_a, "f32")
    yb = O.combine(fw["Y"], dest, w_b, "f32")
    np.testing.assert_allclose(O.combine(fw["Y"], dest, w_a + w_b, "f32"), ya + yb,
                               rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("act", ACTS)
def test_bf16_path_within_rounding_of_exact_path(act):
    T, d, E, f = 64, 32, 4, 48
    P = _params(24, T, d, E, f, act)
    for n in ("x", "w1", "w3", "w2", "w_g"):
        if P[n] is not None:
            P[n] = O.round_bf16(P[n])
    cap = np.full(E, T)
    r, fw32 = _forward(P, 2, 1, act, cap, "f32")
    _, fw16 = _forward(P, 2, 1, act, cap, "bf16")
    for n in ("H", "A", "Y", "y"):
        v = fw16[n][~np.isnan(fw16[n])]
        np.testing.assert_array_equal(O.round_bf16(v), v)          # stored as bf16
    scale = np.sqrt(np.mean(fw32["y"] ** 2))
    err = np.abs(fw16["y"] - fw32["y"])
    assert err.max() < 0.05 * scale and err.max() > 0                # rounding happened
    assert np.mean(err) < 0.01 * scale


# -- backward ------------------------------------------------------------------
def _autograd_reference(P, r, fw, k, renorm, act):
    """Loss = sum(y * dy) through the dense formulation, routing fixed."""
    keep = torch.tensor(fw["dest_row"] >= 0)
    ids = torch.tensor(r["ids"].astype(np.int64))
    leaves = {}
    for n in ("x", "w_g", "w1", "w3", "w2"):
        if P[n] is not None:
            leaves[n] = torch.tensor(P[n], requires_grad=True)
    x = leaves["x"]
    logits = F.linear(x, leaves["w_g"])
    if P["b"] is not None:
        logits = logits + torch.tensor(P["b"], dtype=torch.float64)
    logits.retain_grad()
    p = torch.softmax(logits, dim=1)
    sel = torch.gather(p, 1, ids)
    w = sel / sel.sum(1, keepdim=True) if renorm else sel
    w.retain_grad()
    dense = _dense_expert_outputs(x, leaves["w1"], leaves.get("w3"), leaves["w2"], act)
    T = x.shape[0]
    y = torch.zeros_like(x)
    for j in range(k):
        y = y + (keep[:, j].double() * w[:, j])[:, None] * dense[ids[:, j], torch.arange(T)]
    (y * torch.tensor(P["dy"])).sum().backward()
    g = {n: t.grad.numpy() for n, t in leaves.items()}
    g["logits"] = logits.grad.numpy()
    g["w"] = w.grad.numpy() * keep.numpy()
    return g


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("k,renorm,cap_kind", [(1, 0, "inf"), (2, 1, "inf"), (2, 1, "tight"),
                                               (3, 1, "tight")])
def test_backward_matches_torch_autograd(act, k, renorm, cap_kind):
    T, d, E, f = 41, 10, 5, 14
    P = _params(31 + k, T, d, E, f, act)
    cap = np.full(E, T) if cap_kind == "inf" else np.array([3, 9, 0, 20, 7])
    r, fw = _forward(P, k, renorm, act, cap)
    b = O.layer_backward(fw, P["x"], P["dy"], P["w1"], P["w3"], P["w2"], act, "f32",
                         r["ids"], r["weights"], E, logits=r["logits"], renorm=renorm,
                         w_g=P["w_g"])
    g = _autograd_reference(P, r, fw, k, renorm, act)
    tol = dict(rtol=2e-6, atol=2e-6)
    np.testing.assert_allclose(b["dweights"], g["w"], **tol)
    np.testing.assert_allclose(b["dlogits"], g["logits"], **tol)
    np.testing.assert_allclose(b["dw_g"], g["w_g"], **tol)
    np.testing.assert_allclose(b["dW1"], g["w1"], **tol)
    np.testing.assert_allclose(b["dW2"], g["w2"], **tol)
    if act == "swiglu":
        np.testing.assert_allclose(b["dW3"], g["w3"], **tol)
    np.testing.assert_allclose(b["dx"], g["x"], **tol)
    np.testing.assert_allclose(b["dlogits"].sum(axis=1), 0.0, atol=1e-7)
    assert (b["dweights"][fw["dest_row"] < 0] == 0).all()


def test_backward_finite_differences():
    """Central differences of the oracle's own forward (fp32 path, float64
    arithmetic) on a few coordinates of every parameter."""
    T, d, E, f, k = 9, 6, 3, 7, 2
    act = "swiglu"
    P = _params(41, T, d, E, f, act)
    cap = np.array([4, 9, 2])

    def loss(Q):
        r, fw = _forward(Q, k, 1, act, cap)
        return float((fw["y"] * Q["dy"]).sum()), r

    base, r0 = loss(P)
    _, fw = _forward(P, k, 1, act, cap)
    b = O.layer_backward(fw, P["x"], P["dy"], P["w1"], P["w3"], P["w2"], act, "f32",
                         r0["ids"], r0["weights"], E, logits=r0["logits"], renorm=1,
                         w_g=P["w_g"])
    grads = dict(x=b["dx"], w_g=b["dw_g"], w1=b["dW1"], w3=b["dW3"], w2=b["dW2"])
    rng = np.random.default_rng(5)
    h = 1e-3          # fp32 logits/weights add ~6e-8/(2h) noise; truncation is O(h^2)
    for name, g in grads.items():
        for _ in range(4):
            idx = tuple(int(rng.integers(0, s)) for s in P[name].shape)
            Qp = {n: (v.copy() if isinstance(v, np.ndarray) else v) for n, v in P.items()}
            Qm = {n: (v.copy() if isinstance(v, np.ndarray) else v) for n, v in P.items()}
            Qp[name][idx] += h
            Qm[name][idx] -= h
            lp, rp = loss(Qp)
            lm, rm = loss(Qm)
            assert (rp["ids"] == r0["ids"]).all() and (rm["ids"] == r0["ids"]).all()
            fd = (lp - lm) / (2 * h)
            assert abs(fd - g[idx]) <= 1e-3 * (abs(fd) + 1e-2), (name, idx, fd, g[idx])


def test_dropped_tokens_do_not_reach_weight_gradients():
    T, d, E, f = 50, 8, 3, 12
    P = _params(51, T, d, E, f, "relu")
    cap = np.array([6, 6, 6])
    r, fw = _forward(P, 2, 1, "relu", cap)
    b1 = O.layer_backward(fw, P["x"], P["dy"], P["w1"], None, P["w2"], "relu", "f32",
                          r["ids"], r["weights"], E)
    dropped_only = (fw["dest_row"] < 0).all(axis=1)
    assert dropped_only.any()
    dy2 = P["dy"].copy()
    dy2[dropped_only] *= 1000.0                              # gradient of dropped tokens
    b2 = O.layer_backward(fw, P["x"], dy2, P["w1"], None, P["w2"], "relu", "f32",
                          r["ids"], r["weights"], E)
    np.testing.assert_array_equal(b1["dW1"], b2["dW1"])
    np.testing.assert_array_equal(b1["dW2"], b2["dW2"])
    assert (b2["dx"][dropped_only] == 0).all()


@pytest.mark.parametrize("act", ACTS)
def test_dw_slices_match_full_backward(act):
    """The column-slice form of the weight gradients equals the full
    backward's gradients on the same columns (bf16 rounding points)."""
    rng = np.random.default_rng(70)
    R, d, f = 57, 24, 40
    X = O.round_bf16(rng.standard_normal((R, d)))
    dY = O.round_bf16(rng.standard_normal((R, d)))
    w1 = O.round_bf16(rng.standard_normal((1, f, d)) * 0.2)
    w3 = O.round_bf16(rng.standard_normal((1, f, d)) * 0.2) if act == "swiglu" else None
    w2 = O.round_bf16(rng.standard_normal((1, d, f)) * 0.2)
    e_of = np.zeros(R, dtype=np.int64)
    fw = O.ffn_rows_fwd(X, e_of, w1, w3, w2, act, "bf16")
    bw = O.ffn_rows_bwd(X, e_of, fw["H"], fw["H3"], dY, w1, w3, w2, act, "bf16", 1)
    cols = np.array([0, 7, 39, 12])
    sl = O.ffn_dw_slices(X, dY, w1[0], None if w3 is None else w3[0], w2[0], act, "bf16", cols)
    np.testing.assert_array_equal(sl["dW2"], bw["dW2"][0][:, cols])
    np.testing.assert_array_equal(sl["dW1"], bw["dW1"][0][cols])
    if act == "swiglu":
        np.testing.assert_array_equal(sl["dW3"], bw["dW3"][0][cols])


def test_topk_alternatives():
    l = np.array([1.0, 3.0, 3.0 + 1e-9, 0.5])
    alts = O.topk_alternatives(l, 2, 1e-6)
    assert (2, 1) in alts and (1, 2) in alts and len(alts) == 2
    alts = O.topk_alternatives(np.array([2.0, 1.0, 1.0 + 1e-9, 1.0 - 1e-9]), 2, 1e-6)
    assert set(alts) == {(0, 2), (0, 1), (0, 3)}
    assert O.topk_alternatives(np.array([0.0, 1.0, 2.0]), 2, 1e-6) == [(2, 1)]
    # strict order equals topk() when nothing is near-tied
    l = np.random.default_rng(3).standard_normal((50, 6)).astype(np.float32)
    ids = O.topk(l, 3)
    for t in range(50):
        assert O.topk_alternatives(l[t], 3, 0.0) == [tuple(ids[t])]
