"""GPU parity of the expert FFN (forward and backward), combine and their
backward against the CPU oracle, through the C ABI.

The bf16 cases run on both GEMM kernels (moe_set_gemm_tiles: 1 = 256x256
tiles, 2 = 128x128 tiles, two workgroups per CU) and with dX reading the
weights K-major or from their transposed copy (moe_set_dx_weight_copy); f32
cases run with the small-layer forward kernel (mode 0) and without it
(mode 1).

ReLU cases use dyadic inputs (x, dy in {-2..2}/4, weights in {-2..2}/16):
every GEMM partial sum is exactly representable in fp32, so the kernels and
the oracle agree bit for bit, including the relu'(H) decisions.  GELU and
SwiGLU cases use random inputs and the stated tolerance (fp32 1e-5, bf16
2e-2)."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import RTOL, assert_close, dev, to_dev, to_np, torch_dtype
from paper_2205_01848_amd import binding as B

pytestmark = pytest.mark.gpu


def _enc(a, dt):
    """float64 values -> stored layer dtype (bf16 bits / float32)."""
    return W.to_bf16_bits(a.astype(np.float32)) if dt == "bf16" else a.astype(np.float32)


def _dec(a, dt):
    return O.bf16_to_f64(a) if dt == "bf16" else a.astype(np.float64)


def _problem(E, d, f, rows, slack, act, dt, dyadic, seed):
    rng = np.random.default_rng(seed)
    rows = np.asarray(rows, dtype=np.int64)
    cap = rows + np.asarray(slack, dtype=np.int64)
    off = O.exclusive_offsets(cap)
    R = int(off[-1]) + 5                              # a few rows past the layout
    if dyadic:
        x = rng.integers(-2, 3, (R, d)) / 4.0
        w1 = rng.integers(-2, 3, (E, f, d)) / 16.0
        w3 = rng.integers(-2, 3, (E, f, d)) / 16.0 if act == "swiglu" else None
        w2 = rng.integers(-2, 3, (E, d, f)) / 16.0
        dy = rng.integers(-2, 3, (R, d)) / 4.0
    else:
        x = rng.standard_normal((R, d))
        w1 = rng.standard_normal((E, f, d)) * 0.05
        w3 = rng.standard_normal((E, f, d)) * 0.05 if act == "swiglu" else None
        w2 = rng.standard_normal((E, d, f)) * 0.05
        dy = rng.standard_normal((R, d))
    P = dict(x=_enc(x, dt), w1=_enc(w1, dt), w3=None if w3 is None else _enc(w3, dt),
             w2=_enc(w2, dt), dy=_enc(dy, dt))
    return rows, cap, off, R, P


def _oracle(rows, off, P, act, dt, E):
    valid = np.concatenate([np.arange(off[e], off[e] + rows[e]) for e in range(E)]).astype(np.int64)
    e_of = np.concatenate([np.full(rows[e], e) for e in range(E)]).astype(np.int64)
    X = _dec(P["x"], dt)[valid]
    w1, w2 = _dec(P["w1"], dt), _dec(P["w2"], dt)
    w3 = None if P["w3"] is None else _dec(P["w3"], dt)
    fw = O.ffn_rows_fwd(X, e_of, w1, w3, w2, act, dt)
    bw = O.ffn_rows_bwd(X, e_of, fw["H"], fw["H3"], _dec(P["dy"], dt)[valid], w1, w3, w2, act,
                        dt, E)
    return valid, fw, bw


def _gpu(rows, cap, off, R, P, act, dt, E, d, f, rows_kind="fill", tiles=0, wcopy=0):
    B.moe_set_gemm_tiles(tiles)
    B.moe_set_dx_weight_copy(wcopy)
    try:
        return _gpu_run(rows, cap, off, R, P, act, dt, E, d, f, rows_kind)
    finally:
        B.moe_set_gemm_tiles(0)
        B.moe_set_dx_weight_copy(0)


def _gpu_run(rows, cap, off, R, P, act, dt, E, d, f, rows_kind):
    i32 = lambda a: torch.from_numpy(np.asarray(a, dtype=np.int32)).to(dev())
    td = torch_dtype(dt)
    a = B.ACTS[act]
    code = B.MOE_BF16 if dt == "bf16" else B.MOE_F32
    x, w1, w2, dy = (to_dev(P[n], dt) for n in ("x", "w1", "w2", "dy"))
    w3 = to_dev(P["w3"], dt) if P["w3"] is not None else None
    n_h = B.h_save_planes(a)   # H (GELU) or H1, H3 (SwiGLU), then A = act(H)
    h = torch.full((n_h * R * f,), float("nan"), dtype=td, device=dev())
    y = torch.full((R, d), float("nan"), dtype=td, device=dev())
    ws = B.workspace(B.moe_ffn_fwd_workspace_bytes(code, a, E, d, f, R), dev())
    r_dev = i32(rows if rows_kind == "fill" else cap)
    B.moe_expert_ffn_fwd(a, i32(off), r_dev, x, w1, w3, w2, h, y, ws)
    dx = torch.full((R, d), float("nan"), dtype=td, device=dev())
    dw1 = torch.full((E, f, d), float("nan"), dtype=torch.float32, device=dev())
    dw3 = torch.full((E, f, d), float("nan"), dtype=torch.float32, device=dev()) if w3 is not None else None
    dw2 = torch.full((E, d, f), float("nan"), dtype=torch.float32, device=dev())
    wsb = B.workspace(B.moe_ffn_bwd_workspace_bytes(code, a, E, d, f, R), dev())
    B.moe_expert_ffn_bwd(a, i32(off), r_dev, x, h, w1, w3, w2, dy, dx, dw1, dw3, dw2, wsb)
    torch.cuda.synchronize()
    return dict(h=to_np(h).reshape(n_h, R, f), y=to_np(y), dx=to_np(dx), dw1=to_np(dw1),
                dw3=None if dw3 is None else to_np(dw3), dw2=to_np(dw2))


def _compare(g, valid, fw, bw, act, dt, exact):
    cmp = (lambda got, ref, name: np.testing.assert_array_equal(got, ref, err_msg=name)) if exact \
        else (lambda got, ref, name: assert_close(got, ref, RTOL[dt], name))
    if act != "relu":   # ReLU keeps A alone
        cmp(g["h"][0][valid], fw["H"], "H")
    if act == "swiglu":
        cmp(g["h"][1][valid], fw["H3"], "H3")
    cmp(g["h"][-1][valid], fw["A"], "A")
    cmp(g["y"][valid], fw["Y"], "Y")
    cmp(g["dx"][valid], bw["dX"], "dX")
    cmp(g["dw1"], bw["dW1"], "dW1")
    cmp(g["dw2"], bw["dW2"], "dW2")
    if act == "swiglu":
        cmp(g["dw3"], bw["dW3"], "dW3")


CASES = [
    # E, d, f, rows per expert, slack rows per expert
    (4, 64, 128, [80, 0, 33, 300], [0, 3, 7, 0]),
    (5, 264, 520, [600, 1, 0, 257, 64], [2, 0, 0, 9, 0]),
    (3, 128, 384, [256, 255, 511], [0, 1, 1]),
]


# (dtype, tile mode, dX weight copy): bf16 on both kernels, each with dX
# reading the weights K-major (1) and from the transposed copy (2); f32 with
# its small-layer forward kernel (mode 0: one wavefront per 32x32 block) and
# on 256x256 tiles only (mode 1)
DT_TILES = [("f32", 0, 0), ("f32", 1, 0), ("bf16", 1, 1), ("bf16", 2, 1), ("bf16", 1, 2),
            ("bf16", 2, 2)]


@pytest.mark.parametrize("dt,tiles,wcopy", DT_TILES)
@pytest.mark.parametrize("case", range(len(CASES)))
def test_relu_dyadic_bit_exact(dt, tiles, wcopy, case):
    E, d, f, rows, slack = CASES[case]
    rows, cap, off, R, P = _problem(E, d, f, rows, slack, "relu", dt, True, 10 + case)
    valid, fw, bw = _oracle(rows, off, P, "relu", dt, E)
    g = _gpu(rows, cap, off, R, P, "relu", dt, E, d, f, tiles=tiles, wcopy=wcopy)
    _compare(g, valid, fw, bw, "relu", dt, exact=True)


@pytest.mark.parametrize("act", ["gelu_tanh", "swiglu"])
@pytest.mark.parametrize("dt,tiles,wcopy", DT_TILES)
@pytest.mark.parametrize("case", [0, 1])
def test_gelu_swiglu_random(act, dt, tiles, wcopy, case):
    E, d, f, rows, slack = [(4, 192, 200, [513, 17, 0, 129], [0, 0, 4, 1]),
                            (2, 64, 136, [40, 300], [1, 1])][case]
    rows, cap, off, R, P = _problem(E, d, f, rows, slack, act, dt, False, 20 + case)
    valid, fw, bw = _oracle(rows, off, P, act, dt, E)
    g = _gpu(rows, cap, off, R, P, act, dt, E, d, f, tiles=tiles, wcopy=wcopy)
    _compare(g, valid, fw, bw, act, dt, exact=False)


@pytest.mark.parametrize("dt,tiles,wcopy", DT_TILES)
def test_gelu_large_preactivations(dt, tiles, wcopy):
    """Pre-activations far into both tails (|H| up to about 60): the kernels'
    GELU goes through an exponential that overflows to inf on the negative
    side and must give -0 there, and H itself on the positive side."""
    E, d, f = 2, 64, 136
    rows, cap, off, R, P = _problem(E, d, f, [70, 130], [1, 0], "gelu_tanh", dt, False, 50)
    scale = np.linspace(0.1, 40.0, f)[None, :, None]      # column j of H scaled by scale[j]
    P["w1"] = _enc(_dec(P["w1"], dt) * scale, dt)
    valid, fw, bw = _oracle(rows, off, P, "gelu_tanh", dt, E)
    assert np.abs(fw["H"]).max() > 40 and fw["H"].min() < -40
    g = _gpu(rows, cap, off, R, P, "gelu_tanh", dt, E, d, f, tiles=tiles, wcopy=wcopy)
    _compare(g, valid, fw, bw, "gelu_tanh", dt, exact=False)
    a = g["h"][-1][valid]
    assert np.isfinite(a).all()
    assert (a[fw["H"] < -20] == 0).all()


@pytest.mark.parametrize("tiles", [1, 2])
def test_split_k_weight_gradients_skewed_experts(tiles):
    """One expert holds almost every row, so the dW products split K into
    chunks and add the partial sums in a fixed order."""
    E, d, f = 8, 256, 256
    rows = [6000, 10, 0, 3, 0, 0, 77, 1]
    rows, cap, off, R, P = _problem(E, d, f, rows, [0] * E, "relu", "bf16", True, 30)
    valid, fw, bw = _oracle(rows, off, P, "relu", "bf16", E)
    g = _gpu(rows, cap, off, R, P, "relu", "bf16", E, d, f, tiles=tiles)
    _compare(g, valid, fw, bw, "relu", "bf16", exact=True)


@pytest.mark.parametrize("tiles", [1, 2])
def test_split_k_swiglu_later_experts(tiles):
    """SwiGLU weight gradients with split K on experts other than the first,
    one of them in the upper half: [dW1; dW3] has 2f rows per expert while
    dW1 and dW3 hold f each, so the split-K reduction must step from expert
    to expert by f x d (a stride of 2f x d wrote expert g's sums into expert
    2g's place, past the buffer for g >= E/2)."""
    E, d, f = 4, 128, 136
    rows, cap, off, R, P = _problem(E, d, f, [10, 3000, 0, 2500], [0, 2, 0, 1], "swiglu", "bf16",
                                    False, 80)
    valid, fw, bw = _oracle(rows, off, P, "swiglu", "bf16", E)
    g = _gpu(rows, cap, off, R, P, "swiglu", "bf16", E, d, f, tiles=tiles)
    _compare(g, valid, fw, bw, "swiglu", "bf16", exact=False)


@pytest.mark.parametrize("tiles", [1, 2])
@pytest.mark.parametrize("act", ["relu", "swiglu"])
def test_weight_gradients_many_empty_experts(tiles, act):
    """Most experts empty, one with split K and one small (the c3 pattern at
    a reduced size): gradients exact (ReLU, dyadic) or within tolerance
    (SwiGLU), and +0.0 for every empty expert."""
    E, d, f = 12, 512, 1024
    rows = [0, 0, 3000, 0, 0, 0, 5, 0, 0, 0, 0, 0]
    dyadic = act == "relu"
    rows, cap, off, R, P = _problem(E, d, f, rows, [0, 2, 0, 0, 1, 0, 0, 0, 3, 0, 0, 0], act,
                                    "bf16", dyadic, 90)
    valid, fw, bw = _oracle(rows, off, P, act, "bf16", E)
    g = _gpu(rows, cap, off, R, P, act, "bf16", E, d, f, tiles=tiles)
    _compare(g, valid, fw, bw, act, "bf16", exact=dyadic)
    empty = [e for e in range(E) if rows[e] == 0]
    for name in ("dw1", "dw2", "dw3"):
        if g[name] is not None:
            assert (g[name][empty] == 0).all() and not np.signbit(g[name][empty]).any(), name


@pytest.mark.parametrize("tiles", [1, 2])
def test_padded_static_rows_match_on_filled_rows(tiles):
    """rows = capacity (padded static-shape baseline): filled rows give the
    same results as rows = fill."""
    E, d, f = 3, 64, 128
    rows, cap, off, R, P = _problem(E, d, f, [50, 5, 100], [30, 60, 0], "relu", "bf16", True, 40)
    valid, fw, bw = _oracle(rows, off, P, "relu", "bf16", E)
    g = _gpu(rows, cap, off, R, P, "relu", "bf16", E, d, f, rows_kind="capacity", tiles=tiles)
    np.testing.assert_array_equal(g["y"][valid], fw["Y"])
    np.testing.assert_array_equal(g["dx"][valid], bw["dX"])


@pytest.mark.parametrize("act", ["relu", "gelu_tanh", "swiglu"])
def test_tile_kernels_bit_identical(act):
    """The 256x256 and the 128x128 kernels add every output's products in the
    same order (K steps of 64 in order, two MFMA k-halves per step, the same
    split-K segments), so on random bf16 inputs every output is identical bit
    for bit, and the automatic choice equals both; dX is the same whether it
    reads the weights K-major or from their transposed copy.  Shapes ragged
    in M, N and K with empty, one-row and split-K experts (d and f not
    multiples of the 64-element copy blocks); the backward of the SwiGLU
    case also runs dX with its W3 half starting at k = f."""
    E, d, f = 6, 392, 648
    rows = [700, 1, 0, 129, 300, 5000]
    rows, cap, off, R, P = _problem(E, d, f, rows, [3, 0, 1, 0, 2, 0], act, "bf16", False, 70)
    gs = [_gpu(rows, cap, off, R, P, act, "bf16", E, d, f, tiles=t, wcopy=c)
          for t, c in ((1, 1), (2, 1), (0, 0), (1, 2), (2, 2))]
    valid = np.concatenate([np.arange(off[e], off[e] + rows[e]) for e in range(E)])
    for name in ("h", "y", "dx", "dw1", "dw2", "dw3"):
        if gs[0][name] is None:
            continue
        a = gs[0][name][:, valid] if name == "h" else (gs[0][name][valid] if name in ("y", "dx") else gs[0][name])
        for g in gs[1:]:
            b = g[name][:, valid] if name == "h" else (g[name][valid] if name in ("y", "dx") else g[name])
            np.testing.assert_array_equal(a, b, err_msg=name)
    assert np.isfinite(gs[0]["dw1"]).all()


# ---- combine, combine backward, dispatch backward -----------------------------
@pytest.mark.parametrize("dt,k,d", [("bf16", 2, 512), ("f32", 1, 64), ("bf16", 3, 136),
                                    ("bf16", 5, 1096), ("f32", 2, 584),
                                    # rows of several 4-vector batches per lane plus a
                                    # ragged end (513, 250 and 257 16-byte vectors)
                                    ("bf16", 2, 4104), ("f32", 4, 1000), ("bf16", 1, 2056)])
def test_combine_and_backward(dt, k, d):
    rng = np.random.default_rng(50 + k)
    T, E = 1500, 6
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    counts = O.count_assignments(ids, E)
    cap = counts // 3                                 # drops, also of first choices
    off = O.exclusive_offsets(cap)
    R = int(off[-1])
    s = O.assign_slots(ids, E, cap, off, R)
    dest = s["dest_row"]
    assert (dest < 0).any()
    if k <= 3:     # with 5 picks of 6 experts every token keeps one
        assert ((dest < 0).all(axis=1)).any()
    wts = rng.random((T, k)).astype(np.float32)
    yd = _enc(rng.standard_normal((R, d)), dt)
    dy = _enc(rng.standard_normal((T, d)), dt)
    dxd = _enc(rng.standard_normal((R, d)), dt)
    dl = (rng.standard_normal((T, E)) * 0.1).astype(np.float32)
    wg = _enc(rng.standard_normal((E, d)) * 0.02, dt)
    td = torch_dtype(dt)
    t_dest = torch.from_numpy(dest.astype(np.int32)).to(dev())
    t_w = torch.from_numpy(wts).to(dev())
    y = torch.empty(T, d, dtype=td, device=dev())
    B.moe_combine(to_dev(yd, dt), t_dest, t_w, y)
    dyd = torch.full((R, d), float("nan"), dtype=td, device=dev())
    dwt = torch.empty(T, k, dtype=torch.float32, device=dev())
    B.moe_combine_bwd(to_dev(dy, dt), to_dev(yd, dt), t_dest, t_w, dyd, dwt)
    dx = torch.empty(T, d, dtype=td, device=dev())
    B.moe_dispatch_bwd(to_dev(dxd, dt), t_dest, E, torch.from_numpy(dl).to(dev()), to_dev(wg, dt), dx)
    dx2 = torch.empty(T, d, dtype=td, device=dev())
    B.moe_dispatch_bwd(to_dev(dxd, dt), t_dest, E, None, None, dx2)
    torch.cuda.synchronize()
    rt = RTOL[dt]
    Yd = _dec(yd, dt)
    assert_close(to_np(y), O.combine(Yd, dest, wts, dt), rt, "y")
    dw_ref, dyd_ref = O.combine_bwd(_dec(dy, dt), Yd, dest, wts, dt)
    assert_close(to_np(dwt), dw_ref, 1e-5 if dt == "f32" else 1e-4, "dweights")
    kept = s["src"] >= 0
    assert_close(to_np(dyd)[kept], dyd_ref[kept], rt, "dy_disp")
    Xd = _dec(dxd, dt)
    assert_close(to_np(dx), O.dispatch_bwd(Xd, dest, dl.astype(np.float64), _dec(wg, dt), dt), rt, "dx")
    assert_close(to_np(dx2), O.dispatch_bwd(Xd, dest, None, None, dt), rt, "dx (no gate)")
    assert (to_np(y)[(dest < 0).all(axis=1)] == 0).all()


# gates of 4 to 64 experts; 40 leaves a partial group of eight experts
@pytest.mark.parametrize("dt,E,k,renorm", [("bf16", 8, 2, 1), ("bf16", 64, 1, 0), ("f32", 4, 1, 0),
                                           ("bf16", 16, 3, 1), ("f32", 40, 2, 0),
                                           ("bf16", 40, 3, 1)])
def test_gate_backward(dt, E, k, renorm):
    rng = np.random.default_rng(60 + E)
    T, d = 1100, 264
    x = _enc(rng.standard_normal((T, d)), dt)
    logits = (rng.standard_normal((T, E)) * 2).astype(np.float32)
    ids = O.topk(logits, k)
    dwts = rng.standard_normal((T, k)).astype(np.float32)
    dwts[::7, 0] = 0.0                                 # as for dropped assignments
    dl = torch.empty(T, E, dtype=torch.float32, device=dev())
    dwg = torch.empty(E, d, dtype=torch.float32, device=dev())
    ws = B.workspace(B.moe_gate_bwd_workspace_bytes(T, d, E), dev())
    B.moe_gate_bwd(to_dev(x, dt), torch.from_numpy(logits).to(dev()),
                   torch.from_numpy(ids).to(dev()), torch.from_numpy(dwts).to(dev()), renorm, dl,
                   dwg, ws)
    torch.cuda.synchronize()
    dl_ref, dwg_ref = O.gate_bwd(logits, ids, dwts, renorm, _dec(x, dt))
    assert_close(to_np(dl), dl_ref, 1e-5, "dlogits")
    assert_close(to_np(dwg), dwg_ref, 1e-5, "dw_g")


@pytest.mark.parametrize("renorm", [0, 1])
def test_gate_backward_skips_invalid_cached_ids(renorm):
    """Cached picks with ids outside [0, E): the gate backward leaves them out
    of the normalisation, as moe_cached_weights does in the forward."""
    rng = np.random.default_rng(71)
    T, d, E, k = 700, 136, 8, 2
    x = _enc(rng.standard_normal((T, d)), "bf16")
    logits = (rng.standard_normal((T, E)) * 2).astype(np.float32)
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    ids[::5, 1] = E + 2
    ids[3::11, 0] = -4
    dwts = rng.standard_normal((T, k)).astype(np.float32)
    dwts[ids >= E] = 0.0
    dwts[ids < 0] = 0.0
    t_ids = torch.from_numpy(ids).to(dev())
    t_l = torch.from_numpy(logits).to(dev())
    w = torch.empty(T, k, dtype=torch.float32, device=dev())
    B.moe_cached_weights(t_l, t_ids, renorm, w)
    dl = torch.empty(T, E, dtype=torch.float32, device=dev())
    dwg = torch.empty(E, d, dtype=torch.float32, device=dev())
    ws = B.workspace(B.moe_gate_bwd_workspace_bytes(T, d, E), dev())
    B.moe_gate_bwd(to_dev(x, "bf16"), t_l, t_ids, torch.from_numpy(dwts).to(dev()), renorm, dl,
                   dwg, ws)
    torch.cuda.synchronize()
    assert_close(to_np(w), O.gate_weights(O.softmax(logits), ids, renorm), 1e-6, "weights")
    dl_ref, dwg_ref = O.gate_bwd(logits, ids, dwts, renorm, _dec(x, "bf16"))
    assert_close(to_np(dl), dl_ref, 1e-5, "dlogits")
    assert_close(to_np(dwg), dwg_ref, 1e-5, "dw_g")
