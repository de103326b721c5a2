"""GPU parity of the gate, load count, capacity and dispatch calls against
the CPU oracle (through the C ABI).  Integer results bit-exact."""
import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from gpu_util import NEAR_TIE, assert_close, dev, min_topk_gap, scaled_small, to_dev, to_np, torch_dtype
from paper_2205_01848_amd import binding as B

pytestmark = pytest.mark.gpu


def _run_gate(x_np, wg_np, b_np, k, renorm, dt):
    T, d = x_np.shape
    E = wg_np.shape[0]
    x = to_dev(W.to_bf16_bits(x_np) if dt == "bf16" else x_np.astype(np.float32), dt)
    wg = to_dev(W.to_bf16_bits(wg_np) if dt == "bf16" else wg_np.astype(np.float32), dt)
    b = None if b_np is None else torch.from_numpy(b_np.astype(np.float32)).to(dev())
    logits = torch.empty(T, E, dtype=torch.float32, device=dev())
    ids = torch.empty(T, k, dtype=torch.int32, device=dev())
    w = torch.empty(T, k, dtype=torch.float32, device=dev())
    B.moe_gate_topk(x, wg, b, k, renorm, logits, ids, w)
    torch.cuda.synchronize()
    return to_np(logits), to_np(ids), to_np(w)


# values in {-2..2}/4: every partial sum of the logits is exact in fp32, so
# the kernel's logits equal the oracle's bit for bit, ties included
@pytest.mark.parametrize("T,d,E,k,renorm,dt", [
    (1000, 256, 8, 2, 1, "bf16"),
    (517, 128, 64, 1, 0, "bf16"),
    (333, 64, 33, 3, 1, "bf16"),
    (70, 200, 16, 8, 1, "bf16"),
    (2000, 96, 24, 2, 1, "bf16"),     # 17-32 experts: four 8-row blocks of w_g
    (301, 72, 32, 3, 0, "bf16"),
    (1, 8, 1, 1, 0, "bf16"),
    # long batches: two waves per token tile, then one (whole rows per wave)
    (40001, 72, 8, 2, 1, "bf16"),
    (70001, 136, 40, 2, 1, "bf16"),
    # E <= 8 and 2048 < d <= 4096: the whole-row kernel (5 to 8 chunks of
    # 512 columns), ragged column tails, ragged 4-token groups and 32-token
    # batches, fewer tokens than waves
    (5003, 4096, 8, 2, 1, "bf16"),
    (2049, 2600, 5, 2, 1, "bf16"),
    (64, 2056, 8, 1, 0, "bf16"),
    (9, 3584, 3, 3, 1, "bf16"),
    (20001, 3072, 2, 2, 0, "bf16"),
    # just past its limits: the tiled kernel
    (300, 4104, 8, 2, 1, "bf16"),
    (250, 2056, 9, 2, 0, "bf16"),
    (777, 1800, 12, 3, 0, "bf16"),
    (129, 64, 4, 1, 0, "f32"),
    (300, 40, 64, 4, 1, "f32"),
])
def test_gate_exact_logits_and_ties(T, d, E, k, renorm, dt):
    rng = np.random.default_rng(T + d + E)
    x = rng.integers(-2, 3, (T, d)) / 4.0
    wg = rng.integers(-2, 3, (E, d)) / 4.0
    b = rng.integers(-4, 5, E) / 8.0
    logits, ids, w = _run_gate(x, wg, b, k, renorm, dt)
    r = O.route(x, wg, b.astype(np.float32), k, renorm)
    np.testing.assert_array_equal(logits, r["logits"].astype(np.float64))
    np.testing.assert_array_equal(ids, r["ids"])
    assert_close(w, r["weights"], 1e-5, "weights")
    ties = (np.sort(r["logits"], axis=1)[:, ::-1][:, :-1] ==
            np.sort(r["logits"], axis=1)[:, ::-1][:, 1:]).any() if E > 1 else False
    if T > 100 and E > 1:
        assert ties, "inputs were meant to contain exact ties"


@pytest.mark.parametrize("name", ["c2", "c3", "c5"])
def test_gate_random_inputs(name):
    wl = scaled_small(W, name, T=2000, d=256)
    I = W.make_inputs(wl)
    f64 = O.bf16_to_f64
    r = O.route(f64(I.x), f64(I.w_g), I.bias, wl.k, wl.renorm)
    scale = np.abs(r["logits"]).max()
    assert min_topk_gap(r["logits"], wl.k) > NEAR_TIE * scale, "seed has a near tie"
    logits, ids, w = _run_gate(f64(I.x), f64(I.w_g), I.bias, wl.k, wl.renorm, "bf16")
    assert_close(logits, r["logits"], 1e-5, "logits")
    np.testing.assert_array_equal(ids, r["ids"])
    assert_close(w, r["weights"], 1e-5, "weights")


# ---- count / capacity ---------------------------------------------------------
def test_count_with_faults():
    rng = np.random.default_rng(3)
    T, E, k = 9000, 16, 3
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    ids[5, 1] = E + 3
    ids[77, 2] = ids[77, 0]
    ids[8000, 0] = -1
    counts = torch.empty(E, dtype=torch.int32, device=dev())
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    B.moe_count(torch.from_numpy(ids).to(dev()), E, counts, status)
    np.testing.assert_array_equal(to_np(counts), O.count_assignments(ids, E))
    assert int(status.item()) == O.STATUS_BAD_ID | O.STATUS_DUP_ID


@pytest.mark.parametrize("T,k,E,num,den,cap_min", [
    (256, 1, 4, 5, 4, 0), (8192, 2, 16, 1, 1, 0), (16384, 1, 64, 2, 1, 0),
    (1000, 2, 7, 1, 3, 5), (10, 1, 1, 7, 1, 0)])
def test_capacity_static(T, k, E, num, den, cap_min):
    cap = torch.empty(E, dtype=torch.int32, device=dev())
    off = torch.empty(E + 1, dtype=torch.int32, device=dev())
    B.moe_update_capacity(T, k, E, None, num, den, cap_min, cap, off)
    ref = O.capacity_static(T, k, E, num, den, cap_min)
    np.testing.assert_array_equal(to_np(cap), ref)
    np.testing.assert_array_equal(to_np(off), O.exclusive_offsets(ref))


@pytest.mark.parametrize("num,den,cap_min", [(11, 10, 0), (21, 20, 0), (1, 1, 0), (3, 2, 4)])
def test_capacity_dynamic(num, den, cap_min):
    rng = np.random.default_rng(num)
    E, T = 64, 200000
    counts = rng.integers(0, T, E).astype(np.int32)
    counts[:6] = [0, 50, 90, 100, 1000, T]
    cap = torch.empty(E, dtype=torch.int32, device=dev())
    off = torch.empty(E + 1, dtype=torch.int32, device=dev())
    B.moe_update_capacity(T, 2, E, torch.from_numpy(counts).to(dev()), num, den, cap_min, cap, off)
    ref = O.capacity_dynamic(counts, T, num, den, cap_min)
    np.testing.assert_array_equal(to_np(cap), ref)
    np.testing.assert_array_equal(to_np(off), O.exclusive_offsets(ref))


# ---- dispatch ------------------------------------------------------------------
def _run_dispatch(x_np, ids, E, cap, off, rows_alloc, dt):
    T, d = x_np.shape
    k = ids.shape[1]
    x = to_dev(x_np, dt)
    t_ids = torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).to(dev())
    i32 = lambda a: torch.from_numpy(np.asarray(a, dtype=np.int32)).to(dev())
    counts = torch.empty(E, dtype=torch.int32, device=dev())
    fill = torch.empty(E, dtype=torch.int32, device=dev())
    dest = torch.full((T, k), 12345, dtype=torch.int32, device=dev())
    src = torch.full((max(rows_alloc, 1),), 777, dtype=torch.int32, device=dev())
    xd = torch.zeros(max(rows_alloc, 1), d, dtype=torch_dtype(dt), device=dev())
    status = torch.zeros(1, dtype=torch.int32, device=dev())
    ws = B.workspace(B.moe_dispatch_workspace_bytes(T, E, k), dev())
    B.moe_dispatch(x, t_ids, E, i32(cap), i32(off), rows_alloc, counts, fill, dest, src, xd,
                   status, ws)
    torch.cuda.synchronize()
    return dict(counts=to_np(counts), fill=to_np(fill), dest_row=to_np(dest),
                src=to_np(src)[:rows_alloc], x_disp=xd, status=int(status.item()))


def _check_dispatch(x_np, ids, E, cap, off, rows_alloc, dt="bf16"):
    g = _run_dispatch(x_np, ids, E, cap, off, rows_alloc, dt)
    s = O.assign_slots(ids, E, np.asarray(cap), np.asarray(off), rows_alloc)
    np.testing.assert_array_equal(g["counts"], s["counts"])
    np.testing.assert_array_equal(g["fill"], s["fill"])
    np.testing.assert_array_equal(g["dest_row"], s["dest_row"])
    np.testing.assert_array_equal(g["src"], s["src"])
    assert g["status"] == s["status"]
    # dispatched rows: exact copies (compared as raw bits)
    kept = s["src"] >= 0
    if kept.any():
        rows = np.nonzero(kept)[0]
        tok = s["src"][rows] // ids.shape[1]
        got = g["x_disp"][torch.from_numpy(rows).to(dev())].cpu()
        if dt == "bf16":
            np.testing.assert_array_equal(got.view(torch.int16).numpy().view(np.uint16), x_np[tok])
        else:
            np.testing.assert_array_equal(got.numpy(), x_np[tok])
    return g, s


def _bf16_rows(T, d, seed):
    return W.to_bf16_bits(np.random.default_rng(seed).standard_normal((T, d)).astype(np.float32))


# T*k = 65536 is the largest batch whose rank kernel also does the per-expert
# scan (64 chunks of 1024 assignments); 65538 takes the separate scan launch
@pytest.mark.parametrize("T,E,k,cap_kind", [
    (5000, 8, 2, "static"), (5000, 8, 2, "dynamic"), (777, 64, 1, "tight"),
    (4096, 5, 3, "zero_some"), (3, 4, 2, "tight"), (9000, 32, 2, "exact"),
    (32768, 16, 2, "tight"), (32769, 16, 2, "tight")])
def test_dispatch_random_ids(T, E, k, cap_kind):
    rng = np.random.default_rng(T * 7 + E)
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    counts = O.count_assignments(ids, E)
    if cap_kind == "static":
        cap = O.capacity_static(T, k, E, 1, 1)
    elif cap_kind == "dynamic":
        cap = O.capacity_dynamic(counts, T, 11, 10)
    elif cap_kind == "tight":
        cap = np.maximum(counts // 2, 0)
    elif cap_kind == "zero_some":
        cap = counts.copy()
        cap[::2] = 0
    else:
        cap = counts.copy()
    off = O.exclusive_offsets(cap)
    d = 136 if T < 100 else 64
    _check_dispatch(_bf16_rows(T, d, 1), ids, E, cap, off, int(off[-1]))


@pytest.mark.parametrize("dt,d", [("bf16", 4104), ("f32", 1032)])
def test_dispatch_wide_ragged_rows(dt, d):
    """Rows of several load batches per lane and a ragged end (513 and 258
    16-byte vectors), with drops."""
    rng = np.random.default_rng(d)
    T, E, k = 700, 8, 2
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    cap = np.maximum(O.count_assignments(ids, E) * 2 // 3, 1)
    off = O.exclusive_offsets(cap)
    x = (_bf16_rows(T, d, 5) if dt == "bf16"
         else rng.standard_normal((T, d)).astype(np.float32))
    _check_dispatch(x, ids, E, cap, off, int(off[-1]), dt=dt)


def test_dispatch_cached_zipf_ids_fp32_rows():
    wl = W.small("c4", T=6000, d=32, f=64)
    I = W.make_inputs(wl)
    counts = O.count_assignments(I.ids, wl.E)
    cap = O.capacity_dynamic(counts, wl.T, 1, 1)
    off = O.exclusive_offsets(cap)
    x = np.random.default_rng(2).standard_normal((wl.T, 24)).astype(np.float32)
    g, s = _check_dispatch(x, I.ids, wl.E, cap, off, int(off[-1]), dt="f32")
    assert (g["dest_row"] >= 0).all()


@pytest.mark.parametrize("T", [4500, 33000])   # scan in the rank kernel / its own launch
def test_dispatch_faults_and_region_overflow(T):
    rng = np.random.default_rng(9)
    E, k = 6, 2
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    ids[10, 0] = 99
    ids[11, 1] = -5
    ids[T - 100, 1] = ids[T - 100, 0]
    cap = np.full(E, T // 5)
    off = O.exclusive_offsets(cap)
    rows_alloc = int(off[-1]) - 1000                  # the last region does not fit
    g, s = _check_dispatch(_bf16_rows(T, 16, 3), ids, E, cap, off, rows_alloc)
    assert g["status"] == O.STATUS_BAD_ID | O.STATUS_DUP_ID | O.STATUS_REGION
    # overlapping regions
    off2 = off.copy()
    off2[3] = off2[2] + 100
    _check_dispatch(_bf16_rows(T, 16, 3), ids, E, cap, off2, int(off[-1]))


def test_dispatch_all_to_one_expert_and_empty_batch():
    T, E = 2500, 4
    ids = np.zeros((T, 1), dtype=np.int32)
    cap = np.array([700, 10, 10, 10])
    off = O.exclusive_offsets(cap)
    g, _ = _check_dispatch(_bf16_rows(T, 8, 4), ids, E, cap, off, int(off[-1]))
    assert list(g["fill"]) == [700, 0, 0, 0]
    g = _run_dispatch(np.zeros((0, 8), np.uint16), np.zeros((0, 1), np.int32), E, cap, off, 50,
                      "bf16")
    assert (g["counts"] == 0).all() and (g["fill"] == 0).all() and (g["src"] == -1).all()


@pytest.mark.parametrize("row_align", [256, 7])
def test_aligned_layout_routing_matches_oracle(row_align):
    """Regions aligned to row_align rows: capacities unchanged, offsets on
    multiples of the alignment, and the dispatch (counts, fill, dest_row, src,
    rows) bit-exact against the oracle in the same layout."""
    rng = np.random.default_rng(91)
    T, E, k, d = 5000, 8, 2, 64
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    ids[: T // 3, 0] = 0
    counts = O.count_assignments(ids, E)
    cap_ref = O.capacity_dynamic(counts * 9 // 10, T, 11, 10)       # lagged: some drops
    off_ref = O.exclusive_offsets(cap_ref, row_align)
    R = int(off_ref[-1]) + 3
    t_counts = torch.from_numpy((counts * 9 // 10).astype(np.int32)).to(dev())
    cap = torch.empty(E, dtype=torch.int32, device=dev())
    off = torch.empty(E + 1, dtype=torch.int32, device=dev())
    B.moe_update_capacity(T, k, E, t_counts, 11, 10, 0, cap, off, row_align=row_align)
    x = torch.from_numpy(W.to_bf16_bits(rng.standard_normal((T, d)).astype(np.float32))
                         .view(np.int16)).view(torch.bfloat16).to(dev())
    outs = dict(counts=torch.empty(E, dtype=torch.int32, device=dev()),
                fill=torch.empty(E, dtype=torch.int32, device=dev()),
                dest=torch.empty(T, k, dtype=torch.int32, device=dev()),
                src=torch.empty(R, dtype=torch.int32, device=dev()),
                xd=torch.zeros(R, d, dtype=torch.bfloat16, device=dev()),
                status=torch.zeros(1, dtype=torch.int32, device=dev()))
    ws = B.workspace(B.moe_dispatch_workspace_bytes(T, E, k), dev())
    B.moe_dispatch(x, torch.from_numpy(ids).to(dev()), E, cap, off, R, outs["counts"],
                   outs["fill"], outs["dest"], outs["src"], outs["xd"], outs["status"], ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(cap), cap_ref)
    np.testing.assert_array_equal(to_np(off), off_ref)
    assert (to_np(off)[:-1] % row_align == 0).all()
    s = O.assign_slots(ids, E, cap_ref, off_ref, R)
    np.testing.assert_array_equal(to_np(outs["counts"]), s["counts"])
    np.testing.assert_array_equal(to_np(outs["fill"]), s["fill"])
    np.testing.assert_array_equal(to_np(outs["dest"]), s["dest_row"])
    np.testing.assert_array_equal(to_np(outs["src"]), s["src"])
    assert int(outs["status"].item()) == s["status"]     # duplicates from the forced picks
    kept = s["dest_row"] >= 0
    xd = to_np(outs["xd"])
    X = to_np(x)
    tt, jj = np.nonzero(kept)
    np.testing.assert_array_equal(xd[s["dest_row"][tt, jj]], X[tt])


def test_policy_uploads_aligned_offsets():
    T, E, k = 1000, 4, 2
    pol = B.CapacityPolicy(T, k, E, 0, (11, 10), (3, 2), [500] * E, row_align=256)
    cap = torch.empty(E, dtype=torch.int32, device=dev())
    off = torch.empty(E + 1, dtype=torch.int32, device=dev())
    counts = torch.tensor([400, 600, 500, 500], dtype=torch.int32, device=dev())
    rows, _ = pol.begin(cap, off)
    pol.end(counts)
    assert rows == 4 * 512
    rows, rec = pol.begin(cap, off)              # sees iteration 0's counts: 600 overflowed
    pol.end(counts)
    torch.cuda.synchronize()
    pol.close()
    assert rec
    np.testing.assert_array_equal(to_np(cap), [440, 660, 550, 550])
    np.testing.assert_array_equal(to_np(off), O.exclusive_offsets([440, 660, 550, 550], 256))
    assert rows == int(O.exclusive_offsets([440, 660, 550, 550], 256)[-1])
