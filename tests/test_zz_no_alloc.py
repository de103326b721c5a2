"""The allocation-free dispatch (moe_dispatch_noalloc, for callers that
cannot allocate device memory) against moe_dispatch with a caller workspace,
through the C ABI: bit-identical routing and dispatched rows on two calls in
a row, the second smaller than the first, so nothing left in the library's
fixed scratch by the first call may leak into the second."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_util import dev
from paper_2205_01848_amd import binding as B

pytestmark = pytest.mark.gpu


def _case(seed, T, d, E, k, dt, lag):
    rng = np.random.default_rng(seed)
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    ids[rng.random(T) < 0.4, 0] = 0                    # skewed loads
    if seed % 2:
        ids[5, 0] = E + 1                              # a bad cached id (status bit 1)
    counts = np.bincount(ids[(ids >= 0) & (ids < E)], minlength=E)
    cap = (counts * 9 // 10) if lag else counts        # lagged capacities drop some
    off = np.concatenate([[0], np.cumsum(cap)]).astype(np.int32)
    R = int(off[-1]) + 3
    if dt == "bf16":
        x = torch.from_numpy(W.to_bf16_bits(rng.standard_normal((T, d)).astype(np.float32))
                             .view(np.int16)).view(torch.bfloat16)
    else:
        x = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32))
    i32 = lambda a: torch.from_numpy(np.asarray(a, dtype=np.int32)).to(dev())
    return dict(x=x.to(dev()), ids=i32(ids), cap=i32(cap), off=i32(off), R=R, E=E)


def _outputs(c, d, fn):
    T, k = c["ids"].shape
    R, E = c["R"], c["E"]
    o = dict(counts=torch.full((E,), -7, dtype=torch.int32, device=dev()),
             fill=torch.full((E,), -7, dtype=torch.int32, device=dev()),
             dest_row=torch.full((T, k), -7, dtype=torch.int32, device=dev()),
             src=torch.full((R,), -7, dtype=torch.int32, device=dev()),
             x_disp=torch.zeros(R, d, dtype=c["x"].dtype, device=dev()),
             status=torch.zeros(1, dtype=torch.int32, device=dev()))
    fn(o)
    return o


def _run_both(c):
    d = c["x"].shape[1]
    args = lambda o: (c["x"], c["ids"], c["E"], c["cap"], c["off"], c["R"], o["counts"],
                      o["fill"], o["dest_row"], o["src"], o["x_disp"], o["status"])
    T, k = c["ids"].shape
    ws = B.workspace(B.moe_dispatch_workspace_bytes(T, c["E"], k), dev())
    ref = _outputs(c, d, lambda o: B.moe_dispatch(*args(o), ws))
    got = _outputs(c, d, lambda o: B.moe_dispatch_noalloc(*args(o)))
    torch.cuda.synchronize()
    return ref, got


def test_noalloc_dispatch_matches_dispatch_on_two_calls():
    big = _case(1, 70000, 136, 64, 2, "bf16", lag=True)     # 137 routing chunks: separate scan
    small = _case(2, 3001, 64, 8, 3, "f32", lag=False)      # 9 chunks: scan inside the rank kernel
    for c in (big, small):
        ref, got = _run_both(c)
        for name in ref:
            assert torch.equal(ref[name], got[name]), name
    assert int(small["ids"].shape[0]) < int(big["ids"].shape[0])


def test_noalloc_dispatch_refuses_more_than_its_scratch():
    cap = B.moe_dispatch_noalloc_max_assignments()
    assert cap == 1 << 21
    T, k, E, d = cap // 2 + 1, 2, 4, 8                      # T*k one pair past the limit
    x = torch.empty(T, d, dtype=torch.bfloat16, device=dev())
    ids = torch.zeros(T, k, dtype=torch.int32, device=dev())
    z = lambda n: torch.zeros(n, dtype=torch.int32, device=dev())
    with pytest.raises(B.MoEError, match="workspace"):
        B.moe_dispatch_noalloc(x, ids, E, z(E), z(E + 1), 8, z(E), z(E), z(T * k).view(T, k),
                               z(8), torch.empty(8, d, dtype=torch.bfloat16, device=dev()), z(1))
