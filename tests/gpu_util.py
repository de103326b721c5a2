"""Helpers of the GPU parity tests: host <-> device copies of the seeded
inputs and the tolerance rule.

Tolerance rule (elementwise, on float64 values):
    |got - ref| <= rtol * (|ref| + rms(ref))
with rtol = 1e-5 for fp32 layers and 2e-2 for bf16 layers (fp32
accumulation).  The rms term keeps elements near zero (cancellation) from
demanding more relative accuracy than the tensor's scale carries.
Integer outputs (ids, counts, fill, dest_row, src, status) and the dispatched
rows are compared bit-exactly.
"""
import numpy as np
import torch

RTOL = {"f32": 1e-5, "bf16": 2e-2}

# Two logits closer than 8 fp32 ulps of the largest |logit| are a near tie:
# their order is not decided by the arithmetic (accumulation order differs
# between the kernel and the oracle), so both orders are valid routings.
NEAR_TIE = 8 * 2.0 ** -23


def scaled_small(W, name, **kw):
    """A reduced copy of a named workload whose gate logits keep the full
    config's scale (x_std = sqrt(d_full / d_small)), so routing skew and
    expert loads look like the full config's."""
    import math
    full = W.config(name)
    kw.setdefault("x_std", math.sqrt(full.d / kw.get("d", full.d)))
    return W.small(name, **kw)


def dev():
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    return torch.device("cuda:0")


def to_dev(a, dtype):
    """numpy array (bf16 bits as uint16, or float32/int32) -> device tensor."""
    if a is None:
        return None
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev())
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev())


def to_np(t):
    """device tensor -> float64 numpy (bf16/f32) or int64 (ints)."""
    t = t.detach().cpu()
    if t.dtype in (torch.int32, torch.int64):
        return t.numpy().astype(np.int64)
    return t.float().numpy().astype(np.float64)


def torch_dtype(dt):
    return torch.bfloat16 if dt == "bf16" else torch.float32


def assert_close(got, ref, rtol, name=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{name}: non-finite output"
    if ref.size == 0:
        return
    scale = np.sqrt(np.mean(ref ** 2))
    err = np.abs(got - ref) / (np.abs(ref) + scale + 1e-300)
    i = int(np.argmax(err))
    assert err.flat[i] <= rtol, (f"{name}: max rel err {err.flat[i]:.3e} > {rtol} at flat index "
                                 f"{i}: got {got.flat[i]!r} ref {ref.flat[i]!r}")


def min_topk_gap(logits, k):
    """Smallest gap between the k-th and (k+1)-th largest logit of any token
    (inf when k == E)."""
    l = np.sort(np.asarray(logits, np.float64), axis=1)[:, ::-1]
    if k >= l.shape[1]:
        return np.inf
    gaps = np.abs(l[:, k - 1] - l[:, k])
    # also gaps inside the top k decide the order of the picks
    for j in range(k - 1):
        gaps = np.minimum(gaps, np.abs(l[:, j] - l[:, j + 1]))
    return float(gaps.min())


def relu_kink_bound(n_values, eps=1e-5):
    """Upper bound on how many of n_values ReLU pre-activations fall within
    eps * rms of 0 (where fp32 summation order, not the arithmetic, decides
    relu'(H), so the row is excluded from the dX comparison).  For a
    pre-activation close to normal with standard deviation sigma = rms,
    P(|h| < eps sigma) = erf(eps / sqrt 2) ~ 0.80 eps; the mean is doubled
    for experts whose own scale is below the tensor's rms, then six standard
    deviations of a Poisson count and a floor of 4 are added."""
    import math
    mu = 2 * 0.8 * eps * n_values
    return int(mu + 6 * math.sqrt(mu) + 4)
