"""Shared helpers for the GPU parity tests (tolerances, uploads)."""
import numpy as np
import torch

# Tolerance on max|gpu - ref| / max|ref| per tensor: bf16 storage with float32
# accumulation, and the float32 debug mode.
TOL = {"bf16": 2e-2, "f32": 1e-4}


def rel_err(gpu, ref) -> float:
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    if gpu.size == 0:
        return 0.0
    den = np.max(np.abs(ref))
    num = np.max(np.abs(gpu - ref))
    if den == 0.0:
        return float(num)
    return float(num / den)


# Error statistics of the full-size cases, printed at the end of the session
# (conftest.pytest_terminal_summary): (case, tensor, max-normalised error,
# 99.9th percentile and maximum of the element-wise relative error).
STATS = []


def elem_rel(gpu, ref):
    """Element-wise |gpu - ref| / |ref|, with |ref| floored at 1e-3 max|ref|
    (elements near zero would otherwise dominate with a meaningless ratio)."""
    gpu = np.asarray(gpu, dtype=np.float64).ravel()
    ref = np.asarray(ref, dtype=np.float64).ravel()
    if ref.size == 0:
        return np.zeros(0)
    floor = 1e-3 * max(np.max(np.abs(ref)), 1e-300)
    return np.abs(gpu - ref) / np.maximum(np.abs(ref), floor)


def assert_close(name, gpu, ref, dtype, case=None):
    e = rel_err(gpu, ref)
    assert np.all(np.isfinite(np.asarray(gpu, dtype=np.float64))), "%s has non-finite values" % name
    if case is not None:
        r = elem_rel(gpu, ref)
        STATS.append((case, name, e, float(np.quantile(r, 0.999)) if r.size else 0.0,
                      float(r.max()) if r.size else 0.0))
    assert e <= TOL[dtype], "%s: max rel err %.3e > %.1e" % (name, e, TOL[dtype])
    return e


def dev(a, dtype=None):
    """Upload a numpy array (uint16 -> bfloat16 bit patterns)."""
    if a is None:
        return None
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.to(dtype)


def host(t):
    """Download to float64 numpy (bfloat16 widened exactly)."""
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy().astype(np.float64) if t.is_floating_point() else t.cpu().numpy()


def near_tie_ok(ids_gpu, ids_ref, logits_ref, tol=1e-4):
    """Tokens whose selected ids differ must be near-ties in the reference
    logits: every differing position j picks an expert whose logit is within
    tol*(1+|l|) of the reference's j-th choice. Returns the number of
    differing tokens."""
    diff = np.any(ids_gpu != ids_ref, axis=1)
    for t in np.nonzero(diff)[0]:
        l = logits_ref[t]
        for j in range(ids_ref.shape[1]):
            a, b = l[ids_gpu[t, j]], l[ids_ref[t, j]]
            assert abs(a - b) <= tol * (1 + abs(b)), (t, j, ids_gpu[t], ids_ref[t], a, b)
    return int(diff.sum())
