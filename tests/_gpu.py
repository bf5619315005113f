"""Helpers of the GPU parity tests: host<->device conversion and the error
metrics.  No arithmetic of the layer lives here."""
import sys

import numpy as np
import torch

TOL_F32 = 1e-5      # fp32 outputs: max row-normwise relative error
TOL_BF16 = 2e-2     # bf16 outputs (fp32 accumulation)
NEAR_TIE = 1e-4     # logit margin under which a different top-k is acceptable
MISMATCH_FRAC = 1e-4  # at most this fraction of routings may differ (near-ties only)

DEV = "cuda"


def case(msg: str):
    """Name the case before a GPU step (so a fault can be attributed)."""
    print(f"[gpu case] {msg}", flush=True)
    sys.stdout.flush()


def dev(a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(DEV).to(dtype)


def host(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64) if t.is_floating_point() \
        else t.detach().cpu().numpy()


def rownorm_err(got, ref) -> float:
    """max over rows of max|got - ref| / max|ref| (rows whose reference is all
    zero are compared absolutely)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if got.ndim == 1:
        got, ref = got[None], ref[None]
    got = got.reshape(got.shape[0], -1)
    ref = ref.reshape(ref.shape[0], -1)
    if got.size == 0:
        return 0.0
    num = np.abs(got - ref).max(axis=1)
    den = np.abs(ref).max(axis=1)
    den = np.where(den == 0, 1.0, den)
    return float((num / den).max())


def _adjacent_gaps(logits, alive, k):
    """Boundary margin l_(k) - l_(k+1) and the smallest gap between adjacent
    selected logits, on float32-rounded logits (the decision precision)."""
    l = np.asarray(logits, np.float64).astype(np.float32).astype(np.float64)
    if alive is not None:
        l = np.where(np.asarray(alive, bool)[None, :], l, -np.inf)
    s = -np.sort(-l, axis=1)
    n = min(k + 1, s.shape[1])
    gaps = s[:, :n - 1] - s[:, 1:n]
    gaps = np.where(np.isfinite(gaps), gaps, np.inf)
    boundary = gaps[:, k - 1] if n == k + 1 else np.full(s.shape[0], np.inf)
    inner = gaps[:, :k - 1].min(axis=1) if k > 1 else np.full(s.shape[0], np.inf)
    return boundary, inner


def check_routing(idx_gpu, gate_gpu, idx_ref, gate_ref, logits_ref, k, alive=None):
    """Top-k ids bit-exact except at near-ties: a different selected set is
    allowed only where the k-th and (k+1)-th logits are within NEAR_TIE, a
    different slot order only where two selected logits are within NEAR_TIE.
    Gates of the rows that match are within TOL_F32."""
    idx_gpu = np.asarray(idx_gpu)
    T = idx_gpu.shape[0]
    boundary, inner = _adjacent_gaps(logits_ref, alive, k)
    set_diff = np.array([set(a.tolist()) != set(b.tolist()) for a, b in zip(idx_gpu, idx_ref)])
    ord_diff = np.any(idx_gpu != idx_ref, axis=1) & ~set_diff
    bad = (set_diff & ~(boundary < NEAR_TIE)) | (ord_diff & ~(inner < NEAR_TIE))
    assert not np.any(bad), (
        f"routing differs away from near-ties at tokens {np.nonzero(bad)[0][:10]}")
    n_mis = int(sum(len(set(idx_gpu[t]) ^ set(idx_ref[t])) // 2 for t in np.nonzero(set_diff)[0]))
    assert n_mis <= MISMATCH_FRAC * T * k, f"{n_mis} mismatched routings of {T * k}"
    same = ~(set_diff | ord_diff)
    err = rownorm_err(gate_gpu[same], gate_ref[same])
    assert err <= TOL_F32, f"gate error {err}"
    return int((set_diff | ord_diff).sum()), err
