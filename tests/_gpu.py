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


def check_routing(idx_gpu, gate_gpu, idx_ref, gate_ref, margin, k):
    """Top-k ids bit-exact except at near-ties; gates within TOL_F32."""
    idx_gpu = np.asarray(idx_gpu)
    T = idx_gpu.shape[0]
    diff_rows = np.any(idx_gpu != idx_ref, axis=1)
    near = margin < NEAR_TIE
    assert not np.any(diff_rows & ~near), (
        f"routing differs away from near-ties at tokens {np.nonzero(diff_rows & ~near)[0][:10]}")
    n_mis = int(sum(len(set(idx_gpu[t]) ^ set(idx_ref[t])) // 2 for t in np.nonzero(diff_rows)[0]))
    assert n_mis <= MISMATCH_FRAC * T * k, f"{n_mis} mismatched routings of {T * k}"
    same = ~diff_rows
    err = rownorm_err(gate_gpu[same], gate_ref[same])
    assert err <= TOL_F32, f"gate error {err}"
    return int(diff_rows.sum()), err
