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


# One entry per check_routing call: what the near-tie rule excluded.  The
# test session prints them at its end (tests/conftest.py), so the counts
# appear in the run's output even under -q.
ROUTING_RECORDS = []


def check_routing(idx_gpu, gate_gpu, idx_ref, gate_ref, logits_ref, k, alive=None,
                  renorm=True, label=None):
    """Check a device routing against the oracle's.

    Every token: its slots hold distinct alive experts (as many as are alive,
    up to k), the rest -1 with gate 0.  A token whose ids equal the oracle's
    slot for slot must have the oracle's gates (within TOL_F32).  A token
    whose ids differ is accepted only as a near-tie alternative, judged on
    the oracle's float32 logits l (the decision precision) with l_(k) the
    oracle's k-th largest alive logit and tolerance NEAR_TIE:
      1. every selected expert has l >= l_(k) - NEAR_TIE;
      2. every alive expert left out has l <= l_(k) + NEAR_TIE;
      3. consecutive slots are non-increasing in l up to NEAR_TIE;
      4. its gates equal the oracle's gates of the device's own selection
         (``oracle.moe.selection_gates``) within TOL_F32.
    The (token, slot) routings whose expert differs from the oracle's set
    must stay at or below MISMATCH_FRAC * T * k.
    Returns (tokens that differ, max gate error) and appends a record to
    ROUTING_RECORDS."""
    from oracle.moe import selection_gates   # test infrastructure (the oracle)

    idx_gpu = np.asarray(idx_gpu)
    idx_ref = np.asarray(idx_ref)
    gate_gpu = np.asarray(gate_gpu, np.float64)
    gate_ref = np.asarray(gate_ref, np.float64)
    T = idx_gpu.shape[0]
    l32 = np.asarray(logits_ref, np.float64).astype(np.float32).astype(np.float64)
    E = l32.shape[1] if l32.ndim == 2 else 0
    alive_m = np.ones(E, bool) if alive is None else np.asarray(alive).astype(bool)
    kk = min(k, int(alive_m.sum()))
    assert idx_gpu.shape == (T, k) and gate_gpu.shape == (T, k), "routing shape"
    # validity of every token's selection
    sel = idx_gpu[:, :kk]
    assert np.all((sel >= 0) & (sel < E)), "a slot that must hold an expert holds none"
    assert np.all(alive_m[sel]), "a dead expert was selected"
    if kk > 1:
        s = np.sort(sel, axis=1)
        assert np.all(s[:, 1:] != s[:, :-1]), "an expert repeats within a token"
    assert np.all(idx_gpu[:, kk:] == -1) and np.all(gate_gpu[:, kk:] == 0), \
        "slots beyond the alive experts must be empty"
    diff = np.any(idx_gpu != idx_ref, axis=1)
    same = ~diff
    err_same = rownorm_err(gate_gpu[same], gate_ref[same])
    assert err_same <= TOL_F32, f"gate error {err_same} on tokens routed as the oracle"
    n_set = n_order = n_mis = 0
    err_diff = 0.0
    toks = np.nonzero(diff)[0]
    if toks.size:
        lm = np.where(alive_m[None, :], l32[toks], -np.inf)
        lk = np.take_along_axis(lm, idx_ref[toks, kk - 1:kk].astype(np.int64), axis=1)[:, 0]
        lsel = np.take_along_axis(lm, sel[toks].astype(np.int64), axis=1)
        left_out = np.ones_like(lm, bool)
        np.put_along_axis(left_out, sel[toks].astype(np.int64), False, axis=1)
        left_out &= alive_m[None, :]
        c1 = np.all(lsel >= lk[:, None] - NEAR_TIE, axis=1)
        c2 = np.all(np.where(left_out, lm, -np.inf) <= lk[:, None] + NEAR_TIE, axis=1)
        c3 = np.all(lsel[:, :-1] >= lsel[:, 1:] - NEAR_TIE, axis=1) if kk > 1 else \
            np.ones(toks.size, bool)
        bad = ~(c1 & c2 & c3)
        assert not np.any(bad), (
            f"routing differs away from a near-tie at tokens {toks[bad][:10]} "
            f"(selected within tie {c1[bad][:10]}, excluded within tie {c2[bad][:10]}, "
            f"slot order {c3[bad][:10]})")
        g_own = selection_gates(np.asarray(logits_ref)[toks], idx_gpu[toks], alive=alive_m,
                                renorm=renorm)
        err_diff = rownorm_err(gate_gpu[toks], g_own)
        assert err_diff <= TOL_F32, \
            f"gates of near-tie tokens {toks[:10]} differ from their own selection's: {err_diff}"
        set_diff = np.array([set(a.tolist()) != set(b.tolist())
                             for a, b in zip(idx_gpu[toks], idx_ref[toks])])
        n_set = int(set_diff.sum())
        n_order = int((~set_diff).sum())
        n_mis = int(sum(len(set(idx_gpu[t].tolist()) - set(idx_ref[t].tolist())) for t in toks))
    assert n_mis <= MISMATCH_FRAC * T * k, f"{n_mis} mismatched routings of {T * k}"
    ROUTING_RECORDS.append(dict(label=label or _current_test(), T=T, k=k, tokens_differ=int(diff.sum()),
                                set_differ=n_set, order_differ=n_order, routings_differ=n_mis,
                                gate_err=max(err_same, err_diff)))
    return int(diff.sum()), max(err_same, err_diff)


def _current_test():
    import os
    return os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]
