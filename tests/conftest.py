import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs a real MI355X (HIP device); skipped on CPU-only hosts")


def pytest_collection_modifyitems(config, items):
    # GPU tests need a visible HIP device; on a CPU-only host they are
    # skipped rather than failed so that `-m "not gpu"` and a plain run agree.
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:  # pragma: no cover
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="no HIP device visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    # The routing checks record what the near-tie rule excluded (tokens whose
    # device top-k differs from the oracle's at a near-tie).  Print them at
    # the end of the run, where -q output keeps them.
    mod = sys.modules.get("_gpu")
    recs = getattr(mod, "ROUTING_RECORDS", None) if mod else None
    if not recs:
        return
    tr = terminalreporter
    tr.write_sep("-", "near-tie routing exclusions (device vs oracle top-k)")
    tot_tok = sum(r["T"] for r in recs)
    tot_rt = sum(r["T"] * r["k"] for r in recs)
    tot_diff = sum(r["tokens_differ"] for r in recs)
    tot_mis = sum(r["routings_differ"] for r in recs)
    for r in recs:
        if r["tokens_differ"] or r["T"] >= 4096:
            tr.write_line(
                f"{r['label']}: T={r['T']} k={r['k']}: {r['tokens_differ']} tokens differ "
                f"({r['set_differ']} in the set, {r['order_differ']} in slot order only), "
                f"{r['routings_differ']} of {r['T'] * r['k']} routings, "
                f"max gate err {r['gate_err']:.2e}")
    tr.write_line(f"all {len(recs)} routing checks: {tot_diff} of {tot_tok} tokens excluded "
                  f"as near-ties, {tot_mis} of {tot_rt} routings differ "
                  f"({tot_mis / max(tot_rt, 1):.2e})")
