"""The allocation-free route + count call (moe_route_count_noalloc) against
the workspace call it shares its kernels with (moe_route_count), through the
C ABI: two calls in a row on the library's scratch array, the second with a
smaller input, every output bit-identical; the routing also against the
oracle."""
import numpy as np
import pytest
import torch

import oracle.moe as om
import paper_2601_14327_amd as laep
from workloads import random_case
from _gpu import case, check_routing, dev, host

pytestmark = pytest.mark.gpu


def _run(fn, x, wr, k, bias, E, **kw):
    etn = torch.zeros(E, dtype=torch.int64, device="cuda")
    out = fn(x, wr, k, bias=bias, want_logits=True, want_row_src=True, etn_accum=etn, **kw)
    return list(out) + [etn]


def test_noalloc_route_count_matches_workspace_call():
    # largest first (two-level counting scan: more than 512 wave tiles), then
    # smaller shapes on the same scratch array
    shapes = [(40000, 256, 64, 8, 1.0), (1000, 192, 40, 5, 2.0), (300, 128, 256, 16, 0.5)]
    for T, d, E, k, bstd in shapes:
        c = random_case(31 * T + E, T=T, d_model=d, E=E, k=k, d_ff=64, dtype="bf16",
                        bias_std=bstd, weight_std=0.05)
        x, wr = dev(c["x"], torch.bfloat16), dev(c["w_router"], torch.bfloat16)
        bias = dev(c["bias"], torch.float32)
        case(f"route_count_noalloc T={T} d={d} E={E} k={k}")
        got = _run(laep.moe_route_count_noalloc, x, wr, k, bias, E)
        ref = _run(laep.moe_route_count, x, wr, k, bias, E)
        torch.cuda.synchronize()
        names = ["topk_idx", "topk_gate", "counts", "offsets", "dest_row", "row_src", "logits",
                 "etn"]
        for n, a, b in zip(names, got, ref):
            assert torch.equal(a, b), f"{n} differs from moe_route_count (T={T}, E={E})"
        ridx, rgate, _, rlog = om.route(c["x"], c["w_router"], k, bias=c["bias"])
        check_routing(host(got[0]), host(got[1]), ridx, rgate, rlog, k,
                      label=f"route_count_noalloc T={T} E={E}")
        rc, ro, rd = om.expert_counts(host(got[0]), E)
        np.testing.assert_array_equal(host(got[2]), rc)
        np.testing.assert_array_equal(host(got[3]), ro)
        np.testing.assert_array_equal(host(got[4]), rd)
        np.testing.assert_array_equal(host(got[7]), rc)


def test_noalloc_rejects_oversized_scratch():
    x = torch.zeros((700000, 64), dtype=torch.bfloat16, device="cuda")
    wr = torch.zeros((64, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(laep.LaepError) as ei:
        laep.moe_route_count_noalloc(x, wr, 8)
    assert ei.value.code == 3 and "scratch" in ei.value.msg
