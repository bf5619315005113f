"""C-ABI contract tests that need no GPU: the library loads, exports every
symbol the header declares, rejects invalid arguments on the host before any
HIP call, and its host rearrangement utility matches the oracle."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))
                 if f.endswith(".h"))


@pytest.fixture(scope="module")
def L():
    import paper_2601_14327_amd as laep

    # tests/test_host_sanitizers.py reruns this module against the host
    # sanitizer build of the library
    alt = os.environ.get("LAEP_ABI_TEST_LIB")
    if alt:
        from paper_2601_14327_amd._lib import bind

        return bind(ctypes.CDLL(alt))
    if not os.path.exists(laep.LIB_PATH):
        from paper_2601_14327_amd import build

        build.build()
    return laep.lib()


def _declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M))
    return sorted(names)


def test_header_declares_the_hot_path_calls():
    names = _declared_functions()
    for n in ["moe_route", "moe_expert_counts", "laep_prune_mask", "moe_permute",
              "moe_grouped_ffn_fwd", "moe_grouped_ffn_bwd", "moe_combine", "moe_combine_bwd",
              "moe_permute_bwd", "moe_workspace_bytes", "laep_rearrange", "laep_last_error",
              "moe_route_bwd", "laep_expert_pruning", "laep_compact_experts",
              "laep_repack_experts", "moe_grouped_ffn_fwd_gather",
              "moe_grouped_ffn_fwd_gather_combine"]:
        assert n in names, n


def test_library_exports_every_declared_symbol(L):
    for n in _declared_functions():
        assert hasattr(L, n), f"{n} declared in include/*.h but not exported"


def test_binding_covers_every_declared_symbol():
    from paper_2601_14327_amd._lib import SIGNATURES

    assert set(_declared_functions()) == set(SIGNATURES)


P = ctypes.c_void_p


def _fake(n=1):
    # host memory stands in for device pointers: validation must reject the
    # call before touching it
    buf = (ctypes.c_uint8 * (64 * n))()
    addr = ctypes.addressof(buf)
    return buf, (addr + 15) & ~15


def _err(L):
    return L.laep_last_error().decode()


def test_route_validation(L):
    keep, p = _fake()
    assert L.moe_route(p, p, None, None, 7, 16, 64, 8, 2, 1, None, p, p, None, 0, None) == 2
    assert "dtype" in _err(L)
    assert L.moe_route(p, p, None, None, 1, 16, 64, 8, 9, 1, None, p, p, None, 0, None) == 1
    assert "k=9" in _err(L)
    assert L.moe_route(p, p, None, None, 1, 16, 64, 300, 2, 1, None, p, p, None, 0, None) == 1
    assert L.moe_route(p, p, None, None, 1, 16, 60, 8, 2, 1, None, p, p, None, 0, None) == 1
    assert L.moe_route(None, p, None, None, 1, 16, 64, 8, 2, 1, None, p, p, None, 0, None) == 1
    assert L.moe_route(p + 2, p, None, None, 1, 16, 64, 8, 2, 1, None, p, p, None, 0, None) == 1
    assert "aligned" in _err(L)
    # empty input is a valid no-op that launches nothing
    assert L.moe_route(None, None, None, None, 1, 0, 64, 8, 2, 1, None, None, None, None, 0, None) == 0


def test_counts_validation_and_workspace(L):
    keep, p = _fake()
    need = L.moe_workspace_bytes(1, 1000, 8, 64, 0, 0)
    assert need > 0
    assert L.moe_expert_counts(p, 1000, 8, 64, p, p, p, None, None, p, need - 1, None) == 3
    assert "workspace" in _err(L)
    assert L.moe_expert_counts(p, 1000, 8, 64, None, p, p, None, None, p, need, None) == 1


def test_prune_validation(L):
    keep, p = _fake()
    assert L.laep_prune_mask(p, 0, 100, math.inf, 0.1, p, p, None) == 1
    assert L.laep_prune_mask(p, 8, -1, math.inf, 0.1, p, p, None) == 1
    assert L.laep_prune_mask(p, 8, 100, math.nan, 0.1, p, p, None) == 1
    assert L.laep_prune_mask(None, 8, 100, math.inf, 0.1, p, p, None) == 1


def test_ffn_validation(L):
    keep, p = _fake()
    # d_model not a multiple of 64
    assert L.moe_grouped_ffn_fwd(p, p, p, p, None, 1, 8, 96, 128, 64, p, None, p, 1 << 30, None) == 2
    assert L.moe_grouped_ffn_fwd(p, p, p, p, None, 1, 8, 128, 128, 64, p, None, p, 16, None) == 3
    assert L.moe_grouped_ffn_fwd(p, p, p, p, None, 5, 8, 128, 128, 64, p, None, p, 1 << 30, None) == 2
    # bf16: one expert's weights are addressed with 32-bit offsets (under 2 GiB)
    assert L.moe_grouped_ffn_fwd(p, p, p, p, None, 1, 8, 32768, 16384, 64, p, None, p, 16,
                                 None) == 2
    assert "2 GiB" in _err(L)
    assert L.moe_grouped_ffn_fwd(p, p, p, p, None, 1, 8, 32768, 16320, 64, p, None, p, 16,
                                 None) == 3
    # backward: only bf16
    assert L.moe_grouped_ffn_bwd(p, p, p, None, p, p, p, None, 0, 8, 128, 128, 64, p, p, p, 0,
                                 p, 1 << 30, None) == 2
    assert "LAEP_BF16" in _err(L)
    # the forward's H (h_fwd) is optional but, when given, 16-byte aligned
    assert L.moe_grouped_ffn_bwd(p, p, p, p + 2, p, p, p, None, 1, 8, 128, 128, 64, p, p, p, 0,
                                 p, 1 << 30, None) == 1
    assert "aligned" in _err(L)
    # fused dispatch: bf16 only, R <= T*k, row_src required
    g = L.moe_grouped_ffn_fwd_gather
    assert g(p, p, 10, 2, p, p, p, None, 0, 8, 128, 128, 20, p, None, None, p, 1 << 30,
             None) == 2
    assert g(p, p, 10, 2, p, p, p, None, 1, 8, 128, 128, 21, p, None, None, p, 1 << 30,
             None) == 1
    assert g(p, None, 10, 2, p, p, p, None, 1, 8, 128, 128, 20, p, None, None, p, 1 << 30,
             None) == 1
    # the copy of the dispatched rows must not alias y_perm, and is 16-byte aligned
    q = p + 16
    assert g(p, p, 10, 2, p, p, p, None, 1, 8, 128, 128, 20, q, None, q, p, 1 << 30,
             None) == 1
    assert "alias" in _err(L)
    assert g(p, p, 10, 2, p, p, p, None, 1, 8, 128, 128, 20, q, None, p + 2, p, 1 << 30,
             None) == 1
    assert "aligned" in _err(L)
    # gather + combine: one slot per token only, R <= T, out not aliasing y_perm
    gc = L.moe_grouped_ffn_fwd_gather_combine
    assert gc(p, p, 10, 2, p, p, p, None, p, 1, 8, 128, 128, 20, p, None, None, None, p,
              1 << 30, None) == 2
    assert "one slot per token" in _err(L)
    assert gc(p, p, 10, 1, p, p, p, None, p, 0, 8, 128, 128, 10, p, None, None, None, p,
              1 << 30, None) == 2
    assert gc(p, p, 10, 1, p, p, p, None, p, 1, 8, 128, 128, 11, p, None, None, None, p,
              1 << 30, None) == 1
    assert gc(p, p, 10, 1, p, p, p, None, None, 1, 8, 128, 128, 10, p, None, None, None, p,
              1 << 30, None) == 1
    assert gc(p, p, 10, 1, p, p, p, None, p, 1, 8, 128, 128, 10, p, p, None, None, p, 1 << 30,
              None) == 1
    assert "alias" in _err(L)
    assert gc(p, p, 10, 1, p, p, p, None, p, 1, 8, 128, 128, 10, q, None, None, q, p, 1 << 30,
              None) == 1
    assert "alias" in _err(L)
    # x addressed with 32-bit offsets: T * d_model * 2 bytes under 2 GiB
    assert g(p, p, 1 << 19, 2, p, p, p, None, 1, 8, 2048, 128, 20, p, None, None, p, 1 << 30,
             None) == 2


def test_route_bwd_validation(L):
    keep, p = _fake()
    args = lambda **kw: dict(dict(dgate=p, idx=p, gate=p, logits=None, alive=None, x=p, w=p,
                                  offsets=p, row_src=p, dtype=1, T=16, d=64, E=8, k=2, renorm=1,
                                  dl=None, dw=p, db=None, dx=p, acc=0, ws=p, wsb=1 << 20), **kw)
    call = lambda a: L.moe_route_bwd(a["dgate"], a["idx"], a["gate"], a["logits"], a["alive"],
                                     a["x"], a["w"], a["offsets"], a["row_src"], a["dtype"],
                                     a["T"], a["d"], a["E"], a["k"], a["renorm"], a["dl"],
                                     a["dw"], a["db"], a["dx"], a["acc"], a["ws"], a["wsb"], None)
    assert call(args(row_src=None)) == 1          # renorm needs the dispatch order
    assert "row_src" in _err(L)
    assert call(args(renorm=0)) == 1              # full softmax needs the logits
    assert "logits" in _err(L)
    assert call(args(dtype=5)) == 2
    assert call(args(k=9)) == 1
    assert call(args(wsb=16)) == 3
    assert call(args(dw=None, db=p)) == 1        # dbias comes with dw_router
    assert "dbias" in _err(L)
    assert call(args(w=None, dx=None, dw=None)) == 1
    assert "w_router" in _err(L)
    need = L.moe_workspace_bytes(4, 16, 2, 8, 0, 0)
    assert need >= 16 * 8 * 4
    # the segment partials of the weight gradient grow with d_model
    assert L.moe_workspace_bytes(4, 16, 2, 8, 64, 0) >= need + 64 * 4


def test_calib_validation(L):
    keep, p = _fake()
    assert L.laep_calib_copy(p, p + 2, 64, None) == 1
    assert L.laep_calib_copy(p, p, 60, None) == 1
    assert L.laep_calib_copy(None, p, 64, None) == 1
    assert L.laep_calib_mfma(0, 10, p, None) == 1
    assert L.laep_calib_mfma(8, 0, p, None) == 1
    assert L.laep_calib_mfma(8, 10, None, None) == 1
    # blocked read: block sizes outside [8 KiB, 128 KiB], not a multiple of
    # 8 KiB or not dividing the byte count; null or misaligned pointers
    assert L.laep_calib_read(p, 1 << 20, 4096, p, None) == 1
    assert L.laep_calib_read(p, 1 << 20, 262144, p, None) == 1
    assert L.laep_calib_read(p, 1 << 20, 12288, p, None) == 1
    assert L.laep_calib_read(p, 100000, 8192, p, None) == 1
    assert L.laep_calib_read(None, 1 << 20, 8192, p, None) == 1
    assert L.laep_calib_read(p, 1 << 20, 8192, None, None) == 1
    assert L.laep_calib_read(p + 2, 1 << 20, 8192, p, None) == 1


def test_rowop_validation(L):
    keep, p = _fake()
    assert L.moe_permute(p, 1, p, 10, 2, 12, p, None) == 1
    assert L.moe_combine(p, p, p, 10, 0, 64, 1, p, None) == 1
    assert L.moe_combine_bwd(p, p, p, p, 10, 2, 64, 3, p, p, None) == 2
    assert L.moe_permute_bwd(p, None, 10, 2, 64, 1, p, None) == 1


def test_workspace_sizes_are_monotone(L):
    a = L.moe_workspace_bytes(2, 1024, 1, 16, 256, 256)
    b = L.moe_workspace_bytes(2, 4096, 1, 16, 256, 256)
    assert 0 < a < b
    assert L.moe_workspace_bytes(3, 1024, 1, 16, 256, 256) > 0
    assert L.moe_workspace_bytes(0, 1024, 1, 16, 256, 256) == 0


def _rearrange(L, loads, ng):
    loads = np.ascontiguousarray(loads, dtype=np.float64)
    n = loads.shape[0]
    group_of, order = np.empty(n, np.int32), np.empty(n, np.int32)
    sums = np.empty(max(ng, 1), np.float64)
    rc = L.laep_rearrange(loads.ctypes.data, n, ng, group_of.ctypes.data, order.ctypes.data,
                          sums.ctypes.data)
    return rc, dict(group_of=group_of, order=order, sums=sums[:ng])


def test_rearrange_matches_oracle(L):
    from oracle import laep as olaep
    from paper_2601_14327_amd import laep_rearrange

    rng = np.random.default_rng(0)
    cases = [([40, 30, 20, 10, 5, 5], 2), ([100, 1, 1, 1], 2), ([9, 8, 7, 6, 5], 2)]
    for _ in range(200):
        n = int(rng.integers(1, 80))
        cases.append((rng.integers(0, 1000, n).astype(float).tolist(), int(rng.integers(1, n + 1))))
    for i, (loads, ng) in enumerate(cases):
        rc, got = _rearrange(L, loads, ng)
        assert rc == 0
        if i < 3:   # the Python binding gives the same placement
            b = laep_rearrange(loads, ng)
            for key in got:
                np.testing.assert_array_equal(b[key], got[key])
        want = olaep.rearrange(loads, ng)
        np.testing.assert_array_equal(got["group_of"], want["group_of"])
        np.testing.assert_array_equal(got["order"], want["order"])
        np.testing.assert_array_equal(got["sums"], want["sums"])


def test_rearrange_errors(L):
    from paper_2601_14327_amd import LaepError, laep_rearrange

    with pytest.raises(LaepError):
        laep_rearrange([1.0, 2.0], 0)
    assert _rearrange(L, [1.0, 2.0], 0)[0] == 1
    assert L.laep_rearrange(None, 3, 2, None, None, None) == 1
    # no experts: valid, the group sums are zero
    rc, got = _rearrange(L, [], 3)
    assert rc == 0 and np.all(got["sums"] == 0)


def test_expert_pruning_validation(L):
    keep, p = _fake()
    a3 = (ctypes.c_double * 3)(0.2, 0.4, 0.2)
    ok_args = dict(etn=p, it=2, L=3, E=8, total=100, alpha=a3, beta=0.1, alive=p, n=p, mk=None)

    def call(**kw):
        a = dict(ok_args, **kw)
        return L.laep_expert_pruning(a["etn"], a["it"], a["L"], a["E"], a["total"], a["alpha"],
                                     a["beta"], a["alive"], a["n"], a["mk"], None)

    assert call(it=0) == 1 and "ITER" in _err(L)
    assert call(L=0) == 1
    assert call(L=257, alpha=(ctypes.c_double * 257)()) == 1
    assert call(E=300) == 1
    assert call(etn=None) == 1
    assert call(alpha=None) == 1
    assert call(total=-1) == 1
    assert call(beta=-0.5) == 1
    assert call(alpha=(ctypes.c_double * 3)(0.2, float("nan"), 0.2)) == 1
    assert "alpha[1]" in _err(L)
    assert call(alpha=(ctypes.c_double * 3)(0.2, -1.0, 0.2)) == 1


def test_compact_and_repack_validation(L):
    keep, p = _fake()
    assert L.laep_compact_experts(p, 1, 300, p, p, None) == 1
    assert L.laep_compact_experts(p, 0, 8, p, p, None) == 1
    assert L.laep_compact_experts(None, 1, 8, p, p, None) == 1
    # (expert_map, E, n_out, dtype, d, f, w_r, bias, w_gu, w_d, w_r', bias', w_gu', w_d')
    rp = L.laep_repack_experts
    assert rp(p, 8, 4, 5, 64, 64, p, None, p, p, p, None, p, p, None) == 2
    assert rp(None, 8, 4, 1, 64, 64, p, None, p, p, p, None, p, p, None) == 1
    assert rp(p, 8, -1, 1, 64, 64, p, None, p, p, p, None, p, p, None) == 1
    assert rp(p, 8, 4, 1, 60, 64, p, None, p, p, p, None, p, p, None) == 1
    assert rp(p, 8, 4, 1, 64, 64, p, None, p, p, None, None, p, p, None) == 1
    assert "both" in _err(L)
    assert rp(p, 8, 4, 1, 64, 0, p, None, p, p, p, None, p, p, None) == 1
    assert rp(p, 8, 4, 1, 64, 64, p + 4, None, p, p, p, None, p, p, None) == 1
    assert "aligned" in _err(L)
    # nothing to copy: valid, and enqueues nothing
    assert rp(p, 8, 0, 1, 64, 64, p, None, p, p, p, None, p, p, None) == 0


def test_route_count_noalloc_validation(L):
    """The allocation-free route + count call: the same argument checks as
    moe_route_count, and shapes whose counting scratch exceeds the library's
    array are rejected before anything is enqueued."""
    keep, p = _fake()
    call = lambda T, E, k, x=p, dtype=1, d=64: L.moe_route_count_noalloc(
        x, p, None, None, dtype, T, d, E, k, 1, None, p, p, p, p, p, None, None, None)
    assert call(16, 8, 9) == 1 and "k=9" in _err(L)
    assert call(16, 8, 2, dtype=7) == 2
    assert call(16, 8, 2, x=None) == 1 and "moe_route_count_noalloc" in _err(L)
    assert call(16, 8, 2, x=p + 2) == 1 and "aligned" in _err(L)
    limit = 8 << 20
    assert L.moe_workspace_bytes(1, 691840, 8, 64, 0, 0) <= limit
    assert L.moe_workspace_bytes(1, 691841 + 63, 8, 64, 0, 0) > limit
    assert call(700000, 64, 8) == 3
    assert "scratch" in _err(L) and "moe_route_count" in _err(L)
    assert call(200000, 256, 8) == 3


def test_ffn_bwd_gather_validation(L):
    """The fused backward: without dy_perm it needs dout and the gates; bf16
    only; R <= T*k; x and dout under 2 GiB."""
    keep, p = _fake()
    g = L.moe_grouped_ffn_bwd_gather
    # (dy, dout, gate, x, row_src, T, k, act, h, wgu, wd, off, emap, dtype, E, d, f, R,
    #  dx, dwgu, dwd, acc, ws, wsb, stream)
    ok = lambda **kw: dict(dict(dy=p, dout=None, gate=None, x=p, rs=p, T=10, k=2, dtype=1, R=20,
                                h=None), **kw)
    call = lambda a: g(a["dy"], a["dout"], a["gate"], a["x"], a["rs"], a["T"], a["k"], p,
                       a["h"], p, p, p, None, a["dtype"], 8, 128, 128, a["R"], p, p, p, 0, p,
                       1 << 30, None)
    assert call(ok(dy=None)) == 1 and "dout" in _err(L)
    assert call(ok(dy=None, dout=p)) == 1 and "topk_gate" in _err(L)
    assert call(ok(dtype=0)) == 2
    assert call(ok(R=21)) == 1
    assert call(ok(rs=None)) == 1
    assert call(ok(dy=None, dout=p + 2, gate=p)) == 1 and "aligned" in _err(L)
    big = g(None, p, p, p, p, 1 << 20, 1, p, None, p, p, p, None, 1, 8, 1024, 128, 20, p, p, p,
            0, p, 1 << 40, None)
    assert big == 2 and "2 GiB" in _err(L)
