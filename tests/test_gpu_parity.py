"""GPU parity of every step of the layer against the CPU oracle, through the
C ABI, at sizes the oracle finishes in seconds (several tiles, ragged tails,
edge cases).  Stages are teacher-forced: each GPU stage is fed the GPU's own
upstream outputs and compared with the oracle on those same inputs."""
import math

import numpy as np
import pytest
import torch

import oracle.moe as om
import oracle.laep as ol
import paper_2601_14327_amd as laep
from workloads import WORKLOADS, generate, random_case
from _gpu import (TOL_BF16, TOL_F32, case, check_routing, dev, host, rownorm_err)

pytestmark = pytest.mark.gpu

TD = {"bf16": torch.bfloat16, "f32": torch.float32}


def _route_case(c, k, dtype, renorm=True, alive=None):
    td = TD[dtype]
    x, wr = dev(c["x"], td), dev(c["w_router"], td)
    bias = dev(c["bias"], torch.float32) if "bias" in c else None
    alive_t = None if alive is None else dev(alive.astype(np.uint8), torch.uint8)
    idx, gate, logits = laep.moe_route(x, wr, k, bias=bias, alive=alive_t, renorm=renorm,
                                       want_logits=True)
    torch.cuda.synchronize()
    ridx, rgate, margin, rlog = om.route(c["x"], c["w_router"], k, bias=c.get("bias"),
                                        alive=alive, renorm=renorm)
    return host(idx), host(gate), host(logits), ridx, rgate, margin, rlog


# ---------------------------------------------------------------------------
# routing
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("T,d,E,k,dtype,renorm,bias", [
    (256, 128, 8, 2, "f32", False, 0.0),      # tiny fp32 layer, top-2 of a softmax
    (256, 128, 8, 2, "f32", True, 0.0),
    (1000, 256, 64, 8, "bf16", True, 0.0),    # ragged token tail
    (777, 512, 64, 8, "bf16", True, 2.0),     # biased router
    (333, 192, 40, 5, "bf16", False, 0.0),    # E not a multiple of 32
    (300, 384, 100, 6, "bf16", True, 1.0),    # LDS-staged router, 128-column chunks, 4 expert blocks
    (96, 128, 8, 2, "bf16", False, 0.0),      # LDS-staged router, one 128-column chunk
    (130, 64, 256, 16, "bf16", True, 0.5),    # largest expert count
    (65, 136, 3, 3, "bf16", True, 0.0),       # k = E, d not a multiple of 16
    (1, 64, 1, 1, "f32", True, 0.0),          # one token, one expert
])
def test_route_parity(T, d, E, k, dtype, renorm, bias):
    case(f"route T={T} d={d} E={E} k={k} {dtype} renorm={renorm} bias={bias}")
    c = random_case(T * 7 + E, T=T, d_model=d, E=E, k=k, d_ff=64, dtype=dtype, bias_std=bias,
                    weight_std=0.05)
    idx, gate, logits, ridx, rgate, margin, rlog = _route_case(c, k, dtype, renorm)
    check_routing(idx, gate, ridx, rgate, rlog, k, renorm=renorm)
    assert rownorm_err(logits, rlog) <= TOL_F32


def test_route_with_alive_mask_and_too_few_alive():
    T, d, E, k = 300, 128, 16, 4
    c = random_case(5, T=T, d_model=d, E=E, k=k, d_ff=64, dtype="bf16", weight_std=0.05)
    alive = np.ones(E, bool)
    alive[[0, 3, 4, 9, 15]] = False
    case("route alive mask (11 of 16)")
    idx, gate, logits, ridx, rgate, margin, rlog = _route_case(c, k, "bf16", True, alive)
    check_routing(idx, gate, ridx, rgate, rlog, k, alive)
    assert not np.isin(idx, np.nonzero(~alive)[0]).any()
    assert np.all(np.isneginf(logits[:, ~alive]))
    alive2 = np.zeros(E, bool)
    alive2[[2, 7]] = True
    case("route alive mask (2 of 16 < k)")
    idx, gate, *_ = _route_case(c, k, "bf16", True, alive2)
    assert np.all(idx[:, 2:] == -1) and np.all(gate[:, 2:] == 0)
    assert np.all(np.sort(idx[:, :2], axis=1) == [2, 7])
    np.testing.assert_allclose(gate[:, :2].sum(1), 1.0, rtol=1e-6)


@pytest.mark.parametrize("T,d,E,k,dtype,renorm,dead", [
    (8192, 2048, 64, 8, "bf16", True, False),   # LDS-staged router, whole tiles
    (100, 256, 64, 8, "bf16", True, True),      # ragged: 4 workgroups, last tile half empty
    (33, 128, 16, 4, "bf16", False, False),     # odd number of workgroups
    (1, 64, 8, 2, "f32", True, False),
    (300, 384, 200, 6, "bf16", True, True),     # register path (7 expert blocks)
    (257, 96, 40, 5, "f32", False, True),
])
def test_route_count_matches_route_then_counts(T, d, E, k, dtype, renorm, dead):
    """moe_route_count is bit-identical to moe_route followed by moe_expert_counts."""
    c = random_case(T + 3 * E, T=T, d_model=d, E=E, k=k, d_ff=64, dtype=dtype, bias_std=1.0,
                    weight_std=0.05)
    td = TD[dtype]
    x, w = dev(c["x"], td), dev(c["w_router"], td)
    bias = dev(c["bias"], torch.float32)
    alive = None
    if dead:
        a = np.ones(E, np.uint8)
        a[np.random.default_rng(E).choice(E, E // 4, replace=False)] = 0
        alive = dev(a, torch.uint8)
    case(f"route_count T={T} d={d} E={E} k={k} {dtype} renorm={renorm} dead={dead}")
    idx, gate, logits = laep.moe_route(x, w, k, bias=bias, alive=alive, renorm=renorm,
                                       want_logits=True)
    etn1 = torch.full((E,), 3, dtype=torch.int64, device="cuda")
    counts, offsets, dest, row_src = laep.moe_expert_counts(idx, E, want_row_src=True,
                                                           etn_accum=etn1)
    etn2 = torch.full((E,), 3, dtype=torch.int64, device="cuda")
    f = laep.moe_route_count(x, w, k, bias=bias, alive=alive, renorm=renorm, want_logits=True,
                             want_row_src=True, etn_accum=etn2)
    torch.cuda.synchronize()
    for got, ref, name in zip(f, (idx, gate, counts, offsets, dest, row_src, logits),
                              ("idx", "gate", "counts", "offsets", "dest_row", "row_src",
                               "logits")):
        assert torch.equal(got, ref), name
    assert torch.equal(etn1, etn2)
    rc, ro, rd = om.expert_counts(host(idx), E)
    np.testing.assert_array_equal(host(f[2]), rc)
    np.testing.assert_array_equal(host(f[4]), rd)


def test_route_count_empty_and_validation():
    x = torch.zeros((0, 64), dtype=torch.bfloat16, device="cuda")
    w = dev(np.ones((8, 64), np.float32), torch.bfloat16)
    case("route_count T=0")
    idx, gate, counts, offsets, dest, _, _ = laep.moe_route_count(x, w, 2)
    torch.cuda.synchronize()
    assert host(counts).tolist() == [0] * 8 and host(offsets).tolist() == [0] * 9
    with pytest.raises(laep.LaepError):
        laep.moe_route_count(dev(np.ones((4, 64), np.float32), torch.bfloat16), w, 9)


# ---------------------------------------------------------------------------
# counts / offsets / dispatch permutation
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("T,E,k", [(1, 1, 1), (63, 8, 2), (64, 8, 2), (1000, 64, 8),
                                   (4097, 256, 16), (2000, 16, 1), (500, 5, 5)])
def test_counts_bit_exact(T, E, k):
    rng = np.random.default_rng(T + E)
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    case(f"counts T={T} E={E} k={k}")
    etn = torch.full((E,), 5, dtype=torch.int64, device="cuda")
    counts, offsets, dest, row_src = laep.moe_expert_counts(
        dev(idx, torch.int32), E, want_row_src=True, etn_accum=etn)
    torch.cuda.synchronize()
    rc, ro, rd = om.expert_counts(idx, E)
    np.testing.assert_array_equal(host(counts), rc)
    np.testing.assert_array_equal(host(offsets), ro)
    np.testing.assert_array_equal(host(dest), rd)
    rs = host(row_src)
    np.testing.assert_array_equal(rs[rd], np.arange(T * k))
    np.testing.assert_array_equal(host(etn), rc + 5)


@pytest.mark.parametrize("T,E,k", [(32769, 64, 8), (40000, 5, 2), (131072, 256, 4),
                                   (70000, 16, 1)])
def test_counts_two_level_scan(T, E, k):
    """More than 512 wave tiles: the counting pass scans in two levels (block
    partials, one workgroup over the blocks, then the tile bases)."""
    rng = np.random.default_rng(T + 3 * E)
    idx = np.argsort(rng.random((T, E)), axis=1)[:, :k].astype(np.int32)
    idx[rng.random(T) < 0.01, -1] = -1          # a few unrouted slots
    case(f"counts two-level T={T} E={E} k={k}")
    etn = torch.full((E,), 7, dtype=torch.int64, device="cuda")
    counts, offsets, dest, row_src = laep.moe_expert_counts(
        dev(idx, torch.int32), E, want_row_src=True, etn_accum=etn)
    torch.cuda.synchronize()
    rc, ro, rd = om.expert_counts(idx, E)
    np.testing.assert_array_equal(host(counts), rc)
    np.testing.assert_array_equal(host(offsets), ro)
    np.testing.assert_array_equal(host(dest), rd)
    routed = rd >= 0
    np.testing.assert_array_equal(host(row_src)[rd[routed]], np.nonzero(routed)[0])
    np.testing.assert_array_equal(host(etn), rc + 7)


@pytest.mark.parametrize("T,E,k", [(16384, 64, 8), (16385, 64, 8), (4096, 256, 8),
                                   (4097, 256, 8), (9000, 3, 2), (130, 256, 1)])
def test_counts_mid_sizes(T, E, k):
    """Mid sizes around 16384 (wave tile, expert) pairs, up to 256 experts and
    down to 3, with unrouted slots."""
    rng = np.random.default_rng(T * 7 + E)
    idx = np.argsort(rng.random((T, E)), axis=1)[:, :k].astype(np.int32)
    idx[rng.random(T) < 0.02, -1] = -1
    case(f"counts mid sizes T={T} E={E} k={k}")
    etn = torch.full((E,), 3, dtype=torch.int64, device="cuda")
    counts, offsets, dest, row_src = laep.moe_expert_counts(
        dev(idx, torch.int32), E, want_row_src=True, etn_accum=etn)
    torch.cuda.synchronize()
    rc, ro, rd = om.expert_counts(idx, E)
    np.testing.assert_array_equal(host(counts), rc)
    np.testing.assert_array_equal(host(offsets), ro)
    np.testing.assert_array_equal(host(dest), rd)
    routed = rd >= 0
    np.testing.assert_array_equal(host(row_src)[rd[routed]], np.nonzero(routed)[0])
    np.testing.assert_array_equal(host(etn), rc + 3)


def test_counts_skew_unrouted_and_empty_experts():
    rng = np.random.default_rng(3)
    T, E, k = 3000, 32, 4
    idx = np.full((T, k), -1, np.int32)
    for t in range(T):
        m = rng.integers(1, k + 1)
        idx[t, :m] = rng.choice([0, 1, 2, 5, 31], size=m, replace=False)
    case("counts skewed with unrouted slots")
    counts, offsets, dest = laep.moe_expert_counts(dev(idx, torch.int32), E)
    torch.cuda.synchronize()
    rc, ro, rd = om.expert_counts(idx, E)
    np.testing.assert_array_equal(host(counts), rc)
    np.testing.assert_array_equal(host(offsets), ro)
    np.testing.assert_array_equal(host(dest), rd)


def test_counts_zero_tokens():
    case("counts T=0")
    counts, offsets, dest = laep.moe_expert_counts(
        torch.empty((0, 2), dtype=torch.int32, device="cuda"), 8)
    torch.cuda.synchronize()
    assert host(counts).tolist() == [0] * 8 and host(offsets).tolist() == [0] * 9


# ---------------------------------------------------------------------------
# LAEP prune mask
# ---------------------------------------------------------------------------
def test_prune_mask_parity():
    rng = np.random.default_rng(21)
    cases = [([35, 1, 20, 4, 2, 25, 3, 10], 100, math.inf, 0.1),
             ([35, 1, 20, 4, 2, 25, 3, 10], 100, 0.2, 0.1),
             ([5, 5, 5, 85], 100, math.inf, 0.1), ([5, 5, 90], 100, math.inf, 0.1),
             ([0] * 64, 0, math.inf, 0.05)]
    for _ in range(150):
        E = int(rng.integers(1, 257))
        counts = (rng.pareto(0.8, E) * 40).astype(np.int64)
        total = int(counts.sum())
        cases.append((counts.tolist(), total, float(rng.choice([math.inf, 0.2, 0.4, 1.5])),
                      float(rng.choice([0.0, 0.05, 0.1, 0.3, 1.0]))))
    case(f"prune {len(cases)} cases")
    for counts, total, alpha, beta in cases:
        alive, n = laep.laep_prune_mask(dev(np.array(counts, np.int32), torch.int32), total,
                                        alpha, beta)
        ra, rn, _ = ol.prune_mask(counts, total, alpha, beta)
        np.testing.assert_array_equal(host(alive).astype(bool), ra)
        assert int(host(n)[0]) == rn


# ---------------------------------------------------------------------------
# permute / combine / permute_bwd / combine_bwd
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("T,d,E,k", [(1000, 256, 16, 4), (37, 72, 5, 2), (300, 4096, 8, 1)])
def test_rowops_parity(dtype, T, d, E, k):
    rng = np.random.default_rng(T + d)
    td = TD[dtype]
    c = random_case(T, T=T, d_model=d, E=E, k=k, d_ff=64, dtype=dtype)
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    if T > 10:
        idx[5, -1] = -1   # an unrouted slot
    gate = rng.uniform(0.05, 1, (T, k)).astype(np.float32)
    rc, ro, rd = om.expert_counts(idx, E)
    R = int(ro[E])
    case(f"rowops {dtype} T={T} d={d} k={k}")
    x = dev(c["x"], td)
    dest = dev(rd.astype(np.int32), torch.int32)
    xp = laep.moe_permute(x, dest, k, R)
    torch.cuda.synchronize()
    xq = host(x)
    np.testing.assert_array_equal(host(xp), om.permute(xq, rd, k))    # bit-exact copy
    y = dev(rng.standard_normal((R, d)).astype(np.float32), td)
    g = dev(gate, torch.float32)
    out = laep.moe_combine(y, g, dest)
    dxp = laep.moe_permute_bwd(y, dest, T, k)
    dout = dev(rng.standard_normal((T, d)).astype(np.float32), td)
    dy, dgate = laep.moe_combine_bwd(dout, y, g, dest)
    torch.cuda.synchronize()
    tol = TOL_BF16 if dtype == "bf16" else TOL_F32
    yq, dq = host(y), host(dout)
    assert rownorm_err(host(out), om.combine(yq, gate, rd, k, dtype=dtype)) <= tol
    assert rownorm_err(host(dxp), om.permute_bwd(yq, rd, k, dtype=dtype)) <= tol
    rdy, rdg = om.combine_bwd(dq, yq, gate, rd, k, dtype=dtype)
    routed = rd >= 0
    got_dy = host(dy)
    assert rownorm_err(got_dy, rdy) <= tol
    # dgate is a dot product: bound the error by its condition, sum |dout * y|
    cond = np.zeros((T, k))
    for t in range(T):
        for j in range(k):
            r = rd[t * k + j]
            if r >= 0:
                cond[t, j] = np.abs(dq[t] * yq[r]).sum()
    assert np.all(np.abs(host(dgate) - rdg) <= TOL_F32 * cond + 1e-30)
    if T > 10:
        assert host(dgate)[5, -1] == 0.0


# ---------------------------------------------------------------------------
# grouped SwiGLU FFN
# ---------------------------------------------------------------------------
def _ffn_inputs(seed, counts, d, f, dtype, E_phys=None):
    rng = np.random.default_rng(seed)
    E = len(counts)
    E_phys = E if E_phys is None else E_phys
    R = int(sum(counts))
    c = random_case(seed, T=R, d_model=d, E=E_phys, k=1, d_ff=f, dtype=dtype)
    offsets = np.zeros(E + 1, np.int64)
    offsets[1:] = np.cumsum(counts)
    return c["x"], c["w_gate_up"], c["w_down"], offsets


@pytest.mark.parametrize("dtype,counts,d,f", [
    ("f32", [60, 0, 200, 5, 1, 130, 64, 52], 128, 256),          # tiny fp32 layer shape
    ("bf16", [60, 0, 200, 5, 1, 130, 64, 52], 128, 256),
    ("bf16", [300, 129, 128, 0, 7, 1000, 1, 40], 256, 192),       # ragged, f % 128 = 64
    ("bf16", [0, 0, 0, 513], 320, 128),                           # one expert takes all
    ("bf16", [64] * 16, 512, 512),
    # 512 tiles per product: several per persistent workgroup, with a
    # one-step k-loop in the gate/up (K = d = 64) or the down product (K = f = 64)
    ("bf16", [1024] * 31 + [1000], 64, 512),
    ("bf16", [1000] + [1024] * 31, 1024, 64),
    ("bf16", [300, 0, 513, 64], 2048, 1024),                      # the balanced layer's width
])
def test_ffn_fwd_parity(dtype, counts, d, f):
    x, wgu, wd, offsets = _ffn_inputs(len(counts) * 31 + d, counts, d, f, dtype)
    td = TD[dtype]
    case(f"ffn fwd {dtype} counts={counts} d={d} f={f}")
    y, act = laep.moe_grouped_ffn_fwd(dev(x, td), dev(wgu, td), dev(wd, td),
                                      dev(offsets.astype(np.int32), torch.int32))
    torch.cuda.synchronize()
    ry, ract = om.grouped_ffn_fwd(x, wgu, wd, offsets, dtype=dtype)
    tol = TOL_BF16 if dtype == "bf16" else TOL_F32
    assert rownorm_err(host(y), ry) <= tol
    assert rownorm_err(host(act), ract) <= tol


def test_ffn_fwd_expert_map_with_pruned_slots():
    counts = [100, 0, 37, 0, 250]
    d, f = 256, 128
    x, wgu, wd, offsets = _ffn_inputs(9, counts, d, f, "bf16", E_phys=3)
    emap = np.array([2, -1, 0, -1, 1], np.int32)
    case("ffn fwd expert_map")
    y, _ = laep.moe_grouped_ffn_fwd(dev(x, torch.bfloat16), dev(wgu, torch.bfloat16),
                                    dev(wd, torch.bfloat16),
                                    dev(offsets.astype(np.int32), torch.int32),
                                    expert_map=dev(emap, torch.int32))
    torch.cuda.synchronize()
    ry, _ = om.grouped_ffn_fwd(x, wgu, wd, offsets, expert_map=emap, dtype="bf16")
    assert rownorm_err(host(y), ry) <= TOL_BF16


@pytest.mark.parametrize("T,k,E,d,f,mapped", [
    (300, 4, 8, 256, 128, False),    # ragged tiles, top-4
    (257, 1, 3, 128, 256, False),    # one slot per token
    (700, 8, 12, 192, 192, True),    # expert_map with unused slots, f % 128 = 64
])
def test_ffn_fwd_gather_matches_permute_then_ffn(T, k, E, d, f, mapped):
    rng = np.random.default_rng(T + 13 * E)
    c = random_case(T + E, T=T, d_model=d, E=E + 2 if mapped else E, k=1, d_ff=f, dtype="bf16")
    # k distinct experts per token (as routing gives), expert E-1 never chosen
    # (an empty expert) and expert 0 preferred (a heavy one)
    w = np.r_[3.0, np.ones(E - 2), 0.0]
    ids = np.stack([rng.choice(E, size=k, replace=False, p=w / w.sum()) for _ in range(T)])
    bf = torch.bfloat16
    x, wgu, wd = dev(c["x"], bf), dev(c["w_gate_up"], bf), dev(c["w_down"], bf)
    emap = dev(np.array([(e + 2) if mapped else e for e in range(E)], np.int32), torch.int32) \
        if mapped else None
    idx = dev(ids.astype(np.int32), torch.int32)
    case(f"ffn fwd gather T={T} k={k} E={E} d={d} f={f} mapped={mapped}")
    counts, offsets, dest_row, row_src = laep.moe_expert_counts(idx, E, want_row_src=True)
    x_perm = laep.moe_permute(x, dest_row, k)
    y1, a1 = laep.moe_grouped_ffn_fwd(x_perm, wgu, wd, offsets, expert_map=emap)
    xp_copy = torch.full_like(x_perm, 5.0)
    y2, a2 = laep.moe_grouped_ffn_fwd_gather(x, row_src, k, wgu, wd, offsets, expert_map=emap,
                                            save_act=True, x_perm_out=xp_copy)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    assert torch.equal(a1, a2)
    assert torch.equal(xp_copy, x_perm)   # the dispatched rows written beside the FFN
    # and against the oracle's permute + grouped FFN
    rc, ro, rd = om.expert_counts(ids, E)
    xp = om.permute(c["x"], rd, k)
    ry, ract = om.grouped_ffn_fwd(xp, c["w_gate_up"], c["w_down"], ro,
                                  expert_map=host(emap) if mapped else None, dtype="bf16")
    assert rownorm_err(host(y2), ry) <= TOL_BF16
    assert rownorm_err(host(a2), ract) <= TOL_BF16


@pytest.mark.parametrize("T,k,E,d,f,mapped", [
    (300, 4, 8, 256, 128, False),    # ragged tiles, top-4, an empty expert
    (257, 1, 3, 128, 256, False),    # one slot per token
    (700, 8, 12, 192, 192, True),    # expert_map with unused slots, f % 128 = 64
    (90, 2, 5, 64, 64, False),       # experts shorter than one 64-row k-step
    (1500, 6, 8, 128, 128, False),   # long experts: many k-steps of gathered rows
])
def test_ffn_bwd_gather_matches_permute_then_bwd(T, k, E, d, f, mapped):
    """The weight gradient reading X's routed rows from the token rows through
    row_src (moe_grouped_ffn_bwd_gather) is bit-identical to moe_permute +
    moe_grouped_ffn_bwd, with and without the forward's H, and so is the
    variant that forms dY = g * dout on load (against moe_combine_bwd's
    dy_perm); its weight gradients match the oracle (teacher-forced on the
    GPU's dA and H)."""
    rng = np.random.default_rng(3 * T + E)
    n_phys = E + 2 if mapped else E
    c = random_case(T + 3 * E, T=T, d_model=d, E=n_phys, k=1, d_ff=f, dtype="bf16")
    w = np.r_[3.0, np.ones(E - 2), 0.0] if E > 2 else np.ones(E)
    ids = np.stack([rng.choice(E, size=k, replace=False, p=w / w.sum()) for _ in range(T)])
    bf = torch.bfloat16
    x, wgu, wd = dev(c["x"], bf), dev(c["w_gate_up"], bf), dev(c["w_down"], bf)
    emap_h = np.array([e + 2 for e in range(E)], np.int32) if mapped else None
    emap = dev(emap_h, torch.int32) if mapped else None
    idx = dev(ids.astype(np.int32), torch.int32)
    case(f"ffn bwd gather T={T} k={k} E={E} d={d} f={f} mapped={mapped}")
    counts, offsets, dest_row, row_src = laep.moe_expert_counts(idx, E, want_row_src=True)
    R = T * k
    x_perm = laep.moe_permute(x, dest_row, k)
    ws_f = torch.empty(laep.workspace_bytes(laep.LAEP_CALL_FFN_FWD, R, 1, E, d, f),
                       dtype=torch.uint8, device="cuda")
    _, act = laep.moe_grouped_ffn_fwd(x_perm, wgu, wd, offsets, expert_map=emap, ws=ws_f,
                                      save_act=True)
    h_f = laep.ffn_fwd_h_view(ws_f, R, f, bf)
    dy = dev(rng.standard_normal((R, d)).astype(np.float32), bf)
    zeros = lambda t: torch.zeros(t.shape, dtype=torch.float32, device="cuda")
    for use_h in (False, True):
        h = h_f if use_h else None
        a = laep.moe_grouped_ffn_bwd(dy, x_perm, act, wgu, wd, offsets, h_fwd=h,
                                     expert_map=emap, dw_gate_up=zeros(wgu), dw_down=zeros(wd))
        b = laep.moe_grouped_ffn_bwd_gather(dy, x, row_src, k, act, wgu, wd, offsets, h_fwd=h,
                                            expert_map=emap, dw_gate_up=zeros(wgu),
                                            dw_down=zeros(wd), return_ws=True)
        torch.cuda.synchronize()
        for n, u, g in zip(("dx_perm", "dw_gate_up", "dw_down"), a, b[:3]):
            assert torch.equal(u, g), f"{n} differs (use_h={use_h})"
    # dY formed on load: the same bits as combine_bwd's dy_perm + unfused backward
    y_any = torch.randn((R, d), device="cuda").to(bf)
    dout = dev(rng.standard_normal((T, d)).astype(np.float32), bf)
    gates = dev(rng.uniform(0.05, 1.0, size=(T, k)).astype(np.float32), torch.float32)
    dy_c, dg_c = laep.moe_combine_bwd(dout, y_any, gates, dest_row)
    _, dg_only = laep.moe_combine_bwd(dout, y_any, gates, dest_row, want_dy=False)
    for use_h in (False, True):
        h = h_f if use_h else None
        a = laep.moe_grouped_ffn_bwd(dy_c, x_perm, act, wgu, wd, offsets, h_fwd=h,
                                     expert_map=emap, dw_gate_up=zeros(wgu), dw_down=zeros(wd))
        case(f"ffn bwd gather, dY on load, use_h={use_h}")
        c2 = laep.moe_grouped_ffn_bwd_gather(None, x, row_src, k, act, wgu, wd, offsets,
                                             dout=dout, topk_gate=gates, h_fwd=h,
                                             expert_map=emap, dw_gate_up=zeros(wgu),
                                             dw_down=zeros(wd))
        torch.cuda.synchronize()
        for n, u, g in zip(("dx_perm", "dw_gate_up", "dw_down"), a, c2):
            assert torch.equal(u, g), f"{n} differs with dY on load (use_h={use_h})"
    assert torch.equal(dg_c, dg_only)
    # weight gradients against the oracle, on the oracle's dispatched rows
    dA_g, _ = laep.ffn_bwd_ws_views(b[3], R, f, bf)
    rc, ro, rdst = om.expert_counts(ids, E)
    xp = om.permute(c["x"], rdst, k)
    rgu, rdd = om.grouped_ffn_wgrad(host(dy), xp, host(dA_g), host(h_f), ro, n_phys,
                                    expert_map=emap_h)
    got_gu, got_d = host(b[1]), host(b[2])
    for p in range(n_phys):
        assert rownorm_err(got_gu[p], rgu[p]) <= TOL_F32, p
        assert rownorm_err(got_d[p], rdd[p]) <= TOL_F32, p


def test_ffn_bwd_concurrent_calls_on_two_streams():
    """Two backward calls issued back to back on two caller streams take
    different library side streams (their weight gradients overlap on the GPU)
    and give the same bits as the same calls made one after the other."""
    rng = np.random.default_rng(41)
    T, k, E, d, f = 700, 4, 8, 256, 128
    c = random_case(77, T=T, d_model=d, E=E, k=k, d_ff=f, dtype="bf16")
    bf = torch.bfloat16
    x, wgu, wd = dev(c["x"], bf), dev(c["w_gate_up"], bf), dev(c["w_down"], bf)
    ids = np.stack([rng.choice(E, size=k, replace=False) for _ in range(T)]).astype(np.int32)
    idx = dev(ids, torch.int32)
    case(f"ffn bwd, two concurrent calls T={T} k={k} E={E} d={d} f={f}")
    counts, offsets, dest_row, row_src = laep.moe_expert_counts(idx, E, want_row_src=True)
    R = T * k
    x_perm = laep.moe_permute(x, dest_row, k)
    _, act = laep.moe_grouped_ffn_fwd(x_perm, wgu, wd, offsets, save_act=True)
    dys = [dev(rng.standard_normal((R, d)).astype(np.float32), bf) for _ in range(2)]
    zeros = lambda t: torch.zeros(t.shape, dtype=torch.float32, device="cuda")

    def call(dy):
        return laep.moe_grouped_ffn_bwd_gather(dy, x, row_src, k, act, wgu, wd, offsets,
                                               dw_gate_up=zeros(wgu), dw_down=zeros(wd))

    ref = [call(dy) for dy in dys]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(2)]
    for rep in range(3):
        outs = [None, None]
        for i, st in enumerate(streams):
            st.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(st):
                outs[i] = call(dys[i])
        for st in streams:
            torch.cuda.current_stream().wait_stream(st)
        torch.cuda.synchronize()
        for i in range(2):
            for n, u, g in zip(("dx_perm", "dw_gate_up", "dw_down"), ref[i], outs[i]):
                assert torch.equal(u, g), f"{n} differs (call {i}, repetition {rep})"


def test_ffn_fwd_concurrent_calls_on_two_streams():
    """Two gathered forward calls on two caller streams, each with its own
    workspace (the persistent products' tile counters live there), overlap on
    the GPU and give the same bits as the same calls made one after the other;
    several hundred tiles per product, so every workgroup takes several."""
    rng = np.random.default_rng(43)
    T, k, E, d, f = 2000, 8, 16, 512, 512
    c = random_case(78, T=T, d_model=d, E=E, k=k, d_ff=f, dtype="bf16")
    bf = torch.bfloat16
    wgu, wd = dev(c["w_gate_up"], bf), dev(c["w_down"], bf)
    xs = [dev(rng.standard_normal((T, d)).astype(np.float32), bf) for _ in range(2)]
    ids = np.stack([rng.choice(E, size=k, replace=False) for _ in range(T)]).astype(np.int32)
    idx = dev(ids, torch.int32)
    case(f"ffn fwd, two concurrent calls T={T} k={k} E={E} d={d} f={f}")
    counts, offsets, dest_row, row_src = laep.moe_expert_counts(idx, E, want_row_src=True)

    def call(x):
        return laep.moe_grouped_ffn_fwd_gather(x, row_src, k, wgu, wd, offsets)[0]

    ref = [call(x) for x in xs]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(2)]
    for rep in range(3):
        outs = [None, None]
        for i, st in enumerate(streams):
            st.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(st):
                outs[i] = call(xs[i])
        for st in streams:
            torch.cuda.current_stream().wait_stream(st)
        torch.cuda.synchronize()
        for i in range(2):
            assert torch.equal(ref[i], outs[i]), f"y_perm differs (call {i}, repetition {rep})"


@pytest.mark.parametrize("T,E,d,f,mapped,keep_y", [
    (300, 8, 256, 128, False, False),   # ragged tiles, an empty expert
    (1, 3, 128, 256, False, True),      # a single token
    (777, 12, 192, 192, True, True),    # expert_map with unused slots, f % 128 = 64
    (2100, 40, 320, 128, False, False),  # many small experts, d % 256 = 64
])
def test_ffn_fwd_gather_combine_matches_three_calls(T, E, d, f, mapped, keep_y):
    """One slot per token: the combine folded into the down projection's
    epilogue is bit-identical to gather + FFN + combine, and matches the
    oracle's permute + FFN + combine."""
    rng = np.random.default_rng(T + 7 * E)
    c = random_case(T + E + 1, T=T, d_model=d, E=E + 2 if mapped else E, k=1, d_ff=f,
                    dtype="bf16")
    w = np.r_[3.0, np.ones(E - 2), 0.0]
    ids = rng.choice(E, size=(T, 1), p=w / w.sum())
    gates = rng.uniform(0.05, 1.0, size=(T, 1)).astype(np.float32)
    bf = torch.bfloat16
    x, wgu, wd = dev(c["x"], bf), dev(c["w_gate_up"], bf), dev(c["w_down"], bf)
    emap = dev(np.array([e + 2 for e in range(E)], np.int32), torch.int32) if mapped else None
    idx = dev(ids.astype(np.int32), torch.int32)
    g = dev(gates, torch.float32)
    case(f"ffn fwd gather+combine T={T} E={E} d={d} f={f} mapped={mapped} keep_y={keep_y}")
    counts, offsets, dest_row, row_src = laep.moe_expert_counts(idx, E, want_row_src=True)
    y1, a1 = laep.moe_grouped_ffn_fwd_gather(x, row_src, 1, wgu, wd, offsets, expert_map=emap,
                                            save_act=True)
    out1 = laep.moe_combine(y1, g, dest_row)
    xp_copy = torch.empty((T, d), dtype=bf, device="cuda") if keep_y else None
    out2, y2, a2 = laep.moe_grouped_ffn_fwd_gather_combine(
        x, row_src, g, wgu, wd, offsets, expert_map=emap, keep_y=keep_y, save_act=True,
        x_perm_out=xp_copy)
    torch.cuda.synchronize()
    assert torch.equal(out1, out2)
    if keep_y:
        assert torch.equal(xp_copy, laep.moe_permute(x, dest_row, 1))
    assert torch.equal(a1, a2)
    if keep_y:
        assert torch.equal(y1, y2)
    else:
        assert y2 is None
    rc, ro, rd = om.expert_counts(ids, E)
    xp = om.permute(c["x"], rd, 1)
    ry, _ = om.grouped_ffn_fwd(xp, c["w_gate_up"], c["w_down"], ro,
                               expert_map=host(emap) if mapped else None, dtype="bf16")
    rout = om.combine(ry, gates, rd, 1)
    assert rownorm_err(host(out2), rout) <= TOL_BF16


@pytest.mark.parametrize("use_h", [False, True])
@pytest.mark.parametrize("counts,d,f", [
    ([60, 0, 200, 5, 1, 130, 64, 52], 128, 256),
    ([300, 129, 128, 0, 7, 1000, 1, 40], 256, 192),
    ([300, 0, 513, 64], 2048, 1024),                              # the balanced layer's width
])
def test_ffn_bwd_parity(counts, d, f, use_h):
    x, wgu, wd, offsets = _ffn_inputs(len(counts) + d, counts, d, f, "bf16")
    R = int(offsets[-1])
    E = len(counts)
    rng = np.random.default_rng(4)
    bf = torch.bfloat16
    xt, wgut, wdt = dev(x, bf), dev(wgu, bf), dev(wd, bf)
    off = dev(offsets.astype(np.int32), torch.int32)
    case(f"ffn bwd counts={counts} d={d} f={f} use_h={use_h}")
    ws_f = torch.empty(laep.workspace_bytes(laep.LAEP_CALL_FFN_FWD, R, 1, E, d, f),
                       dtype=torch.uint8, device="cuda")
    _, act = laep.moe_grouped_ffn_fwd(xt, wgut, wdt, off, ws=ws_f, save_act=True)
    h_f = laep.ffn_fwd_h_view(ws_f, R, f, bf) if use_h else None
    dy = dev(rng.standard_normal((R, d)).astype(np.float32), bf)
    dwgu = torch.full(wgut.shape, 7.0, dtype=torch.float32, device="cuda")
    dwd = torch.full(wdt.shape, 7.0, dtype=torch.float32, device="cuda")
    dx, dwgu, dwd, ws = laep.moe_grouped_ffn_bwd(dy, xt, act, wgut, wdt, off, h_fwd=h_f,
                                                 dw_gate_up=dwgu, dw_down=dwd, return_ws=True)
    torch.cuda.synchronize()
    dA_g, hb_g = laep.ffn_bwd_ws_views(ws, R, f, bf)
    act_h, dy_h, dA_h, hb_h = host(act), host(dy), host(dA_g), host(hb_g)
    # dgrad 1 + SwiGLU backward (teacher-forced on the GPU's act_save)
    rdx, rdA, rhb = om.grouped_ffn_dgrad(dy_h, act_h, wgu, wd, offsets, dtype="bf16",
                                         dA_given=dA_h)
    assert rownorm_err(dA_h, rdA) <= TOL_BF16
    assert rownorm_err(host(dx), rdx) <= TOL_BF16
    if use_h:
        # the forward's H against the oracle's; the H_b buffer keeps dH
        _, _, rh = om.grouped_ffn_fwd(x, wgu, wd, offsets, dtype="bf16", return_h=True)
        h_used = host(h_f)
        assert rownorm_err(h_used, rh) <= TOL_BF16
    else:
        assert rownorm_err(hb_h, rhb) <= TOL_BF16
        h_used = hb_h
    # wgrad (teacher-forced on the GPU's dA and the H it used), fp32
    rgu, rd = om.grouped_ffn_wgrad(dy_h, x, dA_h, h_used, offsets, E)
    got_gu, got_d = host(dwgu), host(dwd)
    for e in range(E):
        assert rownorm_err(got_gu[e], rgu[e]) <= TOL_F32, e
        assert rownorm_err(got_d[e], rd[e]) <= TOL_F32, e
    # accumulate adds onto the existing gradient
    case("ffn bwd accumulate")
    laep.moe_grouped_ffn_bwd(dy, xt, act, wgut, wdt, off, h_fwd=h_f, dw_gate_up=dwgu,
                             dw_down=dwd, accumulate=True)
    torch.cuda.synchronize()
    assert rownorm_err(host(dwd).reshape(E, -1), (2 * rd).reshape(E, -1)) <= TOL_F32


@pytest.mark.parametrize("seed", range(24))
def test_ffn_bwd_fuzz(seed):
    """Random ragged expert loads (empty experts, single rows, one heavy
    expert) through the backward products, teacher-forced like the parity
    test above: dA, H_b and dX against the oracle at the GPU's act_save, the
    fp32 weight gradients at the GPU's dA and H_b."""
    rng = np.random.default_rng(700 + seed)
    E = int(rng.integers(1, 13))
    counts = [int(v) for v in rng.choice([0, 1, 3, 64, 255, 256, 257, 600], size=E)]
    if sum(counts) == 0:
        counts[0] = 5
    d = int(rng.choice([64, 128, 192, 320]))
    f = int(rng.choice([64, 128, 192, 256]))
    x, wgu, wd, offsets = _ffn_inputs(800 + seed, counts, d, f, "bf16")
    R = int(offsets[-1])
    bf = torch.bfloat16
    xt, wgut, wdt = dev(x, bf), dev(wgu, bf), dev(wd, bf)
    off = dev(offsets.astype(np.int32), torch.int32)
    use_h = seed % 2 == 1   # odd seeds: dW_d from the forward's H
    case(f"ffn bwd fuzz seed={seed} counts={counts} d={d} f={f} use_h={use_h}")
    ws_f = torch.empty(laep.workspace_bytes(laep.LAEP_CALL_FFN_FWD, R, 1, E, d, f),
                       dtype=torch.uint8, device="cuda")
    _, act = laep.moe_grouped_ffn_fwd(xt, wgut, wdt, off, ws=ws_f, save_act=True)
    h_f = laep.ffn_fwd_h_view(ws_f, R, f, bf) if use_h else None
    dy = dev(rng.standard_normal((R, d)).astype(np.float32), bf)
    dx, dwgu, dwd, ws = laep.moe_grouped_ffn_bwd(dy, xt, act, wgut, wdt, off, h_fwd=h_f,
                                                 return_ws=True)
    torch.cuda.synchronize()
    dA_g, hb_g = laep.ffn_bwd_ws_views(ws, R, f, bf)
    act_h, dy_h, dA_h, hb_h = host(act), host(dy), host(dA_g), host(hb_g)
    rdx, rdA, rhb = om.grouped_ffn_dgrad(dy_h, act_h, wgu, wd, offsets, dtype="bf16",
                                         dA_given=dA_h)
    assert rownorm_err(dA_h, rdA) <= TOL_BF16
    assert rownorm_err(host(dx), rdx) <= TOL_BF16
    if use_h:
        _, _, rh = om.grouped_ffn_fwd(x, wgu, wd, offsets, dtype="bf16", return_h=True)
        h_used = host(h_f)
        assert rownorm_err(h_used, rh) <= TOL_BF16
    else:
        assert rownorm_err(hb_h, rhb) <= TOL_BF16
        h_used = hb_h
    rgu, rd = om.grouped_ffn_wgrad(dy_h, x, dA_h, h_used, offsets, E)
    got_gu, got_d = host(dwgu), host(dwd)
    for e in range(E):
        assert rownorm_err(got_gu[e], rgu[e]) <= TOL_F32, e
        assert rownorm_err(got_d[e], rd[e]) <= TOL_F32, e


# ---------------------------------------------------------------------------
# the whole layer, end to end, tiny fp32 workload
# ---------------------------------------------------------------------------
def _heavy_tailed_counts(rng, E, total):
    """Per-expert row counts with a heavy tail (Pareto 1.1 weights) and about
    15 % empty experts, summing to about `total`."""
    w = rng.pareto(1.1, size=E) + 0.05
    w[rng.random(E) < 0.15] = 0.0
    if w.sum() == 0:
        w[0] = 1.0
    c = [int(v) for v in np.floor(w / w.sum() * total)]
    if sum(c) == 0:
        c[0] = 300
    return c


@pytest.mark.parametrize("seed,E,total,d,f", [
    (0, 64, 80000, 128, 64),    # about 380 row tiles: several tiles per persistent workgroup
    (1, 40, 60000, 64, 256),
    (2, 16, 40000, 256, 128),
])
def test_ffn_fwd_many_tiles(seed, E, total, d, f):
    """Uneven expert loads over hundreds of tiles per product, so every
    persistent workgroup takes several tiles from its XCD's queue."""
    counts = _heavy_tailed_counts(np.random.default_rng(40 + seed), E, total)
    test_ffn_fwd_parity("bf16", counts, d, f)


@pytest.mark.parametrize("seed,use_h", [(0, False), (1, True)])
def test_ffn_bwd_many_tiles(seed, use_h):
    """The backward products over uneven expert loads of about 20k rows."""
    counts = _heavy_tailed_counts(np.random.default_rng(60 + seed), 24, 20000)
    test_ffn_bwd_parity(counts, 128, 128, use_h)


def test_tiny_layer_end_to_end():
    w = WORKLOADS["tiny"]
    c = generate(w)
    td = torch.float32
    case("tiny layer end to end (fp32)")
    plan = laep.MoELayerPlan(w.T, w.d_model, w.E, w.k, w.d_ff, dtype=td, device="cuda")
    out = plan.forward(dev(c["x"], td), dev(c["w_router"], td), dev(c["w_gate_up"], td),
                       dev(c["w_down"], td), renorm=w.renorm)
    torch.cuda.synchronize()
    ref = om.layer_forward(c["x"], c["w_router"], c["w_gate_up"], c["w_down"], w.k,
                           renorm=w.renorm, dtype="f32")
    check_routing(host(plan.topk_idx), host(plan.topk_gate), ref["idx"], ref["gate"],
                  ref["logits"], w.k, renorm=w.renorm)
    ok = np.all(host(plan.topk_idx) == ref["idx"], axis=1)
    assert rownorm_err(host(out)[ok], ref["out"][ok]) <= TOL_F32


@pytest.mark.parametrize("seed", range(48))
def test_layer_fuzz(seed):
    """Random shapes through the whole forward (route + counts, dispatch, FFN,
    combine): routing against the oracle (near-ties allowed), outputs
    teacher-forced on the GPU's routing.  Every fourth case keeps exactly k
    experts alive, every fourth (offset 2) lets one expert take every token."""
    rng = np.random.default_rng(900 + seed)
    E = int(rng.integers(1, 65))
    k = int(rng.integers(1, min(E, 8) + 1))
    T = int(rng.integers(1, 700))
    d = int(rng.choice([64, 128, 192, 256]))
    f = int(rng.choice([64, 128, 192]))
    dtype = "f32" if seed % 3 == 0 else "bf16"
    renorm = bool(seed % 2)
    td = TD[dtype]
    c = random_case(5000 + seed, T=T, d_model=d, E=E, k=k, d_ff=f, dtype=dtype,
                    bias_std=float(rng.choice([0.0, 1.0, 3.0])), weight_std=0.05)
    bias = c["bias"].copy() if "bias" in c else np.zeros(E, np.float32)
    alive = None
    if seed % 4 == 1 and E > k:        # every expert pruned except k
        alive = np.zeros(E, bool)
        alive[rng.choice(E, k, replace=False)] = True
    if seed % 4 == 2:                  # one expert takes every token
        bias[int(rng.integers(E))] += 100.0
    case(f"layer fuzz seed={seed} T={T} d={d} E={E} k={k} f={f} {dtype} renorm={renorm}")
    x = dev(c["x"], td)
    idx, gate, counts, offsets, dest, row_src, logits = laep.moe_route_count(
        x, dev(c["w_router"], td), k, bias=dev(bias, torch.float32),
        alive=None if alive is None else dev(alive.astype(np.uint8), torch.uint8),
        renorm=renorm, want_logits=True, want_row_src=True)
    wgu, wd = dev(c["w_gate_up"], td), dev(c["w_down"], td)
    xp = laep.moe_permute(x, dest, k)
    y, _ = laep.moe_grouped_ffn_fwd(xp, wgu, wd, offsets, save_act=False)
    out = laep.moe_combine(y, gate, dest)
    if dtype == "bf16":   # the dispatch folded into the operand loads gives the same bits
        yg, _ = laep.moe_grouped_ffn_fwd_gather(x, row_src, k, wgu, wd, offsets, rows=T * k)
    if dtype == "bf16" and k == 1:   # and so does the combine folded into the epilogue
        og, _, _ = laep.moe_grouped_ffn_fwd_gather_combine(
            x, row_src, gate, wgu, wd, offsets, rows=T, out=torch.zeros_like(out))
    torch.cuda.synchronize()
    ridx, rgate, _, rlog = om.route(c["x"], c["w_router"], k, bias=bias, alive=alive,
                                   renorm=renorm)
    check_routing(host(idx), host(gate), ridx, rgate, rlog, k, alive, renorm=renorm)
    gi, gg = host(idx), host(gate)
    rc, ro, rd = om.expert_counts(gi, E)
    np.testing.assert_array_equal(host(counts), rc)
    np.testing.assert_array_equal(host(dest), rd)
    ry, _ = om.grouped_ffn_fwd(om.permute(c["x"], rd, k), c["w_gate_up"], c["w_down"], ro,
                               dtype=dtype)
    rout = om.combine(ry, gg, rd, k, dtype=dtype)
    tol = TOL_BF16 if dtype == "bf16" else TOL_F32
    assert rownorm_err(host(y), ry) <= tol
    assert rownorm_err(host(out), rout) <= tol
    if dtype == "bf16":
        assert torch.equal(yg, y)
    if dtype == "bf16" and k == 1:
        assert torch.equal(og, out)


def test_determinism():
    w = WORKLOADS["balanced"]
    c = random_case(11, T=1500, d_model=512, E=64, k=8, d_ff=256, dtype="bf16")
    bf = torch.bfloat16
    args = (dev(c["x"], bf), dev(c["w_router"], bf), dev(c["w_gate_up"], bf),
            dev(c["w_down"], bf))
    case("determinism")
    p1 = laep.MoELayerPlan(1500, 512, 64, 8, 256, dtype=bf, device="cuda", save_act=True)
    p2 = laep.MoELayerPlan(1500, 512, 64, 8, 256, dtype=bf, device="cuda", save_act=True)
    o1 = p1.forward(*args).clone()
    o2 = p2.forward(*args)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)
    assert torch.equal(p1.act_save, p2.act_save)


# ---------------------------------------------------------------------------
# router / gate backward (teacher-forced on the GPU's routing)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("T,d,E,k,dtype,renorm,bias,dead", [
    (500, 256, 16, 4, "bf16", True, 0.0, 0),       # renormalised gates
    (256, 128, 8, 2, "f32", False, 0.0, 0),        # tiny layer: full-softmax gates
    (333, 192, 12, 5, "bf16", True, 1.0, 8),       # 4 alive of 12, k = 5: unroutable slots
    (300, 128, 10, 3, "bf16", False, 0.5, 3),      # full softmax with dead experts
])
def test_route_bwd_parity(T, d, E, k, dtype, renorm, bias, dead):
    c = random_case(T + 17 * E, T=T, d_model=d, E=E, k=k, d_ff=64, dtype=dtype, bias_std=bias)
    td = TD[dtype]
    rng = np.random.default_rng(T)
    alive_np = np.ones(E, bool)
    alive_np[rng.choice(E, dead, replace=False)] = False
    alive = dev(alive_np.astype(np.uint8), torch.uint8) if dead else None
    x, wr = dev(c["x"], td), dev(c["w_router"], td)
    b = dev(c["bias"], torch.float32) if "bias" in c else None
    case(f"route bwd T={T} d={d} E={E} k={k} {dtype} renorm={renorm} dead={dead}")
    idx, gate, logits = laep.moe_route(x, wr, k, bias=b, alive=alive, renorm=renorm,
                                       want_logits=True)
    counts, offsets, dest_row, row_src = laep.moe_expert_counts(idx, E, want_row_src=True)
    dg = dev(rng.standard_normal((T, k)).astype(np.float32), torch.float32)
    dx_in = rng.standard_normal((T, d)).astype(np.float32)
    dx = dev(dx_in, td)
    dx_in = host(dx)   # the rounded values the GPU accumulates onto
    dx, dw, db, dl = laep.moe_route_bwd(dg, idx, gate, x, wr, renorm=renorm, logits=logits,
                                        alive=alive, offsets=offsets, row_src=row_src, dx=dx,
                                        accumulate_dx=True, want_dlogits=True, want_dbias=True)
    torch.cuda.synchronize()
    rl, rw, rb, rx = om.route_bwd(host(dg), host(idx), host(gate), c["x"], c["w_router"],
                                  logits=host(logits), alive=alive_np if dead else None,
                                  renorm=renorm, dtype=dtype, dx_in=dx_in)
    assert rownorm_err(host(dl), rl) <= TOL_F32
    assert rownorm_err(host(dw), rw) <= TOL_F32
    assert rownorm_err(host(db), rb) <= TOL_F32
    assert rownorm_err(host(dx), rx) <= (TOL_BF16 if dtype == "bf16" else TOL_F32)
    # the two halves alone (dx only, weights only) give the same bits
    dx2 = dev(dx_in, td)
    d2, w2, b2, l2 = laep.moe_route_bwd(dg, idx, gate, x, wr, renorm=renorm, logits=logits,
                                        alive=alive, offsets=offsets, row_src=row_src, dx=dx2,
                                        accumulate_dx=True, want_dlogits=True, weights=False)
    d3, w3, b3, _ = laep.moe_route_bwd(dg, idx, gate, x, wr, renorm=renorm, logits=logits,
                                       alive=alive, offsets=offsets, row_src=row_src,
                                       data=False, want_dbias=True)
    torch.cuda.synchronize()
    assert w2 is None and b2 is None and d3 is None
    assert torch.equal(d2, dx) and torch.equal(l2, dl)
    assert torch.equal(w3, dw) and torch.equal(b3, db)


def test_zero_rows_everywhere():
    """No routed rows at all: every call is a no-op on its row outputs, and the
    weight gradients come out as the empty sums they are (zero, or unchanged
    when accumulating)."""
    E, d, f, k = 4, 128, 256, 2
    bf = torch.bfloat16
    rng = np.random.default_rng(7)
    wgu = dev((rng.standard_normal((E, 2 * f, d)) * 0.02).astype(np.float32), bf)
    wd = dev((rng.standard_normal((E, d, f)) * 0.02).astype(np.float32), bf)
    wr = dev((rng.standard_normal((E, d)) * 0.02).astype(np.float32), bf)
    offsets = torch.zeros(E + 1, dtype=torch.int32, device="cuda")
    x0 = torch.empty((0, d), dtype=bf, device="cuda")
    case("zero rows: grouped FFN forward / backward")
    y, act = laep.moe_grouped_ffn_fwd(x0, wgu, wd, offsets)
    assert y.shape == (0, d) and act.shape == (0, 2 * f)
    dwgu = torch.full((E, 2 * f, d), 7.0, device="cuda")
    dwd = torch.full((E, d, f), 7.0, device="cuda")
    laep.moe_grouped_ffn_bwd(x0, x0, act, wgu, wd, offsets, dw_gate_up=dwgu, dw_down=dwd)
    torch.cuda.synchronize()
    assert not dwgu.any() and not dwd.any()
    dwgu.fill_(7.0), dwd.fill_(7.0)
    laep.moe_grouped_ffn_bwd(x0, x0, act, wgu, wd, offsets, dw_gate_up=dwgu, dw_down=dwd,
                             accumulate=True)
    torch.cuda.synchronize()
    assert bool((dwgu == 7.0).all()) and bool((dwd == 7.0).all())
    case("zero tokens: row ops and router backward")
    idx0 = torch.empty((0, k), dtype=torch.int32, device="cuda")
    g0 = torch.empty((0, k), dtype=torch.float32, device="cuda")
    r0 = torch.empty(0, dtype=torch.int32, device="cuda")
    assert laep.moe_permute(x0, r0, k, 0).shape == (0, d)
    assert laep.moe_combine(x0, g0, r0).shape == (0, d)
    dy, dg = laep.moe_combine_bwd(x0, x0, g0, r0)
    assert dy.shape == (0, d) and dg.shape == (0, k)
    assert laep.moe_permute_bwd(x0, r0, 0, k).shape == (0, d)
    dw = torch.full((E, d), 7.0, device="cuda")
    db = torch.full((E,), 7.0, device="cuda")
    dx, dw, db, _ = laep.moe_route_bwd(g0, idx0, g0, x0, wr, offsets=offsets, row_src=r0,
                                       dw_router=dw, want_dbias=True, dbias=db)
    torch.cuda.synchronize()
    assert dx.shape == (0, d) and not dw.any() and not db.any()
    # weights only / data only: nothing else is touched
    dw.fill_(7.0)
    _, w_none, _, _ = laep.moe_route_bwd(g0, idx0, g0, x0, wr, offsets=offsets, row_src=r0,
                                         weights=False)
    assert w_none is None
    torch.cuda.synchronize()
    assert bool((dw == 7.0).all())


def test_calib_kernels():
    """The measurement kernels do the work they are timed on: the copy copies,
    the blocked read XORs each thread's 16-byte chunks, the MFMA loop writes
    one value per lane."""
    rng = np.random.default_rng(5)
    case("calibration kernels")
    src = torch.from_numpy(rng.integers(0, 2**31, size=3 * 65536 // 4, dtype=np.int64)
                           .astype(np.uint32).view(np.int32)).cuda()
    dst = torch.empty_like(src)
    laep.laep_calib_copy(src, dst)
    block = 65536                      # 8 chunks of 16 bytes per thread
    out = torch.empty(src.numel() * 4 // block * 512, dtype=torch.float32, device="cuda")
    laep.laep_calib_read(src, block, out)
    mout = torch.empty(8 * 512, dtype=torch.float32, device="cuda")
    laep.laep_calib_mfma(8, 4, mout)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
    words = src.cpu().numpy().view(np.uint32).reshape(-1, block // 16 // 512, 512, 4)  # [wg, u, t, 4]
    want = np.bitwise_xor.reduce(np.bitwise_xor.reduce(words, axis=3), axis=1).reshape(-1)
    assert np.array_equal(out.cpu().numpy().view(np.uint32), want)
    assert torch.isfinite(mout).all()
