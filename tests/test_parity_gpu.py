"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle on seeded inputs.

Tolerances (stated by the method's accuracy target, fp32 arithmetic):
  * every CPPN output: |gpu - oracle| <= 1e-5 * max(|oracle|, 1)  (relative where |o| >= 1,
    absolute below, since relative error is undefined at the zeros of sine/linear outputs);
  * kept cells: identical sets, except cells whose oracle variance lies within 1e-5 of theta
    (theta is the float32 value the kernel compares against);
  * heap indices, counts and record order: exact.
"""

import math

import numpy as np
import pytest

import oracle
from paper_2608_27612_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = 1e-5
BAND = 1e-5


@pytest.fixture(scope="module")
def emr():
    import torch
    assert torch.cuda.is_available()
    from paper_2608_27612_amd import emr as E
    E.lib()
    return E


def close(g, o):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    return np.abs(g - o) <= TOL * np.maximum(np.abs(o), 1.0)


def pair_genome_source(r, genomes, sources, offs):
    if offs is None:
        return genomes[r // len(sources)], sources[r % len(sources)]
    g = int(np.searchsorted(np.asarray(offs), r, side="right") - 1)
    return genomes[g], sources[r]


def check_discover(emr, genomes, sources, D, theta, offs=None, capacity=None, pop=None, calls=1):
    """Runs the GPU path and the oracle; asserts parity; returns summary stats. With calls > 1 the
    same plan runs that many times (a compiled plan's later calls take their chunks from balanced
    lists): every call's result must equal the first bit for bit, and the last is checked."""
    theta32 = float(np.float32(theta))
    if pop is None:
        pop = emr.emr_pack_population(genomes)
    first = None
    for _ in range(calls):
        res = emr.emr_discover(pop, sources, D, theta32, src_offsets=offs, capacity=capacity)
        total, mx = emr.emr_result_check(res)
        counts, recs = emr.records_to_host(res)
        if first is None:
            first = (total, mx, counts, recs)
            continue
        assert (total, mx) == first[:2] and np.array_equal(counts, first[2])
        for (ga, wa), (gb, wb) in zip(recs, first[3]):
            np.testing.assert_array_equal(ga, gb)
            np.testing.assert_array_equal(wa.view(np.uint32), wb.view(np.uint32))
    offsets = res["pair_offset"].cpu().numpy()
    assert offsets[0] == 0 and np.array_equal(np.diff(offsets), counts) and offsets[-1] == total
    o = oracle.discover(genomes, sources, D, theta32, src_offsets=offs)
    assert len(counts) == len(o["pair_count"])
    n_band = 0
    for r in range(len(counts)):
        lo, hi = o["pair_offset"][r], o["pair_offset"][r + 1]
        op, ow, ov = o["parent"][lo:hi], o["w4"][lo:hi], o["var"][lo:hi]
        gp, gw = recs[r]
        assert np.all(np.diff(gp) > 0), "records not in ascending parent order"
        if counts[r] == len(op) and np.array_equal(gp, op):
            ok = close(gw, ow)
            assert ok.all(), (r, np.argwhere(~ok)[:5], gw[~ok.any(axis=1)][:3], ow[~ok.any(axis=1)][:3])
            continue
        # sets differ: every difference must sit in the band around theta
        g, s = pair_genome_source(r, genomes, sources, offs)
        diff = np.setxor1d(gp, op)
        _, dvar = oracle.eval_parents(g, s, diff)
        assert np.all(np.abs(dvar - theta32) <= BAND), (r, diff[:5], dvar[:5])
        n_band += len(diff)
        common, gi, oi = np.intersect1d(gp, op, return_indices=True)
        assert close(gw[gi], ow[oi]).all()
    assert mx == (int(counts.max()) if len(counts) else 0)
    return {"records": int(total), "band": n_band, "counts": counts}


def check_raw(emr, genomes, sources, D, offs=None):
    pop = emr.emr_pack_population(genomes)
    raw = emr.emr_eval_raw(pop, sources, D, src_offsets=offs).cpu().numpy()
    Q = oracle.n_parents(D)
    parents = np.arange(Q, dtype=np.int64)
    worst = 0.0
    for r in range(raw.shape[0]):
        g, s = pair_genome_source(r, genomes, sources, offs)
        w4, _ = oracle.eval_parents(g, s, parents)
        want = w4.reshape(-1)
        ok = close(raw[r], want)
        assert ok.all(), (r, np.argwhere(~ok)[:5].ravel(), raw[r][~ok][:5], want[~ok][:5])
        worst = max(worst, float(np.max(np.abs(raw[r] - want) / np.maximum(np.abs(want), 1.0))))
    return worst


# ------------------------------------------------------------------------------- grids

def test_grid_positions_exact(emr):
    for D in [0, 1, 2, 3, 4, 5, 8]:
        xy = emr.emr_build_grids(D).cpu().numpy().astype(np.float64)
        np.testing.assert_array_equal(xy, oracle.grid(D))


# ------------------------------------------------------------------------------- raw outputs

def test_raw_single_cppn_depth5(emr):
    genomes, sources, D, _ = W.workload("single_d5")
    check_raw(emr, genomes, sources, D)


def test_raw_population_both_directions(emr):
    genomes = W.population(1, 40, 20, 60)
    check_raw(emr, genomes, W.xor_sources(), 5)


@pytest.mark.parametrize("act", range(6))
def test_raw_each_activation(emr, act):
    # out = linear(act(3*x2 - 2*y2 + 0.5) * 2 + x2): exercises each activation over z in [-5.5, 5.5]
    g = {"kind": np.array([0, 1, 2, 3, 4, 6, 5], np.uint8),
         "act": np.array([0, 0, 0, 0, 0, 0, act], np.uint8), "bias": np.zeros(7, np.float32),
         "src": np.array([2, 3, 4, 6, 2], np.int32), "dst": np.array([6, 6, 6, 5, 5], np.int32),
         "w": np.array([3.0, -2.0, 0.5, 2.0, 1.0], np.float32), "enabled": np.ones(5, np.uint8)}
    check_raw(emr, [g], W.xor_sources(), 6)


def test_raw_large_sine_arguments(emr):
    # a linear chain multiplies x2 by 3^4 = 81 before a sine: |z| up to ~80
    kinds = [0, 1, 2, 3, 4, 6, 5, 5, 5, 5, 5]
    acts = [0] * 5 + [0, 0, 0, 0, 0, 4]
    edges = [(2, 6, 3.0), (6, 7, 3.0), (7, 8, 3.0), (8, 9, 3.0), (9, 10, 1.0), (10, 5, 1.0)]
    g = {"kind": np.array(kinds, np.uint8), "act": np.array(acts, np.uint8),
         "bias": np.zeros(len(kinds), np.float32),
         "src": np.array([e[0] for e in edges], np.int32),
         "dst": np.array([e[1] for e in edges], np.int32),
         "w": np.array([e[2] for e in edges], np.float32), "enabled": np.ones(len(edges), np.uint8)}
    check_raw(emr, [g], W.xor_sources(), 6)


# ------------------------------------------------------------------------------- discovery

@pytest.mark.parametrize("theta", [0.03, 1e-3, 1e-4])
def test_discover_single_cppn_depth5(emr, theta):
    # this seeded CPPN is smooth: nothing passes 0.03 (the oracle agrees), 160 cells pass 1e-4
    genomes, sources, D, _ = W.workload("single_d5")
    st = check_discover(emr, genomes, sources, D, theta)
    assert (st["records"] > 0) == (theta < 0.01)


@pytest.mark.parametrize("D", [5, 6])
def test_discover_xor_population(emr, D):
    genomes = W.population(0, 120 if D == 5 else 40, 20, 60)
    st = check_discover(emr, genomes, W.xor_sources(), D, 0.03)
    assert st["records"] > 0


def test_discover_tabular_population(emr):
    genomes = W.population(2, 12, 40, 120)
    check_discover(emr, genomes, W.tabular_sources(32), 5, 0.03)


def test_discover_per_genome_sources(emr):
    # per-genome (CSR) source lists of varying length, as the hidden->hidden phase uses
    rng = np.random.default_rng(5)
    genomes = W.population(3, 9, 12, 40)
    pts, offs = [], [0]
    for k in range(len(genomes)):
        n = int(rng.integers(0, 7))
        for _ in range(n):
            pts.append((float(rng.uniform(-1, 1)), float(rng.uniform(-1, 1)), int(rng.integers(0, 2))))
        offs.append(len(pts))
    sources = W.sources_array(pts)
    check_discover(emr, genomes, sources, 5, 0.02, offs=offs)


@pytest.mark.parametrize("D", [0, 1, 2, 3, 4])
def test_discover_small_depths(emr, D):
    genomes = W.population(4, 10, 10, 30)
    check_discover(emr, genomes, W.xor_sources(), D, 0.01)


def test_theta_extremes(emr):
    genomes = W.population(6, 6, 10, 30)
    srcs = W.xor_sources()
    st = check_discover(emr, genomes, srcs, 4, -1.0)
    assert st["records"] == len(genomes) * len(srcs) * oracle.n_parents(4)
    st = check_discover(emr, genomes, srcs, 4, math.inf)
    assert st["records"] == 0


def test_constant_cppn_keeps_nothing(emr):
    g = {"kind": np.array([0, 1, 2, 3, 4, 6], np.uint8), "act": np.array([0] * 5 + [1], np.uint8),
         "bias": np.zeros(6, np.float32), "src": np.array([0, 4], np.int32),
         "dst": np.array([5, 5], np.int32), "w": np.array([1.0, 0.5], np.float32),
         "enabled": np.ones(2, np.uint8)}
    srcs = W.sources_array([(0.3, -1.0, 0), (0.1, 0.2, 0)])
    st = check_discover(emr, [g], srcs, 5, 0.0)
    assert st["records"] == 0


def test_infinite_weights_give_nan_variance_never_kept(emr):
    g = {"kind": np.array([0, 1, 2, 3, 4, 6], np.uint8), "act": np.zeros(6, np.uint8),
         "bias": np.zeros(6, np.float32), "src": np.array([2], np.int32),
         "dst": np.array([5], np.int32), "w": np.array([np.inf], np.float32),
         "enabled": np.ones(1, np.uint8)}
    st = check_discover(emr, [g], W.xor_sources()[:1], 4, -1.0)
    assert st["records"] == 0


def test_empty_population_and_no_sources(emr):
    pop = emr.emr_pack_population(W.population(0, 3, 5, 10))
    res = emr.emr_discover(pop, W.xor_sources()[:0], 5, 0.03)
    assert emr.emr_result_check(res) == (0, 0)
    assert int(res["pair_offset"][0].item()) == 0
    pop0 = emr.emr_pack_population([])
    res = emr.emr_discover(pop0, W.xor_sources(), 5, 0.03)
    assert emr.emr_result_check(res) == (0, 0)


def test_one_population_many_calls(emr):
    """A population serves calls with different sources, source layouts and depths in any
    order; each call must be planned for its own arguments."""
    genomes = W.population(21, 24, 20, 60)
    pop = emr.emr_pack_population(genomes)
    xs, ts = W.xor_sources(), W.tabular_sources(8)
    offs = np.array([0] + list(np.cumsum([2 + g % 3 for g in range(len(genomes))])), np.int32)
    csr = np.concatenate([ts[-(2 + g % 3):] if g % 2 else ts[: 2 + g % 3]
                          for g in range(len(genomes))])
    for D, srcs, o in [(5, xs, None), (4, xs, None), (5, ts, None), (5, xs, None),
                       (4, csr, offs), (5, csr, offs), (5, xs, None)]:
        check_discover(emr, genomes, srcs, D, 0.03, offs=o, pop=pop)


def test_capacity_overflow_is_reported(emr):
    """A capacity below the call's total: EMR_E_CAPACITY with the exact total; counts and offsets
    are exact (the records are not: the pool is filled in the order walks finish); a retry at the
    reported total gives the complete output."""
    genomes = W.population(12, 80, 20, 60)
    srcs = W.xor_sources()
    pop = emr.emr_pack_population(genomes)
    full = emr.emr_discover(pop, srcs, 6, 0.01)
    total, mx = emr.emr_result_check(full)
    assert total > 100 and mx < oracle.n_parents(6)
    small = emr.emr_discover(pop, srcs, 6, 0.01, capacity=total // 3)
    with pytest.raises(emr.EmrError) as e:
        emr.emr_result_check(small)
    assert e.value.status == emr.EMR_E_CAPACITY
    assert str(total) in str(e.value)
    np.testing.assert_array_equal(small["pair_count"].cpu().numpy(), full["pair_count"].cpu().numpy())
    np.testing.assert_array_equal(small["pair_offset"].cpu().numpy(), full["pair_offset"].cpu().numpy())
    retry = emr.emr_discover_all(pop, srcs, 6, 0.01, capacity=total // 3)
    assert retry["capacity"] == total
    np.testing.assert_array_equal(retry["parent"].cpu().numpy(), full["parent"][:total].cpu().numpy())
    st = check_discover(emr, genomes, srcs, 6, 0.01, capacity=total, pop=pop)
    assert st["records"] == total


def test_zero_capacity_and_exact_capacity(emr):
    genomes, sources, D, _ = W.workload("single_d5")
    pop = emr.emr_pack_population(genomes)
    res = emr.emr_discover(pop, sources, D, 1e-4, capacity=0)
    with pytest.raises(emr.EmrError) as e:
        emr.emr_result_check(res)
    assert e.value.status == emr.EMR_E_CAPACITY
    total = int(res["pair_offset"][-1].item())
    assert total > 0
    check_discover(emr, genomes, sources, D, 1e-4, capacity=total, pop=pop)


def test_result_checks_wait_for_their_own_call(emr):
    """Each call's flags live in a slot of their own: three calls on three results enqueued back
    to back are checked afterwards, each against its own total (one overflows, the others do
    not), and a workspace with no call to check is refused."""
    genomes, sources, D, _ = W.workload("single_d5")
    Q = oracle.n_parents(D)
    pop = emr.emr_pack_population(genomes)
    res_all = emr.emr_discover(pop, sources, D, -1.0)               # every cell kept
    res_few = emr.emr_discover(pop, sources, D, -1.0, capacity=10)
    res_none = emr.emr_discover(pop, sources, D, 1e30)             # nothing kept
    assert emr.emr_result_check(res_all) == (Q, Q)
    with pytest.raises(emr.EmrError) as e:
        emr.emr_result_check(res_few)
    assert e.value.status == emr.EMR_E_CAPACITY
    assert emr.emr_result_check(res_none) == (0, 0)
    # checked again later (no call in between on these results): the same answers
    assert emr.emr_result_check(res_all) == (Q, Q)
    import torch
    other = dict(res_all)
    other.pop("_struct", None)
    other["workspace"] = torch.empty_like(res_all["workspace"])
    with pytest.raises(emr.EmrError) as e:
        emr.emr_result_check(other)
    assert e.value.status == emr.EMR_E_INVAL


def test_many_pairs_csr_offsets(emr):
    """Per-genome CSR sources with many empty and many busy pairs: the compaction's scan over the
    pairs' totals gives exact offsets (every pair's records where its offset says) for 6000+
    pairs."""
    rng = np.random.default_rng(71)
    genomes = W.population(71, 300, 12, 40)
    pts, offs = [], [0]
    for k in range(len(genomes)):
        n = int(rng.integers(0, 40))
        for _ in range(n):
            pts.append((float(rng.uniform(-1, 1)), float(rng.uniform(-1, 1)), int(rng.integers(0, 2))))
        offs.append(len(pts))
    sources = W.sources_array(pts)
    st = check_discover(emr, genomes, sources, 4, 0.01, offs=offs)
    assert st["records"] > 0 and len(st["counts"]) > 5000


def test_discover_is_deterministic(emr):
    genomes = W.population(8, 60, 20, 60)
    pop = emr.emr_pack_population(genomes)
    a = emr.emr_discover(pop, W.xor_sources(), 6, 0.03)
    emr.emr_result_check(a)
    b = emr.emr_discover(pop, W.xor_sources(), 6, 0.03)
    emr.emr_result_check(b)
    ca, ra = emr.records_to_host(a)
    cb, rb = emr.records_to_host(b)
    np.testing.assert_array_equal(ca, cb)
    for (pa, wa), (pb, wb) in zip(ra, rb):
        np.testing.assert_array_equal(pa, pb)
        np.testing.assert_array_equal(wa.view(np.uint32), wb.view(np.uint32))


def test_direction_duality_bit_exact(emr):
    genomes = W.population(9, 10, 12, 40)
    swapped = []
    for g in genomes:
        h = dict(g)
        k = g["kind"].copy()
        k[0], k[1], k[2], k[3] = 2, 3, 0, 1
        h["kind"] = k
        swapped.append(h)
    pa = emr.emr_pack_population(genomes)
    pb = emr.emr_pack_population(swapped)
    ra = emr.emr_eval_raw(pa, W.sources_array([(0.25, -0.5, 0)]), 5).cpu().numpy()
    rb = emr.emr_eval_raw(pb, W.sources_array([(0.25, -0.5, 1)]), 5).cpu().numpy()
    np.testing.assert_array_equal(ra.view(np.uint32), rb.view(np.uint32))


# ------------------------------------------------------------------------------- full size

@pytest.mark.parametrize("policy", ["always", "off"])
def test_full_size_xor_pop1000_depth7_all_pairs(emr, policy):
    """The benchmark's workload and launch: 1000 genomes x 4 sources at depth 7 in one call, under
    the compiled tier (what the timed steps run) and under the interpreter, every pair and every
    record against the oracle."""
    emr.emr_set_jit(emr.EMR_JIT_ALWAYS if policy == "always" else emr.EMR_JIT_OFF)
    emr.emr_profile_enable(True)
    try:
        genomes, sources, D, theta = W.workload("xor_pop1000_d7")
        pop = emr.emr_pack_population(genomes)
        st = check_discover(emr, genomes, sources, D, theta, pop=pop, calls=2)
        assert st["records"] > 0
        assert emr.emr_jit_info(pop)["state"] == (1 if policy == "always" else 0)
        launches = emr.emr_profile_read()
        assert [r["listed"] for r in launches] == ([False, True] if policy == "always" else
                                                    [False, False])
    finally:
        emr.emr_profile_enable(False)
        emr.emr_set_jit(emr.EMR_JIT_AUTO)


def test_full_size_depth8_compiled(emr):
    """Depth 8 (87,380 positions per source, the paper's depth-7 grid) under the compiled tier:
    200 genomes of the XOR population recipe x 4 sources, every pair against the oracle."""
    emr.emr_set_jit(emr.EMR_JIT_ALWAYS)
    try:
        genomes = W.population(0, 200, 20, 60)
        pop = emr.emr_pack_population(genomes)
        st = check_discover(emr, genomes, W.xor_sources(), 8, 0.03, pop=pop, calls=2)
        assert st["records"] > 0
        assert emr.emr_jit_info(pop)["state"] == 1
    finally:
        emr.emr_set_jit(emr.EMR_JIT_AUTO)


def test_raw_population_with_biases(emr):
    """Nonzero node biases (hidden and output nodes): raw outputs against the oracle."""
    genomes = W.population(51, 60, 20, 60, biases=True)
    check_raw(emr, genomes, W.xor_sources(), 5)


def test_discover_population_with_biases(emr):
    genomes = W.population(52, 150, 20, 60, biases=True)
    st = check_discover(emr, genomes, W.xor_sources(), 6, 0.03)
    assert st["records"] > 0


@pytest.mark.parametrize("D", [5, 6])
def test_config2_xor_pop1000_full(emr, D):
    """The XOR population workload (1000 genomes x 4 sources) at depths 5 and 6, every pair."""
    genomes, sources, _, theta = W.workload("xor_pop1000_d%d" % D)
    st = check_discover(emr, genomes, sources, D, theta)
    assert st["records"] > 0



def test_compaction_over_many_tile_groups_sparse(emr):
    """Depth 8 (342 tiles per pair: the compaction visits only the groups of 64 tiles that the
    discover kernel marked), a population against the oracle."""
    genomes = W.population(31, 24, 20, 60)
    st = check_discover(emr, genomes, W.xor_sources(), 8, 0.03)
    assert st["records"] > 0


def test_compaction_over_many_tile_groups_dense(emr):
    """Depth 8 with theta < 0: every group of every pair is marked and every cell kept, so the
    records of each pair are its raw outputs in parent order, bit for bit; a second call on the
    same result (marks cleared and set again) gives the same records."""
    genomes = W.population(32, 3, 20, 60)
    sources = W.xor_sources()
    D = 8
    Q = oracle.n_parents(D)
    pop = emr.emr_pack_population(genomes)
    raw = emr.emr_eval_raw(pop, sources, D).cpu().numpy()
    res = emr.alloc_result(pop, sources, D)
    for call in range(2):
        emr.emr_discover(pop, sources, D, -1.0, res=res)
        assert emr.emr_result_check(res) == (len(genomes) * len(sources) * Q, Q)
        counts, recs = emr.records_to_host(res)
        assert np.all(counts == Q)
        for r in range(len(counts)):
            gp, gw = recs[r]
            assert np.array_equal(gp, np.arange(Q)), (call, r)
            assert np.array_equal(gw.reshape(-1).view(np.uint32), raw[r].view(np.uint32)), (call, r)


def test_config3_tabular_pop150_full(emr):
    """The tabular workload: 150 genomes (up to 40 hidden nodes, 120 edges) x 33 sources at depth
    6, every pair."""
    genomes, sources, D, theta = W.workload("tabular_pop150")
    st = check_discover(emr, genomes, sources, D, theta)
    assert st["records"] > 0


def test_config4_recurrent_depth10_two_phases(emr):
    """The recurrent workload at depth 10, end to end on the GPU: phase 1 (the XOR sources, all 100
    genomes) against the oracle; the hidden nodes found on the device equal the oracle's hidden
    sources from its own phase 1; phase 2 (per-genome CSR sources, one per hidden node) on 64
    sampled pairs against the oracle at the same sources."""
    genomes, sources, D, theta = W.workload("recurrent_pop100")
    theta32 = float(np.float32(theta))
    pop = emr.emr_pack_population(genomes)
    res = emr.emr_discover(pop, sources, D, theta32)
    emr.emr_result_check(res)
    counts, recs = emr.records_to_host(res)
    o = oracle.discover(genomes, sources, D, theta32)
    same = True
    for r in range(len(counts)):
        lo, hi = o["pair_offset"][r], o["pair_offset"][r + 1]
        gp, gw = recs[r]
        if not np.array_equal(gp, o["parent"][lo:hi]):
            same = False
            g, s = pair_genome_source(r, genomes, sources, None)
            diff = np.setxor1d(gp, o["parent"][lo:hi])
            _, dvar = oracle.eval_parents(g, s, diff)
            assert np.all(np.abs(dvar - theta32) <= BAND)
            common, gi, oi = np.intersect1d(gp, o["parent"][lo:hi], return_indices=True)
            assert close(gw[gi], o["w4"][lo:hi][oi]).all(), r
        else:
            assert close(gw, o["w4"][lo:hi]).all(), r
    # phase 2's sources on the device (hidden nodes of phase 1); the oracle's from its own phase 1
    hs_o, offs_o = oracle.hidden_sources(o, len(genomes), sources, D)
    hs_dev = emr.emr_hidden_sources(pop, sources, D, res)
    hs_g, offs_g = emr.hidden_sources_to_host(hs_dev)
    if same:
        np.testing.assert_array_equal(offs_g, offs_o)
        np.testing.assert_array_equal(hs_g["x"], hs_o["x"].astype(np.float32))
        np.testing.assert_array_equal(hs_g["y"], hs_o["y"].astype(np.float32))
    assert offs_g[-1] >= 64
    # phase 2 end to end on the GPU (per-genome CSR sources from the device), checked on 64 sampled
    # pairs against the oracle evaluated at the same sources
    res2 = emr.emr_discover_all(pop, hs_g, D, theta32, src_offsets=offs_g)
    counts2, recs2 = emr.records_to_host(res2)
    rng = np.random.default_rng(4)
    sample = np.sort(rng.choice(len(counts2), size=64, replace=False))
    owner = np.searchsorted(offs_g, sample, side="right") - 1
    sub_offs = np.zeros(len(genomes) + 1, np.int32)
    np.add.at(sub_offs, owner + 1, 1)
    sub_offs = np.cumsum(sub_offs).astype(np.int32)
    oo = oracle.discover(genomes, hs_g[sample], D, theta32, src_offsets=sub_offs)
    for k, r in enumerate(sample):
        lo, hi = oo["pair_offset"][k], oo["pair_offset"][k + 1]
        op, ow = oo["parent"][lo:hi], oo["w4"][lo:hi]
        gp, gw = recs2[r]
        if np.array_equal(gp, op):
            assert close(gw, ow).all(), r
        else:
            diff = np.setxor1d(gp, op)
            _, dvar = oracle.eval_parents(genomes[owner[k]], hs_g[r], diff)
            assert np.all(np.abs(dvar - theta32) <= BAND), (r, diff[:5], dvar[:5])


def test_flat_and_struct_packing_agree(emr):
    """emr_pack_population_flat (threaded packing, concatenated arrays) and emr_pack_population
    give the same programs: identical raw outputs; validation reports the lowest failing genome."""
    genomes = W.population(41, 300, 20, 60)
    sources = W.xor_sources()
    a = emr.emr_eval_raw(emr.emr_pack_population(genomes, layout="flat"), sources, 5).cpu().numpy()
    b = emr.emr_eval_raw(emr.emr_pack_population(genomes, layout="structs"), sources, 5).cpu().numpy()
    np.testing.assert_array_equal(a, b)
    bad = [dict(g) for g in genomes]
    for k in (250, 77):  # two failures: the lowest index is reported
        g = bad[k]
        src = np.concatenate([g["src"], g["dst"][:1]]).astype(np.int32)
        dst = np.concatenate([g["dst"], g["src"][:1]]).astype(np.int32)
        # close a cycle through a hidden node when the genome has one
        hidden = np.nonzero(np.asarray(g["kind"]) == 5)[0]
        if len(hidden) == 0:
            continue
        h = int(hidden[0])
        bad[k] = dict(g, src=np.concatenate([g["src"], [h, h]]).astype(np.int32),
                      dst=np.concatenate([g["dst"], [h, h]]).astype(np.int32),
                      w=np.concatenate([g["w"], [1.0, 1.0]]).astype(np.float32),
                      enabled=np.concatenate([np.ones(len(g["src"]), np.uint8), [1, 1]]))
    for layout in ("flat", "structs"):
        with pytest.raises(emr.EmrError) as e:
            emr.emr_pack_population(bad, layout=layout)
        assert e.value.status == emr.EMR_E_CYCLE
        assert e.value.bad_index == 77
