"""A workspace reused by consecutive record calls: a call leaves its counters cleared and the next
call of the same plan, capacity and stream does not clear them again. Every call's records must
equal those of a call on a fresh workspace, bit for bit, across changes of theta, interleaved raw
calls, another plan on the same workspace and a capacity overflow."""

import numpy as np
import pytest

from paper_2608_27612_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def emr():
    import torch
    assert torch.cuda.is_available()
    from paper_2608_27612_amd import emr as E
    E.lib()
    return E


def host(emr, res):
    counts, recs = emr.records_to_host(res)
    return counts.copy(), [(p.copy(), w.copy()) for p, w in recs]


def same(a, b):
    np.testing.assert_array_equal(a[0], b[0])
    for (p1, w1), (p2, w2) in zip(a[1], b[1]):
        np.testing.assert_array_equal(p1, p2)
        np.testing.assert_array_equal(w1.view(np.uint32), w2.view(np.uint32))


@pytest.mark.parametrize("depth,n", [(6, 300), (8, 100)])
def test_reused_workspace_equals_fresh(emr, depth, n):
    genomes = W.population(71, n, 20, 60)
    sources = W.xor_sources()
    pop = emr.emr_pack_population(genomes)
    cap = n * len(sources) * emr.emr_grid_count(depth)[1]  # theta < 0 keeps every cell
    res = emr.alloc_result(pop, sources, depth, capacity=cap)

    def fresh(theta):
        r = emr.alloc_result(pop, sources, depth, capacity=cap)
        emr.emr_discover(pop, sources, depth, theta, res=r)
        emr.emr_result_check(r)
        return host(emr, r)

    thetas = [0.03, 0.03, 0.01, -1.0, 0.03, 0.0, 0.02, 0.02]
    want = {t: fresh(np.float32(t).item()) for t in set(thetas)}
    for k, t in enumerate(thetas):
        t32 = np.float32(t).item()
        emr.emr_discover(pop, sources, depth, t32, res=res)
        emr.emr_result_check(res)
        same(host(emr, res), want[t])
        if k == 3:
            # a raw-output call with the same workspace in between
            emr.emr_eval_raw(pop, sources, depth)


def test_another_plan_and_overflow_on_one_workspace(emr):
    genomes = W.population(72, 200, 20, 60)
    sources = W.xor_sources()
    pop = emr.emr_pack_population(genomes)
    D = 7
    res = emr.alloc_result(pop, sources, D)
    emr.emr_discover(pop, sources, D, 0.03, res=res)
    emr.emr_result_check(res)
    first = host(emr, res)
    # a capacity overflow on a small result, then the same plan again
    small = emr.alloc_result(pop, sources, D, capacity=16)
    emr.emr_discover(pop, sources, D, 0.03, res=small)
    with pytest.raises(emr.EmrError):
        emr.emr_result_check(small)
    emr.emr_discover(pop, sources, D, 0.03, res=small)
    with pytest.raises(emr.EmrError):
        emr.emr_result_check(small)
    # another depth (another plan) through the first result's buffers is refused or runs on a
    # fresh clear; the first plan then still gives its records
    other = emr.alloc_result(pop, sources, 6)
    emr.emr_discover(pop, sources, 6, 0.03, res=other)
    emr.emr_result_check(other)
    emr.emr_discover(pop, sources, D, 0.03, res=res)
    emr.emr_result_check(res)
    same(host(emr, res), first)


def test_every_cell_kept_with_a_pool_beyond_2_pow_23(emr):
    """theta < 0 keeps every parent (a variance is never negative): every pair's records are all
    parents in order, each with its children's raw outputs. With 400 pairs at depth 8 the pool
    holds 8.7M records, so pool offsets pass 2^23, where a status word's low half has its top bit
    set (a sign-extended read of it once dropped those records)."""
    genomes = W.population(73, 100, 20, 60)
    sources = W.xor_sources()
    pop = emr.emr_pack_population(genomes)
    D = 8
    Q = emr.emr_grid_count(D)[1]
    cap = 100 * len(sources) * Q
    assert cap > 1 << 23
    raw = emr.emr_eval_raw(pop, sources, D).cpu().numpy().reshape(len(genomes) * len(sources), -1)
    for _ in range(2):
        res = emr.alloc_result(pop, sources, D, capacity=cap)
        emr.emr_discover(pop, sources, D, -1.0, res=res)
        total, mx = emr.emr_result_check(res)
        assert total == cap and mx == Q
        counts, recs = emr.records_to_host(res)
        for r, (p, w) in enumerate(recs):
            np.testing.assert_array_equal(p, np.arange(Q))
            # (equal as floats: a -0.0 node bias may stay -0.0 in one tier and not the other)
            np.testing.assert_array_equal(w.reshape(-1), raw[r, :4 * Q])


@pytest.mark.parametrize("depth,n,in_flight", [(7, 400, 2), (7, 400, 4), (8, 120, 4)])
def test_calls_in_flight_on_their_own_streams(emr, depth, n, in_flight):
    """Results, each with its workspace and stream, take the calls in turn with `in_flight` calls
    in flight (call i is checked after call i + in_flight - 1 is enqueued, as the benchmark's timed
    steps run): every call's records equal those of a single synchronous call on a fresh
    workspace, bit for bit, and every call's check reports the same total. The compiled tier runs
    from the second call on."""
    import torch
    genomes = W.population(72, n, 20, 60)
    sources = W.xor_sources()
    theta = np.float32(0.03).item()
    pop = emr.emr_pack_population(genomes)
    ref = emr.alloc_result(pop, sources, depth)
    emr.emr_discover(pop, sources, depth, theta, res=ref)
    total, _ = emr.emr_result_check(ref)
    want = host(emr, ref)
    bufs = [emr.alloc_result(pop, sources, depth) for _ in range(in_flight)]
    streams = [torch.cuda.Stream() for _ in range(in_flight)]
    got = []

    def check(i):
        t, _ = emr.emr_result_check(bufs[i % in_flight])
        assert t == total, (i, t, total)
        got.append(host(emr, bufs[i % in_flight]))

    n_calls = 3 * in_flight + 1
    lag = in_flight - 1
    for i in range(n_calls):
        emr.emr_discover(pop, sources, depth, theta, res=bufs[i % in_flight],
                         stream=streams[i % in_flight])
        if i >= lag:
            check(i - lag)
    for i in range(n_calls - lag, n_calls):
        check(i)
    assert len(got) == n_calls
    assert emr.emr_jit_info(pop)["state"] == 1
    for g in got:
        same(g, want)
