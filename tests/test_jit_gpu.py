"""GPU tests of the compiled tier: compiled programs produce the interpreter's bits (raw outputs,
records in both placements, streamed chunks) and match the oracle; the policy switches tiers as
documented."""

import numpy as np
import pytest

from paper_2608_27612_amd import workloads as W
from tests.test_parity_gpu import check_discover, check_raw

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def emr():
    import torch
    assert torch.cuda.is_available()
    from paper_2608_27612_amd import emr as E
    E.lib()
    return E


@pytest.fixture(autouse=True)
def default_policy(emr):
    yield
    emr.emr_set_jit(emr.EMR_JIT_AUTO)


def both_tiers(emr, fn):
    """fn(pop) on a fresh population under the interpreter, then under the compiled tier."""
    out = []
    for policy in (emr.EMR_JIT_OFF, emr.EMR_JIT_ALWAYS):
        emr.emr_set_jit(policy)
        out.append(fn(policy))
    return out


def raw_both(emr, genomes, sources, D, offs=None):
    def run(policy):
        pop = emr.emr_pack_population(genomes)
        raw = emr.emr_eval_raw(pop, sources, D, src_offsets=offs).cpu().numpy()
        info = emr.emr_jit_info(pop)
        assert info["state"] == (1 if policy == emr.EMR_JIT_ALWAYS else 0), info
        return raw
    return both_tiers(emr, run)


def records_both(emr, genomes, sources, D, theta, offs=None):
    def run(policy):
        pop = emr.emr_pack_population(genomes)
        res = emr.emr_discover(pop, sources, D, float(np.float32(theta)), src_offsets=offs)
        emr.emr_result_check(res)
        assert emr.emr_jit_info(pop)["state"] == (1 if policy == emr.EMR_JIT_ALWAYS else 0)
        return emr.records_to_host(res)
    (ci, ri), (cj, rj) = both_tiers(emr, run)
    assert np.array_equal(ci, cj)
    for r in range(len(ci)):
        assert np.array_equal(ri[r][0], rj[r][0]), r
        assert np.array_equal(ri[r][1].view(np.uint32), rj[r][1].view(np.uint32)), r
    return ci


def test_raw_outputs_bit_identical_single(emr):
    genomes, sources, D, _ = W.workload("single_d5")
    a, b = raw_both(emr, genomes, sources, D)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_raw_outputs_bit_identical_population(emr):
    a, b = raw_both(emr, W.population(1, 40, 20, 60), W.xor_sources(), 5)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_raw_outputs_bit_identical_large_genomes_many_sources(emr):
    # up to 40 hidden nodes and 120 edges: the wider register windows and sources per walk
    a, b = raw_both(emr, W.population(4, 12, 40, 120), W.tabular_sources(), 4)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("act", range(6))
def test_raw_outputs_bit_identical_each_activation(emr, act):
    g = {"kind": np.array([0, 1, 2, 3, 4, 6, 5], np.uint8),
         "act": np.array([0, 0, 0, 0, 0, 0, act], np.uint8), "bias": np.zeros(7, np.float32),
         "src": np.array([2, 3, 4, 6, 2], np.int32), "dst": np.array([6, 6, 6, 5, 5], np.int32),
         "w": np.array([3.0, -2.0, 0.5, 2.0, 1.0], np.float32),
         "enabled": np.ones(5, np.uint8)}
    a, b = raw_both(emr, [g], W.xor_sources(), 5)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_records_bit_identical_population_depth6(emr):
    records_both(emr, W.population(2, 200, 20, 60), W.xor_sources(), 6, 0.03)


def test_records_bit_identical_tabular(emr):
    records_both(emr, W.population(3, 20, 40, 120), W.tabular_sources(), 5, 0.03)


def test_records_bit_identical_per_genome_sources(emr):
    genomes = W.population(6, 30, 20, 60)
    rng = np.random.default_rng(6)
    offs = np.zeros(len(genomes) + 1, np.int32)
    srcs = []
    for g in range(len(genomes)):
        k = int(rng.integers(0, 7))
        for _ in range(k):
            srcs.append((float(rng.uniform(-1, 1)), float(rng.uniform(-1, 1)), 0))
        offs[g + 1] = offs[g] + k
    records_both(emr, genomes, W.sources_array(srcs), 5, 0.02, offs=offs)


def test_records_bit_identical_uniform_outputs_and_negative_theta(emr):
    # theta < 0 keeps every cell, so uniform outputs (no varying program) produce records too
    genomes = W.population(7, 50, 3, 4)
    counts = records_both(emr, genomes, W.xor_sources(), 4, -1.0)
    assert np.all(counts == (4 ** 4 - 1) // 3)


def test_compiled_tier_matches_the_oracle_pop1000_depth5(emr):
    emr.emr_set_jit(emr.EMR_JIT_ALWAYS)
    genomes, sources, D, theta = W.workload("xor_pop1000_d5")
    pop = emr.emr_pack_population(genomes)
    check_discover(emr, genomes, sources, D, theta, pop=pop)
    assert emr.emr_jit_info(pop)["state"] == 1


def test_compiled_tier_streamed_equals_interpreted_one_shot(emr):
    genomes, sources, _, _ = W.workload("deep_single")
    D, theta = 9, float(np.float32(0.01))
    emr.emr_set_jit(emr.EMR_JIT_OFF)
    pop = emr.emr_pack_population(genomes)
    res = emr.emr_discover(pop, sources, D, theta)
    emr.emr_result_check(res)
    counts, recs = emr.records_to_host(res)
    emr.emr_set_jit(emr.EMR_JIT_ALWAYS)
    pop2 = emr.emr_pack_population(genomes)
    got = {}

    def sink(pair, chunk, parent, w4):
        got.setdefault(pair, []).append((parent, w4))
    emr.emr_discover_stream(pop2, sources, D, theta, sink, chunk_positions=1 << 14)
    assert emr.emr_jit_info(pop2)["state"] == 1
    for r in range(len(counts)):
        parts = got.get(r, [])
        p = np.concatenate([x[0] for x in parts]) if parts else np.zeros(0, np.uint32)
        w = np.concatenate([x[1] for x in parts]) if parts else np.zeros((0, 4), np.float32)
        assert np.array_equal(p.astype(np.int64), recs[r][0])
        assert np.array_equal(w.view(np.uint32), recs[r][1].view(np.uint32))


def test_auto_policy_compiles_on_the_second_call(emr):
    emr.emr_set_jit(emr.EMR_JIT_AUTO)
    genomes = W.population(8, 100, 20, 60)
    sources = W.xor_sources()
    pop = emr.emr_pack_population(genomes)
    res = emr.alloc_result(pop, sources, 5)
    emr.emr_profile_enable(True)
    emr.emr_discover(pop, sources, 5, 0.03, res=res)
    emr.emr_result_check(res)
    assert emr.emr_jit_info(pop)["state"] == 0
    first = emr.records_to_host(res)
    emr.emr_discover(pop, sources, 5, 0.03, res=res)
    emr.emr_result_check(res)
    info = emr.emr_jit_info(pop)
    assert info["state"] == 1 and info["programs"] > 0 and info["code_bytes"] > 0
    second = emr.records_to_host(res)
    recs = emr.emr_profile_read()
    emr.emr_profile_enable(False)
    assert [r["compiled"] for r in recs] == [False, True]
    assert np.array_equal(first[0], second[0])
    for a, b in zip(first[1], second[1]):
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_biased_population_both_tiers(emr):
    """Nonzero node biases: raw outputs of both tiers bit-identical and within tolerance of the
    oracle; records of both tiers against the oracle."""
    genomes = W.population(53, 120, 20, 60, biases=True)
    sources = W.xor_sources()
    a, b = raw_both(emr, genomes, sources, 5)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    for policy in (emr.EMR_JIT_OFF, emr.EMR_JIT_ALWAYS):
        emr.emr_set_jit(policy)
        check_raw(emr, genomes, sources, 5)
        pop = emr.emr_pack_population(genomes)
        check_discover(emr, genomes, sources, 6, 0.03, pop=pop)
        assert emr.emr_jit_info(pop)["state"] == (1 if policy == emr.EMR_JIT_ALWAYS else 0)


@pytest.mark.parametrize("act", range(6))
def test_biased_node_of_each_activation_both_tiers(emr, act):
    # hidden h = act(3 x2 - 2 y2 + 0.5 + 0.7) with a uniform node u = act(x1 + 0.4) feeding it,
    # output = linear(2 h + x2 - 1.25): a bias reaches every activation in both kinds of node
    g = {"kind": np.array([0, 1, 2, 3, 4, 6, 5, 5], np.uint8),
         "act": np.array([0] * 5 + [0, act, act], np.uint8),
         "bias": np.array([0, 0, 0, 0, 0, -1.25, 0.7, 0.4], np.float32),
         "src": np.array([2, 3, 4, 6, 2, 0, 7], np.int32),
         "dst": np.array([6, 6, 6, 5, 5, 7, 6], np.int32),
         "w": np.array([3.0, -2.0, 0.5, 2.0, 1.0, 1.0, 0.75], np.float32),
         "enabled": np.ones(7, np.uint8)}
    a, b = raw_both(emr, [g], W.xor_sources(), 5)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    for policy in (emr.EMR_JIT_OFF, emr.EMR_JIT_ALWAYS):
        emr.emr_set_jit(policy)
        check_raw(emr, [g], W.xor_sources(), 5)
