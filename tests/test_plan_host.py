"""The call tables the kernels read, built on the host exactly as the library builds them (the
library's own packing and planning code, compiled without HIP into the test shim), checked entry by
entry: every record stream, uniform program, bias row, pair id, member, pair record, uniform mark
and workspace region the kernels address lies inside its table. Also shows that the check refuses
each kind of bad entry. Host only."""

import ctypes as C

import numpy as np
import pytest

from paper_2608_27612_amd import emr, workloads as W
from tests import packed_interp as PI


def plan_check(genomes, sources, depth, offs=None, n_parts=3, plant=0):
    arr, keep = emr._genome_array(genomes) if len(genomes) else (None, None)
    src = emr._sources(sources)
    o = None if offs is None else np.ascontiguousarray(offs, dtype=np.int32)
    stats = (C.c_int64 * 5)()
    msg = C.create_string_buffer(512)
    rc = PI.shim().shim_plan_check(None if arr is None else C.byref(arr[0]), len(genomes), n_parts,
                                   src.ctypes.data, len(sources),
                                   None if o is None else o.ctypes.data,
                                   0 if o is not None else len(sources), depth, plant, stats, msg,
                                   len(msg))
    return rc, list(stats), msg.value.decode()


@pytest.mark.parametrize("name", sorted(W.WORKLOADS) + ["xor_pop1000_d5", "xor_pop1000_d8"])
def test_named_workload_tables_in_bounds(name):
    genomes, sources, depth, _ = W.workload(name)
    rc, stats, msg = plan_check(genomes, sources, depth)
    assert rc == 0, msg
    assert stats[0] > 0 and stats[1] >= stats[0]


def test_biased_population_and_per_genome_sources_in_bounds():
    genomes = W.population(5, 120, 40, 120, biases=True)
    rc, _, msg = plan_check(genomes, W.xor_sources(), 9)
    assert rc == 0, msg
    # per-genome sources: uneven counts, some genomes with none, both directions
    rng = np.random.default_rng(3)
    counts = rng.integers(0, 6, len(genomes))
    counts[::7] = 0
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    pts = [(float(rng.uniform(-1, 1)), float(rng.uniform(-1, 1)), int(rng.integers(0, 2)))
           for _ in range(int(offs[-1]))]
    rc, stats, msg = plan_check(genomes, W.sources_array(pts), 6, offs=offs)
    assert rc == 0, msg


def test_packing_in_ranges_relocates_every_descriptor():
    # the same population packed as 1, 2 and 7 ranges (as the library's packing threads do):
    # identical table sizes, and every range's descriptors checked against the words
    genomes = W.population(8, 200, 20, 60, biases=True)
    out = [plan_check(genomes, W.xor_sources(), 7, n_parts=k) for k in (1, 2, 7)]
    for rc, _, msg in out:
        assert rc == 0, msg
    assert out[0][1][:3] == out[1][1][:3] == out[2][1][:3]  # groups, members, bias floats


def test_tiny_and_empty_calls_in_bounds():
    assert plan_check([], W.xor_sources(), 5)[0] == 0
    g = W.single_cppn(0, 8, 20)  # a population of one
    assert plan_check(g, W.sources_array([(0.0, -1.0, 0)]), 0)[0] == 0
    assert plan_check(g, W.sources_array([]), 5)[0] == 0


@pytest.mark.parametrize("plant,what", [(1, "bias rows"), (2, "pair"), (3, "member"),
                                        (4, "descriptor"), (5, "group 1"), (6, "workspace")])
def test_check_refuses_each_kind_of_bad_entry(plant, what):
    genomes = W.population(9, 40, 20, 60)
    rc, _, msg = plan_check(genomes, W.xor_sources(), 6, plant=plant)
    assert rc == 1, msg
    assert what in msg, msg
