"""The allocation-free raw-output entry point (emr_eval_raw_noalloc) through the C ABI: its
outputs equal emr_eval_raw's, bit for bit, on two calls in a row (the second smaller, so stale
scratch contents from the first would show), and a call that needs more than the static scratch is
refused before anything is enqueued."""

import numpy as np
import pytest

import oracle
from paper_2608_27612_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def emr():
    import torch
    assert torch.cuda.is_available()
    from paper_2608_27612_amd import emr as E
    E.lib()
    return E


def run_noalloc(emr, pop, sources, D, offs=None):
    import torch
    n_pairs = emr.n_pairs_of(pop, sources, offs)
    out = torch.full((n_pairs, oracle.n_positions(D)), float("nan"), dtype=torch.float32,
                     device="cuda")
    err = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    emr.emr_eval_raw_noalloc(pop, sources, D, out, err, src_offsets=offs)
    torch.cuda.synchronize()
    return out.cpu().numpy(), int(err.item())


def test_noalloc_raw_equals_eval_raw_two_calls(emr):
    emr.emr_set_jit(emr.EMR_JIT_OFF)
    try:
        cases = [(W.population(61, 80, 20, 60, biases=True), W.xor_sources(), 6, None),
                 (W.population(62, 9, 12, 40), W.tabular_sources(5), 4, None)]
        for genomes, sources, D, offs in cases:
            pop = emr.emr_pack_population(genomes)
            want = emr.emr_eval_raw(pop, sources, D, src_offsets=offs).cpu().numpy()
            got, err = run_noalloc(emr, pop, sources, D, offs)
            assert err == 0
            assert got.shape == want.shape
            assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    finally:
        emr.emr_set_jit(emr.EMR_JIT_AUTO)


def test_noalloc_raw_per_genome_sources_and_reuse(emr):
    genomes = W.population(63, 12, 20, 60)
    ts = W.tabular_sources(6)
    sizes = [g % 4 for g in range(len(genomes))]
    offs = np.array([0] + list(np.cumsum(sizes)), np.int32)
    csr = np.concatenate([ts[:s] for s in sizes])
    pop = emr.emr_pack_population(genomes)
    want = emr.emr_eval_raw(pop, csr, 5, src_offsets=offs).cpu().numpy()
    for _ in range(2):  # the second call reuses the population's host-only plan
        got, err = run_noalloc(emr, pop, csr, 5, offs)
        assert err == 0
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_noalloc_refuses_calls_beyond_the_scratch(emr):
    import torch
    pop = emr.emr_pack_population(W.population(64, 2, 5, 10))
    out = torch.empty(1, dtype=torch.float32, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    # depth 15: 5.6M tiles of geometry alone exceed the scratch
    with pytest.raises(emr.EmrError) as e:
        emr.emr_eval_raw_noalloc(pop, W.xor_sources(), 15, out, err)
    assert e.value.status == emr.EMR_E_LIMIT
