"""GPU tests of the operations on a discovery's CSR records (through the C ABI): the hidden nodes
of Phase 2 (and their iteration), the connection types and weight filter, and Eq. 2's literal
chain rule, each against the oracle.

Where floating point decides an integer (a kept cell, a weight above the filter), the oracle is
applied to the GPU's own float32 records, so both sides decide on the same values; the records
themselves are checked against the oracle's in test_parity_gpu.py."""

import numpy as np
import pytest

import oracle
from paper_2608_27612_amd import workloads as W
from tests.test_parity_gpu import BAND, check_discover, close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def emr():
    import torch
    assert torch.cuda.is_available()
    from paper_2608_27612_amd import emr as E
    E.lib()
    return E


def host_records(emr, res):
    """A checked GPU result as the oracle's records dict (float32 weights as given)."""
    counts, recs = emr.records_to_host(res)
    offs = np.zeros(len(counts) + 1, np.int64)
    np.cumsum(counts, out=offs[1:])
    parent = np.concatenate([p for p, _ in recs]) if len(recs) else np.zeros(0, np.int64)
    w4 = np.concatenate([w for _, w in recs]) if len(recs) else np.zeros((0, 4), np.float32)
    return {"pair_count": counts, "pair_offset": offs, "parent": parent, "w4": w4}


def check_hidden(emr, hs, want_cells, depth):
    """An emr_hidden_sources output equals the given per-genome cells, with exact centres."""
    offs = hs["offsets"].cpu().numpy()
    n = hs["total"]
    assert offs[-1] == n == sum(len(c) for c in want_cells)
    cells = hs["cell"][:n].cpu().numpy().view(np.uint32).astype(np.int64)
    src, _ = emr.hidden_sources_to_host(hs)
    xy = oracle.grid(depth)
    for g, want in enumerate(want_cells):
        got = cells[offs[g]:offs[g + 1]]
        np.testing.assert_array_equal(got, want)
        np.testing.assert_array_equal(src["x"][offs[g]:offs[g + 1]], xy[want - 1, 0].astype(np.float32))
        np.testing.assert_array_equal(src["y"][offs[g]:offs[g + 1]], xy[want - 1, 1].astype(np.float32))
        assert np.all(src["dir"][offs[g]:offs[g + 1]] == 0)


@pytest.mark.parametrize("D", [5, 7])
def test_hidden_sources_match_oracle(emr, D):
    genomes = W.population(81, 120, 20, 60)
    sources = W.xor_sources()
    pop = emr.emr_pack_population(genomes)
    res = emr.emr_discover_all(pop, sources, D, float(np.float32(0.03)))
    hs = emr.emr_hidden_sources(pop, sources, D, res)
    # the same set logic applied by the oracle to the GPU's records
    want = oracle.hidden_cells(host_records(emr, res), len(genomes), sources)
    check_hidden(emr, hs, want, D)
    assert hs["total"] > 0


def test_hidden_sources_iterated_with_known_cells(emr):
    """Phase 2 iterated: the second call's nodes are the children of the phase-2 records that are
    not nodes already; `known` ends as the union of both sets."""
    import torch
    genomes = W.population(82, 60, 20, 60)
    sources = W.xor_sources()
    D, theta = 6, float(np.float32(0.03))
    G = len(genomes)
    pop = emr.emr_pack_population(genomes)
    words = emr.emr_cell_words(D)
    known = torch.zeros(G * words, dtype=torch.int32, device="cuda")
    res1 = emr.emr_discover_all(pop, sources, D, theta)
    hs1 = emr.emr_hidden_sources(pop, sources, D, res1, known=known)
    c1 = oracle.hidden_cells(host_records(emr, res1), G, sources)
    check_hidden(emr, hs1, c1, D)
    src2, offs2 = emr.hidden_sources_to_host(hs1)
    res2 = emr.emr_discover_all(pop, src2, D, theta, src_offsets=offs2)
    check_discover(emr, genomes, src2, D, theta, offs=offs2, pop=pop)
    hs2 = emr.emr_hidden_sources(pop, src2, D, res2, src_offsets=offs2, known=known)
    c2 = oracle.hidden_cells(host_records(emr, res2), G, src2, src_offsets=offs2, exclude=c1)
    check_hidden(emr, hs2, c2, D)
    bits = known.cpu().numpy().view(np.uint32).reshape(G, words)
    for g in range(G):
        want = np.union1d(c1[g], c2[g]) - 1  # grid positions
        got = np.nonzero(np.unpackbits(bits[g].view(np.uint8), bitorder="little"))[0]
        np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("mask", [15, 1, 2, 4, 8, 2 | 4 | 8])
@pytest.mark.parametrize("w_min", [0.1, -1.0])
def test_express_matches_oracle(emr, mask, w_min):
    """Connections of a hidden-to-hidden call (sources at cell centres see all four types) and of
    the input/output call, against the oracle's expression of the same records."""
    genomes = W.population(83, 40, 20, 60)
    sources = W.xor_sources()
    D, theta = 5, float(np.float32(0.02))
    w32 = float(np.float32(w_min))
    pop = emr.emr_pack_population(genomes)
    res1 = emr.emr_discover_all(pop, sources, D, theta)
    hs = emr.emr_hidden_sources(pop, sources, D, res1)
    src2, offs2 = emr.hidden_sources_to_host(hs)
    res2 = emr.emr_discover_all(pop, src2, D, theta, src_offsets=offs2)
    for res, srcs, offs in ((res1, sources, None), (res2, src2, offs2)):
        con = emr.emr_express(pop, srcs, D, res, mask, w32, src_offsets=offs)
        want = oracle.express(host_records(emr, res), srcs, D, mask, w32, n_genomes=len(genomes),
                              src_offsets=offs)
        np.testing.assert_array_equal(con["pair_offset"].cpu().numpy(), want["pair_offset"])
        n = con["total"]
        np.testing.assert_array_equal(con["cell"][:n].cpu().numpy().view(np.uint32), want["cell"])
        np.testing.assert_array_equal(con["w"][:n].cpu().numpy(), want["w"].astype(np.float32))
    if mask == 8 and w_min < 0:
        assert int(con["total"]) > 0  # hidden nodes at kept cells find themselves


def test_chain_filter_matches_oracle(emr):
    """Eq. 2 read literally: the chain-filtered GPU records equal the oracle's chain filter of the
    same records; where the parent-rule sets agree with the oracle's, they equal the oracle's own
    literal chain recursion, i.e. ES-HyperNEAT's division."""
    genomes = W.population(84, 200, 20, 60)
    sources = W.xor_sources()
    D, theta = 7, float(np.float32(0.02))
    pop = emr.emr_pack_population(genomes)
    res = emr.emr_discover_all(pop, sources, D, theta)
    ch = emr.emr_chain_filter(res, D)
    want = oracle.chain_filter(host_records(emr, res), D)
    got = host_records(emr, ch)
    np.testing.assert_array_equal(got["pair_count"], want["pair_count"])
    np.testing.assert_array_equal(got["parent"], want["parent"])
    np.testing.assert_array_equal(got["w4"], want["w4"])
    assert len(got["parent"]) < int(res["pair_offset"][-1].item())
    lit = oracle.discover(genomes, sources, D, theta, oracle.CHAIN)
    eager = oracle.discover(genomes, sources, D, theta, oracle.PARENT)
    g_all = host_records(emr, res)
    for r in range(len(lit["pair_count"])):
        lo, hi = eager["pair_offset"][r], eager["pair_offset"][r + 1]
        glo, ghi = g_all["pair_offset"][r], g_all["pair_offset"][r + 1]
        if not np.array_equal(g_all["parent"][glo:ghi], eager["parent"][lo:hi]):
            continue  # a band cell differs: the chain can differ below it
        a, b = lit["pair_offset"][r], lit["pair_offset"][r + 1]
        c, d = got["pair_offset"][r], got["pair_offset"][r + 1]
        np.testing.assert_array_equal(got["parent"][c:d], lit["parent"][a:b])
        assert close(got["w4"][c:d], lit["w4"][a:b]).all()


def test_phase2_empty_and_capacity(emr):
    genomes = W.population(85, 10, 10, 30)
    sources = W.xor_sources()
    pop = emr.emr_pack_population(genomes)
    res = emr.emr_discover_all(pop, sources, 5, 1e30)  # nothing kept
    assert emr.emr_hidden_sources(pop, sources, 5, res)["total"] == 0
    assert emr.emr_express(pop, sources, 5, res)["total"] == 0
    assert int(emr.emr_chain_filter(res, 5)["pair_offset"][-1].item()) == 0
    res = emr.emr_discover_all(pop, sources, 5, 0.001)
    total = int(res["pair_offset"][-1].item())
    with pytest.raises(emr.EmrError) as e:
        emr.emr_express(pop, sources, 5, res, 15, -1.0, capacity=total)  # 4 per record needed
    assert e.value.status == emr.EMR_E_CAPACITY and str(4 * total) in str(e.value)


def test_hidden_sources_of_skewed_records(emr):
    """Hand-built CSR results whose records are spread as a discovery can spread them at its
    extremes: long runs of empty pairs, pairs of thousands of records crossing the marking's spans
    of 1024 records, incoming pairs holding records (which add no node), and, at depth 8, more
    records than one sweep of the marking kernel's waves covers (8.4M), so its waves loop. Each
    pair's records are distinct parents in ascending order, as a discovery leaves them. The hidden
    nodes equal the oracle's set logic applied to the same records."""
    import torch
    sources = W.xor_sources()  # 3 outgoing sources and 1 incoming per genome
    rng = np.random.default_rng(86)
    for D, G, heavy_share, lo_share in ((7, 24, 0.08, 0.3), (8, 150, 0.7, 0.9)):
        genomes = W.population(86 + D, G, 12, 40)
        n_pairs = G * len(sources)
        _, Q = emr.emr_grid_count(D)
        pop = emr.emr_pack_population(genomes)
        counts = np.zeros(n_pairs, np.int64)
        hot = rng.choice(n_pairs, size=n_pairs // 5, replace=False)
        counts[hot] = rng.integers(1, 40, size=len(hot))
        heavy = rng.choice(n_pairs, size=max(2, int(heavy_share * n_pairs)), replace=False)
        counts[heavy] = rng.integers(int(lo_share * Q), Q + 1, size=len(heavy))
        counts[n_pairs - 1] = 3  # the last pair (incoming) holds records too
        offs = np.zeros(n_pairs + 1, np.int64)
        np.cumsum(counts, out=offs[1:])
        total = int(offs[-1])
        assert D == 7 or total > 8 * 1024 * 1024
        parent = np.concatenate([np.sort(rng.choice(Q, size=int(c), replace=False))
                                 for c in counts]).astype(np.int64)
        res = emr.alloc_result(pop, sources, D, capacity=total)
        res["pair_count"].copy_(torch.from_numpy(counts))
        res["pair_offset"].copy_(torch.from_numpy(offs))
        res["parent"][:total].copy_(torch.from_numpy(parent.astype(np.uint32).view(np.int32)))
        hs = emr.emr_hidden_sources(pop, sources, D, res)
        want = oracle.hidden_cells({"pair_offset": offs, "parent": parent}, G, sources)
        check_hidden(emr, hs, want, D)
        del res, hs
