"""Streamed discovery (emr_discover_stream) on the GPU: chunked output equals the one-shot output,
runs resume from any cursor, bad arguments are refused before any GPU work, and the depth-13
single-CPPN workload matches the oracle on sampled cells."""

import numpy as np
import pytest

import oracle
from paper_2608_27612_amd import workloads as W
from tests.test_parity_gpu import close

pytestmark = pytest.mark.gpu

BAND = 1e-5


@pytest.fixture(scope="module")
def emr():
    import torch  # noqa: F401
    from paper_2608_27612_amd import emr as E
    E.lib()
    return E


def collect(emr, pop, sources, D, theta, chunk, start=0, stop_after=None, offs=None):
    """Runs a stream; returns ({pair: [(chunk, parent, w4), ...]}, cursors delivered, status)."""
    got, order = {}, []

    def sink(pair, chunk_i, parent, w4):
        if stop_after is not None and len(order) == stop_after:
            return False
        got.setdefault(pair, []).append((chunk_i, parent, w4))
        order.append((chunk_i, pair))
        return True

    nxt = emr.emr_discover_stream(pop, sources, D, theta, sink, chunk_positions=chunk,
                                  start=start, src_offsets=offs)
    return got, order, nxt


def concat(parts):
    if not parts:
        return np.zeros(0, np.uint32), np.zeros((0, 4), np.float32)
    return np.concatenate([p for _, p, _ in parts]), np.concatenate([w for _, _, w in parts])


def one_shot(emr, pop, sources, D, theta, offs=None):
    res = emr.emr_discover(pop, sources, D, theta, src_offsets=offs)
    emr.emr_result_check(res)
    return emr.records_to_host(res)


@pytest.mark.parametrize("chunk", [256, 256 * 3, 256 * 64, 1 << 24])
def test_stream_equals_one_shot(emr, chunk):
    genomes = W.population(31, 40, 20, 60)
    sources = W.xor_sources()
    D, theta = 7, float(np.float32(0.02))
    pop = emr.emr_pack_population(genomes)
    counts, recs = one_shot(emr, pop, sources, D, theta)
    got, order, nxt = collect(emr, pop, sources, D, theta, chunk)
    n_pairs = len(counts)
    assert nxt == emr.emr_stream_chunks(D, chunk) * n_pairs
    # deliveries come chunk after chunk, pair after pair
    assert order == sorted(order)
    for r in range(n_pairs):
        p, w = concat(got.get(r, []))
        np.testing.assert_array_equal(p, recs[r][0])
        np.testing.assert_array_equal(w, recs[r][1])  # same kernels, same arithmetic: bit-exact
        for c, parent, _ in got.get(r, []):
            # a chunk's records are parents of the chunk's tiles
            lo, hi = chunk_parent_range(D, chunk, c)
            assert parent.min() >= lo and parent.max() < hi


def chunk_parent_range(D, chunk, c):
    """[lo, hi) of the parent indices whose children lie in chunk c (tiles of 256 positions, the
    first holding levels 1..3)."""
    tpc = chunk // 256

    def tile_parent(T):
        if T == 0:
            return 0
        if D < 4:
            return oracle.n_parents(D)
        return 21 + (T - 1) * 64

    tiles = 1 if D < 4 else 1 + (oracle.n_positions(D) - 84) // 256
    return tile_parent(c * tpc), tile_parent(min(tiles, (c + 1) * tpc))


def test_stream_per_genome_sources_and_small_depths(emr):
    genomes = W.population(32, 12, 20, 60)
    ts = W.tabular_sources(6)
    sizes = [1 + g % 4 for g in range(len(genomes))]
    offs = np.array([0] + list(np.cumsum(sizes)), np.int32)
    csr = np.concatenate([ts[-s:] if g % 2 else ts[:s] for g, s in enumerate(sizes)])
    pop = emr.emr_pack_population(genomes)
    for D in (0, 1, 3, 4, 6):
        theta = float(np.float32(0.01))
        counts, recs = one_shot(emr, pop, csr, D, theta, offs=offs)
        got, _, _ = collect(emr, pop, csr, D, theta, 512, offs=offs)
        for r in range(len(counts)):
            p, w = concat(got.get(r, []))
            np.testing.assert_array_equal(p, recs[r][0])
            np.testing.assert_array_equal(w, recs[r][1])


def test_stream_stop_and_resume(emr):
    genomes = W.population(33, 30, 20, 60)
    sources = W.xor_sources()
    D, theta, chunk = 6, float(np.float32(0.02)), 512
    pop = emr.emr_pack_population(genomes)
    full, full_order, total = collect(emr, pop, sources, D, theta, chunk)
    assert len(full_order) > 20
    n_pairs = len(genomes) * len(sources)
    # stop after 11 deliveries: the 12th is refused and is where the run resumes
    with pytest.raises(emr.EmrError) as e:
        collect(emr, pop, sources, D, theta, chunk, stop_after=11)
    assert e.value.status == emr.EMR_E_ABORTED
    c12, r12 = full_order[11]
    assert e.value.next_cursor == c12 * n_pairs + r12
    rest, rest_order, nxt = collect(emr, pop, sources, D, theta, chunk, start=e.value.next_cursor)
    assert nxt == total
    assert full_order[:11] + rest_order == full_order
    # resuming from any cursor delivers exactly the later deliveries
    for start in [0, 1, n_pairs - 1, n_pairs, 5 * n_pairs + 7, total - 1, total]:
        _, order, _ = collect(emr, pop, sources, D, theta, chunk, start=start)
        assert order == [(c, r) for c, r in full_order if c * n_pairs + r >= start]


def test_stream_refuses_bad_arguments(emr):
    genomes = W.population(34, 4, 10, 30)
    pop = emr.emr_pack_population(genomes)
    sources = W.xor_sources()
    for chunk in [0, 100, 256 + 1, -256]:
        with pytest.raises(emr.EmrError) as e:
            collect(emr, pop, sources, 5, 0.03, chunk)
        assert e.value.status == emr.EMR_E_INVAL
    total = emr.emr_stream_chunks(5, 256) * len(genomes) * len(sources)
    for start in [-1, total + 1]:
        with pytest.raises(emr.EmrError) as e:
            collect(emr, pop, sources, 5, 0.03, 256, start=start)
        assert e.value.status == emr.EMR_E_INVAL
    # a sink that raises stops the run and the exception reaches the caller
    def bad(*args):
        raise ValueError("sink failure")
    with pytest.raises(ValueError):
        emr.emr_discover_stream(pop, sources, 5, 0.0, bad, chunk_positions=256)


def test_stream_deep_single_depth9_matches_oracle(emr):
    """The depth-13 workload's CPPN and sources at depth 9, against the full oracle."""
    genomes, sources, _, theta = W.workload("deep_single")
    theta32 = float(np.float32(theta))
    D = 9
    pop = emr.emr_pack_population(genomes)
    got, _, _ = collect(emr, pop, sources, D, theta32, 1 << 14)
    o = oracle.discover(genomes, sources, D, theta32)
    for r in range(len(sources)):
        p, w = concat(got.get(r, []))
        lo, hi = o["pair_offset"][r], o["pair_offset"][r + 1]
        op, ow = o["parent"][lo:hi], o["w4"][lo:hi]
        diff = np.setxor1d(p, op)
        if len(diff):
            _, dvar = oracle.eval_parents(genomes[0], sources[r], diff)
            assert np.all(np.abs(dvar - theta32) <= BAND), (r, diff[:5], dvar[:5])
        common, gi, oi = np.intersect1d(p, op, return_indices=True)
        assert close(w[gi], ow[oi]).all(), r


def check_deep_against_oracle(genome, sources, D, theta32, parents, samples, rng):
    """Per pair: the delivered parents (a list of ascending arrays) are increasing across
    deliveries and at most Q(D); the sampled records (parent, w4) match the oracle evaluated cell
    by cell and pass theta; random parents are delivered exactly when the oracle's variance is
    above theta (outside the band around it). Returns the records delivered."""
    Q = oracle.n_parents(D)
    kept_total = 0
    for r in range(len(sources)):
        allp = np.concatenate(parents[r]) if parents[r] else np.zeros(0, np.uint32)
        assert np.all(np.diff(allp.astype(np.int64)) > 0)
        assert len(allp) <= Q and (len(allp) == 0 or int(allp[-1]) < Q)
        if samples[r]:
            p = np.concatenate([a for a, _ in samples[r]])
            w = np.concatenate([b for _, b in samples[r]])
            ow, ovar = oracle.eval_parents(genome, sources[r], p)
            assert np.all(ovar > theta32 - BAND)
            assert close(w, ow).all(), r
        cand = np.unique(rng.integers(0, Q, size=4000)).astype(np.uint32)
        _, cvar = oracle.eval_parents(genome, sources[r], cand)
        delivered = np.isin(cand, allp)
        assert np.all(delivered[cvar > theta32 + BAND])
        assert not np.any(delivered[cvar < theta32 - BAND])
        kept_total += len(allp)
    return kept_total


def test_stream_deep_single_depth13_sampled(emr):
    """The depth-13 streamed run (one CPPN with 30 hidden nodes and 90 edges, 4 sources, 358M
    queries, chunks of 2^24 positions): every delivery is well formed, sampled kept records match
    the oracle evaluated cell by cell, and sampled parents are kept exactly when the oracle's
    variance is above theta (outside the band around it)."""
    genomes, sources, D, theta = W.workload("deep_single")
    assert D == 13
    theta32 = float(np.float32(theta))
    pop = emr.emr_pack_population(genomes)
    rng = np.random.default_rng(13)
    parents = {r: [] for r in range(len(sources))}
    samples = {r: [] for r in range(len(sources))}

    def sink(pair, chunk, parent, w4):
        parents[pair].append(parent)
        take = rng.choice(len(parent), size=min(40, len(parent)), replace=False)
        samples[pair].append((parent[take], w4[take]))
        return True

    nxt = emr.emr_discover_stream(pop, sources, D, theta32, sink, chunk_positions=1 << 24)
    assert nxt == emr.emr_stream_chunks(D, 1 << 24) * len(sources)
    assert check_deep_against_oracle(genomes[0], sources, D, theta32, parents, samples, rng) > 0


def test_stream_to_record_file_and_resume(emr, tmp_path):
    """A run written by the record-file sink holds exactly the deliveries a Python sink receives;
    a file cut inside a block (a run that died while writing) resumes at its last whole delivery,
    and the resumed run completes the same file byte for byte."""
    genomes = W.population(35, 40, 20, 60)
    sources = W.xor_sources()
    D, theta, chunk = 7, float(np.float32(0.02)), 256 * 16
    pop = emr.emr_pack_population(genomes)
    n_pairs = len(genomes) * len(sources)
    got, order, total = collect(emr, pop, sources, D, theta, chunk)
    path = str(tmp_path / "run.rec")
    with emr.RecordFile(path, n_pairs) as f:
        assert emr.emr_discover_stream(pop, sources, D, theta, f, chunk_positions=chunk) == total
    n, blocks = emr.read_record_file(path)
    assert n == n_pairs
    assert [(c, r) for r, c, _, _ in blocks] == order
    seen = {}
    for r, c, p, w in blocks:
        k = seen.get(r, 0)
        c0, p0, w0 = got[r][k]
        assert c == c0
        np.testing.assert_array_equal(p, p0)
        np.testing.assert_array_equal(w, w0)
        seen[r] = k + 1
    full = open(path, "rb").read()
    cut_block = len(blocks) // 2
    start = 32 + sum(24 + 20 * len(b[2]) for b in blocks[:cut_block])
    with open(path, "r+b") as fh:
        fh.truncate(start + 24 + 8)
    f = emr.RecordFile(path, n_pairs, resume=True)
    r_, c_ = blocks[cut_block - 1][0], blocks[cut_block - 1][1]
    assert f.cursor == c_ * n_pairs + r_ + 1
    assert emr.emr_discover_stream(pop, sources, D, theta, f, chunk_positions=chunk,
                                   start=f.cursor) == total
    recs, nxt = f.close()
    assert open(path, "rb").read() == full
    assert recs == sum(len(b[2]) for b in blocks)
    # resuming a complete file delivers nothing more
    with emr.RecordFile(path, n_pairs, resume=True) as f:
        assert emr.emr_discover_stream(pop, sources, D, theta, f, chunk_positions=chunk,
                                       start=f.cursor) == total
    assert open(path, "rb").read() == full


def test_stream_deep_single_depth14_to_disk(emr, tmp_path):
    """The same CPPN and sources at depth 14 (358M positions per source: the paper's depth-13
    substrate; 1.43G queries) streamed to a record file on disk in chunks of 2^24 positions, then
    read back and checked against the oracle on sampled records and sampled parents."""
    genomes, sources, _, theta = W.workload("deep_single")
    D = 14
    theta32 = float(np.float32(theta))
    pop = emr.emr_pack_population(genomes)
    path = str(tmp_path / "d14.rec")
    with emr.RecordFile(path, len(sources)) as f:
        nxt = emr.emr_discover_stream(pop, sources, D, theta32, f, chunk_positions=1 << 24)
    assert nxt == emr.emr_stream_chunks(D, 1 << 24) * len(sources)
    n, blocks = emr.read_record_file(path)
    assert n == len(sources)
    rng = np.random.default_rng(14)
    parents = {r: [] for r in range(len(sources))}
    samples = {r: [] for r in range(len(sources))}
    for r, c, p, w in blocks:
        parents[r].append(p)
        take = rng.choice(len(p), size=min(40, len(p)), replace=False)
        samples[r].append((p[take], w[take]))
    assert check_deep_against_oracle(genomes[0], sources, D, theta32, parents, samples, rng) > 0
