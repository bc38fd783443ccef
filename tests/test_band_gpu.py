"""Band values and the band filter on the GPU (emr_band_values, emr_band_filter) against the
oracle.

The oracle evaluates the four neighbour outputs in float64 on the GPU's own float32 connection
weights (the weights the kernel compares against), so each band differs only by the neighbours'
float32 evaluation: every output within 1e-5 * max(|o|, 1) (the CPPN tolerance), and min / max /
|.| are 1-Lipschitz, so |band_gpu - band_oracle| <= 1e-5 * max(1, |w|, the neighbours' |o|) plus the
rounding of one subtraction (~1.2e-7 of the same scale): 1.1e-5 of that scale is the bound. The
filter is exact on the GPU's own band values; against the oracle's, it may differ only for
connections whose oracle band lies within that bound of theta_band."""

import numpy as np
import pytest

import oracle
from paper_2608_27612_amd import workloads as W
from tests.test_oracle_pins import INPUTS, LIN, linear_cppn, mk

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def emr():
    import torch
    assert torch.cuda.is_available()
    from paper_2608_27612_amd import emr as E
    E.lib()
    return E


def conn_to_host(c):
    n = int(c["total"])
    offs = c["pair_offset"].cpu().numpy()
    return {"pair_offset": offs, "pair_count": np.diff(offs),
            "cell": c["cell"][:n].cpu().numpy().view(np.uint32).astype(np.int64),
            "w": c["w"][:n].cpu().numpy()}


def run_band(emr, genomes, sources, D, theta, src_offsets=None, w_min=-1.0):
    pop = emr.emr_pack_population(genomes)
    res = emr.emr_discover_all(pop, sources, D, float(np.float32(theta)), src_offsets=src_offsets)
    conn = emr.emr_express(pop, sources, D, res, emr.EMR_CONN_ALL, float(np.float32(w_min)),
                           src_offsets=src_offsets)
    band = emr.emr_band_values(pop, sources, D, conn, src_offsets=src_offsets)
    return pop, conn, band


def check_band(genomes, sources, D, conn_h, band_g, src_offsets=None):
    want, nb = oracle.band_values(conn_h, genomes, sources, D, src_offsets=src_offsets,
                                  neighbours=True)
    scale = np.maximum(1.0, np.maximum(np.abs(conn_h["w"]), np.abs(nb).max(axis=1)))
    bad = np.abs(band_g - want) > 1.1e-5 * scale
    assert not bad.any(), (np.nonzero(bad)[0][:5], band_g[bad][:5], want[bad][:5])
    return want, scale


@pytest.mark.parametrize("seed,n,D,biases", [(11, 300, 6, False), (12, 200, 5, True)])
def test_band_values_match_oracle(emr, seed, n, D, biases):
    genomes = W.population(seed, n, 20, 60, biases=biases)
    sources = W.xor_sources()
    _, conn, band = run_band(emr, genomes, sources, D, 0.03)
    conn_h = conn_to_host(conn)
    assert len(conn_h["cell"]) > 1000
    check_band(genomes, sources, D, conn_h, band[:len(conn_h["cell"])].cpu().numpy())


def test_band_values_wide_programs(emr):
    """The tabular population's larger CPPNs need the wider register windows."""
    genomes = W.population(21, 40, 40, 120)
    sources = W.tabular_sources(32)
    _, conn, band = run_band(emr, genomes, sources, 5, 0.03)
    conn_h = conn_to_host(conn)
    assert len(conn_h["cell"]) > 500
    check_band(genomes, sources, 5, conn_h, band[:len(conn_h["cell"])].cpu().numpy())


def test_band_values_per_genome_sources(emr):
    """A hidden-to-hidden phase: per-genome sources at the hidden cells."""
    genomes = W.population(31, 60, 20, 60)
    sources = W.xor_sources()
    D = 5
    pop = emr.emr_pack_population(genomes)
    res = emr.emr_discover_all(pop, sources, D, float(np.float32(0.03)))
    hs = emr.emr_hidden_sources(pop, sources, D, res)
    src2, offs2 = emr.hidden_sources_to_host(hs)
    assert len(src2) > 50
    _, conn, band = run_band(emr, genomes, src2, D, 0.03, src_offsets=offs2)
    conn_h = conn_to_host(conn)
    check_band(genomes, src2, D, conn_h, band[:len(conn_h["cell"])].cpu().numpy(),
               src_offsets=offs2)


@pytest.mark.parametrize("a,b,c", [(0.75, -1.5, 0.25), (-2.0, 0.5, 0.0)])
def test_linear_band_closed_form(emr, a, b, c):
    """band = max(|a|, |b|) * side for a x2 + b y2 + c (every output exact in fp32)."""
    g = linear_cppn(a, b, c)
    sources = W.sources_array([(0.0, -1.0, 0), (0.5, 0.5, 1)])
    _, conn, band = run_band(emr, [g], sources, 6, -1.0)  # theta < 0 keeps every cell
    conn_h = conn_to_host(conn)
    offs = conn_h["pair_offset"]
    bg = band[:len(conn_h["cell"])].cpu().numpy()
    side = np.array([2.0 * 0.5 ** oracle.cell(int(F))[2] for F in conn_h["cell"]])
    out = slice(offs[0], offs[1])
    assert offs[1] - offs[0] == oracle.n_positions(6)
    np.testing.assert_array_equal(bg[out], (max(abs(a), abs(b)) * side[out]).astype(np.float32))
    # the incoming pair puts the position in (x1, y1), on which the output does not depend
    np.testing.assert_array_equal(bg[offs[1]:offs[2]], 0.0)


@pytest.mark.parametrize("theta_band", [0.0, 0.05, 0.3])
def test_band_filter(emr, theta_band):
    genomes = W.population(41, 200, 20, 60)
    sources = W.xor_sources()
    D = 6
    _, conn, band = run_band(emr, genomes, sources, D, 0.03, w_min=0.1)
    conn_h = conn_to_host(conn)
    n = len(conn_h["cell"])
    bg = band[:n].cpu().numpy()
    got = emr.emr_band_filter(conn, band, float(np.float32(theta_band)))
    got_h = conn_to_host(got)
    # exact on the GPU's own band values
    same = oracle.band_filter(conn_h, bg, np.float32(theta_band))
    np.testing.assert_array_equal(got_h["pair_offset"], same["pair_offset"])
    np.testing.assert_array_equal(got_h["cell"], same["cell"])
    np.testing.assert_array_equal(got_h["w"], same["w"])
    # against the oracle's band values: differences only within the bound of theta_band
    want, scale = check_band(genomes, sources, D, conn_h, bg)
    kept_g, kept_o = bg > np.float32(theta_band), want > theta_band
    diff = kept_g != kept_o
    assert np.all(np.abs(want[diff] - theta_band) <= 1.1e-5 * scale[diff])
    assert 0 < got_h["pair_offset"][-1] <= n


def test_band_empty_and_everything(emr):
    genomes = W.population(51, 20, 10, 30)
    sources = W.xor_sources()
    # theta above every variance: no records, no connections
    _, conn, band = run_band(emr, genomes, sources, 4, 1e30)
    assert conn["total"] == 0
    out = emr.emr_band_filter(conn, band, 0.0)
    assert out["total"] == 0
    assert np.all(out["pair_offset"].cpu().numpy() == 0)
    # theta_band below 0 keeps every connection (no band is NaN here)
    _, conn, band = run_band(emr, genomes, sources, 4, 0.0)
    out = emr.emr_band_filter(conn, band, -1.0)
    assert out["total"] == conn["total"] > 0
    np.testing.assert_array_equal(conn_to_host(out)["cell"], conn_to_host(conn)["cell"])
    with pytest.raises(emr.EmrError):
        emr.emr_band_filter(conn, band, float("nan"))
