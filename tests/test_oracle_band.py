"""Pins of the oracle's band values and band filter (ES-HyperNEAT's band threshold, which Theorem 1
names beside the variance threshold) against closed forms. No GPU needed.

Band of a connection at cell C (centre (x, y), side d): the CPPN at the same-level neighbour
centres (x -+ d, y) and (x, y -+ d); band = max(min(|w - left|, |w - right|),
min(|w - down|, |w - up|)).
 - a linear output a*x + b*y + c over the position has band max(|a|, |b|) * d at every cell (a
   wrong neighbour distance, a swapped min / max or a dropped axis fails it);
 - |x| has band 0 at the cells next to the ridge x = 0 and d elsewhere (min over both sides);
 - an output that depends on the source only, or a constant, has band 0;
 - the pair's direction decides which inputs carry the position (a swapped direction gives 0);
 - the filter is strict and keeps the order.
"""

import numpy as np
import pytest

import oracle
from paper_2608_27612_amd import workloads as W
from tests.test_oracle_pins import ABS, INPUTS, LIN, linear_cppn, mk


def all_cells(depth):
    """Every cell of the grid as one pair's connections (weights filled in later)."""
    cells = np.arange(1, oracle.n_positions(depth) + 1, dtype=np.int64)
    return {"pair_offset": np.array([0, len(cells)], np.int64), "cell": cells,
            "w": np.zeros(len(cells))}


def with_weights(conn, g, source):
    """The connections' weights: the CPPN at each cell for this source (float64)."""
    s = source
    pts = []
    for F in conn["cell"]:
        x, y, _ = oracle.cell(int(F))
        pts.append((s["x"], s["y"], x, y, 1.0) if int(s["dir"]) == 0 else (x, y, s["x"], s["y"], 1.0))
    out = dict(conn)
    out["w"] = oracle.eval_points(g, np.array(pts))
    return out


def sides(conn):
    return np.array([2.0 * 0.5 ** oracle.cell(int(F))[2] for F in conn["cell"]])


@pytest.mark.parametrize("a,b,c", [(0.75, -1.5, 0.25), (-2.0, 0.5, 0.0), (0.0, 1.25, -0.5),
                                   (1.0, 0.0, 3.0)])
@pytest.mark.parametrize("direction", [0, 1])
def test_linear_output_band_is_max_slope_times_side(a, b, c, direction):
    depth = 5
    if direction == 0:
        g = linear_cppn(a, b, c)  # a x2 + b y2 + c: the position in (x2, y2)
    else:
        g = mk(INPUTS + [6], [0] * 5 + [LIN], [(0, 5, a), (1, 5, b), (4, 5, c)])
    src = W.sources_array([(0.0, -1.0, direction)])
    conn = with_weights(all_cells(depth), g, src[0])
    band = oracle.band_values(conn, [g], src, depth)
    np.testing.assert_array_equal(band, max(abs(a), abs(b)) * sides(conn))


def test_abs_ridge_has_no_band_next_to_it():
    depth = 4
    g = mk(INPUTS + [6], [0] * 5 + [ABS], [(2, 5, 1.0)])  # |x2|
    src = W.sources_array([(0.0, -1.0, 0)])
    conn = with_weights(all_cells(depth), g, src[0])
    band = oracle.band_values(conn, [g], src, depth)
    d = sides(conn)
    x = np.array([oracle.cell(int(F))[0] for F in conn["cell"]])
    next_to_ridge = np.abs(x) == d / 2
    assert next_to_ridge.any() and (~next_to_ridge).any()
    np.testing.assert_array_equal(band[next_to_ridge], 0.0)
    np.testing.assert_array_equal(band[~next_to_ridge], d[~next_to_ridge])


def test_source_only_and_constant_outputs_have_no_band():
    depth = 4
    src = W.sources_array([(0.5, -1.0, 0)])
    for g in (mk(INPUTS + [6], [0] * 5 + [LIN], [(0, 5, 2.0), (1, 5, -1.0)]),  # x1, y1 only
              mk(INPUTS + [6], [0] * 5 + [LIN], [(4, 5, 0.7)])):
        conn = with_weights(all_cells(depth), g, src[0])
        np.testing.assert_array_equal(oracle.band_values(conn, [g], src, depth), 0.0)


def test_direction_decides_which_inputs_hold_the_position():
    depth = 3
    g = linear_cppn(1.0, 0.5, 0.0)  # depends on (x2, y2) only
    out_src = W.sources_array([(0.0, -1.0, 0)])
    in_src = W.sources_array([(0.0, -1.0, 1)])
    conn = with_weights(all_cells(depth), g, out_src[0])
    np.testing.assert_array_equal(oracle.band_values(conn, [g], out_src, depth), sides(conn))
    conn_in = with_weights(all_cells(depth), g, in_src[0])
    np.testing.assert_array_equal(oracle.band_values(conn_in, [g], in_src, depth), 0.0)


def test_neighbours_are_the_same_level_cells():
    """Inside the grid, a cell's four neighbour outputs are the outputs at the adjacent cells of
    its level (the eager grid holds them)."""
    depth = 4
    g = W.single_cppn(3, 8, 20)[0]
    src = W.sources_array([(0.0, -1.0, 0)])
    conn = with_weights(all_cells(depth), g, src[0])
    _, nb = oracle.band_values(conn, [g], src, depth, neighbours=True)
    xy = oracle.grid(depth)
    where = {(float(x), float(y)): i for i, (x, y) in enumerate(xy)}
    checked = 0
    for i, F in enumerate(conn["cell"]):
        x, y, lv = oracle.cell(int(F))
        d = 2.0 * 0.5 ** lv
        for k, (dx, dy) in enumerate([(-d, 0), (d, 0), (0, -d), (0, d)]):
            j = where.get((x + dx, y + dy))
            if j is not None and oracle.cell(j + 1)[2] == lv:
                assert nb[i, k] == conn["w"][j]
                checked += 1
    assert checked > 100


def test_filter_is_strict_and_keeps_order():
    conn = {"pair_offset": np.array([0, 3, 3, 5], np.int64), "cell": np.array([5, 6, 7, 9, 11]),
            "w": np.array([0.1, 0.2, 0.3, 0.4, 0.5])}
    band = np.array([0.3, 0.30000001, np.nan, 1.0, 0.2])
    out = oracle.band_filter(conn, band, 0.3)
    np.testing.assert_array_equal(out["pair_count"], [1, 0, 1])
    np.testing.assert_array_equal(out["pair_offset"], [0, 1, 1, 2])
    np.testing.assert_array_equal(out["cell"], [6, 9])
    np.testing.assert_array_equal(out["w"], [0.2, 0.4])
    allk = oracle.band_filter(conn, band, -1.0)
    np.testing.assert_array_equal(allk["cell"], [5, 6, 9, 11])  # NaN never passes
