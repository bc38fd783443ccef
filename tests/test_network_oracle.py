"""Pins of the oracle's network construction and activation (no GPU): a substrate worked out by
hand from a linear CPPN at depth 1, pruning against reachability from a graph library, activation
against closed forms, a topological-order evaluation of acyclic networks and the fixed point of
recurrent ones, and the XOR fitness on known networks. Planted mistakes show the pins would catch
a wrong step."""

import numpy as np
import pytest
from scipy import optimize, special
from scipy.sparse import csr_matrix
from scipy.sparse.csgraph import shortest_path

import oracle
from paper_2608_27612_amd import workloads as W

LIN = 0
F, B, L, S = oracle.CONN_FORWARD, oracle.CONN_BACKWARD, oracle.CONN_LATERAL, oracle.CONN_SELF


def mk(edges, n_hidden=0, act=LIN):
    """CPPN with inputs x1 y1 x2 y2 bias (nodes 0..4), an output (node 5 + n_hidden) and the given
    (src, dst, w) edges."""
    kinds = [0, 1, 2, 3, 4] + [5] * n_hidden + [6]
    n = len(kinds)
    return {"kind": np.array(kinds, np.uint8), "act": np.array([0] * (n - 1) + [act], np.uint8),
            "bias": np.zeros(n, np.float32),
            "src": np.array([e[0] for e in edges], np.int32),
            "dst": np.array([e[1] for e in edges], np.int32),
            "w": np.array([e[2] for e in edges], np.float32),
            "enabled": np.ones(len(edges), np.uint8)}


# out = x1 + y2: an outgoing source s gives cell C the weight s_x + C_y; an incoming source o
# (the query puts the cell in (x1, y1)) gives C -> o the weight C_x + o_y.
HAND = mk([(0, 5, 1.0), (3, 5, 1.0)])
# Depth 1: the four level-1 cells, heap 1..4 at (-1/2,-1/2), (1/2,-1/2), (-1/2,1/2), (1/2,1/2).
# The root's children vary by 1/4 in both x and y (variance 1/4 for every source): kept.


def hand_build(type_mask, w_min, iterations):
    return oracle.build_networks([HAND], W.xor_sources(), 1, 0.1, type_mask, w_min, iterations)[0]


def edge_set(net):
    return {(int(u), int(v)): float(w) for u, v, w in zip(net["src"], net["dst"], net["w"])}


def test_hand_substrate_without_pruning():
    """Forward connections, w_min 0.1, one hidden-to-hidden phase. Inputs a (-1,-1), bias (0,-1),
    b (1,-1) are nodes 0..2, the output (0,1) node 3, cells 1..4 nodes 4..7. Every input
    reaches every cell (a: -1 + C_y, b: 1 + C_y, bias: C_y, all |w| >= 1/2); every cell reaches
    the output (C_x + 1); of the hidden-to-hidden connections only bottom -> top rows are forward,
    and from cell 1 (x = -1/2) they weigh 0 and fail the filter, from cell 2 they weigh 1."""
    net = hand_build(F, 0.1, 1)
    assert list(net["cells"]) == [1, 2, 3, 4]
    want = {}
    for j, (sx, sy) in enumerate([(-1, -1), (0, -1), (1, -1)]):
        for k, (cx, cy) in enumerate([(-.5, -.5), (.5, -.5), (-.5, .5), (.5, .5)]):
            want[(j, 4 + k)] = sx + cy
    for k, (cx, cy) in enumerate([(-.5, -.5), (.5, -.5), (-.5, .5), (.5, .5)]):
        want[(4 + k, 3)] = cx + 1
    want[(5, 6)] = 1.0
    want[(5, 7)] = 1.0
    assert edge_set(net) == want


def test_hand_substrate_types_and_self_loops():
    """All four types: the hidden-to-hidden phase adds, from each cell h to each cell C,
    h_x + C_y when it is nonzero (|w| > 0.1), self-loops included (cell 1: -1, cell 4: 1;
    cells 2 and 3 weigh 0)."""
    net = hand_build(F | B | L | S, 0.1, 1)
    cells = [(-.5, -.5), (.5, -.5), (-.5, .5), (.5, .5)]
    hh = {(4 + i, 4 + k): hx + cy for i, (hx, hy) in enumerate(cells)
          for k, (cx, cy) in enumerate(cells) if abs(hx + cy) > 0.1}
    got = {k: v for k, v in edge_set(net).items() if k[0] >= 4 and k[1] >= 4}
    assert got == hh
    assert got[(4, 4)] == -1.0 and got[(7, 7)] == 1.0 and (5, 5) not in got and (6, 6) not in got


def test_hand_substrate_pruned_and_activated():
    """w_min 1: only a -> cells 1, 2 (-3/2), b -> cells 3, 4 (3/2) and cells 2, 4 -> output
    (3/2) survive the filter (hidden-to-hidden weights are at most 1). Cell 1 cannot reach the
    output and cell 3 neither: both are cut, leaving cells 2, 4 as nodes 4, 5. The output after
    two steps is sigmoid(3/2 sigmoid(-3/2 a) + 3/2 sigmoid(3/2 b)); after one step 1/2."""
    net = hand_build(F, 1.0, 1)
    assert list(net["cells"]) == [2, 4]
    assert edge_set(net) == {(0, 4): -1.5, (2, 5): 1.5, (4, 3): 1.5, (5, 3): 1.5}
    subs = W.xor_sources()
    pats = oracle.xor_patterns(3, bias_input=1)
    np.testing.assert_array_equal(pats, [[0, 1, 0], [0, 1, 1], [1, 1, 0], [1, 1, 1]])
    a, b = pats[:, 0], pats[:, 2]
    want = special.expit(1.5 * special.expit(-1.5 * a) + 1.5 * special.expit(1.5 * b))
    np.testing.assert_allclose(oracle.activate(net, subs, pats, 2)[:, 0], want, rtol=0, atol=1e-15)
    np.testing.assert_allclose(oracle.activate(net, subs, pats, 7)[:, 0], want, rtol=0, atol=1e-15)
    assert np.all(oracle.activate(net, subs, pats, 1) == 0.5)
    assert np.all(oracle.activate(net, subs, pats, 0) == 0.0)
    fit = 1 - np.mean((want - np.array([0, 1, 1, 0])) ** 2)
    assert abs(oracle.xor_fitness(net, subs, 2, bias_input=1) - fit) < 1e-15


def test_hand_substrate_feedforward_has_no_hidden_to_hidden():
    """No hidden-to-hidden phase (the feedforward configuration)."""
    net = hand_build(F, 0.1, 0)
    assert not any(u >= 4 and v >= 4 for u, v in edge_set(net))
    assert len(edge_set(net)) == 12 + 4


def random_graph(rng, n, n_in, n_out, p):
    """Edges among n nodes (no edges into inputs or out of outputs)."""
    e = []
    for u in range(n):
        if n_in <= u < n_in + n_out:
            continue
        for v in range(n_in, n):
            if rng.random() < p:
                e.append((u, v))
    return e


@pytest.mark.parametrize("seed", range(8))
def test_prune_against_graph_library(seed):
    rng = np.random.default_rng(seed)
    n, n_in, n_out = 30, 3, 2
    edges = random_graph(rng, n, n_in, n_out, 0.06)
    node, emask = oracle.prune(n, range(n_in), range(n_in, n_in + n_out), edges)
    A = np.zeros((n, n))
    for u, v in edges:
        A[u, v] = 1
    D = shortest_path(csr_matrix(A), directed=True, unweighted=True)
    from_in = np.isfinite(D[:n_in]).any(axis=0)
    to_out = np.isfinite(D[:, n_in:n_in + n_out]).any(axis=1)
    want = from_in & to_out
    want[:n_in + n_out] = True
    np.testing.assert_array_equal(node, want)
    np.testing.assert_array_equal(emask, [bool(from_in[u] and to_out[v]) for u, v in edges])


def feedforward(n, n_in, src, dst, w, x):
    """Textbook feedforward pass of a DAG whose edges run from lower to higher node numbers."""
    s = np.zeros(n)
    s[:n_in] = x
    for v in range(n_in, n):
        m = dst == v
        s[v] = special.expit(np.sum(w[m] * s[src[m]]))
    return s


@pytest.mark.parametrize("seed", range(6))
def test_acyclic_activation_equals_topological_evaluation(seed):
    """For a DAG, as many synchronous steps as its longest chain of non-input nodes reach the
    feedforward values, which later steps keep."""
    rng = np.random.default_rng(100 + seed)
    n, n_in = 12, 2
    pairs = [(u, v) for v in range(n_in, n) for u in range(v) if rng.random() < 0.35]
    src = np.array([u for u, _ in pairs])
    dst = np.array([v for _, v in pairs])
    w = rng.normal(0, 2, len(pairs))
    depth = np.zeros(n, int)  # steps until a node holds its final value
    depth[n_in:] = 1  # a node without inputs takes sigmoid(0) at the first step
    for u, v in sorted(pairs, key=lambda e: e[1]):
        depth[v] = max(depth[v], depth[u] + 1)
    # substrate: n_in inputs, then the last node as the only output; others hidden
    subs = W.sources_array([(0, -1, 0)] * n_in + [(0, 1, 1)])
    perm = list(range(n_in)) + [v + 1 for v in range(n_in, n - 1)] + [n_in]  # node -> number
    net = {"cells": np.arange(n - n_in - 1), "src": np.array([perm[u] for u in src]),
           "dst": np.array([perm[v] for v in dst]), "w": w}
    x = rng.normal(size=(3, n_in))
    want = np.array([feedforward(n, n_in, src, dst, w, xi)[n - 1] for xi in x])
    L_ = int(depth.max())
    np.testing.assert_allclose(oracle.activate(net, subs, x, L_)[:, 0], want, atol=1e-14)
    np.testing.assert_allclose(oracle.activate(net, subs, x, L_ + 5)[:, 0], want, atol=1e-14)


def test_recurrent_activation_converges_to_the_fixed_point():
    """With small weights the synchronous update is a contraction: many steps reach the fixed
    point s = sigmoid(W s + U x), found here by a root finder."""
    rng = np.random.default_rng(7)
    n_h = 6
    Wh = rng.normal(0, 0.5, (n_h, n_h))
    U = rng.normal(0, 1.0, (n_h, 2))
    wo = rng.normal(0, 1.0, n_h)
    x = np.array([0.3, -0.8])
    # network numbering: inputs 0, 1; output 2; hidden 3..8
    src, dst, w = [], [], []
    for i in range(n_h):
        for j in range(2):
            src.append(j), dst.append(3 + i), w.append(U[i, j])
        for k in range(n_h):
            src.append(3 + k), dst.append(3 + i), w.append(Wh[i, k])
        src.append(3 + i), dst.append(2), w.append(wo[i])
    net = {"cells": np.arange(n_h), "src": np.array(src), "dst": np.array(dst), "w": np.array(w)}
    subs = W.sources_array([(-1, -1, 0), (1, -1, 0), (0, 1, 1)])
    h = optimize.fsolve(lambda h: h - special.expit(Wh @ h + U @ x), np.full(n_h, 0.5),
                        xtol=1e-14)
    want = special.expit(wo @ h)
    got = oracle.activate(net, subs, x[None, :], 200)[0, 0]
    assert abs(got - want) < 1e-10


def test_xor_fitness_known_networks():
    subs = W.xor_sources()
    empty = {"cells": np.zeros(0, np.int64), "src": np.zeros(0, np.int64),
             "dst": np.zeros(0, np.int64), "w": np.zeros(0)}
    # no edges: the output is sigmoid(0) = 1/2 for every pattern
    assert oracle.xor_fitness(empty, subs, 3, bias_input=1) == 0.75
    assert oracle.xor_fitness(empty, subs, 0, bias_input=1) == 0.5  # output 0 before any step
    # the textbook two-hidden-unit XOR: h1 = OR, h2 = NAND, out = AND; inputs a = node 0,
    # bias = node 1, b = node 2
    k = 20.0
    edges = [(0, 4, k), (2, 4, k), (1, 4, -k / 2), (0, 5, -k), (2, 5, -k), (1, 5, 1.5 * k),
             (4, 3, k), (5, 3, k), (1, 3, -1.5 * k)]
    net = {"cells": np.array([1, 2]), "src": np.array([e[0] for e in edges]),
           "dst": np.array([e[1] for e in edges]), "w": np.array([e[2] for e in edges])}
    f = oracle.xor_fitness(net, subs, 2, bias_input=1)
    assert f > 0.9999
    pats = oracle.xor_patterns(3, bias_input=1)
    h1 = special.expit(k * pats[:, 0] + k * pats[:, 2] - k / 2)
    h2 = special.expit(-k * pats[:, 0] - k * pats[:, 2] + 1.5 * k)
    out = special.expit(k * h1 + k * h2 - 1.5 * k)
    assert abs(f - (1 - np.mean((out - [0, 1, 1, 0]) ** 2))) < 1e-15
    with pytest.raises(ValueError):
        oracle.xor_fitness(empty, W.sources_array([(0, -1, 0), (1, -1, 0), (0, 1, 1),
                                                   (1, 1, 1)]), 1)
    with pytest.raises(ValueError):
        oracle.xor_fitness(empty, subs, 1)  # three inputs but no bias named


def test_assembled_population_invariants():
    """A random population with two hidden-to-hidden phases: the nodes are hidden cells the phases
    found; every kept edge lies on an input-to-output path of the kept graph (graph library);
    every edge is an expressed connection of its phase between two nodes."""
    genomes = W.population(510, 12, 16, 48)
    subs = W.xor_sources()
    D, theta, mask, w_min = 5, 0.02, F | B | L | S, 0.1
    phases, known = oracle.network_phases(genomes, subs, D, theta, 2)
    assert len(phases) >= 2
    nets = oracle.assemble(len(genomes), subs, D, phases, known, mask, w_min)
    for g, net in enumerate(nets):
        assert set(net["cells"]) <= set(known[g])
        n = 4 + len(net["cells"])
        if len(net["src"]) == 0:
            continue
        A = csr_matrix((np.ones(len(net["src"])), (net["src"], net["dst"])), shape=(n, n))
        Dm = shortest_path(A, directed=True, unweighted=True)
        from_in = np.isfinite(Dm[:3]).any(axis=0)
        to_out = np.isfinite(Dm[:, 3])
        assert np.all(from_in[net["src"]] & to_out[net["dst"]])
        assert np.all((from_in & to_out)[4:])  # every kept hidden node is on a path
        assert np.all(np.abs(net["w"]) > w_min)
        assert not np.any(net["dst"] < 3)  # nothing flows into an input


def test_planted_mistakes_fail_the_pins(monkeypatch):
    """A wrong step in the oracle fails a pin: pruning that keeps every node, an activation
    that lets inputs float, and a transposed edge direction for incoming sources."""
    net = hand_build(F, 1.0, 1)
    assert list(net["cells"]) == [2, 4]
    real_prune = oracle.prune
    monkeypatch.setattr(oracle, "prune", lambda n, i, o, e: (np.ones(n, bool),
                                                             np.ones(len(e), bool)))
    assert list(hand_build(F, 1.0, 1)["cells"]) != [2, 4]
    monkeypatch.setattr(oracle, "prune", real_prune)
    real_sig = oracle.sigmoid
    monkeypatch.setattr(oracle, "sigmoid", lambda z: np.tanh(np.asarray(z)))
    pats = oracle.xor_patterns(3, bias_input=1)
    want = special.expit(1.5 * special.expit(-1.5 * pats[:, 0]) + 1.5 * special.expit(1.5 * pats[:, 2]))
    assert oracle.xor_fitness(net, W.xor_sources(), 2, bias_input=1) != pytest.approx(
        1 - np.mean((want - [0, 1, 1, 0]) ** 2), abs=1e-6)
    monkeypatch.setattr(oracle, "sigmoid", real_sig)
    subs = W.xor_sources()
    flipped = subs.copy()
    flipped["dir"][3] = 0  # the output treated as an outgoing source
    assert oracle.build_networks([HAND], flipped, 1, 0.1, F, 1.0, 1)[0]["cells"].tolist() \
        != [2, 4]
