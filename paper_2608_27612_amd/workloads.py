"""Seeded synthetic workloads: random NEAT-style CPPN genomes and substrate source layouts.

This module only *draws* inputs. It holds none of the method's arithmetic (no grid, no CPPN
evaluation, no variance), so both the HIP path and the CPU oracle can consume what it produces
without sharing any computation.

Genome layout (one genome = a dict of numpy arrays):
  nodes 0..4      inputs with roles x1, y1, x2, y2, bias (kind 0..4)
  nodes 5..5+H-1  hidden nodes (kind 5)
  node  5+H       the output node (kind 6)
  kind  u8[n]     node role
  act   u8[n]     activation id (0 linear, 1 sigmoid, 2 tanh, 3 gaussian, 4 sine, 5 abs)
  bias  f32[n]    per-node bias (0 unless drawn, see `biases` below)
  src, dst i32[e] edge endpoints (node ids)
  w     f32[e]    edge weights
  enabled u8[e]   1 = enabled

Recipe (the paper evolves CPPNs with NEAT on XOR / visual / retina / financial tasks; no evolved
genomes are available, so seeded random DAGs of the same size classes stand in for them):
  * a random permutation fixes the topological rank of the hidden nodes;
  * candidate edges are u -> v with u an input or hidden node, v a hidden node or the output, and
    rank(u) < rank(v) (inputs rank first, the output last); there are 5(H+1) + H(H-1)/2 + H;
  * E distinct candidates are drawn uniformly without replacement, in random order;
  * weights are clip(N(0, 1), -3, 3) rounded to float32; activations are uniform over the six
    ids for hidden and output nodes; every edge is enabled;
  * biases are 0, or, when asked for (`biases=True`, test populations that exercise the bias
    terms), clip(N(0, 1), -3, 3) rounded to float32 for every hidden and output node, drawn after
    the genome's other values.
"""

from __future__ import annotations

import numpy as np

N_ACT = 6
KIND_X1, KIND_Y1, KIND_X2, KIND_Y2, KIND_BIAS, KIND_HIDDEN, KIND_OUTPUT = range(7)
DIR_OUT, DIR_IN = 0, 1


def n_candidates(h: int) -> int:
    """Number of admissible edges of a DAG with 5 inputs, h ranked hidden nodes and one output."""
    return 5 * (h + 1) + h * (h - 1) // 2 + h


def _candidate_edges(h: int, rank: np.ndarray):
    """All admissible (u, v) node-id pairs for hidden ranks `rank` (rank[k] of hidden node 5+k)."""
    out = 5 + h
    hidden = list(range(5, 5 + h))
    cand = []
    for u in range(5):
        for v in hidden + [out]:
            cand.append((u, v))
    for a in hidden:
        for b in hidden:
            if rank[a - 5] < rank[b - 5]:
                cand.append((a, b))
    for a in hidden:
        cand.append((a, out))
    assert len(cand) == n_candidates(h)
    return cand


def random_genome(rng: np.random.Generator, n_hidden: int, n_edges: int,
                  biases: bool = False) -> dict:
    """One random CPPN genome following the module recipe."""
    h = int(n_hidden)
    n = 5 + h + 1
    rank = rng.permutation(h)
    cand = _candidate_edges(h, rank)
    e = int(min(n_edges, len(cand)))
    pick = rng.choice(len(cand), size=e, replace=False)
    src = np.array([cand[k][0] for k in pick], dtype=np.int32)
    dst = np.array([cand[k][1] for k in pick], dtype=np.int32)
    w = np.clip(rng.standard_normal(e), -3.0, 3.0).astype(np.float32)
    kind = np.array([0, 1, 2, 3, 4] + [KIND_HIDDEN] * h + [KIND_OUTPUT], dtype=np.uint8)
    act = np.zeros(n, dtype=np.uint8)
    act[5:] = rng.integers(0, N_ACT, size=h + 1)
    bias = np.zeros(n, dtype=np.float32)
    if biases:
        bias[5:] = np.clip(rng.standard_normal(h + 1), -3.0, 3.0).astype(np.float32)
    return {
        "kind": kind,
        "act": act,
        "bias": bias,
        "src": src,
        "dst": dst,
        "w": w,
        "enabled": np.ones(e, dtype=np.uint8),
    }


def depends_on(genome: dict, roles) -> bool:
    """Structural test: is there an enabled path from any input with a kind in `roles` to the output?"""
    kind = genome["kind"]
    n = len(kind)
    adj = [[] for _ in range(n)]
    for s, d, en in zip(genome["src"], genome["dst"], genome["enabled"]):
        if en:
            adj[int(s)].append(int(d))
    out = int(np.nonzero(kind == KIND_OUTPUT)[0][0])
    seen = set()
    stack = [i for i in range(n) if int(kind[i]) in roles]
    while stack:
        u = stack.pop()
        if u in seen:
            continue
        seen.add(u)
        stack.extend(adj[u])
    return out in seen


def population(seed: int, n: int, h_max: int, e_max: int, biases: bool = False) -> list:
    """n genomes with H ~ U{0..h_max} and E ~ U{1..min(e_max, C(H))}, drawn in index order."""
    rng = np.random.default_rng(seed)
    pop = []
    for _ in range(n):
        h = int(rng.integers(0, h_max + 1))
        e = int(rng.integers(1, min(e_max, n_candidates(h)) + 1))
        pop.append(random_genome(rng, h, e, biases))
    return pop


def single_cppn(seed: int, n_hidden: int, n_edges: int) -> list:
    """One genome with exactly (n_hidden, n_edges), redrawn until the output depends on x2 or y2."""
    rng = np.random.default_rng(seed)
    while True:
        g = random_genome(rng, n_hidden, n_edges)
        if depends_on(g, (KIND_X2, KIND_Y2)):
            return [g]


def sources_array(points) -> np.ndarray:
    """Pack [(x, y, dir), ...] into the structured layout the C ABI reads (f32 x, f32 y, i32 dir)."""
    dt = np.dtype([("x", "<f4"), ("y", "<f4"), ("dir", "<i4")])
    arr = np.zeros(len(points), dtype=dt)
    for k, (x, y, d) in enumerate(points):
        arr[k] = (x, y, d)
    return arr


# --- substrate layouts --------------------------------------------------------------------------

def xor_sources():
    """Two inputs at (-1,-1), (1,-1), the bias input at (0,-1) (outgoing queries) and one output at
    (0, 1) (incoming queries)."""
    return sources_array([(-1.0, -1.0, DIR_OUT), (0.0, -1.0, DIR_OUT), (1.0, -1.0, DIR_OUT),
                          (0.0, 1.0, DIR_IN)])


def tabular_sources(n_inputs: int = 32):
    """n_inputs evenly spaced on y = -1 (endpoints included) plus one output at (0, 1)."""
    pts = [(-1.0 + 2.0 * k / (n_inputs - 1), -1.0, DIR_OUT) for k in range(n_inputs)]
    pts.append((0.0, 1.0, DIR_IN))
    return sources_array(pts)


# --- the named workloads --------------------------------------------------------------------------

WORKLOADS = {
    # name: (description, builder)
    "single_d5": "1 CPPN (H=8, E=20), one outgoing source at (0,-1), depth 5, theta 0.03, seed 0",
    "xor_pop1000": "1000 CPPNs (H<=20, E<=60), XOR layout (3 outgoing + 1 incoming), theta 0.03",
    "tabular_pop150": "150 CPPNs (H<=40, E<=120), 32 outgoing + 1 incoming sources, depth 6",
    "recurrent_pop100": "100 CPPNs as the XOR population, depth 10, theta 0.02",
    "deep_single": "1 CPPN (H=30, E=90), XOR layout, depth 13, theta 0.01, streamed",
}


def workload(name: str, seed: int = 0):
    """Return (genomes, sources, depth, theta) for a named workload."""
    if name == "single_d5":
        return single_cppn(seed, 8, 20), sources_array([(0.0, -1.0, DIR_OUT)]), 5, 0.03
    if name.startswith("xor_pop1000"):
        depth = int(name.split("_d")[1]) if "_d" in name else 7
        return population(seed, 1000, 20, 60), xor_sources(), depth, 0.03
    if name == "tabular_pop150":
        return population(seed, 150, 40, 120), tabular_sources(32), 6, 0.03
    if name == "recurrent_pop100":
        return population(seed, 100, 20, 60), xor_sources(), 10, 0.02
    if name == "deep_single":
        return single_cppn(seed, 30, 90), xor_sources(), 13, 0.01
    raise KeyError(name)
