"""ctypes wrapper around the C oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's CPU-baseline leg are
the only callers. The product path (the HIP library and its binding) never imports this module.
"""

from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

PARENT, CHAIN = 0, 1


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (gcc, -O2, no FP contraction, OpenMP over pairs)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math",
                               "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Genome(C.Structure):
    _fields_ = [("n_nodes", C.c_int32), ("n_edges", C.c_int32),
                ("kind", C.c_void_p), ("act", C.c_void_p), ("bias", C.c_void_p),
                ("src", C.c_void_p), ("dst", C.c_void_p), ("w", C.c_void_p),
                ("enabled", C.c_void_p)]


class _Source(C.Structure):
    _fields_ = [("x", C.c_float), ("y", C.c_float), ("dir", C.c_int32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = C.CDLL(_LIB)
        L.orc_n_positions.restype = C.c_int64
        L.orc_n_positions.argtypes = [C.c_int]
        L.orc_n_parents.restype = C.c_int64
        L.orc_n_parents.argtypes = [C.c_int]
        L.orc_cell.argtypes = [C.c_int64, C.POINTER(C.c_double), C.POINTER(C.c_double),
                               C.POINTER(C.c_int)]
        L.orc_grid.argtypes = [C.c_int, C.c_void_p]
        L.orc_act.restype = C.c_double
        L.orc_act.argtypes = [C.c_int, C.c_double]
        L.orc_topo_order.restype = C.c_int
        L.orc_topo_order.argtypes = [C.POINTER(_Genome), C.c_void_p]
        L.orc_eval_points.restype = C.c_int
        L.orc_eval_points.argtypes = [C.POINTER(_Genome), C.c_void_p, C.c_int64, C.c_void_p]
        L.orc_eval_parents.restype = C.c_int
        L.orc_eval_parents.argtypes = [C.POINTER(_Genome), C.POINTER(_Source), C.c_void_p,
                                       C.c_int64, C.c_void_p, C.c_void_p]
        L.orc_discover.restype = C.c_int64
        L.orc_discover.argtypes = [C.POINTER(_Genome), C.c_int32, C.POINTER(_Source), C.c_void_p,
                                   C.c_int32, C.c_int, C.c_double, C.c_int, C.c_void_p, C.c_void_p,
                                   C.c_void_p, C.c_void_p, C.c_int64]
        L.orc_lazy.restype = C.c_int64
        L.orc_lazy.argtypes = [C.POINTER(_Genome), C.POINTER(_Source), C.c_int, C.c_double,
                               C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64,
                               C.POINTER(C.c_int64)]
        L.orc_max_threads.restype = C.c_int
        L.orc_set_threads.restype = None
        L.orc_set_threads.argtypes = [C.c_int]
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _genome_struct(g: dict):
    """Marshal a genome dict into the oracle's struct; returns (struct, keep-alive list)."""
    keep = {
        "kind": np.ascontiguousarray(g["kind"], dtype=np.uint8),
        "act": np.ascontiguousarray(g["act"], dtype=np.uint8),
        "bias": None if g.get("bias") is None else np.ascontiguousarray(g["bias"], np.float32),
        "src": np.ascontiguousarray(g["src"], dtype=np.int32),
        "dst": np.ascontiguousarray(g["dst"], dtype=np.int32),
        "w": np.ascontiguousarray(g["w"], dtype=np.float32),
        "enabled": None if g.get("enabled") is None else np.ascontiguousarray(g["enabled"],
                                                                                np.uint8),
    }
    st = _Genome(len(keep["kind"]), len(keep["src"]), _ptr(keep["kind"]), _ptr(keep["act"]),
                 _ptr(keep["bias"]), _ptr(keep["src"]), _ptr(keep["dst"]), _ptr(keep["w"]),
                 _ptr(keep["enabled"]))
    return st, keep


def _source_struct(s):
    return _Source(float(s["x"]), float(s["y"]), int(s["dir"]))


def n_positions(depth: int) -> int:
    return int(lib().orc_n_positions(depth))


def n_parents(depth: int) -> int:
    return int(lib().orc_n_parents(depth))


def cell(F: int):
    x, y, lv = C.c_double(), C.c_double(), C.c_int()
    lib().orc_cell(F, C.byref(x), C.byref(y), C.byref(lv))
    return x.value, y.value, lv.value


def grid(depth: int) -> np.ndarray:
    xy = np.zeros((n_positions(depth), 2), dtype=np.float64)
    lib().orc_grid(depth, xy.ctypes.data)
    return xy


def act(a: int, z: float) -> float:
    return float(lib().orc_act(a, z))


def topo_order(g: dict):
    st, keep = _genome_struct(g)
    order = np.zeros(len(keep["kind"]), dtype=np.int32)
    rc = lib().orc_topo_order(C.byref(st), order.ctypes.data)
    return None if rc != 0 else order


def eval_points(g: dict, in5: np.ndarray) -> np.ndarray:
    """CPPN output at each row (x1, y1, x2, y2, bias) of in5."""
    st, keep = _genome_struct(g)
    in5 = np.ascontiguousarray(in5, dtype=np.float64).reshape(-1, 5)
    out = np.zeros(len(in5), dtype=np.float64)
    if lib().orc_eval_points(C.byref(st), in5.ctypes.data, len(in5), out.ctypes.data) != 0:
        raise ValueError("cyclic genome")
    return out


def eval_parents(g: dict, source, parents: np.ndarray):
    """(w4[n,4], var[n]) for the given parent heap indices of one (genome, source) pair."""
    st, keep = _genome_struct(g)
    src = _source_struct(source)
    parents = np.ascontiguousarray(parents, dtype=np.int64)
    w4 = np.zeros((len(parents), 4), dtype=np.float64)
    var = np.zeros(len(parents), dtype=np.float64)
    rc = lib().orc_eval_parents(C.byref(st), C.byref(src), parents.ctypes.data, len(parents),
                                w4.ctypes.data, var.ctypes.data)
    if rc != 0:
        raise ValueError("cyclic genome")
    return w4, var


def discover(genomes, sources, depth: int, theta: float, mode: int = PARENT, src_offsets=None):
    """Eager discovery over a population.

    Returns dict(pair_count[n_pairs], pair_offset[n_pairs+1], parent[n], w4[n,4], var[n]).
    `theta` is compared as given (pass the float32 value the kernel uses).
    """
    structs, keeps = [], []
    for g in genomes:
        st, k = _genome_struct(g)
        structs.append(st)
        keeps.append(k)
    garr = (_Genome * max(1, len(structs)))(*structs)
    sarr = (_Source * max(1, len(sources)))(*[_source_struct(s) for s in sources])
    if src_offsets is None:
        n_pairs = len(genomes) * len(sources)
        offs = None
    else:
        offs = np.ascontiguousarray(src_offsets, dtype=np.int32)
        n_pairs = int(offs[-1])
    counts = np.zeros(max(1, n_pairs), dtype=np.int64)
    L = lib()
    args = (garr, len(genomes), sarr, _ptr(offs), len(sources) if offs is None else 0, depth,
            float(theta), mode, counts.ctypes.data)
    total = L.orc_discover(*args, None, None, None, 0)
    if total < 0:
        raise ValueError("cyclic genome")
    parent = np.zeros(max(1, total), dtype=np.int64)
    w4 = np.zeros((max(1, total), 4), dtype=np.float64)
    var = np.zeros(max(1, total), dtype=np.float64)
    total2 = L.orc_discover(*args, parent.ctypes.data, w4.ctypes.data, var.ctypes.data, total)
    assert total2 == total
    counts = counts[:n_pairs]
    offset = np.zeros(n_pairs + 1, dtype=np.int64)
    np.cumsum(counts, out=offset[1:])
    return {"pair_count": counts, "pair_offset": offset, "parent": parent[:total],
            "w4": w4[:total], "var": var[:total]}


def lazy(g: dict, source, depth: int, theta: float):
    """ES-HyperNEAT division phase: (centres[n,2], levels[n], n_queries) of the parents whose
    children were discovered."""
    st, keep = _genome_struct(g)
    src = _source_struct(source)
    L = lib()
    nq = C.c_int64()
    n = L.orc_lazy(C.byref(st), C.byref(src), depth, float(theta), None, None, None, 0,
                   C.byref(nq))
    if n < 0:
        raise ValueError("cyclic genome")
    cx = np.zeros(max(1, n))
    cy = np.zeros(max(1, n))
    lv = np.zeros(max(1, n), dtype=np.int32)
    L.orc_lazy(C.byref(st), C.byref(src), depth, float(theta), cx.ctypes.data, cy.ctypes.data,
               lv.ctypes.data, n, C.byref(nq))
    return np.stack([cx[:n], cy[:n]], axis=1), lv[:n], int(nq.value)


def max_threads() -> int:
    return int(lib().orc_max_threads())


def set_threads(n: int) -> None:
    """Threads the oracle's later calls may use (timing harness only)."""
    lib().orc_set_threads(int(n))


def _pair_sources(sources, n_genomes: int, src_offsets=None):
    """(genome of each pair, source index of each pair) for the two pair layouts: shared sources
    (pair = g * n_shared + j) or per-genome CSR sources (pair = source index)."""
    if src_offsets is None:
        n_src = len(sources)
        pairs = np.arange(n_genomes * n_src)
        return pairs // max(n_src, 1), pairs % max(n_src, 1)
    offs = np.asarray(src_offsets, np.int64)
    pairs = np.arange(int(offs[-1]))
    return np.searchsorted(offs, pairs, side="right") - 1, pairs


def hidden_cells(records, n_genomes: int, sources, src_offsets=None, exclude=None):
    """The hidden nodes a discovery found (Section 2, Phase 1 feeding Phase 2): per genome, the
    heap indices 4P+1 .. 4P+4 of the children of every kept parent P of its outgoing pairs, as a
    set (deduplicated), minus the cells in exclude[g] (the nodes found before, when the hidden-to-
    hidden step is iterated). Returns a list of ascending int64 arrays, one per genome."""
    gen, src = _pair_sources(sources, n_genomes, src_offsets)
    out = []
    for g in range(n_genomes):
        kids = []
        for r in np.nonzero(gen == g)[0]:
            if int(sources[int(src[r])]["dir"]) != 0:
                continue
            lo, hi = records["pair_offset"][r], records["pair_offset"][r + 1]
            P = np.asarray(records["parent"][lo:hi], np.int64)
            kids.append((4 * P[:, None] + np.arange(1, 5)[None, :]).ravel())
        cells = np.unique(np.concatenate(kids)) if kids else np.zeros(0, np.int64)
        if exclude is not None and len(exclude[g]):
            cells = np.setdiff1d(cells, np.asarray(exclude[g], np.int64))
        out.append(cells)
    return out


def sources_at_cells(cells_per_genome, depth: int):
    """Outgoing sources at the centres of the given heap cells, per genome: (sources, offsets) in
    the CSR layout of discover's src_offsets."""
    xy = grid(depth)
    offs = [0]
    parts = []
    for cells in cells_per_genome:
        parts.append(np.asarray(cells, np.int64))
        offs.append(offs[-1] + len(cells))
    src = np.zeros(offs[-1], dtype=[("x", "<f4"), ("y", "<f4"), ("dir", "<i4")])
    if offs[-1]:
        idx = np.concatenate(parts) - 1  # heap cell F sits at grid index F - 1
        src["x"] = xy[idx, 0]
        src["y"] = xy[idx, 1]
    return src, np.array(offs, np.int32)


def hidden_sources(records, genomes_sources, sources, depth: int):
    """Sources of the hidden-to-hidden phase, from this oracle's own phase-1 output (the reading of
    'from every discovered hidden node' used for the recurrent substrate): for each genome, the
    union over its outgoing input sources of the four children 4P+1..4P+4 of every kept parent P,
    deduplicated by heap index in ascending order, each an outgoing source at its cell centre.

    records: the dict returned by discover() for `genomes_sources` genomes x `sources` (shared).
    Returns (sources array, offsets[n_genomes + 1]) in the layout of discover's src_offsets;
    the sources of a genome are ordered by heap index.
    """
    return sources_at_cells(hidden_cells(records, genomes_sources, sources), depth)


def chain_filter(records, depth: int):
    """Eq. 2 read literally on a parent-rule result: a kept parent stays only if its own parent
    was kept by the same rule, recursively up to the root (active at depth 0, then active[d] =
    active[d-1] of the parent and its variance test). Records are per pair in ascending heap
    order, i.e. level by level, so one pass in that order decides every cell after its parent.
    Returns a records dict of the same form (pair_count, pair_offset, parent, w4, var)."""
    counts = np.asarray(records["pair_count"], np.int64)
    offs = np.asarray(records["pair_offset"], np.int64)
    keep = np.zeros(int(offs[-1]), bool)
    for r in range(len(counts)):
        kept = set()
        for i in range(int(offs[r]), int(offs[r + 1])):
            P = int(records["parent"][i])
            if P == 0 or (P - 1) // 4 in kept:
                kept.add(P)
                keep[i] = True
    new_counts = np.array([int(np.sum(keep[offs[r]:offs[r + 1]])) for r in range(len(counts))],
                          np.int64)
    new_offs = np.zeros(len(counts) + 1, np.int64)
    np.cumsum(new_counts, out=new_offs[1:])
    out = {"pair_count": new_counts, "pair_offset": new_offs,
           "parent": np.asarray(records["parent"])[keep], "w4": np.asarray(records["w4"])[keep]}
    if "var" in records:
        out["var"] = np.asarray(records["var"])[keep]
    return out


# Connection types (Section 4, the connection type taxonomy): from the source and target node's y
# coordinates; a self-loop is a connection from a node to itself.
CONN_FORWARD, CONN_BACKWARD, CONN_LATERAL, CONN_SELF = 1, 2, 4, 8


def connection_type(sx, sy, tx, ty) -> int:
    """Self when source and target are the same node (same position), else forward (y_s < y_t),
    backward (y_s > y_t) or lateral (y_s = y_t)."""
    if sx == tx and sy == ty:
        return CONN_SELF
    if sy < ty:
        return CONN_FORWARD
    if sy > ty:
        return CONN_BACKWARD
    return CONN_LATERAL


def express(records, sources, depth: int, type_mask: int, w_min: float, n_genomes=None,
            src_offsets=None):
    """The connections a discovery expresses: every child C = 4P+k (k = 1..4) of a kept parent P
    of pair (genome, source s) is a connection with the CPPN output at C as its weight. An outgoing
    source s connects s -> C, an incoming one C -> s (Section 3.1: the query direction). A
    connection is expressed when its type (Section 4) is in type_mask and its weight magnitude
    exceeds w_min (Section 3.3: the weight magnitude filter, 0.1 in the paper). The weights are
    the records' values as given (pass the float32 outputs the kernels produced to compare the
    filters exactly). Returns dict(pair_count, pair_offset, cell (heap index of C), w)."""
    offs = np.asarray(records["pair_offset"], np.int64)
    n_pairs = len(offs) - 1
    if n_genomes is None:
        n_genomes = n_pairs // max(len(sources), 1) if src_offsets is None else len(src_offsets) - 1
    _, src = _pair_sources(sources, n_genomes, src_offsets)
    xy = grid(depth)
    counts = np.zeros(n_pairs, np.int64)
    cells, ws = [], []
    for r in range(n_pairs):
        s = sources[int(src[r])]
        sx, sy, d = float(s["x"]), float(s["y"]), int(s["dir"])
        for i in range(int(offs[r]), int(offs[r + 1])):
            P = int(records["parent"][i])
            for k in range(4):
                C = 4 * P + 1 + k
                cx, cy = float(xy[C - 1, 0]), float(xy[C - 1, 1])
                t = connection_type(sx, sy, cx, cy) if d == 0 else connection_type(cx, cy, sx, sy)
                w = float(records["w4"][i][k])
                if (t & type_mask) and abs(w) > w_min:
                    cells.append(C)
                    ws.append(w)
                    counts[r] += 1
    pair_offset = np.zeros(n_pairs + 1, np.int64)
    np.cumsum(counts, out=pair_offset[1:])
    return {"pair_count": counts, "pair_offset": pair_offset,
            "cell": np.array(cells, np.int64), "w": np.array(ws, np.float64)}


def band_values(conn, genomes, sources, depth: int, src_offsets=None, neighbours=False):
    """ES-HyperNEAT's band value of every expressed connection. Theorem 1 names a band threshold
    beside the variance threshold and leaves its definition to ES-HyperNEAT, whose pruning step
    keeps a point only when its weight stands out from its neighbours' on both sides along x or
    along y. Here, for connection (pair r, cell C, weight w): C is the centre (x, y) of a level-l
    cell of side d = 2^(1 - l) (its parent's half-width), and the pair's CPPN is queried, in the
    pair's direction, at the four same-level neighbour centres (x - d, y), (x + d, y), (x, y - d),
    (x, y + d); with dl, dr, dd, du the absolute differences between w and those four outputs,
    band = max(min(dl, dr), min(dd, du)) (min and max ignore a NaN operand). conn: the CSR layout
    of express() (pair_offset, cell, w; w as given). float64. Returns the band per connection, and
    with neighbours=True also the [n, 4] neighbour outputs (left, right, down, up)."""
    offs = np.asarray(conn["pair_offset"], np.int64)
    n_pairs = len(offs) - 1
    n_genomes = len(genomes)
    gen, src = _pair_sources(sources, n_genomes, src_offsets)
    assert len(gen) == n_pairs
    n = int(offs[-1])
    band = np.zeros(n, np.float64)
    nb = np.zeros((n, 4), np.float64)
    steps = np.array([[-1.0, 0.0], [1.0, 0.0], [0.0, -1.0], [0.0, 1.0]])
    for r in range(n_pairs):
        lo, hi = int(offs[r]), int(offs[r + 1])
        if hi == lo:
            continue
        s = sources[int(src[r])]
        sx, sy, d = float(s["x"]), float(s["y"]), int(s["dir"])
        pts = []
        for i in range(lo, hi):
            x, y, lv = cell(int(conn["cell"][i]))
            side = 2.0 * 0.5 ** lv
            for k in range(4):
                px, py = x + side * steps[k, 0], y + side * steps[k, 1]
                pts.append((sx, sy, px, py, 1.0) if d == 0 else (px, py, sx, sy, 1.0))
        vals = eval_points(genomes[int(gen[r])], np.array(pts)).reshape(-1, 4)
        w = np.asarray(conn["w"][lo:hi], np.float64)[:, None]
        dist = np.abs(w - vals)
        band[lo:hi] = np.fmax(np.fmin(dist[:, 0], dist[:, 1]), np.fmin(dist[:, 2], dist[:, 3]))
        nb[lo:hi] = vals
    return (band, nb) if neighbours else band


def band_filter(conn, band, theta_band: float):
    """The connections whose band exceeds theta_band (strict; a NaN band never does), in their
    order: dict(pair_count, pair_offset, cell, w) like express()."""
    offs = np.asarray(conn["pair_offset"], np.int64)
    keep = np.asarray(band) > theta_band
    counts = np.array([int(keep[offs[r]:offs[r + 1]].sum()) for r in range(len(offs) - 1)],
                      np.int64)
    pair_offset = np.zeros(len(offs), np.int64)
    np.cumsum(counts, out=pair_offset[1:])
    return {"pair_count": counts, "pair_offset": pair_offset,
            "cell": np.asarray(conn["cell"])[keep], "w": np.asarray(conn["w"])[keep]}


# ----------------------------------------------------------------------------- networks
# The networks the experiments evaluate (Section 5: XOR over its four input patterns), built from
# the discovered substrate. The paper does not spell out this construction; the oracle follows
# ES-HyperNEAT's: substrate nodes plus the hidden nodes of Phase 1 and the hidden-to-hidden
# phase, connected by the expressed connections, then cut down to the nodes that lie on a path
# from an input to an output, and activated synchronously for a fixed number of steps with the
# sigmoid on every non-input node.

def sigmoid(z):
    """1 / (1 + e^-z), elementwise, float64."""
    z = np.asarray(z, np.float64)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = ez / (1.0 + ez)
    return out


def network_phases(genomes, substrate, depth: int, theta: float, iterations: int):
    """Phase 1 on the substrate sources, then up to `iterations` hidden-to-hidden phases, each
    querying the hidden nodes the previous phase found (and only those) as outgoing sources; it
    stops early when no genome found a new node. Returns (phases, known): phases[k] =
    dict(records, sources, src_offsets, cells) (cells: per genome the hidden cells queried in
    phase k, None for the substrate phase), known[g] = every hidden cell of genome g, ascending
    (the children of the kept parents of every outgoing pair of every phase)."""
    G = len(genomes)
    rec = discover(genomes, substrate, depth, theta)
    phases = [{"records": rec, "sources": substrate, "src_offsets": None, "cells": None}]
    new = hidden_cells(rec, G, substrate)
    known = [c.copy() for c in new]
    for _ in range(iterations):
        if not any(len(c) for c in new):
            break
        src, offs = sources_at_cells(new, depth)
        rec = discover(genomes, src, depth, theta, src_offsets=offs)
        phases.append({"records": rec, "sources": src, "src_offsets": offs, "cells": new})
        new = hidden_cells(rec, G, src, offs, exclude=known)
        known = [np.union1d(k, n) for k, n in zip(known, new)]
    return phases, known


def reachable(n_nodes: int, edges, seeds):
    """Boolean mask of the nodes reachable from `seeds` along the directed (u, v) edges."""
    adj = [[] for _ in range(n_nodes)]
    for u, v in edges:
        adj[u].append(v)
    seen = np.zeros(n_nodes, bool)
    stack = list(seeds)
    for s in stack:
        seen[s] = True
    while stack:
        u = stack.pop()
        for v in adj[u]:
            if not seen[v]:
                seen[v] = True
                stack.append(v)
    return seen


def prune(n_nodes: int, inputs, outputs, edges):
    """(node mask, edge mask): a node stays when it is an input or an output, or when it can be
    reached from an input and can reach an output; an edge u -> v stays when u can be reached from
    an input and v can reach an output (so it lies on an input-to-output path)."""
    fwd = reachable(n_nodes, edges, inputs)
    bwd = reachable(n_nodes, [(v, u) for u, v in edges], outputs)
    node = fwd & bwd
    node[list(inputs)] = True
    node[list(outputs)] = True
    emask = np.array([bool(fwd[u] and bwd[v]) for u, v in edges], bool)
    return node, emask


def assemble(n_genomes: int, substrate, depth: int, phases, known, type_mask: int, w_min: float):
    """The pruned networks. Per genome, before pruning: node j < n_sub is substrate source j, node
    n_sub + i is the hidden cell known[g][i]; every connection the phases express (express(), with
    type_mask and w_min) is an edge between the source's node (a substrate node in phase 0, the
    queried hidden cell's node later) and the grid cell's node, in the connection's direction; a
    connection whose grid cell is not a hidden node (an incoming source's cell that no outgoing
    pair reached) is dropped. Then prune(). Returns per genome dict(cells: the kept hidden cells
    ascending (node n_sub + i is cells[i]), src, dst, w: the kept edges with the kept nodes'
    numbers, in the order phase, pair, cell)."""
    n_sub = len(substrate)
    inputs = [j for j in range(n_sub) if int(substrate[j]["dir"]) == 0]
    outputs = [j for j in range(n_sub) if int(substrate[j]["dir"]) != 0]
    raw = [[] for _ in range(n_genomes)]
    for ph in phases:
        offs = ph["src_offsets"]
        conn = express(ph["records"], ph["sources"], depth, type_mask, w_min, n_genomes, offs)
        gen, src = _pair_sources(ph["sources"], n_genomes, offs)
        for r in range(len(conn["pair_count"])):
            g, j = int(gen[r]), int(src[r])
            if ph["cells"] is None:
                s_node, d = j, int(substrate[j]["dir"])
            else:
                cell = int(ph["cells"][g][j - int(offs[g])])
                s_node, d = n_sub + int(np.searchsorted(known[g], cell)), 0
            for i in range(int(conn["pair_offset"][r]), int(conn["pair_offset"][r + 1])):
                c = int(conn["cell"][i])
                pos = int(np.searchsorted(known[g], c))
                if pos == len(known[g]) or int(known[g][pos]) != c:
                    continue
                c_node = n_sub + pos
                raw[g].append((s_node, c_node, float(conn["w"][i])) if d == 0
                              else (c_node, s_node, float(conn["w"][i])))
    nets = []
    for g in range(n_genomes):
        n = n_sub + len(known[g])
        edges = [(u, v) for u, v, _ in raw[g]]
        node, emask = prune(n, inputs, outputs, edges)
        new_id = np.cumsum(node) - 1
        e = [(int(new_id[u]), int(new_id[v]), w) for (u, v, w), k in zip(raw[g], emask) if k]
        nets.append({"cells": np.asarray(known[g], np.int64)[node[n_sub:]],
                     "src": np.array([x[0] for x in e], np.int64),
                     "dst": np.array([x[1] for x in e], np.int64),
                     "w": np.array([x[2] for x in e], np.float64)})
    return nets


def build_networks(genomes, substrate, depth: int, theta: float, type_mask: int, w_min: float,
                   iterations: int):
    """network_phases() then assemble(), all from this oracle's own float64 discovery."""
    phases, known = network_phases(genomes, substrate, depth, theta, iterations)
    return assemble(len(genomes), substrate, depth, phases, known, type_mask, w_min)


def activate(net, substrate, inputs, steps: int):
    """Outputs [n_patterns, n_outputs] of one network after `steps` synchronous updates: the input
    nodes (the outgoing substrate sources, in order) hold the pattern's values throughout, every
    other node starts at 0 and takes sigmoid(sum of w * the source node's previous value) at each
    step."""
    n_sub = len(substrate)
    inputs = np.atleast_2d(np.asarray(inputs, np.float64))
    ins = [j for j in range(n_sub) if int(substrate[j]["dir"]) == 0]
    outs = [j for j in range(n_sub) if int(substrate[j]["dir"]) != 0]
    n = n_sub + len(net["cells"])
    s = np.zeros((len(inputs), n))
    s[:, ins] = inputs
    for _ in range(steps):
        z = np.zeros_like(s)
        for u, v, w in zip(net["src"], net["dst"], net["w"]):
            z[:, v] += w * s[:, u]
        s = sigmoid(z)
        s[:, ins] = inputs
    return s[:, outs]


XOR_TARGETS = np.array([0.0, 1.0, 1.0, 0.0])


def xor_patterns(n_inputs: int, bias_input=None) -> np.ndarray:
    """The four XOR patterns (a, b) = (0,0), (0,1), (1,0), (1,1) as input values in input order:
    a and b are the first and second input other than `bias_input` (the bias input, held at 1;
    None when there is none)."""
    ab = np.array([[0, 0], [0, 1], [1, 0], [1, 1]], np.float64)
    if n_inputs != 2 + (bias_input is not None):
        raise ValueError("XOR needs inputs a, b and at most one bias input")
    out = np.ones((4, n_inputs))
    cols = [j for j in range(n_inputs) if j != bias_input]
    out[:, cols] = ab
    return out


def xor_fitness(net, substrate, steps: int, bias_input=None) -> float:
    """1 - the mean squared error of the single output over the four XOR patterns."""
    n_in = sum(1 for s in substrate if int(s["dir"]) == 0)
    out = activate(net, substrate, xor_patterns(n_in, bias_input), steps)
    if out.shape[1] != 1:
        raise ValueError("XOR needs one output")
    return float(1.0 - np.mean((out[:, 0] - XOR_TARGETS) ** 2))
