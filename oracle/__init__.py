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


def hidden_sources(records, genomes_sources, sources, depth: int):
    """Sources of the hidden-to-hidden phase, from this oracle's own phase-1 output (the reading of
    'from every discovered hidden node' used for the recurrent substrate): for each genome, the
    union over its outgoing input sources of the four children 4P+1..4P+4 of every kept parent P,
    deduplicated by heap index in ascending order, each an outgoing source at its cell centre.

    records: the dict returned by discover() for `genomes_sources` genomes x `sources` (shared).
    Returns (sources array, offsets[n_genomes + 1]) in the layout of discover's src_offsets;
    the sources of a genome are ordered by heap index.
    """
    n_src = len(sources)
    xy = grid(depth)
    out_x, out_y, offs = [], [], [0]
    for g in range(genomes_sources):
        kids = []
        for j in range(n_src):
            if int(sources[j]["dir"]) != 0:
                continue
            r = g * n_src + j
            lo, hi = records["pair_offset"][r], records["pair_offset"][r + 1]
            P = records["parent"][lo:hi].astype(np.int64)
            # heap cell F sits at grid index F - 1: the children 4P+1..4P+4 at 4P..4P+3
            kids.append((4 * P[:, None] + np.arange(4)[None, :]).ravel())
        idx = np.unique(np.concatenate(kids)) if kids else np.zeros(0, np.int64)
        out_x.append(xy[idx, 0])
        out_y.append(xy[idx, 1])
        offs.append(offs[-1] + len(idx))
    src = np.zeros(offs[-1], dtype=[("x", "<f4"), ("y", "<f4"), ("dir", "<i4")])
    if offs[-1]:
        src["x"] = np.concatenate(out_x)
        src["y"] = np.concatenate(out_y)
    return src, np.array(offs, np.int32)
