"""Python binding of include/emr.h (ctypes; argument marshalling only).

Every step of discovery runs in libemr.so's HIP kernels. PyTorch provides device memory and the
current HIP stream; nothing here computes any part of the method. If the library has not been
built the first call raises, so a missing extension can never fall back to another code path.
"""

from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libemr.so")

EMR_OK, EMR_E_INVAL, EMR_E_CYCLE, EMR_E_LIMIT, EMR_E_NOMEM, EMR_E_CAPACITY, EMR_E_DEVICE, \
    EMR_E_ABORTED, EMR_E_IO = 0, -1, -2, -3, -4, -5, -6, -7, -8
EMR_DIR_OUT, EMR_DIR_IN = 0, 1
EMR_MAX_DEPTH = 15

# Every function include/emr.h declares.
ABI_FUNCTIONS = [
    "emr_last_error", "emr_version", "emr_grid_count", "emr_build_grids", "emr_pack_population",
    "emr_free_population", "emr_population_info", "emr_workspace_bytes", "emr_discover",
    "emr_result_check", "emr_eval_raw", "emr_discover_cost", "emr_profile_enable",
    "emr_profile_read", "emr_stream_chunks", "emr_discover_stream", "emr_pack_population_flat",
    "emr_set_jit", "emr_jit_info", "emr_eval_raw_noalloc", "emr_call_check", "emr_cell_words",
    "emr_hidden_workspace_bytes", "emr_hidden_sources", "emr_express_workspace_bytes",
    "emr_express", "emr_chain_workspace_bytes", "emr_chain_filter", "emr_band_workspace_bytes",
    "emr_band_values", "emr_band_filter", "emr_record_file_open",
    "emr_record_file_sink", "emr_record_file_close", "emr_build_networks", "emr_networks_info",
    "emr_networks_phase", "emr_activate", "emr_xor_fitness", "emr_free_networks",
    "emr_copy_to_host",
]
EMR_CONN_FORWARD, EMR_CONN_BACKWARD, EMR_CONN_LATERAL, EMR_CONN_SELF, EMR_CONN_ALL = 1, 2, 4, 8, 15
EMR_NOALLOC_SCRATCH_BYTES = 32 << 20
EMR_JIT_OFF, EMR_JIT_AUTO, EMR_JIT_ALWAYS = 0, 1, 2


class EmrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("emr status %d: %s" % (status, message))
        self.status = status


class emr_genome(C.Structure):
    _fields_ = [("n_nodes", C.c_int32), ("n_edges", C.c_int32), ("kind", C.c_void_p),
                ("act", C.c_void_p), ("bias", C.c_void_p), ("src", C.c_void_p),
                ("dst", C.c_void_p), ("w", C.c_void_p), ("enabled", C.c_void_p)]


class emr_source(C.Structure):
    _fields_ = [("x", C.c_float), ("y", C.c_float), ("dir", C.c_int32)]


class emr_result(C.Structure):
    _fields_ = [("parent", C.c_void_p), ("w4", C.c_void_p), ("capacity", C.c_int64),
                ("pair_count", C.c_void_p), ("pair_offset", C.c_void_p),
                ("workspace", C.c_void_p), ("workspace_bytes", C.c_int64)]


class emr_hidden(C.Structure):
    _fields_ = [("sources", C.c_void_p), ("cell", C.c_void_p), ("capacity", C.c_int64),
                ("offsets", C.c_void_p), ("known", C.c_void_p), ("workspace", C.c_void_p),
                ("workspace_bytes", C.c_int64)]


class emr_connections(C.Structure):
    _fields_ = [("cell", C.c_void_p), ("w", C.c_void_p), ("capacity", C.c_int64),
                ("pair_count", C.c_void_p), ("pair_offset", C.c_void_p),
                ("workspace", C.c_void_p), ("workspace_bytes", C.c_int64)]


class emr_launch_profile(C.Structure):
    _fields_ = [("group_size", C.c_int32), ("window", C.c_int32), ("positions", C.c_int32),
                ("call", C.c_int32), ("tiles", C.c_int64), ("queries", C.c_int64),
                ("slots", C.c_double), ("ms", C.c_float), ("compiled", C.c_int32),
                ("listed", C.c_int32), ("parts", C.c_int32)]


class emr_network_info(C.Structure):
    _fields_ = [("n_genomes", C.c_int32), ("n_substrate", C.c_int32), ("n_inputs", C.c_int32),
                ("n_outputs", C.c_int32), ("depth", C.c_int32), ("phases", C.c_int32),
                ("nodes", C.c_int64), ("edges", C.c_int64), ("node_offset", C.c_void_p),
                ("node_cell", C.c_void_p), ("in_offset", C.c_void_p), ("in_src", C.c_void_p),
                ("in_w", C.c_void_p), ("known", C.c_void_p), ("known_words", C.c_int64)]


class emr_network_phase(C.Structure):
    _fields_ = [("sources", C.c_void_p), ("n_sources", C.c_int32), ("src_offsets", C.c_void_p),
                ("src_cell", C.c_void_p), ("n_pairs", C.c_int64), ("parent", C.c_void_p),
                ("w4", C.c_void_p), ("pair_offset", C.c_void_p), ("records", C.c_int64),
                ("conn_cell", C.c_void_p), ("conn_w", C.c_void_p), ("conn_offset", C.c_void_p),
                ("connections", C.c_int64)]


_lib = None

# int32_t sink(int64_t pair, int64_t chunk, const uint32_t* parent, const float* w4, int64_t n,
#              void* user)
SINK = C.CFUNCTYPE(C.c_int32, C.c_int64, C.c_int64, C.POINTER(C.c_uint32), C.POINTER(C.c_float),
                   C.c_int64, C.c_void_p)


def lib():
    """The loaded libemr.so (raises if it was never built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libemr.so is not built; run __graft_entry__.build() or "
                              "python paper_2608_27612_amd/build.py")
        L = C.CDLL(LIB_PATH)
        P, I32, I64, F32, F64 = C.c_void_p, C.c_int32, C.c_int64, C.c_float, C.c_double
        sig = {
            "emr_last_error": (C.c_char_p, []),
            "emr_version": (I32, []),
            "emr_grid_count": (I32, [I32, P, P]),
            "emr_build_grids": (I32, [I32, P, P]),
            "emr_pack_population": (I32, [P, I32, P, P]),
            "emr_free_population": (None, [P]),
            "emr_population_info": (I32, [P, P, P, P, P]),
            "emr_workspace_bytes": (I32, [P, P, I32, P, I32, I32, I64, P]),
            "emr_discover": (I32, [P, P, I32, P, I32, I32, F32, P, P]),
            "emr_result_check": (I32, [P, P, P, P]),
            "emr_eval_raw": (I32, [P, P, I32, P, I32, I32, P, P, I64, P]),
            "emr_discover_cost": (I32, [P, P, I32, P, I32, I32, F64, P, P, P, P]),
            "emr_profile_enable": (I32, [I32, I32, F64]),
            "emr_profile_read": (I32, [P, I32, P]),
            "emr_stream_chunks": (I32, [I32, I64, P]),
            "emr_pack_population_flat": (I32, [I32, P, P, P, P, P, P, P, P, P, P, P]),
            "emr_discover_stream": (I32, [P, P, I32, P, I32, I32, F32, I64, I64, SINK, P, P, P]),
            "emr_set_jit": (I32, [I32]),
            "emr_eval_raw_noalloc": (I32, [P, P, I32, P, I32, I32, P, P, P]),
            "emr_jit_info": (I32, [P, P, P, P, P, P]),
            "emr_call_check": (I32, [P, I64, P, P, P]),
            "emr_cell_words": (I32, [I32, P]),
            "emr_hidden_workspace_bytes": (I32, [I32, I32, P]),
            "emr_hidden_sources": (I32, [P, P, I32, P, I32, I32, P, P, P]),
            "emr_express_workspace_bytes": (I32, [I64, P]),
            "emr_express": (I32, [P, P, I32, P, I32, I32, P, I32, F32, P, P]),
            "emr_chain_workspace_bytes": (I32, [I64, I32, P]),
            "emr_chain_filter": (I32, [P, I64, I32, P, P]),
            "emr_band_workspace_bytes": (I32, [I64, P]),
            "emr_band_values": (I32, [P, P, I32, P, I32, I32, P, P, P, I64, P]),
            "emr_band_filter": (I32, [P, P, I64, F32, P, P]),
            "emr_record_file_open": (I32, [C.c_char_p, I64, I32, I64, P, P]),
            "emr_record_file_sink": (I32, [I64, I64, P, P, I64, P]),
            "emr_record_file_close": (I32, [P, P, P]),
            "emr_build_networks": (I32, [P, P, I32, I32, F32, I32, F32, I32, P, P]),
            "emr_networks_info": (I32, [P, P]),
            "emr_networks_phase": (I32, [P, I32, P]),
            "emr_activate": (I32, [P, P, I32, I32, P, P]),
            "emr_xor_fitness": (I32, [P, I32, I32, P, P]),
            "emr_free_networks": (None, [P]),
            "emr_copy_to_host": (I32, [P, P, I64, P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status: int):
    if status != EMR_OK:
        raise EmrError(status, lib().emr_last_error().decode())


def _stream_ptr(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


# ----------------------------------------------------------------------------- grids

def emr_grid_count(depth: int):
    n, q = C.c_int64(), C.c_int64()
    _check(lib().emr_grid_count(depth, C.byref(n), C.byref(q)))
    return n.value, q.value


def emr_build_grids(depth: int, stream=None):
    """Device tensor [N(D), 2] of cell centres in heap order."""
    import torch
    n, _ = emr_grid_count(depth)
    xy = torch.empty((n, 2), dtype=torch.float32, device="cuda")
    _check(lib().emr_build_grids(depth, C.c_void_p(xy.data_ptr() if n else 0), _stream_ptr(stream)))
    return xy


# ----------------------------------------------------------------------------- population

class Population:
    """A packed population (owns the library's emr_population)."""

    def __init__(self, handle, n_genomes):
        self.handle = handle
        self.n_genomes = n_genomes

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.emr_free_population(self.handle)
            self.handle = None

    def info(self):
        n = self.n_genomes
        steps = np.zeros(2 * n, np.int32)
        edges = np.zeros(2 * n, np.int32)
        window = np.zeros(n, np.int32)
        _check(lib().emr_population_info(self.handle, None, steps.ctypes.data, edges.ctypes.data,
                                         window.ctypes.data))
        return {"steps": steps.reshape(n, 2), "var_edges": edges.reshape(n, 2), "window": window}


def _genome_array(genomes):
    keep = []
    arr = (emr_genome * max(1, len(genomes)))()
    for i, g in enumerate(genomes):
        k = {
            "kind": np.ascontiguousarray(g["kind"], np.uint8),
            "act": np.ascontiguousarray(g["act"], np.uint8),
            "bias": None if g.get("bias") is None else np.ascontiguousarray(g["bias"], np.float32),
            "src": np.ascontiguousarray(g["src"], np.int32),
            "dst": np.ascontiguousarray(g["dst"], np.int32),
            "w": np.ascontiguousarray(g["w"], np.float32),
            "enabled": None if g.get("enabled") is None else np.ascontiguousarray(g["enabled"],
                                                                                    np.uint8),
        }
        keep.append(k)
        ptr = lambda a: None if a is None else a.ctypes.data  # noqa: E731
        arr[i] = emr_genome(len(k["kind"]), len(k["src"]), ptr(k["kind"]), ptr(k["act"]),
                            ptr(k["bias"]), ptr(k["src"]), ptr(k["dst"]), ptr(k["w"]),
                            ptr(k["enabled"]))
    return arr, keep


def flat_genomes(genomes):
    """The concatenated-array layout of emr_pack_population_flat for a list of genome dicts."""
    n = len(genomes)
    nn = np.fromiter((len(g["kind"]) for g in genomes), np.int64, n)
    ne = np.fromiter((len(g["src"]) for g in genomes), np.int64, n)
    node_off = np.zeros(n + 1, np.int64)
    edge_off = np.zeros(n + 1, np.int64)
    np.cumsum(nn, out=node_off[1:])
    np.cumsum(ne, out=edge_off[1:])

    def cat(key, dtype, per_genome_default):
        parts = [np.asarray(g[key] if g.get(key) is not None else per_genome_default(g), dtype)
                 for g in genomes]
        return np.ascontiguousarray(np.concatenate(parts) if parts else np.zeros(0, dtype), dtype)

    return {
        "n": n, "node_off": node_off, "edge_off": edge_off,
        "kind": cat("kind", np.uint8, None), "act": cat("act", np.uint8, None),
        "bias": cat("bias", np.float32, lambda g: np.zeros(len(g["kind"]), np.float32)),
        "src": cat("src", np.int32, None), "dst": cat("dst", np.int32, None),
        "w": cat("w", np.float32, None),
        "enabled": cat("enabled", np.uint8, lambda g: np.ones(len(g["src"]), np.uint8)),
    }


def emr_pack_population(genomes, layout: str = "flat") -> Population:
    """Validate and pack genomes into device program tables: a list of dicts (see workloads.py),
    through emr_pack_population_flat (layout "flat") or emr_pack_population ("structs"), or the
    concatenated arrays of flat_genomes (a dict; passed as they are)."""
    handle = C.c_void_p()
    bad = C.c_int32(-1)
    if isinstance(genomes, dict):
        layout = "flat"
    if layout == "flat":
        f = genomes if isinstance(genomes, dict) else flat_genomes(genomes)
        d = lambda a: a.ctypes.data if len(a) else None  # noqa: E731
        st = lib().emr_pack_population_flat(f["n"], f["node_off"].ctypes.data, d(f["kind"]),
                                            d(f["act"]), d(f["bias"]), f["edge_off"].ctypes.data,
                                            d(f["src"]), d(f["dst"]), d(f["w"]), d(f["enabled"]),
                                            C.byref(handle), C.byref(bad))
        keep = f
    else:
        arr, keep = _genome_array(genomes)
        st = lib().emr_pack_population(arr, len(genomes), C.byref(handle), C.byref(bad))
    if st != EMR_OK:
        err = EmrError(st, lib().emr_last_error().decode())
        err.bad_index = bad.value
        raise err
    del keep
    return Population(handle, int(f["n"]) if layout == "flat" else len(genomes))


# ----------------------------------------------------------------------------- discovery

# numpy records with emr_source's layout (12 bytes: float x, float y, int32 dir)
SOURCE_DTYPE = np.dtype([("x", "<f4"), ("y", "<f4"), ("dir", "<i4")])
_NO_SOURCE = np.zeros(1, SOURCE_DTYPE)


def _sources(sources):
    """The sources as a contiguous array of emr_source records: an array of SOURCE_DTYPE is
    passed as it is (no per-call conversion); anything else indexable by "x", "y", "dir" is
    converted. Keep the returned array alive until the call that gets its address returns."""
    if isinstance(sources, np.ndarray) and sources.dtype == SOURCE_DTYPE:
        arr = sources if sources.flags.c_contiguous else np.ascontiguousarray(sources)
    else:
        arr = np.array([(float(s["x"]), float(s["y"]), int(s["dir"])) for s in sources],
                       dtype=SOURCE_DTYPE)
    return arr if len(arr) else _NO_SOURCE


_SRC_LAST = [None, None, 0]  # the last sources object passed, its record array and address


def _sources_ptr(sources):
    """(record array, its address) of _sources(sources); a repeated call with the same array
    object reuses the address (an array's data never moves while the cache holds it)."""
    if sources is _SRC_LAST[0]:
        return _SRC_LAST[1], _SRC_LAST[2]
    arr = _sources(sources)
    ptr = arr.ctypes.data
    if isinstance(sources, np.ndarray):
        _SRC_LAST[0], _SRC_LAST[1], _SRC_LAST[2] = sources, arr, ptr
    return arr, ptr


def _offsets(src_offsets):
    if src_offsets is None:
        return None
    return np.ascontiguousarray(src_offsets, dtype=np.int32)


def n_pairs_of(pop: Population, sources, src_offsets=None) -> int:
    return len(sources) if src_offsets is not None else pop.n_genomes * len(sources)


def emr_workspace_bytes(pop: Population, sources, depth: int, src_offsets=None,
                        capacity: int = 0) -> int:
    offs = _offsets(src_offsets)
    b = C.c_int64()
    src = _sources(sources)
    _check(lib().emr_workspace_bytes(pop.handle, src.ctypes.data, len(sources),
                                     None if offs is None else offs.ctypes.data,
                                     0 if offs is not None else len(sources), depth,
                                     int(capacity), C.byref(b)))
    return b.value


# Default capacity of a result: the worst case n_pairs * Q(D) while its buffers stay below this
# many records, else this many (a call that finds more reports its total; emr_discover_all then
# retries at that size).
DEFAULT_CAPACITY = 1 << 22


def alloc_result(pop: Population, sources, depth: int, src_offsets=None, capacity=None):
    """Device buffers for emr_discover (torch tensors): CSR records of `capacity` records."""
    import torch
    _, q = emr_grid_count(depth)
    npairs = n_pairs_of(pop, sources, src_offsets)
    cap = min(npairs * q, DEFAULT_CAPACITY) if capacity is None else int(capacity)
    ws = emr_workspace_bytes(pop, sources, depth, src_offsets, cap)
    return {
        "parent": torch.empty(max(cap, 1), dtype=torch.int32, device="cuda"),
        "w4": torch.empty((max(cap, 1), 4), dtype=torch.float32, device="cuda"),
        "pair_count": torch.empty(max(npairs, 1), dtype=torch.int64, device="cuda"),
        "pair_offset": torch.empty(npairs + 1, dtype=torch.int64, device="cuda"),
        "workspace": torch.empty(max(ws, 256), dtype=torch.uint8, device="cuda"),
        "capacity": cap,
        "n_pairs": npairs,
    }


def _result_struct(res):
    ws = res["workspace"]
    assert ws.data_ptr() % 256 == 0
    return emr_result(res["parent"].data_ptr(), res["w4"].data_ptr(), res["capacity"],
                      res["pair_count"].data_ptr(), res["pair_offset"].data_ptr(),
                      ws.data_ptr(), ws.numel())


def emr_discover(pop: Population, sources, depth: int, theta: float, res=None, src_offsets=None,
                 stream=None, capacity=None):
    """Enqueue eager discovery; returns the result dict (device tensors, see alloc_result).
    `parent` is the int32 view of the library's uint32 heap indices."""
    if res is None:
        res = alloc_result(pop, sources, depth, src_offsets, capacity)
    offs = _offsets(src_offsets)
    out = res.get("_struct")
    if out is None or out.parent != res["parent"].data_ptr() or \
            out.workspace != res["workspace"].data_ptr() or out.w4 != res["w4"].data_ptr() or \
            out.pair_offset != res["pair_offset"].data_ptr() or \
            out.pair_count != res["pair_count"].data_ptr() or out.capacity != res["capacity"]:
        out = _result_struct(res)
        res["_struct"] = out
    src, src_ptr = _sources_ptr(sources)
    _check(lib().emr_discover(pop.handle, src_ptr, len(sources),
                              None if offs is None else offs.ctypes.data,
                              0 if offs is not None else len(sources), depth,
                              C.c_float(theta), C.byref(out), _stream_ptr(stream)))
    return res


def emr_result_check(res, stream=None):
    """Synchronize and check a discover result; returns (total records, largest pair count).
    (The check waits for the call through its workspace's flag slot; a stream is passed only when
    the caller names one.)"""
    out = res.get("_struct") or _result_struct(res)
    chk = res.get("_check_args")
    if chk is None or chk[0] is not out:
        total, mx = C.c_int64(), C.c_int64()
        chk = (out, total, mx, C.byref(out), C.byref(total), C.byref(mx))
        res["_check_args"] = chk
    _, total, mx, p_out, p_total, p_mx = chk
    _check(lib().emr_result_check(p_out, p_total, p_mx,
                                  None if stream is None else _stream_ptr(stream)))
    return total.value, mx.value


def emr_discover_all(pop: Population, sources, depth: int, theta: float, src_offsets=None,
                     stream=None, capacity=None):
    """emr_discover + emr_result_check, retried once at the reported total when the capacity was
    too small; returns the checked result."""
    res = emr_discover(pop, sources, depth, theta, src_offsets=src_offsets, stream=stream,
                       capacity=capacity)
    try:
        emr_result_check(res, stream)
    except EmrError as e:
        if e.status != EMR_E_CAPACITY:
            raise
        total = int(res["pair_offset"][-1].item())
        res = emr_discover(pop, sources, depth, theta, src_offsets=src_offsets, stream=stream,
                           capacity=total)
        emr_result_check(res, stream)
    return res


def emr_eval_raw(pop: Population, sources, depth: int, src_offsets=None, stream=None):
    """Device tensor [n_pairs, N(D)] of raw CPPN outputs."""
    import torch
    n, _ = emr_grid_count(depth)
    npairs = n_pairs_of(pop, sources, src_offsets)
    out = torch.empty((npairs, n), dtype=torch.float32, device="cuda")
    ws_bytes = emr_workspace_bytes(pop, sources, depth, src_offsets, 0)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    offs = _offsets(src_offsets)
    src = _sources(sources)
    _check(lib().emr_eval_raw(pop.handle, src.ctypes.data, len(sources),
                              None if offs is None else offs.ctypes.data,
                              0 if offs is not None else len(sources), depth,
                              C.c_void_p(out.data_ptr() if out.numel() else 0),
                              C.c_void_p(ws.data_ptr()), ws.numel(), _stream_ptr(stream)))
    return out


def emr_eval_raw_noalloc(pop: Population, sources, depth: int, out, err, src_offsets=None,
                         stream=None):
    """emr_eval_raw_noalloc into caller-owned device tensors: out float32 [n_pairs, N(D)] and err
    (one int32 / uint32 word, cleared by the call, error bits after the stream's work)."""
    offs = _offsets(src_offsets)
    src = _sources(sources)
    _check(lib().emr_eval_raw_noalloc(pop.handle, src.ctypes.data, len(sources),
                                      None if offs is None else offs.ctypes.data,
                                      0 if offs is not None else len(sources), depth,
                                      C.c_void_p(out.data_ptr() if out.numel() else 0),
                                      C.c_void_p(err.data_ptr()), _stream_ptr(stream)))


def emr_discover_work(pop: Population, sources, depth: int, src_offsets=None,
                      transcendental_slots: float = 4.0):
    """The algorithmic work of one discover call: {"slots": VALU slots under the cost model,
    "queries": all queries, "evaluated": queries of position-dependent pairs, "flops": useful
    floating-point operations}."""
    offs = _offsets(src_offsets)
    slots, queries, evaluated, flops = C.c_double(), C.c_double(), C.c_double(), C.c_double()
    src = _sources(sources)
    _check(lib().emr_discover_cost(pop.handle, src.ctypes.data, len(sources),
                                   None if offs is None else offs.ctypes.data,
                                   0 if offs is not None else len(sources), depth,
                                   float(transcendental_slots), C.byref(slots), C.byref(queries),
                                   C.byref(evaluated), C.byref(flops)))
    return {"slots": slots.value, "queries": queries.value, "evaluated": evaluated.value,
            "flops": flops.value}


def emr_discover_cost(pop: Population, sources, depth: int, src_offsets=None,
                      transcendental_slots: float = 4.0):
    """(algorithmic VALU slots, queries) of one discover call under the cost model."""
    w = emr_discover_work(pop, sources, depth, src_offsets, transcendental_slots)
    return w["slots"], w["queries"]


def records_to_host(res):
    """Copy a checked result to numpy: (pair counts, per-pair (parent[i], w4[i]) in ascending
    order)."""
    n = res["n_pairs"]
    counts = res["pair_count"][:n].cpu().numpy()
    offs = res["pair_offset"].cpu().numpy()
    total = int(min(offs[-1], res["capacity"]))
    parent = res["parent"][:total].cpu().numpy().view(np.uint32).astype(np.int64)
    w4 = res["w4"][:total].cpu().numpy()
    out = []
    for r in range(n):
        lo, hi = int(offs[r]), int(offs[r] + counts[r])
        out.append((parent[lo:hi], w4[lo:hi]))
    return counts, out


# ----------------------------------------------------------------------------- profiling

def emr_profile_enable(on=True, transcendental_slots: float = 4.0, every: int = 1):
    """on: False/0 off, True/1 every discover launch, "first"/2 a call's first launch only;
    every: time one call in `every`."""
    mode = 2 if on == "first" else int(on)
    _check(lib().emr_profile_enable(mode, int(every), float(transcendental_slots)))


def emr_profile_read():
    """Every launch record held (profiled calls since enable or the last read), in launch order;
    synchronizes on their events and drops them. "first" marks a call's first launch."""
    n = C.c_int32()
    _check(lib().emr_profile_read(None, 0, C.byref(n)))
    arr = (emr_launch_profile * max(1, n.value))()
    _check(lib().emr_profile_read(arr, n.value, C.byref(n)))
    out = []
    for i, r in enumerate(arr[:n.value]):
        out.append({"S": r.group_size, "W": r.window, "P": r.positions, "call": r.call,
                    "tiles": r.tiles, "queries": r.queries, "slots": r.slots, "ms": r.ms,
                    "compiled": bool(r.compiled), "listed": bool(r.listed), "parts": r.parts,
                    "first": i == 0 or arr[i - 1].call != r.call})
    return out


# ----------------------------------------------------------------------------- compiled tier

def emr_set_jit(policy: int):
    """Process-wide compiled-tier policy: EMR_JIT_OFF, EMR_JIT_AUTO (default), EMR_JIT_ALWAYS."""
    _check(lib().emr_set_jit(int(policy)))


def emr_jit_info(pop: Population):
    """The compiled tier of the population's current plan: {"state": 0 not compiled / 1 compiled /
    -1 failed, "programs", "code_bytes", "compile_ms", "load_ms", "error" (when failed)}."""
    st, npg, nb = C.c_int32(), C.c_int64(), C.c_int64()
    cm, lm = C.c_double(), C.c_double()
    _check(lib().emr_jit_info(pop.handle, C.byref(st), C.byref(npg), C.byref(nb), C.byref(cm),
                              C.byref(lm)))
    out = {"state": st.value, "programs": npg.value, "code_bytes": nb.value,
           "compile_ms": cm.value, "load_ms": lm.value}
    if st.value == -1:
        out["error"] = lib().emr_last_error().decode()
    return out


# ----------------------------------------------------------------------------- streaming

def emr_stream_chunks(depth: int, chunk_positions: int = 1 << 24) -> int:
    n = C.c_int64()
    _check(lib().emr_stream_chunks(depth, chunk_positions, C.byref(n)))
    return n.value


class RecordFile:
    """A record file opened by emr_record_file_open; pass it as emr_discover_stream's sink to
    write the run to disk. `cursor` is where a resumed run starts (0 for a new file)."""

    def __init__(self, path: str, n_pairs: int, resume: bool = False, buffer_bytes: int = 0):
        h, cur = C.c_void_p(), C.c_int64()
        _check(lib().emr_record_file_open(os.fsencode(path), n_pairs, int(bool(resume)),
                                          buffer_bytes, C.byref(h), C.byref(cur)))
        self.handle, self.cursor, self.path = h, cur.value, path

    def close(self):
        """Closes the file: (records in the file, cursor after its last delivery)."""
        if self.handle is None:
            raise ValueError("record file already closed")
        recs, nxt = C.c_int64(), C.c_int64()
        h, self.handle = self.handle, None
        _check(lib().emr_record_file_close(h, C.byref(recs), C.byref(nxt)))
        return recs.value, nxt.value

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        if self.handle is not None:
            self.close()


def read_record_file(path: str):
    """Reads a record file (layout in include/emr.h): (n_pairs, [(pair, chunk, parent uint32 [n],
    w4 float32 [n, 4]), ...]) in file order. A trailing partial block is ignored."""
    data = np.fromfile(path, dtype=np.uint8)
    if len(data) < 32 or bytes(data[:8]) != b"EMRRECv1":
        raise ValueError("%s is not a record file" % path)
    n_pairs = int(data[8:16].view(np.int64)[0])
    blocks, pos = [], 32
    while pos + 24 <= len(data):
        pair, chunk, n = (int(v) for v in data[pos:pos + 24].view(np.int64))
        end = pos + 24 + 20 * n
        if n < 1 or end > len(data):
            break
        parent = data[pos + 24:pos + 24 + 4 * n].view(np.uint32).copy()
        w4 = data[pos + 24 + 4 * n:end].view(np.float32).reshape(n, 4).copy()
        blocks.append((pair, chunk, parent, w4))
        pos = end
    return n_pairs, blocks


def emr_discover_stream(pop: Population, sources, depth: int, theta: float, sink,
                        chunk_positions: int = 1 << 24, start: int = 0, src_offsets=None,
                        stream=None) -> int:
    """Streamed eager discovery. `sink(pair, chunk, parent, w4)` receives numpy copies of each
    (chunk, pair) delivery (parent uint32 [n], w4 float32 [n, 4]) and returns True/None to go on,
    False to stop; or `sink` is a RecordFile, whose C sink writes the deliveries to its file.
    Returns the cursor after the run; a stop raises EmrError(EMR_E_ABORTED) whose `next_cursor` is
    the refused delivery's cursor (see emr_discover_stream in include/emr.h)."""
    offs = _offsets(src_offsets)
    errors = []

    def _sink(pair, chunk, parent, w4, n, user):
        try:
            p = np.ctypeslib.as_array(parent, shape=(n,)).copy()
            w = np.ctypeslib.as_array(w4, shape=(n * 4,)).reshape(n, 4).copy()
            return 0 if sink(int(pair), int(chunk), p, w) is not False else 1
        except BaseException as e:  # an exception in the sink stops the run and is re-raised
            errors.append(e)
            return 1

    if isinstance(sink, RecordFile):
        if sink.handle is None:
            raise ValueError("record file is closed")
        cb, user = SINK(("emr_record_file_sink", lib())), sink.handle
    else:
        cb, user = SINK(_sink), None
    nxt = C.c_int64(start)
    src = _sources(sources)
    st = lib().emr_discover_stream(pop.handle, src.ctypes.data, len(sources),
                                   None if offs is None else offs.ctypes.data,
                                   0 if offs is not None else len(sources), depth,
                                   C.c_float(theta), chunk_positions, start, cb, user,
                                   C.byref(nxt), _stream_ptr(stream))
    if errors:
        raise errors[0]
    if st != EMR_OK:
        err = EmrError(st, lib().emr_last_error().decode())
        err.next_cursor = nxt.value
        raise err
    return nxt.value



# ----------------------------------------------------------------------------- after discovery

def emr_call_check(workspace, capacity: int, stream=None):
    """emr_call_check on a call's workspace tensor: (total, largest per pair or genome)."""
    total, mx = C.c_int64(), C.c_int64()
    _check(lib().emr_call_check(C.c_void_p(workspace.data_ptr()), int(capacity), C.byref(total),
                                C.byref(mx), _stream_ptr(stream)))
    return total.value, mx.value


def emr_cell_words(depth: int) -> int:
    w = C.c_int64()
    _check(lib().emr_cell_words(depth, C.byref(w)))
    return w.value


def _rec_struct(rec):
    return rec.get("_struct") or _result_struct(rec)


def emr_hidden_sources(pop: Population, sources, depth: int, rec, src_offsets=None, known=None,
                       capacity=None, stream=None):
    """The hidden nodes of a checked discover result `rec` (same population, sources and depth):
    enqueues emr_hidden_sources and checks it (retrying once at the reported total when the
    capacity was too small). Returns dict(sources int32 [n, 3] device (emr_source records), cell
    uint32-as-int32 [n] device, offsets int64 [n_genomes + 1] device, total). `known`: an int32
    device bitmap of n_genomes * emr_cell_words(depth) words or None."""
    import torch
    G = pop.n_genomes
    cap = int(capacity) if capacity is not None else max(1024, 4 * int(rec["pair_offset"][-1].item()))
    wsb = C.c_int64()
    _check(lib().emr_hidden_workspace_bytes(G, depth, C.byref(wsb)))
    ws = torch.empty(max(wsb.value, 256), dtype=torch.uint8, device="cuda")
    offs = _offsets(src_offsets)
    src = _sources(sources)
    # the call ors its new cells into `known`: a retry starts again from the bits given
    known_before = known.clone() if known is not None else None
    for attempt in range(2):
        out = {"sources": torch.empty((max(cap, 1), 3), dtype=torch.int32, device="cuda"),
               "cell": torch.empty(max(cap, 1), dtype=torch.int32, device="cuda"),
               "offsets": torch.empty(G + 1, dtype=torch.int64, device="cuda")}
        st = emr_hidden(out["sources"].data_ptr(), out["cell"].data_ptr(), cap,
                        out["offsets"].data_ptr(), 0 if known is None else known.data_ptr(),
                        ws.data_ptr(), ws.numel())
        _check(lib().emr_hidden_sources(pop.handle, src.ctypes.data, len(sources),
                                        None if offs is None else offs.ctypes.data,
                                        0 if offs is not None else len(sources), depth,
                                        C.byref(_rec_struct(rec)), C.byref(st),
                                        _stream_ptr(stream)))
        try:
            total, _ = emr_call_check(ws, cap, stream)
        except EmrError as e:
            if e.status != EMR_E_CAPACITY or attempt == 1:
                raise
            cap = int(out["offsets"][-1].item())
            if known is not None:
                known.copy_(known_before)
            continue
        out["total"] = total
        return out


def hidden_sources_to_host(hs):
    """(sources as numpy emr_source records, int32 offsets) of an emr_hidden_sources output, for
    the next emr_discover call's per-genome sources."""
    n = hs["total"]
    src = hs["sources"][:n].cpu().numpy().copy().view(SOURCE_DTYPE).reshape(-1)
    return src, hs["offsets"].cpu().numpy().astype(np.int32)


def emr_express(pop: Population, sources, depth: int, rec, type_mask: int = EMR_CONN_ALL,
                w_min: float = 0.1, src_offsets=None, capacity=None, stream=None):
    """The connections of a checked discover result (see emr_express in include/emr.h), checked;
    returns dict(cell, w, pair_count, pair_offset device tensors, total)."""
    import torch
    n_pairs = rec["n_pairs"]
    cap = int(capacity) if capacity is not None else 4 * int(rec["pair_offset"][-1].item())
    wsb = C.c_int64()
    _check(lib().emr_express_workspace_bytes(n_pairs, C.byref(wsb)))
    ws = torch.empty(max(wsb.value, 256), dtype=torch.uint8, device="cuda")
    out = {"cell": torch.empty(max(cap, 1), dtype=torch.int32, device="cuda"),
           "w": torch.empty(max(cap, 1), dtype=torch.float32, device="cuda"),
           "pair_count": torch.empty(max(n_pairs, 1), dtype=torch.int64, device="cuda"),
           "pair_offset": torch.empty(n_pairs + 1, dtype=torch.int64, device="cuda")}
    st = emr_connections(out["cell"].data_ptr(), out["w"].data_ptr(), cap,
                         out["pair_count"].data_ptr(), out["pair_offset"].data_ptr(),
                         ws.data_ptr(), ws.numel())
    offs = _offsets(src_offsets)
    src = _sources(sources)
    _check(lib().emr_express(pop.handle, src.ctypes.data, len(sources),
                             None if offs is None else offs.ctypes.data,
                             0 if offs is not None else len(sources), depth,
                             C.byref(_rec_struct(rec)), int(type_mask), C.c_float(w_min),
                             C.byref(st), _stream_ptr(stream)))
    out["total"], _ = emr_call_check(ws, cap, stream)
    out["n_pairs"] = n_pairs
    out["capacity"] = cap
    return out


def _conn_struct(conn, workspace=None):
    ws_ptr, ws_n = (0, 0) if workspace is None else (workspace.data_ptr(), workspace.numel())
    return emr_connections(conn["cell"].data_ptr(), conn["w"].data_ptr(), conn["capacity"],
                           conn["pair_count"].data_ptr(), conn["pair_offset"].data_ptr(),
                           ws_ptr, ws_n)


def emr_band_values(pop: Population, sources, depth: int, conn, src_offsets=None, stream=None):
    """ES-HyperNEAT band values of the connections of a checked emr_express result `conn` (see
    emr_band_values in include/emr.h), checked; a float32 device tensor aligned with conn's
    entries."""
    import torch
    n_pairs = conn["n_pairs"]
    wsb = C.c_int64()
    _check(lib().emr_band_workspace_bytes(n_pairs, C.byref(wsb)))
    ws = torch.empty(max(wsb.value, 256), dtype=torch.uint8, device="cuda")
    band = torch.empty(max(conn["capacity"], 1), dtype=torch.float32, device="cuda")
    offs = _offsets(src_offsets)
    src = _sources(sources)
    st = _conn_struct(conn)
    _check(lib().emr_band_values(pop.handle, src.ctypes.data, len(sources),
                                 None if offs is None else offs.ctypes.data,
                                 0 if offs is not None else len(sources), depth, C.byref(st),
                                 C.c_void_p(band.data_ptr()), C.c_void_p(ws.data_ptr()),
                                 ws.numel(), _stream_ptr(stream)))
    emr_call_check(ws, 0, stream)
    return band


def emr_band_filter(conn, band, theta_band: float, capacity=None, stream=None):
    """The connections of `conn` whose band value exceeds theta_band (see emr_band_filter in
    include/emr.h), checked; a dict of the emr_express form."""
    import torch
    n_pairs = conn["n_pairs"]
    cap = int(conn["total"]) if capacity is None else int(capacity)
    wsb = C.c_int64()
    _check(lib().emr_express_workspace_bytes(n_pairs, C.byref(wsb)))
    ws = torch.empty(max(wsb.value, 256), dtype=torch.uint8, device="cuda")
    out = {"cell": torch.empty(max(cap, 1), dtype=torch.int32, device="cuda"),
           "w": torch.empty(max(cap, 1), dtype=torch.float32, device="cuda"),
           "pair_count": torch.empty(max(n_pairs, 1), dtype=torch.int64, device="cuda"),
           "pair_offset": torch.empty(n_pairs + 1, dtype=torch.int64, device="cuda"),
           "capacity": cap, "n_pairs": n_pairs}
    st_in = _conn_struct(conn)
    st_out = _conn_struct(out, ws)
    _check(lib().emr_band_filter(C.byref(st_in), C.c_void_p(band.data_ptr()), n_pairs,
                                 C.c_float(theta_band), C.byref(st_out), _stream_ptr(stream)))
    out["total"], _ = emr_call_check(ws, cap, stream)
    return out


def emr_chain_filter(rec, depth: int, capacity=None, stream=None):
    """Eq. 2's literal chain rule applied to a checked discover result: a result dict of the same
    form (checked)."""
    import torch
    n_pairs = rec["n_pairs"]
    cap = int(rec["pair_offset"][-1].item()) if capacity is None else int(capacity)
    wsb = C.c_int64()
    _check(lib().emr_chain_workspace_bytes(n_pairs, depth, C.byref(wsb)))
    out = {"parent": torch.empty(max(cap, 1), dtype=torch.int32, device="cuda"),
           "w4": torch.empty((max(cap, 1), 4), dtype=torch.float32, device="cuda"),
           "pair_count": torch.empty(max(n_pairs, 1), dtype=torch.int64, device="cuda"),
           "pair_offset": torch.empty(n_pairs + 1, dtype=torch.int64, device="cuda"),
           "workspace": torch.empty(max(wsb.value, 256), dtype=torch.uint8, device="cuda"),
           "capacity": cap, "n_pairs": n_pairs}
    st = _result_struct(out)
    out["_struct"] = st
    _check(lib().emr_chain_filter(C.byref(_rec_struct(rec)), n_pairs, depth, C.byref(st),
                                  _stream_ptr(stream)))
    emr_result_check(out, stream)
    return out


# ----------------------------------------------------------------------------- networks

def _dev_to_host(ptr, n, dtype, stream=None):
    """n elements of dtype from a library-owned device pointer (emr_copy_to_host)."""
    out = np.empty(max(int(n), 0), dtype=dtype)
    if n > 0:
        _check(lib().emr_copy_to_host(out.ctypes.data, C.c_void_p(ptr), out.nbytes,
                                      _stream_ptr(stream)))
    return out


class Networks:
    """The networks of a population (owns the library's emr_networks handle)."""

    def __init__(self, handle):
        self.handle = handle

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.emr_free_networks(self.handle)
            self.handle = None

    def info(self) -> emr_network_info:
        i = emr_network_info()
        _check(lib().emr_networks_info(self.handle, C.byref(i)))
        return i

    def to_host(self, stream=None):
        """Per genome dict(cells: kept hidden cells ascending, src, dst, w: the edges with the
        genome's node numbers, grouped by destination in the library's order)."""
        i = self.info()
        G = i.n_genomes
        node_off = _dev_to_host(i.node_offset, G + 1, np.int64, stream)
        cell = _dev_to_host(i.node_cell, i.nodes, np.uint32, stream)
        in_off = _dev_to_host(i.in_offset, i.nodes + 1, np.int64, stream)
        src = _dev_to_host(i.in_src, i.edges, np.uint32, stream).astype(np.int64)
        w = _dev_to_host(i.in_w, i.edges, np.float32, stream)
        nets = []
        for g in range(G):
            a, b = int(node_off[g]), int(node_off[g + 1])
            e0, e1 = int(in_off[a]), int(in_off[b])
            dst = np.repeat(np.arange(b - a, dtype=np.int64), np.diff(in_off[a:b + 1]))
            nets.append({"cells": cell[a + i.n_substrate:b].astype(np.int64),
                         "substrate_cells": cell[a:a + i.n_substrate],
                         "src": src[e0:e1] - a, "dst": dst, "w": w[e0:e1]})
        return nets

    def known_cells(self, stream=None):
        """Per genome the hidden cells of every phase before pruning (ascending heap indices)."""
        i = self.info()
        bits = _dev_to_host(i.known, i.n_genomes * i.known_words, np.uint32, stream)
        bits = bits.reshape(i.n_genomes, i.known_words)
        return [np.nonzero(np.unpackbits(bits[g].view(np.uint8), bitorder="little"))[0] + 1
                for g in range(i.n_genomes)]

    def phase(self, k: int, stream=None):
        """Phase k on the host: dict(sources, src_offsets, src_cell, records (the oracle's records
        layout: pair_count, pair_offset, parent, w4), conn (pair_count, pair_offset, cell, w))."""
        ph = emr_network_phase()
        _check(lib().emr_networks_phase(self.handle, k, C.byref(ph)))
        G = self.info().n_genomes
        src = np.ctypeslib.as_array(C.cast(ph.sources, C.POINTER(C.c_uint8)),
                                    shape=(ph.n_sources * SOURCE_DTYPE.itemsize,))
        src = src.view(SOURCE_DTYPE).copy()
        offs = None
        if ph.src_offsets:
            offs = np.ctypeslib.as_array(C.cast(ph.src_offsets, C.POINTER(C.c_int32)),
                                         shape=(G + 1,)).copy()
        rec_off = _dev_to_host(ph.pair_offset, ph.n_pairs + 1, np.int64, stream)
        records = {"pair_offset": rec_off, "pair_count": np.diff(rec_off),
                   "parent": _dev_to_host(ph.parent, ph.records, np.uint32, stream).astype(np.int64),
                   "w4": _dev_to_host(ph.w4, 4 * ph.records, np.float32, stream).reshape(-1, 4)}
        c_off = _dev_to_host(ph.conn_offset, ph.n_pairs + 1, np.int64, stream)
        conn = {"pair_offset": c_off, "pair_count": np.diff(c_off),
                "cell": _dev_to_host(ph.conn_cell, ph.connections, np.uint32, stream).astype(np.int64),
                "w": _dev_to_host(ph.conn_w, ph.connections, np.float32, stream)}
        cells = None
        if ph.src_cell:
            cells = _dev_to_host(ph.src_cell, ph.n_sources, np.uint32, stream).astype(np.int64)
        return {"sources": src, "src_offsets": offs, "src_cell": cells, "records": records,
                "conn": conn}

    def activate(self, inputs, steps: int, stream=None):
        """Outputs [n_genomes, n_patterns, n_outputs] (numpy) of emr_activate."""
        import torch
        i = self.info()
        x = np.ascontiguousarray(inputs, dtype=np.float32).reshape(-1, i.n_inputs)
        out = torch.empty(max(1, i.n_genomes * len(x) * i.n_outputs), dtype=torch.float32,
                          device="cuda")
        _check(lib().emr_activate(self.handle, x.ctypes.data, len(x), steps,
                                  C.c_void_p(out.data_ptr()), _stream_ptr(stream)))
        return out[:i.n_genomes * len(x) * i.n_outputs].cpu().numpy().reshape(
            i.n_genomes, len(x), i.n_outputs)

    def xor_fitness(self, bias_input: int, steps: int, out=None, stream=None):
        """emr_xor_fitness into `out` (a float32 device tensor of n_genomes, allocated when None);
        returns the tensor (not synchronized)."""
        import torch
        G = self.info().n_genomes
        if out is None:
            out = torch.empty(G, dtype=torch.float32, device="cuda")
        _check(lib().emr_xor_fitness(self.handle, -1 if bias_input is None else int(bias_input),
                                     steps, C.c_void_p(out.data_ptr()), _stream_ptr(stream)))
        return out


def emr_build_networks(pop: Population, substrate, depth: int, theta: float, type_mask: int,
                       w_min: float, iterations: int, stream=None) -> Networks:
    """emr_build_networks (synchronizing) on a packed population and a substrate (shared
    sources: inputs outgoing, outputs incoming)."""
    src = _sources(substrate)
    h = C.c_void_p()
    _check(lib().emr_build_networks(pop.handle, src.ctypes.data, len(substrate), depth,
                                    C.c_float(theta), type_mask, C.c_float(w_min), iterations,
                                    C.byref(h), _stream_ptr(stream)))
    return Networks(h)
