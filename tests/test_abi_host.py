"""The C-ABI library on the host: it loads, exports every declared symbol, and rejects bad
arguments before touching a device (no GPU needed)."""

import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2608_27612_amd import emr, workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "emr.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(emr_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 10
    assert set(names) == set(emr.ABI_FUNCTIONS)
    lib = C.CDLL(emr.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), name


def test_grid_count():
    for D in range(0, 16):
        n, q = emr.emr_grid_count(D)
        assert n == (4 ** (D + 1) - 4) // 3
        assert q == ((4 ** D - 1) // 3 if D else 0)
    for bad in (-1, 16):
        with pytest.raises(emr.EmrError) as e:
            emr.emr_grid_count(bad)
        assert e.value.status == emr.EMR_E_INVAL


def test_pack_validation_reports_first_bad_genome():
    good = W.population(0, 3, 5, 10)
    cyc = {k: v.copy() for k, v in good[1].items()}
    # add a 2-cycle between the output and a new hidden node
    n = len(cyc["kind"])
    cyc["kind"] = np.append(cyc["kind"], np.uint8(5))
    cyc["act"] = np.append(cyc["act"], np.uint8(0))
    cyc["bias"] = np.append(cyc["bias"], np.float32(0))
    out = int(np.nonzero(cyc["kind"] == 6)[0][0])
    cyc["src"] = np.append(cyc["src"], np.int32([out, n]))
    cyc["dst"] = np.append(cyc["dst"], np.int32([n, out]))
    cyc["w"] = np.append(cyc["w"], np.float32([1, 1]))
    cyc["enabled"] = np.append(cyc["enabled"], np.uint8([1, 1]))
    with pytest.raises(emr.EmrError) as e:
        emr.emr_pack_population([good[0], good[2], cyc, good[1]])
    assert e.value.status == emr.EMR_E_CYCLE
    assert e.value.bad_index == 2
    assert "cycle" in str(e.value)


def test_discover_rejects_null_population():
    L = emr.lib()
    res = emr.emr_result()
    src = emr._sources(W.xor_sources())
    st = L.emr_discover(None, src.ctypes.data, 4, None, 4, 5, C.c_float(0.03), C.byref(res), None)
    assert st == emr.EMR_E_INVAL
    assert b"population" in L.emr_last_error()
    st = L.emr_build_grids(-3, None, None)
    assert st == emr.EMR_E_INVAL


def test_version():
    assert emr.lib().emr_version() >= 100


def test_stream_chunk_count_and_argument_errors():
    """emr_stream_chunks counts tiles of 256 positions (the first holding levels 1..3); streaming
    refuses bad arguments before touching a GPU."""
    from paper_2608_27612_amd import emr
    import oracle
    for D in [0, 3, 4, 7, 13]:
        tiles = 1 if D < 4 else 1 + (oracle.n_positions(D) - 84) // 256
        for chunk in [256, 512, 256 * 7, 1 << 24]:
            assert emr.emr_stream_chunks(D, chunk) == -(-tiles // (chunk // 256))
    assert emr.emr_stream_chunks(13, 1 << 24) == 6
    for chunk in [0, 255, 300, -256]:
        with pytest.raises(emr.EmrError) as e:
            emr.emr_stream_chunks(7, chunk)
        assert e.value.status == emr.EMR_E_INVAL
    with pytest.raises(emr.EmrError) as e:
        emr.emr_stream_chunks(16, 256)
    assert e.value.status == emr.EMR_E_INVAL
    L = emr.lib()
    sink = emr.SINK(lambda *a: 0)
    nxt = C.c_int64(-5)
    st = L.emr_discover_stream(None, None, 0, None, 0, 7, C.c_float(0.03), 256, 0, sink, None,
                               C.byref(nxt), None)
    assert st == emr.EMR_E_INVAL and nxt.value == 0
    st = L.emr_discover_stream(None, None, 0, None, 0, 7, C.c_float(0.03), 256, 0,
                               C.cast(None, emr.SINK), None, None, None)
    assert st == emr.EMR_E_INVAL


def test_network_calls_refuse_null_arguments():
    """Checked on the host before any device work."""
    L = emr.lib()
    h = C.c_void_p()
    subs = W.xor_sources()
    assert L.emr_build_networks(None, subs.ctypes.data, 4, 5, C.c_float(0.02), 1, C.c_float(0.1), 1,
                                C.byref(h), None) == emr.EMR_E_INVAL
    assert L.emr_build_networks(None, subs.ctypes.data, 4, 5, C.c_float(0.02), 1, C.c_float(0.1), 1,
                                None, None) == emr.EMR_E_INVAL
    assert L.emr_activate(None, None, 4, 1, None, None) == emr.EMR_E_INVAL
    assert L.emr_xor_fitness(None, 1, 1, None, None) == emr.EMR_E_INVAL
    assert L.emr_networks_info(None, None) == emr.EMR_E_INVAL
    assert L.emr_networks_phase(None, 0, None) == emr.EMR_E_INVAL
    assert L.emr_copy_to_host(None, None, -1, None) == emr.EMR_E_INVAL
    assert L.emr_copy_to_host(None, None, 0, None) == emr.EMR_OK
    L.emr_free_networks(None)


def test_band_calls_refuse_bad_arguments():
    """Checked on the host before any device work."""
    L = emr.lib()
    b = C.c_int64()
    assert L.emr_band_workspace_bytes(-1, C.byref(b)) == emr.EMR_E_INVAL
    assert L.emr_band_workspace_bytes(1000, C.byref(b)) == emr.EMR_OK and b.value == 16128
    subs = W.xor_sources()
    assert L.emr_band_values(None, subs.ctypes.data, 4, None, 4, 5, None, None, None, 0,
                             None) == emr.EMR_E_INVAL
    assert L.emr_band_filter(None, None, 4, C.c_float(0.1), None, None) == emr.EMR_E_INVAL
    conn = emr.emr_connections(0, 0, 0, 0, 0, 0, 0)
    assert L.emr_band_filter(C.byref(conn), None, -1, C.c_float(0.1), C.byref(conn),
                             None) == emr.EMR_E_INVAL
