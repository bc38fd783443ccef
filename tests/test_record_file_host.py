"""Record files on the host (no GPU): the C sink writes deliveries in the documented layout, a
file cut inside a block resumes at its last whole delivery, and every misuse is refused with its
status."""

import ctypes as C
import os

import numpy as np
import pytest

from paper_2608_27612_amd import emr


def deliveries(seed, n_pairs, n_chunks):
    """Random deliveries in cursor order (chunk-major), some (chunk, pair) skipped as empty."""
    rng = np.random.default_rng(seed)
    out = []
    for chunk in range(n_chunks):
        for pair in range(n_pairs):
            if rng.random() < 0.3:
                continue
            n = int(rng.integers(1, 50))
            parent = np.sort(rng.choice(1 << 20, size=n, replace=False)).astype(np.uint32)
            w4 = rng.standard_normal((n, 4)).astype(np.float32)
            out.append((pair, chunk, parent, w4))
    return out


def sink(f, pair, chunk, parent, w4):
    parent = np.ascontiguousarray(parent, np.uint32)
    w4 = np.ascontiguousarray(w4, np.float32)
    return emr.lib().emr_record_file_sink(pair, chunk, parent.ctypes.data, w4.ctypes.data,
                                          len(parent), f.handle)


def same(blocks, expect):
    assert len(blocks) == len(expect)
    for (p, c, par, w), (ep, ec, epar, ew) in zip(blocks, expect):
        assert (p, c) == (ep, ec)
        assert np.array_equal(par, epar)
        assert np.array_equal(w.view(np.uint32), ew.view(np.uint32))


def test_write_read_round_trip(tmp_path):
    path = str(tmp_path / "a.rec")
    d = deliveries(1, 5, 7)
    f = emr.RecordFile(path, 5)
    assert f.cursor == 0
    for dl in d:
        assert sink(f, *dl) == 0
    recs, nxt = f.close()
    assert recs == sum(len(x[2]) for x in d)
    assert nxt == d[-1][1] * 5 + d[-1][0] + 1
    n_pairs, blocks = emr.read_record_file(path)
    assert n_pairs == 5
    same(blocks, d)
    assert os.path.getsize(path) == 32 + sum(24 + 20 * len(x[2]) for x in d)


@pytest.mark.parametrize("cut", [1, 10, 24, 30])
def test_resume_cuts_a_partial_block(tmp_path, cut):
    path = str(tmp_path / "b.rec")
    d = deliveries(2, 3, 6)
    with emr.RecordFile(path, 3, buffer_bytes=4096) as f:
        for dl in d:
            assert sink(f, *dl) == 0
    full = open(path, "rb").read()
    # a run that died while writing the last block: its bytes are cut short
    last = 24 + 20 * len(d[-1][2])
    cut = min(cut, last - 1)
    with open(path, "r+b") as fh:
        fh.truncate(len(full) - last + (last - cut))
    f = emr.RecordFile(path, 3, resume=True)
    expect_next = d[-2][1] * 3 + d[-2][0] + 1
    assert f.cursor == expect_next
    assert os.path.getsize(path) == len(full) - last
    assert sink(f, *d[-1]) == 0
    recs, nxt = f.close()
    assert open(path, "rb").read() == full
    assert nxt == d[-1][1] * 3 + d[-1][0] + 1
    assert recs == sum(len(x[2]) for x in d)


def test_resume_of_missing_or_whole_file(tmp_path):
    path = str(tmp_path / "c.rec")
    f = emr.RecordFile(path, 2, resume=True)
    assert f.cursor == 0
    assert f.close() == (0, 0)
    d = deliveries(3, 2, 3)
    with emr.RecordFile(path, 2, resume=True) as f:
        for dl in d:
            assert sink(f, *dl) == 0
    f = emr.RecordFile(path, 2, resume=True)
    assert f.cursor == d[-1][1] * 2 + d[-1][0] + 1
    f.close()
    same(emr.read_record_file(path)[1], d)
    # resume = 0 starts over
    f = emr.RecordFile(path, 2)
    assert f.close() == (0, 0)
    assert os.path.getsize(path) == 32


def test_refusals(tmp_path):
    path = str(tmp_path / "d.rec")
    d = deliveries(4, 4, 3)
    f = emr.RecordFile(path, 4)
    assert sink(f, *d[1]) == 0
    assert sink(f, *d[0]) == 1  # a cursor before the file's end
    assert sink(f, *d[2]) == 1  # every delivery after a refusal
    with pytest.raises(emr.EmrError) as e:
        f.close()
    assert e.value.status == emr.EMR_E_INVAL
    assert "precedes" in str(e.value)
    same(emr.read_record_file(path)[1], [d[1]])
    f = emr.RecordFile(path, 4, resume=True)
    p = np.zeros(1, np.uint32)
    w = np.zeros((1, 4), np.float32)
    assert sink(f, 4, 9, p, w) == 1  # pair outside n_pairs
    with pytest.raises(emr.EmrError) as e:
        f.close()
    assert e.value.status == emr.EMR_E_INVAL
    f = emr.RecordFile(path, 4, resume=True)
    assert emr.lib().emr_record_file_sink(0, 9, p.ctypes.data, w.ctypes.data, 0, f.handle) == 1
    with pytest.raises(emr.EmrError):
        f.close()
    assert emr.lib().emr_record_file_sink(0, 0, p.ctypes.data, w.ctypes.data, 1, None) == 1


def test_open_refusals(tmp_path):
    path = str(tmp_path / "e.rec")
    with emr.RecordFile(path, 3):
        pass
    for args, status in [((path, 4, True), emr.EMR_E_INVAL), ((path, 0, False), emr.EMR_E_INVAL),
                         ((str(tmp_path / "no" / "x.rec"), 3, False), emr.EMR_E_IO)]:
        with pytest.raises(emr.EmrError) as e:
            emr.RecordFile(*args)
        assert e.value.status == status, args
    with pytest.raises(emr.EmrError) as e:
        emr.RecordFile(path, 3, buffer_bytes=-1)
    assert e.value.status == emr.EMR_E_INVAL
    other = str(tmp_path / "f.rec")
    open(other, "wb").write(b"not a record file at all, nothing but text")
    with pytest.raises(emr.EmrError) as e:
        emr.RecordFile(other, 3, resume=True)
    assert e.value.status == emr.EMR_E_INVAL
    # a block that this sink could not have written (pair beyond n_pairs)
    bad = bytearray(open(path, "rb").read())
    bad += np.int64([7, 0, 1]).tobytes() + bytes(20)
    open(other, "wb").write(bytes(bad))
    with pytest.raises(emr.EmrError) as e:
        emr.RecordFile(other, 3, resume=True)
    assert e.value.status == emr.EMR_E_INVAL
    assert "malformed" in str(e.value)
    h = C.c_void_p()
    assert emr.lib().emr_record_file_open(None, 3, 0, 0, C.byref(h), None) == emr.EMR_E_INVAL
    assert emr.lib().emr_record_file_close(None, None, None) == emr.EMR_E_INVAL


@pytest.mark.skipif(not os.path.exists("/dev/full"), reason="no /dev/full")
def test_full_disk_is_an_io_error():
    with pytest.raises(emr.EmrError) as e:
        emr.RecordFile("/dev/full", 2)
    assert e.value.status == emr.EMR_E_IO
