"""The host's placement of a discover launch's chunks on its waves (longest processing time first):
every chunk exactly once, lists in assignment order, and the greedy rule's load bound. Host only."""

import ctypes as C

import numpy as np
import pytest

from paper_2608_27612_amd import emr

NO_CHUNK = 0xFFFFFFFF


def lpt(cost, waves, key=None, domain_waves=0, domains=1, n_keys=None):
    lib = C.CDLL(emr.LIB_PATH)
    f = lib.emr_lpt_schedule
    f.restype = C.c_int
    f.argtypes = [C.c_void_p, C.c_void_p, C.c_uint32, C.c_uint32, C.c_uint32, C.c_uint32,
                  C.c_uint32, C.c_void_p, C.c_uint64, C.POINTER(C.c_uint32)]
    cost = np.ascontiguousarray(cost, dtype=np.float32)
    kp, nk = None, 0
    if key is not None:
        key = np.ascontiguousarray(key, dtype=np.uint32)
        kp, nk = key.ctypes.data, int(key.max()) + 1 if len(key) else 0
        if n_keys is not None:
            nk = n_keys
    stride = C.c_uint32(0)
    args = (cost.ctypes.data, kp, nk, len(cost), waves, domain_waves, domains)
    rc = f(*args, None, 0, C.byref(stride))
    if rc < 0:
        return rc, None
    assert rc == 1 and stride.value % 64 == 0 and stride.value >= 64
    table = np.empty(waves * stride.value, dtype=np.uint32)
    assert f(*args, table.ctypes.data, table.size - 1, C.byref(stride)) == 1  # one short: refused
    assert f(*args, table.ctypes.data, table.size, C.byref(stride)) == 0
    return 0, table.reshape(waves, stride.value)


def brute_lpt(cost, waves):
    """The rule restated: costliest chunk first (equal costs by index), to the least loaded wave
    (equal loads: the lowest wave)."""
    load = [0.0] * waves
    lists = [[] for _ in range(waves)]
    for c in sorted(range(len(cost)), key=lambda c: (-float(np.float32(cost[c])), c)):
        w = min(range(waves), key=lambda w: (load[w], w))
        lists[w].append(c)
        load[w] += float(np.float32(cost[c]))
    return lists


@pytest.mark.parametrize("n,waves,seed", [(0, 4, 0), (1, 4, 1), (7, 3, 2), (200, 16, 3),
                                          (1000, 64, 4), (130, 1, 5)])
def test_schedule_is_a_permutation_and_matches_the_rule(n, waves, seed):
    rng = np.random.default_rng(seed)
    cost = rng.lognormal(3.0, 1.5, n).astype(np.float32)
    if n > 10:
        cost[::7] = cost[3]  # ties
    rc, t = lpt(cost, waves)
    assert rc == 0
    ids = t[t != NO_CHUNK]
    assert sorted(ids.tolist()) == list(range(n))
    for w in range(waves):
        row = t[w]
        k = int(np.sum(row != NO_CHUNK))
        assert (row[k:] == NO_CHUNK).all()  # padding only after the list
    want = brute_lpt(cost, waves)
    for w in range(waves):
        got = [int(c) for c in t[w] if c != NO_CHUNK]
        assert got == want[w], w


def test_schedule_load_bound():
    # each wave's load stays within the mean plus the largest chunk (greedy list scheduling)
    rng = np.random.default_rng(7)
    for n, waves in [(5000, 300), (15774, 3072), (100, 200)]:
        cost = rng.lognormal(4.0, 1.2, n).astype(np.float32)
        rc, t = lpt(cost, waves)
        assert rc == 0
        load = np.array([cost[r[r != NO_CHUNK]].astype(np.float64).sum() for r in t])
        assert load.max() <= cost.sum() / waves + cost.max() + 1e-3 * cost.max()


def test_domains_keep_keys_together_and_balance():
    # 8 domains of 4-wave workgroups (wave w in domain (w // 4) % 8); a key's chunks share one
    # domain, each domain is balanced per wave within its largest key, and each domain's chunks
    # follow the one-level rule over its own waves
    rng = np.random.default_rng(11)
    n_groups, per = 400, 11
    gcost = rng.lognormal(3.0, 0.4, n_groups)  # no group above a tenth of a domain's load
    key = np.repeat(np.arange(n_groups), per)
    cost = (np.repeat(gcost, per) * rng.uniform(0.9, 1.1, key.size)).astype(np.float32)
    waves = 4 * 96
    rc, t = lpt(cost, waves, key, 4, 8)
    assert rc == 0
    ids = t[t != NO_CHUNK]
    assert sorted(ids.tolist()) == list(range(cost.size))
    dom_of_wave = (np.arange(waves) // 4) % 8
    dom_of_chunk = np.empty(cost.size, dtype=np.int64)
    for w in range(waves):
        for c in t[w][t[w] != NO_CHUNK]:
            dom_of_chunk[c] = dom_of_wave[w]
    for g in range(n_groups):
        assert len(set(dom_of_chunk[key == g].tolist())) == 1, g
    key_total = np.bincount(key, weights=cost.astype(np.float64))
    dload = np.bincount(dom_of_chunk, weights=cost.astype(np.float64), minlength=8) / (waves / 8)
    assert dload.max() <= dload.mean() + key_total.max() / (waves / 8) + 1e-6
    for d in range(8):
        ws = np.nonzero(dom_of_wave == d)[0]
        mine = np.nonzero(dom_of_chunk == d)[0]
        want = brute_lpt(cost[mine], len(ws))
        for i, w in enumerate(ws):
            got = [int(c) for c in t[w] if c != NO_CHUNK]
            assert got == [int(mine[j]) for j in want[i]]


def test_schedule_rejects_bad_input():
    assert lpt(np.ones(3), 0)[0] == -1
    assert lpt(np.ones(3), 8, None, 4, 2)[0] == -1           # domains without keys
    assert lpt(np.ones(3), 8, np.zeros(3), 4, 4)[0] == -1    # 4 domains of 4 waves > 8 waves
    assert lpt(np.ones(3), 8, np.array([0, 1, 2]), 2, 2, n_keys=2)[0] == -1  # key out of range
    assert lpt(np.array([1.0, np.nan]), 2)[0] == -1
    assert lpt(np.array([1.0, -1.0]), 2)[0] == -1
    assert lpt(np.array([1.0, np.inf]), 2)[0] == -1


def test_few_large_keys_use_all_waves():
    # 4 keys (a call with 4 groups) over 8 domains: one domain per key would idle half the waves,
    # so the placement uses every wave (the one-level rule)
    rng = np.random.default_rng(21)
    key = np.repeat(np.arange(4), 500)
    cost = rng.uniform(90, 110, key.size).astype(np.float32)
    waves = 4 * 64
    rc, t = lpt(cost, waves, key, 4, 8)
    assert rc == 0
    assert (t[:, 0] != NO_CHUNK).all()  # every wave has work
    want = brute_lpt(cost, waves)
    for w in range(waves):
        assert [int(c) for c in t[w] if c != NO_CHUNK] == want[w]
