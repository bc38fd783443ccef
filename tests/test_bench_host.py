"""The benchmark's pipelined steps (host logic only): with depth + 1 calls in flight every call is
checked exactly once, in call order, after the calls it overlaps have been enqueued, and no result
buffer is enqueued again before the check of the call that last used it."""

import types

import pytest

import bench


class _Cuda:
    @staticmethod
    def synchronize():
        pass


_TORCH = types.SimpleNamespace(cuda=_Cuda())


@pytest.mark.parametrize("depth", [0, 1, 2, 3, 5])
@pytest.mark.parametrize("steps", [1, 2, 3, 4, 7, 10])
def test_pipelined_steps_check_every_call_once_and_never_reuse_a_busy_buffer(steps, depth):
    log = []

    def enqueue(i):
        log.append(("enqueue", i))

    def check(i):
        log.append(("check", i))

    bench.pipelined_steps(_TORCH, enqueue, check, steps, 0, depth)
    enq = [i for k, i in log if k == "enqueue"]
    chk = [i for k, i in log if k == "check"]
    assert enq == list(range(steps)) and chk == list(range(steps))
    pos = {e: n for n, e in enumerate(log)}
    nbuf = depth + 1
    for i in range(steps):
        # the call is checked only after the calls up to i + depth are enqueued
        last = min(i + depth, steps - 1)
        assert pos[("check", i)] > pos[("enqueue", last)]
        # its buffer is enqueued again (call i + nbuf) only after its check
        if i + nbuf < steps:
            assert pos[("enqueue", i + nbuf)] > pos[("check", i)]
    # never more than depth + 1 calls between an enqueue and its check
    in_flight = 0
    for k, _ in log:
        in_flight += 1 if k == "enqueue" else -1
        assert 0 <= in_flight <= nbuf


def test_warmup_runs_its_own_calls_first():
    log = []
    bench.pipelined_steps(_TORCH, lambda i: log.append(("e", i)), lambda i: log.append(("c", i)),
                          3, 2, bench.IN_FLIGHT - 1)
    # the warm-up's two calls, then the three timed ones, each checked
    assert [x for x in log if x[0] == "e"] == [("e", 0), ("e", 1), ("e", 0), ("e", 1), ("e", 2)]
    assert sorted(i for k, i in log if k == "c") == [0, 0, 1, 1, 2]
