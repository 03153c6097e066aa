"""Host logic of bench.py's overlapped schedule, on the CPU: the Unique calls
of later steps run on a second stream while earlier steps' Seg-Sum and update
run on the first, in groups of steps over two halves of the sets of Unique
outputs. A recording stand-in for the streams and events checks that every
ordering the events allow keeps each step on its own set and never lets a
Unique overwrite a set that an earlier step still reads."""
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


class Rec:
    """Streams as op lists in host issue order. A wait names the last record
    of its event issued before it on the host (HIP's rule; a wait on an
    event never recorded would not wait at all, so the test rejects it)."""

    def __init__(self):
        self.ops = {"main": [], "side": []}
        self.last = {}  # event -> (stream, index of its latest record op)

    def record(self, i, stream):
        self.last[i] = (stream, len(self.ops[stream]))
        self.ops[stream].append(("record", i))

    def wait(self, i, stream):
        assert i in self.last, f"wait on event {i} before any record of it"
        self.ops[stream].append(("wait", i, self.last[i]))

    def front(self, b, j, stream):
        self.ops[stream].append(("front", b, j))

    def back(self, b, j):
        self.ops["main"].append(("back", b, j))


def _schedule(nsets, steps, first=0):
    rec = Rec()
    pipe = object.__new__(bench.Pipeline)
    pipe.sets = [(f"set{j}", None) for j in range(nsets)]
    pipe.front, pipe.back = rec.front, rec.back
    pipe.run_overlapped(first, steps, None, "main", "side", rec)
    return rec.ops


def _earliest_times(ops):
    """Earliest start and end of every op when each takes one time unit
    after the previous op of its stream and a wait ends no earlier than the
    record it names. Returns {(stream, index): (start, end)}."""
    t = {}
    done = {"main": 0, "side": 0}
    progress = True
    while progress:
        progress = False
        for s in ("main", "side"):
            while done[s] < len(ops[s]):
                k = done[s]
                op = ops[s][k]
                start = t[(s, k - 1)][1] if k else 0
                if op[0] == "wait":
                    if op[2] not in t:
                        break  # the record it names is not placed yet
                    start = max(start, t[op[2]][1])
                t[(s, k)] = (start, start + 1)
                done[s] += 1
                progress = True
    assert all(done[s] == len(ops[s]) for s in ops), "the waits deadlock"
    return t


@pytest.mark.parametrize("nsets,steps", [(2, 1), (2, 7), (4, 2), (4, 3), (4, 7), (4, 200),
                                         (6, 7), (16, 5), (16, 37), (16, 200)])
def test_overlapped_schedule_orders_the_streams(nsets, steps):
    ops = _schedule(nsets, steps, first=5)
    fronts = [op for op in ops["side"] if op[0] == "front"]
    backs = [op for op in ops["main"] if op[0] == "back"]
    # every step once, in order, each on set (step - first) % nsets
    assert [op[1] for op in fronts] == list(range(5, 5 + steps))
    assert [op[1] for op in backs] == list(range(5, 5 + steps))
    assert all(op[2] == (op[1] - 5) % nsets for op in fronts + backs)
    # each event is recorded once, on one stream
    recs = [op[1] for s in ops for op in ops[s] if op[0] == "record"]
    assert len(set(recs)) == len(recs)
    t = _earliest_times(ops)
    span = {ops[s][k][:2]: v for (s, k), v in t.items() if ops[s][k][0] in ("front", "back")}
    for i in range(5, 5 + steps):
        # Seg-Sum and the update of step i start after its Unique ended
        assert span[("back", i)][0] >= span[("front", i)][1]
        # a Unique that reuses step i's set starts after step i ended
        j = i + nsets
        if ("front", j) in span:
            assert span[("front", j)][0] >= span[("back", i)][1]


def test_overlapped_schedule_lets_unique_run_ahead():
    """With groups of two steps (four sets) the side stream runs group 1's
    Unique calls before it first waits for the main one, and then waits
    once per group, for the group two before."""
    ops = _schedule(4, 8)
    side_waits = [op for op in ops["side"] if op[0] == "wait"]
    # the start event, then one wait before each of groups 2 and 3
    assert [op[1] for op in side_waits] == [0, 2, 4]
    assert ops["side"].index(("front", 3, 3)) < ops["side"].index(side_waits[1])
    assert ops["side"].index(side_waits[1]) < ops["side"].index(("front", 4, 0))


@pytest.mark.parametrize("nsets,steps", [(4, 8), (16, 37), (16, 8), (2, 5)])
def test_overlapped_schedule_meets_once_per_group(nsets, steps):
    """The main stream waits once per group of nsets / 2 steps (the last
    group may be short), and never between two steps of one group."""
    G = nsets // 2
    ops = _schedule(nsets, steps)
    main = ops["main"]
    waits = [k for k, op in enumerate(main) if op[0] == "wait"]
    assert len(waits) == (steps + G - 1) // G
    for k in waits:
        nxt = next(op for op in main[k + 1:] if op[0] == "back")
        assert nxt[1] % G == 0  # a group's first step follows each wait


def test_overlapped_schedule_rejects_odd_sets():
    with pytest.raises(ValueError):
        _schedule(3, 4)


def test_cu_mask_words():
    """Bit c of the mask is CU c; the split's two ranges cover every CU once."""
    assert bench.cu_mask_words(0, 32, 256) == [0xFFFFFFFF] + [0] * 7
    assert bench.cu_mask_words(32, 224, 256) == [0] + [0xFFFFFFFF] * 7
    assert bench.cu_mask_words(3, 2, 40) == [0b11000, 0]
    for n in bench.SIDE_CUS.values():
        side = bench.cu_mask_words(0, n, 256)
        main = bench.cu_mask_words(n, 256 - n, 256)
        assert all(a & b == 0 and a | b == 0xFFFFFFFF for a, b in zip(side, main))
        assert n % 32 == 0
    with pytest.raises(ValueError):
        bench.cu_mask_words(250, 8, 256)
    with pytest.raises(ValueError):
        bench.cu_mask_words(0, 0, 256)
