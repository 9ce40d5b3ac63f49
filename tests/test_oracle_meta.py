"""Pins of the oracle's integer metadata and page allocator (CPU only).

The expected tables in the worked example were derived by hand from the
allocation rule (lowest free page first, requests in argument order, a step
takes a page when the cached length is a multiple of the page size); the
random-sequence test checks the invariants any valid allocator must keep.
"""
import json
import os

import numpy as np

from oracle import meta

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_varlen_closed_forms():
    r = np.random.default_rng(0)
    for _ in range(50):
        lens = r.integers(1, 40, size=r.integers(1, 12))
        cu = meta.cu_seqlens(lens)
        assert cu[0] == 0 and len(cu) == len(lens) + 1
        for i in range(len(lens)):
            assert cu[i + 1] - cu[i] == lens[i]
        pos = meta.positions(lens)
        last = meta.last_idx(lens)
        for i, n in enumerate(lens):
            assert list(pos[cu[i]:cu[i + 1]]) == list(range(n))
            assert last[i] == cu[i] + n - 1 and pos[last[i]] == n - 1
        start = r.integers(0, 100, size=len(lens))
        pos2 = meta.positions(lens, start)
        assert np.array_equal(pos2 - np.repeat(start, lens), pos)


def test_page_allocator_worked_example():
    with open(os.path.join(GOLDEN, "page_alloc_example.json")) as f:
        ex = json.load(f)
    a = meta.PageAllocator(**ex["init"])
    for op in ex["ops"]:
        kind = op["op"]
        if kind == "prefill":
            rc = a.prefill(op["slots"], op["lens"])
        elif kind == "step":
            rc = a.step(op["slots"])
        else:
            rc = a.release(op["slots"])
        assert rc == op["rc"], op
        if "pages" in op:
            for slot, pages in op["pages"].items():
                assert a.pages[int(slot)] == pages, (op, slot)
        if "seq_len" in op:
            for slot, n in op["seq_len"].items():
                assert a.seq_len[int(slot)] == n
        if "n_free" in op:
            assert a.n_free() == op["n_free"]


def _snapshot(a):
    return (a.table().copy(), a.seq_lens().copy(), sorted(a.free), list(a.active))


def test_failed_calls_leave_state_unchanged():
    a = meta.PageAllocator(num_pages=6, page_size=4, max_slots=4, max_seq_len=16)
    assert a.prefill([0, 1], [5, 4]) == meta.OK             # pages 0,1 | 2
    before = _snapshot(a)
    assert a.prefill([2, 2], [1, 1]) == meta.ERR_INVALID_ARG   # repeated slot
    assert a.prefill([2], [0]) == meta.ERR_INVALID_ARG         # empty prompt
    assert a.prefill([2], [17]) == meta.ERR_INVALID_ARG        # longer than max
    assert a.prefill([4], [1]) == meta.ERR_INVALID_ARG         # slot out of range
    assert a.prefill([2, 0], [1, 1]) == meta.ERR_SLOT_BUSY
    assert a.prefill([2, 3], [8, 9]) == meta.ERR_OUT_OF_PAGES  # needs 2 + 3 > 3 free
    assert a.step([3]) == meta.ERR_SLOT_EMPTY
    assert a.step([0, 0]) == meta.ERR_INVALID_ARG
    assert a.release([5]) == meta.ERR_INVALID_ARG
    after = _snapshot(a)
    for x, y in zip(before, after):
        assert np.array_equal(np.asarray(x), np.asarray(y))


def test_random_operation_sequences_keep_invariants():
    r = np.random.default_rng(1)
    ps = 16
    a = meta.PageAllocator(num_pages=64, page_size=ps, max_slots=8, max_seq_len=200)
    for _ in range(400):
        kind = r.integers(0, 3)
        slots = list(r.choice(8, size=r.integers(1, 4), replace=False))
        if kind == 0:
            a.prefill(slots, list(r.integers(1, 200, size=len(slots))))
        elif kind == 1:
            a.step(slots)
        else:
            a.release(slots)
        used = [p for s in range(8) for p in a.pages[s]]
        assert len(used) == len(set(used))                       # no page shared
        assert sorted(used + list(a.free)) == list(range(64))    # nothing lost
        for s in range(8):
            assert len(a.pages[s]) == meta.pages_for(a.seq_len[s], ps)
            assert a.active[s] == (a.seq_len[s] > 0)
