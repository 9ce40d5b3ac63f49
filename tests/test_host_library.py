"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, and its host metadata and page allocator agree bit for bit with the
oracle's (no GPU calls)."""
import json
import os
import re

import numpy as np
import pytest

from oracle import meta
from paper_2609_01068_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "outlets.h")


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(outlets_\w+)\s*\(", src, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2609_01068_amd import build
        build.build(verbose=False)
    return B.lib()


def test_library_exports_every_declared_symbol(lib):
    names = header_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(names) == sorted(B.exported_names())


def test_header_is_plain_c():
    src = open(HEADER).read()
    assert 'extern "C"' in src
    for banned in ("torch", "at::", "std::", "hip_runtime", "#ifdef __HIP"):
        assert banned not in src


def test_varlen_meta_matches_oracle(lib):
    r = np.random.default_rng(3)
    for _ in range(100):
        lens = r.integers(1, 300, size=r.integers(1, 40))
        cu, pos, last = B.outlets_varlen_meta(lens)
        assert np.array_equal(cu, meta.cu_seqlens(lens))
        assert np.array_equal(pos, meta.positions(lens))
        assert np.array_equal(last, meta.last_idx(lens))


def test_varlen_meta_rejects_empty_prompt(lib):
    with pytest.raises(B.OutletsError) as e:
        B.outlets_varlen_meta([3, 0, 2])
    assert e.value.rc == B.OUTLETS_ERR_INVALID_ARG


def _check_decode_plan(pages, n_kv, cus):
    """The plan's defining properties: the step's pages (requests in order)
    cut into L contiguous ranges of equal length (+-1); each range's part in
    one request is one segment; segments numbered in page order; pieces of
    at most 64 pages cover every page exactly once."""
    work, cu, lanes = B.outlets_decode_plan(pages, n_kv, cus)
    n, P = len(pages), int(sum(pages))
    L = len(lanes) - 1
    assert 1 <= L <= max(1, 8 * cus // n_kv) and L <= max(1, -(-P // 16))
    assert lanes[0] == 0 and lanes[-1] == len(work) and all(a <= b for a, b in zip(lanes, lanes[1:]))
    start = np.concatenate([[0], np.cumsum(pages)])
    covered = np.zeros(P, dtype=np.int64)
    seg_req, seg_pages = {}, {}
    for ln in range(L):
        lo, hi = P * ln // L, P * (ln + 1) // L
        pos = lo
        for (r, p0, p1, s) in work[lanes[ln]:lanes[ln + 1]]:
            assert 0 <= r < n and 0 <= p0 < p1 <= pages[r] and p1 - p0 <= 64
            assert start[r] + p0 == pos, "pieces of a range are contiguous and in order"
            covered[start[r] + p0:start[r] + p1] += 1
            pos = start[r] + p1
            assert seg_req.setdefault(s, (r, ln)) == (r, ln), "a segment is one request within one range"
            seg_pages.setdefault(s, []).append((p0, p1))
        assert pos == hi
    assert np.all(covered == 1)
    n_segs = len(seg_req)
    assert sorted(seg_req) == list(range(n_segs)) and n_segs <= L + n
    # segments in page order: request-major, consecutive per request
    assert [seg_req[s][0] for s in range(n_segs)] == sorted(seg_req[s][0] for s in range(n_segs))
    assert cu[0] == 0 and cu[-1] == n_segs
    for r in range(n):
        segs = [s for s in range(n_segs) if seg_req[s][0] == r]
        assert segs == list(range(cu[r], cu[r + 1])) and segs
    # a range holds as many segments as requests it touches
    for ln in range(L):
        lo, hi = P * ln // L, P * (ln + 1) // L
        touched = np.unique(np.searchsorted(start, np.arange(lo, hi), side="right") - 1)
        assert len({s for (_, _, _, s) in work[lanes[ln]:lanes[ln + 1]]}) == len(touched)
    assert len(work) <= P // 64 + n_segs
    return work, cu, lanes


def test_decode_plan_ranges_segments_and_pieces(lib):
    r = np.random.default_rng(11)
    cases = [([1], 8, 256), ([3, 1, 2], 8, 256), ([600] * 3, 8, 256), ([1] * 700, 8, 256),
             ([1000, 1, 1, 513], 1, 4), ([64, 65, 127, 128, 129], 2, 16)]
    for _ in range(40):
        n = int(r.integers(1, 300))
        cases.append((list(r.integers(1, 600, size=n)), int(r.choice([1, 2, 8])), int(r.choice([1, 4, 80, 256]))))
    for pages, n_kv, cus in cases:
        _check_decode_plan(pages, n_kv, cus)


def test_decode_plan_at_the_512_request_step_shape(lib):
    # caches of U[256, 8192] tokens plus the new one, 16-token pages
    r = np.random.default_rng(5)
    pages = [(int(x) + 1 + 15) // 16 for x in r.integers(256, 8193, size=512)]
    work, cu, lanes = _check_decode_plan(pages, 8, 256)
    assert len(lanes) - 1 == 256
    assert cu[-1] <= 256 + 512


def test_decode_plan_rejects_bad_sizes(lib):
    for pages in ([], [2, 0, 1], [-3]):
        with pytest.raises(B.OutletsError) as e:
            B.outlets_decode_plan(pages, 8, 256)
        assert e.value.rc == B.OUTLETS_ERR_INVALID_ARG


def _compare(p, o):
    assert p.read(B.OUTLETS_META_PAGE_TABLE) == list(o.table().reshape(-1))
    assert p.read(B.OUTLETS_META_SEQ_LEN) == list(o.seq_lens())


def test_pager_worked_example_matches(lib):
    with open(os.path.join(ROOT, "tests", "golden", "page_alloc_example.json")) as f:
        ex = json.load(f)
    init = ex["init"]
    p = B.Pager(init["num_pages"], init["page_size"], init["max_slots"], init["max_seq_len"])
    o = meta.PageAllocator(**init)
    for op in ex["ops"]:
        if op["op"] == "prefill":
            rc, ro = p.prefill(op["slots"], op["lens"]), o.prefill(op["slots"], op["lens"])
        elif op["op"] == "step":
            rc, ro = p.step(op["slots"]), o.step(op["slots"])
        else:
            rc, ro = p.release(op["slots"]), o.release(op["slots"])
        assert rc == ro == op["rc"], op
        _compare(p, o)


def test_pager_random_sequences_match_oracle(lib):
    r = np.random.default_rng(11)
    for trial in range(8):
        ps = 16
        num_pages, slots_n, max_seq = int(r.integers(8, 200)), int(r.integers(2, 12)), int(r.integers(20, 400))
        p = B.Pager(num_pages, ps, slots_n, max_seq)
        o = meta.PageAllocator(num_pages, ps, slots_n, max_seq)
        for _ in range(300):
            kind = r.integers(0, 3)
            k = int(r.integers(0, 4))
            slots = list(r.integers(-1, slots_n + 1, size=k))     # includes bad and repeated slots
            if kind == 0:
                lens = list(r.integers(-1, max_seq + 2, size=k))
                assert p.prefill(slots, lens) == o.prefill(slots, lens)
            elif kind == 1:
                assert p.step(slots) == o.step(slots)
            else:
                assert p.release(slots) == o.release(slots)
            _compare(p, o)
        p.close()


def test_pager_error_codes_leave_state_unchanged(lib):
    p = B.Pager(6, 4, 4, 16)
    assert p.prefill([0, 1], [5, 4]) == B.OUTLETS_OK
    before = (p.read(0), p.read(1))
    assert p.prefill([2, 2], [1, 1]) == B.OUTLETS_ERR_INVALID_ARG
    assert p.prefill([2, 0], [1, 1]) == B.OUTLETS_ERR_SLOT_BUSY
    assert p.prefill([2, 3], [8, 9]) == B.OUTLETS_ERR_OUT_OF_PAGES
    assert p.step([3]) == B.OUTLETS_ERR_SLOT_EMPTY
    assert p.release([9]) == B.OUTLETS_ERR_INVALID_ARG
    assert (p.read(0), p.read(1)) == before
    assert "slot" in B.last_error() or "range" in B.last_error()
