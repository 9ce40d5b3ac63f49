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
