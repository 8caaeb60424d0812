"""Failure injection for the C block manager, forced from the host: every error leaves the state
unchanged and reports the documented code."""
import ctypes

import numpy as np
import pytest

import paper_2609_39334_amd as tkv


def _same(a, b):
    for k in ("refcount", "block_len", "indexed"):
        np.testing.assert_array_equal(a[k], b[k])
    assert a["seqs"] == b["seqs"]


def _bm():
    bm = tkv.BlockManager(10, 4, 4)
    p, _, _ = bm.extend(-1, [1, 2, 3, 4, 5], True)       # blocks 0, 1
    c, _, _ = bm.extend(p, [6, 7], False)                  # block 2, unsealed
    return bm, p, c


def test_pool_exhaustion_is_atomic():
    bm, p, _ = _bm()
    before = bm.snapshot()
    with pytest.raises(tkv.TkvError) as e:
        bm.extend(p, list(range(100, 129)), True)        # 8 blocks > 7 free
    assert e.value.code == tkv.TKV_ENOMEM
    _same(before, bm.snapshot())
    # a partial hit prefix does not change the need: the same step as a prefix hit + misses
    s, blocks, hits = bm.extend(p, list(range(100, 124)), True)   # 6 blocks fit
    assert list(hits) == [0] * 6


def test_sequence_slots_exhausted():
    bm, p, _ = _bm()
    bm.extend(p, [9], True)
    bm.extend(p, [10], True)
    before = bm.snapshot()
    with pytest.raises(tkv.TkvError) as e:
        bm.extend(p, [11], True)
    assert e.value.code == tkv.TKV_ENOMEM
    _same(before, bm.snapshot())


def test_unknown_and_double_prune():
    bm, p, c = _bm()
    before = bm.snapshot()
    for s in (3, -1, 99):
        with pytest.raises(tkv.TkvError) as e:
            bm.prune(s)
        assert e.value.code == tkv.TKV_ENOSEQ
    _same(before, bm.snapshot())
    bm.prune(c)
    with pytest.raises(tkv.TkvError) as e:
        bm.prune(c)
    assert e.value.code == tkv.TKV_ENOSEQ


def test_extend_from_unsealed_parent_or_dead_parent():
    bm, p, c = _bm()
    before = bm.snapshot()
    with pytest.raises(tkv.TkvError) as e:
        bm.extend(c, [1], True)
    assert e.value.code == tkv.TKV_EINVAL
    with pytest.raises(tkv.TkvError) as e:
        bm.extend(3, [1], True)
    assert e.value.code == tkv.TKV_ENOSEQ
    with pytest.raises(tkv.TkvError) as e:
        bm.extend(-1, [], True)
    assert e.value.code == tkv.TKV_EINVAL
    _same(before, bm.snapshot())


def test_capacity_errors_report_needed_size():
    bm, p, c = _bm()
    L = tkv.lib()
    before = bm.snapshot()
    toks = (ctypes.c_int32 * 9)(*range(9))
    child, n = ctypes.c_int32(), ctypes.c_int32()
    blk = (ctypes.c_int32 * 2)()
    hit = (ctypes.c_uint8 * 2)()
    rc = L.tkv_bm_extend(bm.h, p, toks, 9, 1, ctypes.byref(child), blk, hit, 2, ctypes.byref(n))
    assert rc == tkv.TKV_ECAP and n.value == 3
    rc = L.tkv_bm_extend(bm.h, p, toks, 9, 2, ctypes.byref(child), blk, hit, 2, ctypes.byref(n))
    assert rc == tkv.TKV_EINVAL
    freed = (ctypes.c_int32 * 1)()
    rc = L.tkv_prune(bm.h, c, freed, 1, ctypes.byref(n))
    assert rc == tkv.TKV_ECAP and n.value == 3
    tab = (ctypes.c_int32 * 1)()
    kv = ctypes.c_int32()
    rc = L.tkv_bm_table(bm.h, c, tab, 1, ctypes.byref(n), ctypes.byref(kv))
    assert rc == tkv.TKV_ECAP and n.value == 3
    used = ctypes.c_size_t()
    rc = L.tkv_bm_snapshot(bm.h, None, 0, ctypes.byref(used))
    assert rc == tkv.TKV_ECAP and used.value > 0
    assert "capacity" in tkv.tkv_last_error() or "NULL" in tkv.tkv_last_error() or tkv.tkv_last_error()
    _same(before, bm.snapshot())


def test_bad_create_and_refcount_range():
    with pytest.raises(tkv.TkvError) as e:
        tkv.tkv_bm_create(0, 16, 4)
    assert e.value.code == tkv.TKV_EINVAL
    bm, _, _ = _bm()
    with pytest.raises(tkv.TkvError):
        tkv.tkv_bm_refcount(bm.h, 10)
    assert tkv.tkv_bm_refcount(bm.h, 0) == 2


def test_coalesce_rejects_dead_sequences_and_bad_q_len():
    bm, p, c = _bm()
    with pytest.raises(tkv.TkvError) as e:
        bm.coalesce([p, 3], [1, 1])
    assert e.value.code == tkv.TKV_ENOSEQ
    with pytest.raises(tkv.TkvError) as e:
        bm.coalesce([p], [0])
    assert e.value.code == tkv.TKV_EINVAL


def test_append_errors_leave_state_unchanged():
    bm, p, c = _bm()                                       # c: open step of 2 tokens in block 2; 7 blocks free
    before = bm.snapshot()
    with pytest.raises(tkv.TkvError) as e:
        bm.append(c, list(range(31)))                      # 2 slots left, then 29 tokens = 8 blocks > 7
    assert e.value.code == tkv.TKV_ENOMEM
    _same(before, bm.snapshot())
    for s in (3, -1, 99):
        with pytest.raises(tkv.TkvError) as e:
            bm.append(s, [1])
        assert e.value.code == tkv.TKV_ENOSEQ
    _same(before, bm.snapshot())
    L = tkv.lib()
    toks = np.arange(5, dtype=np.int32)
    dst = np.zeros(5, dtype=np.int32)
    rc = L.tkv_bm_append(bm.h, c, toks.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), 5,
                         dst.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), 4)
    assert rc == tkv.TKV_ECAP
    _same(before, bm.snapshot())
    assert bm.append(c, list(range(30))).tolist()[:2] == [2 * 4 + 2, 2 * 4 + 3]   # 30 tokens fit


def test_seal_errors_leave_state_unchanged():
    bm, p, c = _bm()
    bm.append(c, [8, 9, 10])                               # open step: blocks 2 (full) and 3
    before = bm.snapshot()
    with pytest.raises(tkv.TkvError) as e:
        bm.seal(p)                                         # already sealed
    assert e.value.code == tkv.TKV_EINVAL
    L = tkv.lib()
    n = ctypes.c_int32()
    out = np.zeros(2, dtype=np.int32)
    rc = L.tkv_bm_seal(bm.h, c, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), 1, ctypes.byref(n))
    assert rc == tkv.TKV_ECAP and n.value == 2             # two open blocks need room for two pairs
    _same(before, bm.snapshot())
    assert bm.seal(c) == [] and bm.snapshot()["seqs"][c][1:] == (1, 0)
    with pytest.raises(tkv.TkvError) as e:
        bm.seal(c)
    assert e.value.code == tkv.TKV_EINVAL


def test_fork_errors_leave_state_unchanged():
    bm, p, c = _bm()                                       # 7 blocks and 2 sequence slots free
    before = bm.snapshot()
    with pytest.raises(tkv.TkvError) as e:
        bm.fork(c, [1, 2, 3])                              # 3 children, 2 sequence slots
    assert e.value.code == tkv.TKV_ENOMEM
    _same(before, bm.snapshot())                           # the open step was not sealed either
    with pytest.raises(tkv.TkvError) as e:
        bm.fork(9, [1])
    assert e.value.code == tkv.TKV_ENOSEQ
    _same(before, bm.snapshot())
    kids = bm.fork(c, [5, 6])
    snap = bm.snapshot()["seqs"]
    assert snap[c][1] == 1 and all(snap[k][1:] == (0, 1) for k in kids)
